"""The quantization kernels replace the per-element IEEE fp32 division x / s
by one correctly rounded reciprocal r = RN(1/s) per lane and two fmas per
element: q0 = RN(x r), rem = x - q0 s (exact), q = RN(q0 + rem r).  Because
s is a binary16 value (at most 11 significant bits) this q equals RN(x / s)
for every binary32 x (Markstein's correction step; the margin argument is in
csrc/quantize.hip).  These tests check the identity on the CPU:
exhaustively over all binary16 operand pairs the activation and weight
quantizers can see, and over every binary16 scale with random and
near-midpoint numerators for the KV4 quantizer."""
import os
import subprocess

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))


@pytest.fixture(scope="module")
def checker(tmp_path_factory):
    exe = str(tmp_path_factory.mktemp("divrn") / "div_rn_check")
    subprocess.run(["gcc", "-std=c11", "-O2", "-ffp-contract=off", "-fno-fast-math", "-o", exe,
                    os.path.join(HERE, "arith", "div_rn_check.c"), "-lm"], check=True)
    return exe


@pytest.mark.parametrize("mode", ["fp16", "kv"])
def test_reciprocal_division_is_exact(checker, mode):
    r = subprocess.run([checker, mode], capture_output=True, text=True, timeout=600)
    print(r.stdout)
    assert r.returncode == 0, r.stdout + r.stderr
    assert " 0 mismatches" in r.stdout
