"""The quantization kernels replace the per-element IEEE fp32 division x / s
by one reciprocal r per lane and two fmas per element: q0 = RN(x r),
rem = x - q0 s (exact), q = RN(q0 + rem r).  r may be RN(1/s) or either
binary32 neighbour of it (the hardware reciprocal is within one ulp of 1/s);
the scale itself, RN(amax / qmax), is computed the same way with r = RN(1/qmax).  Because
s is a binary16 value (at most 11 significant bits) this q equals RN(x / s)
for every binary32 x (Markstein's correction step; the margin argument is in
csrc/fmpq.h).  These tests check the identity on the CPU:
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


@pytest.mark.parametrize("mode", ["fp16", "kv", "qmax"])
def test_reciprocal_division_is_exact(checker, mode):
    r = subprocess.run([checker, mode], capture_output=True, text=True, timeout=600)
    print(r.stdout)
    assert r.returncode == 0, r.stdout + r.stderr
    assert " 0 mismatches" in r.stdout


@pytest.mark.parametrize("mode", ["fp16", "kv"])
def test_reciprocal_within_one_ulp_suffices(checker, mode):
    # the kernels take r from the hardware reciprocal (at most one ulp from
    # 1/s): the identity must hold for both binary32 neighbours of RN(1/s)
    r = subprocess.run([checker, mode, "nbr"], capture_output=True, text=True, timeout=900)
    print(r.stdout)
    assert r.returncode == 0, r.stdout + r.stderr
    assert " 0 mismatches" in r.stdout
