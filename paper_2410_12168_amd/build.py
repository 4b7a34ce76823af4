"""Build libcomet.so (gfx950) in-tree with hipcc.

Every HIP source is compiled for gfx950 only, with packed-fp32 instructions
disabled, IEEE fp32 division and square root, fp32 denormals kept, and no
floating-point contraction (fused multiply-adds are written explicitly).

The library carries a stamp: the SHA-256 of its sources (csrc/, the public
header) and of the compiler flags below, as the string
``COMET_SOURCE_STAMP=<hex>`` in its data and from ``comet_build_stamp()``.
``source_stamp()`` recomputes it from the tree, so a loader can tell a library
built from other sources before it loads it.
"""
import hashlib
import os
import re
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
OUT_DIR = os.path.join(HERE, "_build")
LIB = os.path.join(HERE, "libcomet.so")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

SOURCES = ["quantize.hip", "gemm.hip", "gemm_skinny.hip", "kv4.hip", "noalloc.hip", "scheduler.cpp",
           "calib.cpp", "comet_api.cpp"]

# The GEMM's inner loop interleaves MFMAs with the dequantization FMAs: keep
# MFMA results in VGPRs (no accumulator-register copies).
PER_FILE = {"gemm.hip": ["-mllvm", "-amdgpu-mfma-vgpr-form"],
            "gemm_skinny.hip": ["-mllvm", "-amdgpu-mfma-vgpr-form"]}

COMMON = ["-O3", "-std=c++17", "-fPIC", "-Wall", "-ffp-contract=off", "-fvisibility=hidden",
          "-I" + os.path.join(os.path.dirname(HERE), "include")]
DEVICE = ["-x", "hip", "--offload-arch=gfx950",
          "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
          "-fhip-fp32-correctly-rounded-divide-sqrt", "-fno-gpu-flush-denormals-to-zero",
          "-munsafe-fp-atomics"]


HEADER = os.path.join(os.path.dirname(HERE), "include", "comet.h")
STAMP_RE = re.compile(rb"COMET_SOURCE_STAMP=([0-9a-f]{64})")


def source_stamp() -> str:
    """SHA-256 over every file under csrc/ (sorted by name), the public
    header and the build flags."""
    h = hashlib.sha256()
    names = sorted(n for n in os.listdir(CSRC) if not n.startswith("."))
    for name in names + [None]:
        path = HEADER if name is None else os.path.join(CSRC, name)
        h.update((name or "include/comet.h").encode() + b"\0")
        with open(path, "rb") as f:
            h.update(f.read())
        h.update(b"\0")
    # flags without the include path, which depends on where the tree sits
    flags = [f for f in COMMON if not f.startswith("-I")] + DEVICE
    h.update(repr((SOURCES, PER_FILE, flags)).encode())
    return h.hexdigest()


def library_stamp(path: str = LIB):
    """The stamp recorded in a built library file (read from its bytes,
    without loading it), or None."""
    try:
        with open(path, "rb") as f:
            m = STAMP_RE.search(f.read())
    except OSError:
        return None
    return m.group(1).decode() if m else None


def _compile(src: str, verbose: bool, stamp: str) -> str:
    path = os.path.join(CSRC, src)
    obj = os.path.join(OUT_DIR, src + ".o")
    cmd = [HIPCC] + COMMON
    if src.endswith(".hip"):
        cmd += DEVICE + PER_FILE.get(src, [])
    if src == "comet_api.cpp":
        cmd += [f'-DCOMET_SOURCE_STAMP="{stamp}"']
    cmd += ["-c", path, "-o", obj]
    if verbose:
        print(" ".join(cmd), file=sys.stderr)
    r = subprocess.run(cmd, capture_output=True, text=True)
    # hipcc's host pass does not know the packed-fp32 target feature; that
    # warning is expected and harmless.
    msg = "\n".join(l for l in (r.stdout + r.stderr).splitlines()
                    if "packed-fp32-ops" not in l and "not a recognized feature" not in l)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed on {src}:\n{msg}")
    if verbose and msg.strip():
        print(msg, file=sys.stderr)
    return obj


def build(verbose: bool = False) -> str:
    os.makedirs(OUT_DIR, exist_ok=True)
    stamp = source_stamp()
    with ThreadPoolExecutor(len(SOURCES)) as ex:
        objs = list(ex.map(lambda s: _compile(s, verbose, stamp), SOURCES))
    tmp = LIB + ".tmp"
    cmd = [HIPCC, "-shared", "-fPIC", "--offload-arch=gfx950", "-o", tmp] + objs
    if verbose:
        print(" ".join(cmd), file=sys.stderr)
    subprocess.run(cmd, check=True)
    if library_stamp(tmp) != stamp:
        raise RuntimeError("built library does not carry the source stamp")
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
