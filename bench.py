"""Benchmark of the W4Ax hot path on one MI355X.

One step = the whole hot path over one batch: for each linear layer of the
workload, online FMPQ quantization of the fp16 activations (M tokens) and the
W4Ax GEMM against the layer's pre-packed 4-bit weights.  Weight packing is
offline (done once before timing).  Inputs are seeded synthetic tensors of the
layer shapes, resident in HBM before the timed region starts.

Prints ONE JSON line.  ``value`` is effective TOPS = sum over layers of
2*M*N*K divided by the step time.  ``roofline`` describes the dominant kernel
launch of the step, the GEMM of the largest layer: its algorithmic ops
(prefill, MFMA-bound) or bytes (decode, HBM-bound) per launch over its average
launch time, measured with HIP events on the stream the kernels run on.  Its
``traffic`` is the HBM bytes per launch read from the rocprofv3 counter
summary committed under profiles/, reported only while the kernel sources
still hash to the value recorded there (else null).  ``cpu_baseline`` times
the CPU oracle on a bounded sample of the same workload (a few token rows of
every layer) and also checks the GPU output rows of that sample against it.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)
sys.path.insert(0, os.path.join(ROOT, "tests"))

PEAK_MFMA_TFLOPS = 5000.0  # MI355X dense FP8 (= dense INT8) MFMA
PEAK_HBM_GBS = 8000.0

METRIC = "W4Ax GEMM effective TOPS + % int8-MFMA peak / % HBM BW, LLaMA-3-70B shapes"

WORKLOADS = {
    "llama3-70b-prefill": dict(M=4096, layers="LLAMA3_70B"),
    "llama3-8b-prefill": dict(M=2048, layers="LLAMA3_8B"),
    # few-token regime: the gate_up layer streams its 4-bit weights from HBM
    "llama3-70b-decode": dict(M=8, layers="LLAMA3_70B", only="gate_up", rotate=6),
    # LLaMA-3-70B MLP: quantize x, the gate/up GEMM through the SwiGLU entry
    # point (the down projection's input quantized in the GEMM epilogue on
    # 128-row tiles, by the standalone SwiGLU kernel on the other paths),
    # down GEMM
    "llama3-70b-mlp": dict(M=4096, mlp=True),
    # KV4 cache quantization of a prefill batch (8 prompts x 4096 tokens): the
    # K and V rows of every layer (8 KV heads x head_dim 128 = 1024 channels,
    # groups of 128)
    "llama3-70b-kv4": dict(T=32768, C=1024, n_layers=80, G=128),
}

# Sources that determine each GEMM kernel's code; a counter summary applies
# only to the sources it was taken with.
CSRC = os.path.join(ROOT, "paper_2410_12168_amd", "csrc")
KERNEL_SOURCES = {
    "tile": ["gemm.hip", "operand.h", "kernels.h"],
    "skinny": ["gemm_skinny.hip", "operand.h", "kernels.h"],
    "skinny_shared": ["gemm_skinny.hip", "operand.h", "kernels.h"],
    "mid": ["gemm.hip", "operand.h", "kernels.h"],
    "stream": ["gemm_skinny.hip", "operand.h", "kernels.h"],
    "kv4": ["kv4.hip"],
}
def gemm_kind(M: int, N: int, K: int, cus: int) -> str:
    """Which GEMM kernel the library runs for this shape (asked of the library)."""
    import paper_2410_12168_amd as comet

    return comet.KERNEL_NAMES[comet.comet_gemm_kernel(M, N, K, cus)]


def _code_only(text: str) -> str:
    """C++ source without comments and blank lines, so that a comment edit
    does not mark a kernel as changed.  (The kernel sources hold no string
    literal with a comment marker in it.)"""
    import re

    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    lines = (re.sub(r"//.*", "", line).rstrip() for line in text.splitlines())
    return "\n".join(line for line in lines if line.strip())


def kernel_sha(kind: str) -> str:
    """SHA-256 of the code (comments and blank lines removed) of the sources
    that determine this kernel."""
    h = hashlib.sha256()
    for name in KERNEL_SOURCES[kind]:
        with open(os.path.join(CSRC, name), encoding="utf-8") as f:
            h.update(_code_only(f.read()).encode())
    return h.hexdigest()


def profile_path(kind: str, workload: str, layer: str, M: int) -> str:
    if kind == "kv4":
        return os.path.join(ROOT, "profiles", f"kv4_quantize_{workload}_t{M}.txt")
    return os.path.join(ROOT, "profiles", f"w4ax_gemm_{kind}_{workload}_{layer}_m{M}.txt")


def profiled_traffic(kind: str, workload: str, layer: str, M: int):
    """HBM bytes per launch from the committed counter summary of this kernel
    and workload, or None (no summary, or the kernel changed since)."""
    path = profile_path(kind, workload, layer, M)
    if not os.path.exists(path):
        return None
    fields = {}
    with open(path) as f:
        for line in f:
            if ":" in line and not line.startswith((" ", "#")):
                k, v = line.split(":", 1)
                fields[k.strip()] = v.strip()
    if fields.get("kernel_sources_sha256") != kernel_sha(kind):
        return None
    try:
        return int(float(fields["traffic_bytes_per_launch"]))
    except (KeyError, ValueError):
        return None


def warm_up(warmup, step) -> int:
    """Run the untimed warm-up steps and return how many ran: `warmup` if
    given, else 5 and then, for short steps, as many more as cover 20 ms of
    GPU work (one of them timed with events to size the rest), because the
    clock ramps up over the first milliseconds of work."""
    import math

    import torch

    n = 5 if warmup is None else warmup
    for _ in range(n):
        step()
    if warmup is not None:
        return n
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    step()
    e1.record()
    torch.cuda.synchronize()
    extra = max(0, math.ceil(20.0 / max(e0.elapsed_time(e1), 1e-3)) - n - 1)
    for _ in range(extra):
        step()
    return n + 1 + extra


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=None,
                    help="untimed warm-up steps (default: 5, or more for short steps: enough "
                         "for 20 ms of GPU work, since the clock ramps up over the first "
                         "milliseconds)")
    ap.add_argument("--workload", default="llama3-70b-prefill", choices=sorted(WORKLOADS))
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--m", type=int, default=0, help="tokens (default: the workload's)")
    ap.add_argument("--frac8", type=float, default=1 / 16)
    ap.add_argument("--placement", default="contiguous", choices=["contiguous", "random"],
                    help="where the 8-bit blocks sit (a contiguous run, or a seeded random subset)")
    ap.add_argument("--layers", default="",
                    help="comma-separated subset of the workload's layers (default: all)")
    ap.add_argument("--copy-mib", type=int, default=0,
                    help="after timing, run one device-to-device copy of this many MiB (a "
                         "known-size reference for HBM byte counters)")
    ap.add_argument("--unfused", action="store_true",
                    help="llama3-70b-mlp: gate/up GEMM to fp16, then a separate SwiGLU-quantize "
                         "kernel (instead of the fused epilogue)")
    ap.add_argument("--perm", action="store_true",
                    help="calibrated channel permutation: activations with scattered outlier "
                         "channels, map and permutation planned from sampled maxima, permuted "
                         "quantization (weights packed with the same permutation)")
    ap.add_argument("--cpu-rows", type=int, default=512,
                    help="token rows per layer in the CPU-oracle sample (0: skip)")
    ap.add_argument("--no-extras", action="store_true",
                    help="llama3-70b-prefill: skip the other configurations (small case, "
                         "LLaMA-3-8B layers, load-balance sweep with the schedule ablation, "
                         "decode sweep) that the default run reports beside the headline")
    return ap.parse_args()


def main():
    args = parse()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the W4Ax GEMM is a single-GPU kernel and this "
              "build has no multi-GPU path (--gpus must be 1).", file=sys.stderr)
        sys.exit(2)

    import torch

    import paper_2410_12168_amd as comet
    import synth

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    wl = WORKLOADS[args.workload]
    if "T" in wl:
        return bench_kv4(args, wl, dev)
    if wl.get("mlp"):
        return bench_mlp(args, wl, dev)
    M = args.m or wl["M"]
    shapes = getattr(synth, wl["layers"])
    if "only" in wl:
        shapes = {wl["only"]: shapes[wl["only"]]}
    rotate = wl.get("rotate", 1)
    layers = []
    t_setup = time.time()
    wanted = [x for x in args.layers.split(",") if x] or list(shapes)
    for name, (K, N) in shapes.items():
        if name not in wanted:
            continue
        NG = K // 128
        perm = None
        W16 = synth.weights(args.seed, N, K)
        Wd = torch.from_numpy(W16.view(np.int16)).to(dev).view(torch.float16)
        if args.perm:
            # outliers on 0.5% of the channels, scattered; calibrate on 512 rows
            ch = synth.outlier_channels(K, max(1, K // 200), seed=args.seed)
            X16 = synth.calibration_activations(args.seed, M, K, ch)
            X = torch.from_numpy(X16.view(np.int16)).to(dev).view(torch.float16)
            absmax = comet.channel_absmax(X[:512])
            perm_h, prec, _ = comet.plan_channel_perm(absmax, 128, 8.0, 0.2)
            perm = torch.from_numpy(perm_h).to(dev)
            n8 = int((prec == 8).sum())
        else:
            n8 = int(round(NG * args.frac8))
            prec = synth.prec_map(NG, n8, args.placement, seed=args.seed)
            X16 = synth.activations(args.seed, M, K, prec)
            X = torch.from_numpy(X16.view(np.int16)).to(dev).view(torch.float16)
        Wp, sw = comet.pack_w4(Wd, perm=perm)
        torch.cuda.synchronize()
        del Wd
        # several weight copies, used in turn, so that each call streams its
        # weights from HBM instead of the 256 MB last-level cache
        Wps = [Wp] + [Wp.clone() for _ in range(rotate - 1)]
        sws = [sw] + [sw.clone() for _ in range(rotate - 1)]
        nbytes = comet.comet_act_packed_bytes(prec, M, K)
        A = torch.empty(nbytes, dtype=torch.uint8, device=dev)
        sa = torch.empty((NG, M), dtype=torch.float16, device=dev)
        out = torch.empty((M, N), dtype=torch.float16, device=dev)
        layers.append(dict(name=name, M=M, N=N, K=K, prec=prec, X=X, X16=X16, W16=W16, Wp=Wp,
                           sw=sw, Wps=Wps, sws=sws, A=A, sa=sa, out=out, n8=n8, perm=perm,
                           perm_h=None if perm is None else perm.cpu().numpy()))
    t_setup = time.time() - t_setup

    calls = [0]

    def step(ev=None):
        calls[0] += 1
        for i, L in enumerate(layers):
            j = calls[0] % rotate
            if ev is not None:
                ev[i][0].record()
            comet.comet_fmpq_quantize_act_perm(L["X"], L["perm"], L["prec"], L["A"], L["sa"],
                                               L["M"], L["K"])
            if ev is not None:
                ev[i][1].record()
            comet.comet_w4ax_gemm(L["A"], L["prec"], L["sa"], L["Wps"][j], L["sws"][j], L["out"],
                                  L["M"], L["N"], L["K"])
            if ev is not None:
                ev[i][2].record()

    args.warmup = warm_up(args.warmup, step)
    torch.cuda.synchronize()

    # timed region: whole steps; then, queued right behind it so that the GPU
    # does not idle in between, the same steps again with events around each
    # launch (same stream) for the per-kernel durations
    start = torch.cuda.Event(enable_timing=True)
    stop = torch.cuda.Event(enable_timing=True)
    evs = [[[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in layers]
           for _ in range(args.steps)]
    torch.cuda.synchronize()
    start.record()
    for _ in range(args.steps):
        step()
    stop.record()
    for s in range(args.steps):
        step(evs[s])
    torch.cuda.synchronize()
    ms_total = start.elapsed_time(stop)
    ms_per_step = ms_total / args.steps
    q_ms = np.zeros(len(layers))
    g_ms = np.zeros(len(layers))
    for s in range(args.steps):
        for i in range(len(layers)):
            q_ms[i] += evs[s][i][0].elapsed_time(evs[s][i][1])
            g_ms[i] += evs[s][i][1].elapsed_time(evs[s][i][2])
    q_ms /= args.steps
    g_ms /= args.steps

    ops = np.array([2.0 * L["M"] * L["N"] * L["K"] for L in layers])
    # algorithmic HBM bytes of one GEMM call: packed weights and their scales,
    # packed activations and their scales, fp16 output
    gbytes = []
    for L in layers:
        K, N, NG, k8 = L["K"], L["N"], L["K"] // 128, L["n8"] * 128
        gbytes.append(N * K / 2 + 2 * N * NG + M * ((K - k8) / 2 + k8) + 2 * M * NG + 2 * M * N)
    gbytes = np.array(gbytes)
    value = float(ops.sum() / (ms_per_step * 1e-3) / 1e12)
    hbm_bound = "decode" in args.workload
    per_layer = {}
    for i, L in enumerate(layers):
        K, N = L["K"], L["N"]
        NG = K // 128
        k8 = L["n8"] * 128
        qbytes = 2 * M * K + M * ((K - k8) // 2 + k8) + 2 * M * NG
        per_layer[L["name"]] = {
            "K": K, "N": N, "gemm_us": round(g_ms[i] * 1e3, 2),
            "gemm_tops": round(ops[i] / (g_ms[i] * 1e-3) / 1e12, 1),
            "gemm_frac_peak": round(ops[i] / (g_ms[i] * 1e-3) / 1e12 / PEAK_MFMA_TFLOPS, 4),
            "gemm_gbs": round(gbytes[i] / (g_ms[i] * 1e-3) / 1e9, 1),
            "quant_us": round(q_ms[i] * 1e3, 2),
            "quant_gbs": round(qbytes / (q_ms[i] * 1e-3) / 1e9, 1),
        }
    # the dominant kernel launch: the GEMM of the layer with the most work
    d = int(np.argmax(ops))
    D = layers[d]
    kind = gemm_kind(M, D["N"], D["K"], torch.cuda.get_device_properties(0).multi_processor_count)
    if hbm_bound:
        achieved = float(gbytes[d] / (g_ms[d] * 1e-3) / 1e9)
        roof = {"bound": "hbm", "achieved": round(achieved, 1), "peak": PEAK_HBM_GBS,
                "unit": "GB/s", "frac": round(achieved / PEAK_HBM_GBS, 4)}
    else:
        achieved = float(ops[d] / (g_ms[d] * 1e-3) / 1e12)
        roof = {"bound": "mfma", "achieved": round(achieved, 1), "peak": PEAK_MFMA_TFLOPS,
                "unit": "TFLOP/s", "frac": round(achieved / PEAK_MFMA_TFLOPS, 4)}
    roof["traffic"] = profiled_traffic(kind, args.workload, D["name"], M)
    roof["kernel"] = (f"w4ax_gemm {kind} kernel, {D['name']} layer (M={M}, K={D['K']}, "
                      f"N={D['N']}): {'bytes' if hbm_bound else 'ops'} per launch "
                      f"{int(gbytes[d] if hbm_bound else ops[d])}, {g_ms[d] * 1e3:.2f} us per launch")
    roof["alg_bytes_per_launch"] = int(gbytes[d])

    record = {
        "metric": METRIC,
        "value": round(value, 2),
        "unit": "TOPS",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "fp8",
        "data": "synthetic",
        "config": {
            "workload": (f"{args.workload}: quantize+W4Ax GEMM of {'/'.join(per_layer)} at M={M} "
                         f"tokens, G=128, " +
                         (f"calibrated channel permutation ({', '.join(str(L['n8']) for L in layers)}"
                          f" 8-bit blocks)" if args.perm else
                          f"{args.frac8:.4g} of activation blocks 8-bit ({args.placement})")),
            "M": M, "G": 128, "frac8": (round(float(np.mean([L['n8'] / (L['K'] // 128)
                                                          for L in layers])), 4)
                                        if args.perm else args.frac8),
            "perm": bool(args.perm), "placement": args.placement, "seed": args.seed,
            "operands": "int4 weights, int4/int8 activation codes on FP8-E4M3 MFMA, fp32 dequant",
        },
        "roofline": roof,
        "layers": per_layer,
        "setup_s": round(t_setup, 1),
    }

    if args.copy_mib > 0:
        src = torch.empty(args.copy_mib << 20, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        record["copy_mib"] = args.copy_mib

    if args.workload == "llama3-70b-prefill" and not args.no_extras and not args.m and \
            not args.layers and not args.perm:
        record["configs"] = bench_extras(args, dev, layers)

    if args.cpu_rows > 0:
        record["cpu_baseline"] = cpu_baseline(layers, args.cpu_rows)

    print(json.dumps(record), flush=True)


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(layers, rows_per_layer: int) -> dict:
    """Time the CPU oracle on a bounded sample (the first rows of every layer)
    and check the GPU output of those rows against it."""
    import torch

    import oracle
    from parity import out_errors

    threads = os.cpu_count() or 1
    t_total = 0.0
    ops = 0.0
    worst = 0.0
    worst_norm = 0.0
    for L in layers:
        rows = np.arange(min(rows_per_layer, L["M"]))
        W16, X16 = L["W16"], L["X16"][rows]
        if L["perm_h"] is not None:  # offline: permute the weight columns
            W16 = oracle.permute_columns(W16, L["perm_h"])
        qw, sw = oracle.quantize_weight(W16, nthreads=threads)  # offline step, not timed
        t0 = time.perf_counter()
        if L["perm_h"] is not None:
            X16 = oracle.permute_columns(X16, L["perm_h"])
        qa, sa = oracle.quantize_act(X16, L["prec"], nthreads=threads)
        ref = oracle.dequant_gemm(qa, sa, qw, sw, nthreads=threads)
        t_total += time.perf_counter() - t0
        ops += 2.0 * len(rows) * L["N"] * L["K"]
        y = L["out"][: len(rows)].view(torch.int16).cpu().numpy().view(np.float16)
        mx, norm = out_errors(y, ref)
        worst = max(worst, mx)
        worst_norm = max(worst_norm, norm)
    # one thread on the small case (16 x 1024 x 1024, block 3 of 8 in 8 bits):
    # a per-core figure, median of three runs
    import synth

    prec0 = synth.prec_map(8, 1)
    X0, W0 = synth.activations(0, 16, 1024, prec0), synth.weights(0, 1024, 1024)
    qw0, sw0 = oracle.quantize_weight(W0, nthreads=1)
    t1 = []
    for _ in range(3):
        t0 = time.perf_counter()
        qa0, sa0 = oracle.quantize_act(X0, prec0, nthreads=1)
        oracle.dequant_gemm(qa0, sa0, qw0, sw0, nthreads=1)
        t1.append(time.perf_counter() - t0)
    t1 = float(np.median(t1))
    return {
        "value": round(ops / t_total / 1e12, 5), "unit": "TOPS", "cores": threads,
        "kind": "oracle", "seconds": round(t_total, 2), "cpu_model": cpu_model(),
        "rows_per_layer": int(min(rows_per_layer, layers[0]["M"])),
        "sample": ", ".join(f"{L['name']}: first {min(rows_per_layer, L['M'])} of {L['M']} token rows"
                            for L in layers) + " (quantize + fp64-dequant GEMM); value = "
                  "2*rows*N*K summed over the sample / oracle seconds",
        "single_thread_small_case": {
            "workload": "M=16, K=N=1024, G=128, block 3 of 8 in 8 bits (quantize + GEMM), "
                        "median of 3", "seconds": round(t1, 5), "cores": 1,
            "value": round(2.0 * 16 * 1024 * 1024 / t1 / 1e12, 6), "unit": "TOPS"},
        "parity_max_rel": worst, "parity_norm_rel": worst_norm, "parity_ok": worst <= 2e-3,
    }


def _to_dev(a16, dev):
    import torch

    return torch.from_numpy(np.ascontiguousarray(a16).view(np.int16)).to(dev).view(torch.float16)


def _ms_per_call(fn, n: int, warm: int = 2, min_ms: float = 20.0) -> float:
    """Average time of `fn(i)` over back-to-back calls, from HIP events around
    the batch on the current stream (the one the library launches on).

    After the host-side setup between measurements the GPU has idled and its
    clock ramps back up over the first milliseconds of work, so every
    measurement first runs at least `min_ms` of untimed calls (and at least
    `warm`), then times at least n calls and at least `min_ms` of them."""
    import math

    import torch

    for i in range(warm):
        fn(i)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    fn(0)
    e1.record()
    torch.cuda.synchronize()
    reps = max(1, math.ceil(min_ms / max(e0.elapsed_time(e1), 1e-3)))
    for i in range(reps):
        fn(i)
    n = max(n, reps)
    torch.cuda.synchronize()
    e0.record()
    for i in range(n):
        fn(i)
    e1.record()
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) / n


def _rows_err(out, X16, prec, qw, sw, rows) -> float:
    """Max elementwise error (tests/parity.py rule) of the fp16 output rows
    against the CPU oracle."""
    import torch

    import oracle
    from parity import out_errors

    qa, sa = oracle.quantize_act(X16[rows], prec)
    ref = oracle.dequant_gemm(qa, sa, qw, sw)
    idx = torch.from_numpy(np.asarray(rows)).to(out.device)
    y = out[idx].view(torch.int16).cpu().numpy().view(np.float16)
    return out_errors(y, ref)[0]


def _gemm_bytes(M, N, K, n8):
    k8 = 128 * n8
    return N * K / 2 + 2 * N * (K // 128) + M * ((K - k8) / 2 + k8) + 2 * M * (K // 128) + 2 * M * N


def bench_extras(args, dev, main_layers) -> dict:
    """The other benchmark configurations, measured in the same run beside the
    headline (each GEMM timed over back-to-back calls with HIP events; fp16
    outputs of sampled rows checked against the CPU oracle):
      small: M = 16, K = N = 1024, block 3 of 8 in 8 bits (launch-bound);
      llama3_8b: the four LLaMA-3-8B layers at M = 2048;
      load_balance: LLaMA-3-70B down (M = 4096, K = 28672, N = 8192) with 0,
        1/16, 1/4 and 1/2 of the blocks 8-bit, contiguous or random;
      ablation: the schedule modes natural (map order, whole tiles), dp
        (precision-batched order, whole tiles) and cost (the default: plus a
        cost-balanced split of the last wave of tiles) on the load-balance
        points and on the 70B qkv layer;
      decode: LLaMA-3-70B gate_up at M = 1, 8, 32, 128 with six rotated weight
        copies, so every call streams its weights from HBM."""
    import torch

    import oracle
    import paper_2410_12168_amd as comet
    import synth

    cus = torch.cuda.get_device_properties(0).multi_processor_count
    res = {}
    seed = args.seed

    def mode(m):
        if m is None:
            os.environ.pop("COMET_SCHED", None)
        else:
            os.environ["COMET_SCHED"] = m

    # small case
    M, K, N = 16, 1024, 1024
    prec = synth.prec_map(K // 128, 1)
    X16, W16 = synth.activations(seed, M, K, prec), synth.weights(seed, N, K)
    X, Wd = _to_dev(X16, dev), _to_dev(W16, dev)
    Wp, sw = comet.pack_w4(Wd)
    A, sa = comet.quantize_act(X, prec)
    out = torch.empty((M, N), dtype=torch.float16, device=dev)

    def small_both(i):
        comet.comet_fmpq_quantize_act(X, prec, A, sa, M, K)
        comet.comet_w4ax_gemm(A, prec, sa, Wp, sw, out, M, N, K)

    t_both = _ms_per_call(small_both, 200)
    t_gemm = _ms_per_call(lambda i: comet.comet_w4ax_gemm(A, prec, sa, Wp, sw, out, M, N, K), 200)
    qw, osw = oracle.quantize_weight(W16)
    res["small"] = {"workload": "M=16, K=N=1024, G=128, block 3 of 8 in 8 bits",
                    "kernel": comet.KERNEL_NAMES[comet.comet_gemm_kernel(M, N, K, cus)],
                    "quant_plus_gemm_us": round(t_both * 1e3, 2),
                    "gemm_us": round(t_gemm * 1e3, 2),
                    "parity_max_rel": _rows_err(out, X16, prec, qw, osw, np.arange(M))}

    # LLaMA-3-8B layers at M = 2048
    M = 2048
    layers8 = {}
    for name, (K, N) in synth.LLAMA3_8B.items():
        NG = K // 128
        prec = synth.prec_map(NG, NG // 16)
        X16, W16 = synth.activations(seed, M, K, prec), synth.weights(seed, N, K)
        X, Wd = _to_dev(X16, dev), _to_dev(W16, dev)
        Wp, sw = comet.pack_w4(Wd)
        del Wd
        A, sa = comet.quantize_act(X, prec)
        out = torch.empty((M, N), dtype=torch.float16, device=dev)
        tq = _ms_per_call(lambda i: comet.comet_fmpq_quantize_act(X, prec, A, sa, M, K), 10)
        tg = _ms_per_call(lambda i: comet.comet_w4ax_gemm(A, prec, sa, Wp, sw, out, M, N, K), 10)
        ops = 2.0 * M * N * K
        qw, osw = oracle.quantize_weight(W16)
        rows = np.arange(0, M, 256) + 17  # one row in every 256-row tile
        layers8[name] = {"K": K, "N": N, "gemm_us": round(tg * 1e3, 2),
                         "gemm_frac_peak": round(ops / (tg * 1e-3) / 1e12 / PEAK_MFMA_TFLOPS, 4),
                         "quant_us": round(tq * 1e3, 2),
                         "parity_max_rel": _rows_err(out, X16, prec, qw, osw, rows)}
        del X, A, sa, out, Wp, sw
    res["llama3_8b"] = {"M": M, "frac8": 1 / 16, "layers": layers8}

    # load-balance sweep on the 70B down projection, with the schedule ablation
    M, (K, N) = 4096, synth.LLAMA3_70B["down"]
    NG = K // 128
    W16 = synth.weights(seed, N, K)
    Wd = _to_dev(W16, dev)
    Wp, sw = comet.pack_w4(Wd)
    del Wd
    qw, osw = oracle.quantize_weight(W16)
    out = torch.empty((M, N), dtype=torch.float16, device=dev)
    ops = 2.0 * M * N * K
    sweep, abl = {}, {}
    for frac in (0.0, 1 / 16, 1 / 4, 1 / 2):
        for place in ("contiguous", "random"):
            if frac == 0.0 and place == "random":
                continue  # no 8-bit blocks: the same map
            n8 = int(round(NG * frac))
            prec = synth.prec_map(NG, n8, place, seed=seed)
            X16 = synth.activations(seed, M, K, prec)
            X = _to_dev(X16, dev)
            A, sa = comet.quantize_act(X, prec)
            del X
            key = f"f={frac:g},{place}"
            t = {}
            for m in ("natural", "dp", "cost"):
                mode(m)
                t[m] = _ms_per_call(
                    lambda i: comet.comet_w4ax_gemm(A, prec, sa, Wp, sw, out, M, N, K), 5)
            mode(None)
            err = _rows_err(out, X16, prec, qw, osw, np.array([1, 1000, 2600, 4095]))
            sweep[key] = {"n8": n8, "gemm_us": round(t["cost"] * 1e3, 2),
                          "frac_peak": round(ops / (t["cost"] * 1e-3) / 1e12 / PEAK_MFMA_TFLOPS, 4),
                          "parity_max_rel": err}
            abl[f"down {key}"] = {m: round(v * 1e3, 2) for m, v in t.items()}
            del A, sa
    t0 = sweep["f=0,contiguous"]["gemm_us"]
    for v in sweep.values():
        v["t_over_t0"] = round(v["gemm_us"] / t0, 4)
    res["load_balance"] = {"workload": "LLaMA-3-70B down, M=4096, K=28672, N=8192", "points": sweep}
    del Wp, sw, out

    # ablation on the 70B qkv layer of the headline step (640 tiles on 256 CUs)
    for L in main_layers:
        if L["name"] != "qkv":
            continue
        t = {}
        for m in ("natural", "dp", "cost"):
            mode(m)
            t[m] = _ms_per_call(lambda i: comet.comet_w4ax_gemm(
                L["A"], L["prec"], L["sa"], L["Wp"], L["sw"], L["out"], L["M"], L["N"], L["K"]), 10)
        mode(None)
        abl["qkv M=4096 f=1/16 contiguous"] = {m: round(v * 1e3, 2) for m, v in t.items()}
    res["ablation_us"] = {"modes": "natural = map order, whole tiles; dp = precision-batched "
                                   "order, whole tiles; cost = precision-batched + cost-balanced "
                                   "split of the last wave (default)", "gemm_us": abl}

    # decode sweep on the 70B gate_up with rotated weights
    K, N = synth.LLAMA3_70B["gate_up"]
    NG = K // 128
    prec = synth.prec_map(NG, NG // 16)
    W16 = synth.weights(seed, N, K)
    Wd = _to_dev(W16, dev)
    Wp, sw = comet.pack_w4(Wd)
    del Wd
    rot = 6
    Wps = [Wp] + [Wp.clone() for _ in range(rot - 1)]
    sws = [sw] + [sw.clone() for _ in range(rot - 1)]
    qw, osw = oracle.quantize_weight(W16)
    dec = {}
    for M in (1, 8, 32, 128):
        X16 = synth.activations(seed, M, K, prec)
        A, sa = comet.quantize_act(_to_dev(X16, dev), prec)
        out = torch.empty((M, N), dtype=torch.float16, device=dev)
        t = _ms_per_call(lambda i: comet.comet_w4ax_gemm(A, prec, sa, Wps[i % rot], sws[i % rot],
                                                         out, M, N, K), 60, warm=6)
        nbytes = _gemm_bytes(M, N, K, NG // 16)
        rows = np.arange(M) if M <= 32 else np.array([0, 1, 63, 64, 127])
        dec[f"M={M}"] = {"kernel": comet.KERNEL_NAMES[comet.comet_gemm_kernel(M, N, K, cus)],
                         "gemm_us": round(t * 1e3, 2),
                         "gbs": round(nbytes / (t * 1e-3) / 1e9, 1),
                         "frac_hbm": round(nbytes / (t * 1e-3) / 1e9 / PEAK_HBM_GBS, 4),
                         "alg_bytes": int(nbytes),
                         "parity_max_rel": _rows_err(out, X16, prec, qw, osw, rows)}
    res["decode"] = {"workload": "LLaMA-3-70B gate_up, K=8192, N=57344, 1/16 of blocks 8-bit, "
                                 f"{rot} rotated weight copies (back-to-back calls)", "points": dec}
    del Wps, sws
    torch.cuda.empty_cache()
    worst = max([res["small"]["parity_max_rel"]] +
                [v["parity_max_rel"] for v in layers8.values()] +
                [v["parity_max_rel"] for v in sweep.values()] +
                [v["parity_max_rel"] for v in dec.values()])
    res["parity_max_rel"] = worst
    res["parity_ok"] = worst <= 2e-3
    return res


def bench_mlp(args, wl, dev):
    """One LLaMA-3-70B MLP over M tokens: quantize x (K = 8192), gate/up W4Ax
    GEMM (N = 2 x 28672, gate/up rows in 256-wide groups) whose epilogue forms
    h = SiLU(gate) * up and quantizes it for the down projection, then the
    down W4Ax GEMM (28672 -> 8192).  --unfused writes the gate/up output in
    fp16 and runs the SwiGLU quantizer as its own kernel instead."""
    import torch

    import paper_2410_12168_amd as comet
    import synth

    M = args.m or wl["M"]
    (K1, N1), (K2, N2) = synth.LLAMA3_70B["gate_up"], synth.LLAMA3_70B["down"]
    I = N1 // 2
    t_setup = time.time()
    NG1, NG2 = K1 // 128, K2 // 128
    prec1 = synth.prec_map(NG1, int(round(NG1 * args.frac8)), args.placement, seed=args.seed)
    prec2 = synth.prec_map(NG2, int(round(NG2 * args.frac8)), args.placement, seed=args.seed + 1)
    X16 = synth.activations(args.seed, M, K1, prec1)
    X = torch.from_numpy(X16.view(np.int16)).to(dev).view(torch.float16)
    packed = []
    for tid_seed, (N, K) in ((args.seed, (N1, K1)), (args.seed + 1, (N2, K2))):
        Wd = torch.from_numpy(synth.weights(tid_seed, N, K).view(np.int16)).to(dev).view(torch.float16)
        packed.append(comet.pack_w4(Wd))
        del Wd
    (Wp1, sw1), (Wp2, sw2) = packed
    A1 = torch.empty(comet.comet_act_packed_bytes(prec1, M, K1), dtype=torch.uint8, device=dev)
    sa1 = torch.empty((NG1, M), dtype=torch.float16, device=dev)
    A2 = torch.empty(comet.comet_act_packed_bytes(prec2, M, K2), dtype=torch.uint8, device=dev)
    sa2 = torch.empty((NG2, M), dtype=torch.float16, device=dev)
    gu = torch.empty((M, N1), dtype=torch.float16, device=dev) if args.unfused else None
    y = torch.empty((M, N2), dtype=torch.float16, device=dev)
    torch.cuda.synchronize()
    t_setup = time.time() - t_setup

    def step(ev=None):
        comet.comet_fmpq_quantize_act(X, prec1, A1, sa1, M, K1)
        if ev is not None:
            ev[0].record()
        if args.unfused:
            comet.comet_w4ax_gemm(A1, prec1, sa1, Wp1, sw1, gu, M, N1, K1)
            comet.comet_swiglu_quantize(gu, prec2, A2, sa2, M, I)
        else:
            comet.comet_w4ax_gemm_swiglu_quant(A1, prec1, sa1, Wp1, sw1, M, N1, K1, 128, prec2,
                                               A2, sa2)
        if ev is not None:
            ev[1].record()
        comet.comet_w4ax_gemm(A2, prec2, sa2, Wp2, sw2, y, M, N2, K2)

    args.warmup = warm_up(args.warmup, step)
    torch.cuda.synchronize()
    start = torch.cuda.Event(enable_timing=True)
    stop = torch.cuda.Event(enable_timing=True)
    start.record()
    for _ in range(args.steps):
        step()
    stop.record()
    torch.cuda.synchronize()
    ms_per_step = start.elapsed_time(stop) / args.steps
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(2)] for _ in range(args.steps)]
    for k in range(args.steps):
        step(evs[k])
    torch.cuda.synchronize()
    gu_ms = float(np.mean([e[0].elapsed_time(e[1]) for e in evs]))
    ops1, ops2 = 2.0 * M * N1 * K1, 2.0 * M * N2 * K2
    value = (ops1 + ops2) / (ms_per_step * 1e-3) / 1e12
    achieved = ops1 / (gu_ms * 1e-3) / 1e12
    record = {
        "metric": METRIC, "value": round(value, 2), "unit": "TOPS", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "fp8",
        "data": "synthetic",
        "config": {"workload": f"{args.workload}: quantize x, gate/up W4Ax GEMM "
                               f"{'then a separate SwiGLU-quantize kernel' if args.unfused else 'with SwiGLU + down-input quantization fused in its epilogue'}"
                               f", down W4Ax GEMM, M={M} tokens, G=128, {args.frac8:.4g} of "
                               f"activation blocks 8-bit",
                   "M": M, "G": 128, "frac8": args.frac8, "fused": not args.unfused,
                   "seed": args.seed},
        "roofline": {"bound": "mfma", "achieved": round(achieved, 1), "peak": PEAK_MFMA_TFLOPS,
                     "unit": "TFLOP/s", "frac": round(achieved / PEAK_MFMA_TFLOPS, 4),
                     "traffic": None,
                     "kernel": f"gate/up W4Ax GEMM{' + SwiGLU quantizer' if args.unfused else ' with fused SwiGLU epilogue'}"
                               f" (M={M}, K={K1}, N={N1}): {gu_ms * 1e3:.2f} us per step"},
        "setup_s": round(t_setup, 1),
    }
    print(json.dumps(record), flush=True)


def bench_kv4(args, wl, dev):
    """KV4 quantization of a prefill batch's K and V rows, every layer: a step is
    2 * n_layers launches over distinct buffers (the whole set exceeds the
    last-level cache, so each launch streams from HBM)."""
    import torch

    import paper_2410_12168_amd as comet
    import synth

    T, C, G, nl = (args.m or wl["T"]), wl["C"], wl["G"], wl["n_layers"]
    t_setup = time.time()
    X16 = [synth.kv_rows(args.seed + i, T, C) for i in range(2)]
    base = [torch.from_numpy(x.view(np.int16)).to(dev).view(torch.float16) for x in X16]
    # distinct copies per (layer, K/V)
    srcs = [base[i % 2] if i < 2 else base[i % 2].clone() for i in range(2 * nl)]
    codes = [torch.empty((T, C // 2), dtype=torch.uint8, device=dev) for _ in range(2 * nl)]
    params = [torch.empty((T, C // G, 2), dtype=torch.float16, device=dev) for _ in range(2 * nl)]
    torch.cuda.synchronize()
    t_setup = time.time() - t_setup

    def step(ev=None):
        for i in range(2 * nl):
            if ev is not None:
                ev[i][0].record()
            comet.comet_kv4_quantize(srcs[i], codes[i], params[i], T, C, G)
            if ev is not None:
                ev[i][1].record()

    args.warmup = warm_up(args.warmup, step)
    torch.cuda.synchronize()
    start = torch.cuda.Event(enable_timing=True)
    stop = torch.cuda.Event(enable_timing=True)
    start.record()
    for _ in range(args.steps):
        step()
    stop.record()
    torch.cuda.synchronize()
    ms_per_step = start.elapsed_time(stop) / args.steps
    # per-launch durations: events around each launch, on the launch stream
    evs = [[[torch.cuda.Event(enable_timing=True) for _ in range(2)] for _ in range(2 * nl)]
           for _ in range(args.steps)]
    for k in range(args.steps):
        step(evs[k])
    torch.cuda.synchronize()
    launch_ms = float(np.mean([e[0].elapsed_time(e[1]) for ek in evs for e in ek]))
    # algorithmic bytes per launch: fp16 rows in, 4-bit codes and {s, mn} out
    bpl = T * C * 2 + T * C // 2 + T * (C // G) * 4
    gbs = bpl / (launch_ms * 1e-3) / 1e9
    step_gbs = 2 * nl * bpl / (ms_per_step * 1e-3) / 1e9
    record = {
        "metric": "KV4 cache quantization effective GB/s (HBM), LLaMA-3-70B K/V rows",
        "value": round(step_gbs, 1), "unit": "GB/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms_per_step, 4), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "fp16->int4", "data": "synthetic",
        "config": {"workload": f"{args.workload}: asymmetric INT4 groups of {G} over K and V rows "
                               f"of {nl} layers, T={T} tokens x C={C} channels",
                   "T": T, "C": C, "G": G, "layers": nl, "seed": args.seed},
        "roofline": {"bound": "hbm", "achieved": round(gbs, 1), "peak": PEAK_HBM_GBS,
                     "unit": "GB/s", "frac": round(gbs / PEAK_HBM_GBS, 4),
                     "traffic": profiled_traffic("kv4", args.workload, "kv", T),
                     "kernel": f"kv4_quantize, T={T}, C={C}, G={G}: {bpl} bytes per launch, "
                               f"{launch_ms * 1e3:.2f} us per launch",
                     "alg_bytes_per_launch": bpl},
        "setup_s": round(t_setup, 1),
    }
    if args.copy_mib > 0:
        src = torch.empty(args.copy_mib << 20, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        record["copy_mib"] = args.copy_mib
    if args.cpu_rows > 0:
        import oracle

        rows = min(4096, T)
        threads = 1
        t0 = time.perf_counter()
        c_ref, p_ref = oracle.kv4_quantize(X16[0][:rows], G)
        dt = time.perf_counter() - t0
        got_c = codes[0][:rows].cpu().numpy()
        got_p = params[0][:rows].view(torch.int16).cpu().numpy().view(np.uint16)
        record["cpu_baseline"] = {
            "value": round((rows * C * 2 + rows * C // 2 + rows * (C // G) * 4) / dt / 1e9, 4),
            "unit": "GB/s", "cores": threads, "kind": "oracle", "seconds": round(dt, 3),
            "sample": f"first {rows} of {T} K rows of one layer",
            "parity_ok": bool(np.array_equal(got_c, c_ref) and np.array_equal(got_p, p_ref)),
        }
    print(json.dumps(record), flush=True)


if __name__ == "__main__":
    main()
