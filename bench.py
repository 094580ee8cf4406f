"""Benchmark of the kernelized-attention-with-RPE forward pass on one GPU.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload 4]

A step is one krpe_attention_fwd call over the whole workload (all batches and
heads): spectrum of c, feature maps of q and k, the FFT convolution +
contraction kernel and the final division.  Inputs are seeded synthetic data
already resident in device memory when the timed region starts.  Prints one
JSON line with whole-job throughput (tokens/s), the roofline position of the
dominant kernel (timed with HIP events on the library's stream) and the fp64
oracle's throughput on a bounded sample of the same workload on the host CPU.
"""
from __future__ import annotations

import argparse
import ctypes
import json
import math
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "tokens/sec and ms/layer for RPE kernelized attn fwd; % HBM/MFMA roofline"
PEAK_FP32_VECTOR_TFLOPS = 157.3   # MI355X published fp32 vector peak
PEAK_HBM_GBS = 8000.0


def direct_flops(B: int, H: int, n: int, d: int, m: int, b: np.ndarray) -> float:
    """Algorithmic flops of the direct route: for every (query, key) pair with a finite
    b_{j-i}, the feature dot product (2m), the weight c phi(q) phi(k) (1) and its product with
    [v, 1] (2 (d + 1))."""
    pairs = 0
    for h in range(b.shape[0]):
        t = np.arange(-(n - 1), n)
        pairs += int(np.sum((n - np.abs(t))[np.isfinite(b[h])]))
    return B * pairs * (2.0 * m + 1.0 + 2.0 * (d + 1))


BLOCK = 16384   # longest sequence one transform covers; longer ones run in blocks


def conv_stage_flops(B: int, H: int, n: int, d: int, m: int, b: np.ndarray | None = None) -> float:
    """Algorithmic flops of the FFT convolution + contraction stage.

    Per channel (m (d+1) channels per head): two real FFTs of length L = 2n at
    2.5 L log2 L flops each, the pointwise complex product with the spectrum
    over n + 1 bins (6 flops each), forming the channel (1 multiply per
    position) and the contraction with phi(q) (1 multiply-add per position).
    For n > BLOCK, that count at n = BLOCK for every block pair (I, J) of the
    blocked Toeplitz product (nb = ceil(n / BLOCK) blocks each way) whose
    window of b holds a finite entry (the kernel skips the others), per head.
    """
    if n > BLOCK:
        nb = -(-n // BLOCK)
        pair = conv_stage_flops(B, 1, BLOCK, d, m)
        live = 0
        for h in range(H):
            fin = np.isfinite(b[h]) if b is not None else np.ones(2 * n - 1, bool)
            for D in range(-(nb - 1), nb):
                lo = max(D * BLOCK - (BLOCK - 1), -(n - 1))
                hi = min(D * BLOCK + (BLOCK - 1), n - 1)
                if lo <= hi and fin[lo + n - 1:hi + n].any():
                    live += nb - abs(D)
        return live * pair
    L = 2 * n
    per_channel = 5.0 * L * math.log2(L) + 6.0 * (n + 1) + 4.0 * n
    return B * H * m * (d + 1) * per_channel


def conv_stage_bytes(B, H, n, d, m, s_in) -> float:
    """Algorithmic HBM bytes of the stage: read phi(q), phi(k) (fp32) and v once, the spectrum of c
    (2n complex bins per head), write the n x (d+1) numerators and denominator once."""
    return B * H * (2 * n * m * 4 + n * d * s_in + (d + 1) * n * 4) + H * 2 * n * 8


def feature_stage_roofline(B, H, n, d, m, s_in, ms) -> dict:
    """The feature-map stage of the FFT route (phi(q), phi(k) by MFMA with the exp epilogue, then
    the value columns' maxima and scaled pairs): algorithmic HBM bytes (q, k, W read once, v read
    twice, phi(q), phi(k) and the N-padded value pairs written once) and MFMA flops (2 n m d per
    (batch, head) and input) over the stage's event time, as fractions of the HBM and fp32 MFMA
    peaks."""
    N = 1 << max(0, (n - 1).bit_length())
    pairs = (d + 2) // 2
    hbm = B * H * (2 * n * d * s_in + 2 * n * d * s_in + 2 * m * N * 4 + pairs * N * 8) + H * m * d * 4
    flops = 2.0 * 2 * B * H * n * m * d
    gbs = hbm / (ms * 1e-3) / 1e9
    tf = flops / (ms * 1e-3) / 1e12
    return {"ms": ms, "hbm_bytes": hbm, "achieved_gbs": gbs, "hbm_frac": gbs / PEAK_HBM_GBS,
            "mfma_tflops": tf, "mfma_frac": tf / PEAK_FP32_VECTOR_TFLOPS}


def measured_traffic(kernel: str, workload: str):
    """HBM bytes per launch of `kernel` from the committed profiler record, or None when the
    record is for another workload or the device sources changed since the counters were taken."""
    path = os.path.join(ROOT, "profiles", "traffic.json")
    if not os.path.exists(path):
        return None
    rec = json.load(open(path)).get(kernel)
    if not rec or rec.get("workload") != workload:
        return None
    return rec["bytes"] if device_source_hash() == rec.get("source_sha256") else None


def device_source_hash() -> str:
    """sha256 of the translation units the convolution and the other forward kernels are compiled
    from (kernels.hip, conv_top.hip and the headers they include), comments and blank space
    removed (comment edits keep it; host code in the other sources does not change it)."""
    import hashlib
    import re
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2106_12566_amd", "csrc")
    for name in ("common.hpp", "conv.hpp", "conv_top.hip", "fft.hpp", "kernels.hip", "launch.hpp"):
        f = os.path.join(csrc, name)
        text = open(f).read()
        text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
        text = re.sub(r"//[^\n]*", "", text)
        h.update(re.sub(r"\s+", " ", text).encode())
    return h.hexdigest()


class HipEvents:
    """Raw hipEvent_t handles (the library records them on its own stream)."""

    def __init__(self):
        self.lib = ctypes.CDLL("libamdhip64.so")
        self.lib.hipEventCreate.argtypes = [ctypes.POINTER(ctypes.c_void_p)]
        self.lib.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p, ctypes.c_void_p]
        self.lib.hipEventSynchronize.argtypes = [ctypes.c_void_p]
        self.lib.hipEventDestroy.argtypes = [ctypes.c_void_p]

    def create(self) -> int:
        e = ctypes.c_void_p()
        rc = self.lib.hipEventCreate(ctypes.byref(e))
        if rc != 0:
            raise RuntimeError(f"hipEventCreate failed: {rc}")
        return e.value

    def elapsed_ms(self, a: int, b: int) -> float:
        self.lib.hipEventSynchronize(ctypes.c_void_p(b))
        out = ctypes.c_float()
        rc = self.lib.hipEventElapsedTime(ctypes.byref(out), ctypes.c_void_p(a), ctypes.c_void_p(b))
        if rc != 0:
            raise RuntimeError(f"hipEventElapsedTime failed: {rc}")
        return float(out.value)

    def destroy(self, e: int) -> None:
        self.lib.hipEventDestroy(ctypes.c_void_p(e))


def blas_threads() -> int:
    try:
        from threadpoolctl import threadpool_info
        nums = [p.get("num_threads", 1) for p in threadpool_info() if p.get("user_api") == "blas"]
        if nums:
            return int(max(nums))
    except Exception:
        pass
    return len(os.sched_getaffinity(0))


def cpu_baseline(d: dict, budget_s: float, z_gpu: np.ndarray | None, nprf: bool = False, kind: str = "prf"):
    """Time the fp64 oracle (Eq. (10), O(n^2) per head) on whole (batch, head) units.

    Runs units until `budget_s` of wall time is spent (at least one), and
    extrapolates to the full layer.  Also returns the GPU's per-row normwise
    error on the units the oracle computed.
    """
    import oracle
    wl = d["workload"]
    B, H, n = wl.B, d["H"], wl.n
    if n > BLOCK:
        return cpu_baseline_rows(d, budget_s, z_gpu, nprf=nprf, kind=kind)
    units = [(beta, h) for h in range(H) for beta in range(B)]
    rng = np.random.default_rng([2106, 12566, 99])
    rng.shuffle(units)
    t0 = time.perf_counter()
    done = 0
    worst = 0.0
    for beta, h in units:
        z, _ = oracle.attention(d["q"][beta:beta + 1, h:h + 1], d["k"][beta:beta + 1, h:h + 1],
                                d["v"][beta:beta + 1, h:h + 1], d["b"][h:h + 1],
                                None if kind == "elu" else d["W"][h:h + 1], nprf=nprf, kind=kind)
        done += 1
        if z_gpu is not None:
            num = np.max(np.abs(z_gpu[beta, h] - z[0, 0]), axis=-1)
            worst = max(worst, float(np.max(num / np.max(np.abs(z[0, 0]), axis=-1))))
        if time.perf_counter() - t0 >= budget_s:
            break
    elapsed = time.perf_counter() - t0
    per_unit = elapsed / done
    layer_s = per_unit * B * H
    tokens_per_s = B * n / layer_s
    return {
        "value": tokens_per_s,
        "unit": "tokens/s",
        "cores": blas_threads(),
        "kind": "oracle",
        "sample": f"{done} of {B * H} (batch, head) units of {wl.name}, full Eq. (10) per unit in fp64 "
                  f"({elapsed:.1f} s), extrapolated to the layer; BLAS threads as cores, elementwise exp "
                  f"single-threaded",
        "layer_s": layer_s,
    }, worst, done


def cpu_baseline_rows(d: dict, budget_s: float, z_gpu: np.ndarray | None, nprf: bool = False,
                      kind: str = "prf"):
    """As cpu_baseline, on sampled output rows (the oracle's row-at-a-time form of Eq. (10), O(n)
    per row after one feature map per (batch, head)), for sequences whose n x n weight matrix is
    too large to form on the host."""
    import oracle
    wl = d["workload"]
    B, H, n = wl.B, d["H"], wl.n
    rng = np.random.default_rng([2106, 12566, 98])
    t0 = time.perf_counter()
    done, worst = 0, 0.0
    W = None if kind == "elu" else d["W"]
    while True:
        beta, h = int(rng.integers(B)), int(rng.integers(H))
        rows = [(beta, h, int(i)) for i in rng.integers(0, n, 64)]
        z, _ = oracle.attention_rows(d["q"], d["k"], d["v"], d["b"], W, rows, nprf=nprf, kind=kind)
        done += len(rows)
        if z_gpu is not None:
            got = np.stack([z_gpu[bb, hh, i] for bb, hh, i in rows])
            num = np.max(np.abs(got - z), axis=-1)
            worst = max(worst, float(np.max(num / np.max(np.abs(z), axis=-1))))
        if time.perf_counter() - t0 >= budget_s:
            break
    elapsed = time.perf_counter() - t0
    layer_s = elapsed / done * B * H * n
    return {
        "value": B * n / layer_s,
        "unit": "tokens/s",
        "cores": blas_threads(),
        "kind": "oracle",
        "sample": f"{done} sampled rows of {wl.name} in blocks of 64 rows of one (batch, head), Eq. (10) "
                  f"row by row in fp64 (oracle.attention_rows, {elapsed:.1f} s, one feature map per "
                  f"block), extrapolated to the layer's {B * H * n} rows",
        "layer_s": layer_s,
    }, worst, done


def time_config(wid: int, steps: int, warmup: int, route: str, rows: int = 16) -> dict:
    """One synthetic workload at its stated size: forward time (wall clock over `steps` calls
    after `warmup`, inputs resident on the GPU), stage times from the library's HIP events, the
    route taken, the rows evaluated exactly, the convolution's fraction of the fp32 vector peak
    (FFT route) or the exact-row kernel's fp32 MFMA rate (direct route), and the per-row
    normwise error of `rows` sampled rows (plus the first and last) against the fp64 oracle."""
    import torch
    import oracle
    from paper_2106_12566_amd import krpe, synth
    d = synth.make(wid)
    wl = d["workload"]
    B, H, n, dd, m = wl.B, d["H"], wl.n, wl.d, wl.m
    dev = torch.device("cuda", 0)
    tdt = torch.bfloat16 if wl.qkv_dtype == "bf16" else torch.float32
    q, k, v = (torch.from_numpy(d[x]).to(dev).to(tdt) for x in ("q", "k", "v"))
    b, W = torch.from_numpy(d["b"]).to(dev), torch.from_numpy(d["W"]).to(dev)
    out = torch.empty((B, H, n, dd), dtype=torch.float32, device=dev)
    # a causal workload states its mask (read by the route choice only)
    cz = bool(wl.causal)
    ws = torch.empty(krpe.attention_fwd_workspace(B, H, n, dd, m, route=route, causal=cz), dtype=torch.uint8,
                     device=dev)
    hip = HipEvents()
    events = [[hip.create() for _ in range(krpe.STAGE_EVENTS)] for _ in range(steps)]
    for _ in range(warmup):
        krpe.attention_fwd(q, k, v, b, W, out=out, workspace=ws, route=route, causal=cz)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for s in range(steps):
        krpe.attention_fwd(q, k, v, b, W, out=out, workspace=ws, events=events[s], route=route, causal=cz)
    torch.cuda.synchronize()
    ms = 1e3 * (time.perf_counter() - t0) / steps
    stage = [float(np.mean([hip.elapsed_ms(ev[i], ev[i + 1]) for ev in events])) for i in range(4)]
    for ev in events:
        for e in ev:
            hip.destroy(e)
    used = krpe.attention_fwd_route(B, H, n, dd, m, route=route, causal=cz)
    res = {"workload": wl.name, "B": B, "H": H, "n": n, "m": m, "qkv_dtype": wl.qkv_dtype, "route": used,
           "ms_per_layer": ms, "tokens_per_s": B * n / (ms * 1e-3),
           "exact_rows": krpe.attention_fwd_fixed_rows(ws, B, H, n, dd, m)}
    if used == "fft":
        tf = conv_stage_flops(B, H, n, dd, m, d["b"]) / (stage[2] * 1e-3) / 1e12
        res.update({"conv_ms": stage[2], "conv_tflops": tf, "conv_frac": tf / PEAK_FP32_VECTOR_TFLOPS,
                    "rest_ms": stage[0] + stage[1] + stage[3]})
    else:
        tf = direct_flops(B, H, n, dd, m, d["b"]) / (stage[3] * 1e-3) / 1e12
        res.update({"exact_kernel_ms": stage[3], "exact_kernel_tflops": tf,
                    "exact_kernel_frac": tf / PEAK_FP32_VECTOR_TFLOPS})
    rng = np.random.default_rng([2106, 12566, 97, wid])
    sel = [(0, 0, 0), (B - 1, H - 1, n - 1)] + [(int(rng.integers(B)), int(rng.integers(H)), int(rng.integers(n)))
                                                for _ in range(rows)]
    zr, _ = oracle.attention_rows(d["q"], d["k"], d["v"], d["b"], d["W"], sel)
    zg = out.cpu().numpy()
    got = np.stack([zg[bb, hh, i] for bb, hh, i in sel])
    res["parity_rownorm_err_sampled"] = float(np.max(np.max(np.abs(got - zr), axis=-1)
                                                     / np.max(np.abs(zr), axis=-1)))
    res["parity_rows"] = len(sel)
    del ws, out
    return res


def sweep(lengths, ms, heads, steps: int) -> int:
    """Forward time against sequence length with d = 64 (the paper's speed test setting is one
    head), each m and head count, both routes; one JSON line per (H, n, m, route) on stdout."""
    import torch
    from paper_2106_12566_amd import krpe, synth
    dev = torch.device("cuda", 0)
    for H, n, m in ((H, n, m) for H in heads for n in lengths for m in ms):
        if H * n > 16 * 40000:       # keeps the direct route's share of the sweep to seconds
            continue
        dd = synth.custom(1, H, n, 64, m, seed=n)
        q, k, v, b, W = (torch.from_numpy(dd[x]).to(dev) for x in ("q", "k", "v", "b", "W"))
        for rt in ("fft", "direct"):
            ws = torch.empty(krpe.attention_fwd_workspace(1, H, n, 64, m, route=rt), dtype=torch.uint8,
                             device=dev)
            out = torch.empty_like(q)
            krpe.attention_fwd(q, k, v, b, W, out=out, workspace=ws, route=rt)
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            for _ in range(steps):
                krpe.attention_fwd(q, k, v, b, W, out=out, workspace=ws, route=rt)
            torch.cuda.synchronize()
            ms_call = 1e3 * (time.perf_counter() - t0) / steps
            print(json.dumps({"H": H, "n": n, "m": m, "route": rt, "ms": ms_call,
                              "auto": krpe.attention_fwd_route(1, H, n, 64, m)}), flush=True)
            del ws
    return 0


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", type=int, default=4, help="synthetic workload id (1-7)")
    ap.add_argument("--sweep", action="store_true",
                    help="instead: forward time against n (1k .. 40k), one head, d = 64, m = 32/64/128, "
                         "both routes, one JSON line each")
    ap.add_argument("--sweep-heads", default="1", help="comma-separated head counts of the sweep")
    ap.add_argument("--cpu-budget", type=float, default=12.0, help="seconds of oracle time on the host")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-configs", action="store_true",
                    help="skip the per-workload results (workloads 1-5 at their stated sizes, by the route "
                         "the library picks and, where that is the direct one, by the FFT route too)")
    ap.add_argument("--feature-map", choices=["prf", "trf", "elu"], default="prf",
                    help="feature map of Section 2: PRF (Eq. (5)), trigonometric (2m features) or elu + 1 (m = d)")
    ap.add_argument("--route", choices=["auto", "fft", "direct"], default="fft",
                    help="forward route timed: the FFT route of Sec. 3.2 (default: a step then runs the whole "
                         "path, feature maps, Toeplitz products by FFT and contraction), the direct quadratic "
                         "evaluation, or the one the library picks by its cost model")
    ap.add_argument("--backward", action="store_true",
                    help="also time krpe_attention_bwd (dq, dk, dv, db) on the same inputs, reported in config")
    ap.add_argument("--nprf", action="store_true",
                    help="normalise the rows of q and k first (Algorithm 1's NPRF attention)")
    ap.add_argument("--copy-calibration-mib", type=int, default=0,
                    help="after the timed region, copy a buffer of this size (MiB) 3 times, so that "
                         "profiler byte counters can be scaled by a kernel of known traffic")
    args = ap.parse_args()

    if args.gpus != 1:
        print(f"bench.py: this build runs on one GPU only; --gpus {args.gpus} is not supported "
              "(heads are independent, so a multi-GPU run would shard (batch, head) with no "
              "communication; it is not built)", file=sys.stderr)
        return 2

    import torch
    from paper_2106_12566_amd import krpe, synth

    if not os.path.exists(krpe.lib_path()):
        from paper_2106_12566_amd import build
        build.build()
    krpe.load()
    if not torch.cuda.is_available():
        print("bench.py: no GPU visible", file=sys.stderr)
        return 1
    torch.cuda.set_device(0)
    if args.sweep:
        return sweep([1000, 2000, 4000, 8000, 16000, 24000, 32000, 40000], [32, 64, 128],
                     [int(h) for h in args.sweep_heads.split(",")], args.steps)

    d = synth.make(args.workload)
    wl = d["workload"]
    B, H, n, dd, m = wl.B, d["H"], wl.n, wl.d, wl.m
    tdt = torch.bfloat16 if wl.qkv_dtype == "bf16" else torch.float32
    dev = torch.device("cuda", 0)
    q = torch.from_numpy(d["q"]).to(dev).to(tdt)
    k = torch.from_numpy(d["k"]).to(dev).to(tdt)
    v = torch.from_numpy(d["v"]).to(dev).to(tdt)
    b = torch.from_numpy(d["b"]).to(dev)
    W = torch.from_numpy(d["W"]).to(dev)
    out = torch.empty((B, H, n, dd), dtype=torch.float32, device=dev)
    fm = args.feature_map
    if fm == "elu":
        m = dd                       # elu + 1 has one feature per coordinate
    M = 2 * m if fm == "trf" else m  # features per position
    rt = args.route
    cz = bool(wl.causal)  # a causal workload states its mask (read by the route choice only)
    ws = torch.empty(krpe.attention_fwd_workspace(B, H, n, dd, m, nprf=args.nprf, features=fm, route=rt, causal=cz),
                     dtype=torch.uint8, device=dev)
    print(f"bench: workload {wl.name} B={B} H={H} n={n} d={dd} m={m} {wl.qkv_dtype}", file=sys.stderr,
          flush=True)

    hip = HipEvents()
    events = [[hip.create() for _ in range(krpe.STAGE_EVENTS)] for _ in range(args.steps)]

    for _ in range(args.warmup):
        krpe.attention_fwd(q, k, v, b, W, out=out, workspace=ws, nprf=args.nprf, features=fm, route=rt, causal=cz)
    torch.cuda.synchronize()

    t0 = time.perf_counter()
    for s in range(args.steps):
        krpe.attention_fwd(q, k, v, b, W, out=out, workspace=ws, events=events[s], nprf=args.nprf, features=fm,
                           route=rt, causal=cz)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0

    ms_per_step = 1e3 * elapsed / args.steps
    stage_names = ["spectrum", "feature_map", "conv_contract", "combine"]
    stages = {name: float(np.mean([hip.elapsed_ms(ev[i], ev[i + 1]) for ev in events]))
              for i, name in enumerate(stage_names)}
    # per-call device time (first to last event of each step): spread over the timed steps
    per_call = np.array([hip.elapsed_ms(ev[0], ev[4]) for ev in events])
    call_pct = {f"p{q}": float(np.percentile(per_call, q)) for q in (10, 50, 90)}
    for ev in events:
        for e in ev:
            hip.destroy(e)
    tokens = B * n
    value = tokens / (ms_per_step * 1e-3)

    route_used = krpe.attention_fwd_route(B, H, n, dd, m, nprf=args.nprf, features=fm, route=rt, causal=cz)
    s_in = 2 if wl.qkv_dtype == "bf16" else 4
    if route_used == "fft":
        flops = conv_stage_flops(B, H, n, dd, M, d["b"])
        conv_ms = stages["conv_contract"]
        conv_gbs = conv_stage_bytes(B, H, n, dd, M, s_in) / (conv_ms * 1e-3) / 1e9
        roof = {"bound": "alu", "kernel": "k_conv_contract"}
    else:
        flops = direct_flops(B, H, n, dd, M, d["b"])
        conv_ms = stages["combine"]       # the exact-row kernel evaluates every row
        conv_gbs = None
        roof = {"bound": "mfma", "kernel": "k_fixup"}
    achieved_tflops = flops / (conv_ms * 1e-3) / 1e12
    print(f"bench: {ms_per_step:.3f} ms/step, stages {stages}", file=sys.stderr, flush=True)

    result = {
        "metric": METRIC,
        "value": value,
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": wl.name, "B": B, "H": H, "n": n, "d": dd, "m": m,
                   "qkv_dtype": wl.qkv_dtype, "features": wl.features, "bias": wl.bias,
                   "causal": wl.causal, "nprf": args.nprf, "feature_map": fm, "features_per_position": M,
                   "route": route_used, "blocks": -(-n // BLOCK) if route_used == "fft" else None,
                   "ms_per_layer": ms_per_step, "stages_ms": stages, "call_ms_percentiles": call_pct,
                   "conv_stage_hbm_gbs": conv_gbs,
                   "feature_stage_roofline": (feature_stage_roofline(B, H, n, dd, M, s_in, stages["feature_map"])
                                              if route_used == "fft" and n <= BLOCK and fm == "prf" else None),
                   "exact_rows": krpe.attention_fwd_fixed_rows(ws, B, H, n, dd, m)},
        "roofline": {**roof, "achieved": achieved_tflops,
                     "peak": PEAK_FP32_VECTOR_TFLOPS, "unit": "TFLOP/s",
                     "frac": achieved_tflops / PEAK_FP32_VECTOR_TFLOPS,
                     "traffic": (measured_traffic("k_conv_contract", wl.name)
                                 if fm == "prf" and route_used == "fft" else None)},
    }
    if args.backward:
        if fm != "prf":
            raise SystemExit("the backward pass takes PRF features only")
        dz = torch.randn((B, H, n, dd), generator=torch.Generator(device=dev).manual_seed(2106), device=dev)
        wsb = torch.empty(krpe.attention_bwd_workspace(B, H, n, dd, m, nprf=args.nprf), dtype=torch.uint8,
                          device=dev)
        for _ in range(max(1, args.warmup)):
            krpe.attention_bwd(q, k, v, b, W, dz, workspace=wsb, nprf=args.nprf, with_db=True)
        torch.cuda.synchronize()
        t1 = time.perf_counter()
        for _ in range(args.steps):
            krpe.attention_bwd(q, k, v, b, W, dz, workspace=wsb, nprf=args.nprf, with_db=True)
        torch.cuda.synchronize()
        result["config"]["backward_ms"] = 1e3 * (time.perf_counter() - t1) / args.steps
        print(f"bench: backward {result['config']['backward_ms']:.3f} ms/step", file=sys.stderr, flush=True)
        del wsb
    if args.copy_calibration_mib > 0:
        src = torch.ones(args.copy_calibration_mib << 18, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        result["config"]["copy_calibration_bytes"] = src.numel() * 4
    if not args.no_configs and fm == "prf" and not args.nprf and rt != "direct":
        per = {}
        for wid in range(1, 6):
            res = time_config(wid, max(3, min(args.steps, 10)), max(1, min(args.warmup, 3)), "auto")
            if res["route"] == "direct":
                fft = time_config(wid, max(3, min(args.steps, 10)), max(1, min(args.warmup, 3)), "fft")
                res["fft_route"] = {k2: fft[k2] for k2 in ("ms_per_layer", "conv_ms", "conv_frac", "exact_rows",
                                                            "parity_rownorm_err_sampled")}
            per[str(wid)] = res
            print(f"bench: workload {wid} {res['workload']}: {res['ms_per_layer']:.3f} ms/layer ({res['route']})",
                  file=sys.stderr, flush=True)
        result["config"]["per_workload"] = per
    if not args.no_cpu_baseline:
        z_gpu = out.cpu().numpy()
        cb, err, units = cpu_baseline(d, args.cpu_budget, z_gpu, nprf=args.nprf, kind=fm)
        result["cpu_baseline"] = {k2: cb[k2] for k2 in ("value", "unit", "cores", "kind", "sample")}
        result["config"]["parity_rownorm_err"] = err
        result["config"]["parity_units"] = units
    print(json.dumps(result), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
