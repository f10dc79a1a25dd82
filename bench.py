"""Benchmark of the n:m:g hot path on one MI355X.

One step = the whole path on one batch: nmg_compress of a dense weight
(group score, top-n select, pack) followed by nmg_spmm of the packed weight
with a 4096-token activation.  Workload: BERT-base FFN up-projection,
W 3072 x 768 fp32 ~ N(0, 0.02^2), 1:4 (75% sparse), g = 8, X 768 x 4096 fp32
~ N(0, 1); synthetic, seeded.

Inputs are resident in HBM before timing starts.  Steps rotate over enough
distinct buffer sets (> 1 GB in total) that the 256 MB Infinity Cache cannot
serve a step from the previous visit.

Prints ONE JSON line (rank 0).  `value` = useful GFLOP (2 N nnz of the sparse
weight) per step / step time; `roofline` describes nmg_spmm, the dominant
kernel, from HIP events around each of its launches in the timed region;
`cpu_baseline` times the CPU oracle on a bounded sample of the same workload.
"""
from __future__ import annotations

import argparse
import json
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "nmg_spmm useful GFLOP/s + % HBM roofline, BERT-base FFN 3072x768 @ 75% sparse"
HBM_PEAK_GBS = 8000.0           # MI355X HBM3E, GB/s
FP32_MFMA_PEAK_TFLOPS = 157.3   # MI355X dense binary32 matrix peak
FP32_VALU_PEAK_TFLOPS = 78.6    # binary32 vector FMA without packed math (2 FLOP/lane/clk)
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "spmm_bert-ffn-up_traffic.txt")


def parse():
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--kernel", choices=("auto", "mfma", "valu"), default="auto")
    ap.add_argument("--rotate-mb", type=float, default=1100.0,
                    help="total size of the rotated buffer sets")
    ap.add_argument("--cpu-seconds", type=float, default=12.0,
                    help="approximate CPU time budget of the oracle baseline")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    return ap.parse_args()


def source_digest() -> str:
    import hashlib
    with open(os.path.join(ROOT, "paper_2304_07613_amd", "csrc", "nmg.hip"), "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()[:16]


def stored_traffic(digest: str):
    """HBM bytes per spmm launch from the committed rocprofv3 counter summary,
    if it was taken on the current kernel source; else None."""
    try:
        with open(TRAFFIC_FILE) as f:
            text = f.read()
    except OSError:
        return None
    kv = dict(re.findall(r"^(\w+)\s*=\s*(\S+)\s*$", text, re.M))
    if kv.get("source_sha") != digest:
        return None
    try:
        return float(kv["hbm_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU; --gpus {args.gpus} is not supported "
              f"(the path shards by tokens with no communication, see DESIGN.md)",
              file=sys.stderr)
        sys.exit(2)

    import torch

    from paper_2304_07613_amd import nmg, synth

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    nmg.lib()  # raises if the HIP library is missing: there is no fallback
    dev = torch.device("cuda:0")
    wl = synth.FFN_UP
    lin = wl.layers[0]
    L = nmg.Layout(lin.M, lin.K, lin.n, lin.m, lin.g, lin.dtype)
    kernel = nmg.auto_kernel(L, lin.N) if args.kernel == "auto" else args.kernel

    # ---- resident, rotated inputs and outputs
    es = 4
    set_bytes = (lin.M * lin.K + lin.K * lin.N + lin.M * lin.N + L.M * L.C * L.n) * es + \
        (L.M // L.g) * L.C * L.n
    n_sets = max(2, int(args.rotate_mb * 1e6 // set_bytes) + 1)
    sets = []
    for i in range(n_sets):
        W, X = synth.layer_inputs(2, i, lin)
        W, X = W.to(dev), X.to(dev)
        v = torch.empty(L.values_shape, dtype=lin.dtype, device=dev)
        idx = torch.empty(L.indices_shape, dtype=torch.uint8, device=dev)
        Y = torch.empty((lin.M, lin.N), dtype=lin.dtype, device=dev)
        sets.append((W, X, v, idx, Y))
    torch.cuda.synchronize()

    def step(i):
        W, X, v, idx, Y = sets[i % n_sets]
        nmg.compress_into(L, W, v, idx)
        nmg.spmm_into(L, v, idx, X, Y, kernel)

    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()

    # ---- timed region: K steps, events around every launch.  The ctypes
    # arguments are marshalled beforehand so the host never starves the GPU.
    import ctypes
    stream = torch.cuda.current_stream(dev)
    lib = nmg.lib()
    sp = ctypes.c_void_p(stream.cuda_stream)
    lref = ctypes.byref(L.c)
    vp = lambda t: ctypes.c_void_p(t.data_ptr())
    calls = [((lref, vp(W), lin.K, vp(v), vp(idx), sp),
              (lref, nmg.KERNELS[kernel], vp(v), vp(idx), vp(X), lin.N, lin.N, vp(Y), lin.N, sp))
             for (W, X, v, idx, Y) in sets]
    compress_c, spmm_c = lib.nmg_compress, lib.nmg_spmm_with
    K = args.steps
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(K)]
    status = []
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    start = torch.cuda.Event(enable_timing=True)
    stop = torch.cuda.Event(enable_timing=True)
    start.record(stream)
    for s in range(K):
        ca, sa = calls[s % n_sets]
        ev[s][0].record(stream)
        status.append(compress_c(*ca))
        ev[s][1].record(stream)
        status.append(spmm_c(*sa))
        ev[s][2].record(stream)
    stop.record(stream)
    torch.cuda.synchronize()
    if any(status):
        raise nmg.NmgError(next(x for x in status if x), "timed step")
    wall = time.perf_counter() - t0
    ms_step = start.elapsed_time(stop) / K
    compress_ms = sum(e[0].elapsed_time(e[1]) for e in ev) / K
    spmm_ms = sum(e[1].elapsed_time(e[2]) for e in ev) / K

    useful_flop = lin.useful_flop
    value = useful_flop / (ms_step * 1e-3) / 1e9
    alg_bytes = (L.M * L.C * L.n) * es + (L.M // L.g) * L.C * L.n + lin.K * lin.N * es + \
        lin.M * lin.N * es
    spmm_tflops = useful_flop / (spmm_ms * 1e-3) / 1e12
    peak = FP32_MFMA_PEAK_TFLOPS if kernel == "mfma" else FP32_VALU_PEAK_TFLOPS
    digest = source_digest()
    traffic = stored_traffic(digest)
    compress_bytes = lin.M * lin.K * es + (L.M * L.C * L.n) * es + (L.M // L.g) * L.C * L.n

    # ---- kernel-family evidence (outside the timed region)
    family = {}
    W0, X0, v0, idx0, Y0 = sets[0]
    nmg.compress_into(L, W0, v0, idx0)
    for fam in ("mfma", "valu"):
        try:
            for _ in range(3):
                nmg.spmm_into(L, v0, idx0, X0, Y0, fam)
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            reps = 20
            e0.record(stream)
            for r in range(reps):
                Wr, Xr, vr, idxr, Yr = sets[r % n_sets]
                nmg.spmm_into(L, vr, idxr, Xr, Yr, fam)
            e1.record(stream)
            torch.cuda.synchronize()
            family[fam] = round(e0.elapsed_time(e1) / reps * 1e3, 2)
        except nmg.NmgError:
            family[fam] = None
    nmg.spmm_into(L, v0, idx0, X0, Y0, kernel)  # set 0 holds the timed kernel's output again
    torch.cuda.synchronize()

    out = {
        "metric": METRIC,
        "value": round(value, 1),
        "unit": "GFLOP/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": wl.key, "M": lin.M, "K": lin.K, "N": lin.N, "n": lin.n,
                   "m": lin.m, "g": lin.g, "kernel": kernel, "rotated_sets": n_sets,
                   "step": "nmg_compress + nmg_spmm"},
        "roofline": {
            "kernel": f"k_spmm_{kernel}",
            "bound": "mfma" if kernel == "mfma" else "alu",
            "achieved": round(spmm_tflops, 2),
            "peak": peak,
            "unit": "TFLOP/s",
            "frac": round(spmm_tflops / peak, 4),
            "traffic": traffic,
            "algorithmic_bytes": alg_bytes,
            "hbm_frac": round(alg_bytes / (spmm_ms * 1e-3) / (HBM_PEAK_GBS * 1e9), 4),
        },
        "spmm_us": round(spmm_ms * 1e3, 2),
        "spmm_gflops": round(useful_flop / (spmm_ms * 1e-3) / 1e9, 1),
        "compress_us": round(compress_ms * 1e3, 2),
        "compress_gbs": round(compress_bytes / (compress_ms * 1e-3) / 1e9, 1),
        "compress_hbm_frac": round(compress_bytes / (compress_ms * 1e-3) / (HBM_PEAK_GBS * 1e9), 4),
        "spmm_us_by_kernel": family,
        "wall_s_timed": round(wall, 4),
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(args, lin, L, sets[0], dev)
    print(json.dumps(out))


def cpu_baseline(args, lin, L, set0, dev):
    """The CPU oracle (test infrastructure, untuned) on a bounded sample of the
    same workload, on this host's cores; also spot-checks the GPU output of
    that sample against it."""
    import numpy as np

    import oracle

    W, X, v, idx, Y = set0
    Wn, Xn = W.cpu().numpy(), X.cpu().numpy()
    cores = len(os.sched_getaffinity(0))
    t0 = time.perf_counter()
    rv, ridx = oracle.compress(Wn, lin.n, lin.m, lin.g)
    t_compress = time.perf_counter() - t0
    # calibrate: rows of the product that fit the time budget
    probe = lin.g * 8
    t0 = time.perf_counter()
    oracle.spmm(rv[:probe], ridx[:probe // lin.g], Xn, lin.K, lin.n, lin.m, lin.g, cores)
    t_probe = time.perf_counter() - t0
    rows = int(args.cpu_seconds / max(t_probe, 1e-6) * probe) // lin.g * lin.g
    rows = max(lin.g, min(lin.M, rows))
    t0 = time.perf_counter()
    Yref, B = oracle.spmm(rv[:rows], ridx[:rows // lin.g], Xn, lin.K, lin.n, lin.m, lin.g, cores)
    t_spmm = time.perf_counter() - t0
    flop = 2 * lin.N * rows * L.C * L.n
    # spot check of the GPU packing and product on the sample
    nmg_compress_ok = bool(np.array_equal(idx.cpu().numpy(), ridx))
    Yg = Y[:rows].cpu().numpy().astype(np.float64)
    prod_ok = bool((np.abs(Yg - Yref) <= 1e-5 * B).all())
    return {
        "value": round(flop / t_spmm / 1e9, 3),
        "unit": "GFLOP/s",
        "cores": cores,
        "kind": "oracle",
        "sample": f"oracle compress of the full 3072x768 weight ({t_compress:.2f} s) and the "
                  f"binary64 oracle product for the first {rows} of 3072 rows x 4096 tokens "
                  f"({t_spmm:.2f} s, OpenMP over rows)",
        "gpu_matches_sample": nmg_compress_ok and prod_ok,
    }


if __name__ == "__main__":
    main()
