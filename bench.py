"""Benchmark of the n:m:g hot path on one MI355X.

One step = the whole path on one batch: nmg_compress of a dense weight
(group score, top-n select, pack) followed by nmg_spmm of the packed weight
with a 4096-token activation.  Default workload: BERT-base FFN up-projection,
W 3072 x 768 fp32 ~ N(0, 0.02^2), 1:4 (75% sparse), g = 8, X 768 x 4096 fp32
~ N(0, 1); synthetic, seeded.

Inputs are resident in HBM before timing starts.  The other kernel families
are timed on the same buffers first (the evidence behind the automatic
choice; --no-family skips them), then the W untimed warmup steps run, then
the K timed steps.  The GPU reaches its sustained clock only after tens of
milliseconds of work: measured without the family timings, 10 warmup steps
leave the timed steps 13% slower, 100 steps 8%, 400 or more none; the family
timings (about 0.1 s of GPU work) come first so that a short warmup is timed
at that clock as well.  Steps rotate over enough
distinct buffer sets (> 1 GB in total) that the 256 MB Infinity Cache cannot
serve a step from the previous visit.

Default output: ONE JSON line.  `value` = useful GFLOP (2 N nnz of the sparse
weight) per step / step time, from K whole steps launched back to back with
HIP events only at the two ends.  `roofline` describes nmg_spmm, the dominant
kernel: its average launch duration is measured with HIP events around K
back-to-back launches of it alone over the same rotated sets (events between
every kernel would themselves add several microseconds of idle per launch).
`cpu_baseline` times the CPU oracle on a bounded sample of the same workload.

Other modes (not the headline): --workload 1|3 (the other single layers),
--sweep (the n:m x g sweep, one line per point), --stack (the 12-layer fp16
BERT-base linear stack), --stack-layer 0..3 (one of its projections alone,
like --workload), --copy-calibration (a plain device copy of known size, for
scaling the HBM byte counters).
"""
from __future__ import annotations

import argparse
import ctypes
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
FP16_MFMA_PEAK_TFLOPS = 2500.0  # MI355X dense binary16 matrix peak
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "spmm_bert-ffn-up_traffic.txt")
KERNEL_SYMBOL = {"mfma_scalar": "k_spmm_mfma_s", "mfma_general": "k_spmm_mfma",
                 "mfma_f16": "k_spmm_mfma_h", "mfma_direct": "k_spmm_mfma_d",
                 "smfmac_f16": "k_spmm_smfmac", "valu_staged": "k_spmm_valu_s",
                 "valu": "k_spmm_valu", "mfma_wide": "k_spmm_x16", "mfma_split": "k_spmm_x16",
                 "mfma_expand": "k_spmm_mfma_s"}


def parse():
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=1000)
    ap.add_argument("--kernel", choices=("auto", "mfma", "valu", "mfma_general", "mfma_scalar",
                                         "mfma_f16", "mfma_direct", "smfmac_f16",
                                         "valu_staged", "mfma_wide", "mfma_split",
                                         "mfma_expand"),
                    default="auto")
    ap.add_argument("--workload", type=int, choices=(1, 2, 3), default=2)
    ap.add_argument("--sweep", action="store_true")
    ap.add_argument("--stack", action="store_true")
    ap.add_argument("--stack-kernels", default=None,
                    help="with --stack: name=family items, comma-separated (qkv, ao, up, down)")
    ap.add_argument("--stack-layer", type=int, choices=(0, 1, 2, 3), default=None,
                    help="one projection of the fp16 stack (QKV, attention-out, FFN up, FFN down) "
                         "timed like --workload, with the other kernel families")
    ap.add_argument("--chunked", action="store_true",
                    help="the paper's chunked layout beside the group layout on the sweep shapes")
    ap.add_argument("--copy-calibration", action="store_true")
    ap.add_argument("--rotate-mb", type=float, default=1100.0,
                    help="total size of the rotated buffer sets")
    ap.add_argument("--cpu-seconds", type=float, default=10.0,
                    help="approximate CPU time budget of the oracle baseline")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-family", action="store_true",
                    help="skip timing the other kernel family")
    return ap.parse_args()


# The sources that make the profiled kernels (the headline product and the
# converter): the stored traffic figure holds while these are unchanged.
TRAFFIC_SOURCES = ("common.hpp", "k_spmm_mfma_s.hpp", "k_spmm_mfma_s_f32_u8.hip",
                   "k_elementwise.hip")


def traffic_digest() -> str:
    """Digest of the profiled kernels' sources (names and contents) and the header."""
    import hashlib
    from paper_2304_07613_amd import build
    h = hashlib.sha256()
    for p in [os.path.join(build.CSRC, f) for f in TRAFFIC_SOURCES] + [build.HEADER]:
        h.update(os.path.relpath(p, ROOT).encode())
        with open(p, "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def stored_traffic(digest: str):
    """HBM bytes per spmm launch from the committed rocprofv3 counter summary,
    if it was taken on the current sources of the profiled kernels; else None."""
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


class Ctx:
    def __init__(self):
        import torch

        from paper_2304_07613_amd import nmg, synth
        assert torch.cuda.is_available(), "bench.py needs a GPU"
        nmg.lib()  # raises if the HIP library is missing: there is no fallback
        self.torch, self.nmg, self.synth = torch, nmg, synth
        self.dev = torch.device("cuda:0")
        self.stream = torch.cuda.current_stream(self.dev)
        self.sp = ctypes.c_void_p(self.stream.cuda_stream)

    def event(self):
        return self.torch.cuda.Event(enable_timing=True)


def layer_bytes(lin, L):
    es = lin.dtype.itemsize
    packed = L.M * L.C * L.n * es + (L.M // L.g) * L.C * L.n
    return {
        "spmm": packed + lin.K * lin.N * es + lin.M * lin.N * es,
        "compress": lin.M * lin.K * es + packed,
        "set": lin.M * lin.K * es + packed + lin.K * lin.N * es + lin.M * lin.N * es,
    }


def time_layer(ctx, args, workload, layer_no, lin, kernel_req):
    """Rotated resident buffers, warmup, then K timed steps of compress + spmm
    with HIP events around every launch.  Returns timings and the buffers."""
    torch, nmg = ctx.torch, ctx.nmg
    L = nmg.Layout(lin.M, lin.K, lin.n, lin.m, lin.g, lin.dtype)
    kernel = nmg.auto_kernel(L, lin.N) if kernel_req == "auto" else kernel_req
    nb = layer_bytes(lin, L)
    n_sets = max(2, int(args.rotate_mb * 1e6 // nb["set"]) + 1)
    sets = []
    for i in range(n_sets):
        W, X = ctx.synth.layer_inputs(workload, layer_no + 100 * i, lin)
        W, X = W.to(ctx.dev), X.to(ctx.dev)
        v = torch.empty(L.values_shape, dtype=lin.dtype, device=ctx.dev)
        idx = torch.empty(L.indices_shape, dtype=torch.uint8, device=ctx.dev)
        Y = torch.empty((lin.M, lin.N), dtype=lin.dtype, device=ctx.dev)
        sets.append((W, X, v, idx, Y))
    lib = nmg.lib()
    lref = ctypes.byref(L.c)
    vp = lambda t: ctypes.c_void_p(t.data_ptr())
    # arguments marshalled beforehand so the host never starves the GPU
    calls = [((lref, vp(W), lin.K, vp(v), vp(idx), ctx.sp),
              (lref, nmg.KERNELS[kernel], vp(v), vp(idx), vp(X), lin.N, lin.N, vp(Y), lin.N,
               ctx.sp)) for (W, X, v, idx, Y) in sets]
    compress_c, spmm_c = lib.nmg_compress, lib.nmg_spmm_with
    status = []
    family = None
    if not args.no_family:
        # the other kernel families on the same sets (the evidence behind the
        # automatic choice), before the timed region: on a fresh GPU this
        # also brings the clock to its sustained level
        status += [compress_c(*ca) for ca, _ in calls]
        family = family_times(ctx, L, sets, kernel)
    for s in range(args.warmup):
        ca, sa = calls[s % n_sets]
        status += [compress_c(*ca), spmm_c(*sa)]
    torch.cuda.synchronize()

    K = args.steps
    # (1) the timed region: K whole steps back to back, events only at its ends
    start, stop = ctx.event(), ctx.event()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    start.record(ctx.stream)
    for s in range(K):
        ca, sa = calls[s % n_sets]
        status.append(compress_c(*ca))
        status.append(spmm_c(*sa))
    stop.record(ctx.stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    # (2) each kernel's average launch duration: K launches of it alone, back to
    # back over the same rotated sets, between two events (launch gaps included)
    def kernel_ms(which):
        e0, e1 = ctx.event(), ctx.event()
        e0.record(ctx.stream)
        for s in range(K):
            ca, sa = calls[s % n_sets]
            status.append(compress_c(*ca) if which == 0 else spmm_c(*sa))
        e1.record(ctx.stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / K
    compress_ms = kernel_ms(0)
    spmm_ms = kernel_ms(1)
    if any(status):
        raise nmg.NmgError(next(x for x in status if x), "timed step")
    res = {
        "L": L, "kernel": kernel, "n_sets": n_sets, "sets": sets, "wall": wall,
        "ms_step": start.elapsed_time(stop) / K,
        "compress_ms": compress_ms,
        "spmm_ms": spmm_ms,
        "bytes": nb,
    }
    if family is not None:
        res["family"] = family
    return res


def family_times(ctx, L, sets, kernel, reps=50):
    """Mean spmm time of each kernel family on the same rotated sets (outside
    the timed region): the evidence behind the automatic choice."""
    torch, nmg = ctx.torch, ctx.nmg
    out = {}
    for fam in ("smfmac_f16", "mfma_f16", "mfma_wide", "mfma_direct", "mfma_scalar",
                "mfma_general", "mfma_split", "mfma_expand", "valu_staged", "valu"):
        try:
            for r in range(3):
                W, X, v, idx, Y = sets[r % len(sets)]
                nmg.spmm_into(L, v, idx, X, Y, fam)
            e0, e1 = ctx.event(), ctx.event()
            e0.record(ctx.stream)
            for r in range(reps):
                W, X, v, idx, Y = sets[r % len(sets)]
                nmg.spmm_into(L, v, idx, X, Y, fam)
            e1.record(ctx.stream)
            torch.cuda.synchronize()
            out[fam] = round(e0.elapsed_time(e1) / reps * 1e3, 2)
            if fam in nmg.X16_KERNELS:
                # the per-call figure above includes making the prepared
                # operands; the product alone on operands prepared beforehand
                out[fam + "_per_call"] = out[fam]
                prep = [nmg.x16_prepare(v, idx, L) for (W, X, v, idx, Y) in sets]
                e0.record(ctx.stream)
                for r in range(reps):
                    W, X, v, idx, Y = sets[r % len(sets)]
                    nmg.spmm_x16_epilogue(L, prep[r % len(sets)], X, Y=Y)
                e1.record(ctx.stream)
                torch.cuda.synchronize()
                out[fam] = round(e0.elapsed_time(e1) / reps * 1e3, 2)
        except nmg.NmgError:
            out[fam] = None
    for r in range(len(sets)):  # every set holds the chosen kernel's output again
        W, X, v, idx, Y = sets[r]
        nmg.spmm_into(L, v, idx, X, Y, kernel)
    torch.cuda.synchronize()
    return out


def layer_record(lin, res):
    kernel = res["kernel"]
    spmm_s = res["spmm_ms"] * 1e-3
    tflops = lin.useful_flop / spmm_s / 1e12
    matrix = kernel.startswith("mfma") or kernel.startswith("smfmac")
    # binary16 kernels on the binary16 matrix instructions; the others on the
    # binary32 ones; the vector kernels without packed math
    if kernel in ("mfma_f16", "smfmac_f16", "mfma_wide"):
        peak = FP16_MFMA_PEAK_TFLOPS
    else:
        peak = FP32_MFMA_PEAK_TFLOPS if matrix else FP32_VALU_PEAK_TFLOPS
    rec = {
        "roofline": {
            "kernel": KERNEL_SYMBOL.get(kernel, kernel),
            "bound": "mfma" if matrix else "alu",
            "achieved": round(tflops, 2),
            "peak": peak,
            "unit": "TFLOP/s",
            "frac": round(tflops / peak, 4),
            "traffic": None,
            "algorithmic_bytes": res["bytes"]["spmm"],
            "hbm_frac": round(res["bytes"]["spmm"] / spmm_s / (HBM_PEAK_GBS * 1e9), 4),
        },
        "spmm_us": round(res["spmm_ms"] * 1e3, 2),
        "spmm_gflops": round(lin.useful_flop / spmm_s / 1e9, 1),
        "compress_us": round(res["compress_ms"] * 1e3, 2),
        "compress_gbs": round(res["bytes"]["compress"] / (res["compress_ms"] * 1e-3) / 1e9, 1),
        "compress_hbm_frac": round(res["bytes"]["compress"] / (res["compress_ms"] * 1e-3) /
                                   (HBM_PEAK_GBS * 1e9), 4),
    }
    if "family" in res:
        rec["spmm_us_by_kernel"] = res["family"]
    return rec


def cpu_baseline(args, lin, L, set0):
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
    probe = lin.g * max(1, 64 // lin.g)
    t0 = time.perf_counter()
    oracle.spmm(rv[:probe], ridx[:probe // lin.g], Xn, lin.K, lin.n, lin.m, lin.g, cores)
    t_probe = time.perf_counter() - t0
    rows = int(args.cpu_seconds / max(t_probe, 1e-6) * probe) // lin.g * lin.g
    rows = max(lin.g, min(lin.M, rows))
    # repeat the sample until the budget of CPU work has been timed
    reps, t_spmm = 0, 0.0
    while reps == 0 or (t_spmm < args.cpu_seconds and reps < 1000):
        t0 = time.perf_counter()
        Yref, B = oracle.spmm(rv[:rows], ridx[:rows // lin.g], Xn, lin.K, lin.n, lin.m, lin.g,
                              cores)
        t_spmm += time.perf_counter() - t0
        reps += 1
    flop = 2 * lin.N * rows * L.C * L.n * reps
    # the same oracle on one thread, over a sample sized for about a third of
    # the budget
    rows1 = int(args.cpu_seconds / 3 / max(t_probe * cores, 1e-6) * probe) // lin.g * lin.g
    rows1 = max(lin.g, min(lin.M, rows1))
    t0 = time.perf_counter()
    oracle.spmm(rv[:rows1], ridx[:rows1 // lin.g], Xn, lin.K, lin.n, lin.m, lin.g, 1)
    t_one = time.perf_counter() - t0
    flop1 = 2 * lin.N * rows1 * L.C * L.n
    ok = bool(np.array_equal(idx.cpu().numpy(), ridx))
    Yg = Y[:rows].cpu().numpy().astype(np.float64)
    tol = 1e-5 if lin.dtype.itemsize == 4 else 2e-2
    ok = ok and bool((np.abs(Yg - Yref) <= tol * B).all())
    return {
        "value": round(flop / t_spmm / 1e9, 3),
        "unit": "GFLOP/s",
        "cores": cores,
        "kind": "oracle",
        "sample": f"oracle compress of the full {lin.M}x{lin.K} weight ({t_compress:.3f} s), then "
                  f"the binary64 oracle product of the first {rows} of {lin.M} rows x {lin.N} "
                  f"tokens, {reps} time(s) ({t_spmm:.2f} s, OpenMP over rows on {cores} threads)",
        "gpu_matches_sample": ok,
        "single_thread": {"value": round(flop1 / t_one / 1e9, 3), "unit": "GFLOP/s",
                          "sample": f"the first {rows1} rows x {lin.N} tokens once "
                                    f"({t_one:.2f} s, one thread)"},
        "cpu_model": cpu_model(),
    }


def cpu_model() -> str:
    """The host CPU's model name, from /proc/cpuinfo."""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def headline(ctx, args):
    workload, layer = (4, args.stack_layer) if args.stack_layer is not None else (args.workload, 0)
    wl = ctx.synth.WORKLOADS[workload]
    lin = wl.layers[layer]
    res = time_layer(ctx, args, workload, layer, lin, args.kernel)
    rec = layer_record(lin, res)
    if workload == 2:
        rec["roofline"]["traffic"] = stored_traffic(traffic_digest())
    out = {
        "metric": METRIC if workload == 2 else "nmg_spmm useful GFLOP/s",
        "value": round(lin.useful_flop / (res["ms_step"] * 1e-3) / 1e9, 1),
        "unit": "GFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(res["ms_step"], 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32" if lin.dtype.itemsize == 4 else "f16",
        "data": "synthetic",
        "config": {"workload": wl.key if workload != 4 else f"{wl.key}:{lin.name}",
                   "M": lin.M, "K": lin.K, "N": lin.N, "n": lin.n, "m": lin.m, "g": lin.g,
                   "kernel": res["kernel"],
                   "rotated_sets": res["n_sets"], "step": "nmg_compress + nmg_spmm"},
        **rec,
        "wall_s_timed": round(res["wall"], 4),
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(args, lin, res["L"], res["sets"][0])
    print(json.dumps(out), flush=True)


def sweep(ctx, args):
    for j, lin in enumerate(ctx.synth.SWEEP.layers):
        res = time_layer(ctx, args, 5, j, lin, args.kernel)
        rec = layer_record(lin, res)
        W, v = res["sets"][0][0], res["sets"][0][2]
        energy = float(v.double().abs().sum() / W.double().abs().sum())
        print(json.dumps({"metric": "nmg_spmm useful GFLOP/s", "point": lin.name,
                          "value": rec["spmm_gflops"], "unit": "GFLOP/s",
                          "kernel": res["kernel"], "energy": round(energy, 4),
                          "ms_per_step": round(res["ms_step"], 5), **rec}), flush=True)
        del res


def chunked(ctx, args):
    """The paper's chunked layout beside the group layout on the sweep shapes
    it fits (K % m == 0, M % (C(m,n) * g) == 0): kept magnitude of the group
    layout, of the chunked layout's greedy and of its swap search; converter
    and product times (events around `reps` back-to-back launches each)."""
    torch, nmg, synth = ctx.torch, ctx.nmg, ctx.synth
    import math
    reps = max(3, args.steps // 20)

    def timed(fn):
        fn()
        torch.cuda.synchronize()
        a, b = ctx.event(), ctx.event()
        a.record(ctx.stream)
        for _ in range(reps):
            fn()
        b.record(ctx.stream)
        torch.cuda.synchronize()
        return a.elapsed_time(b) / reps * 1e3  # us

    for j, lin in enumerate(synth.SWEEP.layers):
        S = math.comb(lin.m, lin.n) * lin.g
        if lin.n == lin.m or lin.K % lin.m or lin.M % S or S > 256:
            continue
        W, X = synth.layer_inputs(5, j, lin)
        W, X = W.to(ctx.dev), X.to(ctx.dev)
        total = float(W.double().abs().sum())
        v, idx, L = nmg.compress(W, lin.n, lin.m, lin.g)
        pv, pidx, PL = nmg.p_compress(W, lin.n, lin.m, lin.g)
        rv, ridx = nmg.p_refine(W, pidx, PL)
        e = lambda vals: round(float(vals.double().abs().sum()) / total, 5)
        rec = {"mode": "chunked-vs-group", "point": lin.name, "shape": [lin.M, lin.K, lin.N],
               "rows_per_chunk": S,
               "energy_group": e(v), "energy_chunked_greedy": e(pv), "energy_chunked_swap": e(rv),
               "us_compress_group": round(timed(lambda: nmg.compress(W, lin.n, lin.m, lin.g)), 2),
               "us_compress_chunked": round(timed(lambda: nmg.p_compress(W, lin.n, lin.m, lin.g)), 2),
               "us_swap_search": round(timed(lambda: nmg.p_refine(W, pidx, PL)), 2),
               "us_spmm_group": round(timed(lambda: nmg.spmm(v, idx, X, L)), 2),
               "us_spmm_chunked": round(timed(lambda: nmg.p_spmm(pv, pidx, X, PL)), 2),
               "us_spmm_chunked_valu": round(timed(lambda: nmg.p_spmm(pv, pidx, X, PL, "valu")), 2),
               "us_spmm_chunked_mfma": round(timed(lambda: nmg.p_spmm(pv, pidx, X, PL, "mfma")), 2),
               "group_kernel": nmg.auto_kernel(L, lin.N)}
        rec["tflops_spmm_chunked"] = round(lin.useful_flop / rec["us_spmm_chunked"] / 1e6, 2)
        rec["tflops_spmm_group"] = round(lin.useful_flop / rec["us_spmm_group"] / 1e6, 2)
        print(json.dumps(rec), flush=True)


def stack(ctx, args):
    """Forward of the 12-layer fp16 linear stack (48 sparse products, 12 GELU,
    24 residual sums), weights compressed once beforehand."""
    torch, nmg, synth = ctx.torch, ctx.nmg, ctx.synth
    from paper_2304_07613_amd import stack as stack_mod
    from paper_2304_07613_amd.stack import LinearStack
    kernels = dict(stack_mod.DEFAULT_KERNELS)
    for item in filter(None, (args.stack_kernels or "").split(",")):
        name, _, fam = item.partition("=")
        if name not in kernels or fam not in nmg.KERNELS:
            raise SystemExit(f"--stack-kernels: bad item {item!r}")
        kernels[name] = fam
    st = LinearStack.from_workload(4, nmg, keep_dense=False, kernels=kernels)
    torch.cuda.synchronize()
    x = synth.normal((synth.BERT_HIDDEN, synth.BERT_TOKENS), synth.seed_for(4, 0, "X"), 1.0,
                     torch.float16).to(ctx.dev)
    for _ in range(max(1, args.warmup // 5)):
        st.forward(x)
    torch.cuda.synchronize()
    reps = max(1, args.steps // 20)
    a, b = ctx.event(), ctx.event()
    a.record(ctx.stream)
    for _ in range(reps):
        y = st.forward(x)
    b.record(ctx.stream)
    torch.cuda.synchronize()
    ms = a.elapsed_time(b) / reps
    # the same forward captured in a HIP graph and replayed (no host launches)
    graph, _ = st.capture(x)
    graph.replay()
    torch.cuda.synchronize()
    a.record(ctx.stream)
    for _ in range(reps):
        graph.replay()
    b.record(ctx.stream)
    torch.cuda.synchronize()
    ms_graph = a.elapsed_time(b) / reps
    flop = 12 * sum(l.useful_flop for l in synth.bert_stack_layers())
    print(json.dumps({"metric": "BERT-base linear stack forward, useful GFLOP/s",
                      "value": round(flop / (ms * 1e-3) / 1e9, 1), "unit": "GFLOP/s",
                      "ms_per_forward": round(ms, 4),
                      "ms_per_forward_graph": round(ms_graph, 4),
                      "tokens_per_s": round(synth.BERT_TOKENS / (ms * 1e-3), 1),
                      "dtype": "f16 (binary32 accumulate)", "layers": 12, "reps": reps,
                      "kernels": kernels,
                      "finite": bool(torch.isfinite(y.float()).all())}), flush=True)


def copy_calibration(ctx, args):
    """A plain device-to-device copy of known size (torch's copy kernel),
    256 MiB per launch over rotating buffers, for scaling FETCH_SIZE and
    WRITE_SIZE."""
    torch = ctx.torch
    nbytes = 256 << 20
    bufs = [torch.empty(nbytes // 4, dtype=torch.float32, device=ctx.dev).fill_(1.0)
            for _ in range(8)]
    torch.cuda.synchronize()
    a, b = ctx.event(), ctx.event()
    reps = 8
    a.record(ctx.stream)
    for r in range(reps):
        bufs[(2 * r + 1) % 8].copy_(bufs[(2 * r) % 8])
    b.record(ctx.stream)
    torch.cuda.synchronize()
    ms = a.elapsed_time(b) / reps
    print(json.dumps({"mode": "copy-calibration", "bytes_read_per_copy": nbytes,
                      "bytes_written_per_copy": nbytes, "copies": reps,
                      "ms_per_copy": round(ms, 4),
                      "gbs_read_plus_write": round(2 * nbytes / (ms * 1e-3) / 1e9, 1)}),
          flush=True)


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU; --gpus {args.gpus} is not supported: the library "
              f"has no multi-GPU path (the product would shard by tokens with no communication)",
              file=sys.stderr)
        sys.exit(2)
    ctx = Ctx()
    if args.copy_calibration:
        copy_calibration(ctx, args)
    elif args.sweep:
        sweep(ctx, args)
    elif args.stack:
        stack(ctx, args)
    elif args.chunked:
        chunked(ctx, args)
    else:
        headline(ctx, args)


if __name__ == "__main__":
    main()
