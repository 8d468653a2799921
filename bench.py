#!/usr/bin/env python
"""Benchmark of the row-typed star_q projection on one MI355X.

Default workload (one JSON line on stdout): the star_2 FFN up-projection with
bias and GELU at the ~110M-LM FFN shape: M = 8192 rows (8 sequences x 1024
positions), 768 -> 3072 in blocks 384 x 1536, bf16 operands, fp32
accumulation, bf16 output, row type = position in sequence mod 2.  A step is
one pass of the hot path over the batch: the type plan, then the grouped
diagonal + type-gathered off-diagonal MFMA GEMM with the fused bias/GELU
epilogue.  ``value`` counts only the retained block GEMMs
(2 * sum_i M_i (D_diag + s_i (N - r_i)) flops).

Also reported in the same line: the same-code dense control (ordinary XW
through the same kernels), warm and cache-flushed kernel times, the decode
stack (12 layers, M in {1, 8, 32, 64}) in HBM GB/s and FFN tokens/s, the
roofline of the dominant kernel measured with HIP events, and the CPU oracle
timed on this host, plus the FFN training step (M = 16384, forward and
backward) and the fixed-block q sweep (q = 2..16) unless ``--no-extra``.
"""

from __future__ import annotations

import argparse
import hashlib
import json
import os
import statistics
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "⋆-proj TFLOP/s & % bf16 MFMA peak; decode HBM GB/s; speedup vs dense"
PEAK_BF16_TFLOPS = 2500.0  # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0      # MI355X HBM3E
FLUSH_BYTES = 512 << 20    # twice the 256 MB Infinity Cache
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "star_gemm_fwd_cfg2_traffic.json")
GEMM_SRCS = [os.path.join(ROOT, "paper_2609_32814_amd", "csrc", f)
             for f in ("gemm_async.hip", "gemm_common.hpp")]
GEMM_KERNEL = "star_gemm_async_kernel<fwd, star, gelu>"


def gemm_src_hash():
    """SHA-256 of the GEMM sources with // comments and blank lines removed,
    so that the stored traffic counters stay valid across comment edits and
    go stale on any change to the code itself."""
    h = hashlib.sha256()
    for f in GEMM_SRCS:
        with open(f, encoding="utf-8") as fh:
            for line in fh:
                code = line.split("//", 1)[0].rstrip()
                if code:
                    h.update(code.encode() + b"\n")
    return h.hexdigest()


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--trials", type=int, default=12, help="cache-flushed trials per kernel")
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    ap.add_argument("--no-decode", action="store_true")
    ap.add_argument("--no-extra", action="store_true",
                    help="skip the training step and the q sweep")
    ap.add_argument("--all", action="store_true", help=argparse.SUPPRESS)
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="only run a plain 256 MiB device copy (for HBM counter calibration)")
    ap.add_argument("--cpu-seconds", type=float, default=10.0)
    return ap.parse_args()


class Timer:
    """HIP-event timing on torch's current stream (the stream the library
    launches on)."""

    def __init__(self, torch):
        self.torch = torch

    def ev(self):
        return self.torch.cuda.Event(enable_timing=True)


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (got --gpus {args.gpus}); the star projection "
              "is row-local and shards over token rows with one dW all-reduce per step, "
              "which this build does not implement.", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    if args.calibrate_copy:
        calibrate_copy(torch, dev)
        return

    import paper_2609_32814_amd as P
    import synth

    T = Timer(torch)
    flush_buf = torch.empty(FLUSH_BYTES // 4, dtype=torch.float32, device=dev)

    def flush():
        flush_buf.fill_(1.0)

    # ---- primary workload ----------------------------------------------------
    M, K, N, q, SEQ = 8192, 768, 3072, 2, 1024
    alg = P.Algebra.equal(q, K, N)
    dalg = alg.with_law("dense")
    X = synth.gaussian(2, 0, (M, K), 1.0, "bf16")
    W = synth.gaussian(2, 1, (K, N), 0.02, "bf16")
    b = synth.gaussian(2, 2, (N,), 0.02, "f32")
    t = synth.sequence_types(M, q, SEQ)
    Xd, Wd = to_dev_bf16(X, torch, dev), to_dev_bf16(W, torch, dev)
    bd = torch.from_numpy(b.raw).to(dev)
    td = torch.from_numpy(t).to(dev)
    Y = torch.empty((M, N), dtype=torch.bfloat16, device=dev)
    plan = torch.empty(P.star_plan_bytes(q, M), dtype=torch.uint8, device=dev)
    rows = np.bincount(t, minlength=q)
    flops_star = 2 * P.star_count_macs(alg, rows)
    flops_dense = 2 * P.star_count_macs(dalg, rows)

    def run_plan():
        P.star_type_plan(q, td, plan)

    def run_fwd(a):
        P.star_proj_fwd_planned(a, plan, Xd, Wd, bd, "gelu", Y=Y)

    def timed_steps(a, steps, warmup):
        """Step time (type plan + GEMM, launched eagerly and, captured once,
        as a HIP graph replay) and the GEMM's own mean and median duration
        from events on its stream.  The step loops carry no events inside, so
        that event packets do not pad the step."""
        for _ in range(warmup):
            run_plan()
            run_fwd(a)
        torch.cuda.synchronize()
        e0, e1 = T.ev(), T.ev()
        e0.record()
        for _ in range(steps):
            run_plan()
            run_fwd(a)
        e1.record()
        torch.cuda.synchronize()
        eager_ms = e0.elapsed_time(e1) / steps
        # one step captured as a graph (same two kernels), replayed
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            run_plan()
            run_fwd(a)
        for _ in range(warmup):
            g.replay()
        torch.cuda.synchronize()
        e0.record()
        for _ in range(steps):
            g.replay()
        e1.record()
        torch.cuda.synchronize()
        graph_ms = e0.elapsed_time(e1) / steps
        del g
        ks = [(T.ev(), T.ev()) for _ in range(steps)]
        for s0, s1 in ks:
            run_plan()
            s0.record()
            run_fwd(a)
            s1.record()
        torch.cuda.synchronize()
        kern = [s0.elapsed_time(s1) for s0, s1 in ks]
        return eager_ms, graph_ms, statistics.mean(kern), statistics.median(kern)

    def flushed_kernel_ms(a, trials):
        out = []
        for _ in range(trials):
            run_plan()
            flush()
            torch.cuda.synchronize()
            s0, s1 = T.ev(), T.ev()
            s0.record()
            run_fwd(a)
            s1.record()
            torch.cuda.synchronize()
            out.append(s0.elapsed_time(s1))
        return statistics.median(out)

    log("primary: star_2 FFN up-projection M=8192 768->3072 bf16 + bias + GELU")
    eager_ms, graph_ms, kern_mean, kern_med = timed_steps(alg, args.steps, args.warmup)
    step_ms = min(eager_ms, graph_ms)
    # same-code dense control, then a second star pass: alternate the two
    d_eager_ms, d_graph_ms, d_kern_mean, d_kern_med = timed_steps(dalg, args.steps, args.warmup)
    d_step_ms = min(d_eager_ms, d_graph_ms)
    eager_ms2, graph_ms2, kern_mean2, _ = timed_steps(alg, args.steps, args.warmup)
    step_ms2 = min(eager_ms2, graph_ms2)
    star_fl, dense_fl = [], []
    for _ in range(max(1, args.trials // 2)):
        star_fl.append(flushed_kernel_ms(alg, 1))
        dense_fl.append(flushed_kernel_ms(dalg, 1))
    star_flushed, dense_flushed = statistics.median(star_fl), statistics.median(dense_fl)
    ms = min(step_ms, step_ms2)
    kern = min(kern_mean, kern_mean2)
    value = flops_star / (ms * 1e-3) / 1e12
    achieved = flops_star / (kern * 1e-3) / 1e12
    log(f"  star  step {ms*1e3:.1f} us (eager {min(eager_ms, eager_ms2)*1e3:.1f}, graph "
        f"{min(graph_ms, graph_ms2)*1e3:.1f})  kernel mean {kern*1e3:.1f} us  flushed {star_flushed*1e3:.1f} us"
        f"  -> {value:.1f} TFLOP/s step, {achieved:.1f} TFLOP/s kernel")
    log(f"  dense step {d_step_ms*1e3:.1f} us  kernel mean {d_kern_mean*1e3:.1f} us"
        f"  flushed {dense_flushed*1e3:.1f} us")

    traffic = None
    if os.path.exists(TRAFFIC_FILE):
        with open(TRAFFIC_FILE) as f:
            tr = json.load(f)
        if tr.get("gemm_src_sha256") == gemm_src_hash():
            traffic = tr.get("hbm_bytes_per_launch")

    roofline = {"bound": "mfma", "achieved": round(achieved, 2), "peak": PEAK_BF16_TFLOPS,
                "unit": "TFLOP/s", "frac": round(achieved / PEAK_BF16_TFLOPS, 4),
                "traffic": traffic, "kernel": GEMM_KERNEL,
                "kernel_mean_us": round(kern * 1e3, 2)}
    dense_ctrl = {
        "kernel_mean_us": round(d_kern_mean * 1e3, 2),
        "dense_tflops": round(flops_dense / (d_kern_mean * 1e-3) / 1e12, 2),
        "speedup_kernel_warm": round(d_kern_mean / kern, 3),
        "speedup_step_warm": round(d_step_ms / ms, 3),
        "speedup_kernel_flushed": round(dense_flushed / star_flushed, 3),
        "ideal_q2_over_2q_minus_1": round(q * q / (2 * q - 1), 3),
        "star_kernel_flushed_us": round(star_flushed * 1e3, 2),
        "dense_kernel_flushed_us": round(dense_flushed * 1e3, 2),
    }

    result = {
        "metric": METRIC,
        "value": round(value, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": "star_2 FFN up-projection + bias + GELU, M=8192 (8x1024 tokens), "
                               "768->3072 in blocks 384x1536, bf16 in / fp32 acc / bf16 out, "
                               "row type = position mod 2",
                   "M": M, "K": K, "N": N, "q": q, "retained_gflop": round(flops_star / 1e9, 3),
                   "parallelism": "single GPU",
                   "step": "type plan + fused GEMM, the faster of eager launches and a HIP graph replay",
                   "step_us_eager": round(min(eager_ms, eager_ms2) * 1e3, 2),
                   "step_us_graph": round(min(graph_ms, graph_ms2) * 1e3, 2)},
        "roofline": roofline,
        "dense_control": dense_ctrl,
        "mfma_peak_frac_step": round(value / PEAK_BF16_TFLOPS, 4),
    }
    del Y
    torch.cuda.empty_cache()

    # ---- decode stack ------------------------------------------------------------
    if not args.no_decode:
        result["decode"] = bench_decode(P, synth, torch, np, dev, T, flush, args)

    if not args.no_extra:
        result["training"] = bench_training(P, synth, torch, np, dev, T, args)
        result["qsweep"] = bench_qsweep(P, synth, torch, np, dev, T, flush, args)
        result["tensor2"] = bench_tensor2(P, synth, torch, np, dev, T, args)
        result["pilot_ffn"] = bench_pilot_ffn(P, synth, torch, np, dev, T, args)

    # ---- CPU oracle baseline -------------------------------------------------
    if not args.no_cpu:
        import oracle
        oalg = oracle.Alg.equal(q, K, N)
        reps, t0 = 0, time.perf_counter()
        while True:
            oracle.proj_fwd(oalg, t, X.exact, W.exact, b.exact, "gelu")
            reps += 1
            el = time.perf_counter() - t0
            if el >= args.cpu_seconds or reps >= 50:
                break
        cpu_val = flops_star * reps / el / 1e12
        result["cpu_baseline"] = {"value": round(cpu_val, 5), "unit": "TFLOP/s",
                                  "cores": oracle.num_threads(), "kind": "oracle",
                                  "sample": f"the full workload (M=8192) x {reps} repetitions, "
                                            f"{el:.1f} s, fp64 loops",
                                  "gpu_over_cpu": round(value / cpu_val, 1)}
        log(f"  cpu oracle: {cpu_val*1e3:.2f} GFLOP/s on {oracle.num_threads()} threads")

    print(json.dumps(result), flush=True)


def calibrate_copy(torch, dev):
    """A plain device-to-device copy of 256 MiB, five times: the reference
    kernel whose FETCH_SIZE / WRITE_SIZE counters give the scale factor for
    the GEMM's counters."""
    n = 256 << 20
    src = torch.ones(n // 4, dtype=torch.float32, device=dev)
    dst = torch.empty_like(src)
    for _ in range(5):
        dst.copy_(src)
    torch.cuda.synchronize()
    log(f"copy calibration: 5 x {n} bytes read and written")


def decode_weight_bytes(q, D, F, types, L, law="star"):
    """Weight bytes one decode step must read: every block (g, j) that some
    row's support reaches, for the up (D->F) and down (F->D) banks."""
    s_up, r_up = D // q, F // q
    s_dn, r_dn = F // q, D // q
    present = set(int(v) for v in types)
    need = 0
    for g in range(q):
        for j in range(q):
            if law == "dense" or any(g == i or g == j for i in present):
                need += 1
    return L * need * 2 * (s_up * r_up + s_dn * r_dn)


def bench_decode(P, synth, torch, np, dev, T, flush, args):
    D, F, L, q = 768, 3072, 12, 2
    up, dn = P.Algebra.equal(q, D, F), P.Algebra.equal(q, F, D)
    Wu = [to_dev_bf16(synth.gaussian(5, 10 + l, (D, F), 0.02, "bf16"), torch, dev) for l in range(L)]
    Wd = [to_dev_bf16(synth.gaussian(5, 40 + l, (F, D), 0.02, "bf16"), torch, dev) for l in range(L)]
    bu = [torch.from_numpy(synth.gaussian(5, 70 + l, (F,), 0.02, "f32").raw).to(dev) for l in range(L)]
    bdn = [torch.from_numpy(synth.gaussian(5, 100 + l, (D,), 0.02, "f32").raw).to(dev) for l in range(L)]
    out = {"workload": "12-layer star_2 FFN decode stack, d_model 768, d_ff 3072, bf16 weights "
                       "(113.2 MB), h += FFN(h), types = random position mod 2"}
    for M in (1, 8, 32, 64):
        X = to_dev_bf16(synth.gaussian(5, M, (M, D), 1.0, "bf16"), torch, dev)
        types = (synth.decode_positions(5, M) % 2).astype(np.int32)
        td = torch.from_numpy(types).to(dev)
        Y = torch.empty((M, D), dtype=torch.bfloat16, device=dev)
        ws = torch.empty(P.star_workspace_bytes("decode", up, dn, M), dtype=torch.uint8, device=dev)
        res = {}
        for law in ("star", "dense"):
            u, d = up.with_law(law), dn.with_law(law)

            def step():
                P.star_decode(u, d, td, X, Wu, bu, Wd, bdn, "gelu", True, Y=Y, ws=ws, check=False)

            for _ in range(args.warmup):
                step()
            torch.cuda.synchronize()
            n = max(20, args.steps)
            e0, e1 = T.ev(), T.ev()
            e0.record()
            for _ in range(n):
                step()
            e1.record()
            torch.cuda.synchronize()
            warm = e0.elapsed_time(e1) / n
            fl = []
            for _ in range(max(3, args.trials // 2)):
                flush()
                torch.cuda.synchronize()
                s0, s1 = T.ev(), T.ev()
                s0.record()
                step()
                s1.record()
                torch.cuda.synchronize()
                fl.append(s0.elapsed_time(s1))
            flushed = statistics.median(fl)
            nbytes = decode_weight_bytes(q, D, F, types, L, law)
            res[law] = {"step_us_warm": round(warm * 1e3, 1), "step_us_flushed": round(flushed * 1e3, 1),
                        "weight_MB": round(nbytes / 1e6, 1),
                        "GBps_warm": round(nbytes / (warm * 1e-3) / 1e9, 1),
                        "GBps_flushed": round(nbytes / (flushed * 1e-3) / 1e9, 1),
                        "tokens_per_s_warm": round(M / (warm * 1e-3), 1)}
        s = res["star"]
        s["hbm_frac_flushed"] = round(s["GBps_flushed"] / PEAK_HBM_GBS, 4)
        s["speedup_vs_dense_warm"] = round(res["dense"]["step_us_warm"] / s["step_us_warm"], 3)
        out[f"M{M}"] = res
        log(f"  decode M={M}: star {s['step_us_warm']} us warm / {s['step_us_flushed']} us flushed "
            f"({s['GBps_flushed']} GB/s flushed), dense {res['dense']['step_us_warm']} us warm")
    return out


def to_dev_bf16(t, torch, dev):
    import numpy as np
    return torch.from_numpy(np.ascontiguousarray(t.raw).view(np.int16)).view(torch.bfloat16).to(dev)


def bench_training(P, synth, torch, np, dev, T, args):
    """FFN forward + backward at M = 16384 (16 x 1024), 768 -> 3072 -> 768."""
    M, D, F, q = 16384, 768, 3072, 2
    up, dn = P.Algebra.equal(q, D, F), P.Algebra.equal(q, F, D)
    X = to_dev_bf16(synth.gaussian(3, 0, (M, D), 1.0, "bf16"), torch, dev)
    Wu = to_dev_bf16(synth.gaussian(3, 1, (D, F), 0.02, "bf16"), torch, dev)
    Wd = to_dev_bf16(synth.gaussian(3, 2, (F, D), 0.02, "bf16"), torch, dev)
    bu = torch.from_numpy(synth.gaussian(3, 3, (F,), 0.02, "f32").raw).to(dev)
    bd = torch.from_numpy(synth.gaussian(3, 4, (D,), 0.02, "f32").raw).to(dev)
    dY = to_dev_bf16(synth.gaussian(3, 5, (M, D), 1.0, "bf16"), torch, dev)
    t = synth.sequence_types(M, q, 1024)
    td = torch.from_numpy(t).to(dev)
    rows = np.bincount(t, minlength=q)
    res = {}
    for law in ("star", "dense"):
        u, d = up.with_law(law), dn.with_law(law)
        plan = P.star_type_plan(q, td)
        Z = torch.empty((M, F), dtype=torch.bfloat16, device=dev)
        H = torch.empty_like(Z)
        Y = torch.empty((M, D), dtype=torch.bfloat16, device=dev)
        ws = torch.empty(max(P.star_workspace_bytes("bwd_weight", u, None, M),
                             P.star_workspace_bytes("bwd_weight", d, None, M)),
                         dtype=torch.uint8, device=dev)

        def step():
            P.star_type_plan(q, td, plan)
            P.star_proj_fwd_planned(u, plan, X, Wu, bu, "gelu", Z_out=Z, Y=H)
            P.star_proj_fwd_planned(d, plan, H, Wd, bd, "none", Y=Y)
            P.star_ffn_bwd(u, d, td, X, Z, H, Wu, Wd, dY, "gelu", plan=plan, ws=ws)

        for _ in range(args.warmup):
            step()
        torch.cuda.synchronize()
        n = max(10, args.steps // 2)
        e0, e1 = T.ev(), T.ev()
        e0.record()
        for _ in range(n):
            step()
        e1.record()
        torch.cuda.synchronize()
        eager_ms = e0.elapsed_time(e1) / n
        # the same step captured once as a HIP graph and replayed
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            step()
        for _ in range(args.warmup):
            g.replay()
        torch.cuda.synchronize()
        e0.record()
        for _ in range(n):
            g.replay()
        e1.record()
        torch.cuda.synchronize()
        graph_ms = e0.elapsed_time(e1) / n
        del g
        ms = min(eager_ms, graph_ms)
        fl = 3 * 2 * (P.star_count_macs(u, rows) + P.star_count_macs(d, rows))
        res[law] = {"step_ms": round(ms, 4), "tflops": round(fl / (ms * 1e-3) / 1e12, 2),
                    "gflop": round(fl / 1e9, 2), "step_ms_eager": round(eager_ms, 4),
                    "step_ms_graph": round(graph_ms, 4)}
    res["speedup"] = round(res["dense"]["step_ms"] / res["star"]["step_ms"], 3)
    res["mfma_peak_frac"] = round(res["star"]["tflops"] / PEAK_BF16_TFLOPS, 4)
    log("training:", json.dumps(res))
    return res


def bench_tensor2(P, synth, torch, np, dev, T, args):
    """The pilot's law, the tensor square of the two-group law (q = 4, 36
    block products), on the FFN up-projection shape: M = 8192, 768 -> 3072
    in groups of 192 / 768, bias + GELU, interval row types
    floor((p mod 768) / 192); the same-code dense control beside it."""
    M, K, N, q = 8192, 768, 3072, 4
    alg = P.Algebra.equal(q, K, N, "tensor2")
    X = to_dev_bf16(synth.gaussian(6, 0, (M, K), 1.0, "bf16"), torch, dev)
    W = to_dev_bf16(synth.gaussian(6, 1, (K, N), 0.02, "bf16"), torch, dev)
    b = torch.from_numpy(synth.gaussian(6, 2, (N,), 0.02, "f32").raw).to(dev)
    t = ((np.arange(M) % 768) // 192).astype(np.int32)
    td = torch.from_numpy(t).to(dev)
    plan = P.star_type_plan(q, td)
    Y = torch.empty((M, N), dtype=torch.bfloat16, device=dev)
    rows = np.bincount(t, minlength=q)
    res = {"workload": "Q_2 (x) Q_2 FFN up-projection + bias + GELU, M=8192, 768->3072 in groups "
                       "192/768, bf16, row type = floor((p mod 768) / 192)"}
    for law in ("tensor2", "dense"):
        a = alg.with_law(law)
        for _ in range(args.warmup):
            P.star_proj_fwd_planned(a, plan, X, W, b, "gelu", Y=Y)
        torch.cuda.synchronize()
        n = max(20, args.steps)
        ks = [(T.ev(), T.ev()) for _ in range(n)]
        for s0, s1 in ks:
            s0.record()
            P.star_proj_fwd_planned(a, plan, X, W, b, "gelu", Y=Y)
            s1.record()
        torch.cuda.synchronize()
        ms = statistics.mean(s0.elapsed_time(s1) for s0, s1 in ks)
        fl = 2 * P.star_count_macs(a, rows)
        res[law] = {"kernel_us": round(ms * 1e3, 1), "tflops": round(fl / (ms * 1e-3) / 1e12, 1),
                    "gflop": round(fl / 1e9, 3)}
    res["speedup"] = round(res["dense"]["kernel_us"] / res["tensor2"]["kernel_us"], 3)
    res["ideal"] = round(16 / 9, 3)
    res["products_per_type"] = P.star_count_products(alg)[0]
    del X, W, Y, plan
    torch.cuda.empty_cache()

    # the same law through the 12-layer decode stack (d_model 768, d_ff 3072)
    D, F, L = 768, 3072, 12
    up, dn = P.Algebra.equal(q, D, F, "tensor2"), P.Algebra.equal(q, F, D, "tensor2")
    Wu = [to_dev_bf16(synth.gaussian(6, 10 + l, (D, F), 0.02, "bf16"), torch, dev) for l in range(L)]
    Wd = [to_dev_bf16(synth.gaussian(6, 40 + l, (F, D), 0.02, "bf16"), torch, dev) for l in range(L)]
    bu = [torch.from_numpy(synth.gaussian(6, 70 + l, (F,), 0.02, "f32").raw).to(dev) for l in range(L)]
    bdn = [torch.from_numpy(synth.gaussian(6, 100 + l, (D,), 0.02, "f32").raw).to(dev) for l in range(L)]
    dec = {}
    for Md in (1, 64):
        Xd = to_dev_bf16(synth.gaussian(6, 200 + Md, (Md, D), 1.0, "bf16"), torch, dev)
        tdd = torch.from_numpy(((synth.decode_positions(6, Md) % 768) // 192).astype(np.int32)).to(dev)
        Yd = torch.empty((Md, D), dtype=torch.bfloat16, device=dev)
        ws = torch.empty(P.star_workspace_bytes("decode", up, dn, Md), dtype=torch.uint8, device=dev)
        one = {}
        for law in ("tensor2", "dense"):
            u, d = up.with_law(law), dn.with_law(law)
            for _ in range(args.warmup):
                P.star_decode(u, d, tdd, Xd, Wu, bu, Wd, bdn, "gelu", True, Y=Yd, ws=ws, check=False)
            torch.cuda.synchronize()
            n = max(20, args.steps)
            e0, e1 = T.ev(), T.ev()
            e0.record()
            for _ in range(n):
                P.star_decode(u, d, tdd, Xd, Wu, bu, Wd, bdn, "gelu", True, Y=Yd, ws=ws, check=False)
            e1.record()
            torch.cuda.synchronize()
            one[law] = {"step_us_warm": round(e0.elapsed_time(e1) / n * 1e3, 1)}
        dec[f"M{Md}"] = one
    res["decode"] = dec
    log("tensor2:", json.dumps(res))
    return res


def bench_pilot_ffn(P, synth, torch, np, dev, T, args):
    """The pretraining pilot's FFN: bias-free SwiGLU, D = 768, F = 1536, under
    the tensor-square law Q_2 (x) Q_2 with interval row types, one training
    step (three projections forward, their activation and weight gradients)
    at M = 16384 tokens, beside the same-code dense control."""
    M, D, F, q = 16384, 768, 1536, 4
    up, dn = P.Algebra.equal(q, D, F, "tensor2"), P.Algebra.equal(q, F, D, "tensor2")
    X = to_dev_bf16(synth.gaussian(8, 0, (M, D), 1.0, "bf16"), torch, dev)
    Wg = to_dev_bf16(synth.gaussian(8, 1, (D, F), 0.02, "bf16"), torch, dev)
    Wu = to_dev_bf16(synth.gaussian(8, 2, (D, F), 0.02, "bf16"), torch, dev)
    Wd = to_dev_bf16(synth.gaussian(8, 3, (F, D), 0.02, "bf16"), torch, dev)
    dY = to_dev_bf16(synth.gaussian(8, 4, (M, D), 1.0, "bf16"), torch, dev)
    t = ((np.arange(M) % 768) // 192).astype(np.int32)
    td = torch.from_numpy(t).to(dev)
    rows = np.bincount(t, minlength=q)
    res = {"workload": "bias-free SwiGLU FFN 768 -> 2 x 1536 -> 768, Q_2 (x) Q_2, M=16384, bf16, "
                       "row type = floor((p mod 768) / 192); forward + backward; and its 12-layer "
                       "decode stack at M in {1, 48}"}
    for law in ("tensor2", "dense"):
        u, d = up.with_law(law), dn.with_law(law)
        plan = P.star_type_plan(q, td)

        def step():
            P.star_type_plan(q, td, plan)
            Zg, Zu, H, _ = P.star_swiglu_ffn_fwd(u, d, td, X, Wg, None, Wu, None, Wd, None, plan=plan)
            P.star_swiglu_ffn_bwd(u, d, td, X, Zg, Zu, H, Wg, Wu, Wd, dY, plan=plan)

        for _ in range(args.warmup):
            step()
        torch.cuda.synchronize()
        n = max(10, args.steps // 2)
        e0, e1 = T.ev(), T.ev()
        e0.record()
        for _ in range(n):
            step()
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / n
        fl = 3 * 2 * (2 * P.star_count_macs(u, rows) + P.star_count_macs(d, rows))
        res[law] = {"step_ms": round(ms, 4), "tflops": round(fl / (ms * 1e-3) / 1e12, 2),
                    "gflop": round(fl / 1e9, 2)}
    res["speedup"] = round(res["dense"]["step_ms"] / res["tensor2"]["step_ms"], 3)
    del X, Wg, Wu, Wd, dY
    torch.cuda.empty_cache()

    # the pilot's 12-layer gated decode stack (weights 12 x 3 x 768 x 1536 bf16 = 84.9 MB)
    L = 12
    Wgs = [to_dev_bf16(synth.gaussian(8, 10 + l, (D, F), 0.02, "bf16"), torch, dev) for l in range(L)]
    Wus = [to_dev_bf16(synth.gaussian(8, 40 + l, (D, F), 0.02, "bf16"), torch, dev) for l in range(L)]
    Wds = [to_dev_bf16(synth.gaussian(8, 70 + l, (F, D), 0.02, "bf16"), torch, dev) for l in range(L)]
    dec = {}
    for Md in (1, 48):
        Xd = to_dev_bf16(synth.gaussian(8, 200 + Md, (Md, D), 1.0, "bf16"), torch, dev)
        tdd = torch.from_numpy(((synth.decode_positions(8, Md) % 768) // 192).astype(np.int32)).to(dev)
        Yd = torch.empty((Md, D), dtype=torch.bfloat16, device=dev)
        ws = torch.empty(P.star_workspace_bytes("decode", up, dn, Md), dtype=torch.uint8, device=dev)
        one = {}
        for law in ("tensor2", "dense"):
            u, d = up.with_law(law), dn.with_law(law)
            for _ in range(args.warmup):
                P.star_decode_gated(u, d, tdd, Xd, Wgs, None, Wus, None, Wds, None, True, Y=Yd, ws=ws, check=False)
            torch.cuda.synchronize()
            n = max(20, args.steps)
            e0, e1 = T.ev(), T.ev()
            e0.record()
            for _ in range(n):
                P.star_decode_gated(u, d, tdd, Xd, Wgs, None, Wus, None, Wds, None, True, Y=Yd, ws=ws, check=False)
            e1.record()
            torch.cuda.synchronize()
            us = e0.elapsed_time(e1) / n * 1e3
            one[law] = {"step_us_warm": round(us, 1), "tokens_per_s": round(Md / (us * 1e-6), 1)}
        dec[f"M{Md}"] = one
    res["decode"] = dec
    log("pilot_ffn:", json.dumps(res))
    return res


def bench_qsweep(P, synth, torch, np, dev, T, flush, args):
    M = 16384
    out = {}
    for q in (2, 4, 8, 16):
        d = 256 * q
        alg = P.Algebra.equal(q, d, d)
        X = to_dev_bf16(synth.gaussian(4, q, (M, d), 1.0, "bf16"), torch, dev)
        W = to_dev_bf16(synth.gaussian(4, 100 + q, (d, d), (1.0 / d) ** 0.5, "bf16"), torch, dev)
        t = synth.cyclic_types(M, q)
        td = torch.from_numpy(t).to(dev)
        plan = P.star_type_plan(q, td)
        Y = torch.empty((M, d), dtype=torch.bfloat16, device=dev)
        rows = np.bincount(t, minlength=q)
        res = {}
        for law in ("star", "dense"):
            a = alg.with_law(law)
            for _ in range(args.warmup):
                P.star_proj_fwd_planned(a, plan, X, W, Y=Y)
            torch.cuda.synchronize()
            n = max(20, args.steps)
            e0, e1 = T.ev(), T.ev()
            e0.record()
            for _ in range(n):
                P.star_proj_fwd_planned(a, plan, X, W, Y=Y)
            e1.record()
            torch.cuda.synchronize()
            ms = e0.elapsed_time(e1) / n
            fl = 2 * P.star_count_macs(a, rows)
            byts = 2 * (M * d + d * d + M * d)
            res[law] = {"kernel_us": round(ms * 1e3, 1), "tflops": round(fl / (ms * 1e-3) / 1e12, 1),
                        "GBps_algorithmic": round(byts / (ms * 1e-3) / 1e9, 1)}
        res["speedup"] = round(res["dense"]["kernel_us"] / res["star"]["kernel_us"], 3)
        res["ideal"] = round(q * q / (2 * q - 1), 3)
        res["products_per_type"] = P.star_count_products(alg)[0]
        out[f"q{q}"] = res
        del X, W, Y
        torch.cuda.empty_cache()
    log("qsweep:", json.dumps(out))
    return out


if __name__ == "__main__":
    main()
