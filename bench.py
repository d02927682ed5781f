"""Benchmark of one TeraPipe pipeline stage on one MI355X.

A step is one training sequence through the stage: reset the K/V prefix, run
the forward of every token slice in order, then the backward of every slice in
reverse (the weight-gradient GEMMs included: per slice, or once at the end of
the sequence in the deferred mode).  Throughput is algorithmic flops per
second: per layer and slice, 24 n H^2 (projections) + 4 H per causal
(query, key <= query) pair forward, backward twice forward.

Prints one JSON line.  Per-kernel-class times are measured with HIP events on
the stage's stream; `roofline` reports one kernel: the deferred dW GEMM (the
largest single kernel) in the deferred mode, else the class with the largest
total time.  `cpu_baseline` times the fp64 CPU oracle on a bounded sample of
the same workload (one layer, a short slice).
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

# name: (layers, hidden, heads, seq, default slicing, operation-partitioning shard p)
WORKLOADS = {
    "gpt3-175b-stage": (2, 12288, 96, 2048, [256] * 8, 1),
    "gpt3-175b-stage-8k": (2, 12288, 96, 8192, [512] * 16, 1),
    "gpt3-13b-stage": (2, 5120, 40, 2048, [256] * 8, 1),
    "gpt3-1.3b-stage": (2, 2048, 16, 2048, [256] * 8, 1),
    # one GPU's work in the paper's 175B settings: (10) 48 stages of 2 layers,
    # each layer split 8 ways; (9) 96 stages of 1 layer split 4 ways
    "gpt3-175b-op8-stage": (2, 12288, 96, 2048, [256] * 8, 8),
    "gpt3-175b-op4-stage": (1, 12288, 96, 2048, [256] * 8, 4),
}
# pipeline depth K of the paper's setting for each model (Table 1: settings (2), (4), (10), (9))
PAPER_K = {"gpt3-175b-stage": 48, "gpt3-175b-stage-8k": 48, "gpt3-13b-stage": 20,
           "gpt3-1.3b-stage": 12, "gpt3-175b-op8-stage": 48, "gpt3-175b-op4-stage": 96}

PEAK_BF16_TFLOPS = 2500.0  # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0

# HBM bytes per launch of a kernel class on the default workload, from two
# rocprofv3 --pmc passes (FETCH_SIZE, WRITE_SIZE) scaled by the same counters on
# a plain copy of known size (profiles/gemm_bwd_dw_tn_traffic.md).  Reported only
# while the kernel source still has the hash it had when the counters were taken,
# and for the gradient-buffer mode they were taken in.
TRAFFIC = {
    "gemm_bwd_dw_tn": {"workload": "gpt3-175b-stage", "grad_buffers": "overwrite",
                       "source": "paper_2102_07988_amd/csrc/kernels_gemm_dma.hip",
                       "sha256_16": "63b4dc6c732fc8bf", "bytes_per_launch": 4555134686},
}


def measured_traffic(kernel: str, workload: str, grad_buffers: str):
    import hashlib

    t = TRAFFIC.get(kernel)
    if not t or t["workload"] != workload or t["grad_buffers"] != grad_buffers:
        return None
    try:
        h = hashlib.sha256(open(os.path.join(ROOT, t["source"]), "rb").read()).hexdigest()[:16]
    except OSError:
        return None
    return t["bytes_per_launch"] if h == t["sha256_16"] else None


def parse_slicing(s: str, L: int, default):
    if not s:
        return list(default)
    if s.startswith("uniform"):
        n = int(s[len("uniform"):])
        assert L % n == 0
        return [n] * (L // n)
    lens = [int(v) for v in s.split(",")]
    assert sum(lens) == L, "slicing must sum to the sequence length"
    return lens


def cpu_baseline(params0, x, dy, hidden: int, heads: int, n_tokens: int, op_parts: int = 1):
    """Time the fp64 oracle on one layer of the workload (the benchmark's own
    layer-0 parameters): forward + backward of one slice of the first n tokens
    after no context, for n = 16 and n = n_tokens on all host threads, and for
    n = 4 on one thread.  `value` is the all-thread rate at n = n_tokens; every
    point is listed."""
    import ctypes
    import numpy as np
    import torch

    from oracle import OracleStage, slice_flops

    p64 = {k: v.detach().to("cpu").to(torch.float64).numpy() for k, v in params0.items()}
    threads = int(os.environ.get("OMP_NUM_THREADS", "0")) or os.cpu_count()
    try:
        gomp = ctypes.CDLL("libgomp.so.1")
    except OSError:
        gomp = None

    def point(n, nthreads):
        x64 = x[:n].to("cpu").to(torch.float64).numpy()
        dy64 = dy[:n].to("cpu").to(torch.float64).numpy()
        st = OracleStage([p64], hidden, heads, n, op_parts=op_parts)
        if gomp is not None:
            gomp.omp_set_num_threads(nthreads)
        t0 = time.perf_counter()
        st.run_sequence(x64, dy64, [n])
        dt = time.perf_counter() - t0
        if gomp is not None:
            gomp.omp_set_num_threads(threads)
        fl = slice_flops(n, 0, hidden) // op_parts
        return {"len": n, "ctx": 0, "threads": nthreads if gomp is not None else threads,
                "seconds": round(dt, 3), "tflops": fl / dt / 1e12}

    pts = [point(16, threads), point(n_tokens, threads)]
    if gomp is not None:
        pts.append(point(4, 1))
    main = pts[1]
    return {"value": main["tflops"], "unit": "TFLOP/s", "cores": threads, "kind": "oracle",
            "seconds": main["seconds"], "points": pts,
            "sample": f"1 layer of the same shape (H={hidden}, {heads // op_parts} of {heads} "
                      f"heads), one slice of {n_tokens} tokens at context 0, forward+backward, "
                      f"fp64, {threads} threads (points: 16 tokens on {threads} threads, 4 tokens "
                      f"on 1 thread)"}


def _subset(U: int):
    """Model-mode subset in units: a few lengths x a few contexts (Sec. 3.3 fits
    the overhead on a subset of the (i, j) grid)."""
    ks = sorted({k for k in (1, 2, U // 8, U // 4, U // 2, 3 * U // 4) if 1 <= k < U})
    js = sorted({j for j in (1, U // 8, U // 4, U // 2, 3 * U // 4) if 1 <= j < U})
    return ks, js


def _eq5(cost, units, K):
    ts, c = [], 0
    for u in units:
        ts.append(int(cost[u - 1, c]))
        c += u
    return sum(ts) + (K - 1) * max(ts), sum(ts)


def _slicing_summary(tp, cost, unit, K):
    """DP slicing of a table and Eq. 5 latencies of the uniform slicings."""
    U = cost.shape[0]
    t1 = time.perf_counter()
    dp_lens, dp_T = tp.dp_optimal_slicing(cost, unit, K)
    dp_s = time.perf_counter() - t1
    uniform = {str(m): round(_eq5(cost, [U // m] * m, K)[0] / 1e6, 3)
               for m in range(1, U + 1) if U % m == 0}
    best_m = min(uniform, key=uniform.get)
    return {"dp_slicing": dp_lens, "dp_T_ms": round(dp_T / 1e6, 3), "dp_seconds": round(dp_s, 4),
            "uniform_T_ms": uniform, "best_uniform_slices": int(best_m),
            "dp_speedup_vs_best_uniform": round(uniform[best_m] / (dp_T / 1e6), 4),
            "single_slice_T_ms": uniform["1"]}


def pipeline_report(st, tp, L: int, unit: int, K: int, warmup: int, reps: int,
                    run_slicing, dw_ms: float, fine_unit: int, n_layers: int, H: int,
                    deferred: bool, fine_K=(48, 96), op_parts: int = 1):
    """Per-slice cost tables t(len, ctx) = t_fwd + t_bwd of this stage and the
    slicings they give for a pipeline of K such stages (Eq. 5-8, Algorithm 1):

    * the full table measured at every (len, ctx) on a grid of `unit` tokens:
      DP vs uniform vs one slice, and the DP slicing run back to back on the
      stage against the sum of its table entries;
    * the model-mode table (Eq. 9) on the same grid from t(i, 0) plus a fitted
      context overhead: its prediction error on the points it did not measure
      and the latency its DP slicing reaches on the measured table;
    * a model-mode table on a fine grid of `fine_unit` tokens (too many points
      to measure one by one): DP vs uniform slicings for each K in fine_K."""
    import numpy as np

    U = L // unit
    lens = [unit * k for k in range(1, U + 1)]
    ctxs = [unit * j for j in range(U)]
    t0 = time.perf_counter()
    tf, tb = st.profile(lens, ctxs, warmup=warmup, reps=reps)
    prof_s = time.perf_counter() - t0
    cost = np.where(tf >= 0, tf + tb, -1).astype(np.int64)
    # the same table measured once more: the repeat-measurement noise that any
    # model of it is compared against
    tf2, tb2 = st.profile(lens, ctxs, warmup=warmup, reps=reps)
    cost2 = np.where(tf2 >= 0, tf2 + tb2, -1).astype(np.int64)
    rep = {"K": K, "unit": unit, "table_points": int((cost >= 0).sum()),
           "warmup": warmup, "reps": reps, "profile_seconds": round(prof_s, 2)}
    # slice throughput vs (len, ctx): the stage's fwd + bwd flops of one slice
    # (without the deferred once-per-sequence dW GEMMs, which the table does
    # not time) over the measured t_fwd + t_bwd
    pts = []
    n = unit
    while n <= L:
        for c in sorted({0, L // 2 - n if L // 2 >= n else 0, L - n}):
            if c < 0 or (c % unit):
                continue
            t_ns = int(cost[n // unit - 1, c // unit])
            fl = n_layers * (tp.slice_flops(n, c, H) - (24 * n * H * H if deferred else 0))
            fl //= op_parts
            pts.append({"len": n, "ctx": c, "t_ms": round(t_ns / 1e6, 3),
                        "tflops": round(fl / (t_ns * 1e-9) / 1e12, 1),
                        "pct_bf16_peak": round(100 * fl / (t_ns * 1e-9) / 1e12 / PEAK_BF16_TFLOPS, 1)})
        n *= 2
    rep["slice_tflops"] = pts
    rep.update(_slicing_summary(tp, cost, unit, K))
    dp_units = [n // unit for n in rep["dp_slicing"]]
    measured_ms = run_slicing(rep["dp_slicing"])
    table_sum = _eq5(cost, dp_units, K)[1] / 1e6
    rep["back_to_back"] = {
        "slicing": rep["dp_slicing"], "measured_ms": round(measured_ms, 3),
        "measured_minus_deferred_dw_ms": round(measured_ms - dw_ms, 3),
        "table_sum_ms": round(table_sum, 3),
        "ratio": round((measured_ms - dw_ms) / table_sum, 4)}

    # model mode on the same grid (Eq. 9): t(i, 0) for every length plus the
    # context overhead fitted on a subset, judged on the points it did not
    # measure -- against the first measured table, next to how far the second
    # measurement of the same table lies from the first
    ks, js = _subset(U)
    t0 = time.perf_counter()
    mcost, coef = st.profile_model(L, unit, [unit * k for k in ks], [unit * j for j in js],
                                   warmup=warmup, reps=reps)
    mprof_s = time.perf_counter() - t0
    sub = {(k, j) for k in ks for j in js if k + j <= U}
    ov_err, ov_noise, t_err, t_noise, big_err, big_noise = [], [], [], [], [], []
    for k in range(1, U + 1):
        for j in range(1, U - k + 1):
            if (k, j) in sub:
                continue
            i, c = k * unit, j * unit
            actual_ov = cost[k - 1, j] - cost[k - 1, 0]
            again_ov = cost2[k - 1, j] - cost2[k - 1, 0]
            pred_ov = coef[0] + coef[1] * i + coef[2] * c + coef[3] * i * c
            if actual_ov > 0:
                ov_err.append(abs(pred_ov - actual_ov) / actual_ov)
                ov_noise.append(abs(again_ov - actual_ov) / actual_ov)
                # overheads of at least a tenth of the slice's own cost
                if actual_ov >= 0.1 * cost[k - 1, 0]:
                    big_err.append(ov_err[-1])
                    big_noise.append(ov_noise[-1])
            t_err.append(abs(mcost[k - 1, j] - cost[k - 1, j]) / cost[k - 1, j])
            t_noise.append(abs(cost2[k - 1, j] - cost[k - 1, j]) / cost[k - 1, j])
    med = lambda v: round(float(np.median(v)), 4) if v else None
    p90 = lambda v: round(float(np.percentile(v, 90)), 4) if v else None
    m_lens, _ = tp.dp_optimal_slicing(mcost, unit, K)
    m_T = _eq5(cost, [n // unit for n in m_lens], K)[0]
    rep["model"] = {
        "unit": unit, "points_measured": U + len(sub), "profile_seconds": round(mprof_s, 2),
        "coef_ns": [round(v, 6) for v in coef],
        "heldout_points": len(t_err),
        "heldout_overhead_rel_err_median": med(ov_err),
        "heldout_overhead_rel_err_p90": p90(ov_err),
        "repeat_overhead_rel_diff_median": med(ov_noise),
        "repeat_overhead_rel_diff_p90": p90(ov_noise),
        "large_overhead_points": len(big_err),
        "large_overhead_rel_err_median": med(big_err),
        "large_overhead_repeat_rel_diff_median": med(big_noise),
        "heldout_cost_rel_err_median": med(t_err),
        "heldout_cost_rel_err_max": round(float(np.max(t_err)), 4) if t_err else None,
        "repeat_cost_rel_diff_median": med(t_noise),
        "repeat_cost_rel_diff_max": round(float(np.max(t_noise)), 4) if t_noise else None,
        "paper_overhead_rel_err_bound": 0.02,
        "dp_slicing": m_lens, "dp_T_on_measured_table_ms": round(m_T / 1e6, 3),
        "vs_measured_table_dp": round(m_T / (rep["dp_T_ms"] * 1e6), 4)}
    # the tables themselves (int64 ns, entry [len units - 1][ctx units], -1
    # past the sequence end), so every slicing above can be re-derived offline
    # (paper_2102_07988_amd/replay.py)
    rep["tables"] = {"unit": unit, "measured_ns": cost.tolist(), "measured_again_ns": cost2.tolist(),
                     "model_ns": mcost.tolist(), "model_coef_ns": [float(v) for v in coef]}

    # model mode on the fine grid
    if fine_unit and L % fine_unit == 0 and fine_unit < unit:
        Uf = L // fine_unit
        ks, js = _subset(Uf)
        t0 = time.perf_counter()
        fcost, fcoef = st.profile_model(L, fine_unit, [fine_unit * k for k in ks],
                                        [fine_unit * j for j in js], warmup=warmup, reps=reps)
        fprof_s = time.perf_counter() - t0
        rep["model_fine"] = {
            "unit": fine_unit, "points_measured": Uf + sum(1 for k in ks for j in js if k + j <= Uf),
            "table_points": int((fcost >= 0).sum()), "profile_seconds": round(fprof_s, 2),
            "coef_ns": [round(v, 6) for v in fcoef],
            # the fine table is tp_cost_table_from_model(t0_ns, unit, coef) exactly
            "t0_ns": [int(v) for v in fcost[:, 0]], "coef_full": [float(v) for v in fcoef],
            "by_K": {str(k): _slicing_summary(tp, fcost, fine_unit, k) for k in fine_K}}
        rep["_fine_cost"] = fcost
    rep["deferred_dw_ms_per_sequence"] = round(dw_ms, 3)
    rep["note"] = ("T = Eq. 5 over t_fwd + t_bwd tables; in deferred mode the once-per-sequence "
                   "dW GEMMs (deferred_dw_ms) add to the last stage's tail and are not in t")
    return rep


def joint_report(make_stage, tp, L: int, unit: int, K: int, B: int, cost_b1, warmup: int,
                 reps: int):
    """Batch x token plan of Sec. 3.4 for a batch of B sequences: the model-mode
    cost table (Eq. 9, grid of `unit` tokens) of a stage holding b = 1..B
    sequences per batch slice (b = 1: `cost_b1`), the optimal token slicing and
    latency T_b of each group size, and the group sizes chosen by the batch
    split (knapsack over T_b), next to B single sequences and one group of B."""
    import numpy as np
    U = L // unit
    ks, js = _subset(U)
    costs = np.zeros((B, U, U), dtype=np.int64)
    costs[0] = cost_b1
    prof_s = 0.0
    for b in range(2, B + 1):
        stb = make_stage(b)
        t0 = time.perf_counter()
        costs[b - 1], _ = stb.profile_model(L, unit, [unit * k for k in ks],
                                            [unit * j for j in js], warmup=warmup, reps=reps)
        prof_s += time.perf_counter() - t0
        del stb
    groups, T_b, total = tp.joint_slicing(costs, unit, K)
    return {"B": B, "unit": unit, "K": K, "profile_seconds": round(prof_s, 2),
            "T_b_ms": [round(t / 1e6, 3) for t in T_b],
            "T_b_per_sequence_ms": [round(t / (b + 1) / 1e6, 3) for b, t in enumerate(T_b)],
            "groups": [{"sequences": b, "slicing": sl} for b, sl in groups],
            "total_ms": round(total / 1e6, 3),
            "all_single_sequences_ms": round(B * T_b[0] / 1e6, 3),
            "one_group_ms": round(T_b[B - 1] / 1e6, 3)}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--workload", default="gpt3-175b-stage", choices=sorted(WORKLOADS))
    ap.add_argument("--slicing", default="",
                    help="'uniform256', comma-separated lengths, or 'dp' (DP over this stage's "
                         "model-mode cost table at the paper's K for the model)")
    ap.add_argument("--wgrad", default="deferred", choices=["deferred", "per_slice"])
    ap.add_argument("--accumulate-grads", action="store_true",
                    help="each step adds its parameter gradients to the earlier steps' "
                         "(default: each step is a training iteration of one sequence that "
                         "stores its gradients, TP_SEQ_OVERWRITE_GRADS)")
    ap.add_argument("--cpu-baseline-tokens", type=int, default=96)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-kernel-timing", action="store_true")
    ap.add_argument("--eager", action="store_true",
                    help="time eager launches instead of a replayed HIP graph of the sequence")
    ap.add_argument("--no-pipeline", action="store_true",
                    help="skip the cost-table / DP / Eq. 5 pipeline-latency report")
    ap.add_argument("--pipeline-unit", type=int, default=128)
    ap.add_argument("--profile-warmup", type=int, default=3,
                    help="untimed runs per table point of the cost-table profiles")
    ap.add_argument("--profile-reps", type=int, default=10,
                    help="timed runs per table point (median); the paper averages 10 runs")
    ap.add_argument("--pipeline-K", type=int, default=48)
    ap.add_argument("--pipeline-fine-unit", type=int, default=16,
                    help="grid of the model-mode (Eq. 9) table for the uniform-vs-DP sweep; "
                         "0 skips it")
    ap.add_argument("--joint-batch", type=int, default=2,
                    help="batch size B of the Sec. 3.4 batch x token plan in the pipeline "
                         "report (model-mode tables for 1..B sequences per batch slice); "
                         "0 or 1 skips it")
    ap.add_argument("--copy-calibration-mib", type=int, default=0,
                    help="only run a plain device copy of this many MiB (4 times), for "
                         "scaling the HBM byte counters")
    args = ap.parse_args()

    if args.gpus != 1:
        print(json.dumps({"error": "this build runs one pipeline stage on one GPU; "
                                   "--gpus above 1 is not supported", "n_gpus": args.gpus}))
        sys.exit(2)

    import torch

    if args.copy_calibration_mib:
        n = args.copy_calibration_mib * (1 << 20) // 4
        src = torch.ones(n, dtype=torch.float32, device="cuda:0")
        dst = torch.empty_like(src)
        for _ in range(4):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_calibration_bytes_read": n * 4, "bytes_written": n * 4}))
        return

    from paper_2102_07988_amd import synth
    from paper_2102_07988_amd import terapipe as tp

    n_layers, H, heads, L, default_sl, parts = WORKLOADS[args.workload]
    dp_source = None
    lens = parse_slicing(args.slicing, L, default_sl) if args.slicing != "dp" else None
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    # the stage enqueues on its own stream (default priority), captured as a whole
    cs = torch.cuda.Stream(device=dev)
    torch.cuda.set_stream(cs)
    bf = torch.bfloat16
    params = synth.stage_params(n_layers, H, seed=synth.SEED_PARAMS, dtype=bf, device=dev,
                                op_parts=parts)
    x = synth.hidden_states(L, H, seed=synth.SEED_X, dtype=bf, device=dev)
    dy = synth.upstream_grad(L, H, seed=synth.SEED_DY, dtype=bf, device=dev)
    st = tp.Stage(params, H, heads, L, dtype="bf16", wgrad=args.wgrad, op_parts=parts)
    if lens is None:
        # slicing chosen by the DP (Eq. 5-8, Algorithm 1) on this stage's own
        # model-mode cost table (Eq. 9) at the paper's pipeline depth for the model
        unit = max(16, L // 128)
        U = L // unit
        ks = sorted({k for k in (1, 2, U // 8, U // 4, U // 2, 3 * U // 4) if 1 <= k < U})
        js = sorted({j for j in (1, U // 8, U // 4, U // 2, 3 * U // 4) if 1 <= j < U})
        t0 = time.perf_counter()
        cost, coef = st.profile_model(L, unit, [unit * k for k in ks], [unit * j for j in js],
                                      warmup=1, reps=3)
        prof_s = time.perf_counter() - t0
        K = PAPER_K[args.workload]
        lens, T = tp.dp_optimal_slicing(cost, unit, K)
        st.zero_grads()
        dp_source = {"kind": "dp", "table": "model mode (Eq. 9)", "unit": unit, "K": K,
                     "predicted_T_ms": round(T / 1e6, 3), "profile_seconds": round(prof_s, 2)}
    y = torch.empty_like(x)
    dx = torch.empty_like(dy)
    bounds = [0]
    for n in lens:
        bounds.append(bounds[-1] + n)

    def step():
        st.reset(overwrite_grads=not args.accumulate_grads)
        for i in range(len(lens)):
            l, r = bounds[i], bounds[i + 1]
            st.forward(l, r, x[l:r], out=y[l:r])
        for i in range(len(lens) - 1, -1, -1):
            l, r = bounds[i], bounds[i + 1]
            st.backward(l, r, dy[l:r], out=dx[l:r])

    for _ in range(max(1, args.warmup)):
        step()
    torch.cuda.synchronize()
    graph, graph_ok = None, None
    if not args.eager:
        # one whole sequence (reset, every slice forward and backward, the dW
        # GEMMs) captured as a HIP graph and replayed per step: no launch gaps.
        # Replays must reproduce the eager outputs bit for bit.
        y_ref, dx_ref = y.clone(), dx.clone()
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph, stream=cs):
            step()
        graph.replay()
        torch.cuda.synchronize()
        graph_ok = bool(torch.equal(y, y_ref) and torch.equal(dx, dx_ref))
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        if graph is not None:
            graph.replay()
        else:
            step()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    if graph is not None:
        graph_ok = graph_ok and bool(torch.equal(y, y_ref) and torch.equal(dx, dx_ref))
    # per-kernel-class times: HIP events around every launch, in eager steps
    # after the timed region (kernel durations do not depend on graph replay)
    stats, kt_steps = {}, 0
    if not args.no_kernel_timing:
        kt_steps = min(args.steps, 3)
        st.enable_kernel_timing(True)
        st.kernel_stats()  # clears the counters
        for _ in range(kt_steps):
            step()
        stats = st.kernel_stats()
        st.enable_kernel_timing(False)

    flops_step = 0
    c = 0
    for n in lens:
        flops_step += tp.slice_flops(n, c, H) * n_layers // parts
        c += n
    ms = (t1 - t0) * 1e3 / args.steps
    value = flops_step / (ms * 1e-3) / 1e12
    finite = bool(torch.isfinite(y.float()).all() and torch.isfinite(dx.float()).all())

    roofline = None
    kernels = {}
    if stats:
        for name, s in stats.items():
            secs = max(s["total_ms"], 1e-9) * 1e-3
            kernels[name] = {"launches": s["launches"], "ms_per_step": s["total_ms"] / kt_steps,
                             "avg_us": 1e3 * s["total_ms"] / max(1, s["launches"]),
                             "achieved_tflops": round(s["flops"] / secs / 1e12, 2),
                             "achieved_gbs": round(s["bytes"] / secs / 1e9, 1)}
        # the roofline names one kernel: with deferred weight gradients the
        # largest single kernel is the dW GEMM (one launch per call); the slice
        # GEMM classes are larger only in sum, each call being a split GEMM
        # kernel plus its reduction
        dom = max(stats, key=lambda k: stats[k]["total_ms"])
        if args.wgrad == "deferred" and "gemm_bwd_dw_tn" in stats:
            dom = "gemm_bwd_dw_tn"
        s = stats[dom]
        secs = s["total_ms"] * 1e-3
        traffic = measured_traffic(dom, args.workload,
                                   "accumulate" if args.accumulate_grads else "overwrite")
        if dom.startswith("gemm"):
            ach = s["flops"] / secs / 1e12
            roofline = {"kernel": dom, "bound": "mfma", "achieved": round(ach, 2),
                        "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                        "frac": round(ach / PEAK_BF16_TFLOPS, 4), "traffic": traffic,
                        "algorithmic_bytes_per_launch": round(s["bytes"] / s["launches"])}
        else:
            ach = s["bytes"] / secs / 1e9
            roofline = {"kernel": dom, "bound": "hbm", "achieved": round(ach, 1),
                        "peak": PEAK_HBM_GBS, "unit": "GB/s",
                        "frac": round(ach / PEAK_HBM_GBS, 4), "traffic": traffic}

    out = {
        "metric": "slice fwd+bwd TFLOP/s (whole sequence through one pipeline stage)",
        "value": round(value, 3), "unit": "TFLOP/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms, 3), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": args.workload, "layers": n_layers, "hidden": H, "heads": heads,
                   "seq_len": L, "batch": 1, "slicing": lens, "wgrad": args.wgrad,
                   "grad_buffers": "accumulate" if args.accumulate_grads else "overwrite",
                   **({"slicing_source": dp_source} if dp_source else {}),
                   "global_batch": 1,
                   "parallelism": "one pipeline stage" if parts == 1 else
                   f"one pipeline stage, shard of {parts}-way operation partitioning"},
        "pct_bf16_peak": round(100 * value / PEAK_BF16_TFLOPS, 2),
        "flops_per_step": flops_step, "outputs_finite": finite,
        "roofline": roofline, "kernels": kernels,
        "execution": "eager" if graph is None else "hip graph of one sequence, replayed per step",
        "graph_matches_eager": graph_ok,
    }
    if not args.no_pipeline:
        dw_ms = kernels.get("gemm_bwd_dw_tn", {}).get("ms_per_step", 0.0) if args.wgrad == "deferred" else 0.0
        def run_slicing(sl):
            b = [0]
            for n in sl:
                b.append(b[-1] + n)

            def seq():
                st.reset(overwrite_grads=not args.accumulate_grads)
                for i in range(len(sl)):
                    st.forward(b[i], b[i + 1], x[b[i]:b[i + 1]], out=y[b[i]:b[i + 1]])
                for i in range(len(sl) - 1, -1, -1):
                    st.backward(b[i], b[i + 1], dy[b[i]:b[i + 1]], out=dx[b[i]:b[i + 1]])
            seq()
            torch.cuda.synchronize()
            reps = 3
            ta = time.perf_counter()
            for _ in range(reps):
                seq()
            torch.cuda.synchronize()
            return (time.perf_counter() - ta) * 1e3 / reps

        rep = pipeline_report(st, tp, L, args.pipeline_unit, args.pipeline_K,
                              args.profile_warmup, args.profile_reps,
                              run_slicing, dw_ms, args.pipeline_fine_unit, n_layers, H,
                              args.wgrad == "deferred", op_parts=parts)
        fine_cost = rep.pop("_fine_cost", None)
        if args.joint_batch >= 2 and fine_cost is not None:
            rep["joint"] = joint_report(
                lambda b: tp.Stage(params, H, heads, L, dtype="bf16", wgrad=args.wgrad, batch=b,
                                   op_parts=parts),
                tp, L, args.pipeline_fine_unit, PAPER_K[args.workload], args.joint_batch,
                fine_cost, args.profile_warmup, args.profile_reps)
        out["pipeline"] = rep
        st.zero_grads()
    out["mfma_probe_tflops"] = round(tp.measure_mfma_peak(), 1)
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(params[0], x, dy, H, heads, args.cpu_baseline_tokens,
                                           parts)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
