"""GPU: batch slices (Sec. 3.4) -- b sequences move through the stage together,
token t of sequence s being row t * b + s.  Parity against one oracle run per
sequence (gradients summed), a batch-invariance property on the GPU itself,
and the joint batch x token plan on measured cost tables."""
import numpy as np
import pytest
import torch

from stage_harness import (compare, make_batch_inputs, make_inputs, rel_l2, run_gpu,
                           run_gpu_batch, run_oracle_batch)

pytestmark = pytest.mark.gpu

TOL = {"fp32": 1e-4, "bf16": 2e-2}


def _case(n_layers, H, heads, L, b, dtype, fwd, bwd=None, wgrad="per_slice", seeds=(0, 1, 2),
          randomize_ln=False, label="", overwrite=False):
    print(f"case {label}: layers={n_layers} H={H} heads={heads} L={L} batch={b} {dtype} "
          f"{wgrad} fwd={fwd} bwd={bwd} overwrite={overwrite}", flush=True)
    params, x, dy = make_batch_inputs(n_layers, H, L, b, dtype, seeds, randomize_ln)
    got = run_gpu_batch(params, x, dy, H, heads, L, dtype, fwd, bwd, wgrad,
                        overwrite_grads=overwrite)
    ref = run_oracle_batch(params, x, dy, H, heads, L, fwd, bwd)
    return compare(got, ref, TOL[dtype], label)


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
def test_tiny_batch_of_two(dtype):
    """hidden 64, 4 heads (d = 16: the generic attention), two sequences."""
    _case(1, 64, 4, 32, 2, dtype, [8, 8, 16], seeds=(5, 0, 6), randomize_ln=True,
          label="tiny b=2")


@pytest.mark.parametrize("H,heads", [(256, 2), (256, 4)])  # d = 128, 64: matrix-core attention
@pytest.mark.parametrize("wgrad", ["per_slice", "deferred"])
def test_matrix_core_batch_ragged(H, heads, wgrad):
    """Three sequences, ragged forward slices and different backward slices."""
    _case(2, H, heads, 150, 3, "bf16", [37, 1, 29, 83], [50, 7, 93], wgrad, seeds=(11, 12, 13),
          randomize_ln=True, label=f"mfma-attn d={H // heads} b=3")


@pytest.mark.parametrize("wgrad", ["per_slice", "deferred"])
def test_batch_overwrite_grads(wgrad):
    """Three sequences whose batch stores its gradients over NaN-filled buffers
    (TP_SEQ_OVERWRITE_GRADS): the sum of the sequences' gradients, as the
    oracle gives it."""
    _case(2, 256, 2, 150, 3, "bf16", [37, 1, 29, 83], [50, 7, 93], wgrad, seeds=(14, 15, 16),
          randomize_ln=True, label=f"b=3 overwrite {wgrad}", overwrite=True)


def test_batch_long_backward_slice_in_query_chunks():
    """Two sequences and one 2048-token backward slice: the attention backward
    runs it in two 1024-query chunks of stored dS planes (4 heads of d = 128),
    after ragged forward slices; parity against one oracle run per sequence."""
    _case(1, 512, 4, 2048, 2, "bf16", [1100, 948], [2048], "deferred", seeds=(31, 32, 33),
          randomize_ln=True, label="b=2 query chunks")


def test_fp32_batch_ragged():
    _case(2, 128, 4, 100, 2, "fp32", [37, 1, 29, 33], [50, 7, 43], "deferred", seeds=(3, 4, 5),
          randomize_ln=True, label="fp32 b=2")


@pytest.mark.parametrize("wgrad", ["per_slice", "deferred"])
def test_batch_equals_separate_sequences_fp32(wgrad):
    """A batch of b sequences gives each sequence's own results (and the sum of
    their parameter gradients) -- checked against b batch-1 runs on the GPU."""
    H, heads, L, b = 128, 4, 64, 3
    params, x, dy = make_batch_inputs(2, H, L, b, "fp32", (21, 22, 23))
    got = run_gpu_batch(params, x, dy, H, heads, L, "fp32", [16, 48], [40, 24], wgrad)
    gsum = None
    for s in range(b):
        r = run_gpu(params, x[:, s].contiguous(), dy[:, s].contiguous(), H, heads, L, "fp32",
                    [16, 48], [40, 24], wgrad)
        assert rel_l2(got["y"][:, s], r["y"]) < 1e-5
        assert rel_l2(got["dx"][:, s], r["dx"]) < 1e-5
        if gsum is None:
            gsum = r["grads"]
        else:
            for acc, g in zip(gsum, r["grads"]):
                for k in acc:
                    acc[k] = acc[k] + g[k]
    for g, ref in zip(got["grads"], gsum):
        for k in g:
            assert rel_l2(g[k], ref[k]) < 1e-5, k


def test_joint_plan_on_measured_tables():
    """Cost tables measured at batch 1 and 2 (Eq. 4 per batch slice); the C-ABI
    joint plan (token DP per size, then the batch split) equals the oracle's."""
    from paper_2102_07988_amd import terapipe as tp
    from oracle import joint_slicing
    H, heads, L, unit, B = 256, 2, 256, 32, 2
    U = L // unit
    params, _, _ = make_inputs(2, H, L, "bf16", (1, 2, 3))
    dparams = [{k: v.cuda() for k, v in p.items()} for p in params]
    costs = np.zeros((B, U, U), dtype=np.int64)
    lens = [unit * k for k in range(1, U + 1)]
    ctxs = [unit * j for j in range(U)]
    for b in range(1, B + 1):
        st = tp.Stage(dparams, H, heads, L, dtype="bf16", wgrad="deferred", batch=b)
        tf, tb = st.profile(lens, ctxs, warmup=1, reps=3)
        costs[b - 1] = np.where(tf >= 0, tf + tb, -1)
        del st
    for K in (1, 4, 16):
        groups, T_b, total = tp.joint_slicing(costs, unit, K)
        og, oT, ot = joint_slicing(costs, K)
        assert T_b == oT and total == ot
        assert groups == [(b, [unit * u for u in units]) for b, units in og]
    torch.cuda.synchronize()
