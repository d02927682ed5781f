"""GPU: one device's shard of p-way operation partitioning (Table 1's #Op
column): heads / p heads and 4H / p FFN units on the full residual stream,
checked against the shard oracle (itself pinned bit for bit to the full-width
oracle on zero-embedded weights) on the same seeded inputs."""
import pytest
import torch

from stage_harness import (compare, make_batch_inputs, make_inputs, run_gpu, run_gpu_batch,
                           run_oracle, run_oracle_batch)

pytestmark = pytest.mark.gpu

TOL = {"fp32": 1e-4, "bf16": 2e-2}


def _case(n_layers, H, heads, p, L, dtype, fwd, bwd=None, wgrad="per_slice", seeds=(0, 1, 2),
          label=""):
    print(f"case {label}: layers={n_layers} H={H} heads={heads} op_parts={p} L={L} {dtype} "
          f"{wgrad} fwd={fwd} bwd={bwd}", flush=True)
    params, x, dy = make_inputs(n_layers, H, L, dtype, seeds, True, op_parts=p)
    got = run_gpu(params, x, dy, H, heads, L, dtype, fwd, bwd, wgrad, op_parts=p)
    ref = run_oracle(params, x, dy, H, heads, L, fwd, bwd, op_parts=p)
    return compare(got, ref, TOL[dtype], label)


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
@pytest.mark.parametrize("p", [2, 4])
def test_tiny_shard(dtype, p):
    """hidden 64, 4 heads (d = 16): 2 or 1 local heads, FFN 128 or 64."""
    _case(1, 64, 4, p, 32, dtype, [8, 8, 16], seeds=(0, 1, 2), label=f"tiny p={p}")


@pytest.mark.parametrize("wgrad", ["per_slice", "deferred"])
@pytest.mark.parametrize("H,heads,p", [(512, 8, 2), (1024, 8, 8), (1024, 16, 4)])
def test_matrix_core_shard_ragged(H, heads, p, wgrad):
    """bf16, d = 64 or 128 on the matrix-core attention; attention width H/p of
    256, 128 or 256; ragged slices with different backward boundaries."""
    _case(2, H, heads, p, 150, "bf16", [37, 1, 29, 83], [50, 7, 93], wgrad, seeds=(4, 5, 6),
          label=f"H={H} heads={heads} p={p}")


@pytest.mark.parametrize("wgrad", ["per_slice", "deferred"])
def test_shard_stored_ds_backward(wgrad):
    """A 2-way shard with 16 local heads of d = 64 (attention width 1024 on a
    2048 residual) over 1024 tokens: the backward slice ending at 1024 has
    enough key blocks for the stored-dS path, the one ending at 400 takes the
    small-grid kernels."""
    _case(1, 2048, 32, 2, 1024, "bf16", [300, 100, 624], [400, 624], wgrad, seeds=(51, 52, 53),
          label=f"shard p=2 stored dS {wgrad}")


@pytest.mark.parametrize("overwrite", [False, True])
def test_shard_with_batch(overwrite):
    """Operation partitioning and batch slices together (setting (10) of Table 1
    has both): two sequences through an 8-way shard; also with the gradients
    stored over NaN-filled buffers (TP_SEQ_OVERWRITE_GRADS)."""
    H, heads, p, L = 1024, 8, 8, 96
    params, x, dy = make_batch_inputs(2, H, L, 2, "bf16", (7, 8, 9), True, op_parts=p)
    got = run_gpu_batch(params, x, dy, H, heads, L, "bf16", [40, 56], [64, 32], "deferred",
                        op_parts=p, overwrite_grads=overwrite)
    ref = run_oracle_batch(params, x, dy, H, heads, L, [40, 56], [64, 32], op_parts=p)
    compare(got, ref, TOL["bf16"], f"shard p=8 batch 2 overwrite={overwrite}")


def test_random_slicings_shard_with_batch():
    """Eight seeded random forward and backward slicings (lengths 1..160) of
    two sequences through a 2-way shard (2 local heads of d = 128 on a 512
    residual), alternating weight-gradient and gradient-buffer modes, against
    one oracle run per sequence (gradients summed)."""
    import numpy as np
    from paper_2102_07988_amd import terapipe as tp
    H, heads, p, L, b = 512, 4, 2, 400, 2
    params, x, dy = make_batch_inputs(2, H, L, b, "bf16", (71, 72, 73), True, op_parts=p)
    ref = run_oracle_batch(params, x, dy, H, heads, L, [L], op_parts=p)
    rng = np.random.default_rng(3402)
    dparams = [{k: v.cuda() for k, v in q.items()} for q in params]
    xd, dyd = x.cuda(), dy.cuda()
    stages = {w: tp.Stage(dparams, H, heads, L, dtype="bf16", wgrad=w, batch=b, op_parts=p)
              for w in ("per_slice", "deferred")}

    def slicing():
        lens = []
        while sum(lens) < L:
            lens.append(int(min(rng.integers(1, 161), L - sum(lens))))
        return lens

    for case in range(8):
        fwd, bwd = slicing(), slicing()
        wgrad = ("per_slice", "deferred")[case % 2]
        overwrite = case % 4 >= 2
        st = stages[wgrad]
        print(f"case {case}: {wgrad} overwrite={overwrite} fwd={fwd} bwd={bwd}", flush=True)
        if overwrite:
            for g in st.grads:
                for v in g.values():
                    v.fill_(float("nan"))
        else:
            st.zero_grads()
        y, dx = st.run_sequence(xd, dyd, fwd, bwd, overwrite_grads=overwrite)
        torch.cuda.synchronize()
        got = {"y": y.float().cpu().numpy(), "dx": dx.float().cpu().numpy(),
               "grads": [{k: v.cpu().numpy() for k, v in g.items()} for g in st.grads]}
        compare(got, ref, TOL["bf16"], f"shard p=2 batch 2 random slicing {case}")
