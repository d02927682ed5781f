"""Every output and every gradient of the full-width stages against the
whole-sequence float64 oracle (oracle/full.py), on the GPU through the C ABI.

The method computes exactly what processing the sequence whole computes
(Sec. 3.2; Sec. 4 compares against the same optimisation), so one oracle run
of a stage serves every slicing and weight-gradient mode the GPU runs.  The
cases run the benchmark's launch configurations at their real widths, which
select kernel instances that narrower shapes never reach: 256 x 192 output
tiles and their transposing-read swizzle, five-way split dX products, the
XCD-ordered tile walk of the deferred weight-gradient GEMMs (512 tiles and
more), unsplit d = 128 dQ launches.

* GPT-3-175B width (hidden 12288, 96 heads), one layer, 512 tokens: forward
  2 x 256; backward 2 x 256 with per-slice weight gradients and 1 x 512
  deferred; the fp32 validation mode on the same shape (1e-4).
* GPT-3-13B stage (2 layers, hidden 5120, 40 heads, 2048 tokens) on the
  slicing the DP (Algorithm 1) picks from a model-mode cost table (Eq. 9)
  measured on this GPU at the paper's pipeline depth K = 20, slice lengths in
  multiples of 16; and per-slice weight gradients with another backward slicing.
* GPT-3-175B stage (2 layers, 2048 tokens): the benchmark's 8 x 256 with
  deferred weight gradients stored over NaN-filled buffers (as the benchmark
  runs it), the DP slicing at K = 48, and per-slice weight gradients with
  4 x 512 backward slices.
* One GPU's shard of the paper's 175B settings with operation partitioning
  (Table 1 settings (10) and (9)): 8-way (2 layers) and 4-way (1 layer).
* Hidden 11136 (87 heads), whose query/key/value product runs as two split
  launches over column groups, the second ending in a partial tile.
* The largest shapes the stage accepts: hidden 16384 (128 heads, one layer,
  256 tokens in ragged slices), and the longest sequence, 20344 tokens (the
  generic attention's one-row-per-block LDS limit; hidden 256, 2 heads of
  128), in ragged slices of up to 8192 tokens and a short last slice after
  a 20000-token prefix.

Tolerance: rel-L2 2e-2 per tensor in bf16 (y, dx and each of the 12
parameter gradients of every layer), 1e-4 in the fp32 validation mode.
"""
import gc
import time

import pytest
import torch

from oracle.full import stage_forward_backward
from paper_2102_07988_amd import synth

pytestmark = [pytest.mark.gpu, pytest.mark.timeout(900)]

TOL = {"bf16": 2e-2, "fp32": 1e-4}
NAMES = synth.PARAM_NAMES


def log(msg):
    print(f"[{time.strftime('%H:%M:%S')}] {msg}", flush=True)


def rel_l2(a: torch.Tensor, b: torch.Tensor) -> float:
    a = a.to(torch.float64)
    b = b.to(torch.float64)
    nb = float(torch.linalg.vector_norm(b))
    d = float(torch.linalg.vector_norm(a - b))
    return d / nb if nb > 0 else d


def inputs(n_layers, H, L, dtype, op_parts=1):
    dev = torch.device("cuda:0")
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    params = synth.stage_params(n_layers, H, seed=synth.SEED_PARAMS, dtype=tdt, device=dev,
                                op_parts=op_parts)
    x = synth.hidden_states(L, H, seed=synth.SEED_X, dtype=tdt, device=dev)
    dy = synth.upstream_grad(L, H, seed=synth.SEED_DY, dtype=tdt, device=dev)
    return params, x, dy


def oracle(params, x, dy, heads_local):
    t0 = time.time()
    cpu = [{k: v.cpu() for k, v in p.items()} for p in params]
    y, dx, grads = stage_forward_backward(cpu, x.cpu(), dy.cpu(), heads_local, log=log)
    del cpu
    gc.collect()
    log(f"oracle done in {time.time() - t0:.0f} s")
    return {"y": y, "dx": dx, "grads": grads}


def dp_slicing(params, H, heads, L, K, unit, op_parts=1):
    """The DP's slicing (Algorithm 1) on a model-mode cost table (Eq. 9)
    measured on this GPU, as the benchmark's --slicing dp takes it."""
    from paper_2102_07988_amd import terapipe as tp
    st = tp.Stage(params, H, heads, L, dtype="bf16", wgrad="deferred", op_parts=op_parts)
    U = L // unit
    ks = sorted({k for k in (1, 2, U // 8, U // 4, U // 2, 3 * U // 4) if 1 <= k < U})
    js = sorted({j for j in (1, U // 8, U // 4, U // 2, 3 * U // 4) if 1 <= j < U})
    cost, _ = st.profile_model(L, unit, [unit * k for k in ks], [unit * j for j in js],
                               warmup=1, reps=3)
    lens, _ = tp.dp_optimal_slicing(cost, unit, K)
    del st
    torch.cuda.synchronize()
    log(f"DP slicing (K={K}, unit {unit}): {lens}")
    assert sum(lens) == L and all(n % unit == 0 for n in lens)
    return lens


def check_run(ref, params, x, dy, H, heads, L, dtype, fwd, bwd, wgrad, label, op_parts=1,
              overwrite=False):
    """overwrite: the gradient buffers start NaN-filled and the sequence stores
    its gradients (TP_SEQ_OVERWRITE_GRADS, as the benchmark runs it)."""
    from paper_2102_07988_amd import terapipe as tp
    log(f"case {label}: H={H} heads={heads} L={L} {dtype} {wgrad} op_parts={op_parts} "
        f"fwd={fwd} bwd={bwd} overwrite={overwrite}")
    st = tp.Stage(params, H, heads, L, dtype=dtype, wgrad=wgrad, op_parts=op_parts)
    if overwrite:
        for g in st.grads:
            for v in g.values():
                v.fill_(float("nan"))
    y, dx = st.run_sequence(x, dy, fwd, bwd, overwrite_grads=overwrite)
    torch.cuda.synchronize()
    errs = {"y": rel_l2(y.cpu(), ref["y"]), "dx": rel_l2(dx.cpu(), ref["dx"])}
    del y, dx
    for li, g in enumerate(st.grads):
        for k in NAMES:
            errs[f"L{li}.{k}"] = rel_l2(g[k].cpu(), ref["grads"][li][k])
    del st
    gc.collect()
    torch.cuda.empty_cache()
    worst = max(errs, key=errs.get)
    log(f"  [{label}] worst rel-L2 {worst} = {errs[worst]:.3e}; y {errs['y']:.2e}, "
        f"dx {errs['dx']:.2e}")
    bad = {k: v for k, v in errs.items() if not v <= TOL[dtype]}
    assert not bad, f"{label}: rel-L2 above {TOL[dtype]}: {bad}"
    return errs


@pytest.mark.parametrize("dtype", ["bf16", "fp32"])
def test_175b_width_one_layer_512_tokens(dtype):
    H, heads, L = 12288, 96, 512
    params, x, dy = inputs(1, H, L, dtype)
    ref = oracle(params, x, dy, heads)
    check_run(ref, params, x, dy, H, heads, L, dtype, [256, 256], [256, 256], "per_slice",
              "175B width, per-slice dW")
    check_run(ref, params, x, dy, H, heads, L, dtype, [256, 256], [512], "deferred",
              "175B width, deferred dW, one 512-token backward slice")


def test_13b_stage_dp_slicing_full_sequence():
    H, heads, L = 5120, 40, 2048
    params, x, dy = inputs(2, H, L, "bf16")
    lens = dp_slicing(params, H, heads, L, K=20, unit=16)
    ref = oracle(params, x, dy, heads)
    check_run(ref, params, x, dy, H, heads, L, "bf16", lens, None, "deferred",
              "13B stage, DP slicing")
    check_run(ref, params, x, dy, H, heads, L, "bf16", [256] * 8, [400, 352, 304, 256, 224,
                                                                  176, 144, 112, 80],
              "per_slice", "13B stage, per-slice dW, other backward slicing")


def test_175b_stage_full_sequence():
    H, heads, L = 12288, 96, 2048
    params, x, dy = inputs(2, H, L, "bf16")
    lens = dp_slicing(params, H, heads, L, K=48, unit=16)
    ref = oracle(params, x, dy, heads)
    check_run(ref, params, x, dy, H, heads, L, "bf16", [256] * 8, None, "deferred",
              "175B stage, benchmark configuration 8 x 256, gradients stored", overwrite=True)
    check_run(ref, params, x, dy, H, heads, L, "bf16", lens, None, "deferred",
              "175B stage, DP slicing")
    check_run(ref, params, x, dy, H, heads, L, "bf16", [256] * 8, [512] * 4, "per_slice",
              "175B stage, per-slice dW, 4 x 512 backward")


@pytest.mark.parametrize("n_layers,parts", [(2, 8), (1, 4)])
def test_175b_operation_partitioning_shard_full_sequence(n_layers, parts):
    H, heads, L = 12288, 96, 2048
    params, x, dy = inputs(n_layers, H, L, "bf16", op_parts=parts)
    ref = oracle(params, x, dy, heads // parts)
    check_run(ref, params, x, dy, H, heads, L, "bf16", [256] * 8, None, "deferred",
              f"175B {parts}-way shard, {n_layers} layer(s)", op_parts=parts)


def test_maximum_hidden_size():
    """Hidden size 16384 (the LayerNorm kernels' register limit), 128 heads of
    128, one layer; ragged forward and backward slicings, both weight-gradient
    modes."""
    H, heads, L = 16384, 128, 256
    params, x, dy = inputs(1, H, L, "bf16")
    ref = oracle(params, x, dy, heads)
    check_run(ref, params, x, dy, H, heads, L, "bf16", [100, 156], [200, 56], "per_slice",
              "hidden 16384, per-slice dW")
    check_run(ref, params, x, dy, H, heads, L, "bf16", [100, 156], None, "deferred",
              "hidden 16384, deferred dW")


def test_two_group_split_with_ragged_tail():
    """Hidden 11136 (87 heads of 128), one layer, 256 tokens: the tile model runs
    the 33408-wide query/key/value product as two split launches over column
    groups (128 tiles of 256 columns, then the last 2.5 tiles), the second
    ending in a partial tile."""
    H, heads, L = 11136, 87, 256
    params, x, dy = inputs(1, H, L, "bf16")
    ref = oracle(params, x, dy, heads)
    check_run(ref, params, x, dy, H, heads, L, "bf16", [256], None, "deferred",
              "hidden 11136, two-group query/key/value product")


def test_maximum_sequence_length():
    """The longest sequence a stage accepts, 20344 tokens, at hidden 256 (2 heads
    of 128): slices of 8192 tokens and a ragged tail, and a 344-token slice
    after a 20000-token prefix."""
    H, heads, L = 256, 2, 20344
    params, x, dy = inputs(1, H, L, "bf16")
    ref = oracle(params, x, dy, heads)
    check_run(ref, params, x, dy, H, heads, L, "bf16", [8192, 8192, 3960], [5000, 15344],
              "per_slice", "20344 tokens, per-slice dW")
    check_run(ref, params, x, dy, H, heads, L, "bf16", [20000, 344], None, "deferred",
              "20344 tokens, short slice after a 20000-token prefix")
