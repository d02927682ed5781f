"""Pins of the whole-sequence float64 oracle (oracle/full.py), which the
full-width GPU parity tests use where the slice oracle's plain loops are too
slow.

* It equals the slice oracle (tp_oracle.c, itself pinned to autograd, finite
  differences and slicing invariance) on every output and gradient, for
  several layer counts, head counts, sliced runs of the slice oracle, and an
  operation-partitioning shard.
* It equals PyTorch float64 autograd of a textbook pre-LN block built from
  library routines (layer_norm, linear, causal scaled-dot-product attention,
  tanh GELU), so its hand-written backward is checked against an independent
  differentiation, not only against the other oracle.
* Properties: causality (changing later inputs leaves earlier outputs
  unchanged) and a closed form (zero projections make the block the identity,
  dx = dy and the weight gradients of W_o and W2 vanish with zero inputs).
"""
import numpy as np
import pytest
import torch

from oracle import OracleStage, PARAM_NAMES
from oracle.full import stage_forward_backward
from paper_2102_07988_amd import synth
from test_oracle_stage import torch_block_reference


def rel(a, b):
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    nb = np.linalg.norm(b)
    return np.linalg.norm(a - b) / (nb if nb > 0 else 1.0)


def _inputs(n_layers, H, L, seed, op_parts=1):
    params = synth.params_f64(synth.stage_params(n_layers, H, seed=seed, randomize_ln=True,
                                                 op_parts=op_parts))
    x = synth.to_f64(synth.hidden_states(L, H, seed=seed))
    dy = synth.to_f64(synth.upstream_grad(L, H, seed=seed + 1))
    return params, x, dy


@pytest.mark.parametrize("n_layers,H,heads,L,fwd,bwd,op_parts", [
    (1, 64, 4, 32, [8, 8, 16], None, 1),
    (2, 64, 2, 40, [40], [13, 27], 1),
    (2, 128, 8, 48, [16, 1, 31], [48], 1),
    (1, 128, 4, 33, [20, 13], None, 2),
])
def test_equals_slice_oracle(n_layers, H, heads, L, fwd, bwd, op_parts):
    params, x, dy = _inputs(n_layers, H, L, 5 + n_layers, op_parts)
    st = OracleStage(params, H, heads, L, op_parts=op_parts)
    y_ref, dx_ref = st.run_sequence(x, dy, fwd, bwd)
    y, dx, grads = stage_forward_backward(params, x, dy, heads // op_parts)
    assert rel(y.numpy(), y_ref) < 1e-12
    assert rel(dx.numpy(), dx_ref) < 1e-11
    for li in range(n_layers):
        for k in PARAM_NAMES:
            assert rel(grads[li][k].numpy(), st.grads[li][k]) < 1e-11, (li, k)


@pytest.mark.parametrize("n_layers,heads", [(1, 4), (2, 2)])
def test_equals_torch_autograd(n_layers, heads):
    H, L = 64, 32
    params, x, dy = _inputs(n_layers, H, L, 11)
    y_ref, dx_ref, g_ref = torch_block_reference(params, x, dy, heads)
    y, dx, grads = stage_forward_backward(params, x, dy, heads)
    assert rel(y.numpy(), y_ref) < 1e-12
    assert rel(dx.numpy(), dx_ref) < 1e-10
    for li in range(n_layers):
        for k in PARAM_NAMES:
            assert rel(grads[li][k].numpy(), g_ref[li][k]) < 1e-10, (li, k)


def test_causality():
    """Outputs of tokens 0..t depend on inputs 0..t only (Eq. 2 sums over s <= t);
    input gradients of tokens t.. depend on upstream gradients t.. only."""
    H, heads, L, t = 64, 4, 24, 10
    params, x, dy = _inputs(2, H, L, 3)
    y, dx, _ = stage_forward_backward(params, x, dy, heads)
    x2 = x.copy()
    x2[t:] += np.random.default_rng(0).normal(size=x2[t:].shape)
    dy2 = dy.copy()
    dy2[:t] += 1.0
    y2, _, _ = stage_forward_backward(params, x2, dy, heads)
    _, dx2, _ = stage_forward_backward(params, x, dy2, heads)
    assert torch.equal(y[:t], y2[:t]) and not torch.equal(y[t:], y2[t:])
    assert torch.allclose(dx[t:], dx2[t:], rtol=0, atol=1e-12)
    assert not torch.allclose(dx[:t], dx2[:t])


def test_zero_projections_closed_form():
    """With every projection weight and bias zero the block is the identity:
    y = x, dx = dy; the gradients of the output-side biases are column sums of dy
    and the LayerNorm-parameter gradients vanish (nothing downstream of the
    LayerNorms reaches y)."""
    H, heads, L = 64, 4, 16
    params, x, dy = _inputs(1, H, L, 9)
    for k in ("w_qkv", "b_qkv", "w_o", "b_o", "w1", "b1", "w2", "b2"):
        params[0][k] = np.zeros_like(params[0][k])
    y, dx, g = stage_forward_backward(params, x, dy, heads)
    assert torch.equal(y, torch.from_numpy(x))
    assert torch.equal(dx, torch.from_numpy(dy))
    colsum = torch.from_numpy(dy).sum(dim=0)
    assert torch.allclose(g[0]["b2"], colsum, rtol=0, atol=1e-12)
    assert torch.allclose(g[0]["b_o"], colsum, rtol=0, atol=1e-12)
    for k in ("ln1_g", "ln1_b", "ln2_g", "ln2_b", "w_qkv", "b_qkv", "w1"):
        assert float(g[0][k].abs().max()) == 0.0, k
