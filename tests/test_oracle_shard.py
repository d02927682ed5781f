"""One device's shard of p-way operation partitioning (the #Op column of
Table 1): heads / p heads and 4H / p FFN units on the full residual stream,
the output and FC2 projections' partial sums taken as the whole sum.

Pin: a full-width block whose other heads and other FFN units have all-zero
weights and biases computes exactly the shard -- their queries, keys and
values are zero, so their attention output is zero; their FFN pre-activations
are zero and GELU(0) = 0; and every extra term of every sum is an exact zero.
So the shard oracle must equal the (separately pinned) full-width oracle on
the embedded weights bit for bit: outputs, input gradients, K/V caches and the
shard's slices of every parameter gradient."""
import numpy as np
import pytest

from oracle import OracleStage
from paper_2102_07988_amd import synth


def embed(shard, H, p):
    """Full-width parameters holding the shard's weights, zeros elsewhere."""
    A, F = H // p, 4 * H // p
    full = {}
    for k in ("ln1_g", "ln1_b", "b_o", "ln2_g", "ln2_b", "b2"):
        full[k] = shard[k].copy()
    w = np.zeros((3 * H, H))
    b = np.zeros(3 * H)
    for part in range(3):  # q, k, v blocks
        w[part * H:part * H + A] = shard["w_qkv"][part * A:(part + 1) * A]
        b[part * H:part * H + A] = shard["b_qkv"][part * A:(part + 1) * A]
    full["w_qkv"], full["b_qkv"] = w, b
    full["w_o"] = np.zeros((H, H))
    full["w_o"][:, :A] = shard["w_o"]
    full["w1"] = np.zeros((4 * H, H))
    full["w1"][:F] = shard["w1"]
    full["b1"] = np.zeros(4 * H)
    full["b1"][:F] = shard["b1"]
    full["w2"] = np.zeros((H, 4 * H))
    full["w2"][:, :F] = shard["w2"]
    return full


def shard_slice(full_grad, k, H, p):
    A, F = H // p, 4 * H // p
    if k == "w_qkv":
        return np.concatenate([full_grad[i * H:i * H + A] for i in range(3)])
    if k == "b_qkv":
        return np.concatenate([full_grad[i * H:i * H + A] for i in range(3)])
    if k == "w_o":
        return full_grad[:, :A]
    if k in ("w1", "b1"):
        return full_grad[:F]
    if k == "w2":
        return full_grad[:, :F]
    return full_grad


@pytest.mark.parametrize("p", [2, 4])
def test_shard_equals_zero_embedded_full_block(p):
    H, heads, L = 64, 4, 24
    params = synth.params_f64(synth.stage_params(2, H, seed=9, randomize_ln=True, op_parts=p))
    x = synth.to_f64(synth.hidden_states(L, H, seed=3))
    dy = synth.to_f64(synth.upstream_grad(L, H, seed=4))
    shard = OracleStage(params, H, heads, L, op_parts=p)
    ys, dxs = shard.run_sequence(x, dy, [8, 4, 12], [12, 12])
    full = OracleStage([embed(q, H, p) for q in params], H, heads, L)
    yf, dxf = full.run_sequence(x, dy, [8, 4, 12], [12, 12])
    assert np.array_equal(ys, yf) and np.array_equal(dxs, dxf)
    A = H // p
    for li in range(2):
        for which in ("k", "v", "dk", "dv"):
            assert np.array_equal(shard.cache(li, which), full.cache(li, which)[:, :A])
        for k in shard.grads[li]:
            assert np.array_equal(shard.grads[li][k], shard_slice(full.grads[li][k], k, H, p)), k
    # and the shard is not trivially the full block
    assert not np.allclose(ys, OracleStage(synth.params_f64(synth.stage_params(
        2, H, seed=9, randomize_ln=True)), H, heads, L).run_sequence(x, dy, [24])[0])


def test_shard_slicing_invariance_bitwise():
    """The accumulation-order rule holds for shards too: any slicing equals the
    whole sequence bit for bit."""
    H, heads, L, p = 64, 4, 20, 2
    params = synth.params_f64(synth.stage_params(1, H, seed=5, op_parts=p))
    x = synth.to_f64(synth.hidden_states(L, H, seed=6))
    dy = synth.to_f64(synth.upstream_grad(L, H, seed=7))
    a = OracleStage(params, H, heads, L, op_parts=p)
    ya, dxa = a.run_sequence(x, dy, [20])
    b = OracleStage(params, H, heads, L, op_parts=p)
    yb, dxb = b.run_sequence(x, dy, [3, 9, 8], [1, 19])
    assert np.array_equal(ya, yb) and np.array_equal(dxa, dxb)
    for k in a.grads[0]:
        assert np.array_equal(a.grads[0][k], b.grads[0][k]), k


def test_shard_rejects_bad_partitioning():
    params = synth.params_f64(synth.stage_params(1, 64, op_parts=1))
    with pytest.raises(ValueError):
        OracleStage(params, 64, 4, 8, op_parts=3)
