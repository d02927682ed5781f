"""Pins of the row-sampling oracle (oracle/rows.py), the reference for sampled
output rows of full-size stages: it must reproduce the slice-by-slice oracle
(itself pinned to autograd, finite differences and slicing invariance) on
small stages, and honour the causal mask (Sec. 3.1: row t depends on tokens
0..t only)."""
import numpy as np
import pytest

from oracle import OracleStage, PARAM_NAMES
from oracle.rows import stage_output_rows


def _params(rng, n_layers, H):
    shapes = {"ln1_g": (H,), "ln1_b": (H,), "w_qkv": (3 * H, H), "b_qkv": (3 * H,),
              "w_o": (H, H), "b_o": (H,), "ln2_g": (H,), "ln2_b": (H,), "w1": (4 * H, H),
              "b1": (4 * H,), "w2": (H, 4 * H), "b2": (H,)}
    out = []
    for _ in range(n_layers):
        p = {k: rng.normal(0.0, 0.2, size=s) for k, s in shapes.items()}
        p["ln1_g"] += 1.0
        p["ln2_g"] += 1.0
        out.append(p)
    return out


@pytest.mark.parametrize("n_layers,H,heads,L", [(1, 32, 2, 20), (2, 64, 4, 40), (3, 48, 3, 33)])
def test_rows_equal_slice_oracle(n_layers, H, heads, L):
    rng = np.random.default_rng(5 + n_layers)
    params = _params(rng, n_layers, H)
    x = rng.normal(size=(L, H))
    st = OracleStage(params, H, heads, L)
    y = np.concatenate([st.forward(0, 7, x[:7]), st.forward(7, 19, x[7:19]),
                        st.forward(19, L, x[19:])])
    rows = [0, 1, 6, 7, 18, 19, L - 2, L - 1]
    got = stage_output_rows(params, x, heads, rows)
    err = np.abs(got - y[rows]).max() / np.abs(y[rows]).max()
    assert err < 1e-12, err


def test_rows_ignore_later_tokens():
    rng = np.random.default_rng(9)
    H, heads, L = 32, 4, 24
    params = _params(rng, 2, H)
    x = rng.normal(size=(L, H))
    a = stage_output_rows(params, x, heads, [5, 11])
    x2 = x.copy()
    x2[12:] = rng.normal(size=(L - 12, H))
    b = stage_output_rows(params, x2, heads, [5, 11])
    np.testing.assert_array_equal(a, b)
    # and a change at token 11 reaches row 11 but not row 5
    x3 = x.copy()
    x3[11] += 1.0
    c = stage_output_rows(params, x3, heads, [5, 11])
    np.testing.assert_array_equal(a[0], c[0])
    assert np.abs(a[1] - c[1]).max() > 1e-3


def test_rows_reject_out_of_range():
    rng = np.random.default_rng(1)
    params = _params(rng, 1, 16)
    x = rng.normal(size=(8, 16))
    with pytest.raises(ValueError):
        stage_output_rows(params, x, 2, [8])
    with pytest.raises(ValueError):
        stage_output_rows(params, x, 2, [])
    assert set(PARAM_NAMES) == set(params[0])
