"""Selected output rows of a stage of pre-LN blocks at full size, in fp64 --
TEST INFRASTRUCTURE ONLY.

The slice-by-slice oracle (tp_oracle.c) runs plain loops and is far too slow
for a whole sequence at hidden size 12288.  Single rows of the stage output can
still be computed exactly: under the causal mask the output of token t depends
on tokens 0..t only (Sec. 3.1: each position attends to itself and the
positions before it), so every layer but the last is evaluated for tokens
0..T-1 (T = 1 + the largest requested row), and the last layer needs its keys
and values for 0..T-1 plus the requested rows themselves.

The block is the one the slice oracle evaluates (the GPT block of the paper's
Eq. 2-3 with the pre-LayerNorm arrangement of GPT-3):
  u  = LN1(x)            biased variance, eps inside the square root, affine
  [q, k, v] = u W_qkv^T + b_qkv      W_qkv is [3H, H]; head h owns columns
                                     h d .. h d + d - 1 of each of q, k, v
  o_t = sum_{s <= t} softmax_s(q_t . k_s / sqrt(d)) v_s   per head
  x1 = x + o W_o^T + b_o
  y  = x1 + GELU(LN2(x1) W_1^T + b_1) W_2^T + b_2        GELU in tanh form
Library matrix products (numpy) are the only steps beyond the definition; the
sums are not reordered beyond what a matrix product does.
"""
from __future__ import annotations

from typing import Dict, List, Sequence

import numpy as np

_GELU_C = float(np.sqrt(2.0 / np.pi))
_GELU_A = 0.044715


def _ln(x: np.ndarray, g: np.ndarray, b: np.ndarray, eps: float) -> np.ndarray:
    mu = x.mean(axis=-1, keepdims=True)
    var = ((x - mu) ** 2).mean(axis=-1, keepdims=True)
    return (x - mu) / np.sqrt(var + eps) * g + b


def _gelu(z: np.ndarray) -> np.ndarray:
    return 0.5 * z * (1.0 + np.tanh(_GELU_C * (z + _GELU_A * z * z * z)))


def _ffn_residual(p: Dict[str, np.ndarray], x1: np.ndarray, eps: float,
                  chunk: int = 512) -> np.ndarray:
    """x1 + FC2(GELU(FC1(LN2(x1)))), rows in chunks to bound the [rows, 4H] temporaries."""
    out = np.empty_like(x1)
    for a in range(0, x1.shape[0], chunk):
        u2 = _ln(x1[a:a + chunk], p["ln2_g"], p["ln2_b"], eps)
        g = _gelu(u2 @ p["w1"].T + p["b1"])
        out[a:a + chunk] = x1[a:a + chunk] + g @ p["w2"].T + p["b2"]
    return out


def _qkv(p: Dict[str, np.ndarray], x: np.ndarray, eps: float, parts=("q", "k", "v")):
    H = x.shape[1]
    u = _ln(x, p["ln1_g"], p["ln1_b"], eps)
    out = {}
    for i, name in enumerate(("q", "k", "v")):
        if name in parts:
            w = p["w_qkv"][i * H:(i + 1) * H]
            out[name] = u @ w.T + p["b_qkv"][i * H:(i + 1) * H]
    return out


def _block_all_rows(p: Dict[str, np.ndarray], x: np.ndarray, heads: int,
                    eps: float) -> np.ndarray:
    """One block over tokens 0..T-1 (every row)."""
    T, H = x.shape
    d = H // heads
    t = _qkv(p, x, eps)
    q, k, v = t["q"], t["k"], t["v"]
    o = np.empty_like(q)
    future = np.triu(np.ones((T, T), dtype=bool), 1)
    for h in range(heads):
        c = slice(h * d, (h + 1) * d)
        s = (q[:, c] @ k[:, c].T) / np.sqrt(d)
        s[future] = -np.inf
        s -= s.max(axis=1, keepdims=True)
        w = np.exp(s)
        w /= w.sum(axis=1, keepdims=True)
        o[:, c] = w @ v[:, c]
    x1 = x + o @ p["w_o"].T + p["b_o"]
    return _ffn_residual(p, x1, eps)


def _block_rows(p: Dict[str, np.ndarray], x: np.ndarray, rows: Sequence[int], heads: int,
                eps: float) -> np.ndarray:
    """One block's output at the given rows; x holds tokens 0..max(rows)."""
    H = x.shape[1]
    d = H // heads
    kv = _qkv(p, x, eps, parts=("k", "v"))
    k, v = kv["k"], kv["v"]
    xr = x[list(rows)]
    q = _qkv(p, xr, eps, parts=("q",))["q"]
    o = np.empty_like(q)
    for i, t in enumerate(rows):
        for h in range(heads):
            c = slice(h * d, (h + 1) * d)
            s = (k[:t + 1, c] @ q[i, c]) / np.sqrt(d)
            w = np.exp(s - s.max())
            w /= w.sum()
            o[i, c] = w @ v[:t + 1, c]
    x1 = xr + o @ p["w_o"].T + p["b_o"]
    return _ffn_residual(p, x1, eps)


def stage_output_rows(params: List[Dict[str, np.ndarray]], x: np.ndarray, heads: int,
                      rows: Sequence[int], eps: float = 1e-5) -> np.ndarray:
    """Stage output y[rows] (fp64) for input x [>= max(rows) + 1, H] and per-layer
    parameters (weights [out, in]); every layer but the last runs over all of
    tokens 0..max(rows)."""
    rows = [int(r) for r in rows]
    if not rows or min(rows) < 0 or max(rows) >= x.shape[0]:
        raise ValueError("rows out of range")
    T = max(rows) + 1
    h = np.asarray(x[:T], dtype=np.float64)
    ps = [{k: np.asarray(v, dtype=np.float64) for k, v in p.items()} for p in params]
    for p in ps[:-1]:
        h = _block_all_rows(p, h, heads, eps)
    return _block_rows(ps[-1], h, rows, heads, eps)
