"""Whole-sequence forward and backward of a stage at full size, in float64 --
TEST INFRASTRUCTURE ONLY (only tests/ may use it).

Token slicing changes when each token is processed, not what is computed
(Sec. 3.2: a cell runs the slices in order and each slice attends to the keys
and values of every earlier position, Eq. 2; the feed-forward part is per
token, Eq. 3).  So for any slicing the stage's outputs and gradients are those
of the whole sequence processed at once, and those are what this module
computes: the stage output y for an input x [L, H], and the exact gradient of
the scalar sum(y * dy) with respect to x and to every parameter.

The slice oracle (tp_oracle.c) computes the same with plain loops, but is far
too slow at hidden sizes 5120 and 12288.  Here the same pre-LayerNorm block
(the GPT-3 block of the evaluation setting, Sec. 4) is written with library
matrix products (PyTorch CPU, float64) as steps, and differentiated by hand,
one step at a time in reverse (no autograd):

  forward, per layer                     backward, per layer (g_* = dL/d*)
  u  = LN1(x)                            g_W2 = g_y^T a,  g_b2 = sum_t g_y,  g_a = g_y W2
  [q,k,v] = u W_qkv^T + b_qkv            g_z = g_a * GELU'(z)
  o  = causal attention(q, k, v)         g_W1 = g_z^T u2, g_b1 = sum_t g_z,  g_u2 = g_z W1
  x1 = x + o W_o^T + b_o                 g_x1 = g_y + LN2^T(g_u2)  (+ gain/bias grads)
  u2 = LN2(x1)                           g_Wo = g_x1^T o, g_bo = sum_t g_x1, g_o = g_x1 W_o
  z  = u2 W1^T + b1, a = GELU(z)         attention backward per head (below)
  y  = x1 + a W2^T + b2                  g_Wqkv = g_qkv^T u, g_bqkv = sum_t g_qkv, g_u = g_qkv W_qkv
                                         g_x = g_x1 + LN1^T(g_u)   (+ gain/bias grads)

LayerNorm: biased variance, eps inside the square root, affine gain and bias.
GELU: tanh form.  Attention per head h of width d: scores
S = q_h k_h^T / sqrt(d) with keys s > query t removed (the inclusive causal sum
of Eq. 2), P = row softmax of S, o_h = P v_h; its backward
g_P = g_o,h v_h^T, g_v,h = P^T g_o,h, g_S = P * (g_P - rowsum(g_P * P)),
g_q,h = g_S k_h / sqrt(d), g_k,h = g_S^T q_h / sqrt(d).

Parameter shapes are taken from the arrays (attention width A = a third of
the rows of W_qkv, FFN width F = the rows of W1), so one device's shard of
operation partitioning is the same code with `heads` = the shard's heads.
"""
from __future__ import annotations

import math
from typing import Callable, Dict, List, Optional, Sequence, Tuple

import torch

GELU_C = math.sqrt(2.0 / math.pi)
GELU_A = 0.044715
PARAM_NAMES = ("ln1_g", "ln1_b", "w_qkv", "b_qkv", "w_o", "b_o",
               "ln2_g", "ln2_b", "w1", "b1", "w2", "b2")


def _f64(t) -> torch.Tensor:
    return torch.as_tensor(t).to(device="cpu", dtype=torch.float64)


def _ln(x: torch.Tensor, g: torch.Tensor, b: torch.Tensor, eps: float):
    """LayerNorm of every row; returns (u, xhat, rstd)."""
    mean = x.mean(dim=1, keepdim=True)
    xc = x - mean
    rstd = 1.0 / torch.sqrt((xc * xc).mean(dim=1, keepdim=True) + eps)
    xhat = xc * rstd
    return xhat * g + b, xhat, rstd


def _ln_back(gu: torch.Tensor, xhat: torch.Tensor, rstd: torch.Tensor, g: torch.Tensor):
    """Input gradient of u = g * xhat + b, xhat = (x - mean(x)) * rstd(x):
    rstd * (gxh - mean(gxh) - xhat * mean(gxh * xhat)), gxh = gu * g."""
    gxh = gu * g
    return rstd * (gxh - gxh.mean(dim=1, keepdim=True)
                   - xhat * (gxh * xhat).mean(dim=1, keepdim=True))


def _gelu(z: torch.Tensor) -> torch.Tensor:
    return 0.5 * z * (1.0 + torch.tanh(GELU_C * (z + GELU_A * z * z * z)))


def _gelu_grad(z: torch.Tensor) -> torch.Tensor:
    th = torch.tanh(GELU_C * (z + GELU_A * z * z * z))
    return 0.5 * (1.0 + th) + 0.5 * z * (1.0 - th * th) * GELU_C * (1.0 + 3.0 * GELU_A * z * z)


def _probs(qh: torch.Tensor, kh: torch.Tensor, scale: float, future: torch.Tensor):
    """Row softmax of the causal scores of one head, [L, L]."""
    s = (qh @ kh.T) * scale
    s.masked_fill_(future, -math.inf)
    s -= s.max(dim=1, keepdim=True).values
    p = torch.exp(s)
    p /= p.sum(dim=1, keepdim=True)
    return p


def _layer_forward(p: Dict[str, torch.Tensor], x: torch.Tensor, heads: int, eps: float,
                   future: torch.Tensor):
    A = p["w_qkv"].shape[0] // 3
    d = A // heads
    scale = 1.0 / math.sqrt(d)
    u, xh1, rs1 = _ln(x, p["ln1_g"], p["ln1_b"], eps)
    qkv = u @ p["w_qkv"].T + p["b_qkv"]
    q, k, v = qkv[:, :A], qkv[:, A:2 * A], qkv[:, 2 * A:]
    o = torch.empty_like(q)
    for h in range(heads):
        c = slice(h * d, (h + 1) * d)
        o[:, c] = _probs(q[:, c], k[:, c], scale, future) @ v[:, c]
    x1 = x + o @ p["w_o"].T + p["b_o"]
    u2, xh2, rs2 = _ln(x1, p["ln2_g"], p["ln2_b"], eps)
    z = u2 @ p["w1"].T + p["b1"]
    a = _gelu(z)
    y = x1 + a @ p["w2"].T + p["b2"]
    saved = {"u": u, "xh1": xh1, "rs1": rs1, "qkv": qkv, "o": o, "xh2": xh2, "rs2": rs2,
             "u2": u2, "z": z, "a": a}
    return y, saved


def _layer_backward(p: Dict[str, torch.Tensor], s: Dict[str, torch.Tensor], gy: torch.Tensor,
                    heads: int, future: torch.Tensor):
    A = p["w_qkv"].shape[0] // 3
    d = A // heads
    scale = 1.0 / math.sqrt(d)
    g: Dict[str, torch.Tensor] = {}
    # y = x1 + a W2^T + b2
    g["w2"] = gy.T @ s["a"]
    g["b2"] = gy.sum(dim=0)
    gz = (gy @ p["w2"]) * _gelu_grad(s["z"])
    del s["a"], s["z"]
    # z = u2 W1^T + b1
    g["w1"] = gz.T @ s["u2"]
    g["b1"] = gz.sum(dim=0)
    gu2 = gz @ p["w1"]
    del gz, s["u2"]
    # u2 = LN2(x1); the residual carries gy into x1
    g["ln2_g"] = (gu2 * s["xh2"]).sum(dim=0)
    g["ln2_b"] = gu2.sum(dim=0)
    gx1 = gy + _ln_back(gu2, s["xh2"], s["rs2"], p["ln2_g"])
    del gu2
    # x1 = x + o W_o^T + b_o
    g["w_o"] = gx1.T @ s["o"]
    g["b_o"] = gx1.sum(dim=0)
    go = gx1 @ p["w_o"]
    # attention, head by head
    qkv = s["qkv"]
    q, k, v = qkv[:, :A], qkv[:, A:2 * A], qkv[:, 2 * A:]
    gqkv = torch.empty_like(qkv)
    for h in range(heads):
        c = slice(h * d, (h + 1) * d)
        P = _probs(q[:, c], k[:, c], scale, future)
        goh = go[:, c]
        gP = goh @ v[:, c].T
        gqkv[:, 2 * A + h * d:2 * A + (h + 1) * d] = P.T @ goh
        gS = P * (gP - (gP * P).sum(dim=1, keepdim=True))
        del gP, P
        gqkv[:, h * d:(h + 1) * d] = (gS @ k[:, c]) * scale
        gqkv[:, A + h * d:A + (h + 1) * d] = (gS.T @ q[:, c]) * scale
        del gS
    del go
    # [q, k, v] = u W_qkv^T + b_qkv
    g["w_qkv"] = gqkv.T @ s["u"]
    g["b_qkv"] = gqkv.sum(dim=0)
    gu = gqkv @ p["w_qkv"]
    del gqkv
    # u = LN1(x); the residual carries gx1 into x
    g["ln1_g"] = (gu * s["xh1"]).sum(dim=0)
    g["ln1_b"] = gu.sum(dim=0)
    gx = gx1 + _ln_back(gu, s["xh1"], s["rs1"], p["ln1_g"])
    return gx, g


def stage_forward_backward(params: Sequence[Dict[str, object]], x, dy, heads: int,
                           eps: float = 1e-5, log: Optional[Callable[[str], None]] = None
                           ) -> Tuple[torch.Tensor, torch.Tensor, List[Dict[str, torch.Tensor]]]:
    """y = stage(x), and the gradients of sum(y * dy): (y, dx, per-layer
    parameter gradients keyed like `params`), all float64 CPU tensors.

    params: per layer, the twelve tensors named in PARAM_NAMES (weights
    [out, in]); x, dy: [L, H]; heads: heads of each layer (of the shard, for an
    operation-partitioning shard)."""
    ps = [{k: _f64(p[k]) for k in PARAM_NAMES} for p in params]
    h = _f64(x)
    L = h.shape[0]
    future = torch.ones(L, L, dtype=torch.bool).triu_(1)
    saved = []
    for li, p in enumerate(ps):
        h, s = _layer_forward(p, h, heads, eps, future)
        saved.append(s)
        if log:
            log(f"full oracle: layer {li} forward done")
    y = h
    g = _f64(dy)
    grads: List[Optional[Dict[str, torch.Tensor]]] = [None] * len(ps)
    for li in range(len(ps) - 1, -1, -1):
        g, grads[li] = _layer_backward(ps[li], saved[li], g, heads, future)
        saved[li] = None
        if log:
            log(f"full oracle: layer {li} backward done")
    return y, g, grads
