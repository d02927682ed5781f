"""ctypes front end of the fp64 CPU oracle -- TEST INFRASTRUCTURE ONLY.

What is computed is defined in tp_oracle.c (stage forward/backward over token
slices and Algorithm 1 of the paper).  This module adds plain-Python
pieces that need no speed:

* ``eq5_latency`` -- the pipeline latency of a slicing, Eq. 5:
  sum_i t_i + (K - 1) * max_j t_j.
* ``exhaustive_optimal`` -- brute force over every composition of the
  sequence (2^(U-1) of them), the ground truth for the DP on small U.
* ``slice_flops`` / ``paper_tflops_per_gpu`` -- the arithmetic a slice of a
  pre-LN block must do, and the per-GPU TFLOP/s convention of the paper's
  result tables (Tables 2-4 in the appendix).
* ``batch_split`` / ``exhaustive_batch_split`` / ``joint_slicing`` -- the
  batch dimension of Sec. 3.4: groups of sequences, each token-sliced, sizes
  chosen by a one-dimensional knapsack over the per-size latencies.
* ``fit_ctx_model`` / ``cost_table_from_model`` -- the cost estimate of
  Sec. 3.3 (Eq. 9): t(i, j) = t(i, 0) + t_ctx(i, j) with the context overhead
  t_ctx = a0 + a1 i + a2 j + a3 i j fitted by least squares.
"""
from __future__ import annotations

import ctypes
import itertools
import math
import os
from typing import Dict, List, Sequence, Tuple

import numpy as np

from . import build as _build

PARAM_NAMES = ("ln1_g", "ln1_b", "w_qkv", "b_qkv", "w_o", "b_o",
               "ln2_g", "ln2_b", "w1", "b1", "w2", "b2")

_DP = ctypes.POINTER(ctypes.c_double)


class _Params(ctypes.Structure):
    _fields_ = [(n, _DP) for n in PARAM_NAMES]


_lib = None


def load_library():
    global _lib
    if _lib is None:
        path = _build.LIB
        if not os.path.exists(path):
            _build.build(force=False)
        lib = ctypes.CDLL(path)
        lib.or_stage_create.restype = ctypes.c_void_p
        lib.or_stage_create.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                        ctypes.c_double, ctypes.c_void_p, ctypes.c_void_p]
        lib.or_stage_create_ex.restype = ctypes.c_void_p
        lib.or_stage_create_ex.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                           ctypes.c_int, ctypes.c_int, ctypes.c_double,
                                           ctypes.c_void_p, ctypes.c_void_p]
        lib.or_stage_destroy.argtypes = [ctypes.c_void_p]
        lib.or_reset.argtypes = [ctypes.c_void_p]
        lib.or_forward.argtypes = [ctypes.c_void_p, ctypes.c_int, ctypes.c_int, _DP, _DP]
        lib.or_backward.argtypes = [ctypes.c_void_p, ctypes.c_int, ctypes.c_int, _DP, _DP]
        lib.or_get_cache.argtypes = [ctypes.c_void_p, ctypes.c_int, ctypes.c_int, _DP]
        lib.or_cached_len.argtypes = [ctypes.c_void_p]
        lib.or_bwd_frontier.argtypes = [ctypes.c_void_p]
        lib.or_gelu.restype = ctypes.c_double
        lib.or_gelu.argtypes = [ctypes.c_double]
        lib.or_gelu_grad.restype = ctypes.c_double
        lib.or_gelu_grad.argtypes = [ctypes.c_double]
        I64P = ctypes.POINTER(ctypes.c_int64)
        IP = ctypes.POINTER(ctypes.c_int)
        lib.or_dp_optimal_slicing.argtypes = [I64P, ctypes.c_int, ctypes.c_int, ctypes.c_int64,
                                              IP, IP, I64P, I64P, IP]
        _lib = lib
    return _lib


def _ptr(a: np.ndarray):
    assert a.dtype == np.float64 and a.flags["C_CONTIGUOUS"]
    return a.ctypes.data_as(_DP)


def gelu(z: float) -> float:
    return load_library().or_gelu(float(z))


def gelu_grad(z: float) -> float:
    return load_library().or_gelu_grad(float(z))


class OracleStage:
    """A stage of ``n_layers`` pre-LN blocks evaluated slice by slice in fp64.

    ``params`` is a list (one dict per layer) of arrays named by PARAM_NAMES,
    weights stored [out, in]; they are converted to float64 and kept alive.
    Gradients accumulate into ``self.grads`` (same structure, float64, zeroed at
    construction and by ``zero_grads``).  ``op_parts`` p > 1 makes the stage one
    device's shard of p-way operation partitioning: heads / p heads and 4H / p
    FFN units (weights of the shard's shapes), the output and FC2 projections'
    partial sums taken as the whole sum.
    """

    def __init__(self, params: List[Dict[str, np.ndarray]], hidden: int, heads: int,
                 max_seq: int, eps: float = 1e-5, op_parts: int = 1):
        self._lib = load_library()
        self.n_layers = len(params)
        self.hidden, self.heads, self.max_seq = hidden, heads, max_seq
        if heads % op_parts or (4 * hidden) % op_parts or hidden % heads:
            raise ValueError("invalid operation partitioning")
        self.op_parts = op_parts
        self.d = hidden // heads
        self.attn_width = heads // op_parts * self.d
        self.params = [{k: np.ascontiguousarray(np.asarray(p[k], dtype=np.float64))
                        for k in PARAM_NAMES} for p in params]
        self.grads = [{k: np.zeros_like(v) for k, v in p.items()} for p in self.params]
        self._p_structs = (_Params * self.n_layers)()
        self._g_structs = (_Params * self.n_layers)()
        for i in range(self.n_layers):
            for k in PARAM_NAMES:
                setattr(self._p_structs[i], k, _ptr(self.params[i][k]))
                setattr(self._g_structs[i], k, _ptr(self.grads[i][k]))
        self._h = self._lib.or_stage_create_ex(self.n_layers, hidden, heads // op_parts, self.d,
                                               4 * hidden // op_parts, max_seq, eps,
                                               ctypes.addressof(self._p_structs),
                                               ctypes.addressof(self._g_structs))
        if not self._h:
            raise ValueError("invalid oracle stage configuration")

    def __del__(self):
        h = getattr(self, "_h", None)
        if h:
            self._lib.or_stage_destroy(h)
            self._h = None

    def zero_grads(self):
        for g in self.grads:
            for v in g.values():
                v[...] = 0.0

    def reset(self):
        self._lib.or_reset(self._h)

    @property
    def cached_len(self) -> int:
        return self._lib.or_cached_len(self._h)

    @property
    def bwd_frontier(self) -> int:
        return self._lib.or_bwd_frontier(self._h)

    def forward(self, l: int, r: int, x: np.ndarray) -> np.ndarray:
        x = np.ascontiguousarray(x, dtype=np.float64).reshape(r - l, self.hidden)
        y = np.zeros_like(x)
        rc = self._lib.or_forward(self._h, l, r, _ptr(x), _ptr(y))
        if rc != 0:
            raise RuntimeError(f"oracle forward [{l},{r}) failed: {rc}")
        return y

    def backward(self, l: int, r: int, dy: np.ndarray) -> np.ndarray:
        dy = np.ascontiguousarray(dy, dtype=np.float64).reshape(r - l, self.hidden)
        dx = np.zeros_like(dy)
        rc = self._lib.or_backward(self._h, l, r, _ptr(dy), _ptr(dx))
        if rc != 0:
            raise RuntimeError(f"oracle backward [{l},{r}) failed: {rc}")
        return dx

    def try_forward(self, l: int, r: int, x: np.ndarray) -> int:
        x = np.ascontiguousarray(x, dtype=np.float64)
        y = np.zeros_like(x)
        return self._lib.or_forward(self._h, l, r, _ptr(x), _ptr(y))

    def cache(self, layer: int, which: str) -> np.ndarray:
        idx = {"k": 0, "v": 1, "dk": 2, "dv": 3}[which]
        out = np.zeros((self.max_seq, self.attn_width))
        n = self._lib.or_get_cache(self._h, layer, idx, _ptr(out))
        return out[:n].copy()

    def run_sequence(self, x: np.ndarray, dy: np.ndarray, fwd_lens: Sequence[int],
                     bwd_lens: Sequence[int] | None = None) -> Tuple[np.ndarray, np.ndarray]:
        """Reset, forward every slice in order, backward every slice in reverse."""
        L = x.shape[0]
        assert sum(fwd_lens) == L
        bwd_lens = list(fwd_lens) if bwd_lens is None else list(bwd_lens)
        assert sum(bwd_lens) == L
        self.reset()
        y = np.zeros((L, self.hidden))
        pos = 0
        for n in fwd_lens:
            y[pos:pos + n] = self.forward(pos, pos + n, x[pos:pos + n])
            pos += n
        dx = np.zeros((L, self.hidden))
        bounds = np.cumsum([0] + bwd_lens)
        for i in range(len(bwd_lens) - 1, -1, -1):
            l, r = int(bounds[i]), int(bounds[i + 1])
            dx[l:r] = self.backward(l, r, dy[l:r])
        return y, dx


# --------------------------------------------------------------------- slicing

def eq5_latency(costs: Sequence[int], K: int) -> int:
    """Eq. 5 for one slicing: total time on a cell plus (K-1) times the slowest slice."""
    return int(sum(costs)) + (K - 1) * int(max(costs))


def slicing_costs(cost: np.ndarray, units: Sequence[int]) -> List[int]:
    """Per-slice costs t(l_i, sum_{j<i} l_j) (Eq. 4) from a [U][U] table in units."""
    out, ctx = [], 0
    for k in units:
        out.append(int(cost[k - 1, ctx]))
        ctx += k
    return out


def exhaustive_optimal(cost: np.ndarray, K: int) -> Tuple[int, List[Tuple[int, ...]]]:
    """Minimum of Eq. 5 over all 2^(U-1) compositions of U units, and every argmin."""
    U = cost.shape[0]
    best, arg = None, []
    for cuts in itertools.product((0, 1), repeat=U - 1):
        units, run = [], 1
        for c in cuts:
            if c:
                units.append(run)
                run = 1
            else:
                run += 1
        units.append(run)
        T = eq5_latency(slicing_costs(cost, units), K)
        if best is None or T < best:
            best, arg = T, [tuple(units)]
        elif T == best:
            arg.append(tuple(units))
    return best, arg


def dp_optimal_slicing(cost: np.ndarray, K: int, eps: int = 0):
    """Algorithm 1 with the t_max enumeration of Eq. 6-7 (see tp_oracle.c).

    ``cost`` is an int64 [U][U] table: cost[k-1, j] = t(k units, j units of
    context).  Returns (units, T, t_max, thresholds_evaluated)."""
    lib = load_library()
    cost = np.ascontiguousarray(cost, dtype=np.int64)
    U = cost.shape[0]
    assert cost.shape == (U, U)
    out = (ctypes.c_int * U)()
    M = ctypes.c_int()
    T = ctypes.c_int64()
    tmax = ctypes.c_int64()
    ev = ctypes.c_int()
    rc = lib.or_dp_optimal_slicing(cost.ctypes.data_as(ctypes.POINTER(ctypes.c_int64)), U, K,
                                   eps, out, ctypes.byref(M), ctypes.byref(T),
                                   ctypes.byref(tmax), ctypes.byref(ev))
    if rc != 0:
        raise ValueError(f"oracle DP rejected its arguments ({rc})")
    return [out[i] for i in range(M.value)], T.value, tmax.value, ev.value


# ------------------------------------------------------ batch split (Sec. 3.4)

def batch_split(T_b: Sequence[int]) -> Tuple[List[int], int]:
    """Sec. 3.4: cut a batch of B = len(T_b) sequences into groups b_1..b_D
    (sum B) minimising T_{b_1} + ... + T_{b_D}, T_b = T_b[b-1] the optimal
    latency of a group of b sequences (negative: unusable).  The knapsack
    recurrence best[x] = min_b best[x - b] + T_b, b ascending, replaced only on
    a strictly smaller total.  Returns (sizes largest first, total)."""
    B = len(T_b)
    INF = None
    best = [0] + [INF] * B
    last = [0] * (B + 1)
    for x in range(1, B + 1):
        for b in range(1, x + 1):
            t = int(T_b[b - 1])
            if t < 0 or best[x - b] is INF:
                continue
            v = best[x - b] + t
            if best[x] is INF or v < best[x]:
                best[x], last[x] = v, b
    if best[B] is INF:
        raise ValueError("no combination of usable group sizes sums to B")
    sizes, x = [], B
    while x > 0:
        sizes.append(last[x])
        x -= last[x]
    return sorted(sizes, reverse=True), best[B]


def integer_partitions(B: int, largest: int = None):
    """Every multiset of positive integers summing to B, as non-increasing tuples."""
    largest = B if largest is None else largest
    if B == 0:
        yield ()
        return
    for first in range(min(B, largest), 0, -1):
        for rest in integer_partitions(B - first, first):
            yield (first,) + rest


def exhaustive_batch_split(T_b: Sequence[int]) -> Tuple[int, List[Tuple[int, ...]]]:
    """Brute force over all partitions of B: the minimal sum and every argmin."""
    best, arg = None, []
    for part in integer_partitions(len(T_b)):
        if any(T_b[b - 1] < 0 for b in part):
            continue
        v = sum(int(T_b[b - 1]) for b in part)
        if best is None or v < best:
            best, arg = v, [part]
        elif v == best:
            arg.append(part)
    return best, arg


def joint_slicing(costs: np.ndarray, K: int, eps: int = 0):
    """Sec. 3.4 joint plan on [B][U][U] tables (plane b-1: a group of b
    sequences): the token DP per group size, then the batch split.  Returns
    (groups [(b, units)], T_b list, total)."""
    T_b, units = [], []
    for b in range(costs.shape[0]):
        u, T, _, _ = dp_optimal_slicing(costs[b], K, eps)
        T_b.append(T)
        units.append(u)
    sizes, total = batch_split(T_b)
    return [(b, units[b - 1]) for b in sizes], T_b, total


# ------------------------------------------------------------------ flop counts

def slice_flops(n: int, c: int, hidden: int) -> int:
    """Algorithmic flops of forward+backward of one pre-LN block over a slice of
    n tokens after c cached tokens: the four projections cost 24 n H^2 forward
    (QKV 6, output 2, two MLP GEMMs 8 each), the causal attention 4 H per
    (query, key) pair with key <= query (QK^T and PV), and backward twice the
    forward.  Elementwise work (LN, GELU, softmax) is not counted."""
    pairs = n * c + n * (n + 1) // 2
    return 3 * (24 * n * hidden * hidden + 4 * hidden * pairs)


def sequence_flops(lens: Sequence[int], hidden: int, n_layers: int) -> int:
    tot, c = 0, 0
    for n in lens:
        tot += slice_flops(n, c, hidden)
        c += n
    return tot * n_layers


def paper_tflops_per_gpu(hidden: int, n_layers: int, seq_len: int, sequences: int,
                         gpus: int, latency_s: float) -> float:
    """Per-GPU TFLOP/s as the paper's result tables count it: (72 H^2 + 6 H L)
    flops per token per layer (three times a causal forward), for the sequences
    of one data-parallel replica, divided by all GPUs and the iteration time."""
    per_token_layer = 72 * hidden * hidden + 6 * hidden * seq_len
    return per_token_layer * n_layers * seq_len * sequences / (gpus * latency_s) / 1e12


# ------------------------------------------------------- cost model (Eq. 9)

def fit_ctx_model(t0: Sequence[int], unit: int, samples: Sequence[Tuple[int, int, int]]):
    """Least-squares fit of the context overhead of Eq. 9.

    ``t0[k-1]`` is the measured cost of a slice of k*unit tokens with no
    context; each sample (i, j, t) is a measured cost t of a slice of i tokens
    (a multiple of ``unit``) after j > 0 tokens of context, whose overhead is
    t - t(i, 0).  Returns (a0, a1, a2, a3) minimising the sum of squared
    differences between that overhead and a0 + a1 i + a2 j + a3 i j, i and j
    in tokens, the definition of least squares solved by numpy's lstsq on the
    unscaled design in float64."""
    X = np.array([[1.0, float(i), float(j), float(i) * float(j)] for i, j, _ in samples])
    y = np.array([float(t) - float(t0[i // unit - 1]) for i, j, t in samples])
    coef, _, rank, _ = np.linalg.lstsq(X, y, rcond=None)
    if rank < 4:
        raise ValueError("samples do not determine the four coefficients")
    return tuple(float(c) for c in coef)


def _round_half_away(x: float) -> int:
    return int(math.floor(x + 0.5)) if x >= 0 else -int(math.floor(-x + 0.5))


def cost_table_from_model(t0: Sequence[int], unit: int, coef) -> np.ndarray:
    """[U][U] int64 cost table from Eq. 9: entry [k-1, j] is t(k units, j units
    of context) = t(k units, 0) measured, plus, for j > 0, the fitted overhead
    a0 + a1 i + a2 c + a3 i c at i = k*unit, c = j*unit tokens, rounded to the
    nearest nanosecond (halves away from zero) and the sum clamped at 0.
    Entries past the sequence (k + j > U) are -1."""
    U = len(t0)
    a0, a1, a2, a3 = coef
    cost = np.full((U, U), -1, dtype=np.int64)
    for k in range(1, U + 1):
        for j in range(0, U - k + 1):
            if j == 0:
                cost[k - 1, j] = int(t0[k - 1])
            else:
                i, c = k * unit, j * unit
                pred = a0 + a1 * i + a2 * c + a3 * i * c
                cost[k - 1, j] = max(0, int(t0[k - 1]) + _round_half_away(pred))
    return cost
