"""ctypes binding of libterapipe.so (include/terapipe.h), argument marshalling only.

PyTorch provides device memory and the stream; every step of the stage runs in
the library's HIP kernels.  If the library is missing this module raises on
import: there is no fallback path.
"""
from __future__ import annotations

import ctypes
import os
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np
import torch

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "lib", "libterapipe.so")

TP_OK, TP_ERR_INVALID, TP_ERR_ORDER, TP_ERR_UNSUPPORTED, TP_ERR_WORKSPACE, TP_ERR_HIP = (
    0, -1, -2, -3, -4, -5)
DTYPE_BF16, DTYPE_FP32 = 0, 1
SEQ_OVERWRITE_GRADS = 1
SEQ_REUSE_WQKV_COPY = 2
WGRAD_PER_SLICE, WGRAD_DEFERRED = 0, 1

PARAM_FIELDS = ("ln1_g", "ln1_b", "w_qkv", "b_qkv", "w_o", "b_o",
                "ln2_g", "ln2_b", "w_fc1", "b_fc1", "w_fc2", "b_fc2")
# names used by the seeded input module for the same tensors
SYNTH_NAMES = ("ln1_g", "ln1_b", "w_qkv", "b_qkv", "w_o", "b_o",
               "ln2_g", "ln2_b", "w1", "b1", "w2", "b2")

EXPORTED = ("tp_stage_workspace_bytes", "tp_stage_init", "tp_stage_destroy",
            "tp_kv_prefix_reset", "tp_kv_prefix_reset_ex", "tp_slice_forward", "tp_slice_forward_static",
            "tp_slice_backward",
            "tp_profile_slice_cost", "tp_dp_optimal_slicing", "tp_dp_batch_split",
            "tp_dp_joint_slicing", "tp_fit_ctx_model",
            "tp_cost_table_from_model", "tp_profile_cost_model", "tp_status_string",
            "tp_stage_enable_kernel_timing", "tp_stage_kernel_stats", "tp_measure_mfma_peak")


class StageConfig(ctypes.Structure):
    _fields_ = [("n_layers", ctypes.c_int), ("hidden", ctypes.c_int), ("heads", ctypes.c_int),
                ("max_seq", ctypes.c_int), ("dtype", ctypes.c_int), ("wgrad_mode", ctypes.c_int),
                ("ln_eps", ctypes.c_float), ("batch", ctypes.c_int), ("op_parts", ctypes.c_int)]


class LayerPtrs(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in PARAM_FIELDS]


class KernelStat(ctypes.Structure):
    _fields_ = [("name", ctypes.c_char * 48), ("launches", ctypes.c_int64),
                ("total_ms", ctypes.c_double), ("flops", ctypes.c_double),
                ("bytes", ctypes.c_double)]


class TerapipeError(RuntimeError):
    def __init__(self, status: int, what: str):
        self.status = status
        super().__init__(f"{what}: {status_string(status)} ({status})")


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run __graft_entry__.build() "
                          "or python paper_2102_07988_amd/build.py")
    lib = ctypes.CDLL(LIB_PATH)
    vp, ip, i64p = ctypes.c_void_p, ctypes.POINTER(ctypes.c_int), ctypes.POINTER(ctypes.c_int64)
    lib.tp_stage_workspace_bytes.restype = ctypes.c_size_t
    lib.tp_stage_workspace_bytes.argtypes = [ctypes.POINTER(StageConfig)]
    lib.tp_stage_init.restype = ctypes.c_int
    lib.tp_stage_init.argtypes = [ctypes.POINTER(StageConfig), ctypes.POINTER(LayerPtrs),
                                  ctypes.POINTER(LayerPtrs), vp, ctypes.c_size_t, vp,
                                  ctypes.POINTER(vp)]
    lib.tp_stage_destroy.restype = None
    lib.tp_stage_destroy.argtypes = [vp]
    lib.tp_kv_prefix_reset.restype = ctypes.c_int
    lib.tp_kv_prefix_reset.argtypes = [vp]
    lib.tp_kv_prefix_reset_ex.restype = ctypes.c_int
    lib.tp_kv_prefix_reset_ex.argtypes = [vp, ctypes.c_uint]
    for f in (lib.tp_slice_forward, lib.tp_slice_forward_static, lib.tp_slice_backward):
        f.restype = ctypes.c_int
        f.argtypes = [vp, ctypes.c_int, ctypes.c_int, vp, vp]
    lib.tp_profile_slice_cost.restype = ctypes.c_int
    lib.tp_profile_slice_cost.argtypes = [vp, ip, ctypes.c_int, ip, ctypes.c_int, ctypes.c_int,
                                          ctypes.c_int, i64p, i64p]
    lib.tp_dp_optimal_slicing.restype = ctypes.c_int
    lib.tp_dp_optimal_slicing.argtypes = [i64p, ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                          ctypes.c_int64, ip, ip, i64p]
    lib.tp_dp_batch_split.restype = ctypes.c_int
    lib.tp_dp_batch_split.argtypes = [i64p, ctypes.c_int, ip, ip, i64p]
    lib.tp_dp_joint_slicing.restype = ctypes.c_int
    lib.tp_dp_joint_slicing.argtypes = [i64p, ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                        ctypes.c_int, ctypes.c_int64, ip, ip, ip, ip, i64p, i64p]
    dp = ctypes.POINTER(ctypes.c_double)
    lib.tp_fit_ctx_model.restype = ctypes.c_int
    lib.tp_fit_ctx_model.argtypes = [i64p, ctypes.c_int, ctypes.c_int, ip, ip, i64p, ctypes.c_int,
                                     dp]
    lib.tp_cost_table_from_model.restype = ctypes.c_int
    lib.tp_cost_table_from_model.argtypes = [i64p, ctypes.c_int, ctypes.c_int, dp, i64p]
    lib.tp_profile_cost_model.restype = ctypes.c_int
    lib.tp_profile_cost_model.argtypes = [vp, ctypes.c_int, ctypes.c_int, ip, ctypes.c_int, ip,
                                          ctypes.c_int, ctypes.c_int, ctypes.c_int, i64p, dp]
    lib.tp_status_string.restype = ctypes.c_char_p
    lib.tp_status_string.argtypes = [ctypes.c_int]
    lib.tp_stage_enable_kernel_timing.restype = ctypes.c_int
    lib.tp_stage_enable_kernel_timing.argtypes = [vp, ctypes.c_int]
    lib.tp_measure_mfma_peak.restype = ctypes.c_int
    lib.tp_measure_mfma_peak.argtypes = [vp, ctypes.c_int, vp, ctypes.POINTER(ctypes.c_double)]
    lib.tp_stage_kernel_stats.restype = ctypes.c_int
    lib.tp_stage_kernel_stats.argtypes = [vp, ctypes.POINTER(KernelStat), ctypes.c_int]
    return lib


lib = _load()


def status_string(status: int) -> str:
    return lib.tp_status_string(status).decode()


def _check(status: int, what: str):
    if status != TP_OK:
        raise TerapipeError(status, what)


def make_config(n_layers: int, hidden: int, heads: int, max_seq: int, dtype: str = "bf16",
                wgrad: str = "per_slice", ln_eps: float = 1e-5, batch: int = 1,
                op_parts: int = 1) -> StageConfig:
    return StageConfig(n_layers, hidden, heads, max_seq,
                       DTYPE_BF16 if dtype == "bf16" else DTYPE_FP32,
                       WGRAD_PER_SLICE if wgrad == "per_slice" else WGRAD_DEFERRED, ln_eps, batch,
                       op_parts)


def workspace_bytes(cfg: StageConfig) -> int:
    return lib.tp_stage_workspace_bytes(ctypes.byref(cfg))


def torch_dtype(dtype: str):
    return torch.bfloat16 if dtype == "bf16" else torch.float32


def _dp(t: Optional[torch.Tensor]) -> Optional[int]:
    return None if t is None else t.data_ptr()


class Stage:
    """One pipeline stage of ``n_layers`` pre-LN blocks on the current device.

    ``params``: list (per layer) of dicts keyed by the seeded-input names
    (ln1_g, ..., w1, b1, w2, b2), device tensors of the stage dtype, weights
    [out, in].  Gradients are fp32 device tensors in ``self.grads`` (same keys),
    zero at construction.  The stage enqueues on the stream that is current at
    construction.  ``batch`` sequences move through the stage together (a batch
    slice): slice tensors are then [n, batch, hidden] (token-major).  ``op_parts``
    p > 1: the stage is one device's shard of p-way operation partitioning
    (parameters of the shard's shapes, see ``synth.param_shapes``).
    """

    def __init__(self, params: List[Dict[str, torch.Tensor]], hidden: int, heads: int,
                 max_seq: int, dtype: str = "bf16", wgrad: str = "per_slice",
                 ln_eps: float = 1e-5, device=None, batch: int = 1, op_parts: int = 1):
        # the library handle, kept so the stage can be destroyed during interpreter
        # shutdown, after the module's globals have been cleared
        self._lib = lib
        self.n_layers = len(params)
        self.hidden, self.heads, self.max_seq, self.dtype = hidden, heads, max_seq, dtype
        self.batch = batch
        self.tdtype = torch_dtype(dtype)
        self.device = torch.device(device) if device is not None else params[0]["w_qkv"].device
        self.op_parts = op_parts
        self.cfg = make_config(self.n_layers, hidden, heads, max_seq, dtype, wgrad, ln_eps, batch,
                               op_parts)
        for p in params:
            for k in SYNTH_NAMES:
                t = p[k]
                if t.dtype != self.tdtype or not t.is_contiguous() or t.device != self.device:
                    raise ValueError(f"parameter {k}: need a contiguous {self.tdtype} tensor on "
                                     f"{self.device}")
        self.params = params
        self.grads = [{k: torch.zeros(p[k].shape, dtype=torch.float32, device=self.device)
                       for k in SYNTH_NAMES} for p in params]
        nbytes = workspace_bytes(self.cfg)
        if nbytes == 0:
            raise TerapipeError(TP_ERR_INVALID, "stage configuration")
        self.workspace = torch.empty(nbytes, dtype=torch.uint8, device=self.device)
        self.stream = torch.cuda.current_stream(self.device)
        P = (LayerPtrs * self.n_layers)()
        G = (LayerPtrs * self.n_layers)()
        for i in range(self.n_layers):
            for f, k in zip(PARAM_FIELDS, SYNTH_NAMES):
                setattr(P[i], f, params[i][k].data_ptr())
                setattr(G[i], f, self.grads[i][k].data_ptr())
        h = ctypes.c_void_p()
        _check(lib.tp_stage_init(ctypes.byref(self.cfg), P, G, self.workspace.data_ptr(),
                                 nbytes, self.stream.cuda_stream, ctypes.byref(h)), "tp_stage_init")
        self._h = h

    def __del__(self):
        h = getattr(self, "_h", None)
        if h is not None and h.value:
            self._lib.tp_stage_destroy(h)
            self._h = None

    @property
    def handle(self):
        return self._h

    def zero_grads(self):
        for g in self.grads:
            for v in g.values():
                v.zero_()

    def reset(self, overwrite_grads: bool = False, reuse_wqkv_copy: bool = False):
        """Start a sequence.  overwrite_grads: its gradients replace the buffers'
        contents instead of adding to them (TP_SEQ_OVERWRITE_GRADS);
        reuse_wqkv_copy: W_qkv is unchanged, keep its fp16 copy
        (TP_SEQ_REUSE_WQKV_COPY)."""
        flags = ((SEQ_OVERWRITE_GRADS if overwrite_grads else 0) |
                 (SEQ_REUSE_WQKV_COPY if reuse_wqkv_copy else 0))
        if flags:
            _check(lib.tp_kv_prefix_reset_ex(self._h, flags), "tp_kv_prefix_reset_ex")
        else:
            _check(lib.tp_kv_prefix_reset(self._h), "tp_kv_prefix_reset")

    def _io(self, t: torch.Tensor, n: int) -> torch.Tensor:
        shape = (n, self.hidden) if self.batch == 1 else (n, self.batch, self.hidden)
        if t.dtype != self.tdtype or t.device != self.device or tuple(t.shape) != shape:
            raise ValueError(f"expected a {list(shape)} {self.tdtype} tensor on {self.device}")
        return t.contiguous()

    def forward(self, l: int, r: int, x: torch.Tensor, out: Optional[torch.Tensor] = None):
        x = self._io(x, r - l)
        y = torch.empty_like(x) if out is None else out
        _check(lib.tp_slice_forward(self._h, l, r, x.data_ptr(), y.data_ptr()),
               f"tp_slice_forward [{l},{r})")
        return y

    def forward_static(self, l: int, r: int, x: torch.Tensor, out: Optional[torch.Tensor] = None):
        """tp_slice_forward_static: the slice forward with its partial sums in the
        library's static scratch (no allocation by the library)."""
        x = self._io(x, r - l)
        y = torch.empty_like(x) if out is None else out
        _check(lib.tp_slice_forward_static(self._h, l, r, x.data_ptr(), y.data_ptr()),
               f"tp_slice_forward_static [{l},{r})")
        return y

    def backward(self, l: int, r: int, dy: torch.Tensor, out: Optional[torch.Tensor] = None):
        dy = self._io(dy, r - l)
        dx = torch.empty_like(dy) if out is None else out
        _check(lib.tp_slice_backward(self._h, l, r, dy.data_ptr(), dx.data_ptr()),
               f"tp_slice_backward [{l},{r})")
        return dx

    def run_sequence(self, x: torch.Tensor, dy: torch.Tensor, fwd_lens: Sequence[int],
                     bwd_lens: Optional[Sequence[int]] = None,
                     overwrite_grads: bool = False) -> Tuple[torch.Tensor, torch.Tensor]:
        """Reset, forward each slice in order, backward each slice in reverse."""
        L = x.shape[0]
        bwd_lens = list(fwd_lens) if bwd_lens is None else list(bwd_lens)
        assert sum(fwd_lens) == L and sum(bwd_lens) == L
        self.reset(overwrite_grads)
        y = torch.empty_like(x)
        pos = 0
        for n in fwd_lens:
            self.forward(pos, pos + n, x[pos:pos + n], out=y[pos:pos + n])
            pos += n
        dx = torch.empty_like(dy)
        bounds = np.cumsum([0] + bwd_lens)
        for i in range(len(bwd_lens) - 1, -1, -1):
            l, r = int(bounds[i]), int(bounds[i + 1])
            self.backward(l, r, dy[l:r], out=dx[l:r])
        return y, dx

    def profile(self, lens: Sequence[int], ctxs: Sequence[int], warmup: int = 3,
                reps: int = 10) -> Tuple[np.ndarray, np.ndarray]:
        """Median forward / backward ns per (len, ctx), shape [len(lens), len(ctxs)]."""
        nl, nc = len(lens), len(ctxs)
        L = (ctypes.c_int * nl)(*lens)
        C = (ctypes.c_int * nc)(*ctxs)
        tf = np.zeros((nl, nc), dtype=np.int64)
        tb = np.zeros((nl, nc), dtype=np.int64)
        i64p = ctypes.POINTER(ctypes.c_int64)
        _check(lib.tp_profile_slice_cost(self._h, L, nl, C, nc, warmup, reps,
                                         tf.ctypes.data_as(i64p), tb.ctypes.data_as(i64p)),
               "tp_profile_slice_cost")
        return tf, tb

    def profile_model(self, L: int, unit: int, sub_lens: Sequence[int], sub_ctxs: Sequence[int],
                      warmup: int = 3, reps: int = 10) -> Tuple[np.ndarray, Tuple[float, ...]]:
        """Model-mode cost table (Eq. 9): every t(i, 0) measured, the context
        overhead fitted on sub_lens x sub_ctxs.  Returns (int64 [U][U] table of
        t_fwd + t_bwd in ns, (a0, a1, a2, a3))."""
        if L % unit:
            raise ValueError("L must be a multiple of unit")
        U = L // unit
        nl, nc = len(sub_lens), len(sub_ctxs)
        Ls = (ctypes.c_int * nl)(*sub_lens)
        Cs = (ctypes.c_int * nc)(*sub_ctxs)
        cost = np.zeros((U, U), dtype=np.int64)
        coef = (ctypes.c_double * 4)()
        _check(lib.tp_profile_cost_model(self._h, U, unit, Ls, nl, Cs, nc, warmup, reps,
                                         cost.ctypes.data_as(ctypes.POINTER(ctypes.c_int64)),
                                         coef), "tp_profile_cost_model")
        return cost, tuple(coef)

    def enable_kernel_timing(self, on: bool = True):
        _check(lib.tp_stage_enable_kernel_timing(self._h, 1 if on else 0), "kernel timing")

    def kernel_stats(self) -> Dict[str, Dict[str, float]]:
        buf = (KernelStat * 16)()
        n = lib.tp_stage_kernel_stats(self._h, buf, 16)
        if n < 0:
            raise TerapipeError(TP_ERR_HIP, "tp_stage_kernel_stats")
        return {buf[i].name.decode(): {"launches": buf[i].launches, "total_ms": buf[i].total_ms,
                                       "flops": buf[i].flops, "bytes": buf[i].bytes}
                for i in range(n)}


def dp_optimal_slicing(cost: np.ndarray, unit: int, K: int, eps_ns: int = 0):
    """C-ABI DP: cost int64 [U][U] (cost[k-1, j] = t(k units, j units of context)).
    Returns (slice lengths in tokens, Eq. 5 latency)."""
    cost = np.ascontiguousarray(cost, dtype=np.int64)
    U = cost.shape[0]
    if cost.shape != (U, U):
        raise ValueError("cost must be square [U][U]")
    out = (ctypes.c_int * U)()
    M = ctypes.c_int()
    T = ctypes.c_int64()
    _check(lib.tp_dp_optimal_slicing(cost.ctypes.data_as(ctypes.POINTER(ctypes.c_int64)), U, unit,
                                     K, eps_ns, out, ctypes.byref(M), ctypes.byref(T)),
           "tp_dp_optimal_slicing")
    return [out[i] for i in range(M.value)], T.value


def batch_split(T_b: Sequence[int]) -> Tuple[List[int], int]:
    """C-ABI batch split (Sec. 3.4): T_b[b-1] = latency of a group of b
    sequences (negative: unusable).  Returns (group sizes largest first, total)."""
    B = len(T_b)
    t = np.ascontiguousarray(T_b, dtype=np.int64)
    out = (ctypes.c_int * B)()
    D = ctypes.c_int()
    tot = ctypes.c_int64()
    _check(lib.tp_dp_batch_split(t.ctypes.data_as(ctypes.POINTER(ctypes.c_int64)), B, out,
                                 ctypes.byref(D), ctypes.byref(tot)), "tp_dp_batch_split")
    return [out[i] for i in range(D.value)], tot.value


def joint_slicing(costs: np.ndarray, unit: int, K: int, eps_ns: int = 0):
    """C-ABI joint batch x token plan (Sec. 3.4).  costs: int64 [B][U][U], plane
    b-1 the cost table of a batch slice of b sequences.  Returns
    (groups [(b, token lengths)], T_b list, total)."""
    costs = np.ascontiguousarray(costs, dtype=np.int64)
    B, U = costs.shape[0], costs.shape[1]
    if costs.shape != (B, U, U):
        raise ValueError("costs must be [B][U][U]")
    sizes = (ctypes.c_int * B)()
    M = (ctypes.c_int * B)()
    lens = (ctypes.c_int * (B * U))()
    Tb = np.zeros(B, dtype=np.int64)
    D = ctypes.c_int()
    tot = ctypes.c_int64()
    i64p = ctypes.POINTER(ctypes.c_int64)
    _check(lib.tp_dp_joint_slicing(costs.ctypes.data_as(i64p), B, U, unit, K, eps_ns, sizes,
                                   ctypes.byref(D), lens, M, Tb.ctypes.data_as(i64p),
                                   ctypes.byref(tot)), "tp_dp_joint_slicing")
    groups = [(sizes[g], [lens[g * U + i] for i in range(M[g])]) for g in range(D.value)]
    return groups, [int(v) for v in Tb], tot.value


def fit_ctx_model(t0: Sequence[int], unit: int, samples: Sequence[Tuple[int, int, int]]):
    """C-ABI Eq. 9 fit: t0[k-1] = t(k*unit, 0); samples (len, ctx, t) with ctx >= 1.
    Returns (a0, a1, a2, a3) of t_ctx = a0 + a1 len + a2 ctx + a3 len ctx (ns, tokens)."""
    U, n = len(t0), len(samples)
    t0a = np.ascontiguousarray(t0, dtype=np.int64)
    i64p = ctypes.POINTER(ctypes.c_int64)
    sl = (ctypes.c_int * n)(*[s[0] for s in samples])
    sc = (ctypes.c_int * n)(*[s[1] for s in samples])
    st = np.ascontiguousarray([s[2] for s in samples], dtype=np.int64)
    coef = (ctypes.c_double * 4)()
    _check(lib.tp_fit_ctx_model(t0a.ctypes.data_as(i64p), U, unit, sl, sc, st.ctypes.data_as(i64p),
                                n, coef), "tp_fit_ctx_model")
    return tuple(coef)


def cost_table_from_model(t0: Sequence[int], unit: int, coef) -> np.ndarray:
    """C-ABI Eq. 9 cost table, int64 [U][U] (layout of dp_optimal_slicing's input)."""
    U = len(t0)
    t0a = np.ascontiguousarray(t0, dtype=np.int64)
    i64p = ctypes.POINTER(ctypes.c_int64)
    c = (ctypes.c_double * 4)(*coef)
    cost = np.zeros((U, U), dtype=np.int64)
    _check(lib.tp_cost_table_from_model(t0a.ctypes.data_as(i64p), U, unit, c,
                                        cost.ctypes.data_as(i64p)), "tp_cost_table_from_model")
    return cost


def measure_mfma_peak(iters: int = 20000) -> float:
    """Dense bf16 TFLOP/s of a register-only MFMA chain on every SIMD of cuda:0."""
    import torch
    sink = torch.empty(1 << 16, dtype=torch.float32, device="cuda")
    out = ctypes.c_double()
    _check(lib.tp_measure_mfma_peak(ctypes.c_void_p(torch.cuda.current_stream().cuda_stream), iters,
                                    ctypes.c_void_p(sink.data_ptr()), ctypes.byref(out)),
           "tp_measure_mfma_peak")
    return out.value


def slice_flops(n: int, c: int, hidden: int) -> int:
    """Algorithmic flops of one layer's forward+backward over n tokens after c
    cached tokens: 24 n H^2 for the projections and 4 H per causal
    (query, key <= query) pair forward, backward twice forward."""
    pairs = n * c + n * (n + 1) // 2
    return 3 * (24 * n * hidden * hidden + 4 * hidden * pairs)
