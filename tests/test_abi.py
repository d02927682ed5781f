"""The C-ABI library on the host: exports, host-side validation, and the DP.

No GPU is touched here: stage creation only records pointers, and every
rejected call returns before enqueuing device work.
"""
import ctypes
import os
import re

import numpy as np
import pytest

from paper_2102_07988_amd import synth
from paper_2102_07988_amd import terapipe as tp
from oracle import dp_optimal_slicing as oracle_dp, exhaustive_optimal

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_functions():
    src = open(os.path.join(ROOT, "include", "terapipe.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(tp_[a-z_]+)\s*\(", src)))


def test_every_declared_function_is_exported():
    names = declared_functions()
    assert len(names) >= 11
    for n in names:
        assert hasattr(tp.lib, n), n
    assert set(names) == set(tp.EXPORTED)


def test_status_strings():
    for s in (0, -1, -2, -3, -4, -5):
        assert tp.status_string(s) and tp.status_string(s) != "unknown status"


def _fake_layers(n):
    P = (tp.LayerPtrs * n)()
    for i in range(n):
        for j, f in enumerate(tp.PARAM_FIELDS):
            setattr(P[i], f, 0x10000000 + 0x1000 * (16 * i + j))
    return P


def _init(cfg, ws=None, nbytes=None, params=None, grads=None):
    n = cfg.n_layers
    P = _fake_layers(n) if params is None else params
    G = _fake_layers(n) if grads is None else grads
    need = tp.workspace_bytes(cfg)
    h = ctypes.c_void_p()
    rc = tp.lib.tp_stage_init(ctypes.byref(cfg), P, G, 0x7f0000000000 if ws is None else ws,
                              need if nbytes is None else nbytes, None, ctypes.byref(h))
    return rc, h


def test_workspace_size_and_init_validation():
    cfg = tp.make_config(2, 64, 4, 32, "fp32")
    need = tp.workspace_bytes(cfg)
    assert need > 0 and need % 256 == 0
    # bigger dtype, more layers, longer sequence -> more workspace
    assert tp.workspace_bytes(tp.make_config(2, 64, 4, 32, "bf16")) < need
    assert tp.workspace_bytes(tp.make_config(3, 64, 4, 32, "fp32")) > need
    assert tp.workspace_bytes(tp.make_config(2, 64, 4, 64, "fp32")) > need
    rc, h = _init(cfg)
    assert rc == tp.TP_OK and h.value
    tp.lib.tp_stage_destroy(h)
    assert _init(cfg, ws=0x7f0000000001)[0] == tp.TP_ERR_WORKSPACE
    assert _init(cfg, nbytes=need - 1)[0] == tp.TP_ERR_WORKSPACE
    assert _init(cfg, ws=0)[0] == tp.TP_ERR_INVALID
    bad = tp.make_config(2, 64, 5, 32)  # hidden % heads != 0
    assert tp.workspace_bytes(bad) == 0
    assert _init(bad)[0] == tp.TP_ERR_INVALID
    assert _init(tp.make_config(1, 96, 2, 32))[0] == tp.TP_ERR_UNSUPPORTED  # d = 48
    P = _fake_layers(2)
    P[1].w_o = None
    assert _init(cfg, params=P)[0] == tp.TP_ERR_INVALID
    assert _init(tp.make_config(0, 64, 4, 32))[0] == tp.TP_ERR_INVALID


def test_batch_config():
    """Batch slices (Sec. 3.4): 0 means 1; the per-token arenas scale with the
    batch (rows = max_seq * batch); sizes outside 0..64 are invalid."""
    one = tp.workspace_bytes(tp.make_config(2, 64, 4, 32, "fp32", batch=1))
    assert tp.workspace_bytes(tp.make_config(2, 64, 4, 32, "fp32", batch=0)) == one
    two = tp.workspace_bytes(tp.make_config(2, 64, 4, 32, "fp32", batch=2))
    # the same as one sequence twice as long
    assert two == tp.workspace_bytes(tp.make_config(2, 64, 4, 64, "fp32", batch=1))
    assert tp.workspace_bytes(tp.make_config(2, 64, 4, 32, "fp32", batch=65)) == 0
    assert tp.workspace_bytes(tp.make_config(2, 64, 4, 32, "fp32", batch=-1)) == 0
    rc, h = _init(tp.make_config(2, 64, 4, 32, "fp32", batch=4))
    assert rc == tp.TP_OK
    tp.lib.tp_stage_destroy(h)


def test_op_parts_config():
    """Operation-partitioning shards: 0 means 1; heads and 4H must divide by p;
    the arenas of the attention and FFN widths shrink with p."""
    full = tp.workspace_bytes(tp.make_config(2, 64, 4, 32, "fp32", op_parts=1))
    assert tp.workspace_bytes(tp.make_config(2, 64, 4, 32, "fp32", op_parts=0)) == full
    half = tp.workspace_bytes(tp.make_config(2, 64, 4, 32, "fp32", op_parts=2))
    assert 0 < half < full
    assert tp.workspace_bytes(tp.make_config(2, 64, 4, 32, "fp32", op_parts=3)) == 0
    assert tp.workspace_bytes(tp.make_config(2, 64, 4, 32, "fp32", op_parts=-1)) == 0
    rc, h = _init(tp.make_config(2, 64, 4, 32, "fp32", op_parts=4))
    assert rc == tp.TP_OK
    tp.lib.tp_stage_destroy(h)


def test_slice_order_errors_are_host_side():
    cfg = tp.make_config(1, 64, 4, 32, "fp32")
    rc, h = _init(cfg)
    assert rc == tp.TP_OK
    X, Y = 0x7e0000000000, 0x7e0000100000
    f, b = tp.lib.tp_slice_forward, tp.lib.tp_slice_backward
    assert f(h, 8, 16, X, Y) == tp.TP_ERR_ORDER      # must start at the cached length 0
    assert f(h, 0, 0, X, Y) == tp.TP_ERR_INVALID     # empty slice
    assert f(h, -1, 4, X, Y) == tp.TP_ERR_INVALID
    assert f(h, 0, 33, X, Y) == tp.TP_ERR_INVALID    # beyond max_seq
    assert f(h, 0, 8, None, Y) == tp.TP_ERR_INVALID
    assert b(h, 0, 8, X, Y) == tp.TP_ERR_ORDER       # frontier is 0: nothing to go back over
    assert b(h, 0, 8, X, None) == tp.TP_ERR_INVALID
    assert f(None, 0, 8, X, Y) == tp.TP_ERR_INVALID
    assert tp.lib.tp_kv_prefix_reset(None) == tp.TP_ERR_INVALID
    tp.lib.tp_stage_destroy(h)


def test_slices_need_a_started_sequence():
    """A new stage holds no sequence (its dK/dV buffer and fp16 W_qkv copy are
    unset): every slice call is refused on the host until tp_kv_prefix_reset."""
    X, Y = 0x7e0000000000, 0x7e0000100000
    for dtype in ("fp32", "bf16"):
        rc, h = _init(tp.make_config(1, 64, 4, 32, dtype))
        assert rc == tp.TP_OK
        assert tp.lib.tp_slice_forward(h, 0, 8, X, Y) == tp.TP_ERR_ORDER
        assert tp.lib.tp_slice_forward_static(h, 0, 8, X, Y) == tp.TP_ERR_ORDER
        assert tp.lib.tp_slice_backward(h, 0, 8, X, Y) == tp.TP_ERR_ORDER
        tp.lib.tp_stage_destroy(h)


def test_reset_flags_checked_on_the_host():
    """tp_kv_prefix_reset_ex refuses a null stage and unknown flag bits before
    enqueuing anything."""
    assert tp.lib.tp_kv_prefix_reset_ex(None, 0) == tp.TP_ERR_INVALID
    assert tp.lib.tp_kv_prefix_reset_ex(None, tp.SEQ_OVERWRITE_GRADS) == tp.TP_ERR_INVALID
    rc, h = _init(tp.make_config(1, 64, 4, 32, "bf16"))
    assert rc == tp.TP_OK
    for flags in (4, 5, 0x80000000, 0xFFFFFFFF):
        assert tp.lib.tp_kv_prefix_reset_ex(h, flags) == tp.TP_ERR_INVALID
    # still no sequence started
    assert tp.lib.tp_slice_backward(h, 0, 8, 0x7e0000000000, 0x7e0000100000) == tp.TP_ERR_ORDER
    tp.lib.tp_stage_destroy(h)


def test_header_constants_match_the_binding():
    """The #define and enum values of include/terapipe.h are the binding's."""
    src = open(os.path.join(ROOT, "include", "terapipe.h")).read()
    defines = dict((k, int(v.rstrip("u"), 0)) for k, v in
                   re.findall(r"#define\s+(TP_\w+)\s+(\w+)", src) if k != "TERAPIPE_H")
    assert defines == {"TP_SEQ_OVERWRITE_GRADS": tp.SEQ_OVERWRITE_GRADS,
                       "TP_SEQ_REUSE_WQKV_COPY": tp.SEQ_REUSE_WQKV_COPY}
    enums = dict((k, int(v)) for k, v in re.findall(r"\b(TP_[A-Z0-9_]+)\s*=\s*(-?\d+)", src))
    assert enums["TP_OK"] == tp.TP_OK and enums["TP_ERR_HIP"] == tp.TP_ERR_HIP
    assert enums["TP_ERR_ORDER"] == tp.TP_ERR_ORDER
    assert enums["TP_DTYPE_BF16"] == tp.DTYPE_BF16 and enums["TP_DTYPE_FP32"] == tp.DTYPE_FP32
    assert enums["TP_WGRAD_PER_SLICE"] == tp.WGRAD_PER_SLICE
    assert enums["TP_WGRAD_DEFERRED"] == tp.WGRAD_DEFERRED


def test_profile_argument_errors():
    cfg = tp.make_config(1, 64, 4, 32, "fp32")
    rc, h = _init(cfg)
    L = (ctypes.c_int * 1)(8)
    C = (ctypes.c_int * 1)(0)
    out = (ctypes.c_int64 * 1)()
    prof = tp.lib.tp_profile_slice_cost
    assert prof(h, L, 0, C, 1, 1, 1, out, out) == tp.TP_ERR_INVALID
    assert prof(h, L, 1, C, 1, 1, 0, out, out) == tp.TP_ERR_INVALID
    bad = (ctypes.c_int * 1)(0)
    assert prof(h, bad, 1, C, 1, 1, 1, out, out) == tp.TP_ERR_INVALID
    tp.lib.tp_stage_destroy(h)


@pytest.mark.parametrize("kind", ["random", "ties", "linear", "flops"])
def test_dp_identical_to_oracle(kind):
    for U in (1, 2, 5, 12, 40, 128):
        for seed in range(3):
            cost = synth.cost_table(U, kind, seed)
            for K in (1, 2, 4, 12, 48):
                for eps in (0, 3):
                    units, T, _, _ = oracle_dp(cost, K, eps)
                    lens, T2 = tp.dp_optimal_slicing(cost, 16, K, eps)
                    assert T2 == T, (kind, U, seed, K, eps)
                    assert lens == [16 * u for u in units], (kind, U, seed, K, eps)


def test_dp_matches_exhaustive():
    for kind in ("random", "ties", "linear", "flops"):
        for K in (1, 2, 3, 4, 8):
            cost = synth.cost_table(12, kind, 5)
            best, argmins = exhaustive_optimal(cost, K)
            lens, T = tp.dp_optimal_slicing(cost, 1, K)
            assert T == best and tuple(lens) in argmins


def test_dp_long_sequence_identical():
    """8192 tokens in units of 16 (512 units), flop-shaped costs: same answer as the oracle."""
    U = 512
    cost = synth.cost_table(U, "flops", 0)
    units, T, _, _ = oracle_dp(cost, 48)
    lens, T2 = tp.dp_optimal_slicing(cost, 16, 48)
    assert T2 == T and lens == [16 * u for u in units]


def test_dp_rejects_bad_arguments():
    cost = synth.cost_table(6, "random", 0)
    for args in ((cost, 16, 0), (cost, 0, 2)):
        with pytest.raises(tp.TerapipeError) as e:
            tp.dp_optimal_slicing(*args)
        assert e.value.status == tp.TP_ERR_INVALID
    bad = cost.copy()
    bad[2, 1] = -5
    with pytest.raises(tp.TerapipeError):
        tp.dp_optimal_slicing(bad, 16, 2)
    with pytest.raises(tp.TerapipeError):
        tp.dp_optimal_slicing(cost, 16, 2, -1)


def test_static_forward_plans_on_the_host():
    """tp_slice_forward_static plans the slice on the host: a slice whose
    partial sums exceed the static scratch array (here the split output
    projection of a 5120-wide layer over 256 rows) is rejected with
    TP_ERR_WORKSPACE before anything is enqueued, and the order checks of
    tp_slice_forward apply."""
    X, Y = 0x7e0000000000, 0x7e0000100000
    f = tp.lib.tp_slice_forward_static
    rc, h = _init(tp.make_config(1, 5120, 40, 256, "bf16", "deferred"))
    assert rc == tp.TP_OK
    assert f(h, 0, 256, X, Y) == tp.TP_ERR_WORKSPACE
    assert f(h, 8, 16, X, Y) == tp.TP_ERR_ORDER      # still at the sequence start
    assert f(h, 0, 257, X, Y) == tp.TP_ERR_INVALID
    assert f(h, 0, 8, None, Y) == tp.TP_ERR_INVALID
    tp.lib.tp_stage_destroy(h)
