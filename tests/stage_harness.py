"""Shared helpers of the GPU parity tests: build the same seeded stage for the
HIP path (through the C ABI) and for the oracle, run a sequence, compare."""
from __future__ import annotations

import numpy as np
import torch

from paper_2102_07988_amd import synth

PARAM_KEYS = synth.PARAM_NAMES


def rel_l2(a, b) -> float:
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    nb = np.linalg.norm(b)
    d = np.linalg.norm(a - b)
    return float(d / nb) if nb > 0 else float(d)


def make_inputs(n_layers, H, L, dtype, seeds=(0, 1, 2), randomize_ln=False, op_parts=1):
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    sx, sp, sdy = seeds
    params = synth.stage_params(n_layers, H, seed=sp, dtype=tdt, randomize_ln=randomize_ln,
                                op_parts=op_parts)
    x = synth.hidden_states(L, H, seed=sx, dtype=tdt)
    dy = synth.upstream_grad(L, H, seed=sdy, dtype=tdt)
    return params, x, dy


def _nan_grads(st):
    """Gradient buffers an overwriting sequence must never read."""
    for g in st.grads:
        for v in g.values():
            v.fill_(float("nan"))


def run_gpu(params, x, dy, H, heads, L, dtype, fwd_lens, bwd_lens=None, wgrad="per_slice",
            device="cuda:0", op_parts=1, overwrite_grads=False):
    from paper_2102_07988_amd import terapipe as tp
    dparams = [{k: v.to(device).contiguous() for k, v in p.items()} for p in params]
    st = tp.Stage(dparams, H, heads, L, dtype=dtype, wgrad=wgrad, op_parts=op_parts)
    if overwrite_grads:
        _nan_grads(st)
    y, dx = st.run_sequence(x.to(device), dy.to(device), fwd_lens, bwd_lens, overwrite_grads)
    torch.cuda.synchronize()
    out = {"y": y.float().cpu().numpy(), "dx": dx.float().cpu().numpy(),
           "grads": [{k: v.cpu().numpy() for k, v in g.items()} for g in st.grads]}
    del st
    return out


def run_oracle(params, x, dy, H, heads, L, fwd_lens, bwd_lens=None, op_parts=1):
    from oracle import OracleStage
    ost = OracleStage(synth.params_f64(params), H, heads, L, op_parts=op_parts)
    y, dx = ost.run_sequence(synth.to_f64(x), synth.to_f64(dy), fwd_lens, bwd_lens)
    return {"y": y, "dx": dx, "grads": ost.grads}


def make_batch_inputs(n_layers, H, L, batch, dtype, seeds=(0, 1, 2), randomize_ln=False,
                      op_parts=1):
    """Parameters and [L, batch, H] inputs / upstream gradients."""
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    sx, sp, sdy = seeds
    params = synth.stage_params(n_layers, H, seed=sp, dtype=tdt, randomize_ln=randomize_ln,
                                op_parts=op_parts)
    x = synth.batch_hidden_states(L, batch, H, seed=sx, dtype=tdt)
    dy = synth.batch_upstream_grad(L, batch, H, seed=sdy, dtype=tdt)
    return params, x, dy


def run_gpu_batch(params, x, dy, H, heads, L, dtype, fwd_lens, bwd_lens=None, wgrad="per_slice",
                  device="cuda:0", op_parts=1, overwrite_grads=False):
    """One batched stage (batch = x.shape[1]) over the whole sequence; with
    overwrite_grads the gradient buffers start NaN-filled and the sequence
    stores its gradients (TP_SEQ_OVERWRITE_GRADS)."""
    from paper_2102_07988_amd import terapipe as tp
    dparams = [{k: v.to(device).contiguous() for k, v in p.items()} for p in params]
    st = tp.Stage(dparams, H, heads, L, dtype=dtype, wgrad=wgrad, batch=x.shape[1],
                  op_parts=op_parts)
    if overwrite_grads:
        _nan_grads(st)
    y, dx = st.run_sequence(x.to(device), dy.to(device), fwd_lens, bwd_lens, overwrite_grads)
    torch.cuda.synchronize()
    out = {"y": y.float().cpu().numpy(), "dx": dx.float().cpu().numpy(),
           "grads": [{k: v.cpu().numpy() for k, v in g.items()} for g in st.grads]}
    del st
    return out


def run_oracle_batch(params, x, dy, H, heads, L, fwd_lens, bwd_lens=None, op_parts=1):
    """The sequences of a batch are independent: one oracle run per sequence,
    outputs stacked on axis 1, parameter gradients summed."""
    b = x.shape[1]
    ys, dxs, grads = [], [], None
    for s in range(b):
        r = run_oracle(params, x[:, s], dy[:, s], H, heads, L, fwd_lens, bwd_lens, op_parts)
        ys.append(r["y"])
        dxs.append(r["dx"])
        if grads is None:
            grads = [{k: v.copy() for k, v in g.items()} for g in r["grads"]]
        else:
            for acc, g in zip(grads, r["grads"]):
                for k in acc:
                    acc[k] += g[k]
    return {"y": np.stack(ys, axis=1), "dx": np.stack(dxs, axis=1), "grads": grads}


def compare(got, ref, tol, label=""):
    errs = {"y": rel_l2(got["y"], ref["y"]), "dx": rel_l2(got["dx"], ref["dx"])}
    for li, (g, r) in enumerate(zip(got["grads"], ref["grads"])):
        for k in PARAM_KEYS:
            errs[f"L{li}.{k}"] = rel_l2(g[k], r[k])
    worst = max(errs, key=errs.get)
    print(f"[{label}] worst rel-L2 {worst} = {errs[worst]:.3e}", flush=True)
    bad = {k: v for k, v in errs.items() if not (v <= tol)}
    assert not bad, f"{label}: rel-L2 above {tol}: {bad}"
    return errs
