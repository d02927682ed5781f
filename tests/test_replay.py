"""Offline replay of a benchmark report's slicings (paper_2102_07988_amd/replay.py)
on a synthetic report whose tables are seeded int64 families and whose stated
slicings come from the oracle's DP (Algorithm 1, oracle/oracle.py): the replay
through the library's DP must agree, and must flag a report whose slicing was
altered.  CPU only."""
import json

import numpy as np

from oracle import cost_table_from_model as oracle_table
from oracle import dp_optimal_slicing as _oracle_dp


def oracle_dp(cost, unit, K):
    """The oracle's Algorithm 1 (slice lengths in units) as token lengths and T."""
    units, T, _, _ = _oracle_dp(cost, K)
    return [u * unit for u in units], T


def _table(U, rng):
    c = np.full((U, U), -1, dtype=np.int64)
    for k in range(1, U + 1):
        for j in range(U - k + 1):
            c[k - 1, j] = 1000 + 350 * k + 7 * j + 3 * k * j + int(rng.integers(0, 40))
    return c


def _ms(v):
    return round(v / 1e6, 3)


def _report(rng):
    U, unit, K = 16, 128, 48
    measured = _table(U, rng)
    again = _table(U, rng)
    coef = [120.0, 1.5, 2.25, 0.125]
    model = oracle_table(measured[:, 0], unit, coef)
    lens, T = oracle_dp(measured, unit, K)
    mlens, _ = oracle_dp(model, unit, K)
    Uf, fu = 64, 32
    t0 = [800 + 90 * k for k in range(1, Uf + 1)]
    fcost = oracle_table(t0, fu, coef)
    by_K = {}
    for k in (48, 96):
        fl, fT = oracle_dp(fcost, fu, k)
        by_K[str(k)] = {"dp_slicing": fl, "dp_T_ms": _ms(fT)}
    return {"pipeline": {
        "K": K, "dp_slicing": lens, "dp_T_ms": _ms(T),
        "model": {"dp_slicing": mlens},
        "tables": {"unit": unit, "measured_ns": measured.tolist(),
                   "measured_again_ns": again.tolist(), "model_ns": model.tolist(),
                   "model_coef_ns": coef},
        "model_fine": {"unit": fu, "t0_ns": t0, "coef_full": coef, "by_K": by_K}}}


def test_replay_reproduces_the_oracle_slicings(tmp_path):
    from paper_2102_07988_amd import replay
    rep = _report(np.random.default_rng(3))
    results = replay.replay(rep)
    assert results and all(r["ok"] for r in results), [r for r in results if not r["ok"]]
    # the command-line form reads a JSON line from a file
    p = tmp_path / "bench.json"
    p.write_text("log line\n" + json.dumps(rep) + "\n")
    assert replay.main([str(p)]) == 0


def test_replay_flags_an_altered_slicing():
    from paper_2102_07988_amd import replay
    rep = _report(np.random.default_rng(4))
    s = rep["pipeline"]["dp_slicing"]
    if len(s) >= 2:
        s[0], s[1] = s[0] + 128, s[1] - 128
    else:
        s.append(0)
    results = replay.replay(rep)
    assert not next(r for r in results if r["check"] == "measured table: DP slicing")["ok"]
