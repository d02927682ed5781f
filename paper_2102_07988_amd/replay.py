"""Offline replay of the slicing decisions in a benchmark report.

The benchmark's `pipeline` block carries the cost tables it measured (int64 ns,
entry [slice length in units - 1][context in units], -1 past the sequence end):
the full table on its grid, the same table measured once more, the model-mode
table of Eq. 9, and the fine model-mode table as its t(i, 0) column plus fitted
coefficients.  The DP of Sec. 3.3 (Eq. 5-8, Algorithm 1) is deterministic on
integer costs, so every slicing and latency the report states follows from
these tables alone; this module recomputes them with the library's DP (host
code, no device needed) and lists any difference.

    python -m paper_2102_07988_amd.replay BENCH.json   (the JSON line, or a file
                                                        whose last line is it)
"""
from __future__ import annotations

import json
import sys
from typing import List

import numpy as np

from . import terapipe as tp


def _check(name: str, got, want, out: List[dict]) -> None:
    out.append({"check": name, "ok": got == want, "replayed": got, "reported": want})


def replay(report: dict) -> List[dict]:
    """Recompute the DP slicings and Eq. 5 latencies of a report's pipeline block."""
    pipe = report["pipeline"]
    tab = pipe["tables"]
    unit, K = int(tab["unit"]), int(pipe["K"])
    out: List[dict] = []
    measured = np.asarray(tab["measured_ns"], dtype=np.int64)
    lens, T = tp.dp_optimal_slicing(measured, unit, K)
    _check("measured table: DP slicing", lens, pipe["dp_slicing"], out)
    _check("measured table: DP latency (ms)", round(T / 1e6, 3), pipe["dp_T_ms"], out)
    model = np.asarray(tab["model_ns"], dtype=np.int64)
    # the model table is its own j = 0 column plus the fitted overhead
    rebuilt = tp.cost_table_from_model(model[:, 0], unit, tab["model_coef_ns"])
    _check("model table: rebuilt from t(i, 0) and coefficients", bool(np.array_equal(rebuilt, model)),
           True, out)
    mlens, _ = tp.dp_optimal_slicing(model, unit, K)
    _check("model table: DP slicing", mlens, pipe["model"]["dp_slicing"], out)
    fine = pipe.get("model_fine")
    if fine:
        fcost = tp.cost_table_from_model(fine["t0_ns"], int(fine["unit"]), fine["coef_full"])
        for k, summary in fine["by_K"].items():
            flens, fT = tp.dp_optimal_slicing(fcost, int(fine["unit"]), int(k))
            _check(f"fine model table, K = {k}: DP slicing", flens, summary["dp_slicing"], out)
            _check(f"fine model table, K = {k}: DP latency (ms)", round(fT / 1e6, 3),
                   summary["dp_T_ms"], out)
    return out


def _load(path: str) -> dict:
    text = open(path).read().strip()
    if not text:
        raise ValueError(f"{path} is empty")
    try:
        return json.loads(text)
    except json.JSONDecodeError:
        return json.loads(text.splitlines()[-1])


def main(argv: List[str]) -> int:
    if len(argv) != 1:
        print(__doc__)
        return 2
    report = _load(argv[0])
    if "parsed" in report and "pipeline" not in report:
        report = report["parsed"]
    results = replay(report)
    for r in results:
        print(("ok      " if r["ok"] else "DIFFERS ") + r["check"] +
              ("" if r["ok"] else f": replayed {r['replayed']}, reported {r['reported']}"))
    return 0 if all(r["ok"] for r in results) else 1


if __name__ == "__main__":
    sys.exit(main(sys.argv[1:]))
