"""Shared checks of the GPU parity tests (not a test module).

* ``localized_error``: the largest error of one row or one column of U,
  relative to the RMS norm of the reference's rows (columns).  A single
  wrong row of a 3072-row matrix moves the global relative Frobenius error by
  only about 1/sqrt(3072) = 0.018, below the 2e-2 Newton-Schulz tolerance, but
  moves this measure to about 1.  Rounding errors spread over every element
  give a value close to the global relative error; the bound used is
  ``ROW_FACTOR`` times the case's global tolerance (a row of b elements with
  independent rounding errors deviates from the mean error by O(1/sqrt(b)),
  and single-element rows by a chi(1) factor, below 4 for a few hundred rows).
* ``record``: per-case error, tolerance and margin.  When the environment
  variable NORMPRE_PARITY_LOG names a file, the session writes every record
  there as a Markdown table at its end (see conftest.py).
"""
from __future__ import annotations

import numpy as np

ROW_FACTOR = 5.0

RECORDS: list[dict] = []


def localized_error(u, ref) -> float:
    u = np.asarray(u, np.float64)
    ref = np.asarray(ref, np.float64)
    d = u - ref
    worst = 0.0
    for axis in (1, 0):
        dn = np.linalg.norm(d, axis=axis)
        rn = np.linalg.norm(ref, axis=axis)
        rms = float(np.sqrt(np.mean(rn * rn)))
        worst = max(worst, float(dn.max()) / (rms if rms > 0 else 1.0))
    return worst


def record(case: str, quantity: str, err: float, tol: float, **extra) -> None:
    RECORDS.append({"case": case, "quantity": quantity, "err": float(err), "tol": float(tol),
                    "margin": float(tol) / max(float(err), 1e-300), **extra})


def check_update(case: str, u, ref_u, tol: float, **extra) -> float:
    """Global relative Frobenius error and localized (per row / column) error
    of an update against the oracle's; records both and asserts both."""
    den = np.linalg.norm(ref_u)
    err = float(np.linalg.norm(np.asarray(u, np.float64) - ref_u) / (den if den > 0 else 1.0))
    loc = localized_error(u, ref_u)
    record(case, "U rel-Frobenius", err, tol, **extra)
    record(case, "U worst row/col", loc, ROW_FACTOR * tol, **extra)
    assert err < tol, (case, err, tol)
    assert loc < ROW_FACTOR * tol, (case, loc, ROW_FACTOR * tol)
    return err


def write_markdown(path: str) -> None:
    lines = ["| case | quantity | error | tolerance | tol / err | notes |", "|---|---|---|---|---|---|"]
    for r in RECORDS:
        notes = ", ".join(f"{k} {v:.3g}" if isinstance(v, float) else f"{k} {v}" for k, v in r.items()
                          if k not in ("case", "quantity", "err", "tol", "margin"))
        lines.append(f"| {r['case']} | {r['quantity']} | {r['err']:.3e} | {r['tol']:.3e} | {r['margin']:.1f} | {notes} |")
    worst = min(RECORDS, key=lambda r: r["margin"]) if RECORDS else None
    head = [f"{len(RECORDS)} checks."]
    if worst:
        head.append(f"Smallest margin: {worst['margin']:.2f} ({worst['case']}, {worst['quantity']}).")
    with open(path, "w") as f:
        f.write(" ".join(head) + "\n\n" + "\n".join(lines) + "\n")
