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
  variable NORMPRE_PARITY_LOG names a file, the session writes a Markdown
  summary there at its end (see conftest.py): per test function the number
  of checks and the smallest and median margin, then the tightest checks.
"""
from __future__ import annotations

import os
import sys

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


def _test_family() -> str:
    node = os.environ.get("PYTEST_CURRENT_TEST", "?").split(" ")[0]
    return node.split("[")[0]


def record(case: str, quantity: str, err: float, tol: float, **extra) -> None:
    RECORDS.append({"test": _test_family(), "case": case, "quantity": quantity, "err": float(err),
                    "tol": float(tol), "margin": float(tol) / float(err) if err > 0 else float("inf"), **extra})


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


def _row(r: dict) -> str:
    notes = ", ".join(f"{k} {v:.3g}" if isinstance(v, float) else f"{k} {v}" for k, v in r.items()
                      if k not in ("test", "case", "quantity", "err", "tol", "margin"))
    return f"| {_md(r['case'])} | {_md(r['quantity'])} | {r['err']:.3e} | {r['tol']:.3e} | {r['margin']:.1f} | {notes} |"


def _md(text: str) -> str:
    return str(text).replace("|", "\\|")


def write_markdown(path: str, tightest: int = 40) -> None:
    """Per test function: checks, smallest and median tol/err; then the
    `tightest` checks with the smallest margins in full."""
    fams: dict[str, list[dict]] = {}
    for r in RECORDS:
        fams.setdefault(r["test"], []).append(r)
    cmd = "NORMPRE_PARITY_LOG=<file> python -m pytest " + " ".join(sys.argv[1:])
    out = ["# Parity margins of the GPU tests against the oracle", "",
           f"Written at the end of `{cmd}` (repository root).  tol / err > 1 passes; "
           "`U worst row/col` is the largest row or column error relative to the RMS row (column) norm; "
           "inf marks a bit-identical result.", "",
           f"{len(RECORDS)} checks in {len(fams)} test functions.", "",
           "| test | checks | quantities | smallest tol/err (case) | median tol/err |", "|---|---|---|---|---|"]
    for name, rs in sorted(fams.items()):
        w = min(rs, key=lambda r: r["margin"])
        qs = ", ".join(sorted({_md(r["quantity"]) for r in rs}))
        med = float(np.median([r["margin"] for r in rs]))
        out.append(f"| {name} | {len(rs)} | {qs} | {w['margin']:.2f} ({_md(w['case'])}, {_md(w['quantity'])}) | {med:.1f} |")
    out += ["", f"The {min(tightest, len(RECORDS))} checks with the smallest margins:", "",
            "| case | quantity | error | tolerance | tol / err | notes |", "|---|---|---|---|---|---|"]
    out += [_row(r) for r in sorted(RECORDS, key=lambda r: r["margin"])[:tightest]]
    with open(path, "w") as f:
        f.write("\n".join(out) + "\n")
