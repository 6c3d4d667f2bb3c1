"""Acceptance rules for comparing the HIP path against the oracle.

TEST INFRASTRUCTURE, like the rest of this package: only the tests, the smoke check and the
benchmark's CPU-baseline leg use it.

Selection (Sec. 4 "Page-based DELTA"; App. A, Alg. 2).  The oracle decides in float64, the
device in float32, so when two candidate scores at the k-th boundary lie within float32
rounding of each other both choices are correct.  The rule: let tau be the oracle's need-th
largest candidate score (need = K - L).  Candidates scoring above tau*(1+band) must be chosen,
those below tau*(1-band) must not, the recency units must be present, and the set must be
ascending, unique and of size min(K, n_units).  When no other score falls inside the band this
is bit-exact equality with the oracle.

Outputs: |o_dev - o_orc| <= atol + rtol*|o_orc| elementwise (bf16 output, fp32 accumulation).
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

SEL_BAND = 1e-5
OUT_ATOL = 2e-2
OUT_RTOL = 1e-2


@dataclass
class SelectionVerdict:
    ok: bool
    exact: bool                 # device set == oracle set
    band_resolved: int          # units decided inside the band (device differs legitimately)
    reasons: list = field(default_factory=list)


def check_selection(S_oracle: np.ndarray, budget_units: int, recent_units: int,
                    sel_dev: np.ndarray, sel_oracle: np.ndarray,
                    band: float = SEL_BAND) -> SelectionVerdict:
    """Accept the device's unit set sel_dev against the oracle's scores S_oracle."""
    sel_dev = np.asarray(sel_dev, dtype=np.int64)
    sel_oracle = np.asarray(sel_oracle, dtype=np.int64)
    n = len(S_oracle)
    reasons = []
    if len(sel_dev) != min(budget_units, n):
        reasons.append(f"size {len(sel_dev)} != min(K={budget_units}, n={n})")
    if len(sel_dev) and (np.any(np.diff(sel_dev) <= 0) or sel_dev[0] < 0 or sel_dev[-1] >= n):
        reasons.append("not ascending / unique / in range")
    exact = len(sel_dev) == len(sel_oracle) and bool(np.all(sel_dev == sel_oracle))
    if exact:
        return SelectionVerdict(not reasons, True, 0, reasons)
    if n <= budget_units:
        reasons.append("context fits the budget: every unit must be kept")
        return SelectionVerdict(False, False, 0, reasons)
    n_cand = n - recent_units
    need = budget_units - recent_units
    chosen = set(sel_dev.tolist())
    recent = set(range(n_cand, n))
    if not recent <= chosen:
        reasons.append("recency units missing")
    cand = S_oracle[:n_cand]
    order = np.lexsort((np.arange(n_cand), -cand))
    tau = cand[order[need - 1]]
    sure_in = set(np.nonzero(cand > tau * (1 + band))[0].tolist())
    sure_out = set(np.nonzero(cand < tau * (1 - band))[0].tolist())
    if not sure_in <= chosen:
        reasons.append(f"{len(sure_in - chosen)} clearly-above-threshold units missing")
    if chosen & sure_out:
        reasons.append(f"{len(chosen & sure_out)} clearly-below-threshold units chosen")
    resolved = len(chosen.symmetric_difference(set(sel_oracle.tolist()))) // 2
    return SelectionVerdict(not reasons, False, resolved, reasons)


def check_output(o_dev: np.ndarray, o_oracle: np.ndarray, atol: float = OUT_ATOL,
                 rtol: float = OUT_RTOL):
    """Elementwise |o_dev - o_orc| <= atol + rtol*|o_orc|.  Returns (ok, max_abs_err, n_bad)."""
    o_dev = np.asarray(o_dev, dtype=np.float64)
    o_oracle = np.asarray(o_oracle, dtype=np.float64)
    err = np.abs(o_dev - o_oracle)
    bad = ~(err <= atol + rtol * np.abs(o_oracle))       # NaN counts as bad
    return (not bool(bad.any())), float(np.nanmax(err) if err.size else 0.0), int(bad.sum())
