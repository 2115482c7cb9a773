"""Comparison rules between a result under test and the fp64 oracle.

TEST INFRASTRUCTURE ONLY (same import rule as ``oracle.losa_oracle``).

* Block masses: max-abs error.
* Selection (Sec. 4.1, Eq. (3)): the kept sets must be equal, except for blocks
  the fp64 order leaves undecidable at fp32 precision.  A block at oracle rank
  r (1-based) is exempt when the oracle's cumulative interval
  [c_{r-1}, c_r] meets [tau - eps, tau + eps] (the result may stop one block
  early or late there), or when its mass is within ``tie`` of the boundary
  mass mbar(pi(s)) (a near-tie at the cut may swap which block is kept).  In
  addition the kept set's oracle mass must reach tau - eps, and for tau >= 1
  no exemption applies.
* Attention outputs: max-abs and mean-abs error over valid rows.
"""
from __future__ import annotations

import numpy as np


def mass_error(m_test, m_ref) -> float:
    return float(np.max(np.abs(np.asarray(m_test, np.float64) - np.asarray(m_ref, np.float64))))


def compare_selection(row_ptr, col_idx, details, mbar_ref, tau: float,
                      eps: float = 1e-5, tie: float = 1e-6) -> dict:
    """Check a CSR selection against the oracle's per-row selection details.

    ``details`` is the list returned by ``losa_oracle.select_blocks`` (computed
    from ``mbar_ref``).  Returns a summary dict with ``ok`` and the first
    failing row, if any.
    """
    row_ptr = np.asarray(row_ptr, dtype=np.int64)
    col_idx = np.asarray(col_idx, dtype=np.int64)
    mflat = np.asarray(mbar_ref, dtype=np.float64).reshape(len(details), -1)
    n_exact = n_exempt = n_tie = 0
    for r, det in enumerate(details):
        got = col_idx[row_ptr[r]:row_ptr[r + 1]]
        if got.size > 1 and np.any(np.diff(got) <= 0):
            return dict(ok=False, row=r, reason="indices not strictly ascending")
        want = det.omega
        if got.size == want.size and np.array_equal(got, want):
            n_exact += 1
            continue
        if tau >= 1.0 or det.s == 0:
            return dict(ok=False, row=r, reason="mismatch where no exemption applies",
                        got=got.tolist(), want=want.tolist())
        rank = np.empty(det.order.size, dtype=np.int64)
        rank[det.order] = np.arange(det.order.size)
        cum = det.cum
        cprev = np.concatenate([[0.0], cum[:-1]])
        boundary_mass = mflat[r, det.order[det.s - 1]]
        diff = np.setxor1d(got, want)
        tie_used = False
        for j in diff:
            rr = rank[j]
            near_tau = (cprev[rr] <= tau + eps) and (cum[rr] >= tau - eps)
            near_tie = abs(mflat[r, j] - boundary_mass) <= tie
            if not (near_tau or near_tie):
                return dict(ok=False, row=r, reason=f"block {int(j)} differs and is not exempt",
                            got=got.tolist(), want=want.tolist())
            tie_used |= not near_tau
        if mflat[r, got].sum() < tau - eps:
            return dict(ok=False, row=r, reason="kept mass below tau - eps")
        n_exempt += 1
        n_tie += tie_used
    # exempt = rows that differ, all within the exemptions; tie_rows = those
    # among them that needed the near-tie rule (not only the cumulative one)
    return dict(ok=True, rows=len(details), exact=n_exact, exempt=n_exempt, tie_rows=n_tie)


def output_errors(o_test, o_ref, N: int):
    """(max-abs, mean-abs) error over the valid rows n < N of [B,H,N_pad,d]."""
    a = np.asarray(o_test, dtype=np.float64)[:, :, :N]
    b = np.asarray(o_ref, dtype=np.float64)[:, :, :N]
    err = np.abs(a - b)
    return float(err.max()), float(err.mean())
