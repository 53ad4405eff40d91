"""Checkers for properties the paper proves -- test infrastructure only.

Each function returns a list of violations (empty when the property holds), so
that tests can report what failed.

  * ``cover``: every dropped arrival has a representative that was retained,
    arrived earlier, and lies within delta (Definition "delta-substitution",
    Section 2.4; Proposition "greedy is simultaneously a cover and a packing",
    cover part).
  * ``packing``: retained rows are pairwise more than delta apart (same
    Proposition, packing part).
  * ``lowest_index``: no retained row with a smaller id than the representative
    was within delta at the arrival (Appendix "Representative selection").
  * ``score_deficit``: for unit queries, 0 <= max_S q.x - max_R q.z <= delta_hat
    (Theorem "Score deficit", with the measured bound of Appendix "The measured
    bound" in place of delta).
"""
from __future__ import annotations

import numpy as np

from . import dedup


def cover(x, rep, tau: float):
    x = np.asarray(x, dtype=np.float32)
    rep = np.asarray(rep, dtype=np.int64)
    kept = set(np.nonzero(rep < 0)[0].tolist())
    bad = []
    for i in np.nonzero(rep >= 0)[0].tolist():
        r = int(rep[i])
        if r >= i or r not in kept or not dedup.within(x[i], x[r], tau):
            bad.append(i)
    return bad


def packing(x, rep, tau: float, margin: float = 1e-9):
    """Kept pairs must satisfy d^2 > delta^2; pairs within ``margin`` of the
    threshold in binary64 are re-checked exactly."""
    x = np.asarray(x, dtype=np.float32)
    kept = np.nonzero(np.asarray(rep) < 0)[0]
    k64 = x[kept].astype(np.float64)
    n2 = np.einsum("ij,ij->i", k64, k64)
    d2t = float(dedup.delta2(tau))
    bad = []
    for s in range(0, kept.size, 2048):
        g = k64[s:s + 2048] @ k64.T
        d2 = n2[s:s + 2048, None] + n2[None, :] - 2.0 * g
        rows, cols = np.nonzero(d2 <= d2t + margin)
        for a, b in zip(rows.tolist(), cols.tolist()):
            i, j = int(kept[s + a]), int(kept[b])
            if i < j and dedup.within(x[i], x[j], tau):
                bad.append((i, j))
    return bad


def lowest_index(x, rep, tau: float, sample=None):
    """For dropped arrivals (all, or the ``sample`` of ids), the representative
    is the lowest retained id within delta among ids retained before it."""
    x = np.asarray(x, dtype=np.float32)
    rep = np.asarray(rep, dtype=np.int64)
    kept_mask = rep < 0
    idx = np.nonzero(rep >= 0)[0] if sample is None else np.asarray(sample)
    bad = []
    for i in idx.tolist():
        kb = np.nonzero(kept_mask[:i])[0]
        if dedup.decide_one(x, i, kb, tau) != int(rep[i]):
            bad.append(i)
    return bad


def score_deficit(x, rep, queries, dhat: float, tol: float = 1e-12):
    """0 <= max_S q.x - max_R q.z <= dhat * ||q|| (+ rounding tol) per query."""
    x64 = np.asarray(x, dtype=np.float32).astype(np.float64)
    kept = np.asarray(rep) < 0
    q64 = np.asarray(queries, dtype=np.float64)
    s_all = q64 @ x64.T
    top_s = s_all.max(axis=1)
    top_r = s_all[:, kept].max(axis=1)
    gap = top_s - top_r
    qn = np.linalg.norm(q64, axis=1)
    return np.nonzero((gap < -tol) | (gap > dhat * qn + tol))[0].tolist()
