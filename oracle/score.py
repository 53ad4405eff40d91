"""Oracle for dequantized retrieval scoring -- test infrastructure only.

Paper:
  * Section 2.1 and Appendix "Rank invariance, in full": a query's score of a
    record is the inner product q . x.  Scoring the reconstruction x_hat = code*s
    instead of x moves it by |q . (x - x_hat)| <= ||q||_1 ||x - x_hat||_inf
    <= eps ||q||_1 (Hoelder, with the per-coordinate bound of Q_eps).
  * Theorem "Score deficit" and Corollary "top-k delta-cover": what the retained
    set loses is at most delta per query; with the quantized store the two
    bounds add (see oracle.invariants).

Readings:
  * the score of query j against stored record y is the exact real
    s * sum_d q_{j,d} code_{y,d}  (the dequantized record, not its float32
    materialisation), computed here in binary64;
  * the top-k order is (score descending, id ascending); when k exceeds the
    store size the tail is padded with (-inf, -1);
  * the bound returned per query is beta_j = eps * ||q_j||_1.
"""
from __future__ import annotations

import numpy as np


def scores(q, codes_rows, eps: float) -> np.ndarray:
    """(nq x N) binary64 scores s * Q . C^T."""
    q64 = np.asarray(q, dtype=np.float32).astype(np.float64)
    c64 = np.asarray(codes_rows, dtype=np.int64).astype(np.float64)
    return (2.0 * float(eps)) * (q64 @ c64.T)


def topk(s, ids, k: int):
    """Per row, the k best by (score desc, id asc)."""
    s = np.asarray(s, dtype=np.float64)
    ids = np.asarray(ids, dtype=np.int64)
    nq, n = s.shape
    out_s = np.full((nq, k), -np.inf)
    out_i = np.full((nq, k), -1, dtype=np.int64)
    kk = min(k, n)
    for j in range(nq):
        order = np.lexsort((ids, -s[j]))[:kk]
        out_s[j, :kk] = s[j, order]
        out_i[j, :kk] = ids[order]
    return out_s, out_i


def bound(q, eps: float) -> np.ndarray:
    """beta_j = eps * ||q_j||_1 (binary64)."""
    q64 = np.asarray(q, dtype=np.float32).astype(np.float64)
    return float(eps) * np.sum(np.abs(q64), axis=1)


def score_topk(q, codes_rows, ids, eps: float, k: int):
    s = scores(q, codes_rows, eps)
    ts, ti = topk(s, ids, k)
    return ts, ti, bound(q, eps)
