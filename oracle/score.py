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
    """(nq x N) binary64 scores s * Q . C^T.  Codes may be given as integers or
    as binary64 values already holding them (exact below 2^53)."""
    q64 = np.asarray(q, dtype=np.float32).astype(np.float64)
    c = np.asarray(codes_rows)
    c64 = c if c.dtype == np.float64 else c.astype(np.int64).astype(np.float64)
    return (2.0 * float(eps)) * (q64 @ c64.T)


def topk_sorted(s, ids, k: int):
    """Per row, the k best by (score desc, id asc): the whole row sorted."""
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


def topk(s, ids, k: int):
    """Per row, the k best by (score desc, id asc) -- topk_sorted's result,
    found by sorting only the entries at or above the row's k-th largest score
    (every entry tied with it included), which is all the order can take."""
    s = np.asarray(s, dtype=np.float64)
    ids = np.asarray(ids, dtype=np.int64)
    nq, n = s.shape
    if n <= 4 * k:
        return topk_sorted(s, ids, k)
    out_s = np.full((nq, k), -np.inf)
    out_i = np.full((nq, k), -1, dtype=np.int64)
    for j in range(nq):
        kth = np.partition(s[j], n - k)[n - k]          # the k-th largest score
        cand = np.nonzero(s[j] >= kth)[0]
        order = cand[np.lexsort((ids[cand], -s[j, cand]))][:k]
        out_s[j] = s[j, order]
        out_i[j] = ids[order]
    return out_s, out_i


def bound(q, eps: float) -> np.ndarray:
    """beta_j = eps * ||q_j||_1 (binary64)."""
    q64 = np.asarray(q, dtype=np.float32).astype(np.float64)
    return float(eps) * np.sum(np.abs(q64), axis=1)


def score_topk(q, codes_rows, ids, eps: float, k: int):
    s = scores(q, codes_rows, eps)
    ts, ti = topk(s, ids, k)
    return ts, ti, bound(q, eps)


def score_topk_blocked(q, x_rows, ids, eps: float, k: int, block: int = 1 << 16):
    """score_topk over a store given by its float32 rows: each block of rows is
    coded by the Q_eps oracle (oracle.qeps.codes) and scored in binary64, and
    the per-query best k of all blocks are merged by (score desc, id asc).  The
    same definition as score_topk(q, codes(x_rows), ...), without holding every
    code or score at once."""
    from oracle import qeps
    q = np.asarray(q, dtype=np.float32)
    ids = np.asarray(ids, dtype=np.int64)
    nq = q.shape[0]
    best_s = np.full((nq, 0), -np.inf)
    best_i = np.full((nq, 0), -1, dtype=np.int64)
    for b0 in range(0, ids.size, block):
        rows = np.asarray(x_rows[b0:b0 + block], dtype=np.float32)
        c = qeps.codes(rows.reshape(-1), eps).reshape(rows.shape)
        s = scores(q, c, eps)
        bs, bi = topk(s, ids[b0:b0 + block], k)
        best_s = np.concatenate([best_s, bs], axis=1)
        best_i = np.concatenate([best_i, bi], axis=1)
        keep = best_i >= 0
        ms = np.where(keep, best_s, -np.inf)
        out_s = np.full((nq, k), -np.inf)
        out_i = np.full((nq, k), -1, dtype=np.int64)
        for j in range(nq):
            valid = np.nonzero(keep[j])[0]
            order = valid[np.lexsort((best_i[j, valid], -ms[j, valid]))][:k]
            out_s[j, :order.size] = ms[j, order]
            out_i[j, :order.size] = best_i[j, order]
        best_s, best_i = out_s, out_i
    return best_s, best_i, bound(q, eps)


def certify(q, codes_rows, ids, eps: float, k: int, delta_hat: float):
    """Rank-invariance certificate (Appendix "Rank invariance, in full") on the
    exact dequantized scores: query j's top-k cannot change when every score
    moves by at most beta_j + ||q_j||_2 delta_hat iff the margin between ranks
    k and k+1 exceeds twice that (a store with at most k records always
    qualifies).  Returns (flags bool[nq], margins float64[nq], thresholds)."""
    s = scores(q, codes_rows, eps)
    ts, _ = topk(s, ids, k + 1)
    q64 = np.asarray(q, dtype=np.float32).astype(np.float64)
    thr = 2.0 * (bound(q, eps) + np.sqrt(np.sum(q64 * q64, axis=1)) * float(delta_hat))
    margin = np.where(np.isfinite(ts[:, k]), ts[:, k - 1] - ts[:, k], np.inf)
    return margin > thr, margin, thr
