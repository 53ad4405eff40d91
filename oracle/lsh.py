"""Oracle for banded candidate generation over Q_eps codes -- test
infrastructure only.

Paper, Section 2.2 ("Three layers", L1) and Algorithm "admit": each arrival is
quantized coordinatewise with Q_eps, the code vector is divided into bands, and
records sharing a band are the candidates; every candidate is verified in full
precision and the lowest-indexed verified one is the representative; a kept
arrival's bands are added to the index.  Appendix "Band width and quantizer
step": the band width r and the step (eps = rel * sigma) set recall against the
exhaustive pair set; at full recall the result is exhaustive greedy.

Readings taken where the paper is silent:
  * bands are the consecutive coordinate ranges [b r, (b + 1) r), r dividing
    the dimension; a band of two records "matches" iff their r codes are equal
    (a digest is only a way to find equal bands, so hash collisions never make
    candidates);
  * codes are those of oracle.qeps at the band step eps_band (round half to
    even of the exact quotient);
  * the index holds retained records only (Algorithm "admit"), so candidates of
    arrival i are the retained records with id < i sharing a band;
  * the verification is the exact predicate of oracle.dedup.
"""
from __future__ import annotations

import numpy as np

from oracle import dedup, qeps


def band_keys(codes_rows, r: int):
    """Per row, the tuple of its bands' codes (hashable band contents)."""
    c = np.asarray(codes_rows, dtype=np.int64)
    n, d = c.shape
    assert d % r == 0
    nb = d // r
    return [[(b, c[i, b * r:(b + 1) * r].tobytes()) for b in range(nb)] for i in range(n)]


def greedy_lsh(x, tau: float, eps_band: float, r: int):
    """Algorithm "admit" with banded candidates.  Returns rep (global id of the
    representative, -1 kept), the kept ids, delta_hat, the number of candidate
    pairs (distinct (arrival, retained record) pairs sharing a band) and the
    number of pairs verified within delta."""
    x = np.asarray(x, dtype=np.float32)
    n, d = x.shape
    codes = qeps.codes(x.reshape(-1), eps_band).reshape(n, d)
    keys = band_keys(codes, r)
    index: dict = {}
    rep = np.full(n, -1, dtype=np.int64)
    kept = []
    dhat = 0.0
    n_cand = 0
    n_within = 0
    for i in range(n):
        cand = set()
        for k in keys[i]:
            cand.update(index.get(k, ()))
        n_cand += len(cand)
        hit = -1
        for y in sorted(cand):
            if dedup.within(x[i], x[y], tau):
                n_within += 1
                if hit < 0:
                    hit = y
        if hit >= 0:
            rep[i] = hit
            dhat = max(dhat, dedup.dist(x[i], x[hit]))
        else:
            kept.append(i)
            for k in keys[i]:
                index.setdefault(k, []).append(i)
    return dict(rep=rep, kept=np.array(kept, dtype=np.int64), delta_hat=dhat,
                n_candidates=n_cand, n_within=n_within)
