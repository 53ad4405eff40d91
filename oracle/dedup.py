"""Oracle for the epsilon error-bounded near-duplicate test -- test
infrastructure only.

Paper:
  * Section 2.1 ("The proximity relation"), Eq. (identity): for unit vectors
    ||a - b||^2 = 2 - 2 cos(a, b); merging at cos >= t is ||a - b|| <= delta with
    delta = sqrt(2 - 2t).
  * Section 2.3, Algorithm "admit": arrivals are taken in order; an arrival is
    dropped iff some retained record y satisfies ||e_j - e_y|| <= delta, and its
    representative is the lowest-indexed such y; otherwise it is appended to the
    retained set.  The measured bound delta_hat is the largest distance used.
  * Appendix "Implementation details", Algorithm "batch": the same relation and
    witness over a finished sequence; the outputs coincide with the online form.
  * Appendix "Representative selection": greedy first-occurrence, compared
    directly with retained records (the relation is not transitive).
  * Appendix "The measured bound": delta_hat = max ||x - pi(x)||, zero when no
    substitution happens.

Readings (where the paper leaves a choice):
  * the predicate is the squared l2 form  sum_d (a_d - b_d)^2 <= 2 - 2 tau,
    evaluated on the float32 inputs as exact reals, inclusive at equality;
    tau is a binary64 value and 2 - 2 tau is taken as an exact rational;
  * candidates are exhaustive (every retained record), which is what banded
    candidates reproduce at full recall (Appendix "Band width and quantizer
    step: the full grid");
  * ids are 0-based arrival ordinals over the whole stream; rep = -1 marks a
    kept arrival; the retained set is append-only;
  * inputs are used exactly as given (no re-normalisation).
"""
from __future__ import annotations

import hashlib
import math
from fractions import Fraction

import numpy as np

_SCALE = 2.0 ** 149          # every finite float32 times 2^149 is an integer


def delta2(tau: float) -> Fraction:
    """delta^2 = 2 - 2 tau, exact."""
    return 2 - 2 * Fraction(float(tau))


def delta(tau: float) -> float:
    """delta = sqrt(2 - 2 tau) (Eq. identity)."""
    return math.sqrt(2.0 - 2.0 * float(tau))


def _as_ints(v) -> list:
    return [int(t) for t in (np.asarray(v, dtype=np.float32).astype(np.float64) * _SCALE).tolist()]


def d2_exact(a, b) -> Fraction:
    """sum_d (a_d - b_d)^2 on exact reals, for float32 rows a and b."""
    ia, ib = _as_ints(a), _as_ints(b)
    s = sum((p - q) * (p - q) for p, q in zip(ia, ib))
    return Fraction(s, 1 << 298)


def within(a, b, tau: float) -> bool:
    """The merge predicate ||a - b||_2 <= delta, exactly."""
    return d2_exact(a, b) <= delta2(tau)


def dist(a, b) -> float:
    """||a - b||_2 in binary64 (correctly rounded sum of the squared
    differences, each difference exact in binary64 for float32 inputs within
    2^29 of each other)."""
    d = np.asarray(a, np.float64) - np.asarray(b, np.float64)
    return math.sqrt(math.fsum((d * d).tolist()))


# ----------------------------------------------------------------- naive form
def greedy_naive(x, tau: float):
    """Algorithm "admit" with exhaustive candidates, literally: every arrival is
    compared with every retained record in increasing index order, on exact
    rationals.  Pure Python; meant for a few hundred rows."""
    x = np.asarray(x, dtype=np.float32)
    d2t = delta2(tau)
    kept: list[int] = []
    rep = np.full(x.shape[0], -1, dtype=np.int64)
    dhat = 0.0
    ints = [_as_ints(r) for r in x]
    lim = d2t * (1 << 298)
    for i in range(x.shape[0]):
        for y in kept:
            s = sum((p - q) * (p - q) for p, q in zip(ints[i], ints[y]))
            if s <= lim:
                rep[i] = y
                dhat = max(dhat, dist(x[i], x[y]))
                break
        else:
            kept.append(i)
    return dict(rep=rep, kept=np.array(kept, dtype=np.int64), delta_hat=dhat)


# ----------------------------------------------------------------- main form
class Greedy:
    """Streaming form of Algorithm "admit" with exhaustive candidates.

    For each arrival, in order, the squared distances to all retained rows are
    evaluated in binary64 (norms plus one matrix-vector product); any distance
    within a rounding margin of delta^2 is re-decided on exact rationals.  The
    first retained row (lowest index) inside delta is the representative.

    ``block`` only groups the matrix-vector products of consecutive arrivals
    against the rows retained before the group into one matrix product; rows
    retained inside the group are compared one by one, in order.  The outputs
    do not depend on it (checked by the tests).
    """

    def __init__(self, dim: int, tau: float, capacity: int):
        self.tau = float(tau)
        self.d2t = delta2(tau)
        self.d2f = float(self.d2t)
        self.rows = np.empty((capacity, dim), dtype=np.float64)   # retained rows
        self.raw = np.empty((capacity, dim), dtype=np.float32)
        self.norm2 = np.empty(capacity, dtype=np.float64)
        self.ids = np.empty(capacity, dtype=np.int64)
        self.m = 0
        self.n_seen = 0
        self.delta_hat = 0.0
        self.n_exact = 0

    # Rounding margin: |fl(na + nb - 2 a.b) - d^2| <= (D + 3) u (na + nb + 2|a||b|)
    # <= 2 (D + 3) u (na + nb), and 1e-11 (na + nb) covers D <= 10^4.

    def _first_hit(self, xi32, xi, ni, d2row, ids):
        """Lowest position whose exact distance is within delta, else -1."""
        marg = 1e-11 * np.maximum(1.0, ni + self.norm2[:d2row.size])
        cand = np.nonzero(d2row <= self.d2f + marg)[0]
        for c in cand.tolist():
            if d2row[c] < self.d2f - marg[c]:
                return c
            self.n_exact += 1
            if d2_exact(xi32, self.raw[c]) <= self.d2t:
                return c
        return -1

    def ingest(self, x, block: int = 256):
        x = np.asarray(x, dtype=np.float32)
        n = x.shape[0]
        rep = np.full(n, -1, dtype=np.int64)
        max_cos = np.full(n, -np.inf, dtype=np.float64)
        x64 = x.astype(np.float64)
        nx = np.einsum("ij,ij->i", x64, x64)
        dh_call = 0.0
        for b0 in range(0, n, max(1, block)):
            b1 = min(n, b0 + max(1, block))
            m0 = self.m
            g = x64[b0:b1] @ self.rows[:m0].T if m0 else np.zeros((b1 - b0, 0))
            for i in range(b0, b1):
                gid = self.n_seen + i
                # retained before the block: one row of the matrix product
                dots = g[i - b0]
                # retained inside the block so far: direct products
                if self.m > m0:
                    dots = np.concatenate([dots, self.rows[m0:self.m] @ x64[i]])
                d2row = nx[i] + self.norm2[:self.m] - 2.0 * dots
                if dots.size:
                    max_cos[i] = float(np.max(dots))
                c = self._first_hit(x[i], x64[i], nx[i], d2row, self.ids[:self.m])
                if c >= 0:
                    rep[i] = self.ids[c]
                    d = dist(x[i], self.raw[c])
                    dh_call = max(dh_call, d)
                else:
                    k = self.m
                    self.rows[k] = x64[i]
                    self.raw[k] = x[i]
                    self.norm2[k] = nx[i]
                    self.ids[k] = gid
                    self.m += 1
        self.n_seen += n
        self.delta_hat = max(self.delta_hat, dh_call)
        return dict(rep=rep, max_cos=max_cos, delta_hat_call=dh_call,
                    delta_hat_run=self.delta_hat, n_kept=int(np.count_nonzero(rep < 0)))

    @property
    def kept_ids(self):
        return self.ids[:self.m].copy()


def greedy(x, tau: float, batch: int | None = None, block: int = 256):
    """Whole-stream greedy; ``batch`` splits the stream into separate ingest
    calls (outputs are identical for any split)."""
    x = np.asarray(x, dtype=np.float32)
    g = Greedy(x.shape[1], tau, x.shape[0])
    reps, cos = [], []
    bs = x.shape[0] if not batch else batch
    for s in range(0, x.shape[0], max(1, bs)):
        r = g.ingest(x[s:s + bs], block=block)
        reps.append(r["rep"])
        cos.append(r["max_cos"])
    rep = np.concatenate(reps) if reps else np.zeros(0, np.int64)
    return dict(rep=rep, kept=g.kept_ids, delta_hat=g.delta_hat,
                max_cos=np.concatenate(cos) if cos else np.zeros(0),
                n_exact=g.n_exact)


def decide_one(x, i: int, kept_before, tau: float):
    """The decision for arrival i given the retained set at its arrival
    (ascending ids): the lowest retained id within delta, else -1.  Used to
    check sampled decisions of a large stream one by one."""
    x = np.asarray(x, dtype=np.float32)
    kb = np.asarray(kept_before, dtype=np.int64)
    if kb.size == 0:
        return -1
    xi = x[i].astype(np.float64)
    rows = x[kb].astype(np.float64)
    rn = np.einsum("ij,ij->i", rows, rows)
    d2row = rn + xi @ xi - 2.0 * (rows @ xi)
    d2f = float(delta2(tau))
    # the binary64 distance is within 1e-11 (||x_i||^2 + ||y||^2) of the exact
    # one (far more than its rounding error at any dim this library takes);
    # the same margin decides which rows are candidates and which are
    # definitely inside, the rest take the exact test
    tol = 1e-11 * np.maximum(1.0, xi @ xi + rn)
    for c in np.nonzero(d2row <= d2f + tol)[0].tolist():
        if d2row[c] < d2f - tol[c] or within(x[i], x[kb[c]], tau):
            return int(kb[c])
    return -1


def decide_many(x, samples, kept, tau: float, block: int = 1 << 16):
    """decide_one for several arrivals at once: for each i in `samples`, the
    lowest id y in `kept` (ascending ids of the retained set) with y < i and
    x[y] within delta of x[i], else -1.  The retained rows are visited in
    ascending blocks, so the first qualifying id found is the lowest; the
    predicate is decided as in decide_one (binary64 distance, exact integers
    within 1e-11 of delta^2).  For checking sampled decisions of a stream too
    large for `greedy`."""
    x = np.asarray(x, dtype=np.float32)
    kept = np.asarray(kept, dtype=np.int64)
    samples = np.asarray(samples, dtype=np.int64)
    d2f = float(delta2(tau))
    xs = x[samples].astype(np.float64)
    sn = np.einsum("ij,ij->i", xs, xs)
    best = np.full(samples.size, -1, dtype=np.int64)
    for b0 in range(0, kept.size, block):
        ids = kept[b0:b0 + block]
        open_ = (best < 0) & (samples > ids[0])
        if not open_.any():
            continue
        rows = x[ids].astype(np.float64)
        rn = np.einsum("ij,ij->i", rows, rows)
        cols = np.nonzero(open_)[0]
        d2 = rn[:, None] + sn[None, cols] - 2.0 * (rows @ xs[cols].T)
        for c, sidx in enumerate(cols):
            i = int(samples[sidx])
            tol = 1e-11 * np.maximum(1.0, sn[sidx] + rn)   # as in decide_one, per row
            for r in np.nonzero((ids < i) & (d2[:, c] <= d2f + tol))[0].tolist():
                if d2[r, c] < d2f - tol[r] or within(x[i], x[ids[r]], tau):
                    best[sidx] = int(ids[r])
                    break
    return best


def removal_ceiling(x, tau: float):
    """Theorem "removal ceiling" and Corollary "measured bracket": greedy at
    radius delta (tau) and at radius 2 delta (tau' = 4 tau - 3; exact in
    binary64 for tau in [1/2, 1]).  Returns the counts, the attained removal
    1 - |R(delta)|/n, the ceiling 1 - |R(2 delta)|/n and the bracket
    (log2 |R(2 delta)|, log2 |R(delta)|)."""
    tau2 = 4.0 * tau - 3.0
    assert Fraction(tau2) == 4 * Fraction(tau) - 3
    n = np.asarray(x).shape[0]
    r1 = greedy(x, tau)
    r2 = greedy(x, tau2)
    k1 = int(np.count_nonzero(r1["rep"] < 0))
    k2 = int(np.count_nonzero(r2["rep"] < 0))
    return dict(n=n, kept=k1, kept_2delta=k2, tau=tau, tau_2delta=tau2, removal=1.0 - k1 / n,
                ceiling=1.0 - k2 / n, bits_lo=math.log2(k2), bits_hi=math.log2(k1),
                kept_ids=r1["kept"], kept_ids_2delta=r2["kept"])


def deletion_digest(rep) -> str:
    """SHA-256 over the (id, rep) pairs of dropped arrivals, little-endian
    int64, in id order (the deletion-set digest of Section "Determinism")."""
    rep = np.asarray(rep, dtype=np.int64)
    ids = np.nonzero(rep >= 0)[0].astype("<i8")
    pairs = np.stack([ids, rep[ids].astype("<i8")], axis=1) if ids.size else np.zeros((0, 2), "<i8")
    return hashlib.sha256(pairs.tobytes()).hexdigest()
