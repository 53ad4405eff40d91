"""Pins for the scoring oracle (CPU).

Checked against: brute-force sorting on tiny inputs, k = 1 as argmax, exact
rational dot products on dyadic data (where the dequantized store equals the
input), the Hoelder bound eps*||q||_1 of Appendix "Rank invariance, in full" on
every (query, record) pair, and Theorem "Score deficit" combined with the
quantization bound.
"""
from fractions import Fraction

import numpy as np
import pytest

import synth
from oracle import dedup, qeps, score


def _store(seed=0, n=300, d=64, eps=1e-3):
    rng = np.random.default_rng(seed)
    x = synth.unit_rows(rng, n, d).astype(np.float32)
    q = synth.unit_rows(rng, 20, d).astype(np.float32)
    c = qeps.codes(x, eps).reshape(n, d)
    return x, q, c, eps


def test_topk_matches_sorted_brute_force():
    x, q, c, eps = _store()
    ids = np.arange(c.shape[0], dtype=np.int64) * 3 + 5
    s = score.scores(q, c, eps)
    # plant exact ties: copy a record under a larger id
    c2 = np.concatenate([c, c[:10]])
    ids2 = np.concatenate([ids, 10_000 + np.arange(10)])
    s2 = score.scores(q, c2, eps)
    for k in (1, 3, 10, 310, 400):
        ts, ti = score.topk(s2, ids2, k)
        for j in range(q.shape[0]):
            ref = sorted(zip((-s2[j]).tolist(), ids2.tolist()))[:k]
            want_i = [i for _, i in ref] + [-1] * (k - len(ref))
            assert ti[j].tolist() == want_i
            assert np.all(np.isneginf(ts[j, len(ref):]))
    assert s.shape == (q.shape[0], c.shape[0])


def test_k1_is_argmax():
    x, q, c, eps = _store(1)
    ids = np.arange(c.shape[0], dtype=np.int64)
    s = score.scores(q, c, eps)
    _, ti = score.topk(s, ids, 1)
    assert np.array_equal(ti[:, 0], np.argmax(s, axis=1))


def test_dyadic_scores_are_exact_dot_products():
    # eps = 2^-12 and inputs on the grid 2^-11: x_hat == x, so the score is the
    # exact inner product of the raw vectors.
    rng = np.random.default_rng(2)
    eps = 2.0 ** -12
    x = (np.round(synth.unit_rows(rng, 40, 32) * 2048) / 2048).astype(np.float32)
    q = synth.unit_rows(rng, 5, 32).astype(np.float32)
    c = qeps.codes(x, eps).reshape(x.shape)
    assert np.array_equal(qeps.decode(c, eps).reshape(x.shape), x)
    s = score.scores(q, c, eps)
    for j in range(q.shape[0]):
        for y in range(0, x.shape[0], 7):
            exact = sum(Fraction(float(a)) * Fraction(float(b)) for a, b in zip(q[j], x[y]))
            assert s[j, y] == pytest.approx(float(exact), abs=1e-15)


@pytest.mark.parametrize("eps", [1e-4, 1e-3, 1e-2])
def test_hoelder_bound_every_pair(eps):
    x, q, c, _ = _store(3, eps=eps)
    s_hat = score.scores(q, c, eps)
    s_true = q.astype(np.float64) @ x.astype(np.float64).T
    beta = score.bound(q, eps)
    assert np.all(np.abs(s_true - s_hat) <= beta[:, None] * (1 + 1e-12) + 1e-15)
    # the bound is eps*||q||_1 (and not, e.g., eps*||q||_2)
    assert np.allclose(beta, eps * np.abs(q.astype(np.float64)).sum(1), rtol=0, atol=1e-17)


def test_dedup_plus_quantization_bound():
    # Theorem "Score deficit" with delta_hat, plus beta for the quantized store:
    # -beta <= max_S q.x - max_R q.x_hat <= ||q|| delta_hat + beta.
    t = synth.tiny_ingest(n=1200, dup_frac=0.2)
    x, tau, eps = t["x"], t["tau"], t["eps"]
    r = dedup.greedy(x, tau)
    kept = r["kept"]
    c = qeps.codes(x[kept], eps).reshape(kept.size, x.shape[1])
    q = t["q"]
    ts, ti, beta = score.score_topk(q, c, kept, eps, 1)
    top_s = (q.astype(np.float64) @ x.astype(np.float64).T).max(1)
    gap = top_s - ts[:, 0]
    qn = np.linalg.norm(q.astype(np.float64), axis=1)
    assert np.all(gap >= -beta - 1e-12)
    assert np.all(gap <= qn * r["delta_hat"] + beta + 1e-12)


def test_blocked_topk_matches_whole_store():
    """score_topk_blocked over float32 rows equals score_topk over their codes,
    with ties planted across block boundaries."""
    rng = np.random.default_rng(4)
    x = synth.unit_rows(rng, 200, 64).astype(np.float32)
    x[150] = x[3]            # equal scores in different blocks
    x[77] = x[40]
    q = synth.unit_rows(rng, 12, 64).astype(np.float32)
    q[5] = x[3]
    eps = 1e-3
    ids = np.arange(200, dtype=np.int64) * 2 + 1
    c = qeps.codes(x, eps).reshape(x.shape)
    for k in (1, 7, 50, 250):
        ws, wi, wb = score.score_topk(q, c, ids, eps, k)
        bs, bi, bb = score.score_topk_blocked(q, x, ids, eps, k, block=37)
        assert np.array_equal(wi, bi) and np.array_equal(ws, bs) and np.array_equal(wb, bb)


def test_certify_closed_forms():
    """A query equal to one stored row, the others orthogonal to it, has margin
    |q|^2 - 0 at k = 1: certified for small eps and delta_hat, not once
    delta_hat exceeds half the margin.  A duplicated best row has margin 0
    (never certified at k = 1); a store of at most k rows always qualifies."""
    d = 64
    x = np.eye(d, dtype=np.float32)[:10] * np.float32(0.5)
    ids = np.arange(10, dtype=np.int64)
    eps = 2.0 ** -10                       # dyadic: codes are exact, scores exact
    c = qeps.codes(x, eps).reshape(x.shape)
    q = np.zeros((1, d), np.float32)
    q[0, 3] = 1.0
    f, m, t = score.certify(q, c, ids, eps, 1, 0.0)
    assert f[0] and m[0] == 0.5 and t[0] == 2 * eps
    f, m, t = score.certify(q, c, ids, eps, 1, 0.25)
    assert not f[0] and t[0] == 2 * (eps + 0.25)
    x2 = np.concatenate([x, x[3:4]])
    c2 = qeps.codes(x2, eps).reshape(x2.shape)
    f, m, _ = score.certify(q, c2, np.arange(11), eps, 1, 0.0)
    assert not f[0] and m[0] == 0.0
    f, m, _ = score.certify(q, c[:3], ids[:3], eps, 3, 10.0)
    assert f[0] and m[0] == np.inf


def test_topk_selection_equals_the_sorted_definition():
    """topk (partition, then sort of the entries at or above the k-th score)
    gives topk_sorted's result (every row sorted by score desc, id asc), with
    ties planted at the k-th score, ids out of order and k near the row size."""
    rng = np.random.default_rng(31)
    for n, k in ((50, 10), (400, 10), (400, 64), (3000, 50), (41, 10)):
        s = np.round(rng.standard_normal((23, n)), 1)   # many exact ties
        ids = rng.permutation(10 * n)[:n]
        a = score.topk(s, ids, k)
        b = score.topk_sorted(s, ids, k)
        assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])
