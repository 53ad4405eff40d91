"""GPU parity of dequant-fused top-k scoring against the oracle: scores within
1e-5 of the oracle's binary64 scores, ids equal except where the oracle's own
scores are within twice the tolerance of each other, bound eps*||q||_1."""
import numpy as np
import pytest

import synth
from oracle import dedup, qeps, score

pytestmark = pytest.mark.gpu
TOL = 1e-5


def _dev(a):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def _compare(gs, gi, codes_rows, ids, q, eps, k, tol=TOL):
    """gs/gi: GPU top-k.  Every returned id must be a stored id whose oracle
    score is within tol of the GPU score; the returned set must be a valid
    top-k: each GPU score >= the oracle's k-th score - 2 tol."""
    S = score.scores(q, codes_rows, eps)
    ts, ti = score.topk(S, ids, k)
    pos = {int(v): i for i, v in enumerate(ids.tolist())}
    worst = 0.0
    for j in range(q.shape[0]):
        nvalid = min(k, len(ids))
        assert np.all(gi[j, nvalid:] == -1)
        row = [pos[int(v)] for v in gi[j, :nvalid]]
        assert len(set(row)) == nvalid
        err = np.abs(gs[j, :nvalid].astype(np.float64) - S[j, row])
        worst = max(worst, float(err.max()) if nvalid else 0.0)
        assert np.all(err <= tol), (j, err.max())
        assert np.all(S[j, row] >= ts[j, nvalid - 1] - 2 * tol)
        # positions where the oracle order is separated by more than 2 tol agree
        gap_ok = np.ones(nvalid, bool)
        sj = np.concatenate([[np.inf], ts[j, :nvalid], [ts[j, nvalid] if nvalid < k else -np.inf]])
        for p in range(nvalid):
            gap_ok[p] = (sj[p] - sj[p + 1] > 2 * tol) and (sj[p + 1] - sj[p + 2] > 2 * tol)
        assert np.array_equal(gi[j, :nvalid][gap_ok], ti[j, :nvalid][gap_ok])
    return worst


def _store_from_rows(lam, x, tau=1.0, spare=0):
    s = lam.Store(x.shape[1], tau, x.shape[0] + spare)
    xd = _dev(x)
    for b0 in range(0, x.shape[0], 4096):
        s.ingest(xd[b0:b0 + 4096])
    return s


def test_tiny_end_to_end(lam):
    t = synth.tiny_ingest()
    x, tau, eps, k, q = t["x"], t["tau"], t["eps"], t["k"], t["q"]
    ref = dedup.greedy(x, tau)
    kept = ref["kept"]
    s = lam.Store(x.shape[1], tau, x.shape[0])
    xd = _dev(x)
    for b0 in range(0, x.shape[0], 1024):
        s.ingest(xd[b0:b0 + 1024])
    p = s.quantize(eps)
    codes_ref = qeps.codes(x[kept], eps)
    plan = qeps.plan(eps, float(np.abs(x[kept]).max()))
    assert p.bits == plan["bits"]
    assert np.array_equal(s.codes().cpu().numpy().view(np.uint32), qeps.pack(codes_ref, p.bits))
    gs, gi, gb = s.score_topk(_dev(q), k)
    worst = _compare(gs.cpu().numpy(), gi.cpu().numpy(), codes_ref.reshape(kept.size, -1), kept, q, eps, k)
    beta = score.bound(q, eps)
    gbn = gb.cpu().numpy().astype(np.float64)
    assert np.all(gbn >= beta) and np.all(gbn - beta <= np.spacing(gbn.astype(np.float32)))
    print(f"max |score - oracle| = {worst:.3g}")


@pytest.mark.parametrize("k", [1, 10, 16, 17, 50, 64])
@pytest.mark.parametrize("n", [5, 300, 1000])
def test_ragged_sizes_and_k(lam, k, n):
    rng = np.random.default_rng(n * 100 + k)
    x = synth.unit_rows(rng, n, 96).astype(np.float32)
    q = synth.unit_rows(rng, 37, 96).astype(np.float32)
    s = _store_from_rows(lam, x)
    s.quantize(1e-3, absmax=1.0)
    gs, gi, _ = s.score_topk(_dev(q), k)
    c = qeps.codes(x, 1e-3).reshape(n, -1)
    _compare(gs.cpu().numpy(), gi.cpu().numpy(), c, np.arange(n), q, 1e-3, k)


def test_duplicate_rows_tie_break_by_id(lam):
    rng = np.random.default_rng(2)
    base = synth.unit_rows(rng, 40, 64).astype(np.float32)
    x = np.concatenate([base, base + np.float32(0.0)])   # exact copies, later ids
    s = lam.Store(64, 1.0, 80)
    # tau = 1 merges exact copies; keep them by ingesting a slightly moved copy
    x[40:, 0] += np.float32(1e-2)
    s.ingest(_dev(x))
    s.quantize(0.02, absmax=1.0)     # coarse step: moved copies share codes
    c = qeps.codes(x, 0.02).reshape(80, -1)
    q = synth.unit_rows(rng, 8, 64).astype(np.float32)
    gs, gi, _ = s.score_topk(_dev(q), 20)
    _compare(gs.cpu().numpy(), gi.cpu().numpy(), c, np.arange(80), q, 0.02, 20)


def test_invalid_query_rows(lam):
    rng = np.random.default_rng(3)
    x = synth.unit_rows(rng, 200, 64).astype(np.float32)
    s = _store_from_rows(lam, x)
    s.quantize(1e-3)
    q = synth.unit_rows(rng, 4, 64).astype(np.float32)
    q[2, 5] = np.inf
    gs, gi, gb = s.score_topk(_dev(q), 5)
    gs, gi, gb = gs.cpu().numpy(), gi.cpu().numpy(), gb.cpu().numpy()
    assert np.all(np.isnan(gs[2])) and np.all(gi[2] == -1) and np.isnan(gb[2])
    assert np.all(gi[[0, 1, 3]] >= 0)


def test_state_errors(lam):
    rng = np.random.default_rng(4)
    x = synth.unit_rows(rng, 50, 64).astype(np.float32)
    s = _store_from_rows(lam, x, spare=10)
    with pytest.raises(lam.LamError) as e:
        s.score_topk(_dev(x[:2]), 3)
    assert e.value.name == "LAM_ESTATE"
    s.quantize(1e-3)
    s.ingest(_dev(synth.unit_rows(rng, 5, 64).astype(np.float32)))
    with pytest.raises(lam.LamError) as e:
        s.score_topk(_dev(x[:2]), 3)
    assert e.value.name == "LAM_ESTATE"
    s.quantize(1e-3)
    with pytest.raises(lam.LamError) as e:
        s.score_topk(_dev(x[:2]), 65)
    assert e.value.name == "LAM_EINVAL"


def test_corpus_all_queries(lam):
    """361,802 clustered rows quantized at eps = 1e-3, 4,096 queries, top-10:
    the benchmark's launch configuration; every query against the oracle's
    scores of the whole store (in blocks of 256 queries)."""
    cfg = synth.corpus_retrieval()
    x, q, eps, k = cfg["x"], cfg["q"], cfg["eps"], cfg["k"]
    s = _store_from_rows(lam, x)
    p = s.quantize(eps)
    gs, gi, gb = s.score_topk(_dev(q), k)
    gs, gi, gb = gs.cpu().numpy(), gi.cpu().numpy(), gb.cpu().numpy()
    c = qeps.codes(x, eps).reshape(x.shape[0], -1).astype(np.float64)
    assert p.bits == qeps.plan(eps, float(np.abs(x).max()))["bits"]
    ids = np.arange(x.shape[0])
    worst = 0.0
    for j0 in range(0, q.shape[0], 256):
        sl = slice(j0, j0 + 256)
        worst = max(worst, _compare(gs[sl], gi[sl], c, ids, q[sl], eps, k))
    beta = score.bound(q, eps)
    gbn = gb.astype(np.float64)
    assert np.all(gbn >= beta) and np.all(gbn - beta <= np.spacing(gbn.astype(np.float32)))
    print(f"corpus, {q.shape[0]} queries: max |score - oracle| = {worst:.3g}")


@pytest.mark.parametrize("k,d", [(10, 64), (50, 64), (10, 768), (50, 768)])
def test_two_pass_and_overflow_fallback(lam, k, d):
    """A store beyond the sample size takes the threshold/candidate plan (at
    D = 768 its filter pass runs on the screen's pipeline); an all-zero query
    ties every row at score 0, overflows its candidate buffer and must come
    back exact from the fallback (the k lowest ids)."""
    rng = np.random.default_rng(11)
    n = 20000
    x = synth.unit_rows(rng, n, d).astype(np.float32)
    s = _store_from_rows(lam, x)
    s.quantize(1e-3)
    q = synth.unit_rows(rng, 40, d).astype(np.float32)
    q[[3, 17]] = 0.0
    gs, gi, gb = s.score_topk(_dev(q), k)
    gs, gi = gs.cpu().numpy(), gi.cpu().numpy()
    assert np.all(gi[3] == np.arange(k)) and np.all(gs[3] == 0.0)
    assert np.all(gi[17] == np.arange(k))
    c = qeps.codes(x, 1e-3).reshape(n, -1)
    keep = [j for j in range(q.shape[0]) if j not in (3, 17)]
    _compare(gs[keep], gi[keep], c, np.arange(n), q[keep], 1e-3, k)


@pytest.mark.parametrize("k,d", [(17, 64), (50, 64), (64, 64), (50, 768)])
def test_two_pass_ties_broken_by_id(lam, k, d):
    """Exactly equal scores at the k-th place in the two-pass plan: 20,000
    rows are 40 copies of 500 vectors, the copies moved by less than the code
    step so that all copies of a vector share its codes; every query's top-k
    cuts through a group of equal scores, which must be taken in id order."""
    rng = np.random.default_rng(12)
    base = synth.unit_rows(rng, 500, d)
    x = np.tile(base, (40, 1))
    x[:, 0] += np.repeat(np.arange(40), 500) * 1e-6     # distinct rows, identical codes at eps = 0.02
    x = x.astype(np.float32)
    s = _store_from_rows(lam, x)
    s.quantize(0.02, absmax=1.0)
    c = qeps.codes(x, 0.02).reshape(x.shape[0], -1)
    assert np.array_equal(c[:500], c[500:1000])
    q = synth.unit_rows(rng, 24, d).astype(np.float32)
    gs, gi, _ = s.score_topk(_dev(q), k)
    S = score.scores(q, c, 0.02)
    ts, ti = score.topk(S, np.arange(x.shape[0]), k)
    assert np.array_equal(gi.cpu().numpy(), ti)
    assert np.all(np.abs(gs.cpu().numpy().astype(np.float64) - ts) <= TOL)


def test_rank_invariance_certificate(lam):
    """Certified queries have an exact margin above 2 (beta + ||q|| delta_hat)
    (soundness); queries whose exact margin clears that by more than the
    float32 error bound are certified; the top-k equals lam_score_topk's."""
    import torch
    rng = np.random.default_rng(21)
    d, n = 768, 3000
    x = synth.unit_rows(rng, n, d).astype(np.float32)
    x[1500:1600] = synth.near_dups(rng, x[:100].astype(np.float64)).astype(np.float32)
    tau, eps = 0.95, 1e-3
    s = lam.Store(d, tau, n)
    s.ingest(_dev(x))
    info = s.info()
    p = s.quantize(eps)
    kept = s.ids().cpu().numpy()
    codes = qeps.codes(x[kept], eps).reshape(kept.size, d)
    q = np.concatenate([synth.unit_rows(rng, 40, d).astype(np.float32), x[kept[rng.choice(kept.size, 24)]]])
    qd = _dev(q)
    u = 2.0 ** -24
    kappa = 1.01 * (2.0 ** -22 + 2 * d * u / (1 - 2 * d * u) + 2.0 ** -23)
    e = kappa * np.abs(q.astype(np.float64)).sum(axis=1) * (p.absmax + eps)
    n_cert = 0
    for k in (1, 5, 20):
        gs, gi, gb, gc, gm = s.score_topk_certified(qd, k)
        ps, pi, pb = s.score_topk(qd, k)
        assert torch.equal(gi, pi) and torch.equal(gs, ps) and torch.equal(gb, pb)
        flags, margin, thr = score.certify(q, codes, kept, eps, k, info.delta_hat_run)
        gc = gc.cpu().numpy()
        assert np.all(margin[gc] > thr[gc])                         # sound
        assert np.all(gc[margin > thr + 2 * e + 4 * TOL])           # complete away from the error band
        gmn = gm.cpu().numpy().astype(np.float64)
        fin = np.isfinite(margin)
        assert np.all(np.abs(gmn[fin] - margin[fin]) <= 2 * TOL)
        n_cert += int(gc.sum())
    assert 0 < n_cert < 3 * q.shape[0]


def test_certificate_small_store_and_invalid_rows(lam):
    import torch
    rng = np.random.default_rng(22)
    x = synth.unit_rows(rng, 3, 64).astype(np.float32)
    s = lam.Store(64, 1.0, 8)
    s.ingest(_dev(x))
    s.quantize(1e-3)
    q = synth.unit_rows(rng, 4, 64).astype(np.float32)
    q[2, 5] = np.nan
    _, gi, gb, gc, gm = s.score_topk_certified(_dev(q), 3)
    assert gc.cpu().tolist() == [True, True, False, True]
    assert torch.isinf(gm[[0, 1, 3]]).all() and torch.isnan(gm[2])
    for k in (0, 64):
        with pytest.raises(lam.LamError):
            s.score_topk_certified(_dev(q), k)


def _flip_store(n=6000, d=64, group=0):
    """Rows whose hi-only scores order differently from their exact scores:
    with eps = 2^-11 (code step 2^-10) row 100 has codes 1000 on coordinates
    0-3 and row 200 codes 1000, 1000, 1000, 1001 on coordinates 4-7.  The query
    is 1 + 2^-11 on coordinates 0-3 and 1 on 4-7: scaled by 2^14 its first four
    entries are 2^14 + 8, which the fp16 hi part rounds to 2^14 (a tie, to
    even).  Exactly, row 100 scores 4000 (1 + 2^-11) 2^-10 > 4001 2^-10 (row
    200); from the hi part alone row 200 is ahead.  The other rows are random
    unit rows on coordinates 8 and up (score 0); `group` more rows carry row
    200's codes exactly (scores tied with it)."""
    rng = np.random.default_rng(31)
    x = np.zeros((n, d), np.float64)
    x[:, 8:] = synth.unit_rows(rng, n, d - 8)
    x[100] = 0.0
    x[100, 0:4] = 1000 * 2.0 ** -10
    r2 = np.zeros(d)
    r2[4:8] = np.array([1000, 1000, 1000, 1001]) * 2.0 ** -10
    x[200] = r2
    for i in range(group):                       # distinct rows, same codes: moved on a coordinate
        x[300 + i] = r2                          # the query ignores, by less than half a step
        x[300 + i, 8] = (i + 1) * 1e-7
    q = np.zeros((3, d))
    q[:, 0:4] = 1.0 + 2.0 ** -11
    q[:, 4:8] = 1.0
    q[1] = 0.0
    q[1, 8:] = synth.unit_rows(rng, 1, d - 8)[0]
    q[2, 0:4] = 1.0                              # no rounding in the hi part
    return x.astype(np.float32), q.astype(np.float32)


@pytest.mark.parametrize("k,d", [(1, 64), (2, 64), (10, 64), (1, 768), (2, 768)])
def test_rescoring_restores_the_exact_order(lam, k, d):
    """The two-pass plan filters and selects on hi-only scores, then rescores
    the candidates near the k-th: the exact order must come back (row 100
    before row 200), the scores within tolerance of the oracle."""
    x, q = _flip_store(d=d)
    s = _store_from_rows(lam, x)
    eps = 2.0 ** -11
    p = s.quantize(eps)
    c = qeps.codes(x, eps).reshape(x.shape[0], -1)
    assert c[100, 0] == 1000 and c[200, 7] == 1001 and p.bits <= 12
    gs, gi, _ = s.score_topk(_dev(q), k)
    gs, gi = gs.cpu().numpy(), gi.cpu().numpy()
    assert gi[0, 0] == 100 and (k == 1 or gi[0, 1] == 200)
    assert gi[2, 0] == 200                       # 4000 < 4001 when nothing is lost to rounding
    _compare(gs, gi, c, np.arange(x.shape[0]), q, eps, k)


@pytest.mark.parametrize("d", [64, 768])
def test_rescoring_cap_falls_back_exactly(lam, d):
    """600 rows tied with row 200 (identical codes) sit within the rescoring
    band of query 2 (row 200's codes win it): more than the rescoring cap, so
    the query is redone by the exact pass; the k best are the tied rows in id
    order."""
    x, q = _flip_store(d=d, group=600)
    s = _store_from_rows(lam, x)
    eps = 2.0 ** -11
    s.quantize(eps)
    c = qeps.codes(x, eps).reshape(x.shape[0], -1)
    assert all(np.array_equal(c[200], c[300 + i]) for i in (0, 299, 599))
    gs, gi, _ = s.score_topk(_dev(q), 10)
    gi = gi.cpu().numpy()
    assert np.array_equal(gi[2], np.concatenate([[200], np.arange(300, 309)]))
    _compare(gs.cpu().numpy(), gi, c, np.arange(x.shape[0]), q, eps, 10)


@pytest.mark.parametrize("near", [600, 2000])
@pytest.mark.parametrize("k,d", [(1, 64), (10, 64), (16, 768)])
def test_selection_over_many_candidates(lam, near, k, d):
    """The store's first 4,096 rows (the threshold plan's sample) are random
    directions; after them each query has `near` rows whose cosines with it
    run from 0.5 to 0.99, all above the sample's k-th score, so the filter
    pass hands the selection about `near` candidates per query (several per
    lane of its per-lane lists), and the top-k must match the oracle."""
    rng = np.random.default_rng(21)
    nq = 4
    q = synth.unit_rows(rng, nq, d)
    parts = [synth.unit_rows(rng, 4096, d)]
    for j in range(nq):
        parts.append(synth.members(rng, np.repeat(q[j:j + 1], near, axis=0), np.linspace(0.5, 0.99, near)))
    x = np.concatenate(parts).astype(np.float32)
    n = x.shape[0]
    s = _store_from_rows(lam, x)
    eps = 1e-3
    s.quantize(eps)
    assert s.info().size == n
    c = qeps.codes(x, eps).reshape(n, -1)
    S = score.scores(q.astype(np.float32), c, eps)
    assert np.all((S[:, 4096:] >= 0.49).sum(1) >= near)
    gs, gi, _ = s.score_topk(_dev(q.astype(np.float32)), k)
    _compare(gs.cpu().numpy(), gi.cpu().numpy(), c, np.arange(n), q.astype(np.float32), eps, k)
