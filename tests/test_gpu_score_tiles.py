"""GPU parity of the scoring filter pass on its 256 x 256 tile (launches of
at least 1,024 such tiles): odd and even code widths, D = 768 and 1,024, a
ragged query count, an all-zero query that overflows into the exact fallback,
and exact ties at the k-th place taken in id order."""
import numpy as np
import pytest

import synth
from oracle import qeps, score
from test_gpu_score import TOL, _compare, _dev, _store_from_rows

pytestmark = pytest.mark.gpu


def _large(nq, n):
    """The launch holds enough 256 x 256 tiles for the large filter tile."""
    return ((nq + 255) // 256) * ((n + 255) // 256) >= 1024


@pytest.mark.parametrize("k", [10, 50])
def test_large_filter_odd_width(lam, k):
    """90,000 unit rows at D = 768, eps = 5e-4 (9-bit codes), 600 queries:
    half near store rows, one all zero."""
    rng = np.random.default_rng(41)
    n, d, nq = 90000, 768, 600
    assert _large(nq, n)
    x = synth.unit_rows(rng, n, d).astype(np.float32)
    s = _store_from_rows(lam, x)
    p = s.quantize(5e-4)
    assert p.bits % 2 == 1
    q = np.concatenate([synth.unit_rows(rng, nq // 2, d),
                        synth.members(rng, x[rng.choice(n, nq // 2)].astype(np.float64),
                                      rng.uniform(0.9, 0.99, nq // 2))]).astype(np.float32)
    q[3] = 0.0
    gs, gi, _ = s.score_topk(_dev(q), k)
    gs, gi = gs.cpu().numpy(), gi.cpu().numpy()
    assert np.all(gi[3] == np.arange(k)) and np.all(gs[3] == 0.0)
    keep = [j for j in range(nq) if j != 3]
    c = qeps.codes(x, 5e-4).reshape(n, -1)
    _compare(gs[keep], gi[keep], c, np.arange(n), q[keep], 5e-4, k)


def test_large_filter_d1024_even_width(lam):
    """70,000 rows at D = 1,024, codes of 10 bits (absmax 1 declared), 1,000
    queries (four query tiles, the last one ragged)."""
    rng = np.random.default_rng(42)
    n, d, nq = 70000, 1024, 1000
    assert _large(nq, n)
    x = synth.unit_rows(rng, n, d).astype(np.float32)
    s = _store_from_rows(lam, x)
    p = s.quantize(1e-3, absmax=1.0)
    assert p.bits == 10
    q = synth.unit_rows(rng, nq, d).astype(np.float32)
    gs, gi, _ = s.score_topk(_dev(q), 10)
    c = qeps.codes(x, 1e-3).reshape(n, -1)
    _compare(gs.cpu().numpy(), gi.cpu().numpy(), c, np.arange(n), q, 1e-3, 10)


@pytest.mark.parametrize("k", [10, 17])
def test_large_filter_ties_by_id(lam, k):
    """40 copies of 2,250 vectors (identical codes at eps = 0.02): the top-k
    of every query cuts through a group of equal scores, taken in id order."""
    rng = np.random.default_rng(43)
    d, nq = 768, 600
    base = synth.unit_rows(rng, 2250, d)
    x = np.tile(base, (40, 1))
    x[:, 0] += np.repeat(np.arange(40), 2250) * 1e-6
    x = x.astype(np.float32)
    n = x.shape[0]
    assert _large(nq, n)
    s = _store_from_rows(lam, x)
    s.quantize(0.02, absmax=1.0)
    c = qeps.codes(x, 0.02).reshape(n, -1)
    assert np.array_equal(c[:2250], c[2250:4500])
    q = synth.unit_rows(rng, nq, d).astype(np.float32)
    gs, gi, _ = s.score_topk(_dev(q), k)
    S = score.scores(q, c, 0.02)
    ts, ti = score.topk(S, np.arange(n), k)
    assert np.array_equal(gi.cpu().numpy(), ti)
    assert np.all(np.abs(gs.cpu().numpy().astype(np.float64) - ts) <= TOL)
