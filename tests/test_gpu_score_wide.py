"""GPU parity of scoring for codes of 13 to 22 bits (the split form: each code
as c >> 11 and c & 2047 against [2^11 q, q]) against the oracle's binary64
scores of the plain codes: the same tolerance and order checks as for narrow
codes, on both scoring plans, the certificate and scoring from blocks."""
import numpy as np
import pytest

import synth
from oracle import qeps, score
from test_gpu_score import TOL, _compare, _dev, _store_from_rows

pytestmark = pytest.mark.gpu


def _eps_for_bits(absmax, b):
    """An eps whose plan for this absmax has width b (max code about 3/4 of
    the width's range, so that the high part c >> 11 spans its range too)."""
    eps = float(absmax) / (2.0 * 0.75 * 2.0 ** (b - 1))
    assert qeps.plan(eps, absmax)["bits"] == b
    return eps


def _wide_store(lam, x, b):
    s = _store_from_rows(lam, x)
    absmax = float(np.abs(x).max())
    eps = _eps_for_bits(absmax, b)
    p = s.quantize(eps)
    assert p.bits == b
    c = qeps.codes(x, eps).reshape(x.shape[0], -1)
    assert np.abs(c).max() >= 2 ** (b - 2)      # the codes reach the width's upper half
    return s, eps, c


@pytest.mark.parametrize("b", [13, 16, 22])
@pytest.mark.parametrize("k,d", [(10, 768), (50, 64)])
def test_small_store_lists(lam, b, k, d):
    """At most the sample size: one pass of per-lane lists over all rows."""
    rng = np.random.default_rng(100 + b)
    n = 3000
    x = synth.unit_rows(rng, n, d).astype(np.float32)
    s, eps, c = _wide_store(lam, x, b)
    q = np.concatenate([synth.unit_rows(rng, 60, d), x[rng.choice(n, 20)]]).astype(np.float32)
    gs, gi, gb = s.score_topk(_dev(q), k)
    worst = _compare(gs.cpu().numpy(), gi.cpu().numpy(), c, np.arange(n), q, eps, k)
    beta = score.bound(q, eps)
    gbn = gb.cpu().numpy().astype(np.float64)
    assert np.all(gbn >= beta) and np.all(gbn - beta <= np.spacing(gbn.astype(np.float32)))
    print(f"b={b} k={k} d={d}: max |score - oracle| = {worst:.3g}")


@pytest.mark.parametrize("b", [14, 22])
@pytest.mark.parametrize("k,d", [(10, 64), (50, 768)])
def test_large_store_threshold_plan(lam, b, k, d):
    """Beyond the sample size: sample, filter on the hi part, select, rescore
    in binary64 over the split rows; an all-zero query overflows its
    candidate buffer and comes back exact from the fallback."""
    rng = np.random.default_rng(200 + b)
    n = 20000
    x = synth.unit_rows(rng, n, d).astype(np.float32)
    s, eps, c = _wide_store(lam, x, b)
    q = np.concatenate([synth.unit_rows(rng, 30, d), x[rng.choice(n, 10)]]).astype(np.float32)
    q[7] = 0.0
    gs, gi, _ = s.score_topk(_dev(q), k)
    gs, gi = gs.cpu().numpy(), gi.cpu().numpy()
    assert np.all(gi[7] == np.arange(k)) and np.all(gs[7] == 0.0)
    keep = [j for j in range(q.shape[0]) if j != 7]
    _compare(gs[keep], gi[keep], c, np.arange(n), q[keep], eps, k)


def test_certificate_on_wide_codes(lam):
    """Sound (certified => exact margin above 2 (beta + ||q|| delta_hat)) with
    the split form's error constant; the top-k equals lam_score_topk's."""
    import torch
    rng = np.random.default_rng(23)
    d, n, b = 768, 3000, 18
    x = synth.unit_rows(rng, n, d).astype(np.float32)
    s = lam.Store(d, 0.95, n)
    s.ingest(_dev(x))
    info = s.info()
    kept = s.ids().cpu().numpy()
    eps = _eps_for_bits(float(np.abs(x[kept]).max()), b)
    p = s.quantize(eps)
    assert p.bits == b
    codes = qeps.codes(x[kept], eps).reshape(kept.size, d)
    q = np.concatenate([synth.unit_rows(rng, 40, d), x[kept[rng.choice(kept.size, 24)]]]).astype(np.float32)
    qd = _dev(q)
    n_cert = 0
    for k in (1, 5, 20):
        gs, gi, gb, gc, gm = s.score_topk_certified(qd, k)
        ps, pi, pb = s.score_topk(qd, k)
        assert torch.equal(gi, pi) and torch.equal(gs, ps) and torch.equal(gb, pb)
        flags, margin, thr = score.certify(q, codes, kept, eps, k, info.delta_hat_run)
        gc = gc.cpu().numpy()
        assert np.all(margin[gc] > thr[gc])
        n_cert += int(gc.sum())
    assert n_cert > 0


def test_scores_from_blocks_equal_fixed_width(lam):
    """The block codec at a wide width: scoring from the blocks gives the
    fixed-width store's results bit for bit."""
    import torch
    rng = np.random.default_rng(24)
    x = synth.unit_rows(rng, 2000, 256).astype(np.float32)
    s, eps, c = _wide_store(lam, x, 17)
    s.block_encode()
    q = _dev(synth.unit_rows(rng, 20, 256).astype(np.float32))
    for k in (1, 10, 64):
        a = s.score_topk(q, k)
        bb = s.score_topk_blocks(q, k)
        assert all(torch.equal(u, v) for u, v in zip(a, bb))


def test_width_limits(lam):
    """23 bits and more: ESTATE; the allocation-free call takes 12 bits at most."""
    import torch
    rng = np.random.default_rng(25)
    x = synth.unit_rows(rng, 500, 64).astype(np.float32)
    s = _store_from_rows(lam, x)
    absmax = float(np.abs(x).max())
    q = _dev(synth.unit_rows(rng, 4, 64).astype(np.float32))
    s.quantize(_eps_for_bits(absmax, 23))
    with pytest.raises(lam.LamError) as e:
        s.score_topk(q, 5)
    assert e.value.name == "LAM_ESTATE"
    s.quantize(_eps_for_bits(absmax, 13))
    s.info()
    out = (torch.empty((4, 5), dtype=torch.float32, device="cuda"),
           torch.empty((4, 5), dtype=torch.int64, device="cuda"),
           torch.empty(4, dtype=torch.float32, device="cuda"))
    with pytest.raises(lam.LamError) as e:
        s.score_topk_noalloc(q, 5, out)
    assert e.value.name == "LAM_ESTATE"
    gs, gi, _ = s.score_topk(q, 5)                 # the allocating call scores it
    c = qeps.codes(x, _eps_for_bits(absmax, 13)).reshape(500, -1)
    _compare(gs.cpu().numpy(), gi.cpu().numpy(), c, np.arange(500), q.cpu().numpy(), _eps_for_bits(absmax, 13), 5)
