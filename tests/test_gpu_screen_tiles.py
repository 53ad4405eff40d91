"""GPU parity of the screen's two tilings (lam_ctx_set_screen_tile): the
256 x 256 tile, forced on every launch, gives the oracle's decisions on the
benchmark stream (calls that wait, calls that do not, calls split into
chunks), at D = 1,024, on exact ties at D = 768, and where the automatic
choice switches from the small to the large tile within one stream."""
import numpy as np
import pytest
import torch

import synth
from oracle import dedup

pytestmark = pytest.mark.gpu


def _dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def _ctx(lam, policy):
    c = lam.Context(0)
    c.set_screen_tile(policy)
    return c


def _ingest(lam, ctx, x, tau, batch, sync=True):
    s = lam.Store(x.shape[1], tau, x.shape[0], ctx=ctx)
    xd = _dev(x)
    reps = [s.ingest(xd[b0:b0 + batch], sync=sync)[0] for b0 in range(0, x.shape[0], batch)]
    info = s.info()
    return torch.cat(reps).cpu().numpy(), info


_REF = {}


def _subset(tau):
    if tau not in _REF:
        x = synth.subset_ingest()["x"]
        _REF[tau] = (x, dedup.greedy(x, tau, block=512))
    return _REF[tau]


@pytest.mark.parametrize("tau", [0.95, 0.99])
def test_large_tile_subset_parity(lam, tau):
    """The 27,986-row benchmark stream in calls of 1,024 that wait."""
    x, ref = _subset(tau)
    rep, info = _ingest(lam, _ctx(lam, "large"), x, tau, 1024)
    assert np.array_equal(rep, ref["rep"])
    assert abs(info.delta_hat_run - ref["delta_hat"]) <= 1e-12


def test_large_tile_async_and_chunked(lam):
    """Calls that do not wait (the grid covers an upper bound of the store
    size, which the kernel reads), and calls of 10,000 rows split into chunks
    of 4,096 (16 chunk tiles, a 136-tile in-chunk triangle)."""
    x, ref = _subset(0.95)
    ctx = _ctx(lam, "large")
    rep, info = _ingest(lam, ctx, x, 0.95, 1024, sync=False)
    assert np.array_equal(rep, ref["rep"])
    assert info.size == int(np.count_nonzero(ref["rep"] < 0))
    rep, info = _ingest(lam, ctx, x, 0.95, 10000)
    assert np.array_equal(rep, ref["rep"])
    assert abs(info.delta_hat_run - ref["delta_hat"]) <= 1e-12


@pytest.mark.parametrize("policy", ["large", "small"])
def test_d1024_parity(lam, policy):
    """D = 1,024 (16 slabs) on a clustered stream of 9,000 rows, both tiles."""
    x = synth.subset_ingest(seed=11, n=9000, n_traj=200, d=1024)["x"]
    ref = dedup.greedy(x, 0.95, block=512)
    rep, info = _ingest(lam, _ctx(lam, policy), x, 0.95, 2048)
    assert np.array_equal(rep, ref["rep"])
    assert abs(info.delta_hat_run - ref["delta_hat"]) <= 1e-12
    assert 0 < np.count_nonzero(rep >= 0) < x.shape[0]


def test_large_tile_exact_ties(lam):
    """Pairs planted exactly on the threshold at D = 768 (escalated to exact
    integers), screened by the large tile."""
    rng = np.random.default_rng(31)
    a, b, b_in, b_out, tau = synth.dyadic_ties(rng, 150, 768)
    x = np.concatenate([a, b, b_in, b_out, synth.unit_rows(rng, 400, 768).astype(np.float32)])
    x = x[rng.permutation(x.shape[0])]
    ref = dedup.greedy(x, tau)
    assert ref["n_exact"] > 0
    ctx = _ctx(lam, "large")
    s = lam.Store(768, tau, x.shape[0], ctx=ctx)
    xd = _dev(x)
    reps, esc = [], 0
    for b0 in range(0, x.shape[0], 300):
        r, st = s.ingest(xd[b0:b0 + 300])
        reps.append(r.cpu().numpy())
        esc += st["n_exact_escalations"]
    assert np.array_equal(np.concatenate(reps), ref["rep"])
    assert esc > 0


def test_auto_switches_within_stream(lam):
    """The benchmark stream in calls of 4,096 that do not wait, the tile left
    to the automatic choice: the first three calls' launches hold fewer than
    768 large tiles (small tiles), the later ones more (large tiles)."""
    x, ref = _subset(0.95)
    rep, info = _ingest(lam, _ctx(lam, "auto"), x, 0.95, 4096, sync=False)
    assert np.array_equal(rep, ref["rep"])
    assert info.size == int(np.count_nonzero(ref["rep"] < 0))
    # a call's large-tile grid covers the rows seen before it (an upper bound
    # of the store size) times the 16 chunk tiles, plus the in-chunk triangle
    grids = [((4096 * c + 255) // 256) * 16 + 136 for c in range((x.shape[0] + 4095) // 4096 - 1)]
    assert min(grids) < 768 <= max(grids)


def test_policy_values(lam):
    c = lam.Context(0)
    for p in ("auto", "small", "large", 0, 1, 2):
        c.set_screen_tile(p)
    with pytest.raises(lam.LamError) as e:
        c.set_screen_tile(3)
    assert e.value.name == "LAM_EINVAL"
