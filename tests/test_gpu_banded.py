"""Banded candidates (Section 2.2, layer L1; Algorithm "admit" with a band
index; Appendix "Band width and quantizer step") on the device against the
oracle: representatives identical to oracle.lsh.greedy_lsh, delta_hat within
1e-12, the candidate count equal to a count from the band codes, the coarse
step equal to exhaustive greedy (and to the screened store), exact copies at
the finest step, calls that do not wait, clearing, and the argument checks.
At the subset workload's full size (27,986 rows of D = 768 at the shipped
r = 4, eps = 0.2 sigma) sampled decisions are recomputed by the oracle over the
arrival's candidates.

Candidate pairs of the device path: an arrival against retained rows of
earlier chunks (chunks of 4,096 arrivals per call), plus arrivals j < i of its
own chunk with an equal band whether or not j is kept; the sequential oracle
counts retained rows only, so the count is checked against the band codes.
"""
import numpy as np
import pytest
import torch

import synth
from oracle import dedup, lsh, qeps

pytestmark = pytest.mark.gpu
CHUNK = 4096


def _rows(seed=7, n=5000, d=64, n_clusters=100):
    rng = np.random.default_rng(seed)
    rows, _, _ = synth.clustered(rng, synth.cluster_sizes(n, n_clusters), d)
    return rows[rng.permutation(n)].astype(np.float32)


def _ingest(lam, x, tau, eps, r, splits, sync=True, ctx=None):
    s = lam.Store(x.shape[1], tau, x.shape[0], ctx=ctx, eps_band=eps, band_width=r)
    xd = torch.from_numpy(x).cuda()
    reps, stats = [], []
    for a, b in zip(splits[:-1], splits[1:]):
        rep, st = s.ingest(xd[a:b], sync=sync)
        reps.append(rep)
        stats.append(st)
    return s, torch.cat(reps).cpu().numpy(), stats


def _share(x, eps, r):
    """share[i, y]: rows i and y have equal codes in at least one band."""
    c = qeps.codes(x.reshape(-1), eps).reshape(x.shape)
    n, d = x.shape
    out = np.zeros((n, n), dtype=bool)
    for b in range(0, d, r):
        _, g = np.unique(c[:, b:b + r], axis=0, return_inverse=True)
        g = g.reshape(-1)
        out |= g[:, None] == g[None, :]
    return out


def _expected_candidates(x, eps, r, rep, splits):
    share = _share(x, eps, r)
    n = x.shape[0]
    chunk = np.empty(n, dtype=np.int64)
    c = 0
    for a, b in zip(splits[:-1], splits[1:]):
        for s0 in range(a, b, CHUNK):
            chunk[s0:min(b, s0 + CHUNK)] = c
            c += 1
    kept = rep < 0
    idx = np.arange(n)
    store = share & kept[None, :] & (chunk[None, :] < chunk[:, None])
    inner = share & (chunk[None, :] == chunk[:, None]) & (idx[None, :] < idx[:, None])
    return int(store.sum() + inner.sum())


@pytest.mark.parametrize("r,rel", [(4, 0.2), (8, 0.3), (4, 0.3)])
def test_parity_with_oracle(lam, r, rel):
    x = _rows()
    d = x.shape[1]
    eps = rel / np.sqrt(d)
    splits = [0, 700, 700 + 4500, x.shape[0]]          # the middle call spans two chunks
    _, rep, stats = _ingest(lam, x, 0.95, eps, r, splits)
    ref = lsh.greedy_lsh(x, 0.95, eps, r)
    assert np.array_equal(rep, ref["rep"]), np.nonzero(rep != ref["rep"])[0][:10]
    assert abs(stats[-1]["delta_hat_run"] - ref["delta_hat"]) <= 1e-12
    assert stats[-1]["store_size"] == ref["kept"].size
    got = sum(s["n_ambiguous_pairs"] for s in stats)
    assert got == _expected_candidates(x, eps, r, rep, splits)
    print(f"r={r} rel={rel}: kept {ref['kept'].size}, candidates {got} (oracle, retained only: "
          f"{ref['n_candidates']})")


def test_coarse_step_is_exhaustive_greedy(lam):
    """Every code 0: every retained row is a candidate, so rep is exhaustive
    greedy and equals the screened store's.  The second call's candidates
    overflow a fresh context's pair list, so that call repeats from the store
    as it was (the band index rebuilt from the earlier rows)."""
    x = _rows(seed=8, n=5200)
    ctx = lam.Context()
    splits = [0, 1000, 5200]
    _, rep, stats = _ingest(lam, x, 0.95, 4.0, 8, splits, ctx=ctx)
    ref = dedup.greedy(x, 0.95)
    assert np.array_equal(rep, ref["rep"])
    assert abs(stats[-1]["delta_hat_run"] - ref["delta_hat"]) <= 1e-12
    assert stats[1]["n_ambiguous_pairs"] > (1 << 20)      # beyond the initial pair list
    plain = lam.Store(x.shape[1], 0.95, x.shape[0], ctx=ctx)
    rep2, _ = plain.ingest(torch.from_numpy(x).cuda())
    assert np.array_equal(rep2.cpu().numpy(), rep)


def test_exact_copies_at_the_finest_step(lam):
    x = _rows(seed=9, n=3000, d=128)
    src = np.array([5, 17, 800, 1500, 2999])
    x2 = np.concatenate([x, x[src]])
    _, rep, stats = _ingest(lam, x2, 0.95, 2.0 ** -23, 16, [0, 3000, 3005])
    ref = lsh.greedy_lsh(x2, 0.95, 2.0 ** -23, 16)
    assert np.array_equal(rep, ref["rep"])
    assert np.array_equal(rep[-5:], src) and stats[-1]["delta_hat_call"] == 0.0
    assert np.count_nonzero(rep[:3000] >= 0) == 0


def test_calls_that_do_not_wait(lam):
    x = _rows(seed=10, n=6000)
    eps = 0.3 / 8
    splits = [0, 1024, 2048, 3000, 6000]
    s, rep, stats = _ingest(lam, x, 0.95, eps, 8, splits, sync=False)
    assert all(st is None for st in stats)
    ref = lsh.greedy_lsh(x, 0.95, eps, 8)
    assert np.array_equal(rep, ref["rep"])
    info = s.info()
    assert info.size == ref["kept"].size and info.n_seen == x.shape[0]
    assert abs(info.delta_hat_run - ref["delta_hat"]) <= 1e-12
    assert np.array_equal(s.ids().cpu().numpy(), ref["kept"])


def test_clear_empties_the_index(lam):
    x = _rows(seed=11, n=2500)
    eps = 0.2 / 8
    s, rep, _ = _ingest(lam, x, 0.95, eps, 4, [0, 2500])
    s.clear()
    rep2, st = s.ingest(torch.from_numpy(x).cuda())
    assert np.array_equal(rep2.cpu().numpy(), rep)
    assert st["store_size"] == np.count_nonzero(rep < 0)


@pytest.mark.parametrize("r,rel", [(1, 0.01), (64, 2.0)])
def test_extreme_band_widths(lam, r, rel):
    """One coordinate per band (64 bands of one code: many candidates) and a
    single band of all D coordinates (candidates only for equal code
    vectors)."""
    x = _rows(seed=13, n=1000)
    eps = rel / 8
    _, rep, stats = _ingest(lam, x, 0.95, eps, r, [0, 500, 1000])
    ref = lsh.greedy_lsh(x, 0.95, eps, r)
    assert np.array_equal(rep, ref["rep"]) and np.count_nonzero(rep >= 0) > 0
    assert sum(st["n_ambiguous_pairs"] for st in stats) == _expected_candidates(x, eps, r, rep, [0, 500, 1000])


def test_invalid_input_of_a_call_that_does_not_wait(lam):
    """A call that does not wait and holds a NaN leaves the store and its band
    index unchanged; the next call that waits reports it once."""
    x = _rows(seed=14, n=2000)
    eps = 0.3 / 8
    s = lam.Store(64, 0.95, 4000, eps_band=eps, band_width=8)
    xd = torch.from_numpy(x).cuda()
    s.ingest(xd[:1000], sync=False)
    bad = xd[1000:1500].clone()
    bad[7, 3] = float("nan")
    s.ingest(bad, sync=False)
    with pytest.raises(lam.LamError):
        s.info()
    rep2, _ = s.ingest(xd[1000:2000])
    ref = lsh.greedy_lsh(x, 0.95, eps, 8)
    assert np.array_equal(rep2.cpu().numpy(), ref["rep"][1000:])
    assert s.info().size == ref["kept"].size


def test_argument_checks(lam):
    with pytest.raises(lam.LamError):
        lam.Store(64, 0.95, 100, eps_band=0.01, band_width=5)        # does not divide dim
    with pytest.raises(lam.LamError):
        lam.Store(64, 0.95, 100, eps_band=1e-9, band_width=8)        # below 2^-23
    with pytest.raises(ValueError):
        lam.Store(64, 0.95, 100, eps_band=0.01)
    s = lam.Store(64, 0.95, 100, eps_band=0.01, band_width=8)
    x = torch.from_numpy(_rows(seed=12, n=50)).cuda()
    with pytest.raises(lam.LamError):
        s.ingest(x, max_cos=True)
    rep, st = s.ingest(x)
    assert st["n_in"] == 50


@pytest.fixture(scope="module")
def subset_run(lam):
    cfg = synth.subset_ingest()
    x = cfg["x"]
    d = x.shape[1]
    eps = 0.2 / np.sqrt(d)
    splits = list(range(0, x.shape[0], cfg["batch"])) + [x.shape[0]]
    print(f"banded subset ingest: {cfg['name']} r=4 eps={eps:.6f}", flush=True)
    s, rep, stats = _ingest(lam, x, cfg["tau"], eps, 4, splits, sync=False)
    info = s.info()
    return dict(x=x, rep=rep, info=info, eps=eps, tau=cfg["tau"], ids=s.ids().cpu().numpy())


def test_subset_sampled_decisions(subset_run):
    """Sampled arrivals decided again by the oracle: the candidates are the
    rows retained at the arrival that share a band's codes; the representative
    is the lowest candidate within delta, else the arrival is kept."""
    x, rep, eps, tau = subset_run["x"], subset_run["rep"], subset_run["eps"], subset_run["tau"]
    n, d = x.shape
    kept = rep < 0
    assert np.array_equal(subset_run["ids"], np.nonzero(kept)[0])
    codes = qeps.codes(x.reshape(-1), eps).reshape(n, d)
    rng = np.random.default_rng(13)
    samples = np.unique(np.concatenate([rng.integers(0, n, 60), rng.choice(np.nonzero(~kept)[0], 40)]))
    for i in samples:
        eq = (codes[:i] == codes[i]).reshape(i, d // 4, 4).all(axis=2).any(axis=1)
        cand = np.nonzero(eq & kept[:i])[0]
        # binary64 distances decide all but pairs within rounding distance of
        # delta^2, which the exact predicate decides
        d2 = np.sum((x[cand].astype(np.float64) - x[i].astype(np.float64)) ** 2, axis=1)
        d2f = float(dedup.delta2(tau))
        want = -1
        for y, v in zip(cand, d2):
            if (v <= d2f) if abs(v - d2f) > 1e-12 else dedup.within(x[i], x[y], tau):
                want = int(y)
                break
        assert rep[i] == want, (i, rep[i], want)


def test_subset_bound_and_recall(subset_run):
    """Every merge keeps the substitution bound; the banded result removes no
    more than exhaustive greedy would allow by the ceiling, and the run's
    delta_hat is the max merged distance."""
    x, rep, tau = subset_run["x"], subset_run["rep"], subset_run["tau"]
    dropped = np.nonzero(rep >= 0)[0]
    assert np.all(rep[dropped] < dropped) and np.all(rep[rep[dropped]] == -1)
    a = x[dropped].astype(np.float64)
    b = x[rep[dropped]].astype(np.float64)
    dist = np.sqrt(np.sum((a - b) ** 2, axis=1))
    assert np.all(dist <= dedup.delta(tau) * (1 + 1e-12))
    assert abs(subset_run["info"].delta_hat_run - dist.max()) <= 1e-12
    print(f"banded subset: removal {dropped.size / rep.size:.4f}")
