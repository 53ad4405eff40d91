"""Pins for the banded-candidate oracle (CPU): limiting cases that reduce to
exhaustive greedy or to exact-duplicate removal, the candidate definition by
brute force, and the substitution bound on every merge."""
import numpy as np

import synth
from oracle import dedup, lsh, qeps


def _rows(seed=0, n=300, d=64):
    rng = np.random.default_rng(seed)
    base = synth.unit_rows(rng, n - 60, d)
    dups = synth.near_dups(rng, base[rng.integers(0, n - 60, 60)])
    x = np.concatenate([base, dups]).astype(np.float32)
    return x[rng.permutation(n)]


def test_coarse_step_reduces_to_exhaustive_greedy():
    """A step larger than every coordinate makes every code 0, so every band
    matches and every retained record is a candidate: exhaustive greedy."""
    x = _rows()
    r = lsh.greedy_lsh(x, 0.95, eps_band=4.0, r=8)
    ref = dedup.greedy(x, 0.95)
    assert np.array_equal(r["rep"], ref["rep"]) and r["delta_hat"] == ref["delta_hat"]


def test_fine_step_keeps_only_equal_bands():
    """A step far below the coordinates' spacing makes two bands equal only
    for equal coordinates: near duplicates never become candidates, and an
    exact copy of a retained record merges into that record."""
    x = _rows()
    first = lsh.greedy_lsh(x, 0.95, eps_band=1e-9, r=16)
    assert np.count_nonzero(first["rep"] >= 0) == 0     # no exact copies among the rows
    src = first["kept"][[3, 50, 120, 200, 299]]
    x2 = np.concatenate([x, x[src]])
    r = lsh.greedy_lsh(x2, 0.95, eps_band=1e-9, r=16)
    assert np.array_equal(r["rep"][-5:], src) and np.count_nonzero(r["rep"][:300] >= 0) == 0


def test_candidates_by_brute_force():
    """The candidate count equals a brute-force count of (arrival, earlier
    retained record) pairs with at least one equal band."""
    x = _rows(seed=1, n=200)
    eps, w = 0.02, 8
    r = lsh.greedy_lsh(x, 0.95, eps, w)
    c = qeps.codes(x.reshape(-1), eps).reshape(x.shape)
    kept = set(r["kept"].tolist())
    n = 0
    for i in range(x.shape[0]):
        for y in range(i):
            if y in kept and any(np.array_equal(c[i, b:b + w], c[y, b:b + w]) for b in range(0, 64, w)):
                n += 1
    assert n == r["n_candidates"]


def test_merges_keep_the_substitution_bound():
    x = _rows(seed=2)
    for eps, w in ((0.01, 4), (0.05, 8), (0.2, 16)):
        r = lsh.greedy_lsh(x, 0.95, eps, w)
        dropped = np.nonzero(r["rep"] >= 0)[0]
        assert all(dedup.within(x[i], x[r["rep"][i]], 0.95) for i in dropped)
        assert np.all(r["rep"][dropped] < dropped)
        assert r["delta_hat"] <= dedup.delta(0.95)
        assert r["n_within"] <= r["n_candidates"]
