"""Pins for the near-duplicate oracle (CPU).

The streaming oracle is checked against: the pure-Python brute force of
Algorithm "admit" on exact integers (tiny inputs), the closed forms of
Eq. (identity) printed by the paper, hand-built threshold cases, the cover and
packing properties of greedy first-occurrence, Theorem "Score deficit" and its
tight example, invariance to how the stream is split into calls, and the
planted structure of the tiny-ingest workload.
"""
import math
import os

import numpy as np
import pytest

import synth
from oracle import dedup, invariants

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def _rows(path):
    return [l.split() for l in open(os.path.join(GOLD, path)) if l.strip() and l[0] != "#"]


def test_delta_closed_form_matches_paper_table():
    for t, d in _rows("delta_table.txt"):
        assert round(dedup.delta(float(t)), 4) == pytest.approx(float(d), abs=5e-5)
        assert float(dedup.delta2(float(t))) == pytest.approx(2 - 2 * float(t), abs=1e-15)


def test_double_radius_threshold():
    # Theorem "removal ceiling": radius 2 delta is the threshold t' = 4t - 3.
    for t in (0.99, 0.95, 0.90):
        assert dedup.delta(4 * t - 3) == pytest.approx(2 * dedup.delta(t), rel=1e-12)
        assert dedup.delta2(4 * t - 3) == 4 * dedup.delta2(t) or \
            abs(float(dedup.delta2(4 * t - 3)) - 4 * float(dedup.delta2(t))) < 1e-15


def test_inclusive_threshold_exact_case():
    # tau = 0.875 gives delta^2 = 0.25 exactly; a = (0.5, 0, ...), b = 0 sit at
    # exactly that distance and must merge (the test is inclusive).
    a = np.zeros(64, np.float32)
    a[0] = 0.5
    b = np.zeros(64, np.float32)
    assert dedup.delta2(0.875) == 0.25
    assert dedup.within(a, b, 0.875)
    r = dedup.greedy(np.stack([b, a]), 0.875)
    assert r["rep"].tolist() == [-1, 0] and r["delta_hat"] == 0.5
    # one float32 ulp further and it must not merge
    a2 = a.copy()
    a2[0] = np.nextafter(np.float32(0.5), np.float32(1))
    assert not dedup.within(a2, b, 0.875)
    assert dedup.greedy(np.stack([b, a2]), 0.875)["rep"].tolist() == [-1, -1]


def test_l2_rule_not_cosine_rule():
    # Rows a little longer than unit: cos(a, b) >= tau but ||a - b||^2 > 2 - 2 tau.
    # The paper's rule is the l2 distance (Algorithm "admit"), so no merge.
    d = 8
    a = np.zeros(d)
    a[0] = 1.0
    c = 0.9501
    b = np.zeros(d)
    b[0], b[1] = c, math.sqrt(1 - c * c)
    a32, b32 = (1.01 * a).astype(np.float32), (1.01 * b).astype(np.float32)
    cos = float(a32 @ b32) / (np.linalg.norm(a32) * np.linalg.norm(b32))
    assert cos >= 0.95
    assert not dedup.within(a32, b32, 0.95)
    assert dedup.greedy(np.stack([a32, b32]), 0.95)["rep"].tolist() == [-1, -1]


def _mixed(seed, n, d=96, tau=0.95):
    rng = np.random.default_rng(seed)
    base, _, _ = synth.clustered(rng, synth.cluster_sizes(n // 2, max(1, n // 16)), d,
                                 cmin=0.9, cmax=0.999)
    a, b = synth.near_threshold_pairs(rng, n // 8, d, tau, spread=2e-7)
    x = np.concatenate([base.astype(np.float32), a, b])
    return x[rng.permutation(x.shape[0])]


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_stream_matches_brute_force(seed):
    x = _mixed(seed, 160)
    for tau in (0.95, 0.99, 0.9):
        ref = dedup.greedy_naive(x, tau)
        got = dedup.greedy(x, tau, block=16)
        assert np.array_equal(got["rep"], ref["rep"])
        assert np.array_equal(got["kept"], ref["kept"])
        assert got["delta_hat"] == pytest.approx(ref["delta_hat"], abs=1e-15)


def _ties(seed, n_pairs=24, d=96):
    rng = np.random.default_rng(seed)
    a, b, b_in, b_out, tau = synth.dyadic_ties(rng, n_pairs, d)
    x = np.concatenate([a, b, b_in, b_out])
    return x[rng.permutation(x.shape[0])], a, b, b_in, b_out, tau


def test_dyadic_ties_sit_on_the_threshold():
    _, a, b, b_in, b_out, tau = _ties(0)
    for k in range(a.shape[0]):
        assert dedup.d2_exact(a[k], b[k]) == dedup.delta2(tau)
        assert dedup.within(a[k], b_in[k], tau)
        assert not dedup.within(a[k], b_out[k], tau)


@pytest.mark.parametrize("seed", [1, 2])
def test_exact_path_is_exercised(seed):
    x, *_, tau = _ties(seed)
    r = dedup.greedy(x, tau, block=8)
    assert r["n_exact"] > 0          # ties reach the rational check
    ref = dedup.greedy_naive(x, tau)
    assert np.array_equal(r["rep"], ref["rep"])
    assert r["delta_hat"] == ref["delta_hat"]


def test_planted_mistake_is_caught():
    # A representative that is not the lowest index fails lowest_index.
    x = _mixed(3, 128)
    r = dedup.greedy(x, 0.95)
    rep = r["rep"].copy()
    i = int(np.nonzero(rep >= 0)[0][0])
    bad = rep.copy()
    bad[i] = int(np.nonzero(rep[:i] < 0)[0][-1]) if rep[i] != np.nonzero(rep[:i] < 0)[0][-1] else -1
    assert invariants.lowest_index(x, bad, 0.95, sample=[i]) == [i]


def test_planted_cover_mistakes_are_caught():
    """Proposition "greedy is a cover and a packing", cover part: a dropped
    arrival whose representative lies outside delta, arrived later, or was
    itself dropped is reported, and only that arrival."""
    x = _mixed(4, 160)
    tau = 0.95
    rep = dedup.greedy(x, tau)["rep"]
    assert invariants.cover(x, rep, tau) == []
    dropped = np.nonzero(rep >= 0)[0]
    kept = np.nonzero(rep < 0)[0]
    i = int(dropped[-1])
    far = [int(k) for k in kept if k < i and not dedup.within(x[i], x[k], tau)][0]
    for wrong in (far,                                       # retained and earlier, but outside delta
                  int(kept[kept > i][0]) if np.any(kept > i) else i,   # not earlier
                  int(dropped[0])):                          # not retained
        bad = rep.copy()
        bad[i] = wrong
        assert invariants.cover(x, bad, tau) == [i]


def test_planted_packing_mistake_is_caught():
    """Packing part: marking a dropped arrival as retained puts two retained
    rows within delta of each other, and the pair is reported."""
    x = _mixed(5, 160)
    tau = 0.95
    rep = dedup.greedy(x, tau)["rep"]
    assert invariants.packing(x, rep, tau) == []
    i = int(np.nonzero(rep >= 0)[0][0])
    bad = rep.copy()
    bad[i] = -1
    found = invariants.packing(x, bad, tau)
    assert (int(rep[i]), i) in found
    assert all(i in pr for pr in found)


def test_planted_score_deficit_mistake_is_caught():
    """Theorem "Score deficit": on the tight example the deficit equals
    delta_hat, so a claimed bound just below it is reported, and a retained
    set that loses the best record for some query shows a deficit the bound
    does not cover."""
    a = np.array([1.0, 0.0], np.float32)
    b = np.array([0.96, 0.28], np.float32)
    x = np.stack([b, a])
    rep = np.array([-1, 0])
    dh = float(np.linalg.norm(a.astype(np.float64) - b))
    q = ((a.astype(np.float64) - b) / dh)[None, :]
    assert invariants.score_deficit(x, rep, q, dh, tol=1e-12) == []
    assert invariants.score_deficit(x, rep, q, dh * (1 - 1e-9), tol=0.0) == [0]
    # on the tiny workload, queries along retained rows pass with the run's
    # delta_hat; dropping one of those rows (a representative far away) leaves
    # its query a deficit near 1, far above the bound, and only that query fails
    t = synth.tiny_ingest()
    x = t["x"][:600]
    r = dedup.greedy(x, t["tau"])
    kept = np.nonzero(r["rep"] < 0)[0]
    qq = x[kept[5:25]].astype(np.float64)
    qq /= np.linalg.norm(qq, axis=1, keepdims=True)
    assert invariants.score_deficit(x, r["rep"], qq, r["delta_hat"]) == []
    bad = r["rep"].copy()
    bad[kept[7]] = kept[0]
    assert invariants.score_deficit(x, bad, qq, r["delta_hat"]) == [2]


@pytest.fixture(scope="module")
def tiny():
    return synth.tiny_ingest()


@pytest.fixture(scope="module")
def tiny_result(tiny):
    return dedup.greedy(tiny["x"], tiny["tau"])


def test_tiny_cover_packing_lowest_index(tiny, tiny_result):
    x, tau, rep = tiny["x"], tiny["tau"], tiny_result["rep"]
    assert invariants.cover(x, rep, tau) == []
    assert invariants.packing(x, rep, tau) == []
    rng = np.random.default_rng(0)
    dropped = np.nonzero(rep >= 0)[0]
    assert invariants.lowest_index(x, rep, tau, sample=rng.choice(dropped, 60, replace=False)) == []
    assert 0 < tiny_result["delta_hat"] <= dedup.delta(tau)


def test_tiny_planted_structure(tiny, tiny_result):
    # Planted copies sit at cosine 0.96..0.995 from their source (inside
    # delta at tau = 0.95); unrelated Gaussian rows are far apart.  So every
    # merge joins rows of one source, and a source with a single planted copy
    # keeps exactly one of the two.
    src, rep = tiny["source"], tiny_result["rep"]
    dropped = np.nonzero(rep >= 0)[0]
    assert np.all(src[dropped] == src[rep[dropped]])
    vals, counts = np.unique(src, return_counts=True)
    pairs = vals[counts == 2]
    kept_per_src = np.bincount(src[rep < 0], minlength=src.max() + 1)
    assert np.all(kept_per_src[pairs] == 1)
    assert np.all(kept_per_src[vals] >= 1)
    assert tiny_result["rep"].size - np.count_nonzero(rep >= 0) == np.count_nonzero(rep < 0)


def test_tiny_partition_invariance(tiny, tiny_result):
    # Appendix "Implementation details": online and batch forms coincide; any
    # split of the stream into calls gives the same outputs.
    x, tau = tiny["x"][:1500], tiny["tau"]
    ref = dedup.greedy(x, tau)
    for batch, block in ((1, 1), (7, 3), (64, 64), (1024, 256)):
        got = dedup.greedy(x, tau, batch=batch, block=block)
        assert np.array_equal(got["rep"], ref["rep"])
        assert got["delta_hat"] == ref["delta_hat"]
    # a prefix of the stream takes the same decisions as the whole stream did
    assert np.array_equal(ref["rep"], tiny_result["rep"][:1500])
    assert dedup.deletion_digest(ref["rep"]) == dedup.deletion_digest(tiny_result["rep"][:1500])


def test_score_deficit_theorem(tiny, tiny_result):
    # Theorem "Score deficit": 0 <= max_S q.x - max_R q.z <= delta_hat for unit q.
    rng = np.random.default_rng(4)
    q = synth.unit_rows(rng, 200, tiny["x"].shape[1])
    # queries aimed at dropped rows make the deficit non-trivial
    dropped = np.nonzero(tiny_result["rep"] >= 0)[0][:200]
    q2 = tiny["x"][dropped].astype(np.float64)
    q2 /= np.linalg.norm(q2, axis=1, keepdims=True)
    for qq in (q, q2):
        assert invariants.score_deficit(tiny["x"], tiny_result["rep"], qq, tiny_result["delta_hat"]) == []


def test_score_deficit_tight_example():
    # S = {a, b}, ||a - b|| = delta, R = {b}: q = (a - b)/delta has deficit delta.
    a = np.array([1.0, 0.0], np.float32)
    b = np.array([0.96, 0.28], np.float32)       # cos = 0.96, delta^2 = 2 - 2*0.96 (float32 rows)
    tau = 1.0 - float(dedup.d2_exact(a, b)) / 2  # threshold placed exactly at their distance
    assert dedup.within(a, b, tau) or dedup.within(a, b, tau - 1e-15)
    x = np.stack([b, a])
    r = dedup.greedy(x, tau - 1e-12)
    assert r["rep"].tolist() == [-1, 0]
    q = (a.astype(np.float64) - b) / np.linalg.norm(a.astype(np.float64) - b)
    gap = float(q @ a) - float(q @ b)
    assert gap == pytest.approx(r["delta_hat"], rel=1e-12)


def test_deletion_digest_is_order_sensitive():
    r1 = np.array([-1, 0, -1, 2], np.int64)
    r2 = np.array([-1, 0, -1, 0], np.int64)
    assert dedup.deletion_digest(r1) != dedup.deletion_digest(r2)
    assert dedup.deletion_digest(r1) == dedup.deletion_digest(r1.copy())


def test_decide_one_matches_stream(tiny, tiny_result):
    x, tau, rep = tiny["x"], tiny["tau"], tiny_result["rep"]
    kept = rep < 0
    for i in (0, 1, 10, 500, 2000, 4095):
        assert dedup.decide_one(x, i, np.nonzero(kept[:i])[0], tau) == rep[i]


def test_decide_many_matches_decide_one():
    """The blocked form gives decide_one's answer for every sampled arrival,
    including exact ties on the threshold and blocks smaller than the set."""
    rng = np.random.default_rng(11)
    a, b, b_in, b_out, tau = synth.dyadic_ties(rng, 40, 64)
    x = np.concatenate([a, b, b_in, b_out, synth.unit_rows(rng, 120, 64).astype(np.float32)])
    x = x[rng.permutation(x.shape[0])]
    ref = dedup.greedy(x, tau)
    kept = np.nonzero(ref["rep"] < 0)[0]
    samples = np.arange(x.shape[0])
    got = dedup.decide_many(x, samples, kept, tau, block=17)
    one = [dedup.decide_one(x, int(i), kept[kept < i], tau) for i in samples]
    assert got.tolist() == one == ref["rep"].tolist()


def test_decide_on_rows_that_are_not_unit():
    """decide_one and decide_many on rows of norm 1/2 to 64 with pairs planted
    exactly on the threshold and one float32 ulp either side (the library
    takes such rows as given): both equal the pure-Python brute force on exact
    integers, so their candidate margins scale with the rows' norms."""
    rng = np.random.default_rng(12)
    rows = []
    for scale in (0.5, 4.0, 64.0):
        a, b, b_in, b_out, tau = synth.dyadic_ties(rng, 12, 64)
        # a * scale stays on a power-of-two grid; b keeps b - a = (e_i - e_j)/4
        a_s = (a.astype(np.float64) * scale).astype(np.float32)
        for bb in (b, b_in, b_out):
            d = bb.astype(np.float64) - a.astype(np.float64)
            rows.append((a_s.astype(np.float64) + d).astype(np.float32))
        rows.append(a_s)
        rows.append((synth.unit_rows(rng, 20, 64) * scale).astype(np.float32))
    x = np.concatenate(rows)
    x = x[rng.permutation(x.shape[0])]
    ref = dedup.greedy_naive(x, tau)
    assert np.count_nonzero(ref["rep"] >= 0) > 20          # the planted pairs merge
    kept = np.nonzero(ref["rep"] < 0)[0]
    samples = np.arange(x.shape[0])
    one = [dedup.decide_one(x, int(i), kept[kept < i], tau) for i in samples]
    assert one == ref["rep"].tolist()
    assert dedup.decide_many(x, samples, kept, tau, block=13).tolist() == ref["rep"].tolist()
    assert np.array_equal(dedup.greedy(x, tau, block=7)["rep"], ref["rep"])


def test_removal_ceiling_closed_forms():
    """Orthonormal rows are sqrt(2) apart: at tau = 0.95 (2 delta = 0.63)
    nothing merges in either pass; at tau = 0.6 (delta = 0.89 < sqrt(2) < 2
    delta = 1.79) nothing merges at delta and everything merges into the
    first row at 2 delta.  Identical rows merge at any radius."""
    e = np.eye(64, dtype=np.float32)[:40]
    r = dedup.removal_ceiling(e, 0.95)
    assert (r["kept"], r["kept_2delta"], r["removal"], r["ceiling"]) == (40, 40, 0.0, 0.0)
    r = dedup.removal_ceiling(e, 0.6)
    assert (r["kept"], r["kept_2delta"]) == (40, 1)
    assert r["ceiling"] == 1 - 1 / 40 and r["bits_lo"] == 0.0 and r["bits_hi"] == math.log2(40)
    same = np.repeat(e[:1], 9, axis=0)
    r = dedup.removal_ceiling(same, 0.99)
    assert (r["kept"], r["kept_2delta"]) == (1, 1)


def test_removal_ceiling_packing_and_order():
    """Theorem "removal ceiling": the 2 delta pass returns a 2 delta-packing
    (every pair of its survivors is more than 2 delta apart, brute force), no
    larger than the delta pass, so the ceiling bounds the attained removal."""
    t = synth.tiny_ingest()
    x = t["x"][:700]
    for tau in (0.95, 0.9, 0.75):
        r = dedup.removal_ceiling(x, tau)
        p = x[r["kept_ids_2delta"]].astype(np.float64)
        nn = np.einsum("ij,ij->i", p, p)
        d2 = nn[:, None] + nn[None, :] - 2.0 * (p @ p.T)   # binary64, error ~1e-13
        iu = np.triu_indices(p.shape[0], 1)
        assert np.all(d2[iu] > 4 * float(dedup.delta2(tau)) - 1e-9)
        assert r["kept_2delta"] <= r["kept"] and r["ceiling"] >= r["removal"]
        assert r["bits_lo"] <= r["bits_hi"]
