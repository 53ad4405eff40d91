"""GPU parity of the greedy near-duplicate test (Algorithm "admit") against the
oracle: identical representatives (bit-exact decisions), deletion digest,
delta_hat within 1e-12, max-cos within the screen bound; invariance to how the
stream is split into calls; exact ties; error paths."""
import numpy as np
import pytest
import torch

import synth
from oracle import dedup, invariants, qeps, score

pytestmark = pytest.mark.gpu


def _dev(a):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def _ingest(lam, x, tau, batch, capacity=None, max_cos=False):
    s = lam.Store(x.shape[1], tau, capacity or x.shape[0])
    reps, stats, cos = [], [], []
    xd = _dev(x)
    for b0 in range(0, x.shape[0], batch):
        r = s.ingest(xd[b0:b0 + batch], max_cos=max_cos)
        reps.append(r[0].cpu().numpy())
        stats.append(r[1])
        if max_cos:
            cos.append(r[2].cpu().numpy())
    rep = np.concatenate(reps) if reps else np.zeros(0, np.int64)
    return s, rep, stats, (np.concatenate(cos) if max_cos else None)


@pytest.fixture(scope="module")
def tiny():
    t = synth.tiny_ingest()
    t["ref"] = dedup.greedy(t["x"], t["tau"])
    return t


def test_tiny_parity(lam, tiny):
    s, rep, stats, cos = _ingest(lam, tiny["x"], tiny["tau"], tiny["batch"], max_cos=True)
    ref = tiny["ref"]
    assert np.array_equal(rep, ref["rep"])
    assert dedup.deletion_digest(rep) == dedup.deletion_digest(ref["rep"])
    assert np.array_equal(s.ids().cpu().numpy(), ref["kept"])
    assert abs(stats[-1]["delta_hat_run"] - ref["delta_hat"]) <= 1e-12
    assert sum(st["n_kept"] for st in stats) == ref["kept"].size
    # max cos: screened in fp16 with fp32 accumulation, within the screen bound
    fin = np.isfinite(ref["max_cos"])
    assert np.array_equal(np.isfinite(cos), fin)
    assert np.max(np.abs(cos[fin] - ref["max_cos"][fin])) <= 1.1e-3


@pytest.mark.parametrize("batch", [1, 7, 64, 1000, 4096])
def test_tiny_partition_invariance(lam, tiny, batch):
    x = tiny["x"] if batch >= 64 else tiny["x"][:600]
    ref = tiny["ref"]["rep"][: x.shape[0]]
    _, rep, stats, _ = _ingest(lam, x, tiny["tau"], batch)
    assert np.array_equal(rep, ref)


def test_repeat_runs_identical(lam, tiny):
    d = set()
    for _ in range(3):
        _, rep, _, _ = _ingest(lam, tiny["x"], tiny["tau"], 1024)
        d.add(dedup.deletion_digest(rep))
    assert len(d) == 1


def test_exact_ties_and_escalation(lam):
    rng = np.random.default_rng(5)
    a, b, b_in, b_out, tau = synth.dyadic_ties(rng, 200, 128)
    x = np.concatenate([a, b, b_in, b_out, synth.unit_rows(rng, 300, 128).astype(np.float32)])
    x = x[rng.permutation(x.shape[0])]
    ref = dedup.greedy(x, tau)
    assert ref["n_exact"] > 0
    _, rep, stats, _ = _ingest(lam, x, tau, 256)
    assert np.array_equal(rep, ref["rep"])
    assert sum(st["n_exact_escalations"] for st in stats) > 0
    assert abs(stats[-1]["delta_hat_run"] - ref["delta_hat"]) <= 1e-12
    # exact ties sit at delta^2 exactly: the smallest decided margin is 0
    assert min(st["min_margin_d2"] for st in stats) == 0.0


@pytest.mark.parametrize("d", [32, 96, 160, 4096])
def test_ragged_dims_parity(lam, d):
    """Dimensions where the reduction is shorter than one slab of 64 (32),
    ends in a partial slab (96, 160), or is the largest allowed (4,096, the
    kernel for any length): planted near-duplicates at cosine 0.93-0.99
    around tau = 0.95, so that merges, misses and ambiguous pairs all occur."""
    rng = np.random.default_rng(d)
    n_base = 500 if d < 4096 else 200
    base = synth.unit_rows(rng, n_base, d)
    dups = synth.members(rng, base[rng.integers(0, n_base, n_base // 2)],
                         rng.uniform(0.93, 0.99, n_base // 2))
    x = np.concatenate([base, dups]).astype(np.float32)
    x = x[rng.permutation(x.shape[0])]
    ref = dedup.greedy(x, 0.95)
    _, rep, stats, cos = _ingest(lam, x, 0.95, 128, max_cos=True)
    assert np.array_equal(rep, ref["rep"]), np.nonzero(rep != ref["rep"])[0][:10]
    assert abs(stats[-1]["delta_hat_run"] - ref["delta_hat"]) <= 1e-12
    fin = np.isfinite(ref["max_cos"])
    assert np.array_equal(fin, np.isfinite(cos))
    # the screen's bound for unit rows: 2 (2^-11 + 2^-22) from the fp16
    # operands plus the fp32 accumulation's 2 D 2^-24 (1.1e-3 up to D = 1,024)
    tol = 1.1e-3 if d <= 1024 else 2 * (2.0 ** -11 + 2.0 ** -22) + 2 * d * 2.0 ** -24 + 1e-5
    assert np.max(np.abs(cos[fin] - ref["max_cos"][fin])) <= tol
    assert 0 < np.count_nonzero(rep >= 0) < n_base // 2


def test_inclusive_threshold_pair(lam):
    a = np.zeros((1, 64), np.float32)
    a[0, 0] = 0.5
    x = np.concatenate([np.zeros((1, 64), np.float32), a])
    _, rep, stats, _ = _ingest(lam, x, 0.875, 2)
    assert rep.tolist() == [-1, 0]
    assert stats[-1]["delta_hat_call"] == 0.5


_SUBSET_REF = {}


def _subset_ref(tau):
    if tau not in _SUBSET_REF:
        x = synth.subset_ingest()["x"]
        _SUBSET_REF[tau] = (x, dedup.greedy(x, tau, block=512))
    return _SUBSET_REF[tau]


@pytest.mark.parametrize("tau", [0.95, 0.99])
def test_subset_parity(lam, tau):
    """27,986 clustered rows in batches of 1,024 (the benchmark's launch
    configuration), exhaustive parity with the oracle."""
    x, ref = _subset_ref(tau)
    _, rep, stats, _ = _ingest(lam, x, tau, 1024)
    assert np.array_equal(rep, ref["rep"])
    assert abs(stats[-1]["delta_hat_run"] - ref["delta_hat"]) <= 1e-12
    amb = sum(st["n_ambiguous_pairs"] for st in stats)
    print(f"tau={tau}: kept {np.count_nonzero(rep < 0)} of {rep.size}, ambiguous pairs {amb}")


def test_subset_multi_chunk_calls(lam):
    """Calls of 10,000 rows: each is split into chunks of 4,096, 4,096 and
    1,808 rows inside the library (the last call is ragged)."""
    x, ref = _subset_ref(0.95)
    _, rep, stats, _ = _ingest(lam, x, 0.95, 10000)
    assert np.array_equal(rep, ref["rep"])
    assert abs(stats[-1]["delta_hat_run"] - ref["delta_hat"]) <= 1e-12


def test_ingest_after_failed_quantize(lam):
    """A quantize call that fails on the device in between two ingests leaves
    the second ingest's decisions unchanged."""
    x, ref = _subset_ref(0.95)
    s = lam.Store(x.shape[1], 0.95, x.shape[0])
    xd = _dev(x)
    r1, _ = s.ingest(xd[:5000])
    bad = torch.zeros(4096, dtype=torch.float32, device="cuda")
    bad[17] = float("nan")
    with pytest.raises(lam.LamError):
        lam.quantize(bad, 1e-3, absmax=1.0)
    r2, _ = s.ingest(xd[5000:12000])
    rep = torch.cat([r1, r2]).cpu().numpy()
    ref12 = dedup.greedy(x[:12000], 0.95, block=512)
    assert np.array_equal(rep, ref12["rep"])


def test_gpu_output_invariants(lam):
    cfg = synth.subset_ingest()
    x, tau = cfg["x"][:6000], 0.95
    _, rep, stats, _ = _ingest(lam, x, tau, 1024)
    assert invariants.cover(x, rep, tau) == []
    assert invariants.packing(x, rep, tau) == []
    assert stats[-1]["delta_hat_run"] <= dedup.delta(tau)


def test_errors_leave_store_unchanged(lam):
    rng = np.random.default_rng(1)
    x = synth.unit_rows(rng, 300, 64).astype(np.float32)
    s = lam.Store(64, 0.95, 400)
    s.ingest(_dev(x[:100]))
    size = s.size
    bad = x[100:200].copy()
    bad[50, 3] = np.nan
    with pytest.raises(lam.LamError) as e:
        s.ingest(_dev(bad))
    assert e.value.name == "LAM_EINVAL" and s.size == size and s.info().n_seen == 100
    for v in (300.0, 255.9375, -255.95):   # 2^8 x would overflow the screen's float16 operand
        big = x[100:200].copy()
        big[7, 0] = v
        with pytest.raises(lam.LamError) as e:
            s.ingest(_dev(big))
        assert e.value.name == "LAM_EINVAL" and s.size == size
    with pytest.raises(lam.LamError) as e:
        s.ingest(_dev(synth.unit_rows(rng, 301, 64).astype(np.float32)))
    assert e.value.name == "LAM_ECAPACITY" and s.size == size
    # the store still works and matches the oracle on the clean stream
    rep2, _ = s.ingest(_dev(x[100:]))
    ref = dedup.greedy(x, 0.95)
    assert np.array_equal(rep2.cpu().numpy(), ref["rep"][100:])


def test_empty_batch(lam):
    import torch
    s = lam.Store(64, 0.95, 10)
    rep, st = s.ingest(torch.empty((0, 64), dtype=torch.float32, device="cuda"))
    assert rep.numel() == 0 and st["n_in"] == 0 and s.size == 0
    assert st["min_margin_d2"] == float("inf")


# ----------------------------------------------------------------- calls that do not wait

def _ingest_async(lam, x, tau, batch, sync_every=0):
    """Ingest in batches with sync=False (every `sync_every`-th call waits)."""
    s = lam.Store(x.shape[1], tau, x.shape[0])
    xd = _dev(x)
    reps = []
    for k, b0 in enumerate(range(0, x.shape[0], batch)):
        sync = sync_every > 0 and k % sync_every == sync_every - 1
        reps.append(s.ingest(xd[b0:b0 + batch], sync=sync)[0])
    info = s.info()
    rep = torch.cat(reps).cpu().numpy() if reps else np.zeros(0, np.int64)
    return s, rep, info


def test_subset_async_parity(lam):
    """The benchmark's stream with calls that return before the device is done."""
    x, ref = _subset_ref(0.95)
    _, rep, info = _ingest_async(lam, x, 0.95, 1024)
    assert np.array_equal(rep, ref["rep"])
    assert info.size == int(np.count_nonzero(ref["rep"] < 0)) and info.n_seen == x.shape[0]
    assert abs(info.delta_hat_run - ref["delta_hat"]) <= 1e-12


def test_async_mixed_with_waiting_calls(lam):
    x, ref = _subset_ref(0.95)
    _, rep, info = _ingest_async(lam, x[:9000], 0.95, 700, sync_every=3)
    ref9 = dedup.greedy(x[:9000], 0.95, block=512)
    assert np.array_equal(rep, ref9["rep"])
    assert info.size == int(np.count_nonzero(ref9["rep"] < 0))


def test_async_exact_ties(lam):
    """Exact ties decided on the device inside calls that do not wait."""
    rng = np.random.default_rng(5)
    a, b, b_in, b_out, tau = synth.dyadic_ties(rng, 200, 128)
    x = np.concatenate([a, b, b_in, b_out, synth.unit_rows(rng, 300, 128).astype(np.float32)])
    x = x[rng.permutation(x.shape[0])]
    ref = dedup.greedy(x, tau)
    assert ref["n_exact"] > 0
    _, rep, info = _ingest_async(lam, x, tau, 256)
    assert np.array_equal(rep, ref["rep"])
    assert abs(info.delta_hat_run - ref["delta_hat"]) <= 1e-12


def test_async_invalid_input_reported_later(lam):
    """A call that did not wait and met NaN leaves the store and its outputs
    untouched; the next waiting call reports it once; later calls are decided
    as if it had not happened."""
    rng = np.random.default_rng(3)
    x = synth.unit_rows(rng, 900, 64).astype(np.float32)
    bad = x[300:600].copy()
    bad[123, 7] = np.nan
    s = lam.Store(64, 0.95, 2000)
    r1, st1 = s.ingest(_dev(x[:300]), sync=False)
    assert st1 is None
    rb = torch.full((300,), -7, dtype=torch.int64, device="cuda")
    s.ingest(_dev(bad), rep=rb, sync=False)
    r3, _ = s.ingest(_dev(x[600:]), sync=False)
    with pytest.raises(lam.LamError) as e:
        s.info()
    assert e.value.name == "LAM_EINVAL"
    info = s.info()   # reported once
    good = np.concatenate([x[:300], x[600:]])
    ref = dedup.greedy(good, 0.95)
    assert info.n_seen == 600 and info.size == int(np.count_nonzero(ref["rep"] < 0))
    assert np.array_equal(torch.cat([r1, r3]).cpu().numpy(), ref["rep"])
    assert (rb.cpu().numpy() == -7).all()


def _small_rows(rng, n, d):
    """Unit rows whose coordinates all lie near 1/sqrt(d) in magnitude."""
    v = np.sign(rng.standard_normal((n, d))) + 0.1 * rng.standard_normal((n, d))
    return (v / np.linalg.norm(v, axis=1, keepdims=True)).astype(np.float32)


def test_store_codec_width_follows_retained_rows(lam):
    """The store codec's measured absmax is max |x| over the retained rows
    only: a dropped near-duplicate with a larger coordinate, an invalid call
    that did not wait and a cleared store's old rows must not count.  The
    magnitudes make each of those mistakes change the code width."""
    rng = np.random.default_rng(11)
    d, tau, eps = 64, 0.95, 1e-3
    u = _small_rows(rng, 1, d - 1)[0]
    def planted(c0):
        r = np.zeros(d, np.float64)
        r[0] = c0
        r[1:] = np.sqrt(1.0 - c0 * c0) * u
        return r.astype(np.float32)
    keep_big, drop_bigger = planted(0.5), planted(0.6)       # cos 0.993: the second is dropped
    x = np.concatenate([_small_rows(rng, 300, d), keep_big[None], _small_rows(rng, 200, d),
                        drop_bigger[None], _small_rows(rng, 100, d)])
    bad = _small_rows(rng, 50, d)
    bad[3] = planted(0.9)
    bad[7, 5] = np.nan
    s = lam.Store(d, tau, 2000)
    s.ingest(_dev(x[:250]), sync=False)
    s.ingest(_dev(bad), sync=False)
    with pytest.raises(lam.LamError):
        s.info()                                  # the invalid call is reported once
    s.ingest(_dev(x[250:500]), sync=False)
    s.ingest(_dev(x[500:]))                       # a call that waits
    ref = dedup.greedy(x, tau)
    kept = ref["kept"]
    assert ref["rep"][501] == 300                 # the planted pair merged
    p = s.quantize(eps)
    a = np.abs(x[kept]).max()
    assert p.absmax == a == np.float32(0.5)
    assert p.bits == qeps.plan(eps, float(a))["bits"] == 9
    assert np.array_equal(s.codes().cpu().numpy().view(np.uint32), qeps.pack(qeps.codes(x[kept], eps), p.bits))
    q = _small_rows(rng, 8, d)
    gs, gi, _ = s.score_topk(_dev(q), 5)
    S = score.scores(q, qeps.codes(x[kept], eps).reshape(kept.size, -1), eps)
    want_s, want_i = score.topk(S, kept, 5)
    assert np.array_equal(gi.cpu().numpy(), want_i)
    assert np.all(np.abs(gs.cpu().numpy() - want_s) <= 1e-5)

    s.clear()
    y = _small_rows(rng, 400, d)
    s.ingest(_dev(y), sync=False)
    refy = dedup.greedy(y, tau)
    p = s.quantize(eps)
    a = np.abs(y[refy["kept"]]).max()
    assert p.absmax == a and a < 0.2
    assert p.bits == qeps.plan(eps, float(a))["bits"] == 8
    assert np.array_equal(s.codes().cpu().numpy().view(np.uint32),
                          qeps.pack(qeps.codes(y[refy["kept"]], eps), p.bits))


@pytest.mark.parametrize("tau", [0.95, 0.99])
def test_removal_ceiling_subset(lam, tau):
    """Theorem "removal ceiling" on the subset stream: both greedy passes
    (tau and 4 tau - 3) match the oracle's counts exactly."""
    x = synth.subset_ingest()["x"]
    ref = dedup.removal_ceiling(x, tau)
    got = lam.removal_ceiling(_dev(x), tau, batch=1024)
    for key in ("n", "kept", "kept_2delta", "tau_2delta", "removal", "ceiling", "bits_lo", "bits_hi"):
        assert got[key] == ref[key], key
    assert got["delta_hat"] <= dedup.delta(tau) and got["delta_hat_2delta"] <= 2 * dedup.delta(tau)
    print(f"tau={tau}: removal {got['removal']:.4f} ceiling {got['ceiling']:.4f} "
          f"({got['frac_of_ceiling']:.3f} of it), bits [{got['bits_lo']:.3f}, {got['bits_hi']:.3f}]")


def test_removal_ceiling_errors(lam):
    x = _dev(np.eye(64, dtype=np.float32)[:10])
    for tau in (0.5, 1.5, float("nan")):
        with pytest.raises(lam.LamError) as e:
            lam.removal_ceiling(x, tau)
        assert e.value.name == "LAM_EINVAL"
    r = lam.removal_ceiling(x, 0.6, batch=3)
    assert (r["kept"], r["kept_2delta"]) == (10, 1)


def test_largest_accepted_coordinates(lam):
    """Coordinates just below the accepted limit (|x| < 255.9375, where 2^8 x
    is still a finite float16) are screened with a finite operand: a near
    copy of such a row merges, a sign-flipped one and the unit rows do not,
    exactly as the oracle decides."""
    rng = np.random.default_rng(8)
    u = synth.unit_rows(rng, 40, 64).astype(np.float32)
    big = u[:4].copy()
    big[:, 0] = np.float32(255.93)
    near = big.copy()
    near[:, 1] += np.float32(0.05)
    flip = big.copy()
    flip[:, 0] = -flip[:, 0]
    x = np.concatenate([u[4:20], big, near, flip, u[20:]])
    ref = dedup.greedy(x, 0.95)
    s = lam.Store(64, 0.95, x.shape[0])
    rep, st = s.ingest(_dev(x))
    assert np.array_equal(rep.cpu().numpy(), ref["rep"])
    assert np.all(ref["rep"][20:24] == np.arange(16, 20))   # the near copies merge into the big rows
    assert abs(st["delta_hat_run"] - ref["delta_hat"]) <= 1e-12


def test_store_maxima_after_calls_that_wait_and_calls_that_do_not(lam):
    """The store's max |x| and max ||x||^2 / 2, kept by the appends, cover
    every retained row when calls that do not wait are followed by one that
    waits (it settles the earlier calls first, then appends its own rows): the
    store's codec then takes the exact maximum as its absmax."""
    rng = np.random.default_rng(21)
    x = synth.unit_rows(rng, 3000, 128).astype(np.float32)
    x[2900, 5] = np.float32(0.9)      # the largest coordinate arrives in the last call
    s = lam.Store(128, 0.95, x.shape[0])
    xd = _dev(x)
    s.ingest(xd[:1000], sync=False)
    s.ingest(xd[1000:2000], sync=False)
    rep, _ = s.ingest(xd[2000:])      # waits
    p = s.quantize(1e-3)              # absmax measured: the appends' maximum
    ref = dedup.greedy(x, 0.95)
    kept = ref["kept"]
    assert p.absmax == float(np.abs(x[kept]).max()) == np.float32(0.9)
    assert np.array_equal(rep.cpu().numpy(), ref["rep"][2000:])


def test_store_quantize_declared_absmax_against_store_maximum(lam):
    """With a declared absmax the store's exact maximum |x| decides ERANGE
    before any code is written (the largest coordinate arrives in a call that
    does not wait); the failed call leaves the store unquantized, and the exact
    maximum itself is accepted."""
    rng = np.random.default_rng(22)
    x = synth.unit_rows(rng, 2000, 128).astype(np.float32)
    x[1500, 7] = np.float32(0.75)
    s = lam.Store(128, 0.95, x.shape[0])
    xd = _dev(x)
    s.ingest(xd[:1000], sync=False)
    s.ingest(xd[1000:], sync=False)
    ref = dedup.greedy(x, 0.95)
    kept = ref["kept"]
    a = np.abs(x[kept]).max()
    assert a == np.float32(0.75)
    below = float(np.nextafter(np.float32(0.75), np.float32(0)))
    with pytest.raises(lam.LamError) as e:
        s.quantize(1e-3, absmax=below)
    assert e.value.name == "LAM_ERANGE"
    with pytest.raises(lam.LamError) as e:
        s.score_topk(_dev(x[:4]), 3)
    assert e.value.name == "LAM_ESTATE"
    p = s.quantize(1e-3, absmax=0.75)
    assert p.absmax == np.float32(0.75)
    assert np.array_equal(s.codes().cpu().numpy().view(np.uint32), qeps.pack(qeps.codes(x[kept], 1e-3), p.bits))
    assert s.info().size == kept.size


def test_clear_resets_bookkeeping_and_pending_errors(lam):
    """lam_store_clear drops the error report of a pending invalid call and
    resets the device bookkeeping before the next ingest uses it: the next
    stream's ids start at 0, its delta_hat and its codec width are its own."""
    cfg = synth.subset_ingest()
    x, y = cfg["x"][:3000], cfg["x"][3000:7000]
    s = lam.Store(768, 0.95, 8000)
    s.ingest(_dev(x), sync=False)
    bad = x[:64].copy()
    bad[5, 3] = np.nan
    s.ingest(_dev(bad), sync=False)
    s.clear()
    info = s.info()                      # no error: the pending report was dropped
    assert (info.size, info.n_seen, info.delta_hat_run) == (0, 0, 0.0)
    reps = [s.ingest(_dev(y[b0:b0 + 1000]), sync=False)[0] for b0 in range(0, y.shape[0], 1000)]
    ref = dedup.greedy(y, 0.95, block=512)
    assert np.array_equal(torch.cat(reps).cpu().numpy(), ref["rep"])
    info = s.info()
    assert info.size == int(ref["kept"].size) and info.n_seen == y.shape[0]
    assert abs(info.delta_hat_run - ref["delta_hat"]) <= 1e-12
    p = s.quantize(1e-3)
    assert p.absmax == np.abs(y[ref["kept"]]).max()
