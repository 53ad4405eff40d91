"""The large online-store workload at its full size -- 1,048,576 rows of
D = 1,024 (16,384 clusters plus 20 % planted near-duplicates) streamed in
batches of 4,096 at tau = 0.95 with calls that do not wait, the store coded at
eps = 1e-3, and 16,384 queries scored top-50 -- checked on sampled outputs the
oracle computes one by one, and on properties that hold at any size.

The rows are drawn on the device (synth.online_store_device: the same recipe
as synth.online_store, whose host draw takes minutes at this size).
"""
import numpy as np
import pytest
import torch

import synth
from oracle import dedup, qeps, score

pytestmark = pytest.mark.gpu
TOL = 1e-5


@pytest.fixture(scope="module")
def run(lam):
    cfg = synth.online_store_device(device="cuda")
    x, q = cfg["x"], cfg["q"]
    n, d = x.shape
    tau, eps, k, batch = cfg["tau"], cfg["eps"], cfg["k"], cfg["batch"]
    print(f"online store: {cfg['name']}", flush=True)
    s = lam.Store(d, tau, n)
    reps = []
    for b0 in range(0, n, batch):
        reps.append(s.ingest(x[b0:b0 + batch], sync=False)[0])
    info = s.info()
    rep = torch.cat(reps).cpu().numpy()
    print(f"ingested: kept {info.size} of {n}, delta_hat {info.delta_hat_run:.6f}", flush=True)
    p = s.quantize(eps)
    gs, gi, gb = s.score_topk(q, k)
    torch.cuda.synchronize()
    out = dict(x=x.cpu().numpy(), q=q.cpu().numpy(), rep=rep, info=info, p=p, ids=s.ids().cpu().numpy(),
               codes=s.codes().cpu().numpy().view(np.uint32), gs=gs.cpu().numpy(), gi=gi.cpu().numpy(),
               gb=gb.cpu().numpy(), tau=tau, eps=eps, k=k)
    del s
    torch.cuda.empty_cache()
    return out


def test_store_bookkeeping(run):
    rep, info = run["rep"], run["info"]
    kept = np.nonzero(rep < 0)[0]
    assert info.n_seen == rep.size and info.size == kept.size
    assert np.array_equal(run["ids"], kept)            # retained ids ascending, in arrival order
    dropped = np.nonzero(rep >= 0)[0]
    assert np.all(rep[dropped] < dropped)              # representatives arrived earlier ...
    assert np.all(rep[rep[dropped]] == -1)             # ... and were retained
    assert info.delta_hat_run <= dedup.delta(run["tau"])
    print(f"kept fraction {kept.size / rep.size:.4f}")


def test_sampled_decisions(run):
    """Decisions of 1,024 arrivals, four from each of the 256 batches, and of
    64 more dropped ones, recomputed by the oracle against the retained set at
    their arrival."""
    x, rep, tau = run["x"], run["rep"], run["tau"]
    rng = np.random.default_rng(2)
    n = rep.size
    batch = 4096
    per_batch = np.concatenate([b0 + rng.choice(min(batch, n - b0), 4, replace=False) for b0 in range(0, n, batch)])
    samples = np.unique(np.concatenate([per_batch, rng.choice(np.nonzero(rep >= 0)[0], 64, replace=False)]))
    assert samples.size >= 1024
    kept = np.nonzero(rep < 0)[0]
    want = dedup.decide_many(x, samples, kept, tau)
    assert np.array_equal(rep[samples], want), samples[rep[samples] != want]
    print(f"{samples.size} sampled decisions equal the oracle's ({np.count_nonzero(want >= 0)} dropped)")


def test_cover_on_dropped_sample(run):
    """Every sampled dropped arrival is within delta of its representative
    (Proposition "greedy is a cover"), and delta_hat bounds the distances."""
    x, rep, tau = run["x"], run["rep"], run["tau"]
    rng = np.random.default_rng(3)
    dropped = np.nonzero(rep >= 0)[0]
    pick = rng.choice(dropped, min(4000, dropped.size), replace=False)
    a = x[pick].astype(np.float64)
    b = x[rep[pick]].astype(np.float64)
    d2 = np.sum((a - b) ** 2, axis=1)
    d2f = float(dedup.delta2(tau))
    near = np.abs(d2 - d2f) <= 1e-9
    assert np.all((d2 <= d2f) | near)
    for i in pick[near]:
        assert dedup.within(x[i], x[rep[i]], tau)
    assert np.sqrt(d2.max()) <= run["info"].delta_hat_run * (1 + 1e-12)


def test_store_codes_sampled_rows(run):
    """Q_eps codes of sampled retained rows equal the oracle's, bit for bit."""
    x, ids, p = run["x"], run["ids"], run["p"]
    d = x.shape[1]
    rng = np.random.default_rng(4)
    rows = np.sort(rng.choice(ids.size, 3000, replace=False))
    ref = qeps.codes(x[ids[rows]], run["eps"]).reshape(rows.size, d)
    words_per_row = d * p.bits // 32
    got = np.stack([qeps.unpack(run["codes"][r * words_per_row:(r + 1) * words_per_row], p.bits, d)
                    for r in rows])
    assert np.array_equal(got, ref)
    assert p.bits == qeps.plan(run["eps"], float(np.abs(x[ids]).max()))["bits"]


def test_sampled_queries_topk(run):
    """Top-50 of 256 sampled queries against the oracle over every retained
    row."""
    x, q, ids, eps, k = run["x"], run["q"], run["ids"], run["eps"], run["k"]
    gs, gi, gb = run["gs"], run["gi"], run["gb"]
    rng = np.random.default_rng(5)
    qs = np.sort(rng.choice(q.shape[0], 256, replace=False))
    ts, ti, beta = score.score_topk_blocked(q[qs], x[ids], ids, eps, k)
    xs = set(ids.tolist())
    for n_, j in enumerate(qs):
        assert len(set(gi[j].tolist())) == k and all(int(v) in xs for v in gi[j])
        cg = qeps.codes(x[gi[j]], eps).reshape(k, -1)
        sg = score.scores(q[j:j + 1], cg, eps)[0]
        assert np.all(np.abs(gs[j].astype(np.float64) - sg) <= TOL)
        assert np.all(sg >= ts[n_, k - 1] - 2 * TOL)
        sj = np.concatenate([[np.inf], ts[n_], [-np.inf]])
        sep = np.array([(sj[p] - sj[p + 1] > 2 * TOL) and (sj[p + 1] - sj[p + 2] > 2 * TOL) for p in range(k)])
        assert np.array_equal(gi[j][sep], ti[n_][sep])
    gbn = gb[qs].astype(np.float64)
    assert np.all(gbn >= beta) and np.all(gbn - beta <= np.spacing(gbn.astype(np.float32)))
