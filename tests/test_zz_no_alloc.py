"""The allocation-free scoring entry point (lam_score_topk_noalloc) against
lam_score_topk: the same kernels on a fixed per-device workspace, so scores,
ids and bounds must be identical, on two calls in a row (the second with fewer
queries, so the workspace holds the first call's leftovers), for a store small
enough for the single-pass plan and one large enough for the threshold plan
at k = 10 and k = 50; and the query limit is checked on the host."""
import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu


def _store(lam, n, d, seed):
    g = torch.Generator(device="cuda").manual_seed(seed)
    x = torch.randn((n, d), generator=g, device="cuda", dtype=torch.float64)
    x = (x / x.norm(dim=1, keepdim=True)).to(torch.float32).contiguous()
    s = lam.Store(d, 0.95, n)
    for b0 in range(0, n, 4096):
        s.ingest(x[b0:b0 + 4096], sync=False)
    s.quantize(1e-3)
    s.info()   # settles the calls that did not wait
    return s, g


def _queries(g, nq, d):
    q = torch.randn((nq, d), generator=g, device="cuda", dtype=torch.float64)
    return (q / q.norm(dim=1, keepdim=True)).to(torch.float32).contiguous()


def _outs(nq, k):
    return (torch.full((nq, k), 7.0, dtype=torch.float32, device="cuda"),
            torch.full((nq, k), -7, dtype=torch.int64, device="cuda"),
            torch.full((nq,), 7.0, dtype=torch.float32, device="cuda"))


@pytest.mark.parametrize("n,d,k", [(3000, 128, 10), (20000, 768, 10), (20000, 768, 50)])
def test_noalloc_equals_score_topk(lam, n, d, k):
    s, g = _store(lam, n, d, seed=n + k)
    for nq in (256, 37):   # the second call is smaller
        q = _queries(g, nq, d)
        want = s.score_topk(q, k)
        got = s.score_topk_noalloc(q, k, out=_outs(nq, k))
        torch.cuda.synchronize()
        for w, h in zip(want, got):
            assert torch.equal(w, h), (n, d, k, nq)
        assert np.all(got[1].cpu().numpy() >= 0)


def test_noalloc_limits(lam):
    s, g = _store(lam, 500, 64, seed=5)
    q = _queries(g, 257, 64)
    with pytest.raises(lam.LamError) as e:
        s.score_topk_noalloc(q, 5, out=_outs(257, 5))
    assert e.value.name == "LAM_EINVAL"
    # an empty call is accepted and writes nothing
    out = _outs(0, 5)
    s.score_topk_noalloc(q[:0], 5, out=out)
