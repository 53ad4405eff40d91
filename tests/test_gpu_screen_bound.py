"""Empirical pin of the screen's error bound (the stated delta of the
decisions): pairs planted around the merge threshold, a third of them inside
the band the screen leaves to the exact test and the rest just outside it,
where the screen's fp16 MFMA decision stands alone.  Every decision must equal the exact
predicate (Eq. identity, Alg. "admit"); a bound that understated the screen's
error would turn some of the outside pairs the wrong way.

Rows (synth.threshold_band_device, drawn on the device): 200,000 unit rows a_i
(Gaussian, and a heavy-tailed half whose coordinates span several binades of
fp16), all mutually far apart (largest cosine about 0.27), ingested first;
then one arrival b_i per a_i at cosine tau + U(-3e-3, 3e-3) to a_i.  The
screen's band is about +-1.1e-3 in cosine for unit rows at D = 768, so about a
third of the pairs are ambiguous and the rest are decided by the screen.
"""
import numpy as np
import pytest
import torch

import synth
from oracle import dedup

pytestmark = pytest.mark.gpu
N = 200_000
D = 768
TAU = 0.95


def _exact_within(a, b, tau):
    """The exact predicate for row pairs: binary64 squared distances (error
    below 1e-13 here) decide all but pairs within 1e-10 of delta^2, which take
    the rational definition."""
    d2 = np.sum((a.astype(np.float64) - b.astype(np.float64)) ** 2, axis=1)
    d2f = float(dedup.delta2(tau))
    out = d2 <= d2f
    for i in np.nonzero(np.abs(d2 - d2f) <= 1e-10)[0]:
        out[i] = dedup.within(a[i], b[i], tau)
    return out, d2


def test_decisions_near_the_threshold(lam):
    ad, bd = synth.threshold_band_device(seed=21, n=N, d=D, tau=TAU, spread=3e-3)
    xd = torch.cat([ad, bd])
    a, b = ad.cpu().numpy(), bd.cpu().numpy()
    print(f"screen bound pin: {N} pairs at cosine {TAU} +- 3e-3, D = {D}", flush=True)
    s = lam.Store(D, TAU, 2 * N)
    reps, amb, margin = [], 0, float("inf")
    for b0 in range(0, 2 * N, 4096):
        rep, st = s.ingest(xd[b0:b0 + 4096])
        reps.append(rep)
        amb += st["n_ambiguous_pairs"]
        margin = min(margin, st["min_margin_d2"])
    rep = torch.cat(reps).cpu().numpy()
    # the a rows are far apart: all kept
    assert np.all(rep[:N] == -1)
    want, d2 = _exact_within(a, b, TAU)
    got = rep[N:]
    assert np.all((got == -1) | (got == np.arange(N)))   # only the planted partner can represent b_i
    assert np.array_equal(got == np.arange(N), want), np.nonzero((got == np.arange(N)) != want)[0][:10]
    # the screen left the pairs near the threshold to the exact test
    d2f = float(dedup.delta2(TAU))
    inner = int(np.count_nonzero(np.abs(d2 - d2f) <= 1e-3))
    assert inner <= amb <= N
    # the smallest margin the exact test saw is the planted pairs' smallest
    assert abs(margin - np.min(np.abs(d2 - d2f))) <= 1e-12
    print(f"merged {int(want.sum())} of {N}; ambiguous pairs {amb}; pairs within 1e-3 of delta^2 in d^2: {inner}")
