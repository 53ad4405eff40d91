"""GPU parity of the per-block codec of the store's codes against the oracle
(oracle/blockcodec.py): widths, row offsets and bit-plane words bit for bit,
decode equal to the store's Q_eps decode, scores equal to the fixed-width
scorer's, sizes and ratios as defined."""
import numpy as np
import pytest
import torch

import synth
from test_gpu_score import _compare
from oracle import blockcodec, dedup, qeps

pytestmark = pytest.mark.gpu


def _dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def _store(lam, x, tau, eps, batch=1024, spare=0):
    s = lam.Store(x.shape[1], tau, x.shape[0] + spare)
    xd = _dev(x)
    for b0 in range(0, x.shape[0], batch):
        s.ingest(xd[b0:b0 + batch])
    p = s.quantize(eps)
    return s, p


@pytest.fixture(scope="module")
def subset():
    cfg = synth.subset_ingest()
    return cfg, dedup.greedy(cfg["x"], 0.95)


@pytest.mark.parametrize("eps", [1e-2, 1e-3, 1e-4])
def test_subset_store_blocks_bit_exact(lam, subset, eps):
    """The whole 27,986-row subset stream at tau = 0.95, its store coded at
    each eps: the fixed-width codes and the block encoding equal the oracle's
    bit for bit, and top-10 scores of the stream's 1,024 queries match the
    oracle's."""
    cfg, ref = subset
    x = cfg["x"]
    s, p = _store(lam, x, 0.95, eps)
    kept = s.ids().cpu().numpy()
    assert np.array_equal(kept, ref["kept"])
    codes = qeps.codes(x[kept], eps).reshape(kept.size, -1)
    assert p.bits == qeps.plan(eps, float(np.abs(x[kept]).max()))["bits"]
    assert np.array_equal(s.codes().cpu().numpy().view(np.uint32), qeps.pack(codes, p.bits))
    ref = blockcodec.encode(codes)
    st = s.block_encode()
    w, ro, d = s.block_export()
    assert np.array_equal(w.cpu().numpy(), ref["widths"])
    assert np.array_equal(ro.cpu().numpy().astype(np.uint64), ref["row_off"])
    assert np.array_equal(d.cpu().numpy().view(np.uint32), ref["data"])
    sz = blockcodec.sizes(ref, codes.size)
    assert st["data_bytes"] == sz["data_bytes"] and st["meta_bytes"] == sz["meta_bytes"]
    assert st["bits_per_code"] == pytest.approx(sz["bits_per_code"], rel=1e-12)
    assert st["plain_bits"] == p.bits
    assert st["composite_ratio"] == pytest.approx(x.shape[0] * x.shape[1] * 4 / sz["total_bytes"], rel=1e-12)
    # lossless: the decode is the store's Q_eps decode, bit for bit
    assert torch.equal(s.block_decode(), s.dequantize())
    q = cfg["q"]
    gs, gi, _ = s.score_topk(torch.from_numpy(q).cuda(), 10)
    worst = _compare(gs.cpu().numpy(), gi.cpu().numpy(), codes, kept, q, eps, 10)
    assert worst <= 1e-5
    print(f"eps={eps}: b={p.bits}, {st['bits_per_code']:.3f} bits/code, codec x{st['codec_ratio']:.2f}, "
          f"composite x{st['composite_ratio']:.2f}")


def test_scores_from_blocks_equal_fixed_width(lam):
    t = synth.tiny_ingest()
    s, p = _store(lam, t["x"], t["tau"], t["eps"])
    s.block_encode()
    q = _dev(t["q"])
    for k in (1, 10, 64):
        a = s.score_topk(q, k)
        b = s.score_topk_blocks(q, k)
        assert all(torch.equal(u, v) for u, v in zip(a, b))


def test_zero_blocks_and_state(lam):
    """All-zero rows cost no data words; a stale encoding is refused."""
    rng = np.random.default_rng(3)
    x = synth.unit_rows(rng, 40, 96).astype(np.float32)
    x[5] = 0.0
    s, p = _store(lam, x, 1.0, 1e-3, spare=4)
    st = s.block_encode()
    w, ro, d = s.block_export()
    ro = ro.cpu().numpy()
    kept = s.ids().cpu().numpy().tolist()
    r5 = kept.index(5)
    assert ro[r5 + 1] == ro[r5] and w.cpu().numpy()[r5].tolist() == [0, 0, 0]
    s.ingest(_dev(synth.unit_rows(rng, 1, 96).astype(np.float32)))
    s.quantize(1e-3)
    with pytest.raises(lam.LamError) as e:
        s.block_decode()
    assert e.value.name == "LAM_ESTATE"
    s.block_encode()
    assert torch.equal(s.block_decode(), s.dequantize())
