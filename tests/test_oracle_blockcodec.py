"""Pins for the per-block codec oracle (CPU): the zigzag map and block widths
by their definitions, packing against the Q_eps oracle's definitional packer,
closed-form sizes, and the round trip."""
import numpy as np

import synth
from oracle import blockcodec, qeps


def test_zigzag_definition_and_inverse():
    q = np.arange(-600, 601)
    u = blockcodec.zigzag(q)
    assert u.tolist() == [2 * v if v >= 0 else -2 * v - 1 for v in q.tolist()]
    assert sorted(u.tolist()) == list(range(1201))          # a bijection onto [0, 1200]
    assert np.array_equal(blockcodec.unzigzag(u), q)


def test_widths_closed_forms():
    d = 64
    c = np.zeros((3, d), dtype=np.int64)
    c[1, 0] = -1            # u = 1 -> 1 bit
    c[1, 40] = 3            # u = 6 -> 3 bits
    c[2, :32] = 511         # u = 1022 -> 10 bits
    c[2, 32:] = -512        # u = 1023 -> 10 bits
    e = blockcodec.encode(c)
    assert e["widths"].tolist() == [[0, 0], [1, 3], [10, 10]]
    assert e["row_off"].tolist() == [0, 0, 4, 24]          # all-zero blocks cost no words
    assert e["data"][:4].tolist() == [1, 0, 1 << 8, 1 << 8]   # -1 -> u 1 (code 0); 3 -> u 6 (code 8, planes 1, 2)
    assert np.array_equal(blockcodec.decode(e, d), c)
    s = blockcodec.sizes(e, c.size)
    assert s["data_bytes"] == 24 * 4 and s["meta_bytes"] == 6 + 4 * 8


def test_block_words_are_bit_planes():
    """Word t of a block, read as an integer, is sum_j bit_t(u_j) 2^j -- checked
    on a hand example and against a big-integer transpose on random blocks."""
    u = np.zeros(32, dtype=np.int64)
    u[0], u[5], u[31] = 1, 6, 5          # 0b1, 0b110, 0b101
    assert blockcodec.bitplanes(u, 3).tolist() == [(1 << 0) | (1 << 31), 1 << 5, (1 << 5) | (1 << 31)]
    rng = np.random.default_rng(0)
    c = rng.integers(-300, 301, size=(5, 96))
    e = blockcodec.encode(c)
    off = 0
    for r in range(5):
        for k in range(3):
            w = int(e["widths"][r, k])
            uu = blockcodec.zigzag(c[r, 32 * k:32 * (k + 1)])
            assert w == max(int(v).bit_length() for v in uu)
            # transpose through one big integer: bit (t * 32 + j) = bit t of u_j
            big = 0
            for j, v in enumerate(uu.tolist()):
                for t in range(w):
                    big |= ((v >> t) & 1) << (t * 32 + j)
            assert e["data"][off:off + w].tolist() == [(big >> (32 * t)) & 0xFFFFFFFF for t in range(w)]
            off += w


def test_round_trip_on_store_codes():
    t = synth.tiny_ingest()
    x = t["x"][:500]
    c = qeps.codes(x, 1e-3).reshape(x.shape)
    e = blockcodec.encode(c)
    assert np.array_equal(blockcodec.decode(e, x.shape[1]), c)
    s = blockcodec.sizes(e, c.size)
    b = qeps.plan(1e-3, float(np.abs(x).max()))["bits"]
    assert s["bits_per_code"] < b              # blocks narrower than the global width pay for the metadata
