"""Oracle for the per-block fixed-length codec of the retained store -- test
infrastructure only.

Paper, Section 2.2 ("Three layers", L2) and Section "Composite reduction:
deduplication x byte codec": retained embeddings are compressed further by an
error-bounded byte codec, and the storage reductions of deduplication and of the
codec multiply.  The paper's codec is cuSZp; here the fixed-length block stage
is applied to the Q_eps codes themselves, so the decoded values are exactly the
Q_eps reconstruction and the score bound eps * ||q||_1 is unchanged.

Readings taken where the paper is silent:
  * a block is 32 consecutive codes of one row (rows hold dim / 32 blocks);
  * codes are mapped to unsigned integers by the zigzag map
    u = 2q for q >= 0 and -2q - 1 for q < 0, and a block is stored with the bit
    width w of its largest u (w = 0 when every u is zero, so an all-zero block
    costs no data words);
  * a block occupies exactly w 32-bit words in bit-plane (bit-shuffled) order:
    bit j of word t is bit t of code j's zigzag value, so each word is one bit
    plane of the block; blocks of a row follow each other, rows follow each
    other;
  * metadata: one byte (the width) per block and one 64-bit word offset per
    row; bits per code = (data words * 32 + blocks * 8 + rows * 64) / codes.
"""
from __future__ import annotations

import numpy as np

BLOCK = 32


def zigzag(q) -> np.ndarray:
    q = np.asarray(q, dtype=np.int64)
    return np.where(q >= 0, 2 * q, -2 * q - 1)


def unzigzag(u) -> np.ndarray:
    u = np.asarray(u, dtype=np.int64)
    return np.where(u % 2 == 0, u // 2, -(u + 1) // 2)


def width(u_block) -> int:
    """Bits of the largest value (0 for an all-zero block)."""
    return int(int(np.max(u_block)).bit_length()) if len(u_block) else 0


def bitplanes(u, w: int) -> np.ndarray:
    """The w bit planes of 32 unsigned values: word t has bit j = bit t of u[j]."""
    u = np.asarray(u, dtype=np.int64)
    assert u.size == BLOCK
    return np.array([sum(((int(u[j]) >> t) & 1) << j for j in range(BLOCK)) for t in range(w)],
                    dtype=np.uint32)


def encode(codes_rows):
    """codes_rows: (rows, dim) integer codes, dim a multiple of 32.  Returns
    dict(widths uint8 (rows, dim/32), row_off uint64 (rows + 1), data uint32)."""
    c = np.asarray(codes_rows, dtype=np.int64)
    rows, dim = c.shape
    assert dim % BLOCK == 0
    nb = dim // BLOCK
    u = zigzag(c).reshape(rows, nb, BLOCK)
    widths = np.zeros((rows, nb), dtype=np.uint8)
    parts = []
    row_off = np.zeros(rows + 1, dtype=np.uint64)
    off = 0
    for r in range(rows):
        row_off[r] = off
        for k in range(nb):
            w = width(u[r, k])
            widths[r, k] = w
            parts.append(bitplanes(u[r, k], w))
            off += w
    row_off[rows] = off
    data = np.concatenate(parts) if parts else np.zeros(0, np.uint32)
    return dict(widths=widths, row_off=row_off, data=data.astype(np.uint32))


def decode(enc, dim: int) -> np.ndarray:
    """Inverse of encode: (rows, dim) int64 codes."""
    widths, row_off, data = enc["widths"], enc["row_off"], enc["data"]
    rows, nb = widths.shape
    out = np.zeros((rows, dim), dtype=np.int64)
    for r in range(rows):
        off = int(row_off[r])
        for k in range(nb):
            w = int(widths[r, k])
            if w:
                planes = data[off:off + w].astype(np.int64)
                uu = np.zeros(BLOCK, dtype=np.int64)
                for t in range(w):
                    uu |= ((planes[t] >> np.arange(BLOCK)) & 1) << t
                out[r, k * BLOCK:(k + 1) * BLOCK] = unzigzag(uu)
            off += w
    return out


def sizes(enc, n_codes: int) -> dict:
    rows = enc["widths"].shape[0]
    data_bytes = int(enc["data"].size) * 4
    meta_bytes = int(enc["widths"].size) + (rows + 1) * 8
    total = data_bytes + meta_bytes
    return dict(data_bytes=data_bytes, meta_bytes=meta_bytes, total_bytes=total,
                bits_per_code=8.0 * total / n_codes if n_codes else 0.0)
