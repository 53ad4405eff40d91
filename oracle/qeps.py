"""Oracle for the quantizer Q_eps -- test infrastructure only.

Paper, Section 2.2 ("Three layers", L1): each coordinate is quantized as
Q_eps(x) = round(x / 2 eps).  The step is s = 2 eps, so the reconstruction
x_hat = q * s is within eps of x in every coordinate (Section 2.1 and
Appendix "Rank invariance, in full": cell-mates differ by at most 2 eps per
coordinate).

Readings taken where the paper is silent:
  * round() is round-half-to-even of the exact real quotient x / s, where x is
    the float32 input and s = 2*eps is the binary64 doubling of eps;
  * codes are integers of the narrowest two's-complement width b that holds
    +-M, M = Q_eps(A) for the declared (or measured) absmax A:
    b = max(1, ceil(log2(2M + 1))) in "bits" mode, or the smallest of
    {8, 16, 32} in "bytes" mode; M >= 2^31 is out of range;
  * element i occupies bits [i*b, (i+1)*b) of a little-endian stream of uint32
    words, least significant bit first; unused tail bits are zero;
  * decode materialises x_hat as float32(float64(q * s)), i.e. round-to-nearest
    to binary64, then to binary32; the bound is stated on the exact q * s.
"""
from __future__ import annotations

from fractions import Fraction

import numpy as np

BITS, BYTES = "bits", "bytes"


def step(eps: float) -> float:
    """s = 2 eps (exact in binary64)."""
    return 2.0 * float(eps)


# ---------------------------------------------------------------- definition
def q_exact(x: float, eps: float) -> int:
    """Q_eps of one float32 value, on exact rationals (Python's round() of a
    Fraction rounds half to even)."""
    return round(Fraction(float(np.float32(x))) / Fraction(step(eps)))


def codes_exact(x, eps: float) -> np.ndarray:
    """Q_eps elementwise by the exact definition (pure Python; small inputs)."""
    xs = np.asarray(x, dtype=np.float32).ravel().tolist()
    s = Fraction(step(eps))
    return np.array([round(Fraction(v) / s) for v in xs], dtype=np.int64)


# ---------------------------------------------------------------- vectorised
def codes(x, eps: float) -> np.ndarray:
    """Q_eps elementwise.  The binary64 quotient is correctly rounded, so
    rint() of it equals the exact result except when a half-integer lies
    within two ulps of it; those elements are recomputed exactly."""
    x = np.asarray(x, dtype=np.float32).ravel()
    if not np.all(np.isfinite(x)):
        raise ValueError("non-finite input")
    s = step(eps)
    qf = x.astype(np.float64) / s
    q = np.rint(qf)
    frac = qf - np.floor(qf)
    near = np.abs(frac - 0.5) <= 4.0 * np.spacing(np.abs(qf))
    out = q.astype(np.int64)
    idx = np.nonzero(near)[0]
    if idx.size:
        sf = Fraction(s)
        out[idx] = [round(Fraction(float(x[i])) / sf) for i in idx.tolist()]
    return out


def max_code(absmax: float, eps: float) -> int:
    """M = Q_eps(A) for the absmax A (float32); Q_eps is monotone, so every
    |code| of an input with |x| <= A is at most M."""
    return q_exact(abs(float(np.float32(absmax))), eps)


def width(m: int, mode: str = BITS) -> int:
    """Narrowest two's-complement width holding +-m."""
    if m < 0 or m >= 2 ** 31:
        raise ValueError("code range out of 32 bits")
    b = max(1, int(m).bit_length() + 1)          # == ceil(log2(2m + 1)), at least 1
    if mode == BITS:
        return b
    if mode == BYTES:
        return next(w for w in (8, 16, 32) if w >= b)
    raise ValueError(mode)


def plan(eps: float, absmax: float, mode: str = BITS):
    m = max_code(absmax, eps)
    return dict(eps=float(eps), step=step(eps), max_code=m, bits=width(m, mode), mode=mode)


# ---------------------------------------------------------------- packing
def pack_exact(q, b: int) -> np.ndarray:
    """The packed stream by its definition: one big integer, element i at bit
    i*b, then cut into 32-bit little-endian words."""
    q = np.asarray(q, dtype=np.int64).ravel().tolist()
    mask = (1 << b) - 1
    acc = 0
    for i, c in enumerate(q):
        acc |= (c & mask) << (i * b)
    nwords = (len(q) * b + 31) // 32
    return np.array([(acc >> (32 * w)) & 0xFFFFFFFF for w in range(nwords)], dtype=np.uint32)


def pack(q, b: int) -> np.ndarray:
    """Vectorised form of ``pack_exact``.  Bit fields of different elements are
    disjoint, so summing them (exactly, in float64 below 2^53) equals OR-ing."""
    q = np.asarray(q, dtype=np.int64).ravel()
    n = q.size
    nwords = (n * b + 31) // 32
    if n == 0:
        return np.zeros(0, dtype=np.uint32)
    u = (q & ((1 << b) - 1)).astype(np.uint64)
    pos = np.arange(n, dtype=np.int64) * b
    w = pos >> 5
    v = u << (pos & 31).astype(np.uint64)
    lo = (v & np.uint64(0xFFFFFFFF)).astype(np.float64)
    hi = (v >> np.uint64(32)).astype(np.float64)
    acc = np.bincount(w, weights=lo, minlength=nwords + 1)
    acc += np.bincount(w + 1, weights=hi, minlength=nwords + 1)
    return acc[:nwords].astype(np.uint64).astype(np.uint32)


def unpack(words, b: int, n: int) -> np.ndarray:
    """Inverse of ``pack``: sign-extended int64 codes."""
    words = np.asarray(words, dtype=np.uint32)
    w64 = np.concatenate([words.astype(np.uint64), np.zeros(1, np.uint64)])
    pos = np.arange(n, dtype=np.int64) * b
    wi = pos >> 5
    v = w64[wi] | (w64[wi + 1] << np.uint64(32))
    u = ((v >> (pos & 31).astype(np.uint64)) & np.uint64((1 << b) - 1)).astype(np.int64)
    return u - ((u >> (b - 1)) & 1) * (1 << b)


# ---------------------------------------------------------------- decode, bound
def decode(q, eps: float) -> np.ndarray:
    """x_hat = float32(float64(q * s))."""
    return (np.asarray(q, dtype=np.int64).astype(np.float64) * step(eps)).astype(np.float32)


def bound_violations(x, q, eps: float) -> int:
    """Number of elements with |x - q*s| > eps on exact reals
    (equivalently, q is not a nearest integer to x/s)."""
    x = np.asarray(x, dtype=np.float32).ravel()
    q = np.asarray(q, dtype=np.int64).ravel()
    s = step(eps)
    qf = x.astype(np.float64) / s
    r = np.abs(qf - q)                          # |x/s - q| up to a few ulps of x/s
    tol = 1e-12 + 4.0 * np.spacing(np.abs(qf))
    bad = r > 0.5 + tol
    unsure = np.abs(r - 0.5) <= tol
    n_bad = int(np.count_nonzero(bad))
    sf = Fraction(s)
    for i in np.nonzero(unsure)[0].tolist():
        if abs(Fraction(float(x[i])) / sf - int(q[i])) > Fraction(1, 2):
            n_bad += 1
    return n_bad


def encode(x, eps: float, absmax: float | None = None, mode: str = BITS):
    """Q_eps plan + codes + packed words; raises ValueError on non-finite input
    or |x| > absmax (codes never saturate)."""
    x = np.asarray(x, dtype=np.float32).ravel()
    if not np.all(np.isfinite(x)):
        raise ValueError("non-finite input")
    a = float(np.max(np.abs(x))) if absmax is None else float(np.float32(absmax))
    if x.size and float(np.max(np.abs(x))) > a:
        raise ValueError("|x| exceeds the declared absmax")
    p = plan(eps, a, mode)
    q = codes(x, eps)
    return pack(q, p["bits"]), q, p
