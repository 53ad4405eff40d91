"""Pins for the quantizer oracle (CPU).

Each test checks oracle.qeps against something fixed outside it: the exact
rational definition of Section 2.2 (L1), hand-worked values, the textbook
special case of a dyadic step, the per-element bound, and the paper's printed
2 eps sqrt(D) values.
"""
import math
import os
from fractions import Fraction

import numpy as np
import pytest

from oracle import qeps

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def _adversarial(rng, eps, n=2000):
    """Values at (k + 1/2) s and a few float32 ulps around it."""
    s = 2 * eps
    k = rng.integers(-3000, 3000, n)
    base = ((k + 0.5) * s).astype(np.float32)
    out = [base]
    for d in (1, 2):
        out.append(np.nextafter(base, np.float32(np.inf)))
        out.append(np.nextafter(base, np.float32(-np.inf)))
        base = out[-2]
    return np.concatenate(out)


@pytest.mark.parametrize("eps", [1e-4, 1e-3, 1e-2, 0.25, 2.0 ** -10, 3e-3])
def test_codes_match_exact_definition(eps):
    rng = np.random.default_rng(11)
    x = np.concatenate([
        rng.uniform(-1, 1, 4000).astype(np.float32),
        (0.04 * rng.standard_normal(4000)).astype(np.float32),
        _adversarial(rng, eps),
        np.array([0.0, -0.0, eps, -eps, 2 * eps, 3 * eps], dtype=np.float32),
    ])
    assert np.array_equal(qeps.codes(x, eps), qeps.codes_exact(x, eps))


def test_hand_worked_values():
    # eps = 0.25, s = 0.5: x/s = 0.5 -> 0 (tie to even), 1.5 -> 2, 2.5 -> 2,
    # -0.5 -> 0, -1.5 -> -2; the float32 just above 0.25 gives 1.
    x = np.array([0.25, 0.75, 1.25, -0.25, -0.75, np.nextafter(np.float32(0.25), np.float32(1))],
                 dtype=np.float32)
    assert qeps.codes(x, 0.25).tolist() == [0, 2, 2, 0, -2, 1]
    # eps = 1e-3: float32(0.001) = 0.00100000004749745 and binary64 0.002 is
    # 0.0020000000000000000416..., so x/s = 0.5000000237... rounds to 1,
    # although in decimal 0.001/0.002 is exactly one half.
    assert qeps.codes(np.array([0.001, -0.001], np.float32), 1e-3).tolist() == [1, -1]


@pytest.mark.parametrize("k", [1, 3, 8, 11, 20])
def test_dyadic_step_reduces_to_ldexp_rint(k):
    # eps = 2^-k: s = 2^(1-k) and x/s = ldexp(x, k-1) is exact, so Q_eps is the
    # textbook round-half-even of a scaled value.
    rng = np.random.default_rng(k)
    eps = 2.0 ** -k
    x = np.concatenate([rng.uniform(-1, 1, 20000), _adversarial(rng, eps)]).astype(np.float32)
    x = x[np.abs(x.astype(np.float64) / (2 * eps)) < 2 ** 30]
    ref = np.rint(np.ldexp(x.astype(np.float64), k - 1)).astype(np.int64)
    assert np.array_equal(qeps.codes(x, eps), ref)


@pytest.mark.parametrize("eps", [1e-4, 1e-3, 1e-2])
def test_bound_and_nearest(eps):
    # |x - q s| <= eps on every element, and no neighbouring code is closer.
    rng = np.random.default_rng(5)
    x = np.concatenate([rng.uniform(-1, 1, 50000), _adversarial(rng, eps)]).astype(np.float32)
    q = qeps.codes(x, eps)
    assert qeps.bound_violations(x, q, eps) == 0
    s = Fraction(2 * eps)
    for i in rng.integers(0, x.size, 300).tolist():
        xv = Fraction(float(x[i]))
        d0 = abs(xv - q[i] * s)
        assert d0 <= s / 2
        assert d0 <= abs(xv - (q[i] + 1) * s) and d0 <= abs(xv - (q[i] - 1) * s)
    # a planted violation is detected
    q2 = q.copy()
    q2[7] += 1
    assert qeps.bound_violations(x, q2, eps) >= 1


def test_width_closed_form():
    # b = ceil(log2(2M + 1)), at least 1 bit
    for m in list(range(0, 300)) + [2 ** 20 - 1, 2 ** 20, 2 ** 31 - 1]:
        b = qeps.width(m)
        assert b == max(1, math.ceil(math.log2(2 * m + 1) - 1e-12))
        assert -(2 ** (b - 1)) <= -m and m <= 2 ** (b - 1) - 1
    with pytest.raises(ValueError):
        qeps.width(2 ** 31)
    assert [qeps.width(m, "bytes") for m in (0, 127, 128, 32767, 32768)] == [8, 8, 16, 16, 32]


@pytest.mark.parametrize("eps,bits", [(1e-2, 7), (1e-3, 10), (1e-4, 14)])
def test_raw_workload_widths(eps, bits):
    # Inputs in (-1, 1): M = round((1 - tiny) / 2 eps) = 50 / 500 / 5000.
    a = np.float32(np.nextafter(np.float32(1.0), np.float32(0.0)))
    p = qeps.plan(eps, float(a))
    assert p["max_code"] == round(0.5 / eps) and p["bits"] == bits


def test_pack_hand_worked():
    # b=4, codes 1,-1,7,-8,0,3,-2,5 -> nibbles (LSB first) 1,F,7,8,0,3,E,5
    assert qeps.pack([1, -1, 7, -8, 0, 3, -2, 5], 4).tolist() == [0x5E3087F1]
    # b=7, codes 63,-64,1 -> 0x3F | 0x40<<7 | 1<<14
    assert qeps.pack([63, -64, 1], 7).tolist() == [0x603F]
    # b=12 crosses a word: FFF,000,7FF,800 -> FF000FFF, 00008007
    assert qeps.pack([-1, 0, 2047, -2048], 12).tolist() == [0xFF000FFF, 0x00008007]
    assert qeps.pack_exact([-1, 0, 2047, -2048], 12).tolist() == [0xFF000FFF, 0x00008007]


@pytest.mark.parametrize("b", [1, 2, 3, 5, 7, 8, 10, 13, 14, 16, 17, 24, 31, 32])
def test_pack_matches_definition_and_roundtrips(b):
    rng = np.random.default_rng(b)
    for n in (0, 1, 31, 32, 33, 257, 1000):
        q = rng.integers(-(2 ** (b - 1)), 2 ** (b - 1), n)
        w = qeps.pack(q, b)
        assert w.size == (n * b + 31) // 32
        assert np.array_equal(w, qeps.pack_exact(q, b))
        assert np.array_equal(qeps.unpack(w, b, n), q)


@pytest.mark.parametrize("eps", [1e-4, 1e-3, 1e-2])
def test_encode_decode_idempotent_over_full_range(eps):
    # encode(decode(c)) == c for every c of the width the (-1, 1) range needs.
    b = qeps.plan(eps, 0.999)["bits"]
    c = np.arange(-(2 ** (b - 1)) + 1, 2 ** (b - 1), dtype=np.int64)
    assert np.array_equal(qeps.codes(qeps.decode(c, eps), eps), c)


@pytest.mark.parametrize("eps", [1e-4, 1e-3])
def test_float32_materialisation_excess_is_half_ulp(eps):
    # The bound is on the exact q*s; the float32 x_hat may sit up to half a
    # float32 ulp beyond it (reading of the decode precision).
    rng = np.random.default_rng(3)
    x = rng.uniform(-1, 1, 100000).astype(np.float32)
    q = qeps.codes(x, eps)
    xh = qeps.decode(q, eps).astype(np.float64)
    err = np.abs(x.astype(np.float64) - xh)
    ulp = np.spacing(np.abs(xh).astype(np.float32)).astype(np.float64)
    assert np.all(err <= eps + 0.5 * ulp + 1e-18)


def test_linf_cell_bound_matches_paper():
    # Table "margin_cert": 2 eps sqrt(768), and cell-mates are within 2 eps.
    rows = [l.split() for l in open(os.path.join(GOLD, "linf_bound.txt")) if l[0] != "#"]
    for eps, val in rows:
        assert round(2 * float(eps) * math.sqrt(768), 4) == pytest.approx(float(val), abs=1e-4)
    rng = np.random.default_rng(9)
    eps = 1e-2
    x = rng.uniform(-1, 1, 200000).astype(np.float32)
    q = qeps.codes(x, eps)
    order = np.argsort(q, kind="stable")
    qs, xs = q[order], x[order].astype(np.float64)
    same = qs[1:] == qs[:-1]
    assert np.all(np.abs(xs[1:] - xs[:-1])[same] <= 2 * eps)


def test_encode_rejects_bad_input():
    with pytest.raises(ValueError):
        qeps.encode(np.array([np.nan], np.float32), 1e-3)
    with pytest.raises(ValueError):
        qeps.encode(np.array([0.5, 0.7], np.float32), 1e-3, absmax=0.6)
