"""GPU parity of Q_eps encode/decode against the oracle (bit-exact codes and
decoded float32), through the C ABI."""
import numpy as np
import pytest

import synth
from oracle import qeps

pytestmark = pytest.mark.gpu


def _dev(a):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def _words(t):
    return t.cpu().numpy().view(np.uint32)


def _check(lam, x, eps, absmax=None, mode="bits"):
    codes, p = lam.quantize(_dev(x), eps, absmax=absmax, mode=mode)
    words_ref, q_ref, plan = qeps.encode(x, eps, absmax=absmax, mode=mode)
    assert (p.bits, p.max_code) == (plan["bits"], plan["max_code"])
    assert p.code_bytes == 4 * words_ref.size
    assert np.array_equal(_words(codes), words_ref), "packed codes differ"
    xh = lam.dequantize(codes, p).cpu().numpy()
    assert np.array_equal(xh.view(np.uint32), qeps.decode(q_ref, eps).view(np.uint32)), "decode differs"
    return q_ref, xh


@pytest.mark.parametrize("eps", [1e-4, 1e-3, 1e-2, 0.25, 2.0 ** -10, 3e-3])
@pytest.mark.parametrize("n", [1, 31, 33, 4095, 4096, 4097, 50001])
def test_codes_bit_exact_ragged(lam, eps, n):
    rng = np.random.default_rng(n)
    x = rng.uniform(-1, 1, n).astype(np.float32)
    _check(lam, x, eps)


@pytest.mark.parametrize("eps", [2.0 ** -10, 0.25, 1e-3, 1e-4])
def test_near_ties(lam, eps):
    rng = np.random.default_rng(7)
    s = 2 * eps
    k = rng.integers(-400, 400, 20000)
    base = ((k + 0.5) * s).astype(np.float32)
    x = np.concatenate([base, np.nextafter(base, np.float32(1)), np.nextafter(base, np.float32(-1)),
                        np.array([0.0, -0.0, eps, -eps], np.float32)])
    _check(lam, x, eps, absmax=float(np.abs(x).max()))
    assert np.array_equal(qeps.codes(x, eps), qeps.codes_exact(x, eps))


@pytest.mark.parametrize("mode", ["bits", "bytes"])
def test_declared_and_measured_absmax(lam, mode):
    rng = np.random.default_rng(3)
    x = (0.04 * rng.standard_normal(100003)).astype(np.float32)
    _check(lam, x, 1e-3, absmax=None, mode=mode)
    _check(lam, x, 1e-3, absmax=1.0, mode=mode)


def test_errors_do_not_saturate(lam):
    x = np.linspace(-1, 1, 10000).astype(np.float32)
    with pytest.raises(lam.LamError) as e:
        lam.quantize(_dev(x), 1e-3, absmax=0.5)
    assert e.value.name == "LAM_ERANGE"
    x[123] = np.nan
    with pytest.raises(lam.LamError) as e:
        lam.quantize(_dev(x), 1e-3, absmax=1.0)
    assert e.value.name == "LAM_EINVAL"
    with pytest.raises(lam.LamError) as e:
        lam.quantize(_dev(x), 1e-3)
    assert e.value.name == "LAM_EINVAL"


def test_empty_input(lam):
    import torch
    codes, p = lam.quantize(torch.empty(0, dtype=torch.float32, device="cuda"), 1e-3, absmax=1.0)
    assert p.n == 0 and p.code_bytes == 0
    assert lam.dequantize(codes, p).numel() == 0


@pytest.mark.parametrize("eps,bits", [(1e-4, 14), (1e-3, 10), (1e-2, 7)])
def test_raw_workload_full_size(lam, eps, bits):
    """2^26 values, half N(0, 0.04^2) and half U(-1, 1): codes bit-exact, the
    bound on every element, the launch configuration the benchmark times."""
    cfg = synth.raw_qeps()
    x = cfg["x"]
    q_ref, xh = _check(lam, x, eps, absmax=1.0)
    assert qeps.plan(eps, 1.0)["bits"] >= bits
    assert qeps.bound_violations(x, q_ref, eps) == 0


def test_quantize_async_codes_and_status(lam):
    """The asynchronous encode writes the codes of the waiting one and reports
    invalid elements through the caller's counters instead of a status."""
    import torch
    x = np.linspace(-1, 1, 100003).astype(np.float32)
    status = torch.zeros(2, dtype=torch.int32, device="cuda")
    c1, p1 = lam.quantize(_dev(x), 1e-3, absmax=1.0)
    c2, p2 = lam.quantize_async(_dev(x), 1e-3, 1.0, status)
    assert (p1.bits, p1.max_code, p1.code_bytes) == (p2.bits, p2.max_code, p2.code_bytes)
    assert torch.equal(c1, c2)
    assert status.tolist() == [0, 0]
    y = x.copy()
    y[5] = np.nan
    y[70001] = 1.5
    lam.quantize_async(_dev(y), 1e-3, 1.0, status)
    s = status.tolist()
    assert s[0] > 0 and s[1] > 0
    status.zero_()
    y = x.copy()
    y[123] = -1.25
    lam.quantize_async(_dev(y), 1e-3, 1.0, status)
    s = status.tolist()
    assert s[0] == 0 and s[1] > 0
    with pytest.raises(lam.LamError) as e:
        lam.quantize_async(_dev(x), 1e-3, 0.0, status)
    assert e.value.name == "LAM_EINVAL"


def test_quantize_async_empty_and_counts_accumulate(lam):
    """An empty input queues nothing and leaves the counters as they were;
    counts from several calls add up until the caller clears them."""
    import torch
    status = torch.zeros(2, dtype=torch.int32, device="cuda")
    codes, p = lam.quantize_async(torch.empty(0, dtype=torch.float32, device="cuda"), 1e-3, 1.0, status)
    assert p.n == 0 and p.code_bytes == 0 and status.tolist() == [0, 0]
    y = np.linspace(-1, 1, 5000).astype(np.float32)
    y[10] = 3.0
    lam.quantize_async(_dev(y), 1e-3, 1.0, status)
    one = status.tolist()
    lam.quantize_async(_dev(y), 1e-3, 1.0, status)
    two = status.tolist()
    assert one[0] == 0 and one[1] > 0 and two == [0, 2 * one[1]]
