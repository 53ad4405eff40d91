"""The C ABI library loads and exports what include/lam.h declares; the
host-only width plan agrees with the oracle (CPU, no GPU calls)."""
import os
import re
import subprocess

import numpy as np
import pytest

from oracle import qeps

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "lam.h")
LIB = os.path.join(ROOT, "paper_2609_32256_amd", "liblam.so")


def _declared():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(lam_[a-z0-9_]+)\s*\(", text)))


def test_header_declares_the_boundary():
    names = _declared()
    for n in ("lam_quantize", "lam_dequantize", "lam_dedup_ingest", "lam_score_topk", "lam_store_quantize",
              "lam_qeps_plan", "lam_ctx_create", "lam_store_create"):
        assert n in names


@pytest.mark.skipif(not os.path.exists(LIB), reason="liblam.so not built")
def test_library_exports_every_declared_symbol():
    out = subprocess.run(["nm", "-D", "--defined-only", LIB], capture_output=True, text=True, check=True).stdout
    exported = set(re.findall(r"\sT\s(lam_[a-z0-9_]+)$", out, flags=re.M))
    missing = [n for n in _declared() if n not in exported]
    assert not missing, missing


@pytest.mark.skipif(not os.path.exists(LIB), reason="liblam.so not built")
def test_binding_loads_and_plan_matches_oracle():
    import paper_2609_32256_amd as lam
    assert lam.abi_version() == 1
    assert set(lam.EXPORTED) <= set(_declared())
    rng = np.random.default_rng(0)
    for eps in (1e-4, 1e-3, 1e-2, 0.25, 3e-3, 2.0 ** -20):
        for a in list(rng.uniform(0, 2, 20).astype(np.float32)) + [np.float32(0.0), np.float32(0.999)]:
            for mode in ("bits", "bytes"):
                ref = qeps.plan(eps, float(a), mode)
                got = lam.qeps_plan(eps, float(a), mode, 1000)
                assert (got.bits, got.max_code) == (ref["bits"], ref["max_code"]), (eps, a, mode)
                assert got.code_bytes == 4 * ((1000 * ref["bits"] + 31) // 32)
    # ties of the plan's rounding: A = (k + 1/2) s with a dyadic step
    for k in range(0, 40):
        a = (k + 0.5) * 0.5
        assert lam.qeps_plan(0.25, a).max_code == qeps.max_code(a, 0.25)


@pytest.mark.skipif(not os.path.exists(LIB), reason="liblam.so not built")
def test_plan_rejects_bad_arguments():
    import paper_2609_32256_amd as lam
    for args in ((float("nan"), 1.0), (0.0, 1.0), (1e-3, -1.0), (1e-3, float("inf"))):
        with pytest.raises(lam.LamError) as e:
            lam.qeps_plan(*args)
        assert e.value.name == "LAM_EINVAL"
    with pytest.raises(lam.LamError) as e:
        lam.qeps_plan(1e-9, 100.0)
    assert e.value.name == "LAM_ERANGE"
