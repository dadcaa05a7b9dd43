"""The compiler's resource report of every kernel (written by the build next to the
objects): no kernel keeps anything in scratch memory (a spill, or a kernel-argument
struct copied to the stack because a pointer into it outlives its use, made the merge
kernel 15x slower once) apart from one bounded exception below, every kernel's LDS fits
a CU (160 KB on gfx950), and the
attention kernel's registers fit two waves per SIMD (its design point: 256 per wave,
so the other wave of the SIMD keeps the matrix core busy through each one's softmax)."""
import json
import os

import pytest

RES = os.path.join(os.path.dirname(__file__), "..", "_build", "kernel_resources.json")


def _report():
    if not os.path.exists(RES):
        pytest.skip("the library has not been built here")
    with open(RES) as f:
        d = json.load(f)
    assert d, "empty resource report"
    return d


# The head_dim-256 attention kernel stores a few loop-invariant values (at most 64 bytes
# per lane) once before its key loop and reloads them only in the branch that masks a
# 32-key unit crossing the tail diagonal (a handful of units per workgroup). The
# spill-free forms of that mask (masking inside the row max and the exponentials of
# every unit) measured 6-7% slower over the whole update.
ALLOWED_SCRATCH = {"_ZN2tu12_GLOBAL__N_16k_attnILi256E": 64}


def test_no_kernel_uses_scratch():
    for name, r in _report().items():
        limit = max([v for k, v in ALLOWED_SCRATCH.items() if name.startswith(k)], default=0)
        assert r.get("scratch_bytes", 0) <= limit, f"{name}: {r['scratch_bytes']} bytes of scratch per lane"


def test_lds_fits_a_cu():
    for name, r in _report().items():
        assert r.get("lds_bytes", 0) <= 160 * 1024, f"{name}: {r['lds_bytes']} bytes of LDS"


def test_attention_registers_fit_two_waves_per_simd():
    att = {n: r for n, r in _report().items() if "k_attnILi" in n}
    assert len(att) == 3, sorted(att)      # head_dim 64, 128, 256
    for name, r in att.items():
        assert r["vgprs"] + r["agprs"] <= 256 and r["waves_per_simd"] >= 2, f"{name}: {r}"
