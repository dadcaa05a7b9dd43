"""The compiler's resource report of every kernel (written by the build next to the
objects): no kernel keeps anything in scratch memory (a spill, or a kernel-argument
struct copied to the stack because a pointer into it outlives its use, made the merge
kernel 15x slower once), every kernel's LDS fits a CU (160 KB on gfx950), and the
attention kernel's registers fit one wave per SIMD (its design point)."""
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


def test_no_kernel_uses_scratch():
    for name, r in _report().items():
        assert r.get("scratch_bytes", 0) == 0, f"{name}: {r['scratch_bytes']} bytes of scratch per lane"


def test_lds_fits_a_cu():
    for name, r in _report().items():
        assert r.get("lds_bytes", 0) <= 160 * 1024, f"{name}: {r['lds_bytes']} bytes of LDS"


def test_attention_registers_fit_one_wave_per_simd():
    att = {n: r for n, r in _report().items() if "k_attnILi" in n}
    assert len(att) == 3, sorted(att)      # head_dim 64, 128, 256
    for name, r in att.items():
        assert r["vgprs"] + r["agprs"] <= 512, f"{name}: {r}"
