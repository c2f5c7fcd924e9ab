"""Register and scratch use of the built kernels, as the compiler reported it
when the library was last built: no kernel may spill to scratch memory (a
spill turns every register access of the epilogue or inner loop into a
memory round trip, which is how a small code change can double a kernel's
time without changing its results)."""
import os

import pytest

from paper_2609_35139_amd import build as _b


def _rows():
    if not os.path.exists(_b.RESOURCES):
        pytest.skip("library not built here (run __graft_entry__.build())")
    rows = []
    for line in open(_b.RESOURCES):
        name, *kv = line.split()
        rows.append((name, dict(x.split("=") for x in kv)))
    return rows


def test_every_source_reported():
    rows = _rows()
    assert any("gemm_nt_kernel" in n for n, _ in rows)
    assert any("attention_kernel" in n for n, _ in rows)
    assert any("layernorm_kernel" in n for n, _ in rows)


def test_no_kernel_spills_to_scratch():
    bad = [(n, r) for n, r in _rows() if r.get("scratch") not in ("0",)]
    assert not bad, bad


def test_resource_remarks_parse():
    text = ("x.hip:1:1: remark: Function Name: _Z3fooPf [-Rpass-analysis=kernel-resource-usage]\n"
            "x.hip:1:1: remark:     VGPRs: 12 [-Rpass-analysis=kernel-resource-usage]\n"
            "x.hip:1:1: remark:     ScratchSize [bytes/lane]: 16 [-Rpass-analysis=kernel-resource-usage]\n"
            "x.hip:1:1: remark:     Occupancy [waves/SIMD]: 8 [-Rpass-analysis=kernel-resource-usage]\n")
    assert _b._resources(text) == [{"kernel": "_Z3fooPf", "VGPRs": 12, "ScratchSize": 16,
                                     "Occupancy": 8}]
