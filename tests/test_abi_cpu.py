"""The C-ABI library loads and exports every entry point its header declares
(no GPU calls here beyond a device count)."""
import ctypes
import os
import re

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "packserve.h")


def _declared():
    src = open(HEADER).read()
    return sorted(set(re.findall(r"^\s*(?:ps_status|const char\*)\s+(ps_\w+)\s*\(", src, re.M)))


def test_header_declares_the_entry_points():
    names = _declared()
    for n in ("ps_create", "ps_destroy", "ps_load_instances", "ps_score_window",
              "ps_score_window_dev", "ps_probe_hits_dev", "ps_commit", "ps_read_state",
              "ps_table_info", "ps_last_error", "ps_schedule_window_dev",
              "ps_replay_window_dev"):
        assert n in names


def test_library_exports_every_declared_symbol():
    import paper_2609_33224_amd as ps
    lib = ps.load_library()
    missing = [n for n in _declared() if not hasattr(lib, n)]
    assert not missing, missing


def test_library_is_built_from_these_sources():
    """ps_build_id() names the sources the library was compiled from: a
    stale libpackserve.so (sources changed, no rebuild) fails here."""
    import paper_2609_33224_amd as ps
    from paper_2609_33224_amd import build
    assert ps.ps_build_id() == build.source_hash()


def test_struct_layouts_match_header():
    import paper_2609_33224_amd as ps
    assert ps.PS_REQ_DTYPE.itemsize == 24
    assert ps.PS_RESULT_DTYPE.itemsize == 20
    # float alpha[6]; int n_seg; int seg_ub[32]; float beta[32][3]; float gamma[32];
    # 4 floats; 2 ints; int64 (8-aligned); uint32; uint64 -> 720 bytes
    assert ctypes.sizeof(ps.PsModel) == 720
    assert ctypes.sizeof(ps.binding.PsInstances) == 56


def test_errors_without_a_context():
    import paper_2609_33224_amd as ps
    lib = ps.load_library()
    assert lib.ps_create(0, None) == ps.binding.PS_E_INVAL
    assert lib.ps_destroy(None) == 0
    assert lib.ps_load_instances(None, None, None) == ps.binding.PS_E_INVAL
    assert lib.ps_score_window(None, None, 0, None, 0, None) == ps.binding.PS_E_INVAL
    assert lib.ps_commit(None, None, 0, None, None, 0, None) == ps.binding.PS_E_INVAL
    assert lib.ps_schedule_window_dev(None, None, 0, None, 0, None, None, None, None) == ps.binding.PS_E_INVAL
    assert lib.ps_replay_window_dev(None, None, 0, None, 0, None, None, None, None) == ps.binding.PS_E_INVAL
    assert b"ctx is NULL" in lib.ps_last_error(None)


def test_no_device_reports_an_error(monkeypatch):
    import torch
    if torch.cuda.is_available():
        pytest.skip("a GPU is present")
    import paper_2609_33224_amd as ps
    with pytest.raises(ps.PackServeError) as e:
        ps.ps_create(0)
    assert e.value.code in (ps.binding.PS_E_DEVICE, ps.binding.PS_E_INVAL)


def test_build_spill_report_parser():
    """The build refuses kernels that spill vector registers: the report
    parser picks each kernel's spill count out of the compiler's remarks."""
    from paper_2609_33224_amd import build
    txt = ("k.hip:1:1: remark: Function Name: kern_a [-Rpass-analysis=kernel-resource-usage]\n"
           "k.hip:1:1: remark:     VGPRs: 128 [-Rpass-analysis=kernel-resource-usage]\n"
           "k.hip:1:1: remark:     VGPRs Spill: 3 [-Rpass-analysis=kernel-resource-usage]\n"
           "    1 | __global__ void kern_a() {\n"
           "k.hip:9:1: remark: Function Name: kern_b [-Rpass-analysis=kernel-resource-usage]\n"
           "k.hip:9:1: remark:     VGPRs Spill: 0 [-Rpass-analysis=kernel-resource-usage]\n")
    assert build.vgpr_spills(txt) == {"kern_a": 3, "kern_b": 0}
