"""The C-ABI library builds, loads without a GPU and exports every entry
point include/pc.h declares; argument errors are reported before any
device work (no compute call is made here)."""
import ctypes
import os
import re
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "pc.h")


def declared_functions():
    src = open(HEADER).read()
    return sorted(set(re.findall(r"^\s*(?:int|const char \*)\s*(pc_\w+)\s*\(", src, re.M)))


@pytest.fixture(scope="module")
def libpc():
    import paper_2602_16100_amd as pc
    if not os.path.exists(pc.LIB_PATH):
        from paper_2602_16100_amd import _build
        _build.build(force=False)
    return pc


def test_header_declares_the_four_checks():
    f = declared_functions()
    for name in ("pc_eval_selectors", "pc_trace_flows", "pc_masked_reach", "pc_report"):
        assert name in f


def test_library_exports_every_declared_symbol(libpc):
    out = subprocess.run(["nm", "-D", "--defined-only", libpc.LIB_PATH], capture_output=True, text=True,
                         check=True).stdout
    exported = set(re.findall(r"\sT\s+(pc_\w+)$", out, re.M))
    assert set(declared_functions()) <= exported
    assert set(libpc.EXPORTED) == set(declared_functions())
    L = libpc.lib()
    for name in declared_functions():
        assert getattr(L, name) is not None


def test_version_matches_header(libpc):
    v = int(re.search(r"#define PC_VERSION (\d+)", open(HEADER).read()).group(1))
    assert libpc.version() == v


def test_null_context_is_einval(libpc):
    L = libpc.lib()
    EINVAL = libpc.PC_EINVAL
    assert L.pc_eval_selectors(None, None, 0, 0, None, None, 0, 0, None, None, None) == EINVAL
    assert L.pc_eval_affinity(None, None, 0, 0, None, 0, None, 0, None, 0, None, None, None, None) == EINVAL
    assert L.pc_score_preferred(None, None, 0, 0, None, None, 0, None, 0, None, None, 0, None, None, None,
                                None) == EINVAL
    assert L.pc_update_nodes(None, None, 0, 0, None, None, 0, 0, None, 0, None, None, None) == EINVAL
    assert L.pc_eval_selectors_count(None, None, 0, 0, None, None, 0, 0, None, None) == EINVAL
    assert L.pc_probe_selectors(None, None, 0, 0, None, None, 0, 0, None, None, 0, None, None) == EINVAL
    assert L.pc_report_counts(None, 0, None, 0, None, 0, None, None, 0, None, None, 0, None, None, None,
                              None) == EINVAL
    assert L.pc_synthesize_paths(None, 0, None, None, 0, None, None, 0, None, None, None, None, 0, None, 0, None,
                                 None, 0, 0, None, None, None, None) == EINVAL
    assert L.pc_trace_flows(None, 0, None, None, 0, None, None, None, 0, None, None, 0, 0, None, None) == EINVAL
    assert L.pc_trace_flows_delta(None, 0, None, None, 0, None, None, None, 0, None, None, 0, 0, None, 0, None, None,
                                  None, None, None) == EINVAL
    assert L.pc_masked_reach(None, 0, None, None, 0, None, 0, None, None, None, None, None) == EINVAL
    assert L.pc_report(None, 0, None, 0, None, 0, None, 0, None, 0, None, None, 0, None, None, None, None) == EINVAL
    f = ctypes.c_uint32()
    assert L.pc_data_errors(None, None, ctypes.byref(f), 0) == EINVAL
    assert L.pc_trace_keep_tables(None, 1) == EINVAL
    assert L.pc_create(None, 0) == EINVAL
    assert L.pc_destroy(None) == libpc.PC_OK


def test_no_device_is_reported_not_faked(libpc):
    import torch
    if torch.cuda.is_available():
        pytest.skip("a GPU is present")
    h = ctypes.c_void_p()
    assert libpc.lib().pc_create(ctypes.byref(h), 0) == libpc.PC_EDEVICE
    with pytest.raises(libpc.PCError):
        libpc.Context(0)
