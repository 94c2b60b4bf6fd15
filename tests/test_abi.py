"""The C ABI: libtc.so loads on a machine without a GPU, exports exactly the
functions include/tc.h declares, and its pure host helpers and argument
checks behave as documented (no device work is started by these calls)."""
import ctypes as C
import os
import re
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "tc.h")


def _declared():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(tc_[a-z0-9_]+)\s*\(", src)))


@pytest.fixture(scope="module")
def tcmod():
    from paper_2401_07788_amd import tc
    if not os.path.exists(tc.LIB_PATH):
        pytest.fail("libtc.so is not built (run __graft_entry__.build())")
    tc.lib()
    return tc


@pytest.mark.parametrize("which", ["LIB_PATH", "DEBUG_LIB_PATH"])
def test_exports_match_header(tcmod, which):
    declared = _declared()
    assert "tc_aqsgd_step" in declared and "tc_topk_compress" in declared
    path = getattr(tcmod, which)
    out = subprocess.run(["nm", "-D", "--defined-only", path], capture_output=True, text=True,
                         check=True).stdout
    exported = sorted({ln.split()[-1] for ln in out.splitlines() if " T " in ln})
    assert exported == declared
    assert sorted(tcmod.EXPORTS) == declared
    tcmod.load(path)


def test_efmix_counts_from_the_library(tcmod, orc):
    for k in (0, 1, 2, 3277, 3278, 2 ** 40 + 1):
        assert tcmod.efmix_counts(k) == orc.efmix_counts(k)
        assert sum(tcmod.efmix_counts(k)) == k


def test_debug_library_refuses_overlapping_buffers(tcmod):
    """the aliasing precondition is checked on the host before any device
    call, so it runs here; the release library does not check it"""
    D = tcmod.load(tcmod.DEBUG_LIB_PATH)
    R = tcmod.load(tcmod.LIB_PATH)
    n_seg, L, k = 2, 1000, 10
    c = tcmod.Codec(1, 0, 0, 0, n_seg, L, k)
    base = 1 << 40                      # never dereferenced: the checks fail first
    x = C.c_void_p(base)
    e_overlap = C.cast(C.c_void_p(base + 4 * L), C.POINTER(C.c_float))
    p = tcmod.Payload(base + (1 << 30), base + (2 << 30), None, None, None)
    assert D.tc_ef_step(C.byref(c), x, 0, e_overlap, C.byref(p), None, 0, None) == tcmod.TC_ERR_PRECONDITION
    assert b"overlap" in D.tc_last_error()
    # a payload whose values run into its indices
    p2 = tcmod.Payload(base + (1 << 30), base + (1 << 30) + 4, None, None, None)
    c2 = tcmod.Codec(1, 0, 0, 0, n_seg, L, k)
    assert D.tc_topk_compress(C.byref(c2), x, 0, C.byref(p2), None, 0, None) == tcmod.TC_ERR_PRECONDITION
    # the receiver side: AQ-SGD output over the buffer
    c3 = tcmod.Codec(1, 2, 0, 0, n_seg, L, k)
    p3 = tcmod.Payload(base + (1 << 30), base + (2 << 30), None, None, None)
    m_r = C.c_void_p(base)
    assert D.tc_aqsgd_reconstruct(C.byref(c3), C.byref(p3), m_r, 2, 4, C.c_void_p(base + (3 << 30)), n_seg,
                                  C.c_void_p(base + 2 * L), None) == tcmod.TC_ERR_PRECONDITION
    assert R.tc_status_str(tcmod.TC_ERR_PRECONDITION)


def test_host_helpers(tcmod, orc):
    for L, num, den in [(16384, 1, 10), (393216, 3, 10), (2 ** 27, 1, 10), (100, 7, 100), (5, 0, 3), (7, 1, 0)]:
        assert tcmod.topk_count(L, num, den) == orc.topk_count(L, num, den)
    for G, b in [(768, 4), (32768, 2), (5, 6), (33, 3), (1, 1), (100, 8)]:
        assert tcmod.quant_group_bytes(G, b) == orc.quant_group_bytes(G, b)
    assert tcmod.quant_group_bytes(10, 32) == 40
    assert tcmod.quant_group_bytes(10, 9) == 0
    for s in range(8):
        assert tcmod.status_str(s) != "unknown status"


def test_validation_before_any_device_call(tcmod):
    L = tcmod.lib()
    p = tcmod.Payload(None, None, None, None)
    # NULL codec
    assert L.tc_topk_compress(None, None, 0, C.byref(p), None, 0, None) == 1
    # bad kind, reserved field, k > seg_len, bad bit width
    for c, fn in [
        (tcmod.Codec(7, 0, 0, 0, 1, 10, 1), L.tc_topk_compress),
        (tcmod.Codec(1, 0, 0, 5, 1, 10, 1), L.tc_topk_compress),
        (tcmod.Codec(1, 0, 0, 0, 1, 10, 11), L.tc_topk_compress),
        (tcmod.Codec(2, 0, 9, 0, 1, 10, 0), L.tc_quant_pack),
        (tcmod.Codec(1, 0, 0, 0, 1, 1 << 32, 1), L.tc_topk_compress),
    ]:
        assert fn(C.byref(c), None, 0, C.byref(p), None, 0, None) == 2
        assert L.tc_last_error()
    # quantization codec to the TopK entry point
    c = tcmod.Codec(2, 0, 4, 0, 1, 10, 0)
    assert L.tc_topk_compress(C.byref(c), None, 0, C.byref(p), None, 0, None) == 2
    # AQ-SGD: n_seg must equal n_ids
    c = tcmod.Codec(1, 2, 0, 0, 4, 10, 3)
    assert L.tc_aqsgd_step(C.byref(c), None, 2, None, 10, None, 3, C.byref(p), None, 0, None) == 2
    # empty tensors are a no-op that succeeds
    c = tcmod.Codec(1, 0, 0, 0, 0, 10, 0)
    assert L.tc_topk_compress(C.byref(c), None, 0, C.byref(p), None, 0, None) == 0


def test_noalloc_refuses_shapes_beyond_its_scratch(tcmod):
    """the allocation-free AQ-SGD sender checks the scratch a shape needs
    against its fixed maximum on the host, before any device call (pointers
    below are never dereferenced)"""
    R = tcmod.load(tcmod.LIB_PATH)
    base = 1 << 40
    n_ids, L, k = 600, 40000, 12000     # many two-workgroup segments at once
    c = tcmod.Codec(1, 2, 0, 0, n_ids, L, k)
    p = tcmod.Payload(base + (1 << 34), base + (2 << 34), None, None, None)
    a, m, ids = C.c_void_p(base), C.c_void_p(base + (1 << 32)), C.c_void_p(base + (3 << 34))
    st = R.tc_aqsgd_step_noalloc(C.byref(c), a, 2, m, 1000, ids, n_ids, C.byref(p), None)
    assert st == tcmod.TC_ERR_WORKSPACE
    assert b"scratch" in R.tc_last_error()
    # the argument checks of tc_aqsgd_step come first
    assert R.tc_aqsgd_step_noalloc(C.byref(c), a, 2, m, 1000, ids, n_ids - 1, C.byref(p), None) == 2
    assert R.tc_aqsgd_step_noalloc(C.byref(c), a, 2, m, 0, ids, n_ids, C.byref(p), None) == 2
    assert R.tc_aqsgd_step_noalloc(None, a, 2, m, 1000, ids, n_ids, C.byref(p), None) == 1
    assert tcmod.NOALLOC_SCRATCH_BYTES == 4 << 20


def test_raise_device_errors_checks_bits_first(tcmod):
    R = tcmod.load(tcmod.LIB_PATH)
    assert R.tc_raise_device_errors(0x10) == tcmod.TC_ERR_ARG
    assert b"unknown" in R.tc_last_error()
