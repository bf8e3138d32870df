"""The C ABI library loads, exports every function include/unison.h declares
and rejects bad arguments on the host, without touching a GPU."""
import ctypes as C
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "unison.h")
LIB = os.path.join(ROOT, "paper_2609_09643_amd", "libunison.so")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(unison_[a-z0-9_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(LIB):
        pytest.fail("libunison.so not built; run __graft_entry__.build()")
    from paper_2609_09643_amd import unison
    return unison.lib()


def test_every_declared_symbol_is_exported(lib):
    names = declared_functions()
    assert len(names) >= 18
    for n in names:
        assert hasattr(lib, n), n


def test_host_side_validation(lib):
    from paper_2609_09643_amd import unison as U
    d = U.Dims(4, 1, 16, 1, 0)
    size = C.c_size_t()
    assert lib.unison_workspace_size(C.byref(d), C.byref(size)) == 0 and size.value > 0
    bad = U.Dims(0, 1, 16, 1, 0)
    assert lib.unison_workspace_size(C.byref(bad), C.byref(size)) == U.E_INVALID
    bad = U.Dims(1, 1, (1 << 20) + 1, 1, 0)
    assert lib.unison_workspace_size(C.byref(bad), C.byref(size)) == U.E_INVALID
    ctx = C.c_void_p()
    # misaligned or short workspace
    assert lib.unison_create(C.byref(ctx), C.byref(d), None, C.c_void_p(0x1001), size) == U.E_INVALID
    assert lib.unison_create(C.byref(ctx), C.byref(d), None, C.c_void_p(0x1000),
                             C.c_size_t(size.value - 1)) == U.E_INVALID
    # a context over a fake (never dereferenced) address: no HIP call happens
    assert lib.unison_create(C.byref(ctx), C.byref(d), None, C.c_void_p(0x100000), size) == 0
    assert lib.unison_run(ctx, 0xFF, 0, 1) == U.E_NOT_READY
    hd = (C.c_uint32 * 51)()
    hn = (C.c_uint32 * 51)()
    assert lib.unison_read_hazard(ctx, 0, hd, hn) == U.E_NOT_READY
    assert lib.unison_read_hazard(ctx, 4, hd, hn) == U.E_INVALID
    assert lib.unison_read_hazard(ctx, 0, None, hn) == U.E_INVALID
    p = (U.SimParams * 4)()
    assert lib.unison_set_params(ctx, p) == U.E_NOT_READY
    assert b"traces" in lib.unison_last_error(ctx)
    assert lib.unison_kendall(None, 1, 1, 1, C.c_void_p(8), C.c_void_p(8), None, C.c_void_p(8),
                              C.c_void_p(8)) == U.E_INVALID
    assert lib.unison_kendall(None, 1, 5000, 5000, C.c_void_p(8), C.c_void_p(8), None,
                              C.c_void_p(8), C.c_void_p(8)) == U.E_INVALID
    assert lib.unison_score_fixed(None, 1, C.c_void_p(8), C.c_void_p(8), C.c_void_p(8),
                                  C.c_void_p(8), C.c_void_p(8), 17, 0, 0, C.c_void_p(8)) == U.E_INVALID
    assert lib.unison_score_fixed(None, 1, C.c_void_p(8), C.c_void_p(8), C.c_void_p(8),
                                  C.c_void_p(8), C.c_void_p(8), 12, 0, 33, C.c_void_p(8)) == U.E_INVALID
    assert lib.unison_strerror(U.E_BAD_TRACE) == b"trace breaks the event format"
    assert lib.unison_debug_cache_slots(ctx, -2) == U.E_INVALID
    assert lib.unison_debug_cache_slots(ctx, 0) == 0 and lib.unison_debug_cache_slots(ctx, -1) == 0
    assert lib.unison_debug_cache_slots(None, 1) == U.E_INVALID
    lib.unison_destroy(ctx)


def test_struct_layouts_match_header():
    from paper_2609_09643_amd import unison as U
    assert C.sizeof(U.SimParams) == 128
    assert U.COUNTERS_DTYPE.itemsize == 25 * 8
    assert U.RECORD_DTYPE.itemsize == 16
    assert C.sizeof(U.TraceBatch) == 8 + 9 * 8
