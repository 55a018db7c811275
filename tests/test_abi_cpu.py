"""libep.so on the CPU: it loads, exports every function include/*.h declares, and
rejects bad arguments before touching a device.  No compute call is made here."""
import ctypes
import glob
import os
import re

import pytest

from paper_2609_40093_amd import _lib

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(_lib.LIB_PATH):
        from paper_2609_40093_amd import build
        build.build()
    return _lib.load()


def declared_functions():
    names = set()
    for path in glob.glob(os.path.join(ROOT, "include", "*.h")):
        text = open(path).read()
        text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)
        text = re.sub(r"//[^\n]*", " ", text)
        for m in re.finditer(r"\b(ep_[a-z0-9_]+)\s*\([^;{}]*\)\s*;", text):
            names.add(m.group(1))
    return sorted(names)


# the C ABI the hot path's scope table names, in its own words
BOUNDARY = ("ep_last_error", "ep_staging_alloc", "ep_staging_free", "ep_staging_ptrs", "ep_layout_workspace_bytes",
            "ep_dispatch_layout", "ep_layout_validate", "ep_dispatch", "ep_combine")


def declaration_comments():
    """The comment block right before each ep_* declaration of include/ep.h."""
    text = open(os.path.join(ROOT, "include", "ep.h")).read()
    out = {}
    for m in re.finditer(r"/\*((?:(?!\*/).)*)\*/\s*((?:[a-z_]+\s+\**)+)(ep_[a-z0-9_]+)\s*\(", text, flags=re.S):
        out[m.group(3)] = m.group(1)
    return out


def test_headers_declare_the_boundary():
    names = declared_functions()
    for required in BOUNDARY:
        assert required in names, required


@pytest.mark.parametrize("name", [n for n in BOUNDARY if n != "ep_last_error"])
def test_boundary_calls_cite_the_paper(name):
    comment = declaration_comments().get(name, "")
    assert re.search(r"Sec\. \d", comment), f"{name}: no section of the paper cited in its declaration"


@pytest.mark.parametrize("name", declared_functions())
def test_symbol_exported(lib, name):
    assert hasattr(lib, name), f"{name} declared in include/ but not exported"


def test_binding_covers_every_symbol():
    assert set(declared_functions()) <= set(_lib.SIGNATURES)


def test_status_names(lib):
    assert lib.ep_abi_version() == _lib.ABI_VERSION == 6
    assert lib.ep_status_name(0) == b"EP_OK"
    assert lib.ep_status_name(5) == b"EP_ERR_TIMEOUT"
    assert lib.ep_status_name(99) == b"EP_ERR_UNKNOWN"


def test_workspace_bytes(lib):
    n = ctypes.c_size_t()
    assert lib.ep_layout_workspace_bytes(128, 2, 16, ctypes.byref(n)) == 0
    assert n.value == 256                           # one tile: header only
    assert lib.ep_layout_workspace_bytes(4096, 2, 8, ctypes.byref(n)) == 0
    assert n.value == 256 + 8 * 9 * 4               # 8 tiles of 16 x 64 entries: 8 counts + error word
    assert lib.ep_layout_workspace_bytes(32768, 8, 256, ctypes.byref(n)) == 0
    assert n.value == 256 + 64 * 257 * 4            # 64 tiles of 16 x 4 x 64 entries (16K counts)
    assert lib.ep_layout_workspace_bytes(20000, 4, 2048, ctypes.byref(n)) == 0
    assert n.value == 256 + 8 * 2049 * 4            # 8 tiles of 4 x 40 x 64 entries
    assert lib.ep_layout_workspace_bytes(-1, 2, 16, ctypes.byref(n)) == _lib.EP_ERR_INVALID_ARG
    assert lib.ep_layout_workspace_bytes(4, 2, 4096, ctypes.byref(n)) == _lib.EP_ERR_INVALID_ARG
    assert b"bad sizes" in lib.ep_last_error()


@pytest.mark.parametrize("T,k,E,R", [(-1, 2, 8, 4), (4, 0, 8, 4), (4, 9, 8, 4), (4, 2, 8, 3),
                                     (4, 2, 0, 1), (4, 2, 4096, 8), (1 << 30, 8, 16, 4)])
def test_layout_rejects_bad_sizes(lib, T, k, E, R):
    dummy = ctypes.c_void_p(16)   # never dereferenced: the call must fail first
    st = lib.ep_dispatch_layout(dummy, T, k, E, R, dummy, dummy, dummy, dummy, dummy, None, dummy, 1 << 20, None)
    assert st == _lib.EP_ERR_INVALID_ARG
    assert lib.ep_last_error()


def test_layout_rejects_null_and_small_workspace(lib):
    d = ctypes.c_void_p(16)
    assert lib.ep_dispatch_layout(d, 4, 2, 8, 4, None, d, d, d, d, None, d, 1 << 20, None) == _lib.EP_ERR_INVALID_ARG
    assert lib.ep_dispatch_layout(None, 4, 2, 8, 4, d, d, d, d, d, None, d, 1 << 20, None) == _lib.EP_ERR_INVALID_ARG
    assert lib.ep_dispatch_layout(d, 40000, 2, 8, 4, d, d, d, d, d, None, d, 256, None) == _lib.EP_ERR_INVALID_ARG
    assert b"workspace" in lib.ep_last_error()


@pytest.mark.parametrize("T,k,E,R", [(-1, 2, 8, 4), (4, 0, 8, 4), (4, 9, 8, 4), (4, 2, 8, 3), (4, 2, 4096, 8)])
def test_fused_dispatch_rejects_bad_arguments(lib, T, k, E, R):
    """ep_dispatch_fused checks the layout's arguments, then the dispatch's (a NULL
    staging), before it touches a device."""
    d = ctypes.c_void_p(16)   # never dereferenced: the call must fail first
    st = lib.ep_dispatch_fused(d, T, k, E, R, d, d, d, d, d, None, d, 1 << 20, d, 512, None, 0, 1, None)
    assert st == _lib.EP_ERR_INVALID_ARG
    assert b"ep_dispatch_fused" in lib.ep_last_error()
    good = lib.ep_dispatch_fused(d, 4, 2, 8, 4, d, d, d, d, d, None, d, 1 << 20, d, 512, None, 0, 1, None)
    assert good == _lib.EP_ERR_INVALID_ARG and b"staging is NULL" in lib.ep_last_error()


@pytest.mark.parametrize("args", [(7, 10, 64, 4, 1, 0), (0, 0, 64, 4, 1, 0), (0, 10, 12, 4, 1, 0),
                                  (0, 10, 64, 0, 1, 0), (0, 10, 64, 4, 9, 0), (1, 10, 64, 4, 1, -1)])
def test_staging_alloc_rejects_bad_arguments(lib, args):
    out = ctypes.c_void_p()
    assert lib.ep_staging_alloc(*args, ctypes.byref(out)) == _lib.EP_ERR_INVALID_ARG
    assert not out.value


def test_null_staging_calls(lib):
    v = _lib.StagingView()
    assert lib.ep_staging_ptrs(None, 0, ctypes.byref(v)) == _lib.EP_ERR_INVALID_ARG
    assert lib.ep_staging_set_wait(None, 10, 1) == _lib.EP_ERR_INVALID_ARG
    assert lib.ep_staging_status(None, None) == _lib.EP_ERR_INVALID_ARG
    assert lib.ep_staging_free(None) == 0
    assert lib.ep_dispatch(None, 4, 64, 2, None, None, None, 0, 1, None) == _lib.EP_ERR_INVALID_ARG
    assert lib.ep_combine(None, 0, 1, None, None, None, 4, 64, 2, None, 0, None) == _lib.EP_ERR_INVALID_ARG
    assert lib.ep_staging_set_mode(None, 0, 0) == _lib.EP_ERR_INVALID_ARG
    assert lib.ep_staging_set_inbound(None, 0, None) == _lib.EP_ERR_INVALID_ARG
    assert lib.ep_graph_legs_sdma(None, 1) == _lib.EP_ERR_INVALID_ARG
    assert lib.ep_graph_legs_sdma(None, 0) == _lib.EP_ERR_INVALID_ARG
    g = ctypes.c_double()
    assert lib.ep_pcie_probe(None, None, 16, 1, ctypes.byref(g)) == _lib.EP_ERR_INVALID_ARG
    assert lib.ep_pcie_probe(ctypes.c_void_p(16), ctypes.c_void_p(16), 16, 4, ctypes.byref(g)) == \
        _lib.EP_ERR_INVALID_ARG
    assert lib.ep_sim_peers_set_delays(None, None, None) == _lib.EP_ERR_INVALID_ARG
    assert lib.ep_sim_peers_start(None, 0, ctypes.byref(ctypes.c_void_p())) == _lib.EP_ERR_INVALID_ARG
    assert lib.ep_sim_peers_stop(None) == 0
    assert lib.ep_copy_probe(ctypes.c_void_p(16), ctypes.c_void_p(16), 15, None) == _lib.EP_ERR_INVALID_ARG
    # store policy 0, 1 or 2 only; a row size with no probe instance
    for pol in (3, -1):
        assert lib.ep_stream_probe(ctypes.c_void_p(16), None, 4, 1024, 0, 1, pol, None) == _lib.EP_ERR_INVALID_ARG
        assert b"store_policy" in lib.ep_last_error()
    assert lib.ep_stream_probe(ctypes.c_void_p(16), None, 4, 3072, 0, 1, 0, None) == _lib.EP_ERR_INVALID_ARG


def test_trace_without_launches(lib):
    assert ctypes.sizeof(_lib.TraceStat) == 48 + 8 + 6 * 8    # ep_trace_stat in include/ep.h
    assert lib.ep_trace_reset() == 0
    arr = (_lib.TraceStat * 4)()
    n = ctypes.c_int32(-1)
    assert lib.ep_trace_read(arr, 4, ctypes.byref(n)) == 0 and n.value == 0
    assert lib.ep_trace_read(None, 4, ctypes.byref(n)) == _lib.EP_ERR_INVALID_ARG


def test_binding_fails_loudly_without_library(tmp_path):
    with pytest.raises(RuntimeError, match="not built"):
        _lib.load(str(tmp_path / "libep.so"))


def test_binding_rejects_host_tensors_before_the_library():
    """A host tensor where the library expects device memory is refused in Python."""
    torch = pytest.importorskip("torch")
    import paper_2609_40093_amd as ep
    with pytest.raises(ValueError, match="must be a device tensor"):
        ep.copy_probe(torch.empty(64, dtype=torch.uint8), torch.empty(64, dtype=torch.uint8))


@pytest.mark.parametrize("T,k,E,R", [(-1, 2, 8, 4), (4, 0, 8, 4), (4, 9, 8, 4), (4, 2, 8, 3), (4, 2, 4096, 8),
                                     (1 << 30, 8, 16, 4)])
def test_static_layout_rejects_bad_arguments_before_the_device(lib, T, k, E, R):
    """ep_dispatch_layout_static checks every argument before it touches a device."""
    dummy = ctypes.c_void_p(16)   # never dereferenced: the call must fail first
    st = lib.ep_dispatch_layout_static(dummy, T, k, E, R, dummy, dummy, dummy, dummy, dummy, None, dummy, None)
    assert st == _lib.EP_ERR_INVALID_ARG
    assert b"ep_dispatch_layout_static" in lib.ep_last_error()
    st = lib.ep_dispatch_layout_static(dummy, 4, 2, 8, 4, dummy, dummy, dummy, dummy, dummy, None, None, None)
    assert st == _lib.EP_ERR_INVALID_ARG and b"status_dev" in lib.ep_last_error()
