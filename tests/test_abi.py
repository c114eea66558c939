"""Host-side checks of the C ABI: the library loads, exports every symbol the
header declares, and rejects bad arguments before touching the GPU."""
import ctypes
import os
import re

import pytest

from paper_2603_14806_amd import trimul as T

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "tri_mul.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(tri_mul_[a-z_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(T.LIB_PATH):
        from paper_2603_14806_amd import build
        build.build()
    return T.lib()


def test_header_declares_the_calls():
    names = declared_functions()
    for n in ("tri_mul_init", "tri_mul_outgoing", "tri_mul_incoming", "tri_mul_block_accumulate",
              "tri_mul_destroy", "tri_mul_last_error", "tri_mul_workspace_size"):
        assert n in names


def test_library_exports_every_declared_symbol(lib):
    for n in declared_functions():
        assert hasattr(lib, n), n
    assert set(declared_functions()) == set(T.SIGNATURES)


def test_struct_layouts():
    assert ctypes.sizeof(T.Params) == 4 * 4 + 4 + 4 + 10 * 8   # 5 scalars, padding, 10 pointers
    assert ctypes.sizeof(T.BlockView) == 9 * 8 + 2 * 4


def test_null_arguments_rejected_without_gpu(lib):
    h = ctypes.c_void_p()
    assert lib.tri_mul_init(ctypes.byref(h), None, None) == T.TRI_MUL_EINVAL
    assert "null" in T.last_error()
    assert lib.tri_mul_init(None, None, None) == T.TRI_MUL_EINVAL
    n = ctypes.c_size_t()
    assert lib.tri_mul_workspace_size(None, 16, ctypes.byref(n)) == T.TRI_MUL_EINVAL
    assert lib.tri_mul_outgoing(None, 16, 0, 16, 16, 16, 1 << 20, None) == T.TRI_MUL_EINVAL
    assert lib.tri_mul_incoming(None, 16, 0, 16, 16, 16, 1 << 20, None) == T.TRI_MUL_EINVAL
    assert lib.tri_mul_block_accumulate(None, None, 16, 16, 16, 0, 0, 0, None) == T.TRI_MUL_EINVAL
    assert lib.tri_mul_destroy(None) == T.TRI_MUL_OK
    assert T.last_error() == ""


def test_bad_params_rejected_without_gpu(lib):
    h = ctypes.c_void_p()
    fake = [16 * (i + 1) for i in range(10)]           # never dereferenced
    p = T.Params(128, 128, 7, 0, 1e-5, *fake)
    assert lib.tri_mul_init(ctypes.byref(h), ctypes.byref(p), None) == T.TRI_MUL_EINVAL
    p = T.Params(64, 128, T.TRI_MUL_BF16, 0, 1e-5, *fake)
    assert lib.tri_mul_init(ctypes.byref(h), ctypes.byref(p), None) == T.TRI_MUL_EUNSUPPORTED
    assert "128" in T.last_error()
    p = T.Params(128, 128, T.TRI_MUL_BF16, 0, 0.0, *fake)
    assert lib.tri_mul_init(ctypes.byref(h), ctypes.byref(p), None) == T.TRI_MUL_EINVAL
    p = T.Params(128, 128, T.TRI_MUL_BF16, 0, 1e-5, *(fake[:3] + [None] + fake[4:]))
    assert lib.tri_mul_init(ctypes.byref(h), ctypes.byref(p), None) == T.TRI_MUL_EINVAL
    assert not h.value


def test_last_error_is_thread_local(lib):
    import threading
    assert lib.tri_mul_init(None, None, None) == T.TRI_MUL_EINVAL
    seen = []
    th = threading.Thread(target=lambda: seen.append(T.last_error()))
    th.start()
    th.join()
    assert seen == [""]
    assert T.last_error() != ""
