"""Host-side checks of the C ABI: the library loads, exports every symbol the
header declares, and rejects bad arguments before touching the GPU."""
import ctypes
import os
import re

import pytest

from paper_2603_14806_amd import trimul as T

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADERS = [os.path.join(ROOT, "include", h) for h in ("tri_mul.h", "opm.h", "triattn.h", "tri_mul_check.h")]


def declared_functions():
    names = set()
    for header in HEADERS:
        text = open(header).read()
        text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
        names |= set(re.findall(r"\b((?:tri_mul|opm|tri_attn)_[a-z_]+)\s*\(", text))
    return sorted(names)


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
    assert ctypes.sizeof(T.Grads) == 10 * 8
    assert ctypes.sizeof(T.OpmParams) == 3 * 4 + 4 + 2 * 8      # 3 ints, padding, 2 pointers
    assert ctypes.sizeof(T.OpmBlockView) == 8 * 8 + 2 * 4
    assert ctypes.sizeof(T.TriAttnView) == 2 * 8 + 2 * 4 + 3 * 8 + 2 * 4


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
    assert lib.opm_init(ctypes.byref(h), None, None) == T.TRI_MUL_EINVAL
    bad = T.OpmParams(16, 128, T.TRI_MUL_F32, 16, None)
    assert lib.opm_init(ctypes.byref(h), ctypes.byref(bad), None) == T.TRI_MUL_EUNSUPPORTED
    assert lib.opm_accumulator_size(None, 4, 4, ctypes.byref(n)) == T.TRI_MUL_EINVAL
    assert lib.opm_block_accumulate(None, None, 16, 16, None, 16, 16, 16, 1 << 20, None) == T.TRI_MUL_EINVAL
    assert lib.opm_forward(None, 16, 16, None, 4, 4, 16, 16, 1 << 20, None) == T.TRI_MUL_EINVAL
    assert lib.opm_destroy(None) == T.TRI_MUL_OK
    assert lib.tri_attn_chunk(None, 16, 16, 16, 16, None, None, 16, None) == T.TRI_MUL_EINVAL
    bad = T.TriAttnView(1, 64, 4, T.TRI_MUL_F32, 60, 0, 64, 0, 1)        # ld_bias not a multiple of 8
    assert lib.tri_attn_state_size(ctypes.byref(bad), ctypes.byref(n)) == T.TRI_MUL_EINVAL
    good = T.TriAttnView(2, 64, 4, T.TRI_MUL_F32, 64, 0, 64, 0, 1)
    assert lib.tri_attn_state_size(ctypes.byref(good), ctypes.byref(n)) == T.TRI_MUL_OK
    assert n.value == (2 * 64 * 4 * 32 + 2 * 2 * 4 * 64) * 4
    assert lib.tri_attn_forward(None, 16, 16, 16, None, 1, 64, 4, 64, 0, 16, None) == T.TRI_MUL_EINVAL


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


def test_block_view_leading_dimension_bounds(lib):
    # validation runs before the handle's contents are used, so a dummy
    # (non-null, never dereferenced) handle reaches the view checks
    dummy = ctypes.c_void_p(16)
    base = dict(n_total=4096, row0=0, col0=0, rows=256, cols=256, k0=0, klen=256, k_index=0, k_count=2)
    v = T.BlockView(**base, ld_a=65536 + 8, ld_b=256)
    assert lib.tri_mul_block_accumulate(dummy, ctypes.byref(v), 16, 16, 16, None, None, None, None) == \
        T.TRI_MUL_EUNSUPPORTED
    assert "65536" in T.last_error()
    v = T.BlockView(**base, ld_a=256, ld_b=1 << 24)
    assert lib.tri_mul_block_accumulate(dummy, ctypes.byref(v), 16, 16, 16, None, None, None, None) == \
        T.TRI_MUL_EUNSUPPORTED
    v = T.BlockView(**base, ld_a=252, ld_b=256)   # below klen
    assert lib.tri_mul_block_accumulate(dummy, ctypes.byref(v), 16, 16, 16, None, None, None, None) == \
        T.TRI_MUL_EINVAL
