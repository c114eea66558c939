"""Thin Python binding of libtrimul.so (the C ABI in include/tri_mul.h,
include/opm.h and include/triattn.h).

Argument marshalling only: every step of the update runs in the library's HIP
kernels.  PyTorch provides device memory and streams.  The functions keep the
C names; TriMul and OuterProductMean are small convenience wrappers that own
a handle.
"""
import ctypes
import os

import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libtrimul.so")

TRI_MUL_OK, TRI_MUL_EINVAL, TRI_MUL_EUNSUPPORTED, TRI_MUL_ENOMEM, TRI_MUL_EHIP = 0, -1, -2, -3, -4
TRI_MUL_F32, TRI_MUL_BF16 = 0, 1
TRI_MUL_OUTGOING, TRI_MUL_INCOMING = 0, 1
DTYPE_CODE = {"f32": TRI_MUL_F32, "bf16": TRI_MUL_BF16}
TORCH_DTYPE = {TRI_MUL_F32: torch.float32, TRI_MUL_BF16: torch.bfloat16}
WEIGHT_FIELDS = ("ln_in_w", "ln_in_b", "w_a", "w_ga", "w_b", "w_gb", "w_g", "ln_out_w", "ln_out_b", "w_o")
# weight (and weight-gradient) shapes for c_z = c = 128
WEIGHT_SHAPES = {"ln_in_w": (128,), "ln_in_b": (128,), "w_a": (128, 128), "w_ga": (128, 128), "w_b": (128, 128),
                 "w_gb": (128, 128), "w_g": (128, 128), "ln_out_w": (128,), "ln_out_b": (128,), "w_o": (128, 128)}

_vp = ctypes.c_void_p
_i32, _i64 = ctypes.c_int32, ctypes.c_int64


class Params(ctypes.Structure):
    _fields_ = [("c_z", _i32), ("c", _i32), ("dtype", _i32), ("out_dtype", _i32), ("ln_eps", ctypes.c_float)] + \
               [(name, _vp) for name in WEIGHT_FIELDS]


class BlockView(ctypes.Structure):
    _fields_ = [("n_total", _i64), ("row0", _i64), ("col0", _i64), ("rows", _i64), ("cols", _i64),
                ("k0", _i64), ("klen", _i64), ("ld_a", _i64), ("ld_b", _i64),
                ("k_index", _i32), ("k_count", _i32)]


class OpmParams(ctypes.Structure):
    """opm_params_t."""
    _fields_ = [("d", _i32), ("c_z", _i32), ("out_dtype", _i32), ("w_o", _vp), ("b_o", _vp)]


class OpmBlockView(ctypes.Structure):
    """opm_block_view_t."""
    _fields_ = [("n_total", _i64), ("s_total", _i64), ("row0", _i64), ("rows", _i64), ("col0", _i64),
                ("cols", _i64), ("s0", _i64), ("slen", _i64), ("k_index", _i32), ("k_count", _i32)]


class TriAttnView(ctypes.Structure):
    """tri_attn_view_t."""
    _fields_ = [("rows", _i64), ("n", _i64), ("heads", _i32), ("out_dtype", _i32), ("ld_bias", _i64),
                ("k0", _i64), ("klen", _i64), ("k_index", _i32), ("k_count", _i32)]


class LoadCheck(ctypes.Structure):
    """tri_mul_load_check_t (include/tri_mul_check.h)."""
    _fields_ = [("tiles", _i64), ("loads", _i64), ("elems", _i64), ("bad_tiles", _i64), ("bad_desc", _i64),
                ("bad_elem", _i64)]


TRI_MUL_OPERAND_BLOCKED, TRI_MUL_OPERAND_ROW_MAJOR, TRI_MUL_OPERAND_TRANSPOSED = 0, 1, 2


class Grads(ctypes.Structure):
    """tri_mul_grads_t: device pointers of the float32 weight gradients."""
    _fields_ = [(name, _vp) for name in WEIGHT_FIELDS]


# name -> (restype, argtypes); the same order and meaning as include/tri_mul.h
SIGNATURES = {
    "tri_mul_init": (ctypes.c_int, [ctypes.POINTER(_vp), ctypes.POINTER(Params), _vp]),
    "tri_mul_destroy": (ctypes.c_int, [_vp]),
    "tri_mul_last_error": (ctypes.c_char_p, []),
    "tri_mul_workspace_size": (ctypes.c_int, [_vp, _i64, ctypes.POINTER(ctypes.c_size_t)]),
    "tri_mul_panel_size": (ctypes.c_int, [_vp, _i64, ctypes.POINTER(ctypes.c_size_t)]),
    "tri_mul_outgoing": (ctypes.c_int, [_vp, _vp, _vp, _i64, _vp, _vp, ctypes.c_size_t, _vp]),
    "tri_mul_incoming": (ctypes.c_int, [_vp, _vp, _vp, _i64, _vp, _vp, ctypes.c_size_t, _vp]),
    "tri_mul_update_noalloc": (ctypes.c_int, [_vp, _vp, _vp, _i64, _i32, _vp, _vp]),
    "tri_mul_block_accumulate": (ctypes.c_int, [_vp, ctypes.POINTER(BlockView), _vp, _vp, _vp, _vp, _vp, _vp, _vp]),
    "tri_mul_block_workspace_size": (ctypes.c_int, [_vp, ctypes.POINTER(BlockView), ctypes.POINTER(ctypes.c_size_t)]),
    "tri_mul_block_accumulate_ws": (ctypes.c_int, [_vp, ctypes.POINTER(BlockView), _vp, _vp, _vp, _vp, _vp, _vp, _vp,
                                                    ctypes.c_size_t, _vp]),
    "tri_mul_block_accumulator_size": (ctypes.c_int, [_vp, ctypes.POINTER(BlockView), ctypes.POINTER(ctypes.c_size_t)]),
    "tri_mul_block_repack": (ctypes.c_int, [_vp, ctypes.POINTER(BlockView), _vp, _vp, _vp, _vp, ctypes.c_size_t, _vp]),
    "tri_mul_block_accumulate_packed": (ctypes.c_int, [_vp, ctypes.POINTER(BlockView), _vp, ctypes.c_size_t, _vp, _vp,
                                                        _vp, _vp, _i32, _vp]),
    "tri_mul_block_panel_size": (ctypes.c_int, [_vp, _i64, _i64, ctypes.POINTER(ctypes.c_size_t)]),
    "tri_mul_block_project": (ctypes.c_int, [_vp, _vp, _i64, _vp, _i64, _i64, _i64, _i64, _i64, _i32, _vp, _vp, _vp]),
    "tri_mul_block_accumulate_blocked": (ctypes.c_int, [_vp, ctypes.POINTER(BlockView), _vp, _vp, _vp, _vp, _vp,
                                                         _vp, _i32, _vp]),
    "tri_mul_block_accumulate_transposed": (ctypes.c_int, [_vp, ctypes.POINTER(BlockView), _vp, _vp, _vp, _vp,
                                                            _vp, _vp, _i32, _vp]),
    "tri_mul_project": (ctypes.c_int, [_vp, _vp, _vp, _i64, _i32, _vp, _vp, _vp]),
    "tri_mul_contract": (ctypes.c_int, [_vp, _vp, _vp, _i64, _vp, _vp]),
    "tri_mul_contract_transposed": (ctypes.c_int, [_vp, _vp, _vp, _i64, _vp, _vp]),
    "tri_mul_epilogue": (ctypes.c_int, [_vp, _vp, _vp, _vp, _i64, _vp, _vp]),
    "tri_mul_contract_backward_workspace_size": (ctypes.c_int, [_vp, _i64, ctypes.POINTER(ctypes.c_size_t)]),
    "tri_mul_contract_backward": (ctypes.c_int, [_vp, _vp, _vp, _vp, _i64, _vp, _vp, _vp, ctypes.c_size_t, _vp]),
    "tri_mul_backward_workspace_size": (ctypes.c_int, [_vp, _i64, ctypes.POINTER(ctypes.c_size_t)]),
    "tri_mul_outgoing_backward": (ctypes.c_int, [_vp, _vp, _vp, _i64, _vp, _vp, ctypes.POINTER(Grads), _vp,
                                                 ctypes.c_size_t, _vp]),
    "tri_mul_incoming_backward": (ctypes.c_int, [_vp, _vp, _vp, _i64, _vp, _vp, ctypes.POINTER(Grads), _vp,
                                                 ctypes.c_size_t, _vp]),
    "tri_mul_outgoing_backward_saved": (ctypes.c_int, [_vp, _vp, _vp, _i64, _vp, _vp, _vp, _vp, _vp,
                                                        ctypes.POINTER(Grads), _vp, ctypes.c_size_t, _vp]),
    "tri_mul_incoming_backward_saved": (ctypes.c_int, [_vp, _vp, _vp, _i64, _vp, _vp, _vp, _vp, _vp,
                                                        ctypes.POINTER(Grads), _vp, ctypes.c_size_t, _vp]),
    "opm_init": (ctypes.c_int, [ctypes.POINTER(_vp), ctypes.POINTER(OpmParams), _vp]),
    "opm_destroy": (ctypes.c_int, [_vp]),
    "opm_accumulator_size": (ctypes.c_int, [_vp, _i64, _i64, ctypes.POINTER(ctypes.c_size_t)]),
    "opm_workspace_size": (ctypes.c_int, [_vp, _i64, _i64, _i64, ctypes.POINTER(ctypes.c_size_t)]),
    "opm_block_accumulate": (ctypes.c_int, [_vp, ctypes.POINTER(OpmBlockView), _vp, _vp, _vp, _vp, _vp, _vp,
                                            ctypes.c_size_t, _vp]),
    "opm_forward_workspace_size": (ctypes.c_int, [_vp, _i64, _i64, ctypes.POINTER(ctypes.c_size_t)]),
    "opm_forward": (ctypes.c_int, [_vp, _vp, _vp, _vp, _i64, _i64, _vp, _vp, ctypes.c_size_t, _vp]),
    "tri_mul_check_contract_loads": (ctypes.c_int, [ctypes.c_int, ctypes.c_int, _i64, _i64, _i64, _i64, _i64, _i64,
                                                    _i64, ctypes.c_int, ctypes.c_uint64, ctypes.c_uint64, ctypes.c_int,
                                                    ctypes.c_int, ctypes.POINTER(LoadCheck)]),
    "tri_mul_check_contract_result": (ctypes.c_int, [_i64, _i64, ctypes.c_int, ctypes.c_uint64, ctypes.c_int,
                                                      ctypes.POINTER(LoadCheck)]),
    "tri_attn_state_size": (ctypes.c_int, [ctypes.POINTER(TriAttnView), ctypes.POINTER(ctypes.c_size_t)]),
    "tri_attn_chunk": (ctypes.c_int, [ctypes.POINTER(TriAttnView), _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp]),
    "tri_attn_forward": (ctypes.c_int, [_vp, _vp, _vp, _vp, _vp, _i64, _i64, ctypes.c_int32, _i64, ctypes.c_int32,
                                        _vp, _vp]),
}

_lib = None


class TriMulError(RuntimeError):
    def __init__(self, code, msg):
        super().__init__(f"tri_mul error {code}: {msg}")
        self.code = code


def lib():
    """Load libtrimul.so from the package directory (it must have been built:
    python -m paper_2603_14806_amd.build).  There is no fallback."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing; build it with `python -m paper_2603_14806_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in SIGNATURES.items():
            f = getattr(L, name)
            f.restype, f.argtypes = res, args
        _lib = L
    return _lib


def last_error():
    return lib().tri_mul_last_error().decode()


def _check(rc):
    if rc != TRI_MUL_OK:
        raise TriMulError(rc, last_error())


def _ptr(t):
    if t is None:
        return None
    if not isinstance(t, torch.Tensor):
        return t                       # already an address (int) or None
    if t.device.type != "cuda":
        raise ValueError("tensors passed to the library must live on the GPU")
    return t.data_ptr()


def _stream(stream):
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    return stream.cuda_stream if hasattr(stream, "cuda_stream") else stream


# ---------------------------------------------------------------- C names

def tri_mul_init(weights, dtype="bf16", out_dtype="f32", eps=1e-5, c_z=128, c=128, stream=None):
    """weights: dict of device tensors (WEIGHT_FIELDS) in the storage dtype."""
    p = Params(c_z, c, DTYPE_CODE[dtype], DTYPE_CODE[out_dtype], eps,
               *[_ptr(weights[n]) for n in WEIGHT_FIELDS])
    h = _vp()
    _check(lib().tri_mul_init(ctypes.byref(h), ctypes.byref(p), _stream(stream)))
    return h


def tri_mul_destroy(h):
    _check(lib().tri_mul_destroy(h))


def tri_mul_workspace_size(h, N):
    n = ctypes.c_size_t()
    _check(lib().tri_mul_workspace_size(h, N, ctypes.byref(n)))
    return n.value


def tri_mul_panel_size(h, N):
    n = ctypes.c_size_t()
    _check(lib().tri_mul_panel_size(h, N, ctypes.byref(n)))
    return n.value


def tri_mul_outgoing(h, z, mask, N, out, ws, ws_bytes, stream=None):
    _check(lib().tri_mul_outgoing(h, _ptr(z), _ptr(mask), N, _ptr(out), _ptr(ws), ws_bytes, _stream(stream)))


def tri_mul_incoming(h, z, mask, N, out, ws, ws_bytes, stream=None):
    _check(lib().tri_mul_incoming(h, _ptr(z), _ptr(mask), N, _ptr(out), _ptr(ws), ws_bytes, _stream(stream)))


def tri_mul_update_noalloc(h, z, mask, N, direction, out, stream=None):
    _check(lib().tri_mul_update_noalloc(h, _ptr(z), _ptr(mask), N, direction, _ptr(out), _stream(stream)))


def tri_mul_block_accumulate(h, view, a_panel, b_panel, acc, mask, z_tile, out_tile, stream=None):
    _check(lib().tri_mul_block_accumulate(h, ctypes.byref(view), _ptr(a_panel), _ptr(b_panel), _ptr(acc),
                                          _ptr(mask), _ptr(z_tile), _ptr(out_tile), _stream(stream)))


def tri_mul_block_workspace_size(h, view):
    n = ctypes.c_size_t()
    _check(lib().tri_mul_block_workspace_size(h, ctypes.byref(view), ctypes.byref(n)))
    return n.value


def tri_mul_block_accumulate_ws(h, view, a_panel, b_panel, acc, mask, z_tile, out_tile, ws, ws_bytes, stream=None):
    _check(lib().tri_mul_block_accumulate_ws(h, ctypes.byref(view), _ptr(a_panel), _ptr(b_panel), _ptr(acc),
                                             _ptr(mask), _ptr(z_tile), _ptr(out_tile), _ptr(ws), ws_bytes,
                                             _stream(stream)))


def tri_mul_block_accumulator_size(h, view):
    n = ctypes.c_size_t()
    _check(lib().tri_mul_block_accumulator_size(h, ctypes.byref(view), ctypes.byref(n)))
    return n.value


def tri_mul_block_repack(h, view, a_panel, b_panel, mask, ws, ws_bytes, stream=None):
    _check(lib().tri_mul_block_repack(h, ctypes.byref(view), _ptr(a_panel), _ptr(b_panel), _ptr(mask), _ptr(ws),
                                      ws_bytes, _stream(stream)))


def tri_mul_block_accumulate_packed(h, view, ws, ws_bytes, acc, mask, z_tile, out_tile, reserve_cus=0, stream=None):
    _check(lib().tri_mul_block_accumulate_packed(h, ctypes.byref(view), _ptr(ws), ws_bytes, _ptr(acc), _ptr(mask),
                                                 _ptr(z_tile), _ptr(out_tile), reserve_cus, _stream(stream)))


def tri_mul_block_panel_size(h, rows, klen):
    n = ctypes.c_size_t()
    _check(lib().tri_mul_block_panel_size(h, rows, klen, ctypes.byref(n)))
    return n.value


def tri_mul_block_project(h, z_tile, ld_z, mask, n_total, row0, col0, rows, cols, direction, a_panel, b_panel,
                          stream=None):
    _check(lib().tri_mul_block_project(h, _ptr(z_tile), ld_z, _ptr(mask), n_total, row0, col0, rows, cols,
                                       direction, _ptr(a_panel), _ptr(b_panel), _stream(stream)))


def tri_mul_block_accumulate_blocked(h, view, a_panel, b_panel, acc, mask, z_tile, out_tile, reserve_cus=0,
                                     stream=None):
    _check(lib().tri_mul_block_accumulate_blocked(h, ctypes.byref(view), _ptr(a_panel), _ptr(b_panel), _ptr(acc),
                                                  _ptr(mask), _ptr(z_tile), _ptr(out_tile), reserve_cus,
                                                  _stream(stream)))


def tri_mul_block_accumulate_transposed(h, view, at_panel, bt_panel, acc, mask, z_tile, out_tile, reserve_cus=0,
                                        stream=None):
    _check(lib().tri_mul_block_accumulate_transposed(h, ctypes.byref(view), _ptr(at_panel), _ptr(bt_panel),
                                                     _ptr(acc), _ptr(mask), _ptr(z_tile), _ptr(out_tile),
                                                     reserve_cus, _stream(stream)))


def tri_mul_project(h, z, mask, N, direction, a_panels, b_panels, stream=None):
    _check(lib().tri_mul_project(h, _ptr(z), _ptr(mask), N, direction, _ptr(a_panels), _ptr(b_panels),
                                 _stream(stream)))


def tri_mul_contract(h, a_panels, b_panels, N, c_out, stream=None):
    _check(lib().tri_mul_contract(h, _ptr(a_panels), _ptr(b_panels), N, _ptr(c_out), _stream(stream)))


def tri_mul_contract_transposed(h, at_panels, bt_panels, N, c_out, stream=None):
    _check(lib().tri_mul_contract_transposed(h, _ptr(at_panels), _ptr(bt_panels), N, _ptr(c_out), _stream(stream)))


def tri_mul_epilogue(h, c_in, z, mask, N, out, stream=None):
    _check(lib().tri_mul_epilogue(h, _ptr(c_in), _ptr(z), _ptr(mask), N, _ptr(out), _stream(stream)))


def tri_mul_contract_backward_workspace_size(h, N):
    n = ctypes.c_size_t()
    _check(lib().tri_mul_contract_backward_workspace_size(h, N, ctypes.byref(n)))
    return n.value


def tri_mul_contract_backward(h, dC, a_panels, b_panels, N, dA, dB, ws, ws_bytes, stream=None):
    _check(lib().tri_mul_contract_backward(h, _ptr(dC), _ptr(a_panels), _ptr(b_panels), N, _ptr(dA), _ptr(dB),
                                           _ptr(ws), ws_bytes, _stream(stream)))


def tri_mul_backward_workspace_size(h, N):
    n = ctypes.c_size_t()
    _check(lib().tri_mul_backward_workspace_size(h, N, ctypes.byref(n)))
    return n.value


def tri_mul_layer_backward(h, direction, z, mask, N, dout, dz, grads, ws, ws_bytes, stream=None):
    """grads: dict WEIGHT_FIELDS -> float32 device tensors (overwritten)."""
    g = Grads(*[_ptr(grads[n]) for n in WEIGHT_FIELDS])
    f = lib().tri_mul_incoming_backward if direction in (TRI_MUL_INCOMING, "incoming") else lib().tri_mul_outgoing_backward
    _check(f(h, _ptr(z), _ptr(mask), N, _ptr(dout), _ptr(dz), ctypes.byref(g), _ptr(ws), ws_bytes, _stream(stream)))


def tri_mul_layer_backward_saved(h, direction, z, mask, N, a_panels, b_panels, c_result, dout, dz, grads, ws,
                                 ws_bytes, stream=None):
    """The layer backward from the forward's saved A, B panels and C result."""
    g = Grads(*[_ptr(grads[n]) for n in WEIGHT_FIELDS])
    f = (lib().tri_mul_incoming_backward_saved if direction in (TRI_MUL_INCOMING, "incoming")
         else lib().tri_mul_outgoing_backward_saved)
    _check(f(h, _ptr(z), _ptr(mask), N, _ptr(a_panels), _ptr(b_panels), _ptr(c_result), _ptr(dout), _ptr(dz),
             ctypes.byref(g), _ptr(ws), ws_bytes, _stream(stream)))


# ---------------------------------------------------------------- wrapper

class TriMul:
    """Owns a handle and allocates outputs / workspace with torch."""

    def __init__(self, weights, dtype="bf16", out_dtype="f32", eps=1e-5, device="cuda", stream=None):
        self.dtype, self.out_dtype = dtype, out_dtype
        self.device = torch.device(device)
        wd = {k: v.to(self.device, TORCH_DTYPE[DTYPE_CODE[dtype]]).contiguous() for k, v in weights.items()}
        self.h = tri_mul_init(wd, dtype, out_dtype, eps, stream=stream)
        torch.cuda.synchronize(self.device)
        self._ws = None

    def close(self):
        if self.h:
            tri_mul_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def workspace(self, N):
        need = tri_mul_workspace_size(self.h, N)
        if self._ws is None or self._ws.numel() < need:
            self._ws = None
            self._ws = torch.empty(need, dtype=torch.uint8, device=self.device)
        return self._ws, need

    def _out(self, N, out):
        if out is None:
            out = torch.empty((N, N, 128), dtype=TORCH_DTYPE[DTYPE_CODE[self.out_dtype]], device=self.device)
        return out

    def outgoing(self, z, mask=None, out=None, stream=None):
        N = z.shape[0]
        out = self._out(N, out)
        ws, need = self.workspace(N)
        tri_mul_outgoing(self.h, z, mask, N, out, ws, need, stream)
        return out

    def incoming(self, z, mask=None, out=None, stream=None):
        N = z.shape[0]
        out = self._out(N, out)
        ws, need = self.workspace(N)
        tri_mul_incoming(self.h, z, mask, N, out, ws, need, stream)
        return out

    def __call__(self, z, mask=None, direction="outgoing", out=None, stream=None):
        return (self.outgoing if direction == "outgoing" else self.incoming)(z, mask, out, stream)

    def project(self, z, mask=None, direction="outgoing", stream=None):
        """Returns the two operands in the library's panel layout (flat
        tensors; see panel_to_dense)."""
        N = z.shape[0]
        t = TORCH_DTYPE[DTYPE_CODE[self.dtype]]
        n = tri_mul_panel_size(self.h, N) // torch.empty((), dtype=t).element_size()
        A = torch.empty(n, dtype=t, device=self.device)
        B = torch.empty(n, dtype=t, device=self.device)
        tri_mul_project(self.h, z, mask, N, TRI_MUL_OUTGOING if direction == "outgoing" else TRI_MUL_INCOMING,
                        A, B, stream)
        return A, B

    def contract(self, A, B, N, stream=None):
        """A, B in the panel layout (project / dense_to_panel); returns C in
        the result layout (flat; see result_to_dense)."""
        C = torch.empty(N * (-(-N // 32) * 32) * 128, dtype=torch.float32, device=self.device)
        tri_mul_contract(self.h, A, B, N, C, stream)
        return C

    def contract_transposed(self, AT, BT, N, stream=None):
        """The same C as contract(A, B, N) from the operands transposed,
        i.e. from project(z, mask, <the opposite direction>)."""
        C = torch.empty(N * (-(-N // 32) * 32) * 128, dtype=torch.float32, device=self.device)
        tri_mul_contract_transposed(self.h, AT, BT, N, C, stream)
        return C

    def epilogue(self, C, z, mask=None, out=None, stream=None):
        """C in the result layout (contract / dense_to_result)."""
        N = z.shape[0]
        out = self._out(N, out)
        tri_mul_epilogue(self.h, C, z, mask, N, out, stream)
        return out

    def contract_backward(self, dC, A, B, N, stream=None):
        """Gradients of the contraction: dC in the result layout, A, B in the
        panel layout; returns (dA, dB), both in the result layout (flat)."""
        n = N * (-(-N // 32) * 32) * 128
        dA = torch.empty(n, dtype=torch.float32, device=self.device)
        dB = torch.empty(n, dtype=torch.float32, device=self.device)
        wsb = tri_mul_contract_backward_workspace_size(self.h, N)
        ws = torch.empty(wsb, dtype=torch.uint8, device=self.device)
        tri_mul_contract_backward(self.h, dC, A, B, N, dA, dB, ws, wsb, stream)
        return dA, dB

    def backward(self, z, dout, mask=None, direction="outgoing", stream=None, saved=None):
        """Gradients of sum(out * dout) for the update of z: returns (dz,
        grads) with grads a dict of float32 tensors shaped like the weights.
        saved = (AT, BT, C) skips the recomputation of the forward: AT, BT
        from project(z, mask, <the opposite direction>) -- the direction's
        operands transposed, as the full calls leave them in their workspace
        -- and C the direction's contraction (contract_transposed(AT, BT))."""
        N = z.shape[0]
        cz = 128
        if tuple(z.shape) != (N, N, cz) or tuple(dout.shape) != (N, N, cz):
            raise ValueError(f"z and dout must be [N, N, {cz}], got {tuple(z.shape)} and {tuple(dout.shape)}")
        if dout.dtype != TORCH_DTYPE[DTYPE_CODE[self.out_dtype]] or z.dtype != TORCH_DTYPE[DTYPE_CODE[self.dtype]]:
            raise ValueError("z must have the storage dtype and dout the output dtype of the layer")
        if not (z.is_contiguous() and dout.is_contiguous()):
            raise ValueError("z and dout must be contiguous")
        grads = {k: torch.empty(v, dtype=torch.float32, device=self.device) for k, v in WEIGHT_SHAPES.items()}
        dz = torch.empty_like(z)
        wsb = tri_mul_backward_workspace_size(self.h, N)
        ws = torch.empty(wsb, dtype=torch.uint8, device=self.device)
        if saved is None:
            tri_mul_layer_backward(self.h, direction, z, mask, N, dout, dz, grads, ws, wsb, stream)
        else:
            tri_mul_layer_backward_saved(self.h, direction, z, mask, N, *saved, dout, dz, grads, ws, wsb, stream)
        return dz, grads

    def block_accumulate(self, view, a_panel, b_panel, acc, mask=None, z_tile=None, out_tile=None, stream=None,
                         ws=None):
        """One ring step; with `ws` (a uint8 device tensor of at least
        block_workspace_size(view) bytes) through the repacking entry point."""
        if ws is None:
            tri_mul_block_accumulate(self.h, view, a_panel, b_panel, acc, mask, z_tile, out_tile, stream)
        else:
            tri_mul_block_accumulate_ws(self.h, view, a_panel, b_panel, acc, mask, z_tile, out_tile, ws,
                                        ws.numel() * ws.element_size(), stream)

    def block_workspace_size(self, view):
        return tri_mul_block_workspace_size(self.h, view)

    def block_accumulator_size(self, view):
        return tri_mul_block_accumulator_size(self.h, view)

    def block_repack(self, view, a_panel, b_panel, mask, ws, stream=None):
        tri_mul_block_repack(self.h, view, a_panel, b_panel, mask, ws, ws.numel() * ws.element_size(), stream)

    def block_accumulate_packed(self, view, ws, acc, mask=None, z_tile=None, out_tile=None, reserve_cus=0,
                                stream=None):
        tri_mul_block_accumulate_packed(self.h, view, ws, ws.numel() * ws.element_size(), acc, mask, z_tile,
                                        out_tile, reserve_cus, stream)

    def block_panel_size(self, rows, klen):
        return tri_mul_block_panel_size(self.h, rows, klen)

    def block_project(self, z_tile, mask, n_total, row0, col0, direction="outgoing", ld_z=None, stream=None):
        """The tile's two blocked panels (new bf16 device tensors of
        block_panel_size elements / 2): z_tile [rows][ld_z][c_z] holds pairs
        (row0 + i, col0 + j), j < cols = z_tile.shape[1] unless ld_z is given."""
        d = TRI_MUL_INCOMING if direction in (TRI_MUL_INCOMING, "incoming") else TRI_MUL_OUTGOING
        rows, cols = z_tile.shape[0], z_tile.shape[1]
        ldz = cols if ld_z is None else ld_z
        m, k = (cols, rows) if d == 1 else (rows, cols)
        n = tri_mul_block_panel_size(self.h, m, k) // 2
        a = torch.empty(n, dtype=torch.bfloat16, device=z_tile.device)
        b = torch.empty_like(a)
        tri_mul_block_project(self.h, z_tile, ldz, mask, n_total, row0, col0, rows, cols, d, a, b, stream)
        return a, b

    def block_accumulate_blocked(self, view, a_panel, b_panel, acc, mask=None, z_tile=None, out_tile=None,
                                 reserve_cus=0, stream=None):
        tri_mul_block_accumulate_blocked(self.h, view, a_panel, b_panel, acc, mask, z_tile, out_tile, reserve_cus,
                                         stream)

    def block_accumulate_transposed(self, view, at_panel, bt_panel, acc, mask=None, z_tile=None, out_tile=None,
                                    reserve_cus=0, stream=None):
        """The ring step from the panels block_project writes with the
        opposite direction (the operands transposed)."""
        tri_mul_block_accumulate_transposed(self.h, view, at_panel, bt_panel, acc, mask, z_tile, out_tile,
                                            reserve_cus, stream)


# ------------------------------------------------------ panel layout views

def _panel_dims(N, c=128):
    T, S = -(-N // 256), -(-N // 32)
    return c, T, S


def panel_to_dense(P, N, c=128, klen=None):
    """Panel-layout operand (flat) of N rows and klen (default N)
    contraction indices -> dense [c][N][klen] (a view copy)."""
    K = N if klen is None else klen
    T, S = -(-N // 256), -(-K // 32)
    X = P.reshape(c, T, S, 256, 32).permute(0, 1, 3, 2, 4).reshape(c, T * 256, S * 32)
    return X[:, :N, :K]


def dense_to_panel(X):
    """Dense [c][N][N] -> flat panel-layout operand (zero padding)."""
    c, N = X.shape[0], X.shape[1]
    _, T, S = _panel_dims(N, c)
    Y = torch.zeros((c, T * 256, S * 32), dtype=X.dtype, device=X.device)
    Y[:, :N, :N] = X
    return Y.reshape(c, T, 256, S, 32).permute(0, 1, 3, 2, 4).contiguous().reshape(-1)


def result_to_dense(Cr, N, c=128, cols=None):
    """Result-layout C (flat) over N rows and `cols` columns (default N) ->
    dense [c][N][cols] (a device tile's packed accumulator has this layout)."""
    cols = N if cols is None else cols
    J = -(-cols // 32)
    return Cr.reshape(N, J, c, 32).permute(2, 0, 1, 3).reshape(c, N, J * 32)[:, :, :cols]


def dense_to_result(C):
    """Dense [c][N][N] -> flat result-layout C (zero padding)."""
    c, N = C.shape[0], C.shape[1]
    J = -(-N // 32)
    Y = torch.zeros((c, N, J * 32), dtype=C.dtype, device=C.device)
    Y[:, :, :N] = C
    return Y.reshape(c, N, J, 32).permute(1, 2, 0, 3).contiguous().reshape(-1)


# ---------------------------------------------------------------- outer product mean (include/opm.h)

def opm_init(w_o, b_o=None, out_dtype="f32", d=32, c_z=128, stream=None):
    """w_o: [c_z][d * d] bf16 device tensor; b_o: [c_z] bf16 device tensor or None."""
    p = OpmParams(d, c_z, DTYPE_CODE[out_dtype], _ptr(w_o), _ptr(b_o))
    h = _vp()
    _check(lib().opm_init(ctypes.byref(h), ctypes.byref(p), _stream(stream)))
    return h


def opm_destroy(h):
    _check(lib().opm_destroy(h))


def opm_accumulator_size(h, rows, cols):
    n = ctypes.c_size_t()
    _check(lib().opm_accumulator_size(h, rows, cols, ctypes.byref(n)))
    return n.value


def opm_workspace_size(h, rows, cols, slen):
    n = ctypes.c_size_t()
    _check(lib().opm_workspace_size(h, rows, cols, slen, ctypes.byref(n)))
    return n.value


def opm_block_accumulate(h, view, a, b, mask, acc, out_tile, ws, ws_bytes, stream=None):
    _check(lib().opm_block_accumulate(h, ctypes.byref(view), _ptr(a), _ptr(b), _ptr(mask), _ptr(acc),
                                      _ptr(out_tile), _ptr(ws), ws_bytes, _stream(stream)))


def opm_forward_workspace_size(h, S, N):
    n = ctypes.c_size_t()
    _check(lib().opm_forward_workspace_size(h, S, N, ctypes.byref(n)))
    return n.value


def opm_forward(h, a, b, mask, S, N, out, ws, ws_bytes, stream=None):
    _check(lib().opm_forward(h, _ptr(a), _ptr(b), _ptr(mask), S, N, _ptr(out), _ptr(ws), ws_bytes,
                             _stream(stream)))


class OuterProductMean:
    """Owns an opm handle and allocates outputs / workspaces with torch."""

    def __init__(self, w_o, b_o=None, out_dtype="f32", device="cuda", stream=None):
        self.out_dtype = out_dtype
        self.device = torch.device(device)
        self._w = w_o.to(self.device, torch.bfloat16).contiguous()
        self._b = None if b_o is None else b_o.to(self.device, torch.bfloat16).contiguous()
        self.h = opm_init(self._w, self._b, out_dtype, stream=stream)
        torch.cuda.synchronize(self.device)

    def close(self):
        if self.h:
            opm_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def _out(self, rows, cols):
        return torch.empty((rows, cols, 128), dtype=TORCH_DTYPE[DTYPE_CODE[self.out_dtype]], device=self.device)

    def forward(self, a, b, mask=None, stream=None):
        """a, b: [S][N][32] bf16 device tensors; mask: [S][N] uint8 or None -> out [N][N][128]."""
        S, N = a.shape[0], a.shape[1]
        if a.dtype != torch.bfloat16 or b.dtype != torch.bfloat16 or a.shape != b.shape or a.shape[2] != 32:
            raise ValueError("a and b must be [S][N][32] bf16 tensors of the same shape")
        if not (a.is_contiguous() and b.is_contiguous()):
            raise ValueError("a and b must be contiguous")
        out = self._out(N, N)
        n = opm_forward_workspace_size(self.h, S, N)
        ws = torch.empty(n, dtype=torch.uint8, device=self.device)
        opm_forward(self.h, a, b, mask, S, N, out, ws, n, stream)
        return out

    def accumulator(self, rows, cols):
        return torch.empty(opm_accumulator_size(self.h, rows, cols) // 4, dtype=torch.float32, device=self.device)

    def block_accumulate(self, view, a, b, mask, acc, out_tile=None, stream=None):
        n = opm_workspace_size(self.h, view.rows, view.cols, view.slen)
        ws = torch.empty(n, dtype=torch.uint8, device=self.device)
        opm_block_accumulate(self.h, view, a, b, mask, acc, out_tile, ws, n, stream)


# ---------------------------------------------------------------- triangle attention core (include/triattn.h)

def tri_attn_state_size(view):
    n = ctypes.c_size_t()
    _check(lib().tri_attn_state_size(ctypes.byref(view), ctypes.byref(n)))
    return n.value


def tri_attn_chunk(view, q, k, v, bias, mask, state, out, stream=None):
    _check(lib().tri_attn_chunk(ctypes.byref(view), _ptr(q), _ptr(k), _ptr(v), _ptr(bias), _ptr(mask), _ptr(state),
                                _ptr(out), _stream(stream)))


def tri_attn_forward(q, k, v, bias, mask, rows, n, heads, ld_bias, out_dtype, out, stream=None):
    _check(lib().tri_attn_forward(_ptr(q), _ptr(k), _ptr(v), _ptr(bias), _ptr(mask), rows, n, heads, ld_bias,
                                  DTYPE_CODE.get(out_dtype, out_dtype), _ptr(out), _stream(stream)))


def triangle_attention(q, k, v, bias, mask=None, out_dtype="f32", stream=None):
    """q, k, v: [rows][n][heads][32] bf16 device tensors; bias: [heads][n][ld] bf16 with ld % 8 == 0
    (a view [heads][n][n] of such a tensor is fine); mask: [n] uint8 or None -> out [rows][n][heads][32]."""
    rows, n, heads, d = q.shape
    if d != 32 or k.shape != q.shape or v.shape != q.shape:
        raise ValueError("q, k, v must be [rows][n][heads][32] of one shape")
    if not (q.is_contiguous() and k.is_contiguous() and v.is_contiguous()):
        raise ValueError("q, k and v must be contiguous")
    if bias.dim() != 3 or bias.shape[0] != heads or bias.shape[1] != n or bias.stride(2) != 1 or bias.stride(0) != n * bias.stride(1):
        raise ValueError("bias must be [heads][n][ld] with unit column stride")
    out = torch.empty((rows, n, heads, 32), dtype=TORCH_DTYPE[DTYPE_CODE[out_dtype]], device=q.device)
    tri_attn_forward(q, k, v, bias, mask, rows, n, heads, bias.stride(1), out_dtype, out, stream)
    return out


def check_contract_loads(a_mode, b_mode, M, N, K, lda=0, ldb=0, a_stride=0, b_stride=0, batch=128, a_bytes=0,
                         b_bytes=0, grid=256, all_channels=False):
    """Host-side walk over the contraction kernel's loads for one launch shape
    (tri_mul_check_contract_loads); returns the counts as a dict."""
    out = LoadCheck()
    _check(lib().tri_mul_check_contract_loads(a_mode, b_mode, M, N, K, lda, ldb, a_stride, b_stride, batch, a_bytes,
                                              b_bytes, grid, int(all_channels), ctypes.byref(out)))
    return {name: getattr(out, name) for name, _ in LoadCheck._fields_}


def check_contract_result(M, N, batch=128, c_bytes=0, all_channels=False):
    """Host-side walk over the contraction kernel's accesses to a pair-blocked
    C (tri_mul_check_contract_result); returns the counts as a dict."""
    out = LoadCheck()
    _check(lib().tri_mul_check_contract_result(M, N, batch, c_bytes, int(all_channels), ctypes.byref(out)))
    return {name: getattr(out, name) for name, _ in LoadCheck._fields_}
