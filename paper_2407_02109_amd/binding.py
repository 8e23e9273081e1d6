"""ctypes binding of the Flash Swin C ABI (``include/fla_swin.h``).

Argument marshalling only: every step of the attention runs inside ``libfla_swin.so``.
Tensors are passed as raw device pointers (``tensor.data_ptr()``); the stream defaults to
PyTorch's current HIP stream.  If the library has not been built, the first call raises
``FlaError`` -- there is no fallback.
"""
from __future__ import annotations

import ctypes
import os
import threading

FLA_PAD_MASK = 0
FLA_PAD_KVTOKEN = 1

_LIB_NAME = "libfla_swin.so"
_lib = None
_lock = threading.Lock()


class FlaError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__("fla_swin: %s (status %d)" % (message, status))
        self.status = status


def library_path() -> str:
    return os.path.join(os.path.dirname(os.path.abspath(__file__)), _LIB_NAME)


def _declare(lib):
    P, I, D = ctypes.c_void_p, ctypes.c_int, ctypes.POINTER(ctypes.c_double)
    fwd_args = [P, P, P, P, I, I, I, I, I, I, I, I, P]
    lib.fla_swin_attn_fwd.argtypes = fwd_args
    lib.fla_swin_attn_fwd.restype = I
    lib.fla_swin_attn_fwd_f32.argtypes = fwd_args
    lib.fla_swin_attn_fwd_f32.restype = I
    lib.fla_status_string.argtypes = [I]
    lib.fla_status_string.restype = ctypes.c_char_p
    lib.fla_swin_attn_work.argtypes = [I, I, I, I, I, I, I, I, I, D, D]
    lib.fla_swin_attn_work.restype = I
    IP = ctypes.POINTER(ctypes.c_int)
    ms_args = [P, P, P, P, I, I, I, IP, I, I, I, I, P]
    lib.fla_swin_attn_ms_fwd.argtypes = ms_args
    lib.fla_swin_attn_ms_fwd.restype = I
    lib.fla_swin_attn_ms_fwd_f32.argtypes = ms_args
    lib.fla_swin_attn_ms_fwd_f32.restype = I
    lib.fla_swin_attn_ms_work.argtypes = [I, I, I, IP, I, I, I, I, I, D, D]
    lib.fla_swin_attn_ms_work.restype = I


def load_library():
    """Load (once) and return the ctypes handle of libfla_swin.so."""
    global _lib
    if _lib is not None:
        return _lib
    with _lock:
        if _lib is None:
            path = library_path()
            if not os.path.exists(path):
                raise FlaError(-1, "%s is not built; run __graft_entry__.build()" % path)
            lib = ctypes.CDLL(path)
            _declare(lib)
            _lib = lib
    return _lib


def _ptr(x):
    if x is None:
        return None
    if isinstance(x, int):
        return x
    return x.data_ptr()


def _stream(stream):
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def _check(rc):
    if rc != 0:
        raise FlaError(rc, fla_status_string(rc))


def fla_status_string(status: int) -> str:
    return load_library().fla_status_string(int(status)).decode()


def fla_swin_attn_fwd(q, k, v, out, B, heads, Hgrid, Wgrid, head_dim, window, shift,
                      pad_mode=FLA_PAD_MASK, stream=None, check=True) -> int:
    """bf16 forward.  q, k, v, out: tensors or raw device addresses."""
    rc = load_library().fla_swin_attn_fwd(
        _ptr(q), _ptr(k), _ptr(v), _ptr(out), B, heads, Hgrid, Wgrid, head_dim,
        window, shift, pad_mode, _stream(stream))
    if check:
        _check(rc)
    return rc


def fla_swin_attn_fwd_f32(q, k, v, out, B, heads, Hgrid, Wgrid, head_dim, window, shift,
                          pad_mode=FLA_PAD_MASK, stream=None, check=True) -> int:
    """fp32 forward.  q, k, v, out: tensors or raw device addresses."""
    rc = load_library().fla_swin_attn_fwd_f32(
        _ptr(q), _ptr(k), _ptr(v), _ptr(out), B, heads, Hgrid, Wgrid, head_dim,
        window, shift, pad_mode, _stream(stream))
    if check:
        _check(rc)
    return rc


def fla_swin_attn_work(B, heads, Hgrid, Wgrid, head_dim, window, shift, pad_mode, elem_bytes):
    """(flops, bytes) of one call, computed by the library on the host."""
    f, b = ctypes.c_double(), ctypes.c_double()
    rc = load_library().fla_swin_attn_work(B, heads, Hgrid, Wgrid, head_dim, window, shift,
                                           pad_mode, elem_bytes, ctypes.byref(f), ctypes.byref(b))
    _check(rc)
    return f.value, b.value


def _grid_array(grids):
    """(H, W) pairs -> (n, c_int array of 2n), or (0, None) for None."""
    if grids is None:
        return 0, None
    flat = [int(t) for hw in grids for t in hw]
    return len(flat) // 2, (ctypes.c_int * max(len(flat), 1))(*flat)


def fla_swin_attn_ms_fwd(q, k, v, out, B, heads, grids, head_dim, window, shift,
                         pad_mode=FLA_PAD_MASK, stream=None, check=True) -> int:
    """Multi-scale bf16 forward; grids: sequence of (H, W), tokens of each grid one after
    the other in q, k, v and out."""
    n, arr = _grid_array(grids)
    rc = load_library().fla_swin_attn_ms_fwd(
        _ptr(q), _ptr(k), _ptr(v), _ptr(out), B, heads, n, arr, head_dim, window, shift,
        pad_mode, _stream(stream))
    if check:
        _check(rc)
    return rc


def fla_swin_attn_ms_fwd_f32(q, k, v, out, B, heads, grids, head_dim, window, shift,
                             pad_mode=FLA_PAD_MASK, stream=None, check=True) -> int:
    """Multi-scale fp32 forward."""
    n, arr = _grid_array(grids)
    rc = load_library().fla_swin_attn_ms_fwd_f32(
        _ptr(q), _ptr(k), _ptr(v), _ptr(out), B, heads, n, arr, head_dim, window, shift,
        pad_mode, _stream(stream))
    if check:
        _check(rc)
    return rc


def fla_swin_attn_ms_work(B, heads, grids, head_dim, window, shift, pad_mode, elem_bytes):
    """(flops, bytes) of one multi-scale call."""
    n, arr = _grid_array(grids)
    f, b = ctypes.c_double(), ctypes.c_double()
    rc = load_library().fla_swin_attn_ms_work(B, heads, n, arr, head_dim, window, shift, pad_mode,
                                              elem_bytes, ctypes.byref(f), ctypes.byref(b))
    _check(rc)
    return f.value, b.value


def swin_attn_ms(q, k, v, grids, window, shift, pad_mode=FLA_PAD_MASK, out=None, stream=None):
    """Tensor-level multi-scale wrapper: q [B, sum(H*W), heads, d]; k/v with one more row
    (the shared pad token) in KV-token mode.  Allocates ``out`` when not given."""
    import torch
    if q.dtype not in (torch.bfloat16, torch.float32):
        raise TypeError("q must be bfloat16 or float32")
    for t in (q, k, v):
        if t.dtype != q.dtype or not t.is_cuda or not t.is_contiguous():
            raise ValueError("q, k, v must share dtype and be contiguous device tensors")
    B, L, heads, d = q.shape
    if out is None:
        out = torch.empty_like(q)
    fn = fla_swin_attn_ms_fwd if q.dtype == torch.bfloat16 else fla_swin_attn_ms_fwd_f32
    fn(q, k, v, out, B, heads, grids, d, window, shift, pad_mode, stream)
    return out


def swin_attn(q, k, v, Hgrid, Wgrid, window, shift, pad_mode=FLA_PAD_MASK, out=None, stream=None):
    """Tensor-level convenience wrapper: q [B, L, heads, d] (bf16 or fp32, on the GPU,
    contiguous), k/v [B, L(+1), heads, d].  Allocates ``out`` when not given."""
    import torch
    if q.dtype not in (torch.bfloat16, torch.float32):
        raise TypeError("q must be bfloat16 or float32")
    for t in (q, k, v):
        if t.dtype != q.dtype or not t.is_cuda or not t.is_contiguous():
            raise ValueError("q, k, v must share dtype and be contiguous device tensors")
    B, L, heads, d = q.shape
    if out is None:
        out = torch.empty_like(q)
    fn = fla_swin_attn_fwd if q.dtype == torch.bfloat16 else fla_swin_attn_fwd_f32
    fn(q, k, v, out, B, heads, Hgrid, Wgrid, d, window, shift, pad_mode, stream)
    return out
