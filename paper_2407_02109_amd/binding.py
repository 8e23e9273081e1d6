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
    lse_args = [P, P, P, P, P, I, I, I, I, I, I, I, I, P]
    ms_lse_args = [P, P, P, P, P, I, I, I, IP, I, I, I, I, P]
    for name, args in (("fla_swin_attn_fwd_lse", lse_args), ("fla_swin_attn_fwd_lse_f32", lse_args),
                       ("fla_swin_attn_ms_fwd_lse", ms_lse_args),
                       ("fla_swin_attn_ms_fwd_lse_f32", ms_lse_args)):
        getattr(lib, name).argtypes = args
        getattr(lib, name).restype = I
    Z = ctypes.c_size_t
    bwd_args = [P, P, P, P, P, P, P, P, P, P, Z, I, I, I, I, I, I, I, I, P]
    ms_bwd_args = [P, P, P, P, P, P, P, P, P, P, Z, I, I, I, IP, I, I, I, I, P]
    for name, args in (("fla_swin_attn_bwd", bwd_args), ("fla_swin_attn_bwd_f32", bwd_args),
                       ("fla_swin_attn_ms_bwd", ms_bwd_args), ("fla_swin_attn_ms_bwd_f32", ms_bwd_args)):
        getattr(lib, name).argtypes = args
        getattr(lib, name).restype = I
    lib.fla_swin_attn_bwd_noalloc.argtypes = [P] * 9 + [I, I, I, I, I, I, I, I, P]
    lib.fla_swin_attn_bwd_noalloc.restype = I
    lib.fla_swin_attn_bwd_workspace.argtypes = [I, I, I, IP, I, I, I, ctypes.POINTER(Z)]
    lib.fla_swin_attn_bwd_workspace.restype = I
    lib.fla_swin_attn_bwd_work.argtypes = [I, I, I, IP, I, I, I, I, I, D, D]
    lib.fla_swin_attn_bwd_work.restype = I
    F = ctypes.c_float
    rope_args = [P, P, P, P, I, I, I, I, I, I, I, I, F, F, P]
    for name in ("fla_swin_attn_rope_fwd", "fla_swin_attn_rope_fwd_f32"):
        getattr(lib, name).argtypes = rope_args
        getattr(lib, name).restype = I
    lib.fla_swin_attn_rope_fwd_lse.argtypes = [P, P, P, P, P, I, I, I, I, I, I, I, I, F, F, P]
    lib.fla_swin_attn_rope_fwd_lse.restype = I
    lib.fla_swin_attn_rope_bwd.argtypes = [P] * 10 + [Z, I, I, I, I, I, I, I, I, F, F, P]
    lib.fla_swin_attn_rope_bwd.restype = I
    lib.fla_cycle_scan.argtypes = [P] * 7 + [Z, I, I, I, I, I, P]
    lib.fla_cycle_scan.restype = I
    lib.fla_cycle_scan_workspace.argtypes = [I, I, I, I, I, ctypes.POINTER(Z)]
    lib.fla_cycle_scan_workspace.restype = I
    lib.fla_cycle_scan_work.argtypes = [I, I, I, I, I, D, D]
    lib.fla_cycle_scan_work.restype = I


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
    _check_shapes(q, k, v, sum(int(h) * int(w) for h, w in grids), pad_mode, *([out] if out is not None else []))
    B, L, heads, d = q.shape
    if out is None:
        out = torch.empty_like(q)
    fn = fla_swin_attn_ms_fwd if q.dtype == torch.bfloat16 else fla_swin_attn_ms_fwd_f32
    fn(q, k, v, out, B, heads, grids, d, window, shift, pad_mode, stream)
    return out


def swin_attn(q, k, v, Hgrid, Wgrid, window, shift, pad_mode=FLA_PAD_MASK, out=None, stream=None):
    """Tensor-level convenience wrapper: q [B, L, heads, d] or [B, Hgrid, Wgrid, heads, d]
    (bf16 or fp32, on the GPU, contiguous), k/v likewise ([B, L + 1, heads, d] in KV-token
    mode).  Allocates ``out`` (q's shape) when not given."""
    import torch
    if q.dtype not in (torch.bfloat16, torch.float32):
        raise TypeError("q must be bfloat16 or float32")
    for t in (q, k, v):
        if t.dtype != q.dtype or not t.is_cuda or not t.is_contiguous():
            raise ValueError("q, k, v must share dtype and be contiguous device tensors")
    shape = q.shape
    flat = lambda t: t.reshape(t.shape[0], t.shape[1] * t.shape[2], t.shape[3], t.shape[4]) if t.dim() == 5 else t
    q4, k4, v4 = flat(q), flat(k), flat(v)
    if q.dim() == 5 and (q.shape[1], q.shape[2]) != (Hgrid, Wgrid):
        raise ValueError("q is %s but the grid is %dx%d" % (tuple(q.shape), Hgrid, Wgrid))
    _check_shapes(q4, k4, v4, Hgrid * Wgrid, pad_mode, *([flat(out)] if out is not None else []))
    if out is None:
        out = torch.empty_like(q)
    out4 = flat(out)
    B, L, heads, d = q4.shape
    fn = fla_swin_attn_fwd if q.dtype == torch.bfloat16 else fla_swin_attn_fwd_f32
    fn(q4, k4, v4, out4, B, heads, Hgrid, Wgrid, d, window, shift, pad_mode, stream)
    return out.reshape(shape)


# ---- training: forward with log-sum-exp, backward ------------------------------------------

def fla_swin_attn_fwd_lse(q, k, v, out, lse, B, heads, Hgrid, Wgrid, head_dim, window, shift,
                          pad_mode=FLA_PAD_MASK, stream=None, check=True, f32=False) -> int:
    """Training forward (bf16, or fp32 with f32=True): out and lse [B, heads, L] fp32."""
    fn = load_library().fla_swin_attn_fwd_lse_f32 if f32 else load_library().fla_swin_attn_fwd_lse
    rc = fn(_ptr(q), _ptr(k), _ptr(v), _ptr(out), _ptr(lse), B, heads, Hgrid, Wgrid, head_dim,
            window, shift, pad_mode, _stream(stream))
    if check:
        _check(rc)
    return rc


def fla_swin_attn_ms_fwd_lse(q, k, v, out, lse, B, heads, grids, head_dim, window, shift,
                             pad_mode=FLA_PAD_MASK, stream=None, check=True, f32=False) -> int:
    """Multi-scale training forward."""
    n, arr = _grid_array(grids)
    lib = load_library()
    fn = lib.fla_swin_attn_ms_fwd_lse_f32 if f32 else lib.fla_swin_attn_ms_fwd_lse
    rc = fn(_ptr(q), _ptr(k), _ptr(v), _ptr(out), _ptr(lse), B, heads, n, arr, head_dim, window,
            shift, pad_mode, _stream(stream))
    if check:
        _check(rc)
    return rc


def fla_swin_attn_bwd_workspace(B, heads, grids, window, shift, pad_mode=FLA_PAD_MASK) -> int:
    """Workspace bytes the backward needs (0 in mask mode)."""
    n, arr = _grid_array(grids)
    out = ctypes.c_size_t()
    _check(load_library().fla_swin_attn_bwd_workspace(B, heads, n, arr, window, shift, pad_mode,
                                                      ctypes.byref(out)))
    return out.value


def fla_swin_attn_bwd(q, k, v, out, dout, lse, dq, dk, dv, workspace, workspace_bytes, B, heads,
                      Hgrid, Wgrid, head_dim, window, shift, pad_mode=FLA_PAD_MASK, stream=None,
                      check=True, f32=False) -> int:
    """Backward (bf16, or fp32 with f32=True); all tensors as raw addresses or tensors."""
    lib = load_library()
    fn = lib.fla_swin_attn_bwd_f32 if f32 else lib.fla_swin_attn_bwd
    rc = fn(_ptr(q), _ptr(k), _ptr(v), _ptr(out), _ptr(dout), _ptr(lse), _ptr(dq), _ptr(dk), _ptr(dv),
            _ptr(workspace), int(workspace_bytes), B, heads, Hgrid, Wgrid, head_dim, window, shift,
            pad_mode, _stream(stream))
    if check:
        _check(rc)
    return rc


def fla_swin_attn_bwd_noalloc(q, k, v, out, dout, lse, dq, dk, dv, B, heads, Hgrid, Wgrid, head_dim, window,
                              shift, pad_mode=FLA_PAD_MASK, stream=None, check=True) -> int:
    """Allocation-free bf16 backward: the library's static device scratch is the workspace."""
    lib = load_library()
    rc = lib.fla_swin_attn_bwd_noalloc(_ptr(q), _ptr(k), _ptr(v), _ptr(out), _ptr(dout), _ptr(lse), _ptr(dq),
                                       _ptr(dk), _ptr(dv), B, heads, Hgrid, Wgrid, head_dim, window, shift,
                                       pad_mode, _stream(stream))
    if check:
        _check(rc)
    return rc


def fla_swin_attn_ms_bwd(q, k, v, out, dout, lse, dq, dk, dv, workspace, workspace_bytes, B, heads,
                         grids, head_dim, window, shift, pad_mode=FLA_PAD_MASK, stream=None,
                         check=True, f32=False) -> int:
    """Multi-scale backward."""
    n, arr = _grid_array(grids)
    lib = load_library()
    fn = lib.fla_swin_attn_ms_bwd_f32 if f32 else lib.fla_swin_attn_ms_bwd
    rc = fn(_ptr(q), _ptr(k), _ptr(v), _ptr(out), _ptr(dout), _ptr(lse), _ptr(dq), _ptr(dk), _ptr(dv),
            _ptr(workspace), int(workspace_bytes), B, heads, n, arr, head_dim, window, shift,
            pad_mode, _stream(stream))
    if check:
        _check(rc)
    return rc


def fla_swin_attn_bwd_work(B, heads, grids, head_dim, window, shift, pad_mode, elem_bytes):
    """(flops, bytes) of one backward call."""
    n, arr = _grid_array(grids)
    f, b = ctypes.c_double(), ctypes.c_double()
    _check(load_library().fla_swin_attn_bwd_work(B, heads, n, arr, head_dim, window, shift, pad_mode,
                                                 elem_bytes, ctypes.byref(f), ctypes.byref(b)))
    return f.value, b.value


def _check_shapes(q, k, v, L, pad_mode, *like_q):
    """Raise ValueError unless q [B, L, heads, d] and k, v [B, L (+1 in KV-token mode), heads, d]
    (and every tensor in like_q has q's shape): the C ABI trusts the sizes it is given, so a
    mismatch here would read or write outside the tensors."""
    if q.dim() != 4 or q.shape[1] != L:
        raise ValueError("q must be [B, %d, heads, head_dim], got %s" % (L, tuple(q.shape)))
    rows = L + (1 if pad_mode == FLA_PAD_KVTOKEN else 0)
    want = (q.shape[0], rows, q.shape[2], q.shape[3])
    for name, t in (("k", k), ("v", v)):
        if tuple(t.shape) != want:
            raise ValueError("%s must be %s, got %s" % (name, want, tuple(t.shape)))
    for t in like_q:
        if tuple(t.shape) != tuple(q.shape):
            raise ValueError("expected a tensor of q's shape %s, got %s" % (tuple(q.shape), tuple(t.shape)))


def _check_tensors(*ts):
    import torch
    t0 = ts[0]
    if t0.dtype not in (torch.bfloat16, torch.float32):
        raise TypeError("tensors must be bfloat16 or float32")
    for t in ts:
        if t.dtype != t0.dtype or not t.is_cuda or not t.is_contiguous():
            raise ValueError("tensors must share dtype and be contiguous device tensors")
    return t0.dtype == torch.float32


def swin_attn_fwd_train(q, k, v, grids, window, shift, pad_mode=FLA_PAD_MASK, stream=None):
    """Training forward over a grid list ((H, W), ...): returns (out, lse)."""
    import torch
    f32 = _check_tensors(q, k, v)
    _check_shapes(q, k, v, sum(int(h) * int(w) for h, w in grids), pad_mode)
    B, L, heads, d = q.shape
    out = torch.empty_like(q)
    lse = torch.empty((B, heads, L), dtype=torch.float32, device=q.device)
    fla_swin_attn_ms_fwd_lse(q, k, v, out, lse, B, heads, grids, d, window, shift, pad_mode, stream,
                             f32=f32)
    return out, lse


def swin_attn_bwd(q, k, v, out, dout, lse, grids, window, shift, pad_mode=FLA_PAD_MASK, stream=None):
    """Backward over a grid list: returns (dq, dk, dv); allocates the workspace it needs."""
    import torch
    f32 = _check_tensors(q, k, v, out, dout)
    if lse.dtype != torch.float32 or not lse.is_contiguous():
        raise ValueError("lse must be a contiguous float32 tensor")
    _check_shapes(q, k, v, sum(int(h) * int(w) for h, w in grids), pad_mode, out, dout)
    B, L, heads, d = q.shape
    if tuple(lse.shape) != (B, heads, L):
        raise ValueError("lse must be [B, heads, L] = %s, got %s" % ((B, heads, L), tuple(lse.shape)))
    dq, dk, dv = torch.empty_like(q), torch.empty_like(k), torch.empty_like(v)
    nbytes = fla_swin_attn_bwd_workspace(B, heads, grids, window, shift, pad_mode)
    ws = torch.empty(max(nbytes, 16), dtype=torch.uint8, device=q.device)
    fla_swin_attn_ms_bwd(q, k, v, out, dout, lse, dq, dk, dv, ws, nbytes, B, heads, grids, d, window,
                         shift, pad_mode, stream, f32=f32)
    return dq, dk, dv


# ---- forward with 2-D RoPE fused into its prologue ---------------------------------------

def fla_swin_attn_rope_fwd(q, k, v, out, B, heads, Hgrid, Wgrid, head_dim, window, shift,
                           pad_mode=FLA_PAD_MASK, rope_theta=10000.0, rope_scale=1.0, stream=None,
                           check=True, f32=False) -> int:
    """Forward of RoPE-rotated q and k (bf16, or fp32 with f32=True)."""
    lib = load_library()
    fn = lib.fla_swin_attn_rope_fwd_f32 if f32 else lib.fla_swin_attn_rope_fwd
    rc = fn(_ptr(q), _ptr(k), _ptr(v), _ptr(out), B, heads, Hgrid, Wgrid, head_dim, window, shift,
            pad_mode, float(rope_theta), float(rope_scale), _stream(stream))
    if check:
        _check(rc)
    return rc


def swin_attn_rope(q, k, v, Hgrid, Wgrid, window, shift, pad_mode=FLA_PAD_MASK, rope_theta=10000.0,
                   rope_scale=1.0, out=None, stream=None):
    """Tensor-level RoPE forward; allocates ``out`` when not given."""
    import torch
    f32 = _check_tensors(q, k, v)
    _check_shapes(q, k, v, Hgrid * Wgrid, pad_mode, *([out] if out is not None else []))
    B, L, heads, d = q.shape
    if out is None:
        out = torch.empty_like(q)
    fla_swin_attn_rope_fwd(q, k, v, out, B, heads, Hgrid, Wgrid, d, window, shift, pad_mode, rope_theta,
                           rope_scale, stream, f32=f32)
    return out


def fla_swin_attn_rope_fwd_lse(q, k, v, out, lse, B, heads, Hgrid, Wgrid, head_dim, window, shift,
                               pad_mode=FLA_PAD_MASK, rope_theta=10000.0, rope_scale=1.0, stream=None,
                               check=True) -> int:
    """bf16 RoPE training forward: out and lse of the rotated q, k."""
    lib = load_library()
    rc = lib.fla_swin_attn_rope_fwd_lse(_ptr(q), _ptr(k), _ptr(v), _ptr(out), _ptr(lse), B, heads, Hgrid, Wgrid,
                                        head_dim, window, shift, pad_mode, float(rope_theta), float(rope_scale),
                                        _stream(stream))
    if check:
        _check(rc)
    return rc


def fla_swin_attn_rope_bwd(q, k, v, out, dout, lse, dq, dk, dv, workspace, workspace_bytes, B, heads,
                           Hgrid, Wgrid, head_dim, window, shift, pad_mode=FLA_PAD_MASK, rope_theta=10000.0,
                           rope_scale=1.0, stream=None, check=True) -> int:
    """bf16 RoPE backward: gradients with respect to the unrotated q, k and v."""
    lib = load_library()
    rc = lib.fla_swin_attn_rope_bwd(_ptr(q), _ptr(k), _ptr(v), _ptr(out), _ptr(dout), _ptr(lse), _ptr(dq),
                                    _ptr(dk), _ptr(dv), _ptr(workspace), int(workspace_bytes), B, heads, Hgrid,
                                    Wgrid, head_dim, window, shift, pad_mode, float(rope_theta), float(rope_scale),
                                    _stream(stream))
    if check:
        _check(rc)
    return rc


def swin_attn_rope_fwd_train(q, k, v, Hgrid, Wgrid, window, shift, pad_mode=FLA_PAD_MASK, rope_theta=10000.0,
                             rope_scale=1.0, stream=None):
    """bf16 RoPE training forward on one grid: returns (out, lse)."""
    import torch
    if _check_tensors(q, k, v):
        raise ValueError("RoPE training takes bf16 tensors")
    _check_shapes(q, k, v, int(Hgrid) * int(Wgrid), pad_mode)
    B, L, heads, d = q.shape
    out = torch.empty_like(q)
    lse = torch.empty((B, heads, L), dtype=torch.float32, device=q.device)
    fla_swin_attn_rope_fwd_lse(q, k, v, out, lse, B, heads, Hgrid, Wgrid, d, window, shift, pad_mode, rope_theta,
                               rope_scale, stream)
    return out, lse


def swin_attn_rope_bwd(q, k, v, out, dout, lse, Hgrid, Wgrid, window, shift, pad_mode=FLA_PAD_MASK,
                       rope_theta=10000.0, rope_scale=1.0, stream=None):
    """bf16 RoPE backward on one grid: returns (dq, dk, dv) of the unrotated q, k, v."""
    import torch
    if _check_tensors(q, k, v, out, dout):
        raise ValueError("RoPE training takes bf16 tensors")
    _check_shapes(q, k, v, int(Hgrid) * int(Wgrid), pad_mode, out, dout)
    B, L, heads, d = q.shape
    if lse.dtype != torch.float32 or tuple(lse.shape) != (B, heads, L) or not lse.is_contiguous():
        raise ValueError("lse must be a contiguous float32 [B, heads, L] tensor")
    dq, dk, dv = torch.empty_like(q), torch.empty_like(k), torch.empty_like(v)
    nbytes = fla_swin_attn_bwd_workspace(B, heads, [(Hgrid, Wgrid)], window, shift, pad_mode)
    ws = torch.empty(max(nbytes, 16), dtype=torch.uint8, device=q.device)
    fla_swin_attn_rope_bwd(q, k, v, out, dout, lse, dq, dk, dv, ws, nbytes, B, heads, Hgrid, Wgrid, d, window,
                           shift, pad_mode, rope_theta, rope_scale, stream)
    return dq, dk, dv


_autograd_fn = None


def _swin_attention_function():
    """torch.autograd.Function over the training forward (keeps out and lse) and the backward
    kernels; built on first use so that importing the package does not import torch."""
    global _autograd_fn
    if _autograd_fn is not None:
        return _autograd_fn
    import torch

    class SwinAttention(torch.autograd.Function):
        @staticmethod
        def forward(ctx, q, k, v, grids, window, shift, pad_mode, rope):
            q, k, v = q.contiguous(), k.contiguous(), v.contiguous()
            if rope is None:
                out, lse = swin_attn_fwd_train(q, k, v, grids, window, shift, pad_mode)
            else:
                (H, W), = grids
                out, lse = swin_attn_rope_fwd_train(q, k, v, H, W, window, shift, pad_mode, rope[0], rope[1])
            ctx.save_for_backward(q, k, v, out, lse)
            ctx.cfg = (grids, window, shift, pad_mode, rope)
            return out

        @staticmethod
        def backward(ctx, dout):
            q, k, v, out, lse = ctx.saved_tensors
            grids, window, shift, pad_mode, rope = ctx.cfg
            dout = dout.contiguous()
            if rope is None:
                dq, dk, dv = swin_attn_bwd(q, k, v, out, dout, lse, grids, window, shift, pad_mode)
            else:
                (H, W), = grids
                dq, dk, dv = swin_attn_rope_bwd(q, k, v, out, dout, lse, H, W, window, shift, pad_mode, rope[0],
                                                rope[1])
            return dq, dk, dv, None, None, None, None, None

    _autograd_fn = SwinAttention
    return SwinAttention


def swin_attention(q, k, v, grids, window, shift, pad_mode=FLA_PAD_MASK, rope=None):
    """Differentiable Flash Swin attention (torch autograd): q [B, L, heads, 64], k and v the
    same (one more row, the pad token, in KV-token mode), on the current stream.  grids is
    [(H, W)] or a multi-scale grid list; rope = (theta, scale) fuses 2-D RoPE of q and k
    (bf16, one grid).  The forward keeps each query's log-sum-exp for the backward."""
    grids = [(int(h), int(w)) for h, w in grids]
    if rope is not None:
        if len(grids) != 1:
            raise ValueError("RoPE takes a single grid")
        rope = (float(rope[0]), float(rope[1]))
    return _swin_attention_function().apply(q, k, v, grids, int(window), int(shift), int(pad_mode), rope)


# ---- Cycle-scan (Sec. 3.5) ----------------------------------------------------------------

def fla_cycle_scan_workspace(B, L, d, N, repeats=3) -> int:
    """Workspace bytes of one fla_cycle_scan call."""
    n = ctypes.c_size_t()
    _check(load_library().fla_cycle_scan_workspace(B, L, d, N, repeats, ctypes.byref(n)))
    return n.value


def fla_cycle_scan(x, delta, A, Bm, Cm, y, workspace, workspace_bytes, B, L, d, N, repeats=3, stream=None,
                   check=True) -> int:
    """fp32 Cycle-scan through the C ABI.  Tensors or raw device addresses."""
    rc = load_library().fla_cycle_scan(_ptr(x), _ptr(delta), _ptr(A), _ptr(Bm), _ptr(Cm), _ptr(y), _ptr(workspace),
                                       workspace_bytes, B, L, d, N, repeats, _stream(stream))
    if check:
        _check(rc)
    return rc


def fla_cycle_scan_work(B, L, d, N, repeats=3):
    """(exponentials, bytes) of one Cycle-scan call."""
    e, b = ctypes.c_double(), ctypes.c_double()
    _check(load_library().fla_cycle_scan_work(B, L, d, N, repeats, ctypes.byref(e), ctypes.byref(b)))
    return e.value, b.value


def cycle_scan(x, delta, A, Bm, Cm, repeats=3, out=None, stream=None):
    """Cycle-scan of x [B, L, d] with delta [B, L, d], A [d, N], Bm, Cm [B, L, N] (contiguous fp32
    device tensors); returns y [B, L, d].  Allocates the output (unless given) and the workspace."""
    import torch
    for t in (x, delta, A, Bm, Cm):
        if t.dtype != torch.float32 or not t.is_cuda or not t.is_contiguous():
            raise ValueError("Cycle-scan tensors must be contiguous float32 device tensors")
    if x.dim() != 3 or tuple(delta.shape) != tuple(x.shape):
        raise ValueError("x and delta must be [B, L, d] of one shape")
    B, L, d = x.shape
    if A.dim() != 2 or A.shape[0] != d:
        raise ValueError("A must be [d, N], got %s" % (tuple(A.shape),))
    N = A.shape[1]
    for name, t in (("Bm", Bm), ("Cm", Cm)):
        if tuple(t.shape) != (B, L, N):
            raise ValueError("%s must be %s, got %s" % (name, (B, L, N), tuple(t.shape)))
    y = torch.empty_like(x) if out is None else out
    if tuple(y.shape) != tuple(x.shape) or y.dtype != torch.float32 or not y.is_contiguous():
        raise ValueError("out must be a contiguous float32 tensor of x's shape")
    nws = fla_cycle_scan_workspace(B, L, d, N, repeats)
    ws = torch.empty(max(nws, 4), dtype=torch.uint8, device=x.device)
    fla_cycle_scan(x, delta, A, Bm, Cm, y, ws, ws.numel(), B, L, d, N, repeats, stream)
    return y

