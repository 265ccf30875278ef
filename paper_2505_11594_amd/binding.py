"""Thin ctypes binding over ``libsage_mi355x.so`` (declared in include/sage_mi355x.h).

Argument marshalling only: every step of the attention path runs in the HIP
kernels.  torch supplies device memory and the current stream.  If the
library has not been built, ``lib()`` raises: there is no fallback path.
"""
from __future__ import annotations

import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libsage_mi355x.so")

SAGE_OK, SAGE_ERR_INVALID_ARG, SAGE_ERR_UNSUPPORTED, SAGE_ERR_HIP, SAGE_ERR_WORKSPACE = 0, 1, 2, 3, 4
SAGE_FMT_MXFP4, SAGE_FMT_NV16_E4M3 = 0x0, 0x1
SAGE_IN_FP16, SAGE_IN_BF16 = 0x0, 0x4
SAGE_OUT_F32 = 0x8
SAGE_NO_SMOOTH_K = 0x10
SAGE_SMOOTH_Q = 0x20
SAGE_BKV64 = 0x40
SAGE_BKV256 = 0x80
SAGE_WG256 = 0x100       # 256 queries per workgroup (MXFP4, 256-key tiles, non-causal, no smoothing Q)


def bkv_flag(bkv: int) -> int:
    """The fmt bit that selects a KV tile of ``bkv`` keys (64, 128 or 256)."""
    return {64: SAGE_BKV64, 128: 0, 256: SAGE_BKV256}[bkv]
SAGE_ROLE_Q, SAGE_ROLE_K, SAGE_ROLE_V = 0, 1, 2

_lib = None


class SageError(RuntimeError):
    def __init__(self, fn: str, status: int):
        super().__init__("%s failed: %s" % (fn, status_string(status)))
        self.status = status


def lib():
    """Load the in-tree HIP library (raises if it has not been built).

    torch is imported first: its wheel carries its own HIP runtime under the
    same soname as ROCm's, and the runtime loaded first is the one every
    later library binds to.  Loading this library before torch would map
    ROCm's runtime next to torch's, and device pointers and streams would
    cross between the two."""
    global _lib
    if _lib is None:
        import torch  # noqa: F401  (see above)
        if not os.path.exists(LIB_PATH):
            raise RuntimeError("libsage_mi355x.so is not built; run __graft_entry__.build() "
                               "or python paper_2505_11594_amd/build.py")
        L = ctypes.CDLL(LIB_PATH)
        vp, i, u, sz = ctypes.c_void_p, ctypes.c_int, ctypes.c_uint, ctypes.c_size_t
        L.sage_quant_sizes.argtypes = [i, i, i, i, i, u, ctypes.POINTER(sz), ctypes.POINTER(sz)]
        L.sage_quant_workspace_size.argtypes = [i, i, i, i, i, u]
        L.sage_quant_workspace_size.restype = sz
        L.sage_quant_fp4.argtypes = [vp, i, i, i, i, i, u, vp, vp, vp, vp, sz, vp]
        L.sage_attn_fp4_workspace_size.argtypes = [i, i, i, i, u]
        L.sage_attn_fp4_workspace_size.restype = sz
        L.sage_attn_fp4_fwd.argtypes = [vp, vp, vp, vp, i, i, i, i, i, u, vp]
        L.sage_attn_fp4_fwd_ws.argtypes = [vp, vp, vp, vp, i, i, i, i, i, u, vp, sz, vp]
        L.sage_attn_fp4_fwd_noalloc.argtypes = [vp, vp, vp, vp, i, i, i, i, i, u, vp]
        L.sage_attn_fp4_fwd_prequant.argtypes = [vp] * 7 + [i, i, i, i, i, u, vp]
        L.sage_attn_bf16_fwd.argtypes = [vp, vp, vp, vp, i, i, i, i, i, u, vp]
        L.sage_quant_int8_sizes.argtypes = [i, i, i, i, i, u, ctypes.POINTER(sz), ctypes.POINTER(sz)]
        L.sage_quant_int8.argtypes = [vp, i, i, i, i, i, u, vp, vp, vp, vp, sz, vp]
        L.sage_attn_int8_workspace_size.argtypes = [i, i, i, i, u]
        L.sage_attn_int8_workspace_size.restype = sz
        L.sage_attn_int8_fwd.argtypes = [vp, vp, vp, vp, vp, i, i, i, i, i, u, vp]
        L.sage_attn_int8_fwd_ws.argtypes = [vp, vp, vp, vp, vp, i, i, i, i, i, u, vp, sz, vp]
        L.sage_attn_int8_fwd_prequant.argtypes = [vp] * 8 + [i, i, i, i, i, u, vp]
        L.sage_attn_int8_bwd.argtypes = [vp] * 9 + [i, i, i, i, i, u, vp]
        L.sage_attn_int8_bwd_ws.argtypes = [vp] * 9 + [i, i, i, i, i, u, vp, sz, vp]
        L.sage_attn_int8_bwd_workspace_size.argtypes = [i, i, i, i, u]
        L.sage_attn_int8_bwd_workspace_size.restype = sz
        L.sage_attn_int8_bwd_min_workspace_size.argtypes = [i, i, i, i, u]
        L.sage_attn_int8_bwd_min_workspace_size.restype = sz
        L.sage_status_string.argtypes = [i]
        L.sage_status_string.restype = ctypes.c_char_p
        L.sage_version.restype = ctypes.c_char_p
        for name in ("sage_quant_sizes", "sage_quant_fp4", "sage_attn_fp4_fwd", "sage_attn_fp4_fwd_ws",
                     "sage_attn_fp4_fwd_noalloc", "sage_attn_fp4_fwd_prequant", "sage_attn_bf16_fwd", "sage_quant_int8_sizes",
                     "sage_quant_int8", "sage_attn_int8_fwd", "sage_attn_int8_fwd_ws",
                     "sage_attn_int8_fwd_prequant", "sage_attn_int8_bwd", "sage_attn_int8_bwd_ws"):
            getattr(L, name).restype = i
        _lib = L
    return _lib


def status_string(status: int) -> str:
    return lib().sage_status_string(int(status)).decode()


def _check(fn: str, rc: int):
    if rc != SAGE_OK:
        raise SageError(fn, rc)


def _stream():
    import torch
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def _ptr(t):
    return ctypes.c_void_p(t.data_ptr()) if t is not None else None


def _in_flag(t) -> int:
    import torch
    if t.dtype == torch.bfloat16:
        return SAGE_IN_BF16
    if t.dtype == torch.float16:
        return SAGE_IN_FP16
    raise TypeError("inputs must be bf16 or fp16, got %s" % t.dtype)


def _shape(t):
    if t.dim() != 4 or not t.is_contiguous() or not t.is_cuda:
        raise ValueError("expected a contiguous 4-d [B, H, N, D] device tensor")
    return tuple(int(s) for s in t.shape)


def _check_qkv(q, k, v):
    """q, k and v must share shape, 16-bit dtype and device: the kernels read
    all three with q's element type and size."""
    shp = _shape(q)
    _in_flag(q)
    for t, what in ((k, "k"), (v, "v")):
        if _shape(t) != shp or t.dtype != q.dtype or t.device != q.device:
            raise ValueError("%s must match q: shape %s, dtype %s, device %s; got %s, %s, %s"
                             % (what, shp, q.dtype, q.device, tuple(t.shape), t.dtype, t.device))
    return shp


def _check_tensor(t, what: str, shape, dtype, device):
    """A caller-supplied buffer must match what the kernels will write or read
    (the C ABI receives bare pointers and cannot check it)."""
    if not t.is_contiguous() or t.device != device or t.dtype != dtype or tuple(t.shape) != tuple(shape):
        raise ValueError("%s must be a contiguous %s tensor of shape %s on %s, got %s %s on %s"
                         % (what, dtype, tuple(shape), device, t.dtype, tuple(t.shape), t.device))


def _check_workspace(ws, device):
    import torch
    if ws.dtype != torch.uint8 or ws.dim() != 1 or not ws.is_contiguous() or ws.device != device:
        raise ValueError("workspace must be a contiguous 1-d uint8 tensor on %s" % device)


def _check_quantized(pair, what: str, nbytes, device):
    import torch
    for t, n, part in zip(pair[:2], nbytes, ("codes", "scales")):
        if t.dtype != torch.uint8 or not t.is_contiguous() or t.device != device or t.numel() != n:
            raise ValueError("%s %s must be %d contiguous uint8 bytes on %s" % (what, part, n, device))


def quant_sizes(role: int, B: int, H: int, N: int, D: int, fmt: int):
    c, s = ctypes.c_size_t(), ctypes.c_size_t()
    _check("sage_quant_sizes", lib().sage_quant_sizes(role, B, H, N, D, fmt, ctypes.byref(c), ctypes.byref(s)))
    return c.value, s.value


def sage_quant_fp4(x, role: int, fmt: int = SAGE_FMT_MXFP4):
    """Quantize one tensor; returns (codes uint8, scales uint8, mean fp32 or None) on the device:
    role K with smoothing K: the channel mean [B,H,D]; role Q with SAGE_SMOOTH_Q: the query-block
    means [B,H,ceil(N/128),D]."""
    import torch
    B, H, N, D = _shape(x)
    fmt = fmt | _in_flag(x)
    cb, sb = quant_sizes(role, B, H, N, D, fmt)
    codes = torch.empty(cb, dtype=torch.uint8, device=x.device)
    scales = torch.empty(sb, dtype=torch.uint8, device=x.device)
    kmean = None
    ws = None
    if role == SAGE_ROLE_Q and (fmt & SAGE_SMOOTH_Q):
        kmean = torch.empty((B, H, (N + 127) // 128, D), dtype=torch.float32, device=x.device)
    if role == SAGE_ROLE_K and not (fmt & SAGE_NO_SMOOTH_K):
        kmean = torch.empty((B, H, D), dtype=torch.float32, device=x.device)
        wsb = int(lib().sage_quant_workspace_size(role, B, H, N, D, fmt))
        ws = torch.empty(max(wsb, 8), dtype=torch.uint8, device=x.device)
    _check("sage_quant_fp4", lib().sage_quant_fp4(_ptr(x), role, B, H, N, D, fmt, _ptr(codes), _ptr(scales),
                                                  _ptr(kmean), _ptr(ws), ws.numel() if ws is not None else 0,
                                                  _stream()))
    return codes, scales, kmean


def attn_fp4_workspace_size(B: int, H: int, N: int, D: int, fmt: int) -> int:
    return int(lib().sage_attn_fp4_workspace_size(B, H, N, D, fmt))


def _out(q, out_f32: bool):
    import torch
    return torch.empty(q.shape, dtype=torch.float32 if out_f32 else q.dtype, device=q.device)


def _check_o(o, q, out_f32: bool):
    import torch
    _check_tensor(o, "out", q.shape, torch.float32 if out_f32 else q.dtype, q.device)


def sage_attn_fp4_fwd(q, k, v, causal: bool = False, fmt: int = SAGE_FMT_MXFP4, out_f32: bool = True,
                      out=None, workspace=None):
    """O = attention(Q, K, V) through the FP4 path.  With ``workspace`` (a uint8 device
    tensor of at least attn_fp4_workspace_size bytes) no allocation happens inside."""
    B, H, N, D = _check_qkv(q, k, v)
    fmt = fmt | _in_flag(q) | (SAGE_OUT_F32 if out_f32 else 0)
    o = _out(q, out_f32) if out is None else out
    _check_o(o, q, out_f32)
    if workspace is not None:
        _check_workspace(workspace, q.device)
    if workspace is None:
        rc = lib().sage_attn_fp4_fwd(_ptr(q), _ptr(k), _ptr(v), _ptr(o), B, H, N, D, int(bool(causal)), fmt, _stream())
        _check("sage_attn_fp4_fwd", rc)
    else:
        rc = lib().sage_attn_fp4_fwd_ws(_ptr(q), _ptr(k), _ptr(v), _ptr(o), B, H, N, D, int(bool(causal)), fmt,
                                        _ptr(workspace), workspace.numel(), _stream())
        _check("sage_attn_fp4_fwd_ws", rc)
    return o


def sage_attn_fp4_fwd_noalloc(q, k, v, causal: bool = False, fmt: int = SAGE_FMT_MXFP4, out_f32: bool = True,
                              out=None):
    """sage_attn_fp4_fwd on the library's fixed per-GPU scratch (no device allocation
    inside the C call; ``out`` may be preallocated).  Calls that overlap on one GPU race."""
    B, H, N, D = _check_qkv(q, k, v)
    fmt = fmt | _in_flag(q) | (SAGE_OUT_F32 if out_f32 else 0)
    o = _out(q, out_f32) if out is None else out
    _check_o(o, q, out_f32)
    rc = lib().sage_attn_fp4_fwd_noalloc(_ptr(q), _ptr(k), _ptr(v), _ptr(o), B, H, N, D, int(bool(causal)), fmt,
                                         _stream())
    _check("sage_attn_fp4_fwd_noalloc", rc)
    return o


def sage_attn_fp4_fwd_prequant(qq, kq, vq, shape, causal: bool = False, fmt: int = SAGE_FMT_MXFP4,
                               in_bf16: bool = True, out_f32: bool = True, out=None):
    """Attention kernel alone on (codes, scales) pairs from sage_quant_fp4."""
    import torch
    B, H, N, D = shape
    fmt = fmt | (SAGE_IN_BF16 if in_bf16 else SAGE_IN_FP16) | (SAGE_OUT_F32 if out_f32 else 0)
    dev = qq[0].device
    for pair, role, what in ((qq, SAGE_ROLE_Q, "q"), (kq, SAGE_ROLE_K, "k"), (vq, SAGE_ROLE_V, "v")):
        _check_quantized(pair, what, quant_sizes(role, B, H, N, D, fmt), dev)
    odt = torch.float32 if out_f32 else (torch.bfloat16 if in_bf16 else torch.float16)
    if out is None:
        out = torch.empty(shape, dtype=odt, device=dev)
    _check_tensor(out, "out", shape, odt, dev)
    rc = lib().sage_attn_fp4_fwd_prequant(_ptr(qq[0]), _ptr(qq[1]), _ptr(kq[0]), _ptr(kq[1]), _ptr(vq[0]),
                                          _ptr(vq[1]), _ptr(out), B, H, N, D, int(bool(causal)), fmt, _stream())
    _check("sage_attn_fp4_fwd_prequant", rc)
    return out


def sage_attn_bf16_fwd(q, k, v, causal: bool = False, out_f32: bool = True, out=None):
    """bf16-MFMA comparison kernel of the same structure."""
    B, H, N, D = _check_qkv(q, k, v)
    flags = _in_flag(q) | (SAGE_OUT_F32 if out_f32 else 0)
    o = _out(q, out_f32) if out is None else out
    _check_o(o, q, out_f32)
    rc = lib().sage_attn_bf16_fwd(_ptr(q), _ptr(k), _ptr(v), _ptr(o), B, H, N, D, int(bool(causal)), flags, _stream())
    _check("sage_attn_bf16_fwd", rc)
    return o


# ---------------------------------------------------------------- 8-bit attention
def quant_int8_sizes(role: int, B: int, H: int, N: int, D: int, flags: int = 0):
    c, s = ctypes.c_size_t(), ctypes.c_size_t()
    _check("sage_quant_int8_sizes",
           lib().sage_quant_int8_sizes(role, B, H, N, D, flags, ctypes.byref(c), ctypes.byref(s)))
    return c.value, s.value


def sage_quant_int8(x, role: int, flags: int = 0):
    """psi for one role; returns (codes int8, scales fp32, mean fp32 or None) on the device
    (role K with smoothing K: the channel mean [B,H,D])."""
    import torch
    B, H, N, D = _shape(x)
    flags = flags | _in_flag(x)
    cb, sb = quant_int8_sizes(role, B, H, N, D, flags)
    codes = torch.empty(cb, dtype=torch.int8, device=x.device)
    scales = torch.empty(sb // 4, dtype=torch.float32, device=x.device)
    kmean, ws = None, None
    if role == SAGE_ROLE_K and not (flags & SAGE_NO_SMOOTH_K):
        kmean = torch.empty((B, H, D), dtype=torch.float32, device=x.device)
        wsb = int(lib().sage_quant_workspace_size(role, B, H, N, D, 0))
        ws = torch.empty(max(wsb, 8), dtype=torch.uint8, device=x.device)
    _check("sage_quant_int8", lib().sage_quant_int8(_ptr(x), role, B, H, N, D, flags, _ptr(codes), _ptr(scales),
                                                    _ptr(kmean), _ptr(ws), ws.numel() if ws is not None else 0,
                                                    _stream()))
    return codes, scales, kmean


def attn_int8_workspace_size(B: int, H: int, N: int, D: int, flags: int = 0) -> int:
    return int(lib().sage_attn_int8_workspace_size(B, H, N, D, flags))


def sage_attn_int8_fwd(q, k, v, causal: bool = False, flags: int = 0, out_f32: bool = True, lse: bool = True,
                       out=None, lse_out=None, workspace=None):
    """Algorithm 2's 8-bit attention forward.  Returns (O, L) with L = m + log l
    [B,H,N] fp32 (None when ``lse`` is False).  With ``workspace`` (uint8, at
    least attn_int8_workspace_size bytes) no allocation happens inside."""
    import torch
    B, H, N, D = _check_qkv(q, k, v)
    flags = flags | _in_flag(q) | (SAGE_OUT_F32 if out_f32 else 0)
    o = _out(q, out_f32) if out is None else out
    _check_o(o, q, out_f32)
    L = None
    if lse:
        L = torch.empty((B, H, N), dtype=torch.float32, device=q.device) if lse_out is None else lse_out
        _check_tensor(L, "lse_out", (B, H, N), torch.float32, q.device)
    if workspace is not None:
        _check_workspace(workspace, q.device)
    if workspace is None:
        rc = lib().sage_attn_int8_fwd(_ptr(q), _ptr(k), _ptr(v), _ptr(o), _ptr(L), B, H, N, D, int(bool(causal)),
                                      flags, _stream())
        _check("sage_attn_int8_fwd", rc)
    else:
        rc = lib().sage_attn_int8_fwd_ws(_ptr(q), _ptr(k), _ptr(v), _ptr(o), _ptr(L), B, H, N, D, int(bool(causal)),
                                         flags, _ptr(workspace), workspace.numel(), _stream())
        _check("sage_attn_int8_fwd_ws", rc)
    return o, L


def sage_attn_int8_fwd_prequant(qq, kq, vq, shape, causal: bool = False, in_bf16: bool = True,
                                out_f32: bool = True, lse: bool = True, flags: int = 0):
    """The 8-bit attention kernel alone on (codes, scales) pairs from sage_quant_int8
    (flags: SAGE_BKV64 as given to sage_quant_int8)."""
    import torch
    B, H, N, D = shape
    flags = flags | (SAGE_IN_BF16 if in_bf16 else SAGE_IN_FP16) | (SAGE_OUT_F32 if out_f32 else 0)
    dev = qq[0].device
    for pair, role, what in ((qq, SAGE_ROLE_Q, "q"), (kq, SAGE_ROLE_K, "k"), (vq, SAGE_ROLE_V, "v")):
        cb, sb = quant_int8_sizes(role, B, H, N, D, flags & SAGE_BKV64)
        for t, n, part, dt in ((pair[0], cb, "codes", torch.int8), (pair[1], sb // 4, "scales", torch.float32)):
            if t.dtype != dt or not t.is_contiguous() or t.device != dev or t.numel() != n:
                raise ValueError("%s %s must be %d contiguous %s elements on %s" % (what, part, n, dt, dev))
    out = torch.empty(shape, dtype=torch.float32 if out_f32 else (torch.bfloat16 if in_bf16 else torch.float16),
                      device=dev)
    L = torch.empty((B, H, N), dtype=torch.float32, device=dev) if lse else None
    rc = lib().sage_attn_int8_fwd_prequant(_ptr(qq[0]), _ptr(qq[1]), _ptr(kq[0]), _ptr(kq[1]), _ptr(vq[0]),
                                           _ptr(vq[1]), _ptr(out), _ptr(L), B, H, N, D, int(bool(causal)), flags,
                                           _stream())
    _check("sage_attn_int8_fwd_prequant", rc)
    return out, L


def attn_int8_bwd_workspace_size(B: int, H: int, N: int, D: int, flags: int = 0) -> int:
    return int(lib().sage_attn_int8_bwd_workspace_size(B, H, N, D, flags))


def attn_int8_bwd_min_workspace_size(B: int, H: int, N: int, D: int, flags: int = 0) -> int:
    return int(lib().sage_attn_int8_bwd_min_workspace_size(B, H, N, D, flags))


def sage_attn_int8_bwd(q, k, v, o, lse, dout, causal: bool = False, flags: int = 0, workspace=None, out=None):
    """Algorithm 3's 8-bit attention backward: returns (dQ, dK, dV) fp32 [B,H,N,D].
    o, lse: the forward's fp32 output and L.  ``out``: three preallocated fp32
    tensors; with ``workspace`` nothing is allocated inside."""
    import torch
    B, H, N, D = _shape(q)
    for t in (k, v, dout):
        if _shape(t) != (B, H, N, D) or t.dtype != q.dtype:
            raise ValueError("q, k, v, dout must have the same shape and dtype")
    if _shape(o) != (B, H, N, D) or o.dtype != torch.float32:
        raise ValueError("o must be the fp32 forward output")
    if tuple(lse.shape) != (B, H, N) or lse.dtype != torch.float32 or not lse.is_contiguous():
        raise ValueError("lse must be fp32 [B,H,N]")
    for t, what in ((k, "k"), (v, "v"), (dout, "dout"), (o, "o"), (lse, "lse")):
        if t.device != q.device:
            raise ValueError("%s must be on %s" % (what, q.device))
    flags = flags | _in_flag(q)
    dq, dk, dv = out if out is not None else [torch.empty((B, H, N, D), dtype=torch.float32, device=q.device)
                                              for _ in range(3)]
    for t, what in ((dq, "dq"), (dk, "dk"), (dv, "dv")):
        _check_tensor(t, what, (B, H, N, D), torch.float32, q.device)
    if workspace is not None:
        _check_workspace(workspace, q.device)
    ptrs = [_ptr(t) for t in (q, k, v, o, lse, dout, dq, dk, dv)]
    if workspace is None:
        _check("sage_attn_int8_bwd", lib().sage_attn_int8_bwd(*ptrs, B, H, N, D, int(bool(causal)), flags, _stream()))
    else:
        _check("sage_attn_int8_bwd_ws", lib().sage_attn_int8_bwd_ws(*ptrs, B, H, N, D, int(bool(causal)), flags,
                                                                  _ptr(workspace), workspace.numel(), _stream()))
    return dq, dk, dv


def version() -> str:
    return lib().sage_version().decode()
