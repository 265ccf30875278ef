"""CPU oracle for microscaled-FP4 attention (SageAttention3 forward, arXiv 2505.11594).

TEST INFRASTRUCTURE ONLY: the test suite, the package's smoke check and the
benchmark's CPU-baseline leg are the only callers.  The product path (the HIP
library and its Python binding) never imports this module.

The arithmetic lives in ``sage_oracle.c`` (plain C, compiled with
``-ffp-contract=off``, no fast-math); this file only builds it and marshals
numpy arrays.  Every function cites the passage of the paper it follows in
the C source.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "sage_oracle.c")
_SRC_I8 = os.path.join(_HERE, "sage_oracle_int8.c")
_LIB = os.path.join(_HERE, "liboracle.so")

FMT_MX, FMT_NV16, FMT_NONE = 0, 1, 2
IN_FP16, IN_BF16 = 0, 1
ROLE_Q, ROLE_K, ROLE_V = 0, 1, 2
NO_SMOOTH_K, DIRECT_P, R_LITERAL, SMOOTH_Q, OCP_SCALE = 1, 2, 4, 8, 16
# the P step in the fused order a GPU evaluates it (orc_p_tile; for the test that bounds its differences)
FUSED_P = 256
# 8-bit attention (Algorithm 2) flags: NO_SMOOTH_K, and
I8_STATIC_P, I8_IDENTITY, I8_DP_INT8 = 32, 64, 128
# P^ of Algorithm 2 in the fused order a GPU evaluates it (for the test that bounds its differences)
I8_FUSED_P = 512
# P of Algorithm 3 in the fused order (for the test that bounds its differences)
I8_FUSED_BWD = 1024

_lib = None


def build(force: bool = False) -> str:
    """Compile sage_oracle.c into liboracle.so (gcc, no fast-math, no FP contraction)."""
    newest = max(os.path.getmtime(_SRC), os.path.getmtime(_SRC_I8))
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < newest:
        tmp = _LIB + ".tmp%d" % os.getpid()
        cmd = ["gcc", "-O2", "-fPIC", "-shared", "-ffp-contract=off", "-fno-fast-math",
               "-pthread", "-o", tmp, _SRC, _SRC_I8, "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(tmp, _LIB)
    return _LIB


def lib():
    global _lib
    if _lib is None:
        build()
        L = ctypes.CDLL(_LIB)
        u8p = ctypes.POINTER(ctypes.c_uint8)
        L.orc_e2m1_encode.restype = ctypes.c_uint8
        L.orc_e2m1_encode.argtypes = [ctypes.c_float]
        L.orc_e2m1_decode.restype = ctypes.c_float
        L.orc_e2m1_decode.argtypes = [ctypes.c_uint8]
        L.orc_e4m3_encode.restype = ctypes.c_uint8
        L.orc_e4m3_encode.argtypes = [ctypes.c_float]
        L.orc_e4m3_decode.restype = ctypes.c_float
        L.orc_e4m3_decode.argtypes = [ctypes.c_uint8]
        L.orc_e8m0_exponent.restype = ctypes.c_int
        L.orc_e8m0_exponent.argtypes = [ctypes.c_float]
        L.orc_e8m0_exponent_floor.restype = ctypes.c_int
        L.orc_e8m0_exponent_floor.argtypes = [ctypes.c_float]
        L.orc_e8m0_decode.restype = ctypes.c_float
        L.orc_e8m0_decode.argtypes = [ctypes.c_uint8]
        L.orc_widen.restype = ctypes.c_float
        L.orc_widen.argtypes = [ctypes.c_uint16, ctypes.c_int]
        L.orc_phi_block.restype = ctypes.c_uint8
        L.orc_phi_block.argtypes = [ctypes.c_void_p, ctypes.c_int, ctypes.c_int, ctypes.c_void_p]
        L.orc_phi_block_ex.restype = ctypes.c_uint8
        L.orc_phi_block_ex.argtypes = [ctypes.c_void_p, ctypes.c_int, ctypes.c_int, ctypes.c_uint, ctypes.c_void_p]
        L.orc_kmean.restype = ctypes.c_long
        L.orc_kmean.argtypes = [ctypes.c_void_p, ctypes.c_int] + [ctypes.c_int] * 4 + [ctypes.c_void_p]
        L.orc_quant.restype = ctypes.c_long
        L.orc_quant.argtypes = ([ctypes.c_void_p, ctypes.c_int, ctypes.c_int] + [ctypes.c_int] * 4 +
                                [ctypes.c_int, ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p])
        L.orc_attn2.restype = ctypes.c_int
        L.orc_attn2.argtypes = ([ctypes.c_void_p] * 3 + [ctypes.c_int] * 9 + [ctypes.c_uint] +
                                [ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p, ctypes.c_void_p,
                                 ctypes.c_void_p, ctypes.c_int])
        L.orc_quant_smooth_q.restype = None
        L.orc_quant_smooth_q.argtypes = ([ctypes.c_void_p, ctypes.c_int] + [ctypes.c_int] * 6 +
                                         [ctypes.c_void_p] * 3)
        L.orc_attn.restype = ctypes.c_int
        L.orc_attn.argtypes = ([ctypes.c_void_p] * 3 + [ctypes.c_int] * 8 + [ctypes.c_uint] +
                               [ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p, ctypes.c_void_p,
                                ctypes.c_void_p, ctypes.c_int])
        L.orc_exact_attn.restype = ctypes.c_int
        L.orc_exact_attn.argtypes = ([ctypes.c_void_p] * 3 + [ctypes.c_int] * 6 +
                                     [ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p, ctypes.c_int])
        L.orc_p_tile.restype = ctypes.c_int
        L.orc_p_tile.argtypes = ([ctypes.c_void_p, ctypes.c_int, ctypes.c_float, ctypes.c_int, ctypes.c_int,
                                  ctypes.c_uint] + [ctypes.c_void_p] * 12)
        L.orc_fp4mm.restype = ctypes.c_long
        L.orc_fp4mm.argtypes = [ctypes.c_void_p] * 4 + [ctypes.c_int] * 4 + [ctypes.c_void_p]
        L.orc_psi_block.restype = ctypes.c_float
        L.orc_psi_block.argtypes = [ctypes.c_void_p, ctypes.c_long, ctypes.c_void_p]
        L.orc_quant_int8.restype = ctypes.c_long
        L.orc_quant_int8.argtypes = ([ctypes.c_void_p, ctypes.c_int, ctypes.c_int] + [ctypes.c_int] * 6 +
                                     [ctypes.c_void_p] * 3)
        L.orc_attn_int8.restype = ctypes.c_int
        L.orc_attn_int8.argtypes = ([ctypes.c_void_p] * 3 + [ctypes.c_int] * 8 + [ctypes.c_uint] +
                                    [ctypes.c_void_p, ctypes.c_int64] + [ctypes.c_void_p] * 4 + [ctypes.c_int])
        L.orc_attn_int8_bwd.restype = ctypes.c_int
        L.orc_attn_int8_bwd.argtypes = ([ctypes.c_void_p] * 6 + [ctypes.c_int] * 8 + [ctypes.c_uint] +
                                        [ctypes.c_void_p] * 6 + [ctypes.c_int])
        _lib = L
    return _lib


def _ptr(a: np.ndarray):
    assert a.flags["C_CONTIGUOUS"]
    return a.ctypes.data_as(ctypes.c_void_p)


def default_threads() -> int:
    try:
        return max(1, len(os.sched_getaffinity(0)))
    except AttributeError:  # pragma: no cover
        return os.cpu_count() or 1


def block_size(fmt: int) -> int:
    return 32 if fmt == FMT_MX else 16


# ---------------------------------------------------------------- codecs
def e2m1_encode(y: float) -> int:
    return int(lib().orc_e2m1_encode(float(y)))


def e2m1_decode(c: int) -> float:
    return float(lib().orc_e2m1_decode(int(c)))


def e4m3_encode(s: float) -> int:
    return int(lib().orc_e4m3_encode(float(s)))


def e4m3_decode(b: int) -> float:
    return float(lib().orc_e4m3_decode(int(b)))


def e8m0_exponent(amax: float) -> int:
    return int(lib().orc_e8m0_exponent(float(amax)))


def e8m0_exponent_floor(amax: float) -> int:
    """The alternative E8M0 rule of the OCP_SCALE ablation: floor(log2 amax) - 2."""
    return int(lib().orc_e8m0_exponent_floor(float(amax)))


def e8m0_decode(b: int) -> float:
    return float(lib().orc_e8m0_decode(int(b)))


def widen(bits: int, in_dtype: int) -> float:
    return float(lib().orc_widen(int(bits), int(in_dtype)))


def phi_block(x: np.ndarray, fmt: int, flags: int = 0):
    """phi on one block: returns (codes uint8[n], scale byte).  flags may hold
    OCP_SCALE (the floor rule for E8M0 scales)."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    codes = np.zeros(x.size, dtype=np.uint8)
    sb = lib().orc_phi_block_ex(_ptr(x), x.size, fmt, flags, _ptr(codes))
    return codes, int(sb)


def dequant_block(codes: np.ndarray, sb: int, fmt: int) -> np.ndarray:
    s = e8m0_decode(sb) if fmt == FMT_MX else e4m3_decode(sb)
    return np.array([e2m1_decode(c) for c in codes], dtype=np.float64) * s


# ---------------------------------------------------------------- tensors
def kmean(k_bits: np.ndarray, in_dtype: int):
    """mu [B,H,D] fp32 and the count of inexact fp64 column sums."""
    B, H, N, D = k_bits.shape
    k_bits = np.ascontiguousarray(k_bits, dtype=np.uint16)
    mu = np.zeros((B, H, D), dtype=np.float32)
    inexact = lib().orc_kmean(_ptr(k_bits), in_dtype, B, H, N, D, _ptr(mu))
    return mu, int(inexact)


def quant_smooth_q(q_bits: np.ndarray, in_dtype: int, fmt: int, bq: int = 128):
    """phi(Q_i - mean(Q_i)) over query blocks of bq rows (smoothing Q, Algorithm 1).
    Returns (codes [B,H,N,D] one per byte, scales [B,H,N,D/n], qbar fp32 [B,H,ceil(N/bq),D])."""
    B, H, N, D = q_bits.shape
    q_bits = np.ascontiguousarray(q_bits, dtype=np.uint16)
    n = 32 if fmt == FMT_MX else 16
    codes = np.zeros((B, H, N, D), dtype=np.uint8)
    scales = np.zeros((B, H, N, D // n), dtype=np.uint8)
    qbar = np.zeros((B, H, (N + bq - 1) // bq, D), dtype=np.float32)
    lib().orc_quant_smooth_q(_ptr(q_bits), in_dtype, B, H, N, D, bq, fmt, _ptr(codes), _ptr(scales), _ptr(qbar))
    return codes, scales, qbar


def quant(x_bits: np.ndarray, in_dtype: int, role: int, fmt: int, smooth_k: bool = True):
    """Logical-layout quantization (one code per byte); see orc_quant in the C source.

    Returns (codes, scales, mu or None, inexact_kmean_columns)."""
    B, H, N, D = x_bits.shape
    n = block_size(fmt)
    x_bits = np.ascontiguousarray(x_bits, dtype=np.uint16)
    if role == ROLE_V:
        Np = (N + n - 1) // n * n
        codes = np.zeros((B, H, D, Np), dtype=np.uint8)
        scales = np.zeros((B, H, D, Np // n), dtype=np.uint8)
    else:
        codes = np.zeros((B, H, N, D), dtype=np.uint8)
        scales = np.zeros((B, H, N, D // n), dtype=np.uint8)
    mu = np.zeros((B, H, D), dtype=np.float32) if role == ROLE_K else None
    inexact = lib().orc_quant(_ptr(x_bits), in_dtype, role, B, H, N, D, fmt, int(bool(smooth_k)),
                              _ptr(codes), _ptr(scales), _ptr(mu) if mu is not None else None)
    return codes, scales, mu, int(inexact)


def attn(q_bits, k_bits, v_bits, in_dtype: int, causal: bool, fmt: int, bkv: int,
         rows=None, flags: int = 0, nthreads: int | None = None, bq: int = 128):
    """Algorithm 1 on the listed rows (smoothing Q when flags has SMOOTH_Q,
    with query blocks of bq rows).

    rows: flat ids ((b*H + h)*N + i); None = every row.
    Returns (out [nrows, D] fp32, tie_tol [nrows] fp32, counters dict)."""
    B, H, N, D = q_bits.shape
    q_bits = np.ascontiguousarray(q_bits, dtype=np.uint16)
    k_bits = np.ascontiguousarray(k_bits, dtype=np.uint16)
    v_bits = np.ascontiguousarray(v_bits, dtype=np.uint16)
    if rows is None:
        rows = np.arange(B * H * N, dtype=np.int64)
    rows = np.ascontiguousarray(rows, dtype=np.int64)
    out = np.zeros((rows.size, D), dtype=np.float32)
    tol = np.zeros(rows.size, dtype=np.float32)
    cnt = np.zeros(5, dtype=np.int64)
    rc = lib().orc_attn2(_ptr(q_bits), _ptr(k_bits), _ptr(v_bits), in_dtype, B, H, N, D, int(bool(causal)),
                         fmt, bkv, bq, flags, _ptr(rows), rows.size, _ptr(out), _ptr(tol), _ptr(cnt),
                         nthreads or default_threads())
    if rc != 0:
        raise ValueError("orc_attn2: invalid arguments")
    counters = dict(inexact_s=int(cnt[0]), inexact_o=int(cnt[1]), tie_codes=int(cnt[2]), skipped_tiles=int(cnt[3]),
                    alt_scales=int(cnt[4]))
    return out, tol, counters


def exact_attn(q_bits, k_bits, v_bits, in_dtype: int, causal: bool, rows=None, nthreads: int | None = None):
    """fp64 softmax(Q K^T / sqrt(D)) V on the unquantized inputs for the listed rows."""
    B, H, N, D = q_bits.shape
    q_bits = np.ascontiguousarray(q_bits, dtype=np.uint16)
    k_bits = np.ascontiguousarray(k_bits, dtype=np.uint16)
    v_bits = np.ascontiguousarray(v_bits, dtype=np.uint16)
    if rows is None:
        rows = np.arange(B * H * N, dtype=np.int64)
    rows = np.ascontiguousarray(rows, dtype=np.int64)
    out = np.zeros((rows.size, D), dtype=np.float64)
    rc = lib().orc_exact_attn(_ptr(q_bits), _ptr(k_bits), _ptr(v_bits), in_dtype, B, H, N, D, int(bool(causal)),
                              _ptr(rows), rows.size, _ptr(out), nthreads or default_threads())
    if rc != 0:
        raise ValueError("orc_exact_attn: invalid arguments")
    return out


def p_tile(S, m_old: float, D: int, fmt: int, flags: int = 0):
    """One tile of the online softmax and the two-level quantization of P~,
    in Algorithm 1's order (FUSED_P: the fused order).

    Returns dict(m_new, alpha, s1, rowsum, p2, codes, sbytes, lo, hi, sb_lo, sb_hi, cont):
    lo/hi bound every accepted P~2 value per key, sb_lo/sb_hi every accepted
    block scale byte, cont = sum(hi - lo)."""
    S = np.ascontiguousarray(S, dtype=np.float32)
    bkv = S.size
    n = 1 if fmt == FMT_NONE else block_size(fmt)
    outs = [np.zeros(1, dtype=np.float32) for _ in range(4)]
    p2 = np.zeros(bkv, dtype=np.float32)
    codes = np.zeros(bkv, dtype=np.uint8)
    sbytes = np.zeros(max(bkv // n, 1), dtype=np.uint8)
    lo = np.zeros(bkv, dtype=np.float64)
    hi = np.zeros(bkv, dtype=np.float64)
    sb_lo = np.zeros(max(bkv // n, 1), dtype=np.uint8)
    sb_hi = np.zeros(max(bkv // n, 1), dtype=np.uint8)
    cont = np.zeros(1, dtype=np.float64)
    rc = lib().orc_p_tile(_ptr(S), bkv, float(m_old), D, fmt, flags, *[_ptr(o) for o in outs],
                          _ptr(p2), _ptr(codes), _ptr(sbytes), _ptr(lo), _ptr(hi), _ptr(sb_lo), _ptr(sb_hi),
                          _ptr(cont))
    if rc != 0:
        raise ValueError("orc_p_tile: fully masked tile")
    return dict(m_new=float(outs[0][0]), alpha=float(outs[1][0]), s1=float(outs[2][0]), rowsum=float(outs[3][0]),
                p2=p2, codes=codes, sbytes=sbytes, lo=lo, hi=hi, sb_lo=sb_lo, sb_hi=sb_hi, cont=float(cont[0]))


def fp4mm(ac, as_, bc, bs, fmt: int):
    """C = FP4MM(A^, s_A, B^, s_B) with A [M,K], B [N,K] codes (one per byte) and scale bytes."""
    M, K = ac.shape
    Nn = bc.shape[0]
    C = np.zeros((M, Nn), dtype=np.float32)
    arrs = [np.ascontiguousarray(a, dtype=np.uint8) for a in (ac, as_, bc, bs)]
    inexact = lib().orc_fp4mm(*[_ptr(a) for a in arrs], M, Nn, K, fmt, _ptr(C))
    return C, int(inexact)


def metrics(o_ref: np.ndarray, o: np.ndarray) -> dict:
    """CosSim, relative L1 and RMSE over the flattened outputs (Appendix, accuracy metrics), fp64."""
    a = np.asarray(o_ref, dtype=np.float64).ravel()
    b = np.asarray(o, dtype=np.float64).ravel()
    cos = float((a * b).sum() / (np.sqrt((a * a).sum()) * np.sqrt((b * b).sum())))
    l1 = float(np.abs(a - b).sum() / np.abs(a).sum())
    rmse = float(np.sqrt(((a - b) ** 2).mean()))
    return dict(cossim=cos, l1=l1, rmse=rmse)


# ---------------------------------------------------------------- Algorithm 2
def psi_block(x: np.ndarray):
    """Per-block INT8 quantization psi (Eq. psi): returns (codes int8[n], scale)."""
    x = np.ascontiguousarray(x, dtype=np.float32).ravel()
    codes = np.zeros(x.size, dtype=np.int8)
    s = lib().orc_psi_block(_ptr(x), x.size, _ptr(codes))
    return codes, float(np.float32(s))


def quant_int8(x_bits: np.ndarray, in_dtype: int, role: int, blk: int, smooth_k: bool = True):
    """psi over blocks of blk rows (role K: of K - mean(K) unless smooth_k is
    False).  Returns (codes int8 [B,H,N,D], scales fp32 [B,H,ceil(N/blk)],
    mu fp32 [B,H,D] or None)."""
    B, H, N, D = x_bits.shape
    x_bits = np.ascontiguousarray(x_bits, dtype=np.uint16)
    codes = np.zeros((B, H, N, D), dtype=np.int8)
    scales = np.zeros((B, H, (N + blk - 1) // blk), dtype=np.float32)
    mu = np.zeros((B, H, D), dtype=np.float32)
    sm = role == ROLE_K and smooth_k
    lib().orc_quant_int8(_ptr(x_bits), in_dtype, role, B, H, N, D, blk, int(sm), _ptr(codes), _ptr(scales),
                         _ptr(mu))
    return codes, scales, (mu if sm else None)


def attn_int8(q_bits, k_bits, v_bits, in_dtype: int, causal: bool, bkv: int, rows=None, flags: int = 0,
              bq: int = 128, nthreads: int | None = None):
    """Algorithm 2 (the 8-bit attention forward) on the listed rows.

    Returns (out [nrows, D] fp32, lse [nrows] fp32, tie_tol [nrows] fp32, counters dict)."""
    B, H, N, D = q_bits.shape
    arrs = [np.ascontiguousarray(a, dtype=np.uint16) for a in (q_bits, k_bits, v_bits)]
    if rows is None:
        rows = np.arange(B * H * N, dtype=np.int64)
    rows = np.ascontiguousarray(rows, dtype=np.int64)
    out = np.zeros((rows.size, D), dtype=np.float32)
    lse = np.zeros(rows.size, dtype=np.float32)
    tol = np.zeros(rows.size, dtype=np.float32)
    cnt = np.zeros(2, dtype=np.int64)
    rc = lib().orc_attn_int8(*[_ptr(a) for a in arrs], in_dtype, B, H, N, D, int(bool(causal)), bq, bkv, flags,
                             _ptr(rows), rows.size, _ptr(out), _ptr(lse), _ptr(tol), _ptr(cnt),
                             nthreads or default_threads())
    if rc != 0:
        raise ValueError("orc_attn_int8: invalid arguments")
    return out, lse, tol, dict(tie_codes=int(cnt[0]), skipped_tiles=int(cnt[1]))


def attn_int8_bwd(q_bits, k_bits, v_bits, do_bits, o, lse, in_dtype: int, causal: bool, bkv: int, flags: int = 0,
                  bq: int = 128, tolerance: bool = True, nthreads: int | None = None):
    """Algorithm 3 (the 8-bit attention backward) for every head.  o: the forward's
    output fp32 [B,H,N,D]; lse: its L fp32 [B,H,N].  Returns (dq, dk, dv) fp32
    [B,H,N,D] and, with tolerance, the per-element tolerances (tq, tk, tv)."""
    B, H, N, D = q_bits.shape
    arrs = [np.ascontiguousarray(a, dtype=np.uint16) for a in (q_bits, k_bits, v_bits, do_bits)]
    o = np.ascontiguousarray(o, dtype=np.float32).reshape(B, H, N, D)
    lse = np.ascontiguousarray(lse, dtype=np.float32).reshape(B, H, N)
    outs = [np.zeros((B, H, N, D), dtype=np.float32) for _ in range(6 if tolerance else 3)]
    tp = [_ptr(x) for x in outs[3:]] if tolerance else [None] * 3
    rc = lib().orc_attn_int8_bwd(*[_ptr(a) for a in arrs], _ptr(o), _ptr(lse), in_dtype, B, H, N, D,
                                 int(bool(causal)), bq, bkv, flags, *[_ptr(x) for x in outs[:3]], *tp,
                                 nthreads or default_threads())
    if rc != 0:
        raise ValueError("orc_attn_int8_bwd: invalid arguments")
    return tuple(outs[:3]) + ((tuple(outs[3:]),) if tolerance else ())
