"""Host-side readers of the library's physical quantized layouts (test code).

The library stores FP4 codes two per byte (element 2i in the low nibble), K^
with its tokens permuted inside each 64-token group and V^ transposed, with
token counts padded to 128 (include/sage_mi355x.h).  These helpers turn the
device buffers back into the oracle's logical layout: one code per byte,
natural token order.
"""
import numpy as np


def pad128(n):
    return (n + 127) // 128 * 128


def unpack_nibbles(b):
    b = np.asarray(b, dtype=np.uint8)
    out = np.empty(b.shape[:-1] + (b.shape[-1] * 2,), dtype=np.uint8)
    out[..., 0::2] = b & 0xF
    out[..., 1::2] = b >> 4
    return out


def k_stored_position(t, fmt=0):
    """Stored row of token t: MXFP4 permutes inside 64-token groups
    (o = 32h + 16t' + 4g + r -> 32t' + 8g + 4h + r), NV16 inside 32-token groups
    (o = 16h + 4g + r -> 8g + 4h + r)."""
    t = np.asarray(t)
    if fmt == 0:
        o = t & 63
        h, tt, g, r = o >> 5, (o >> 4) & 1, (o >> 2) & 3, o & 3
        return (t & ~63) | (tt << 5) | (g << 3) | (h << 2) | r
    o = t & 31
    h, g, r = o >> 4, (o >> 2) & 3, o & 3
    return (t & ~31) | (g << 3) | (h << 2) | r


def block_size(fmt):
    return 32 if fmt == 0 else 16


def q_logical(codes, scales, B, H, N, D, fmt):
    n = block_size(fmt)
    c = unpack_nibbles(np.asarray(codes).reshape(B, H, N, D // 2))
    s = np.asarray(scales).reshape(B, H, N, D // n)
    return c, s


def k_logical(codes, scales, B, H, N, D, fmt):
    """Returns (codes [B,H,N,D], scales [B,H,N,D/n], tail_codes, tail_scales)."""
    n = block_size(fmt)
    Np = pad128(N)
    c = unpack_nibbles(np.asarray(codes).reshape(B, H, Np, D // 2))
    s = np.asarray(scales).reshape(B, H, Np, D // n)
    pos = k_stored_position(np.arange(Np), fmt)
    return c[:, :, pos[:N]], s[:, :, pos[:N]], c[:, :, pos[N:]], s[:, :, pos[N:]]


def v_logical(codes, scales, B, H, N, D, fmt):
    """Returns (codes [B,H,D,Nn], scales [B,H,D,Nn/n], tail codes, tail scales) with Nn = N rounded up to n."""
    n = block_size(fmt)
    Np = pad128(N)
    Nn = (N + n - 1) // n * n
    c = unpack_nibbles(np.asarray(codes).reshape(B, H, D, Np // 2))
    s = np.asarray(scales).reshape(B, H, D, Np // n)
    return c[..., :Nn], s[..., :Nn // n], c[..., Nn:], s[..., Nn // n:]
