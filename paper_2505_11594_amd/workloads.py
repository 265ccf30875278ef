"""Seeded synthetic workloads (inputs only; no attention or quantization arithmetic).

The paper measures kernel speed on sweeps and accuracy on real CogVideoX
Q, K, V (Sec. 4, Table 1), none of which is available here.  These seeded
generators stand in for them: i.i.d. normal Q, K, V with the shapes of the
five benchmark configurations, plus the structures the paper's method is
designed for -- a per-channel bias on K shared by all tokens (what smoothing
K removes, Algorithm 1 preprocessing) and rare large-magnitude rows (what
per-block microscaling contains, Sec. 1).

Recipe (every configuration):
  * numpy ``default_rng(1000 + index)``; Q, K, V drawn in that order as
    float32 standard normals of shape [B, H, N, D];
  * optional K channel bias: one D-vector per (b, h), drawn next, with the
    stated variance (N(0, 4) means standard deviation 2), added to every token;
  * optional outliers: round(frac * N) rows per (b, h), chosen without
    replacement, first for Q then for K, multiplied by ``outlier_scale``;
  * cast once to the 16-bit input type with round-to-nearest-even; the raw
    16-bit patterns are what both the GPU path and the oracle consume.
"""
from __future__ import annotations

from dataclasses import dataclass, field
import numpy as np

IN_FP16, IN_BF16 = 0, 1
FMT_MX, FMT_NV16 = 0, 1


@dataclass(frozen=True)
class Workload:
    name: str
    B: int
    H: int
    N: int
    D: int
    causal: bool
    in_dtype: int
    fmts: tuple = (FMT_MX,)
    bkv: int = 128
    k_bias_var: float = 0.0
    outlier_frac: float = 0.0
    outlier_scale: float = 20.0
    seed: int = 1000

    @property
    def ops(self) -> float:
        """Attention operations 4 B H N^2 D, halved when causal."""
        o = 4.0 * self.B * self.H * self.N * self.N * self.D
        return o / 2 if self.causal else o


# The five benchmark configurations, in order.
CONFIGS = [
    Workload("b1h1n128d64_fp16", 1, 1, 128, 64, False, IN_FP16, (FMT_MX,), bkv=64, seed=1000),
    Workload("b4h32n4096d128_kbias4", 4, 32, 4096, 128, False, IN_BF16, (FMT_MX,), bkv=256, k_bias_var=4.0,
             seed=1001),
    Workload("b1h32n32768d128_outliers", 1, 32, 32768, 128, False, IN_BF16, (FMT_MX,), bkv=256,
             outlier_frac=0.01, outlier_scale=20.0, seed=1002),
    Workload("b8h32n8192d128_causal_kbias1", 8, 32, 8192, 128, True, IN_BF16, (FMT_MX,), bkv=256, k_bias_var=1.0,
             seed=1003),
    Workload("b1h24n76800d64_kbias4", 1, 24, 76800, 64, False, IN_BF16, (FMT_NV16, FMT_MX), k_bias_var=4.0, seed=1004),
]


def to_bits(x: np.ndarray, in_dtype: int) -> np.ndarray:
    """Round float32 to fp16/bf16 (nearest-even) and return the uint16 bit patterns."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    if in_dtype == IN_FP16:
        return x.astype(np.float16).view(np.uint16)
    u = x.view(np.uint32).astype(np.uint64)
    # round to nearest even on the upper 16 bits (inputs are finite)
    r = ((u + 0x7FFF + ((u >> 16) & 1)) >> 16).astype(np.uint16)
    return r


def from_bits(b: np.ndarray, in_dtype: int) -> np.ndarray:
    """Widen uint16 fp16/bf16 bit patterns to float32 (exact)."""
    b = np.ascontiguousarray(b, dtype=np.uint16)
    if in_dtype == IN_FP16:
        return b.view(np.float16).astype(np.float32)
    return (b.astype(np.uint32) << 16).view(np.float32)


def generate(w: Workload, B: int | None = None, H: int | None = None, N: int | None = None):
    """Draw (q, k, v) uint16 bit arrays [B, H, N, D] for a workload (optionally resized)."""
    B = w.B if B is None else B
    H = w.H if H is None else H
    N = w.N if N is None else N
    return make_inputs(B, H, N, w.D, w.in_dtype, w.seed, k_bias_var=w.k_bias_var,
                       outlier_frac=w.outlier_frac, outlier_scale=w.outlier_scale)


def make_inputs(B, H, N, D, in_dtype, seed, k_bias_var=0.0, outlier_frac=0.0, outlier_scale=20.0):
    rng = np.random.default_rng(seed)
    shape = (B, H, N, D)
    q = rng.standard_normal(shape, dtype=np.float32)
    k = rng.standard_normal(shape, dtype=np.float32)
    v = rng.standard_normal(shape, dtype=np.float32)
    if k_bias_var > 0:
        bias = rng.standard_normal((B, H, 1, D), dtype=np.float32) * np.float32(np.sqrt(k_bias_var))
        k += bias
    if outlier_frac > 0:
        n_out = int(round(outlier_frac * N))
        for x in (q, k):
            for b in range(B):
                for h in range(H):
                    idx = rng.choice(N, size=n_out, replace=False)
                    x[b, h, idx, :] *= np.float32(outlier_scale)
    return to_bits(q, in_dtype), to_bits(k, in_dtype), to_bits(v, in_dtype)


def sample_rows(w: Workload, per_head_tiles: int = 8, tile: int = 64, rows_per_tile: int = 64,
                B: int | None = None, H: int | None = None, N: int | None = None, seed: int = 7,
                heads=None):
    """Flat row ids ((b*H + h)*N + i) of a seeded sample of query tiles per head:
    always the first and last tile, plus (causal) the tile that ends on a KV-tile
    boundary, then random tiles; ``rows_per_tile`` rows of each (all if >= tile).
    ``heads``: the flat (b*H + h) heads to sample (default: all)."""
    B = w.B if B is None else B
    H = w.H if H is None else H
    N = w.N if N is None else N
    rng = np.random.default_rng(seed)
    ntile = (N + tile - 1) // tile
    rows = []
    for bh in (range(B * H) if heads is None else heads):
        pick = {0, ntile - 1}
        if w.causal:
            pick.add(min(ntile - 1, (w.bkv // tile)))
        while len(pick) < min(per_head_tiles, ntile):
            pick.add(int(rng.integers(0, ntile)))
        for t in sorted(pick):
            lo, hi = t * tile, min(N, (t + 1) * tile)
            idx = np.arange(lo, hi)
            if rows_per_tile < idx.size:
                idx = np.sort(rng.choice(idx, size=rows_per_tile, replace=False))
            rows.extend((bh * N + idx).tolist())
    return np.asarray(rows, dtype=np.int64)
