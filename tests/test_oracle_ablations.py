"""Pins for the oracle's accuracy ablations (no GPU).

- C3, the E8M0 scale rule: the default is the smallest power of two 2^e with
  6 2^e >= amax (nothing clips).  The alternative, flag OCP_SCALE, is the
  floor rule 2^(floor(log2 amax) - 2), which clips block values in (6, 8) 2^e
  to 6.  Pinned against floor(log2) in fp64 and a brute-force nearest-value
  search over the E2M1 grid, and end to end: the two rules give bit-identical
  attention when every block maximum is 4 2^k and differ otherwise.
- C9, the first-level constant with E8M0 scales: R = 6 against the literal
  448*6 of the E4M3 analysis (Sec. 3.2).
- Fig. 3 (d, e): the error of the P scales and of P~ itself, direct against
  two-level quantization of P~ (Sec. 3.2), with NVFP4-style E4M3 scales.
"""
import math

import numpy as np
import pytest

import oracle
from paper_2505_11594_amd import workloads as wl

GRID = np.array([0.0, 0.5, 1.0, 1.5, 2.0, 3.0, 4.0, 6.0])


def amax_samples(rng):
    e = rng.integers(-120, 120, 400)
    m = rng.uniform(0.5, 1.0, 400)
    vals = list(np.ldexp(m, e))
    for k in range(-20, 21):
        for base in (4.0, 6.0, 8.0, 3.0, 7.0):
            vals.append(math.ldexp(base, k))
        vals.append(math.ldexp(6.0, k) * (1 + 2.0 ** -23))   # one ulp above 6 2^k
        vals.append(math.ldexp(8.0, k) * (1 - 2.0 ** -24))   # one ulp below 8 2^k
    return np.array(vals, dtype=np.float32)


def test_ocp_exponent_is_floor_log2_minus_2():
    rng = np.random.default_rng(80)
    for a in amax_samples(rng):
        ef = oracle.e8m0_exponent_floor(float(a))
        assert ef == math.floor(math.log2(float(a))) - 2
        # the default (ceil) rule is the floor rule, raised by one exactly when
        # the block max would exceed the largest FP4 value at the floor scale
        ed = oracle.e8m0_exponent(float(a))
        assert ed == (ef if float(a) <= math.ldexp(6.0, ef) else ef + 1)
    assert oracle.e8m0_exponent_floor(0.0) == -127


def brute_e2m1(y: float) -> int:
    """Nearest E2M1 value to |y| with saturation at 6, ties to the even code;
    the sign bit follows y."""
    a = min(abs(y), 6.0)
    d = np.abs(GRID - a)
    best = np.flatnonzero(d == d.min())
    code = int(best[0]) if best.size == 1 else int(best[best % 2 == 0][0])
    return code | (8 if math.copysign(1.0, y) < 0 else 0)


def test_ocp_block_codes_brute_force():
    rng = np.random.default_rng(81)
    clipped = 0
    for trial in range(300):
        x = (rng.standard_normal(32) * 2.0 ** rng.integers(-10, 10)).astype(np.float32)
        if trial % 3 == 0:
            x[rng.integers(0, 32)] *= np.float32(rng.uniform(1.0, 8.0))
        codes, sb = oracle.phi_block(x, oracle.FMT_MX, oracle.OCP_SCALE)
        amax = float(np.abs(x).max())
        e = math.floor(math.log2(amax)) - 2
        assert sb == e + 127
        for xi, c in zip(x, codes):
            y = math.ldexp(float(xi), -e)
            assert c == brute_e2m1(y), (xi, e, c)
            clipped += abs(y) > 6.0
        # the default rule on the same block never clips
        dcodes, dsb = oracle.phi_block(x, oracle.FMT_MX)
        assert all(abs(math.ldexp(float(xi), -(dsb - 127))) <= 6.0 for xi in x)
    assert clipped > 0          # the sample reaches the clipping range


def _blocks_with_max(rng, shape, axis_len_blocks, axis, top):
    """Random bf16-exact values in (-3.5, 3.5) 2^k whose every 32-block (along
    `axis`) has one element of magnitude exactly `top` 2^k."""
    x = (rng.uniform(-3.5, 3.5, shape)).astype(np.float32)
    x = np.round(x * 16) / 16                        # 6 significant bits: exact in bf16
    xm = np.moveaxis(x, axis, -1)
    for idx in np.ndindex(xm.shape[:-1]):
        for b in range(axis_len_blocks):
            j = b * 32 + int(rng.integers(0, 32))
            xm[idx + (j,)] = top * (1 if rng.random() < 0.5 else -1)
    return np.moveaxis(xm, -1, axis)


def test_ocp_attention_matches_default_when_every_block_max_is_4_times_a_power_of_two():
    """With every Q, K, V block max at 4 2^k both rules pick the same scale,
    and with N <= 32 the only unmasked P block holds the tile max (scale 2^0
    under both), so the outputs are bit-identical; one block max at 7 2^k
    makes them differ (it clips under the floor rule)."""
    rng = np.random.default_rng(82)
    B, H, N, D = 1, 2, 32, 64
    q = _blocks_with_max(rng, (B, H, N, D), D // 32, 3, 4.0)
    k = _blocks_with_max(rng, (B, H, N, D), D // 32, 3, 4.0)
    v = _blocks_with_max(rng, (B, H, N, D), 1, 2, 4.0)
    qb, kb, vb = wl.to_bits(q, 1), wl.to_bits(k, 1), wl.to_bits(v, 1)
    assert np.array_equal(wl.from_bits(qb, 1), q)
    f = oracle.NO_SMOOTH_K          # K' = K, so its block maxima stay as built
    a, _, _ = oracle.attn(qb, kb, vb, wl.IN_BF16, False, oracle.FMT_MX, 64, flags=f)
    b, _, _ = oracle.attn(qb, kb, vb, wl.IN_BF16, False, oracle.FMT_MX, 64, flags=f | oracle.OCP_SCALE)
    assert np.array_equal(a, b)
    q2 = q.copy()
    j = int(np.flatnonzero(np.abs(q2[0, 0, 5, :32]) == 4.0)[0])
    q2[0, 0, 5, j] = 7.0 * np.sign(q2[0, 0, 5, j])
    qb2 = wl.to_bits(q2, 1)
    a2, _, _ = oracle.attn(qb2, kb, vb, wl.IN_BF16, False, oracle.FMT_MX, 64, flags=f)
    b2, _, _ = oracle.attn(qb2, kb, vb, wl.IN_BF16, False, oracle.FMT_MX, 64, flags=f | oracle.OCP_SCALE)
    assert not np.array_equal(a2[5], b2[5])
    assert np.array_equal(np.delete(a2, 5, axis=0), np.delete(b2, 5, axis=0))


def _metrics(fmt, flags, seed, N=512, D=128, k_bias_var=1.0, outlier_frac=0.0):
    q, k, v = wl.make_inputs(1, 2, N, D, wl.IN_BF16, seed=seed, k_bias_var=k_bias_var, outlier_frac=outlier_frac)
    rows = np.arange(0, 2 * N, 2, dtype=np.int64)
    ex = oracle.exact_attn(q, k, v, wl.IN_BF16, False, rows=rows)
    out, _, _ = oracle.attn(q, k, v, wl.IN_BF16, False, fmt, 128, rows=rows, flags=flags)
    return oracle.metrics(ex, out)


@pytest.mark.parametrize("seed", [90, 91])
def test_r6_beats_the_literal_448x6_with_e8m0_scales(seed):
    """C9: with E8M0 scales the literal 448*6 puts the tile max at a 2^9
    scale where it rounds from 5.25 to 6 (14% error on the largest P value);
    R = 6 maps it exactly onto code 6."""
    a = _metrics(oracle.FMT_MX, 0, seed)
    b = _metrics(oracle.FMT_MX, oracle.R_LITERAL, seed)
    assert a["l1"] < b["l1"] and a["rmse"] < b["rmse"] and a["cossim"] > b["cossim"]


def test_r_literal_tile_max_lands_at_5_25_times_2_to_9():
    """The arithmetic behind C9: P~2 at the tile max is 2688 = 5.25 * 2^9, so
    its E8M0 exponent is 9 and its code is 6 (5.25 rounds up)."""
    S = np.zeros(128, dtype=np.float32)
    S[3] = 10.0
    r = oracle.p_tile(S, 10.0, 128, oracle.FMT_MX, flags=oracle.R_LITERAL)
    assert abs(r["p2"][3] - 2688.0) <= 2688.0 * 2.0 ** -20
    assert int(r["sbytes"][0]) - 127 == 9 and r["codes"][3] == 7
    r6 = oracle.p_tile(S, 10.0, 128, oracle.FMT_MX)
    assert int(r6["sbytes"][0]) - 127 == 0 and r6["codes"][3] == 7


def _p_errors(flags, rng, trials=300):
    """Mean relative error of the E4M3 P scales and of the reconstructed P~
    (relative to each row's max), over tiles of Gaussian scores."""
    D = 128
    c2 = 1.0 / (math.log(2.0) * math.sqrt(D))
    s_err, p_err = [], []
    for _ in range(trials):
        S = (rng.standard_normal(128) * rng.uniform(5, 40)).astype(np.float32)
        m = float(S.max()) + float(rng.uniform(0, 10))
        r = oracle.p_tile(S, m, D, oracle.FMT_NV16, flags=flags)
        pt = np.exp2(c2 * (S.astype(np.float64) - m))                 # P~ exactly
        s1 = r["s1"]
        for b in range(128 // 16):
            blk = slice(16 * b, 16 * b + 16)
            s_exact = (pt[blk] / s1).max() / 6.0                     # the scale phi asks for
            s_q = oracle.e4m3_decode(int(r["sbytes"][b]))
            s_err.append(abs(s_q - s_exact) / s_exact if s_exact > 0 else 0.0)
            deq = np.array([oracle.e2m1_decode(int(c)) for c in r["codes"][blk]]) * s_q * s1
            p_err.append(np.abs(deq - pt[blk]).mean() / pt.max())
    return float(np.mean(s_err)), float(np.mean(p_err))


def test_two_level_lowers_the_scale_and_p_errors():
    """Fig. 3 (d, e): direct quantization leaves the scales of P~ in
    [0, 1/6], where E4M3 has few values and subnormal steps; the two-level
    scheme moves them into the full E4M3 range, which lowers both the error
    of the scales and the error of the reconstructed P~."""
    rng = np.random.default_rng(95)
    sd, pd = _p_errors(oracle.DIRECT_P, rng)
    rng = np.random.default_rng(95)
    s2, p2 = _p_errors(0, rng)
    assert s2 < sd and p2 < pd
    assert s2 < 0.05             # E4M3 with 3 mantissa bits: at most 1/16 relative error for normals
