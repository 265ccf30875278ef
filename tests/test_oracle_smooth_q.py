"""Pins for the oracle's smoothing Q (no GPU).

Algorithm 1 quantizes Q_i - mean(Q_i) for every block of B_q query rows and
adds GEMV(mean(Q_i), K_j^T) back to the scores.  Each test checks the oracle
against something independent of it: textbook softmax attention (the
decomposition q K^T = (q - qbar) K^T + qbar K^T is exact), numpy's own block
mean, the FP4 round-trip bound, and the paper's smoothing ablation (smoothing
Q raises accuracy when Q has a channel bias).
"""
import numpy as np
import pytest

import oracle
from paper_2505_11594_amd import workloads as wl

from test_oracle_attn import textbook_attention


def q_with_channel_bias(B, H, N, D, seed, bias_std=2.0):
    """bf16 bits of (Q, K, V) where Q carries one per-channel bias per head."""
    q, k, v = wl.make_inputs(B, H, N, D, wl.IN_BF16, seed=seed, k_bias_var=1.0)
    rng = np.random.default_rng(seed + 7)
    qf = wl.from_bits(q, 1) + rng.standard_normal((B, H, 1, D)).astype(np.float32) * np.float32(bias_std)
    return wl.to_bits(qf, 1), k, v


@pytest.mark.parametrize("bq", [16, 64, 128])
@pytest.mark.parametrize("causal", [False, True])
@pytest.mark.parametrize("N", [200, 256])
def test_smooth_q_identity_quantizer_equals_textbook_softmax(bq, causal, N):
    q, k, v = q_with_channel_bias(1, 2, N, 64, seed=40 + bq)
    out, _, _ = oracle.attn(q, k, v, wl.IN_BF16, causal, oracle.FMT_NONE, 64, flags=oracle.SMOOTH_Q, bq=bq)
    out = out.reshape(1, 2, N, 64)
    for h in range(2):
        ref = textbook_attention(wl.from_bits(q[0, h], 1), wl.from_bits(k[0, h], 1), wl.from_bits(v[0, h], 1), causal)
        err = np.abs(out[0, h] - ref).max() / np.abs(ref).max()
        assert err < 2e-6, err


@pytest.mark.parametrize("fmt", [oracle.FMT_MX, oracle.FMT_NV16])
@pytest.mark.parametrize("N,bq", [(300, 128), (64, 128), (130, 32)])
def test_smooth_q_block_mean_and_codes(fmt, N, bq):
    D = 64
    q, _, _ = q_with_channel_bias(1, 2, N, D, seed=50 + N)
    codes, scales, qbar = oracle.quant_smooth_q(q, wl.IN_BF16, fmt, bq)
    qf = wl.from_bits(q, 1).astype(np.float64)
    nqb = (N + bq - 1) // bq
    assert qbar.shape == (1, 2, nqb, D)
    for b in range(nqb):
        ref = qf[:, :, b * bq:(b + 1) * bq].mean(axis=2).astype(np.float32)   # numpy's fp64 mean, rounded
        assert np.array_equal(qbar[:, :, b], ref)
    n = 32 if fmt == oracle.FMT_MX else 16
    x = (wl.from_bits(q, 1) - np.repeat(qbar, bq, axis=2)[:, :, :N]).astype(np.float32)
    for h in range(2):
        for t in range(0, N, max(1, N // 17)):
            for blk in range(D // n):
                deq = oracle.dequant_block(codes[0, h, t, blk * n:(blk + 1) * n], int(scales[0, h, t, blk]), fmt)
                xs = x[0, h, t, blk * n:(blk + 1) * n].astype(np.float64)
                s = oracle.e8m0_decode(int(scales[0, h, t, blk])) if fmt == oracle.FMT_MX else \
                    oracle.e4m3_decode(int(scales[0, h, t, blk]))
                assert np.all(np.abs(deq - xs) <= s * (1 + 2 ** -6) + 1e-30)


def test_smooth_q_constant_rows_leave_only_p_and_v_error():
    """Identical rows in every query block: Q - qbar is exactly 0, the codes
    are 0, and S is the GEMV alone, so the MXFP4 result is closer to exact
    attention than without smoothing Q."""
    N, D, bq = 256, 64, 128
    rng = np.random.default_rng(60)
    rows = rng.standard_normal((1, 2, N // bq, D)).astype(np.float32) * 1.5
    qf = np.repeat(rows, bq, axis=2)
    q = wl.to_bits(qf, 1)
    _, k, v = wl.make_inputs(1, 2, N, D, wl.IN_BF16, seed=61, k_bias_var=1.0)
    codes, _, qbar = oracle.quant_smooth_q(q, wl.IN_BF16, oracle.FMT_MX, bq)
    assert not codes.any()
    assert np.array_equal(np.repeat(qbar, bq, axis=2), wl.from_bits(q, 1))
    ex = oracle.exact_attn(q, k, v, wl.IN_BF16, False).reshape(-1, D)
    sm, _, _ = oracle.attn(q, k, v, wl.IN_BF16, False, oracle.FMT_MX, 128, flags=oracle.SMOOTH_Q)
    ns, _, _ = oracle.attn(q, k, v, wl.IN_BF16, False, oracle.FMT_MX, 128)
    a, b = oracle.metrics(ex, sm), oracle.metrics(ex, ns)
    assert a["l1"] < 0.8 * b["l1"] and a["cossim"] > b["cossim"]


@pytest.mark.parametrize("fmt", [oracle.FMT_MX, oracle.FMT_NV16])
def test_smooth_q_helps_when_q_has_a_channel_bias(fmt):
    """The paper's smoothing ablation: smoothing Q raises accuracy."""
    N, D = 512, 128
    q, k, v = q_with_channel_bias(1, 2, N, D, seed=70, bias_std=3.0)
    rows = np.arange(0, 2 * N, 3, dtype=np.int64)
    ex = oracle.exact_attn(q, k, v, wl.IN_BF16, False, rows=rows)
    sm, _, _ = oracle.attn(q, k, v, wl.IN_BF16, False, fmt, 128, rows=rows, flags=oracle.SMOOTH_Q)
    ns, _, _ = oracle.attn(q, k, v, wl.IN_BF16, False, fmt, 128, rows=rows)
    a, b = oracle.metrics(ex, sm), oracle.metrics(ex, ns)
    assert a["l1"] < b["l1"] and a["rmse"] < b["rmse"] and a["cossim"] > b["cossim"]
