"""GPU parity of smoothing Q (Algorithm 1: phi(Q_i - mean(Q_i)) over blocks of
128 query rows, plus GEMV(mean(Q_i), K'^T) added to the scores) against the
oracle, in both formats: bit-exact codes, scales and block means; attention
within the same bar as without smoothing (2e-3 + the oracle's per-row tie
bound)."""
import numpy as np
import pytest

import oracle
from paper_2505_11594_amd import binding as bd
from paper_2505_11594_amd import workloads as wl

from _gpu import to_dev, torch_dev, say
from _layout import q_logical
from test_gpu_attn import check, o_rows
from test_oracle_smooth_q import q_with_channel_bias

pytestmark = pytest.mark.gpu


def q_bias_inputs(B, H, N, D, in_dtype, seed, bias_std=2.0):
    """(q, k, v) bits with a per-channel bias on Q (and on K)."""
    q, k, v = wl.make_inputs(B, H, N, D, in_dtype, seed=seed, k_bias_var=1.0, outlier_frac=0.02)
    rng = np.random.default_rng(seed + 7)
    qf = wl.from_bits(q, in_dtype) + rng.standard_normal((B, H, 1, D)).astype(np.float32) * np.float32(bias_std)
    return wl.to_bits(qf, in_dtype), k, v


@pytest.mark.parametrize("fmt", [0, 1])
@pytest.mark.parametrize("shape", [(1, 1, 1, 64), (1, 2, 100, 128), (2, 1, 128, 64), (1, 1, 129, 128),
                                   (1, 3, 300, 128), (1, 1, 1000, 64)])
@pytest.mark.parametrize("in_dtype", [0, 1])
def test_quant_q_smooth_bit_exact(fmt, shape, in_dtype):
    B, H, N, D = shape
    say("quant Q smooth", shape, "fmt", fmt, "dtype", in_dtype)
    q, _, _ = q_bias_inputs(B, H, N, D, in_dtype, seed=400 + N + D)
    torch = torch_dev()
    codes, scales, qbar = bd.sage_quant_fp4(to_dev(q, in_dtype), bd.SAGE_ROLE_Q, fmt | bd.SAGE_SMOOTH_Q)
    torch.cuda.synchronize()
    c, s = q_logical(codes.cpu().numpy(), scales.cpu().numpy(), B, H, N, D, fmt)
    oc, os_, oqbar = oracle.quant_smooth_q(q, in_dtype, fmt, 128)
    assert np.array_equal(qbar.cpu().numpy().view(np.uint32), oqbar.view(np.uint32))
    assert int((c != oc).sum()) == 0 and int((s != os_).sum()) == 0


def gpu_attn_sq(q, k, v, in_dtype, causal, bkv, extra=0, fmt=0):
    torch = torch_dev()
    f = fmt | bd.SAGE_SMOOTH_Q | extra | bd.bkv_flag(bkv)
    o = bd.sage_attn_fp4_fwd(to_dev(q, in_dtype), to_dev(k, in_dtype), to_dev(v, in_dtype), causal=causal, fmt=f)
    torch.cuda.synchronize()
    return o


@pytest.mark.parametrize("fmt", [0, 1])
@pytest.mark.parametrize("N", [1, 64, 100, 257, 640])
@pytest.mark.parametrize("D", [64, 128])
@pytest.mark.parametrize("causal", [False, True])
@pytest.mark.parametrize("bkv", [64, 128])
def test_attn_smooth_q_edge_shapes(fmt, N, D, causal, bkv):
    say("attn smooth-Q edge fmt=%d N=%d D=%d causal=%d bkv=%d" % (fmt, N, D, causal, bkv))
    in_dtype = 1 if (N + D) % 2 else 0
    q, k, v = q_bias_inputs(1, 2, N, D, in_dtype, seed=500 + N)
    o = gpu_attn_sq(q, k, v, in_dtype, causal, bkv, fmt=fmt)
    ref, tie, _ = oracle.attn(q, k, v, in_dtype, causal, fmt, bkv, flags=oracle.SMOOTH_Q)
    check(o.cpu().numpy().reshape(-1, D), ref, tie, "smooth-Q edge")


@pytest.mark.parametrize("N", [1, 100, 300, 512, 640])
@pytest.mark.parametrize("D", [64, 128])
@pytest.mark.parametrize("causal", [False, True])
def test_attn_smooth_q_bkv256_edge_shapes(N, D, causal):
    say("attn smooth-Q bkv256 edge N=%d D=%d causal=%d" % (N, D, causal))
    in_dtype = 1 if (N + D) % 2 else 0
    q, k, v = q_bias_inputs(1, 2, N, D, in_dtype, seed=530 + N)
    o = gpu_attn_sq(q, k, v, in_dtype, causal, 256)
    ref, tie, _ = oracle.attn(q, k, v, in_dtype, causal, oracle.FMT_MX, 256, flags=oracle.SMOOTH_Q)
    check(o.cpu().numpy().reshape(-1, D), ref, tie, "smooth-Q bkv256 edge")


def test_attn_smooth_q_without_smoothing_k():
    q, k, v = q_bias_inputs(1, 2, 300, 128, 1, seed=510)
    o = gpu_attn_sq(q, k, v, 1, False, 128, extra=bd.SAGE_NO_SMOOTH_K)
    ref, tie, _ = oracle.attn(q, k, v, 1, False, oracle.FMT_MX, 128, flags=oracle.SMOOTH_Q | oracle.NO_SMOOTH_K)
    check(o.cpu().numpy().reshape(-1, 128), ref, tie, "smooth-Q, no smooth-K")


@pytest.mark.parametrize("ci,fmt", [(1, 0), (3, 0), (4, 1)])
def test_attn_smooth_q_full_size_sampled_rows(ci, fmt):
    """Full-size workloads (non-causal, causal, and the D=64 long sequence in the
    16-element E4M3 format) with smoothing Q; the oracle computes a seeded
    sample of rows."""
    w = wl.CONFIGS[ci]
    say("attn smooth-Q config", ci, w.name, "fmt", fmt)
    q, k, v = wl.generate(w)
    o = gpu_attn_sq(q, k, v, w.in_dtype, w.causal, w.bkv, fmt=fmt)
    BH = w.B * w.H
    heads = sorted({0, BH - 1} | set(np.random.default_rng(ci + 50).choice(BH, min(BH, 4), replace=False).tolist()))
    rows = wl.sample_rows(w, per_head_tiles=3, tile=128, rows_per_tile=8, heads=heads, seed=ci + 50)
    ref, tie, cnt = oracle.attn(q, k, v, w.in_dtype, w.causal, fmt, w.bkv, rows=rows, flags=oracle.SMOOTH_Q)
    got = o_rows(o, rows, w.D)
    check(got, ref, tie, w.name + " smooth-Q")
    ex = oracle.exact_attn(q, k, v, w.in_dtype, w.causal, rows=rows)
    say("accuracy vs exact (sampled rows)", oracle.metrics(ex, got), cnt)


def test_attn_smooth_q_raises_accuracy_on_q_bias():
    """The paper's smoothing ablation, on the GPU output: with a channel bias on
    Q, smoothing Q lowers the error against exact attention."""
    B, H, N, D = 1, 4, 1024, 128
    q, k, v = q_with_channel_bias(B, H, N, D, seed=520, bias_std=3.0)
    torch = torch_dev()
    sm = gpu_attn_sq(q, k, v, 1, False, 128).cpu().numpy().reshape(-1, D)
    ns = bd.sage_attn_fp4_fwd(to_dev(q, 1), to_dev(k, 1), to_dev(v, 1), fmt=bd.SAGE_FMT_MXFP4)
    torch.cuda.synchronize()
    ns = ns.cpu().numpy().reshape(-1, D)
    rows = np.arange(0, B * H * N, 5, dtype=np.int64)
    ex = oracle.exact_attn(q, k, v, 1, False, rows=rows)
    a, b = oracle.metrics(ex, sm[rows]), oracle.metrics(ex, ns[rows])
    say("smooth-Q", a, "without", b)
    assert a["l1"] < b["l1"] and a["cossim"] > b["cossim"]


def test_attn_smooth_q_prequant_is_unsupported():
    torch = torch_dev()
    q, k, v = q_bias_inputs(1, 1, 128, 64, 1, seed=530)
    qq = bd.sage_quant_fp4(to_dev(q, 1), bd.SAGE_ROLE_Q, bd.SAGE_SMOOTH_Q)
    kq = bd.sage_quant_fp4(to_dev(k, 1), bd.SAGE_ROLE_K)
    vq = bd.sage_quant_fp4(to_dev(v, 1), bd.SAGE_ROLE_V)
    torch.cuda.synchronize()
    with pytest.raises(bd.SageError) as ex:
        bd.sage_attn_fp4_fwd_prequant(qq[:2], kq[:2], vq[:2], (1, 1, 128, 64), fmt=bd.SAGE_SMOOTH_Q)
    assert ex.value.status == bd.SAGE_ERR_UNSUPPORTED
