"""GPU parity of the microscaled-FP4 attention forward (Algorithm 1 without
smoothing Q, two-level P quantization of Sec. 3.2) against the oracle.

Bar: |O_gpu - O_oracle| <= 2e-3 per element (fp32 output), plus, per row, the
oracle's tie_tol: the largest change any other accepted evaluation of the P
step can make.  The oracle evaluates P~, s_P1 and P~2 = P~/s_P1 in Algorithm
1's order; the kernel evaluates P~2 fused (exp2 of one fma, v_exp_f32 within
1 ulp) and takes the E8M0 exponent of each block from scores.  Codes whose
value lies within the two orders' difference of a rounding boundary, and
block scales within it of a boundary (notably the block of the tile max,
whose plain-order P~2 lands one ulp above 6 on a few percent of tiles and
then takes 2^1), may legitimately differ; tie_tol sums their effect."""
import numpy as np
import pytest

import oracle
from paper_2505_11594_amd import binding as bd
from paper_2505_11594_amd import workloads as wl

from _gpu import to_dev, torch_dev, say

pytestmark = pytest.mark.gpu

TOL = 2e-3


def gpu_attn(q, k, v, in_dtype, causal, fmt, bkv, out_f32=True, **kw):
    torch = torch_dev()
    f = fmt | bd.bkv_flag(bkv)
    o = bd.sage_attn_fp4_fwd(to_dev(q, in_dtype), to_dev(k, in_dtype), to_dev(v, in_dtype), causal=causal, fmt=f,
                             out_f32=out_f32, **kw)
    torch.cuda.synchronize()
    return o


def o_rows(o, rows, D):
    torch = torch_dev()
    flat = o.reshape(-1, D)
    idx = torch.from_numpy(rows).to(o.device)
    return flat.index_select(0, idx).float().cpu().numpy()


ALT = 1e-4    # a row whose tie_tol exceeds this has an accepted alternative P code or block scale


def check(got, ref, tie_tol, label, extra=None):
    err = np.abs(got - ref).max(axis=1)
    lim = TOL + tie_tol + (0 if extra is None else extra)
    bad = err > lim
    one = tie_tol <= ALT
    say("%s: rows=%d max_err=%.3g; rows with one accepted P step: %d, max_err %.3g; rows with alternatives: %d, "
        "max_err %.3g, max err/(2e-3 + tie_tol) %.3f" %
        (label, len(err), float(err.max()), int(one.sum()), float(err[one].max()) if one.any() else 0.0,
         int((~one).sum()), float(err[~one].max()) if (~one).any() else 0.0, float((err / lim).max())))
    assert not bad.any(), "%s: %d rows over the bar, worst err %.3g at row %d" % (
        label, int(bad.sum()), float(err[bad].max()), int(np.flatnonzero(bad)[0]))


@pytest.mark.parametrize("fmt", [0, 1])
@pytest.mark.parametrize("N", [1, 64, 100, 257, 640])
@pytest.mark.parametrize("D", [64, 128])
@pytest.mark.parametrize("causal", [False, True])
@pytest.mark.parametrize("bkv", [64, 128])
def test_attn_edge_shapes(fmt, N, D, causal, bkv):
    say("attn edge fmt=%d N=%d D=%d causal=%d bkv=%d" % (fmt, N, D, causal, bkv))
    in_dtype = 1 if (N + D) % 2 else 0
    q, k, v = wl.make_inputs(1, 2, N, D, in_dtype, seed=200 + N, k_bias_var=4.0, outlier_frac=0.02)
    o = gpu_attn(q, k, v, in_dtype, causal, fmt, bkv)
    ref, tie, _ = oracle.attn(q, k, v, in_dtype, causal, fmt, bkv)
    check(o.cpu().numpy().reshape(-1, D), ref, tie, "edge")


@pytest.mark.parametrize("N", [1, 100, 257, 300, 512, 640, 1000])
@pytest.mark.parametrize("D", [64, 128])
@pytest.mark.parametrize("causal", [False, True])
@pytest.mark.parametrize("out_f32", [True, False])
def test_attn_bkv256_edge_shapes(N, D, causal, out_f32):
    """256-key tiles (MXFP4): tails that end inside the tile's lower or upper
    128 keys (N = 100, 300, 640, 1000), an exact multiple of the tile (512),
    one token; 16-bit and fp32 outputs."""
    say("attn bkv256 edge N=%d D=%d causal=%d out_f32=%d" % (N, D, causal, out_f32))
    in_dtype = 1 if (N + D) % 2 else 0
    q, k, v = wl.make_inputs(1, 2, N, D, in_dtype, seed=300 + N, k_bias_var=4.0, outlier_frac=0.02)
    o = gpu_attn(q, k, v, in_dtype, causal, 0, 256, out_f32=out_f32)
    ref, tie, _ = oracle.attn(q, k, v, in_dtype, causal, oracle.FMT_MX, 256)
    got = o.float().cpu().numpy().reshape(-1, D)
    # a 16-bit output adds its own rounding: half an ulp of |O| <= max|V|
    extra = None if out_f32 else np.abs(ref).max(axis=1) * (2.0 ** -8 if in_dtype == 1 else 2.0 ** -11)
    check(got, ref, tie, "bkv256 edge", extra)


def test_attn_bkv256_rejected_for_nv16_and_with_bkv64():
    torch = torch_dev()
    q = torch.zeros((1, 1, 128, 64), dtype=torch.float16, device="cuda:0")
    with pytest.raises(RuntimeError):
        bd.sage_attn_fp4_fwd(q, q, q, fmt=bd.SAGE_FMT_NV16_E4M3 | bd.SAGE_BKV256)
    with pytest.raises(RuntimeError):
        bd.sage_attn_fp4_fwd(q, q, q, fmt=bd.SAGE_BKV64 | bd.SAGE_BKV256)


def test_attn_config0_all_rows():
    w = wl.CONFIGS[0]
    q, k, v = wl.generate(w)
    o = gpu_attn(q, k, v, w.in_dtype, w.causal, 0, w.bkv)
    ref, tie, cnt = oracle.attn(q, k, v, w.in_dtype, w.causal, oracle.FMT_MX, w.bkv)
    check(o.cpu().numpy().reshape(-1, w.D), ref, tie, w.name)
    ex = oracle.exact_attn(q, k, v, w.in_dtype, w.causal)
    say("accuracy vs exact", oracle.metrics(ex, o.cpu().numpy().reshape(-1, w.D)))


_GEN = {}


def generate_cached(ci):
    """Full-size inputs of workload ci, generated once per test session."""
    if ci not in _GEN:
        _GEN.clear()
        _GEN[ci] = wl.generate(wl.CONFIGS[ci])
    return _GEN[ci]


@pytest.mark.parametrize("b", [0, 1, 2, 3])
def test_attn_config1_all_rows(b):
    """B4 H32 N4096 D128 (K channel bias of variance 4) in the benchmark's launch
    configuration (one launch over all four batches, 256-key tiles): every
    row of batch b against the oracle."""
    ci = 1
    w = wl.CONFIGS[ci]
    say("attn config", ci, w.name, "batch", b, "all rows")
    q, k, v = generate_cached(ci)
    o = gpu_attn(q, k, v, w.in_dtype, w.causal, 0, w.bkv)
    rows = np.arange(b * w.H * w.N, (b + 1) * w.H * w.N, dtype=np.int64)
    ref, tie, cnt = oracle.attn(q, k, v, w.in_dtype, w.causal, 0, w.bkv, rows=rows)
    got = o_rows(o, rows, w.D)
    check(got, ref, tie, "%s batch %d" % (w.name, b))
    if b == 0:
        sub = rows[:: 64]
        ex = oracle.exact_attn(q, k, v, w.in_dtype, w.causal, rows=sub)
        say("accuracy vs exact (every 64th row)", oracle.metrics(ex, got[:: 64]), cnt)


WG = bd.SAGE_WG256


@pytest.mark.parametrize("ci,fmt,bkv,whole,shape", [(2, 0, None, True, WG), (2, 0, None, False, 0),
                                                    (2, 0, 128, False, 0), (3, 0, None, True, 0),
                                                    (3, 0, 128, False, 0), (4, 1, None, True, 0),
                                                    (4, 0, None, True, 0), (4, 0, 256, False, 0)])
def test_attn_configs_full_size_sampled_rows(ci, fmt, bkv, whole, shape):
    """The benchmark's launch configuration at full size (each workload's own
    KV tile, plus the other tile on the long, causal and D = 64 workloads;
    on the B1 H32 N32768 D128 workload 256-query workgroups as the bench step
    launches them, and the 128-query shape on sampled rows).  With whole=True
    the oracle computes 8 whole 128-row query tiles on each of 8 heads (first
    and last tile always, the tile ending on a KV-tile boundary when causal,
    the rest seeded); otherwise 8 rows of 4 tiles."""
    w = wl.CONFIGS[ci]
    assert fmt in w.fmts
    bkv = bkv or w.bkv
    say("attn config", ci, w.name, "fmt", fmt, "bkv", bkv, "whole tiles" if whole else "sampled rows",
        "256-query workgroups" if shape else "")
    q, k, v = generate_cached(ci)
    o = gpu_attn(q, k, v, w.in_dtype, w.causal, fmt | shape, bkv)
    BH = w.B * w.H
    rng = np.random.default_rng(ci)
    heads = sorted({0, BH - 1} | set(rng.choice(np.arange(1, BH - 1), min(BH - 2, 6), replace=False).tolist()))
    if whole:
        rows = wl.sample_rows(w, per_head_tiles=8, tile=128, rows_per_tile=128, heads=heads, seed=ci)
    else:
        rows = wl.sample_rows(w, per_head_tiles=4, tile=128, rows_per_tile=8, heads=heads, seed=ci)
    ref, tie, cnt = oracle.attn(q, k, v, w.in_dtype, w.causal, fmt, bkv, rows=rows)
    got = o_rows(o, rows, w.D)
    check(got, ref, tie, w.name)
    sub = rows[:: 16] if whole else rows
    ex = oracle.exact_attn(q, k, v, w.in_dtype, w.causal, rows=sub)
    say("accuracy vs exact (sampled rows)", oracle.metrics(ex, got[:: 16] if whole else got), cnt)


@pytest.mark.parametrize("fmt,bkv", [(0, 128), (1, 128), (0, 256), (0, 64)])
def test_attn_deterministic_and_entry_points_agree(fmt, bkv):
    """Two calls, the caller-workspace entry point and the prequantized one give
    the same bits (each KV tile size of the format)."""
    torch = torch_dev()
    w = wl.CONFIGS[1]
    q, k, v = wl.generate(w, B=1, H=4, N=2048)
    a = gpu_attn(q, k, v, w.in_dtype, False, fmt, bkv)
    b = gpu_attn(q, k, v, w.in_dtype, False, fmt, bkv)
    assert torch.equal(a, b)
    f = fmt | bd.bkv_flag(bkv)
    qd, kd, vd = (to_dev(x, w.in_dtype) for x in (q, k, v))
    ws = torch.empty(bd.attn_fp4_workspace_size(1, 4, 2048, 128, f | bd.SAGE_IN_BF16 | bd.SAGE_OUT_F32),
                     dtype=torch.uint8, device="cuda")
    c = bd.sage_attn_fp4_fwd(qd, kd, vd, causal=False, fmt=f, workspace=ws)
    qq = bd.sage_quant_fp4(qd, bd.SAGE_ROLE_Q, fmt)
    kq = bd.sage_quant_fp4(kd, bd.SAGE_ROLE_K, fmt)
    vq = bd.sage_quant_fp4(vd, bd.SAGE_ROLE_V, fmt)
    e = bd.sage_attn_fp4_fwd_prequant(qq[:2], kq[:2], vq[:2], (1, 4, 2048, 128), fmt=f)
    torch.cuda.synchronize()
    assert torch.equal(a, c) and torch.equal(a, e)


@pytest.mark.parametrize("in_dtype", [0, 1])
def test_attn_16bit_output(in_dtype):
    torch = torch_dev()
    q, k, v = wl.make_inputs(1, 2, 384, 128, in_dtype, seed=31)
    o = gpu_attn(q, k, v, in_dtype, False, 0, 128, out_f32=False)
    assert o.dtype == (torch.bfloat16 if in_dtype == 1 else torch.float16)
    ref, tie, _ = oracle.attn(q, k, v, in_dtype, False, oracle.FMT_MX, 128)
    rnd = np.abs(ref).max(axis=1) * (2.0 ** -8 if in_dtype == 1 else 2.0 ** -11)
    check(o.float().cpu().numpy().reshape(-1, 128), ref, tie, "16-bit out", extra=rnd)


def test_attn_no_smooth_k_matches_oracle_ablation():
    q, k, v = wl.make_inputs(1, 2, 512, 128, 1, seed=32, k_bias_var=4.0)
    o = gpu_attn(q, k, v, 1, False, bd.SAGE_NO_SMOOTH_K, 128)
    ref, tie, _ = oracle.attn(q, k, v, 1, False, oracle.FMT_MX, 128, flags=oracle.NO_SMOOTH_K)
    check(o.cpu().numpy().reshape(-1, 128), ref, tie, "no smooth-K")


def test_attn_closed_form_q_zero():
    """Q = 0: O is the mean of the dequantized V (every P code 6 at unit scale)."""
    torch = torch_dev()
    q, k, v = wl.make_inputs(1, 1, 300, 128, 1, seed=33)
    q[:] = 0
    o = gpu_attn(q, k, v, 1, False, 0, 128).cpu().numpy().reshape(-1, 128)
    vc, vs, _, _ = oracle.quant(v, 1, oracle.ROLE_V, oracle.FMT_MX)
    E2M1 = np.array([0, .5, 1, 1.5, 2, 3, 4, 6, -0., -.5, -1, -1.5, -2, -3, -4, -6])
    vdeq = E2M1[vc[0, 0]] * np.repeat(2.0 ** (vs[0, 0].astype(np.float64) - 127), 32, axis=1)
    expect = vdeq[:, :300].mean(axis=1)
    assert np.abs(o - expect[None, :]).max() < 1e-5


def test_binding_rejects_mismatched_buffers():
    """The C ABI takes bare pointers, so the binding checks every caller-supplied
    buffer against what the kernels will write or read; nothing is launched."""
    torch = torch_dev()
    q = torch.zeros((1, 2, 100, 64), dtype=torch.bfloat16, device="cuda:0")
    bad_out = [torch.zeros((1, 2, 100, 64), dtype=torch.bfloat16, device="cuda:0"),      # fp32 expected
               torch.zeros((1, 2, 100, 32), dtype=torch.float32, device="cuda:0"),
               torch.zeros((1, 2, 64, 100), dtype=torch.float32, device="cuda:0").transpose(2, 3)]
    for o in bad_out:
        with pytest.raises(ValueError):
            bd.sage_attn_fp4_fwd(q, q, q, out=o)
        with pytest.raises(ValueError):
            bd.sage_attn_bf16_fwd(q, q, q, out=o)
    with pytest.raises(ValueError):
        bd.sage_attn_fp4_fwd(q, q, q, workspace=torch.zeros(1 << 20, dtype=torch.float32, device="cuda:0"))
    # k and v of another dtype with the right shape (fp16 or fp32 read as bf16,
    # a 1-byte dtype read past its end) or on the host
    others = [torch.zeros((1, 2, 100, 64), dtype=dt, device="cuda:0")
              for dt in (torch.float16, torch.float32, torch.uint8, torch.int8, torch.bool)]
    others.append(torch.zeros((1, 2, 100, 64), dtype=torch.bfloat16))
    for x in others:
        for fwd in (bd.sage_attn_fp4_fwd, bd.sage_attn_bf16_fwd, bd.sage_attn_int8_fwd):
            with pytest.raises((ValueError, TypeError)):
                fwd(q, x, q)
            with pytest.raises((ValueError, TypeError)):
                fwd(q, q, x)
    qq = bd.sage_quant_fp4(q, bd.SAGE_ROLE_Q)
    kq = bd.sage_quant_fp4(q, bd.SAGE_ROLE_K)
    vq = bd.sage_quant_fp4(q, bd.SAGE_ROLE_V)
    with pytest.raises(ValueError):      # K^ holds Np = 128 rows, Q^ holds N = 100
        bd.sage_attn_fp4_fwd_prequant(kq[:2], kq[:2], vq[:2], (1, 2, 100, 64))
    with pytest.raises(ValueError):
        bd.sage_attn_fp4_fwd_prequant(qq[:2], kq[:2], vq[:2], (1, 2, 100, 64), out_f32=False,
                                      out=torch.zeros((1, 2, 100, 64), dtype=torch.float32, device="cuda:0"))
    o = bd.sage_attn_fp4_fwd_prequant(qq[:2], kq[:2], vq[:2], (1, 2, 100, 64))      # the matching call runs
    torch.cuda.synchronize()
    assert o.shape == (1, 2, 100, 64) and o.dtype == torch.float32


@pytest.mark.parametrize("N,D", [(1, 64), (100, 128), (257, 64), (300, 128), (640, 128), (1000, 64)])
def test_attn_wg256_same_bits_as_default(N, D):
    """SAGE_WG256 (256 queries per workgroup, each K^/V^T tile shared by 8
    waves) changes who loads a tile, not what any wave computes: the output is
    bit-identical to the default 128-query workgroups, fp32 and 16-bit."""
    torch = torch_dev()
    say("attn wg256 N=%d D=%d" % (N, D))
    in_dtype = 1 if N % 2 else 0
    q, k, v = wl.make_inputs(2, 3, N, D, in_dtype, seed=700 + N, k_bias_var=4.0, outlier_frac=0.02)
    got = None
    for out_f32 in (True, False):
        a = gpu_attn(q, k, v, in_dtype, False, 0, 256, out_f32=out_f32)
        qd, kd, vd = (to_dev(x, in_dtype) for x in (q, k, v))
        b = bd.sage_attn_fp4_fwd(qd, kd, vd, causal=False, fmt=bd.SAGE_BKV256 | bd.SAGE_WG256, out_f32=out_f32)
        torch.cuda.synchronize()
        assert torch.equal(a, b)
        if out_f32:
            got = b.cpu().numpy().reshape(-1, D)
    ref, tie, _ = oracle.attn(q, k, v, in_dtype, False, oracle.FMT_MX, 256)
    check(got, ref, tie, "wg256")


def test_attn_wg256_bench_workload_same_bits():
    """The bench workload (B1 H32 N32768 D128, outlier rows) with SAGE_WG256:
    every output bit equal to the default launch."""
    torch = torch_dev()
    w = wl.CONFIGS[2]
    q, k, v = generate_cached(2)
    a = gpu_attn(q, k, v, w.in_dtype, False, 0, 256)
    qd, kd, vd = (to_dev(x, w.in_dtype) for x in (q, k, v))
    b = bd.sage_attn_fp4_fwd(qd, kd, vd, causal=False, fmt=bd.SAGE_BKV256 | bd.SAGE_WG256)
    torch.cuda.synchronize()
    assert torch.equal(a, b)
