"""GPU parity of the 8-bit attention forward (Algorithm 2) against the oracle,
through the C ABI: psi codes, scales and the smoothing mean bit-exact in every
role; O within 2e-3 + the oracle's per-row tie bound (codes of P^ whose
pre-rounding value lies within 8 ulp of a rounding midpoint, where the GPU's
exp2 may pick the other neighbour); L within 1e-5 (1 + |L|)."""
import numpy as np
import pytest

import oracle
from paper_2505_11594_amd import binding as bd
from paper_2505_11594_amd import workloads as wl

from _gpu import to_dev, torch_dev, say
from _layout import pad128
from test_gpu_attn import check, o_rows

pytestmark = pytest.mark.gpu

BKV = 128      # the default KV tile; SAGE_BKV64 selects 64


def bkv_flag(bkv):
    return bd.SAGE_BKV64 if bkv == 64 else 0


def v_stored_position(t):
    """Column of token t in V^T: inside each 32-token group, token 8g + 4h + r
    sits at 16h + 4g + r."""
    t = np.asarray(t)
    o = t & 31
    g, h, r = o >> 3, (o >> 2) & 1, o & 3
    return (t & ~31) | (h << 4) | (g << 2) | r


def logical_i8(codes, scales, role, B, H, N, D, bkv=BKV):
    """Device buffers -> the oracle's layout, and the padding that must be zero."""
    c = codes.cpu().numpy()
    s = scales.cpu().numpy()
    if role == bd.SAGE_ROLE_Q:
        return c.reshape(B, H, N, D), s.reshape(B, H, -1), np.zeros(0), np.zeros(0)
    Np = pad128(N)
    nb = (N + bkv - 1) // bkv
    s = s.reshape(B, H, Np // bkv)
    if role == bd.SAGE_ROLE_K:
        c = c.reshape(B, H, Np, D)
        return c[:, :, :N], s[:, :, :nb], c[:, :, N:], s[:, :, nb:]
    vt = c.reshape(B, H, D, Np)
    pos = v_stored_position(np.arange(N))
    logical = np.transpose(vt[:, :, :, pos], (0, 1, 3, 2))
    tail = np.setdiff1d(np.arange(Np), pos)
    return logical, s[:, :, :nb], vt[:, :, :, tail], s[:, :, nb:]


def gpu_i8(q, k, v, in_dtype, causal, flags=0, out_f32=True, bkv=BKV):
    torch = torch_dev()
    flags |= bkv_flag(bkv)
    o, L = bd.sage_attn_int8_fwd(to_dev(q, in_dtype), to_dev(k, in_dtype), to_dev(v, in_dtype), causal=causal,
                                 flags=flags, out_f32=out_f32)
    torch.cuda.synchronize()
    return o, L


def check_lse(got, ref, label):
    err = np.abs(got - ref)
    lim = 1e-5 * (1 + np.abs(ref))
    say("%s: L max err %.3g" % (label, float(err.max())))
    assert np.all(err <= lim), "%s: L off by %.3g" % (label, float(err.max()))


@pytest.mark.parametrize("shape", [(1, 1, 1, 64), (1, 2, 100, 128), (2, 1, 128, 64), (1, 1, 129, 128),
                                   (1, 3, 300, 128), (1, 1, 1000, 64)])
@pytest.mark.parametrize("in_dtype", [0, 1])
@pytest.mark.parametrize("smooth", [True, False])
@pytest.mark.parametrize("bkv", [64, 128])
def test_quant_int8_bit_exact(shape, in_dtype, smooth, bkv):
    B, H, N, D = shape
    say("quant int8", shape, "dtype", in_dtype, "smooth", smooth, "bkv", bkv)
    q, k, v = wl.make_inputs(B, H, N, D, in_dtype, seed=700 + N + D, k_bias_var=4.0, outlier_frac=0.02)
    torch = torch_dev()
    for role, x, blk in ((bd.SAGE_ROLE_Q, q, 128), (bd.SAGE_ROLE_K, k, bkv), (bd.SAGE_ROLE_V, v, bkv)):
        flags = (0 if smooth else bd.SAGE_NO_SMOOTH_K) | bkv_flag(bkv)
        codes, scales, mu = bd.sage_quant_int8(to_dev(x, in_dtype), role, flags)
        torch.cuda.synchronize()
        c, s, ctail, stail = logical_i8(codes, scales, role, B, H, N, D, bkv)
        oc, os_, omu = oracle.quant_int8(x, in_dtype, role, blk, smooth_k=smooth)
        assert np.array_equal(c, oc), role
        assert np.array_equal(s.view(np.uint32), os_.view(np.uint32)), role
        assert not ctail.any() and not stail.any()
        if omu is not None:
            assert np.array_equal(mu.cpu().numpy().view(np.uint32), omu.view(np.uint32))


def test_quant_int8_zero_blocks():
    """All-zero blocks (Q rows 0..127; K constant per channel, so K' = 0)
    get s = 0 and zero codes."""
    B, H, N, D = 1, 1, 256, 128
    q, k, v = wl.make_inputs(B, H, N, D, 1, seed=710)
    q[:, :, :128] = 0
    k[:] = k[:, :, :1]
    torch = torch_dev()
    for role, x, blk in ((bd.SAGE_ROLE_Q, q, 128), (bd.SAGE_ROLE_K, k, BKV)):
        codes, scales, _ = bd.sage_quant_int8(to_dev(x, 1), role, bkv_flag(BKV))
        torch.cuda.synchronize()
        c, s, _, _ = logical_i8(codes, scales, role, B, H, N, D)
        oc, os_, _ = oracle.quant_int8(x, 1, role, blk)
        assert np.array_equal(c, oc) and np.array_equal(s, os_)
    assert os_.max() == 0.0


@pytest.mark.parametrize("N", [1, 64, 100, 257, 640])
@pytest.mark.parametrize("D", [64, 128])
@pytest.mark.parametrize("causal", [False, True])
@pytest.mark.parametrize("bkv", [64, 128])
def test_attn_int8_edge_shapes(N, D, causal, bkv):
    say("attn int8 edge N=%d D=%d causal=%d bkv=%d" % (N, D, causal, bkv))
    in_dtype = 1 if (N + D) % 2 else 0
    q, k, v = wl.make_inputs(1, 2, N, D, in_dtype, seed=720 + N, k_bias_var=4.0, outlier_frac=0.02)
    o, L = gpu_i8(q, k, v, in_dtype, causal, bkv=bkv)
    ref, lref, tie, _ = oracle.attn_int8(q, k, v, in_dtype, causal, bkv)
    check(o.cpu().numpy().reshape(-1, D), ref, tie, "int8 edge")
    check_lse(L.cpu().numpy().ravel(), lref, "int8 edge")


def test_attn_int8_no_smooth_k_and_zero_scales():
    """The ablation flag, and a tile whose K block is all zero after
    smoothing (c_t = 0 in the kernel's log2-domain scores)."""
    q, k, v = wl.make_inputs(1, 2, 300, 128, 1, seed=730, k_bias_var=4.0)
    o, L = gpu_i8(q, k, v, 1, False, flags=bd.SAGE_NO_SMOOTH_K)
    ref, lref, tie, _ = oracle.attn_int8(q, k, v, 1, False, BKV, flags=oracle.NO_SMOOTH_K)
    check(o.cpu().numpy().reshape(-1, 128), ref, tie, "int8 no smooth-K")
    check_lse(L.cpu().numpy().ravel(), lref, "int8 no smooth-K")
    k2 = k.copy()
    k2[:] = k2[:, :, :1]                     # every key equal: K' = 0, s_K = 0 on every tile
    for causal in (False, True):
        o, L = gpu_i8(q, k2, v, 1, causal)
        ref, lref, tie, _ = oracle.attn_int8(q, k2, v, 1, causal, BKV)
        check(o.cpu().numpy().reshape(-1, 128), ref, tie, "int8 zero K'")
        check_lse(L.cpu().numpy().ravel(), lref, "int8 zero K'")


@pytest.mark.parametrize("in_dtype", [0, 1])
def test_attn_int8_16bit_output(in_dtype):
    torch = torch_dev()
    q, k, v = wl.make_inputs(1, 2, 384, 128, in_dtype, seed=740)
    o, _ = gpu_i8(q, k, v, in_dtype, False, out_f32=False)
    assert o.dtype == (torch.bfloat16 if in_dtype == 1 else torch.float16)
    ref, _, tie, _ = oracle.attn_int8(q, k, v, in_dtype, False, BKV)
    rnd = np.abs(ref).max(axis=1) * (2.0 ** -8 if in_dtype == 1 else 2.0 ** -11)
    check(o.float().cpu().numpy().reshape(-1, 128), ref, tie, "int8 16-bit out", extra=rnd)


def test_attn_int8_entry_points_agree_and_deterministic():
    torch = torch_dev()
    B, H, N, D = 1, 4, 2048, 128
    q, k, v = wl.make_inputs(B, H, N, D, 1, seed=750, k_bias_var=1.0)
    qd, kd, vd = (to_dev(x, 1) for x in (q, k, v))
    a, la = bd.sage_attn_int8_fwd(qd, kd, vd)
    b, lb = bd.sage_attn_int8_fwd(qd, kd, vd)
    ws = torch.empty(bd.attn_int8_workspace_size(B, H, N, D, bd.SAGE_IN_BF16 | bd.SAGE_OUT_F32), dtype=torch.uint8,
                     device="cuda")
    c, lc = bd.sage_attn_int8_fwd(qd, kd, vd, workspace=ws)
    qq = bd.sage_quant_int8(qd, bd.SAGE_ROLE_Q)
    kq = bd.sage_quant_int8(kd, bd.SAGE_ROLE_K)
    vq = bd.sage_quant_int8(vd, bd.SAGE_ROLE_V)
    e, le = bd.sage_attn_int8_fwd_prequant(qq[:2], kq[:2], vq[:2], (B, H, N, D))
    torch.cuda.synchronize()
    for x, y in ((a, b), (a, c), (a, e), (la, lb), (la, lc), (la, le)):
        assert torch.equal(x, y)
    n, ln = bd.sage_attn_int8_fwd(qd, kd, vd, lse=False)
    torch.cuda.synchronize()
    assert ln is None and torch.equal(a, n)


def test_attn_int8_closed_form_q_zero():
    """Q = 0: O is the mean of the dequantized V, L = ln(#keys)."""
    q, k, v = wl.make_inputs(1, 1, 300, 128, 1, seed=760)
    q[:] = 0
    o, L = gpu_i8(q, k, v, 1, True)
    vc, vs, _ = oracle.quant_int8(v, 1, oracle.ROLE_V, BKV)
    vd = vc[0, 0].astype(np.float64) * np.repeat(vs[0, 0].astype(np.float64), BKV)[:300, None]
    cnt = np.arange(1, 301)
    expect = np.cumsum(vd, axis=0) / cnt[:, None]
    assert np.abs(o.cpu().numpy().reshape(300, 128) - expect).max() < 1e-5 * np.abs(vd).max()
    assert np.abs(L.cpu().numpy().ravel() - np.log(cnt)).max() < 1e-5 * np.log(300)


@pytest.mark.parametrize("ci", [0, 1, 2, 3, 4])
def test_attn_int8_workloads_sampled_rows(ci):
    """The five workloads at full size (64-key tiles); the oracle computes a
    seeded sample of rows."""
    w = wl.CONFIGS[ci]
    say("attn int8 workload", ci, w.name)
    q, k, v = wl.generate(w)
    o, L = gpu_i8(q, k, v, w.in_dtype, w.causal)
    BH = w.B * w.H
    heads = sorted({0, BH - 1} | set(np.random.default_rng(ci + 70).choice(BH, min(BH, 4), replace=False).tolist()))
    rows = wl.sample_rows(w, per_head_tiles=3, tile=128, rows_per_tile=8, heads=heads, seed=ci + 70)
    ref, lref, tie, cnt = oracle.attn_int8(q, k, v, w.in_dtype, w.causal, BKV, rows=rows)
    got = o_rows(o, rows, w.D)
    check(got, ref, tie, w.name + " int8")
    check_lse(L.reshape(-1)[torch_dev().from_numpy(rows).to(L.device)].cpu().numpy(), lref, w.name + " int8")
    ex = oracle.exact_attn(q, k, v, w.in_dtype, w.causal, rows=rows)
    say("int8 accuracy vs exact (sampled rows)", oracle.metrics(ex, got), cnt)


def test_binding_rejects_mismatched_buffers():
    torch = torch_dev()
    q = torch.zeros((1, 2, 100, 64), dtype=torch.bfloat16, device="cuda:0")
    f32 = lambda *s: torch.zeros(s, dtype=torch.float32, device="cuda:0")
    with pytest.raises(ValueError):
        bd.sage_attn_int8_fwd(q, q, q, out=torch.zeros_like(q))
    with pytest.raises(ValueError):
        bd.sage_attn_int8_fwd(q, q, q, lse_out=f32(1, 2, 64))
    qq = bd.sage_quant_int8(q, bd.SAGE_ROLE_Q)
    kq = bd.sage_quant_int8(q, bd.SAGE_ROLE_K)
    vq = bd.sage_quant_int8(q, bd.SAGE_ROLE_V)
    with pytest.raises(ValueError):      # K^ holds Np = 128 rows, Q^ holds N = 100
        bd.sage_attn_int8_fwd_prequant(kq[:2], kq[:2], vq[:2], (1, 2, 100, 64))
    o, L = bd.sage_attn_int8_fwd(q, q, q)
    with pytest.raises(ValueError):
        bd.sage_attn_int8_bwd(q, q, q, o, L, q, out=[f32(1, 2, 100, 64), f32(1, 2, 100, 64), torch.zeros_like(q)])
    torch.cuda.synchronize()
