"""The no-allocation entry point sage_attn_fp4_fwd_noalloc: the same outputs as
sage_attn_fp4_fwd bit for bit, on two calls in a row of which the second is
smaller (the fixed scratch keeps the first call's contents), in both formats
and several KV tiles; and shapes whose workspace exceeds the scratch are
rejected on the host before any HIP call.  Collected last: a failure here
hides no other test."""
import os

import numpy as np
import pytest

from paper_2505_11594_amd import binding as bd
from paper_2505_11594_amd import workloads as wl

from _gpu import to_dev, torch_dev, say

FAKE = 0x10000  # aligned, non-null; never dereferenced because validation fails first


def test_noalloc_rejects_shapes_beyond_the_scratch():
    """Host only (no GPU): the size check comes before any HIP call."""
    if not os.path.exists(bd.LIB_PATH):
        import __graft_entry__
        __graft_entry__.build()
    L = bd.lib()
    limit = (256 << 20)
    # B1 H32 N32768 D128 fits; twice the heads does not
    assert bd.attn_fp4_workspace_size(1, 32, 32768, 128, bd.SAGE_BKV256) <= limit
    assert bd.attn_fp4_workspace_size(1, 64, 32768, 128, bd.SAGE_BKV256) > limit
    rc = L.sage_attn_fp4_fwd_noalloc(FAKE, FAKE, FAKE, FAKE, 1, 64, 32768, 128, 0, bd.SAGE_BKV256, None)
    assert rc == bd.SAGE_ERR_WORKSPACE
    rc = L.sage_attn_fp4_fwd_noalloc(None, FAKE, FAKE, FAKE, 1, 1, 128, 128, 0, 0, None)
    assert rc == bd.SAGE_ERR_INVALID_ARG


@pytest.mark.gpu
@pytest.mark.parametrize("fmt,bkv", [(0, 256), (0, 64), (1, 128), (0, 128)])
def test_noalloc_matches_the_allocating_entry_point(fmt, bkv):
    torch = torch_dev()
    f = fmt | bd.bkv_flag(bkv)
    for (B, H, N, D, causal, dtype, seed) in [(2, 3, 1000, 128, False, 1, 500), (1, 2, 300, 64, True, 0, 501)]:
        say("noalloc fmt=%d bkv=%d B=%d H=%d N=%d D=%d causal=%d" % (fmt, bkv, B, H, N, D, causal))
        q, k, v = wl.make_inputs(B, H, N, D, dtype, seed=seed, k_bias_var=4.0, outlier_frac=0.02)
        qd, kd, vd = (to_dev(x, dtype) for x in (q, k, v))
        ref = bd.sage_attn_fp4_fwd(qd, kd, vd, causal=causal, fmt=f)
        got = bd.sage_attn_fp4_fwd_noalloc(qd, kd, vd, causal=causal, fmt=f)
        out16 = bd.sage_attn_fp4_fwd_noalloc(qd, kd, vd, causal=causal, fmt=f, out_f32=False)
        ref16 = bd.sage_attn_fp4_fwd(qd, kd, vd, causal=causal, fmt=f, out_f32=False)
        torch.cuda.synchronize()
        assert torch.equal(got, ref)
        assert torch.equal(out16, ref16)
        assert np.isfinite(got.cpu().numpy()).all()


@pytest.mark.gpu
def test_noalloc_256_query_workgroups():
    """The bench step's launch shape (256-key tiles, 256-query workgroups,
    non-causal) through the no-allocation entry point: two calls in a row, the
    second smaller, each bit-equal to the allocating entry point."""
    torch = torch_dev()
    f = bd.SAGE_BKV256 | bd.SAGE_WG256
    for (B, H, N, D, dtype, seed) in [(2, 3, 1000, 128, 1, 510), (1, 2, 300, 64, 0, 511)]:
        say("noalloc wg256 B=%d H=%d N=%d D=%d" % (B, H, N, D))
        q, k, v = wl.make_inputs(B, H, N, D, dtype, seed=seed, k_bias_var=4.0, outlier_frac=0.02)
        qd, kd, vd = (to_dev(x, dtype) for x in (q, k, v))
        ref = bd.sage_attn_fp4_fwd(qd, kd, vd, causal=False, fmt=f)
        got = bd.sage_attn_fp4_fwd_noalloc(qd, kd, vd, causal=False, fmt=f)
        torch.cuda.synchronize()
        assert torch.equal(got, ref)
        assert np.isfinite(got.cpu().numpy()).all()
