"""The C-ABI library loads without a GPU, exports every declared symbol and
rejects invalid arguments on the host before any HIP call (no GPU needed)."""
import ctypes
import os
import re

import pytest

from paper_2505_11594_amd import binding as bd

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "sage_mi355x.h")

FAKE = 0x10000  # aligned, non-null; never dereferenced because validation fails first


def declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(sage_[a-z0-9_]+)\s*\(", src)))


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(bd.LIB_PATH):
        import __graft_entry__
        __graft_entry__.build()
    return bd.lib()


def test_every_declared_symbol_is_exported(L):
    names = declared_functions()
    assert len(names) >= 9
    for n in names:
        assert hasattr(L, n), n


def test_status_strings(L):
    assert bd.status_string(0) == "SAGE_OK"
    assert bd.status_string(1) == "SAGE_ERR_INVALID_ARG"
    assert bd.status_string(99) == "SAGE_ERR_UNKNOWN"
    assert "gfx950" in bd.version()


def _attn(L, **kw):
    a = dict(q=FAKE, k=FAKE, v=FAKE, o=FAKE, B=1, H=1, N=128, D=128, causal=0, fmt=0)
    a.update(kw)
    return L.sage_attn_fp4_fwd(a["q"], a["k"], a["v"], a["o"], a["B"], a["H"], a["N"], a["D"], a["causal"], a["fmt"], None)


@pytest.mark.parametrize("bad", [dict(q=None), dict(o=None), dict(q=FAKE + 2), dict(B=0), dict(H=-1), dict(N=0),
                                 dict(D=96), dict(D=256), dict(causal=2), dict(fmt=0x200), dict(fmt=0x3),
                                 dict(fmt=0x40 | 0x80), dict(N=1 << 30),
                                 dict(N=(1 << 24) + 1), dict(D=64, N=(1 << 25) + 1)])
def test_attn_invalid_args_rejected_on_host(L, bad):
    assert _attn(L, **bad) == bd.SAGE_ERR_INVALID_ARG


def test_attn_unsupported(L):
    # smoothing Q needs the GEMV term, which prequantized inputs lack
    for f in (0, bd.SAGE_FMT_NV16_E4M3):
        assert L.sage_attn_fp4_fwd_prequant(FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 1, 1, 128, 128, 0,
                                            f | bd.SAGE_SMOOTH_Q, None) == bd.SAGE_ERR_UNSUPPORTED
    # 256-key tiles exist for MXFP4 only; rejected before any allocation or launch
    assert _attn(L, fmt=bd.SAGE_FMT_NV16_E4M3 | bd.SAGE_BKV256) == bd.SAGE_ERR_UNSUPPORTED
    assert L.sage_attn_fp4_fwd_prequant(FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 1, 1, 128, 128, 0,
                                        bd.SAGE_FMT_NV16_E4M3 | bd.SAGE_BKV256, None) == bd.SAGE_ERR_UNSUPPORTED


def test_smooth_q_workspace_and_quant_arguments(L):
    B, H, N, D = 2, 3, 300, 128
    nqb, Np = 3, 384
    extra = L.sage_attn_fp4_workspace_size(B, H, N, D, bd.SAGE_SMOOTH_Q) - L.sage_attn_fp4_workspace_size(B, H, N, D, 0)
    # block means [B,H,nqb,D] and the GEMV bias [B,H,nqb,Np], each rounded up to 256 bytes
    assert extra >= B * H * nqb * (D + Np) * 4 and extra < B * H * nqb * (D + Np) * 4 + 512
    # role Q with smoothing Q needs the mean output; role Q without it must not get one
    assert L.sage_quant_fp4(FAKE, 0, 1, 1, 128, 128, bd.SAGE_SMOOTH_Q, FAKE, FAKE, None, None, 0,
                            None) == bd.SAGE_ERR_INVALID_ARG
    assert L.sage_quant_fp4(FAKE, 0, 1, 1, 128, 128, 0, FAKE, FAKE, FAKE, None, 0, None) == bd.SAGE_ERR_INVALID_ARG


def test_quant_sizes_and_validation(L):
    c, s = bd.quant_sizes(bd.SAGE_ROLE_Q, 2, 3, 100, 128, 0)
    assert (c, s) == (2 * 3 * 100 * 64, 2 * 3 * 100 * 4)
    c, s = bd.quant_sizes(bd.SAGE_ROLE_K, 2, 3, 100, 128, 1)
    assert (c, s) == (2 * 3 * 128 * 64, 2 * 3 * 128 * 8)
    c, s = bd.quant_sizes(bd.SAGE_ROLE_V, 1, 1, 300, 64, 0)
    assert (c, s) == (64 * 384 // 2, 64 * 384 // 32)
    assert L.sage_quant_workspace_size(1, 1, 2, 1000, 128, 0) == 2 * 2 * 128 * 8
    assert L.sage_quant_workspace_size(0, 1, 2, 1000, 128, 0) == 0
    assert L.sage_quant_workspace_size(1, 1, 2, 1000, 128, bd.SAGE_NO_SMOOTH_K) == 0
    with pytest.raises(bd.SageError):
        bd.quant_sizes(3, 1, 1, 10, 128, 0)
    # role K with smoothing needs kmean and a workspace
    rc = L.sage_quant_fp4(FAKE, 1, 1, 1, 128, 128, 0, FAKE, FAKE, None, FAKE, 1 << 20, None)
    assert rc == bd.SAGE_ERR_INVALID_ARG
    rc = L.sage_quant_fp4(FAKE, 1, 1, 1, 1000, 128, 0, FAKE, FAKE, FAKE, FAKE, 8, None)
    assert rc == bd.SAGE_ERR_WORKSPACE
    # kmean must be NULL for other roles; misaligned input
    assert L.sage_quant_fp4(FAKE, 0, 1, 1, 128, 128, 0, FAKE, FAKE, FAKE, None, 0, None) == bd.SAGE_ERR_INVALID_ARG
    assert L.sage_quant_fp4(FAKE + 8, 0, 1, 1, 128, 128, 0, FAKE, FAKE, None, None, 0, None) == bd.SAGE_ERR_INVALID_ARG


def test_workspace_variant_validation(L):
    need = bd.attn_fp4_workspace_size(1, 2, 1000, 128, 0)
    assert need > 2 * 1000 * 64 * 3
    rc = L.sage_attn_fp4_fwd_ws(FAKE, FAKE, FAKE, FAKE, 1, 2, 1000, 128, 0, 0, FAKE, need - 1, None)
    assert rc == bd.SAGE_ERR_WORKSPACE
    rc = L.sage_attn_fp4_fwd_ws(FAKE, FAKE, FAKE, FAKE, 1, 2, 1000, 128, 0, 0, FAKE + 16, need, None)
    assert rc == bd.SAGE_ERR_INVALID_ARG


def test_prequant_and_bf16_validation(L):
    args = [FAKE] * 7 + [1, 1, 128, 128, 0, 0, None]
    bad = list(args)
    bad[3] = FAKE + 1
    assert L.sage_attn_fp4_fwd_prequant(*bad) == bd.SAGE_ERR_INVALID_ARG
    assert L.sage_attn_bf16_fwd(FAKE, FAKE, FAKE, FAKE, 1, 1, 128, 128, 0, 0, None) == bd.SAGE_ERR_INVALID_ARG
    assert L.sage_attn_bf16_fwd(FAKE, FAKE, FAKE, FAKE, 1, 1, 128, 128, 0, bd.SAGE_IN_BF16 | bd.SAGE_BKV64,
                                None) == bd.SAGE_ERR_INVALID_ARG


def test_int8_sizes_and_validation(L):
    B, H, N, D = 2, 3, 300, 128
    assert bd.quant_int8_sizes(bd.SAGE_ROLE_Q, B, H, N, D) == (B * H * N * D, B * H * 3 * 4)
    assert bd.quant_int8_sizes(bd.SAGE_ROLE_K, B, H, N, D) == (B * H * 384 * D, B * H * 3 * 4)
    assert bd.quant_int8_sizes(bd.SAGE_ROLE_V, B, H, N, D) == (B * H * D * 384, B * H * 3 * 4)
    # 64-key tiles: scale blocks of 64 rows
    assert bd.quant_int8_sizes(bd.SAGE_ROLE_K, B, H, N, D, bd.SAGE_BKV64) == (B * H * 384 * D, B * H * 6 * 4)
    # only the 16-bit dtype, fp32 output, no-smoothing-K and KV-tile bits are accepted
    for f in (bd.SAGE_FMT_NV16_E4M3, bd.SAGE_SMOOTH_Q, 0x80):
        with pytest.raises(bd.SageError):
            bd.quant_int8_sizes(bd.SAGE_ROLE_Q, 1, 1, 128, 128, f)
        assert L.sage_attn_int8_workspace_size(1, 1, 128, 128, f) == 0
        assert L.sage_attn_int8_fwd(FAKE, FAKE, FAKE, FAKE, None, 1, 1, 128, 128, 0, f, None) == bd.SAGE_ERR_INVALID_ARG
    ws = bd.attn_int8_workspace_size(1, 2, 1000, 128, bd.SAGE_BKV64)
    assert ws >= 2 * (1000 + 2 * 1024) * 128
    assert L.sage_attn_int8_fwd_ws(FAKE, FAKE, FAKE, FAKE, None, 1, 2, 1000, 128, 0, 0, FAKE, ws - 1,
                                   None) == bd.SAGE_ERR_WORKSPACE
    # shapes, pointers, alignment, causal
    for bad in (dict(D=96), dict(N=0), dict(causal=2), dict(q=None), dict(o=FAKE + 4), dict(lse=FAKE + 2)):
        a = dict(q=FAKE, o=FAKE, lse=None, D=128, N=128, causal=0)
        a.update(bad)
        rc = L.sage_attn_int8_fwd(a["q"], FAKE, FAKE, a["o"], a["lse"], 1, 1, a["N"], a["D"], a["causal"], 0, None)
        assert rc == bd.SAGE_ERR_INVALID_ARG, bad
    # role K with smoothing needs kmean and a large enough workspace; other roles take no kmean
    assert L.sage_quant_int8(FAKE, 1, 1, 1, 128, 128, 0, FAKE, FAKE, None, FAKE, 1 << 20,
                             None) == bd.SAGE_ERR_INVALID_ARG
    assert L.sage_quant_int8(FAKE, 1, 1, 1, 1000, 128, 0, FAKE, FAKE, FAKE, FAKE, 8, None) == bd.SAGE_ERR_WORKSPACE
    assert L.sage_quant_int8(FAKE, 2, 1, 1, 128, 128, 0, FAKE, FAKE, FAKE, None, 0, None) == bd.SAGE_ERR_INVALID_ARG
    assert L.sage_quant_int8(FAKE, 0, 1, 1, 128, 128, 0, FAKE, FAKE + 2, None, None, 0,
                             None) == bd.SAGE_ERR_INVALID_ARG
    pre = [FAKE] * 6 + [FAKE, None, 1, 1, 128, 128, 0, 0, None]
    bad = list(pre)
    bad[1] = FAKE + 2
    assert L.sage_attn_int8_fwd_prequant(*bad) == bd.SAGE_ERR_INVALID_ARG


def test_int8_bwd_validation(L):
    args = lambda **kw: [kw.get(n, FAKE) for n in ("q", "k", "v", "o", "lse", "do", "dq", "dk", "dv")]
    ok = args()
    assert L.sage_attn_int8_bwd_workspace_size(1, 2, 1000, 128, 0) > 2 * 1000 * 128 * 5
    assert L.sage_attn_int8_bwd_workspace_size(1, 2, 1000, 128, bd.SAGE_BKV64) == 0
    assert L.sage_attn_int8_bwd_workspace_size(1, 2, 1000, 96, 0) == 0
    assert L.sage_attn_int8_bwd(*ok, 1, 1, 128, 128, 0, bd.SAGE_BKV64, None) == bd.SAGE_ERR_UNSUPPORTED
    for f in (bd.SAGE_FMT_NV16_E4M3, bd.SAGE_SMOOTH_Q, 0x80):
        assert L.sage_attn_int8_bwd(*ok, 1, 1, 128, 128, 0, f, None) == bd.SAGE_ERR_INVALID_ARG
    for bad in (dict(q=None), dict(lse=None), dict(dv=None), dict(o=FAKE + 4), dict(do=FAKE + 8), dict(lse=FAKE + 2)):
        assert L.sage_attn_int8_bwd(*args(**bad), 1, 1, 128, 128, 0, 0, None) == bd.SAGE_ERR_INVALID_ARG, bad
    assert L.sage_attn_int8_bwd(*ok, 1, 1, 128, 128, 2, 0, None) == bd.SAGE_ERR_INVALID_ARG
    need = L.sage_attn_int8_bwd_min_workspace_size(1, 1, 128, 128, 0)
    assert L.sage_attn_int8_bwd_ws(*ok, 1, 1, 128, 128, 0, 0, FAKE, need - 1, None) == bd.SAGE_ERR_WORKSPACE
    # the recommended size adds the stored dS^ state of every head: codes of
    # every (query block, KV block) pair, one s_dS per pair, row sums per pair
    for B, H, N, D in ((1, 2, 1000, 128), (2, 3, 300, 64), (1, 1, 1, 128)):
        lo = L.sage_attn_int8_bwd_min_workspace_size(B, H, N, D, 0)
        hi = L.sage_attn_int8_bwd_workspace_size(B, H, N, D, 0)
        nb = (N + 127) // 128
        assert 0 < lo < hi and hi - lo == B * H * (nb * nb * (16384 + 4) + nb * nb * 128 * 4)
    assert L.sage_attn_int8_bwd_min_workspace_size(1, 2, 1000, 96, 0) == 0
    assert L.sage_attn_int8_bwd_min_workspace_size(1, 2, 1000, 128, bd.SAGE_BKV64) == 0
    # the stored state is capped at 64 GiB: at 32 heads of 65536 tokens only 15 heads fit
    per = 512 * 512 * (16384 + 4) + 512 * 65536 * 4
    lo = L.sage_attn_int8_bwd_min_workspace_size(1, 32, 65536, 128, 0)
    assert L.sage_attn_int8_bwd_workspace_size(1, 32, 65536, 128, 0) - lo == ((64 << 30) // per) * per


def test_product_path_does_not_import_oracle():
    import paper_2505_11594_amd
    pkg = os.path.dirname(paper_2505_11594_amd.__file__)
    for root, _, files in os.walk(pkg):
        for f in files:
            if f.endswith((".py", ".hip", ".h", ".cpp")):
                src = open(os.path.join(root, f)).read()
                assert "import oracle" not in src and "from oracle" not in src and "sage_oracle" not in src, f


def test_per_head_size_limit(L):
    """One head may hold Np * D <= 2^31 elements: the largest accepted N at
    D = 128 is 2^24, at D = 64 2^25; one token more is rejected by every size
    query."""
    for D, nmax in ((128, 1 << 24), (64, 1 << 25)):
        assert L.sage_attn_fp4_workspace_size(1, 1, nmax, D, 0) > 0
        assert L.sage_attn_fp4_workspace_size(1, 1, nmax + 1, D, 0) == 0
        assert L.sage_attn_int8_workspace_size(1, 1, nmax, D, 0) > 0
        assert L.sage_attn_int8_workspace_size(1, 1, nmax + 1, D, 0) == 0
        assert bd.attn_int8_bwd_min_workspace_size(1, 1, nmax + 1, D) == 0


def test_wg256_only_where_implemented(L):
    """256-query workgroups need MXFP4 with 256-key tiles, non-causal, no smoothing Q."""
    W, B256 = bd.SAGE_WG256, bd.SAGE_BKV256
    assert _attn(L, fmt=W) == bd.SAGE_ERR_UNSUPPORTED                                  # 128-key tiles
    assert _attn(L, fmt=W | bd.SAGE_BKV64) == bd.SAGE_ERR_UNSUPPORTED
    assert _attn(L, fmt=W | B256, causal=1) == bd.SAGE_ERR_UNSUPPORTED
    assert _attn(L, fmt=W | B256 | bd.SAGE_SMOOTH_Q) == bd.SAGE_ERR_UNSUPPORTED
    assert _attn(L, fmt=W | B256 | bd.SAGE_FMT_NV16_E4M3) == bd.SAGE_ERR_UNSUPPORTED
    args = [FAKE] * 7 + [1, 1, 128, 128]
    assert L.sage_attn_fp4_fwd_prequant(*args, 1, W | B256, None) == bd.SAGE_ERR_UNSUPPORTED
    assert L.sage_attn_fp4_fwd_prequant(*args, 0, W, None) == bd.SAGE_ERR_UNSUPPORTED
