"""GPU parity of the quantization kernels: bit-exact FP4 codes, scale bytes and
the smoothing-K mean against the oracle (phi of Sec. 3.1; smoothing K of
Algorithm 1; V blocked along tokens as in the appendix on transposing V)."""
import numpy as np
import pytest

import oracle
from paper_2505_11594_amd import binding as bd
from paper_2505_11594_amd import workloads as wl

from _gpu import to_dev, torch_dev, say
from _layout import q_logical, k_logical, v_logical

pytestmark = pytest.mark.gpu


def gpu_quant(x_bits, in_dtype, role, fmt, smooth=True):
    torch = torch_dev()
    x = to_dev(x_bits, in_dtype)
    f = fmt | (0 if smooth else bd.SAGE_NO_SMOOTH_K)
    codes, scales, kmean = bd.sage_quant_fp4(x, role, f)
    torch.cuda.synchronize()
    return codes.cpu().numpy(), scales.cpu().numpy(), (kmean.cpu().numpy() if kmean is not None else None)


def check_role(x_bits, in_dtype, role, fmt, smooth=True):
    B, H, N, D = x_bits.shape
    gc, gs, gmu = gpu_quant(x_bits, in_dtype, role, fmt, smooth)
    oc, os_, omu, inexact = oracle.quant(x_bits, in_dtype, role, fmt, smooth_k=smooth)
    if role == bd.SAGE_ROLE_Q:
        c, s = q_logical(gc, gs, B, H, N, D, fmt)
    elif role == bd.SAGE_ROLE_K:
        c, s, tc, ts = k_logical(gc, gs, B, H, N, D, fmt)
        assert np.all(tc == 0)
        assert np.all(ts == (127 if fmt == 0 else 0))
        if smooth:
            assert inexact == 0
            assert np.array_equal(gmu.view(np.uint32), omu.view(np.uint32))
    else:
        c, s, tc, ts = v_logical(gc, gs, B, H, N, D, fmt)
        assert np.all(tc == 0)
        assert np.all(ts == 0)
    nbad_c = int((c != oc).sum())
    nbad_s = int((s != os_).sum())
    assert nbad_c == 0 and nbad_s == 0, (role, fmt, nbad_c, nbad_s)


@pytest.mark.parametrize("fmt", [0, 1])
@pytest.mark.parametrize("role", [0, 1, 2])
@pytest.mark.parametrize("shape", [(1, 1, 1, 64), (1, 2, 31, 128), (2, 1, 100, 64), (1, 1, 129, 128),
                                   (1, 3, 300, 128), (1, 1, 640, 64)])
@pytest.mark.parametrize("in_dtype", [0, 1])
def test_quant_edge_shapes(fmt, role, shape, in_dtype):
    B, H, N, D = shape
    say("quant edge", shape, "role", role, "fmt", fmt, "dtype", in_dtype)
    q, k, v = wl.make_inputs(B, H, N, D, in_dtype, seed=100 + N + D, k_bias_var=4.0, outlier_frac=0.05)
    check_role((q, k, v)[role], in_dtype, role, fmt)


@pytest.mark.parametrize("fmt", [0, 1])
@pytest.mark.parametrize("role", [0, 1, 2])
def test_quant_special_values(fmt, role):
    """Rounding ties at every E2M1 midpoint, zeros, -0, saturation-scale
    magnitudes and tiny values, for both scale formats."""
    rng = np.random.default_rng(5)
    B, H, N, D = 1, 2, 256, 128
    x = rng.standard_normal((B, H, N, D)).astype(np.float32)
    mids = np.array([0.25, 0.75, 1.25, 1.75, 2.5, 3.5, 5.0, 6.0, 0.5, 4.0], np.float32)
    for t in range(0, N, 4):
        e = float(2.0 ** rng.integers(-6, 6))
        x[0, 0, t, :10] = mids * e
        x[0, 0, t, 10:20] = -mids * e
        x[0, 0, t, 31] = 6.0 * e               # block max exactly 6 * 2^e
    x[0, 1, :16] = 0.0                           # all-zero blocks
    x[0, 1, 16:32] = -0.0
    x[0, 1, 32:48] *= 3000.0                     # large magnitudes (E4M3 scale saturates above 2688)
    x[0, 1, 48:64] *= 2.0 ** -10                 # tiny magnitudes (E4M3 subnormal scales; K mean stays exact)
    bits = wl.to_bits(x, 1)
    check_role(bits, 1, role, fmt, smooth=(role != 1))
    check_role(bits, 1, role, fmt, smooth=True)


@pytest.mark.parametrize("ci", range(5))
def test_quant_configs_full_size(ci):
    """Bit-exact at the benchmark sizes (every element for the two smaller
    configurations; six whole heads of the larger ones)."""
    w = wl.CONFIGS[ci]
    say("quant config", ci, w.name)
    q, k, v = wl.generate(w)
    for fmt in w.fmts:
        for role, x in ((0, q), (1, k), (2, v)):
            if ci >= 2:
                gc, gs, gmu = gpu_quant(x, w.in_dtype, role, fmt)
                B, H, N, D = x.shape
                heads = sorted({0, B * H - 1} | set(np.random.default_rng(ci).choice(B * H, 4, replace=False).tolist()))
                xs = x.reshape(B * H, 1, N, D)[heads]
                oc, os_, omu, inexact = oracle.quant(np.ascontiguousarray(xs), w.in_dtype, role, fmt)
                if role == 0:
                    c, s = q_logical(gc, gs, B, H, N, D, fmt)
                elif role == 1:
                    c, s, _, _ = k_logical(gc, gs, B, H, N, D, fmt)
                    assert inexact == 0
                    assert np.array_equal(gmu.reshape(B * H, D)[heads].view(np.uint32), omu.reshape(len(heads), D).view(np.uint32))
                else:
                    c, s, _, _ = v_logical(gc, gs, B, H, N, D, fmt)
                c = c.reshape((B * H,) + c.shape[2:])[heads]
                s = s.reshape((B * H,) + s.shape[2:])[heads]
                assert np.array_equal(c, oc.reshape(c.shape)), (ci, role, fmt)
                assert np.array_equal(s, os_.reshape(s.shape)), (ci, role, fmt)
            else:
                check_role(x, w.in_dtype, role, fmt)


@pytest.mark.parametrize("fmt", [0, 1])
def test_quant_work_split_ragged(fmt):
    """The V quantizer walks contiguous ranges of (head, 128-token tile), one
    workgroup per CU: 409 heads x 10 tiles = 4090 tiles make, on 256 CUs, 16
    tiles per workgroup, a grid of 256 (so the XCD remap is on) and a last
    workgroup with 10; the last tile of every head is partial (N = 1270).  The
    K quantizer's steps of four units per thread end inside a workgroup's
    range.  Every code, scale and the mean against the oracle, all roles."""
    B, H, N, D = 1, 409, 1270, 64
    say("quant work split", (B, H, N, D), "fmt", fmt)
    q, k, v = wl.make_inputs(B, H, N, D, 1, seed=4090 + fmt, k_bias_var=4.0, outlier_frac=0.02)
    for role, x in ((0, q), (1, k), (2, v)):
        check_role(x, 1, role, fmt)
