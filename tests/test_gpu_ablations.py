"""The paper's accuracy orderings on the HIP kernels' own outputs (against
exact fp64 attention on sampled rows): Table 1(a), NVFP4-style E4M3 scales
beat MXFP4; the smoothing ablation, smoothing K beats no smoothing when K
carries a channel bias.  The oracle side of the same ablations is pinned in
test_oracle_ablations and test_oracle_attn."""
import numpy as np
import pytest

import oracle
from paper_2505_11594_amd import binding as bd
from paper_2505_11594_amd import workloads as wl

from _gpu import to_dev, torch_dev, say

pytestmark = pytest.mark.gpu

B, H, N, D = 1, 2, 2048, 128


def _inputs():
    return wl.make_inputs(B, H, N, D, wl.IN_BF16, seed=600, k_bias_var=4.0)


def _gpu_metrics(q, k, v, flags, rows, ex):
    torch = torch_dev()
    o = bd.sage_attn_fp4_fwd(to_dev(q, 1), to_dev(k, 1), to_dev(v, 1), fmt=flags)
    torch.cuda.synchronize()
    return oracle.metrics(ex, o.cpu().numpy().reshape(-1, D)[rows])


def test_gpu_nv16_beats_mxfp4_and_smoothing_k_helps():
    q, k, v = _inputs()
    rows = np.arange(0, B * H * N, 4, dtype=np.int64)
    ex = oracle.exact_attn(q, k, v, wl.IN_BF16, False, rows=rows)
    mx = _gpu_metrics(q, k, v, bd.SAGE_FMT_MXFP4, rows, ex)
    nv = _gpu_metrics(q, k, v, bd.SAGE_FMT_NV16_E4M3, rows, ex)
    mx_ns = _gpu_metrics(q, k, v, bd.SAGE_FMT_MXFP4 | bd.SAGE_NO_SMOOTH_K, rows, ex)
    nv_ns = _gpu_metrics(q, k, v, bd.SAGE_FMT_NV16_E4M3 | bd.SAGE_NO_SMOOTH_K, rows, ex)
    say("mx", mx, "nv16", nv, "mx no-smooth-K", mx_ns, "nv16 no-smooth-K", nv_ns)
    assert nv["cossim"] > mx["cossim"] and nv["l1"] < mx["l1"] and nv["rmse"] < mx["rmse"]
    for a, b in ((mx, mx_ns), (nv, nv_ns)):
        assert a["cossim"] > b["cossim"] and a["l1"] < b["l1"] and a["rmse"] < b["rmse"]
