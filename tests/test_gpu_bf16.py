"""GPU check of the bf16-MFMA comparison kernel (FlashAttention forward,
Sec. 2) against the definition: fp64 softmax(Q K^T / sqrt(D)) V.

Tolerance from the arithmetic: the only rounding beyond fp32 is P to bf16
(relative error <= 2^-9 per probability), which moves both the weighted sum
and the normaliser, so |O - O_exact| <= 2^-8 max|V| per row; fp32 scores and
accumulation add about 1e-5."""
import numpy as np
import pytest

import oracle
from paper_2505_11594_amd import binding as bd
from paper_2505_11594_amd import workloads as wl

from _gpu import to_dev, torch_dev, say

pytestmark = pytest.mark.gpu


def run(q, k, v, causal, out_f32=True):
    torch = torch_dev()
    o = bd.sage_attn_bf16_fwd(to_dev(q, 1), to_dev(k, 1), to_dev(v, 1), causal=causal, out_f32=out_f32)
    torch.cuda.synchronize()
    return o


def check(got, ex, v_rows_max, label):
    err = np.abs(got - ex).max(axis=1)
    lim = 2.0 ** -8 * v_rows_max + 2e-5
    say("%s: rows=%d max_err=%.3g max_ratio=%.3f" % (label, len(err), float(err.max()), float((err / lim).max())))
    assert np.all(err <= lim), label


@pytest.mark.parametrize("N", [1, 64, 100, 257, 700])
@pytest.mark.parametrize("D", [64, 128])
@pytest.mark.parametrize("causal", [False, True])
def test_bf16_edge_shapes(N, D, causal):
    q, k, v = wl.make_inputs(1, 2, N, D, 1, seed=300 + N, k_bias_var=1.0)
    o = run(q, k, v, causal).cpu().numpy().reshape(-1, D)
    ex = oracle.exact_attn(q, k, v, 1, causal)
    vmax = np.abs(wl.from_bits(v, 1)).max()
    check(o, ex, np.full(o.shape[0], vmax), "bf16 edge")


@pytest.mark.parametrize("ci", [1, 2, 3])
def test_bf16_configs_sampled_rows(ci):
    torch = torch_dev()
    w = wl.CONFIGS[ci]
    q, k, v = wl.generate(w)
    o = run(q, k, v, w.causal)
    BH = w.B * w.H
    heads = sorted({0, BH - 1} | set(np.random.default_rng(ci).choice(BH, min(BH, 4), replace=False).tolist()))
    rows = wl.sample_rows(w, per_head_tiles=3, tile=128, rows_per_tile=8, heads=heads, seed=ci)
    got = o.reshape(-1, w.D).index_select(0, torch.from_numpy(rows).to(o.device)).cpu().numpy()
    ex = oracle.exact_attn(q, k, v, 1, w.causal, rows=rows)
    vmax = np.abs(wl.from_bits(v, 1)).max()
    check(got, ex, np.full(got.shape[0], vmax), w.name)
    say("bf16 accuracy vs exact", oracle.metrics(ex, got))


def test_bf16_16bit_output_and_rejects_fp16():
    torch = torch_dev()
    q, k, v = wl.make_inputs(1, 1, 300, 128, 1, seed=41)
    o = run(q, k, v, False, out_f32=False)
    assert o.dtype == torch.bfloat16
    ex = oracle.exact_attn(q, k, v, 1, False)
    vmax = np.abs(wl.from_bits(v, 1)).max()
    err = np.abs(o.float().cpu().numpy().reshape(-1, 128) - ex).max()
    assert err <= 2.0 ** -8 * vmax + np.abs(ex).max() * 2.0 ** -8
    q16 = to_dev(q, 0)
    with pytest.raises(bd.SageError):
        bd.sage_attn_bf16_fwd(q16, q16, q16)
