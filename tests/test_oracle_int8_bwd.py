"""Pins for the oracle of the 8-bit attention backward (Algorithm 3), no GPU.

- identity mode (no psi anywhere) against central finite differences of
  textbook fp64 softmax attention: the gradients of sum(O * dO) with respect
  to Q, K and V, including the smoothing-K term of dQ;
- closed forms: dO = 0 gives zero gradients; doubling dO doubles every
  gradient bit for bit (psi is equivariant under powers of two and every
  step is linear in dO);
- permuting whole query blocks (with dO, O and L) permutes dQ and leaves dK,
  dV unchanged up to the fp32 order of accumulation;
- the paper's claims: the quantized gradients stay close to the exact ones,
  and keeping dP = dO V^T in 16-bit is more accurate for dQ than INT8
  (Table 1(c)).
"""
import math

import numpy as np
import pytest

import oracle
from paper_2505_11594_amd import workloads as wl


def textbook_forward(q, k, v, causal):
    S = q @ k.T / math.sqrt(q.shape[1])
    if causal:
        S = np.where(np.tril(np.ones_like(S, dtype=bool)), S, -np.inf)
    P = np.exp(S - S.max(axis=1, keepdims=True))
    P /= P.sum(axis=1, keepdims=True)
    return P @ v


def fd_gradients(q, k, v, do, causal, h=1e-5):
    """Central differences of sum(O * dO) in fp64."""
    grads = []
    for which in range(3):
        base = [q.copy(), k.copy(), v.copy()]
        g = np.zeros_like(base[which])
        for idx in np.ndindex(g.shape):
            xp = [b.copy() for b in base]
            xm = [b.copy() for b in base]
            xp[which][idx] += h
            xm[which][idx] -= h
            g[idx] = ((textbook_forward(*xp, causal) - textbook_forward(*xm, causal)) * do).sum() / (2 * h)
        grads.append(g)
    return grads


def small_case(N, D, seed, k_bias_var=1.0):
    q, k, v = wl.make_inputs(1, 1, N, D, wl.IN_BF16, seed=seed, k_bias_var=k_bias_var)
    rng = np.random.default_rng(seed + 1)
    do = wl.to_bits(rng.standard_normal((1, 1, N, D)).astype(np.float32), 1)
    return q, k, v, do


@pytest.mark.parametrize("causal", [False, True])
@pytest.mark.parametrize("smooth", [True, False])
def test_identity_mode_matches_finite_differences(causal, smooth):
    N, D, bq, bkv = 20, 16, 8, 4
    q, k, v, do = small_case(N, D, seed=900 + causal)
    fl = oracle.I8_IDENTITY | (0 if smooth else oracle.NO_SMOOTH_K)
    o, lse, _, _ = oracle.attn_int8(q, k, v, 1, causal, bkv, flags=fl, bq=bq)
    dq, dk, dv = oracle.attn_int8_bwd(q, k, v, do, o, lse, 1, causal, bkv, flags=fl, bq=bq, tolerance=False)
    qf, kf, vf, gf = (wl.from_bits(x[0, 0], 1).astype(np.float64) for x in (q, k, v, do))
    gq, gk, gv = fd_gradients(qf, kf, vf, gf, causal)
    for got, ref in ((dq, gq), (dk, gk), (dv, gv)):
        assert np.abs(got[0, 0] - ref).max() <= 2e-5 * (1 + np.abs(ref).max())


def quantized_case(N=300, D=64, seed=910, causal=False, bkv=64, k_bias_var=1.0):
    q, k, v, do = small_case(N, D, seed, k_bias_var)
    o, lse, _, _ = oracle.attn_int8(q, k, v, 1, causal, bkv)
    return q, k, v, do, o.reshape(1, 1, N, D), lse.reshape(1, 1, N)


def test_zero_do_gives_zero_gradients():
    q, k, v, do, o, lse = quantized_case()
    z = np.zeros_like(do)
    dq, dk, dv = oracle.attn_int8_bwd(q, k, v, z, o, lse, 1, False, 64, tolerance=False)
    assert not dq.any() and not dk.any() and not dv.any()


@pytest.mark.parametrize("causal", [False, True])
def test_doubling_do_doubles_every_gradient_exactly(causal):
    q, k, v, do, o, lse = quantized_case(causal=causal)
    d2 = wl.to_bits(wl.from_bits(do, 1) * np.float32(2.0), 1)
    a = oracle.attn_int8_bwd(q, k, v, do, o, lse, 1, causal, 64, tolerance=False)
    b = oracle.attn_int8_bwd(q, k, v, d2, o, lse, 1, causal, 64, tolerance=False)
    for x, y in zip(a, b):
        assert np.array_equal(2 * x, y)


def test_permuting_query_blocks():
    N, bq = 512, 128
    q, k, v, do, o, lse = quantized_case(N=N)
    perm = np.concatenate([b * bq + np.arange(bq) for b in (2, 0, 3, 1)])
    a = oracle.attn_int8_bwd(q, k, v, do, o, lse, 1, False, 64, tolerance=False)
    b = oracle.attn_int8_bwd(q[:, :, perm], k, v, do[:, :, perm], o[:, :, perm], lse[:, :, perm], 1, False, 64,
                             tolerance=False)
    assert np.array_equal(a[0][:, :, perm], b[0])
    for x, y in ((a[1], b[1]), (a[2], b[2])):
        assert np.abs(x - y).max() <= 1e-5 * np.abs(x).max()


def exact_gradients(q, k, v, do, causal):
    qf, kf, vf, gf = (wl.from_bits(x[0, 0], 1).astype(np.float64) for x in (q, k, v, do))
    D = qf.shape[1]
    S = qf @ kf.T / math.sqrt(D)
    if causal:
        S = np.where(np.tril(np.ones_like(S, dtype=bool)), S, -np.inf)
    P = np.exp(S - S.max(axis=1, keepdims=True))
    P /= P.sum(axis=1, keepdims=True)
    O = P @ vf
    dP = gf @ vf.T
    dS = P * (dP - (gf * O).sum(axis=1, keepdims=True))
    return dS @ kf / math.sqrt(D), dS.T @ qf / math.sqrt(D), P.T @ gf


def cos(a, b):
    a, b = a.ravel().astype(np.float64), b.ravel().astype(np.float64)
    return float(a @ b / (np.linalg.norm(a) * np.linalg.norm(b)))


@pytest.mark.parametrize("causal", [False, True])
def test_quantized_gradients_close_to_exact(causal):
    q, k, v, do, o, lse = quantized_case(N=512, D=128, causal=causal)
    dq, dk, dv = oracle.attn_int8_bwd(q, k, v, do, o, lse, 1, causal, 64, tolerance=False)
    gq, gk, gv = exact_gradients(q, k, v, do, causal)
    for got, ref in ((dq, gq), (dk, gk), (dv, gv)):
        assert cos(got[0, 0], ref) > 0.99


def test_fp16_dp_beats_int8_dp_for_dq():
    """Table 1(c): quantizing dO V^T to INT8 loses accuracy in dQ."""
    q, k, v, do, o, lse = quantized_case(N=512, D=128, seed=920)
    gq, _, _ = exact_gradients(q, k, v, do, False)
    a = oracle.attn_int8_bwd(q, k, v, do, o, lse, 1, False, 64, tolerance=False)[0]
    b = oracle.attn_int8_bwd(q, k, v, do, o, lse, 1, False, 64, flags=oracle.I8_DP_INT8, tolerance=False)[0]
    ea, eb = np.abs(a[0, 0] - gq).sum() / np.abs(gq).sum(), np.abs(b[0, 0] - gq).sum() / np.abs(gq).sum()
    assert cos(a[0, 0], gq) > cos(b[0, 0], gq) and ea < eb


@pytest.mark.parametrize("N,D", [(640, 128), (257, 64)])
@pytest.mark.parametrize("causal", [False, True])
def test_fused_order_p_within_tolerance_and_tightness(N, D, causal):
    """Algorithm 3 with P = exp(S - L) in the fused order a GPU uses
    (exp2(fma(acc, c_t, -Lb)) instead of exp2(fl32(u - Lb))) stays inside the
    plain-order tolerance, per element of dQ, dK and dV.  Reported per
    gradient: the largest observed difference over the tolerance at that
    element, where a code flipped (error above 2e-5 of max |grad|), and the
    median tolerance relative to max |grad| -- the tolerance's tightness."""
    # a K channel bias and 2% outlier rows: large scores make the two orders differ most
    q, k, v = wl.make_inputs(1, 2, N, D, wl.IN_BF16, seed=930 + N + causal, k_bias_var=4.0, outlier_frac=0.02)
    do = wl.to_bits(np.random.default_rng(931 + N).standard_normal((1, 2, N, D)).astype(np.float32), 1)
    o, lse, _, _ = oracle.attn_int8(q, k, v, 1, causal, 128)
    o, lse = o.reshape(1, 2, N, D), lse.reshape(1, 2, N)
    *a, tol = oracle.attn_int8_bwd(q, k, v, do, o, lse, 1, causal, 128)
    f = oracle.attn_int8_bwd(q, k, v, do, o, lse, 1, causal, 128, flags=oracle.I8_FUSED_BWD, tolerance=False)
    for name, x, y, t in zip(("dQ", "dK", "dV"), a, f, tol):
        err = np.abs(x - y)
        floor = 2e-5 * np.abs(x).max()
        assert np.all(err <= t + floor), name
        flip = err > floor
        ratio = float((err[flip] / t[flip]).max()) if flip.any() else 0.0
        print("%s causal=%d: %d elements moved beyond 2e-5 of max|%s|, worst move / tolerance there %.3f, "
              "median tolerance / max|%s| %.2g" % (name, causal, int(flip.sum()), name, ratio, name,
                                                   float(np.median(t) / np.abs(x).max())))
