"""Pins for the oracle's codecs (no GPU).

E2M1, E4M3 and E8M0 follow the paper's data-type section (Sec. 3.1, NVFP4 vs
MXFP4) and the value counts printed in the appendix analysis of two-level
quantization; everything here is checked against hand-worked values, the
bit-layout definitions, or an independent library cast.
"""
import os

import numpy as np
import pytest

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _rows(name):
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.split("#")[0].strip()
            if line:
                yield line.split()


def test_e2m1_decode_all_codes():
    vals = [0, .5, 1, 1.5, 2, 3, 4, 6]
    for c in range(16):
        v = oracle.e2m1_decode(c)
        expect = vals[c & 7] * (-1 if c & 8 else 1)
        assert v == expect
        assert np.signbit(v) == bool(c & 8)
    # {E2M1}_n = 8 non-negative values (appendix analysis)
    assert len({abs(oracle.e2m1_decode(c)) for c in range(16)}) == 8


def test_e2m1_encode_hand_worked_ties_and_saturation():
    for x, code in _rows("e2m1_rne.txt"):
        xf = np.float32(float(x))
        assert oracle.e2m1_encode(float(xf)) == int(code, 16), (x, code)


def test_e2m1_encode_is_nearest_with_even_ties():
    # brute force over a dense grid: the code's value is a nearest grid point,
    # and on exact ties the even code wins
    grid = np.array([0, .5, 1, 1.5, 2, 3, 4, 6])
    for y in np.linspace(0, 7, 7001).astype(np.float32):
        c = oracle.e2m1_encode(float(y))
        d = np.abs(grid - min(float(y), 6.0))
        best = np.flatnonzero(d == d.min())
        assert (c & 7) in best
        if best.size == 2:
            assert (c & 7) % 2 == 0


def test_e4m3_table_and_paper_counts():
    vals = [oracle.e4m3_decode(c) for c in range(0x7F)]
    assert all(b > a for a, b in zip(vals, vals[1:]))  # strictly increasing codes 0..0x7E
    assert np.isnan(oracle.e4m3_decode(0x7F))
    pins = {}
    codes = {}
    enc = []
    for row in _rows("e4m3_pins.txt"):
        a, b = row
        if a.startswith("0x"):
            codes[int(a, 16)] = float(b)
        elif a.startswith("count") or a.startswith("grid") or a.startswith("e2m1"):
            pins[a] = int(b)
        else:
            enc.append((float(a), int(b, 16)))
    for c, v in codes.items():
        assert oracle.e4m3_decode(c) == v
    nonneg = np.array(vals)
    assert int((nonneg <= 0.167).sum()) == pins["count_le_0.167"] == 35
    assert int((nonneg <= 448).sum()) == pins["count_le_448"] == 127
    assert nonneg.max() == 448.0
    assert pins["count_le_0.167"] * pins["e2m1_count"] == pins["grid_direct"] == 280
    assert pins["count_le_448"] * pins["e2m1_count"] == pins["grid_two_level"] == 1016
    for x, c in enc:
        assert oracle.e4m3_encode(float(np.float32(x))) == c, (x, c)


def test_e4m3_encode_matches_torch_cast_in_range():
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(0)
    xs = np.concatenate([rng.uniform(0, 448, 4000), np.exp(rng.uniform(np.log(1e-3), np.log(448), 4000)),
                         np.array([oracle.e4m3_decode(c) for c in range(1, 0x7E)]) * 1.0000001]).astype(np.float32)
    t = torch.from_numpy(xs).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    mine = np.array([oracle.e4m3_encode(float(x)) for x in xs], dtype=np.uint8)
    assert np.array_equal(mine, t)


def test_e8m0_rule_hand_cases_and_property():
    cases = {6.0: 0, 7.0: 1, 4.0: 0, 3.0: -1, 3.0000002: 0, 0.75: -3, 12.0: 1, 12.000001: 2, 1.0: -2}
    for a, e in cases.items():
        assert oracle.e8m0_exponent(float(np.float32(a))) == e, a
    assert oracle.e8m0_exponent(0.0) == -127
    rng = np.random.default_rng(1)
    for a in np.exp(rng.uniform(-60, 60, 5000)).astype(np.float32):
        e = oracle.e8m0_exponent(float(a))
        assert 6.0 * 2.0 ** e >= a > 3.0 * 2.0 ** e
    assert oracle.e8m0_decode(127) == 1.0 and oracle.e8m0_decode(0) == 2.0 ** -127


def test_widen_fp16_bf16_exact():
    torch = pytest.importorskip("torch")
    bits = np.arange(0, 65536, 7, dtype=np.uint16)
    f16 = bits.view(np.float16).astype(np.float32)
    bf = torch.from_numpy(bits.view(np.int16).copy()).view(torch.bfloat16).float().numpy()
    for i in range(0, bits.size, 97):
        b = int(bits[i])
        w16 = oracle.widen(b, oracle.IN_FP16)
        wbf = oracle.widen(b, oracle.IN_BF16)
        assert (np.isnan(w16) and np.isnan(f16[i])) or w16 == f16[i]
        assert (np.isnan(wbf) and np.isnan(bf[i])) or wbf == bf[i]


@pytest.mark.parametrize("fmt", [oracle.FMT_MX, oracle.FMT_NV16])
def test_phi_roundtrip_bound_and_exact_max(fmt):
    n = oracle.block_size(fmt)
    rng = np.random.default_rng(2 + fmt)
    for trial in range(300):
        x = (rng.standard_normal(n) * np.exp(rng.uniform(-8, 8))).astype(np.float32)
        if fmt == oracle.FMT_NV16:
            # keep amax / 6 inside the E4M3 normal range [2^-6, 448] (no saturation,
            # relative scale rounding <= 2^-4)
            x *= np.float32(np.clip(np.abs(x).max(), 6 * 2.0 ** -6, 6 * 400) / np.abs(x).max())
        codes, sb = oracle.phi_block(x, fmt)
        deq = oracle.dequant_block(codes, sb, fmt)
        s = oracle.e8m0_decode(sb) if fmt == oracle.FMT_MX else oracle.e4m3_decode(sb)
        # FP4 grid step at the block scale is at most 2 s (between 4 and 6): error <= s
        assert np.all(np.abs(x - deq) <= s * 1.0000001)
        # every dequantized value is a grid point times the scale, |.| <= 6 s
        assert np.all(np.abs(deq) <= 6 * s)
        assert np.all(np.sign(deq[deq != 0]) == np.sign(x[deq != 0]))
    # block max lands exactly on 6 when amax = 6 * 2^e (MX) or amax / 6 is an E4M3 value (NV16)
    x = rng.standard_normal(n).astype(np.float32)
    x[3] = 6.0 * (2.0 ** 5) if fmt == oracle.FMT_MX else 6.0 * 1.375
    x[:] = np.clip(x, -abs(x[3]), abs(x[3]))
    codes, sb = oracle.phi_block(x, fmt)
    assert codes[3] == 7
    assert oracle.dequant_block(codes, sb, fmt)[3] == x[3]


def test_phi_zero_block():
    for fmt in (oracle.FMT_MX, oracle.FMT_NV16):
        codes, sb = oracle.phi_block(np.zeros(oracle.block_size(fmt), np.float32), fmt)
        assert np.all(codes == 0)
        assert sb == (0 if fmt == oracle.FMT_MX else 0)


def test_fp4mm_brute_force():
    rng = np.random.default_rng(3)
    for fmt in (oracle.FMT_MX, oracle.FMT_NV16):
        n = oracle.block_size(fmt)
        M, Nn, K = 9, 7, 128
        ac = rng.integers(0, 16, (M, K), dtype=np.uint8)
        bc = rng.integers(0, 16, (Nn, K), dtype=np.uint8)
        if fmt == oracle.FMT_MX:
            as_ = rng.integers(120, 135, (M, K // n), dtype=np.uint8)
            bs = rng.integers(120, 135, (Nn, K // n), dtype=np.uint8)
            sv = lambda b: 2.0 ** (b.astype(np.float64) - 127)
        else:
            as_ = rng.integers(1, 0x7E, (M, K // n), dtype=np.uint8)
            bs = rng.integers(1, 0x7E, (Nn, K // n), dtype=np.uint8)
            tab = np.array([oracle.e4m3_decode(c) for c in range(256)])
            sv = lambda b: tab[b]
        C, inexact = oracle.fp4mm(ac, as_, bc, bs, fmt)
        assert inexact == 0
        tab2 = np.array([0, .5, 1, 1.5, 2, 3, 4, 6, -0., -.5, -1, -1.5, -2, -3, -4, -6])
        A = tab2[ac] * np.repeat(sv(as_), n, axis=1)
        Bm = tab2[bc] * np.repeat(sv(bs), n, axis=1)
        ref = (A @ Bm.T).astype(np.float32)   # fp64 matmul, exact here, rounded once
        assert np.array_equal(C, ref)
