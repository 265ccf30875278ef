"""Hardware probes (gfx950): the semantics the attention kernels rely on,
checked against independent CPU definitions.

- v_cvt_scalef32_pk_fp4_f32 against the oracle's E2M1 encoder (nearest even,
  saturation at +-6, sign of zero kept) on every fp32 multiple of 1/64 in
  (-16, 16), ties included, and with power-of-two scales;
- v_exp_f32 against the correctly rounded exp2 over the arguments the kernels
  use: its error must stay within the 8-ulp window inside which the oracle
  treats an FP4 or INT8 code of P as tie-ambiguous; and it must never decrease
  its output as its argument grows, on every fp32 in [-130, 0];
- v_cvt_pk_u8_f32 against rint with clamping to [0, 255];
- v_cvt_pk_fp8_f32 / v_cvt_f32_fp8 against the oracle's E4M3 codec (the NV16
  kernel encodes and decodes its second-level P scales with them), on every
  rounding midpoint of [0, 448] and a sweep of the range;
- v_cvt_scalef32_pk_bf16_fp4: it applies only the power-of-two part of its
  scale operand, so an E4M3 scale cannot be folded into it;
- the register layouts of the FP4 block-scaled, int8 and bf16 32x32 MFMAs
  against numpy products (and, for FP4, the oracle's exact FP4MM).
"""
import ctypes
import os

import numpy as np
import pytest

import oracle
from paper_2505_11594_amd import build as hipbuild
from paper_2505_11594_amd import workloads as wl

from _gpu import torch_dev

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def P():
    torch_dev()          # torch's HIP runtime first: the library binds to the runtime loaded first
    if not os.path.exists(hipbuild.PROBES_LIB):
        pytest.fail("libsage_probes.so is not built")
    L = ctypes.CDLL(hipbuild.PROBES_LIB)
    vp = ctypes.c_void_p
    L.sage_probe_cvt_fp4.argtypes = [vp, vp, ctypes.c_int, ctypes.c_float, vp]
    L.sage_probe_exp2.argtypes = [vp, vp, ctypes.c_int, vp]
    L.sage_probe_cvt_u8.argtypes = [vp, vp, ctypes.c_int, vp]
    L.sage_probe_cvt_fp8.argtypes = [vp, vp, ctypes.c_int, vp, vp]
    L.sage_probe_cvt_bf16_fp4.argtypes = [vp, vp, vp, ctypes.c_int, vp]
    L.sage_probe_mfma_fp4.argtypes = [vp] * 6
    L.sage_probe_mfma_i8.argtypes = [vp] * 4
    L.sage_probe_mfma_bf16.argtypes = [vp] * 4
    return L


def dptr(t):
    return ctypes.c_void_p(t.data_ptr())


def run(fn, *args):
    torch = torch_dev()
    assert fn(*args, ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)) == 0
    torch.cuda.synchronize()


@pytest.mark.parametrize("e", [0, -3, 5])
def test_cvt_fp4_matches_the_e2m1_definition(P, e):
    torch = torch_dev()
    x = (np.arange(-1023, 1024, dtype=np.float64) / 64.0 * 2.0 ** e).astype(np.float32)   # ties at k/4 included
    x = np.concatenate([x, np.array([-0.0, 0.0, 100.0 * 2.0 ** e, -7.0 * 2.0 ** e], dtype=np.float32)])
    if x.size % 2:
        x = np.concatenate([x, np.array([1.0], dtype=np.float32)])
    xd = torch.from_numpy(x).cuda()
    cd = torch.empty(x.size, dtype=torch.uint8, device="cuda")
    run(P.sage_probe_cvt_fp4, dptr(xd), dptr(cd), x.size, np.float32(2.0 ** e))
    got = cd.cpu().numpy()
    ref = np.array([oracle.e2m1_encode(float(v) * 2.0 ** -e) for v in x], dtype=np.uint8)
    assert np.array_equal(got, ref)


def test_exp2_error_within_the_tie_window(P):
    torch = torch_dev()
    rng = np.random.default_rng(7)
    x = np.concatenate([rng.uniform(-130.0, 0.0, 1 << 20), rng.uniform(-1.0, 8.0, 1 << 18),
                        np.linspace(-126.0, 3.0, 1 << 16)]).astype(np.float32)
    xd = torch.from_numpy(x).cuda()
    yd = torch.empty_like(xd)
    run(P.sage_probe_exp2, dptr(xd), dptr(yd), x.size)
    y = yd.cpu().numpy().astype(np.float64)
    ref = np.exp2(x.astype(np.float64))
    normal = ref >= 2.0 ** -126
    ulp = np.spacing(ref[normal].astype(np.float32)).astype(np.float64)
    err = np.abs(y[normal] - ref[normal]) / ulp
    assert err.max() <= 2.0, err.max()          # the oracle's tie window is 8 ulp


def test_exp2_is_monotone_on_every_fp32_in_minus130_0(P):
    # the 8-bit backward's dV kernel takes the block maximum of P = exp2(arg) as
    # exp2 of the block maximum of arg: exact when v_exp_f32 never decreases
    torch = torch_dev()
    top = int(np.float32(130.0).view(np.int32))            # bit patterns 0 .. |-130| of the magnitude
    chunk = 1 << 27
    prev = None
    for start in range(0, top + 1, chunk):
        n = min(chunk, top + 1 - start)
        mag = torch.arange(start, start + n, dtype=torch.int32, device="cuda").view(torch.float32)
        xd = (-mag).contiguous()                            # -0, then decreasing to -130
        yd = torch.empty_like(xd)
        run(P.sage_probe_exp2, dptr(xd), dptr(yd), n)
        assert bool((yd[1:] <= yd[:-1]).all()), "exp2 increases somewhere in chunk %d" % (start // chunk)
        if prev is not None:
            assert float(yd[0]) <= prev
        prev = float(yd[-1])
        del mag, xd, yd
    assert prev == 0.0 or prev < 2.0 ** -126


def test_cvt_pk_u8_rounds_to_nearest_even_and_clamps(P):
    # the 8-bit forward forms its P codes rint(127 2^{u-t}) with this convert
    torch = torch_dev()
    x = np.arange(-64, 4160, dtype=np.float64) / 16.0                  # -4 .. 260 in steps of 1/16, ties included
    x = np.concatenate([x, [0.49999997, 0.50000006, 126.49999, 126.5, 127.5, 254.5, 255.49998, 1e6, -1e6, -0.0]])
    x = x.astype(np.float32)
    xd = torch.from_numpy(x).cuda()
    yd = torch.empty(x.size, dtype=torch.uint8, device="cuda")
    run(P.sage_probe_cvt_u8, dptr(xd), dptr(yd), x.size)
    want = np.clip(np.rint(x.astype(np.float64)), 0, 255).astype(np.uint8)   # numpy rint: nearest even
    assert np.array_equal(yd.cpu().numpy(), want)


def fp4_case(seed, lo, hi):
    rng = np.random.default_rng(seed)
    a = rng.integers(0, 16, (32, 64)).astype(np.uint8)
    b = rng.integers(0, 16, (32, 64)).astype(np.uint8)
    as_ = rng.integers(lo, hi, (32, 2)).astype(np.uint8)
    bs = rng.integers(lo, hi, (32, 2)).astype(np.uint8)
    return a, as_, b, bs


def gpu_fp4mm(P, a, as_, b, bs):
    torch = torch_dev()
    ad, bd_, asd, bsd = (torch.from_numpy(np.ascontiguousarray(t)).cuda() for t in (a, b, as_, bs))
    cd = torch.empty((32, 32), dtype=torch.float32, device="cuda")
    run(P.sage_probe_mfma_fp4, dptr(ad), dptr(asd), dptr(bd_), dptr(bsd), dptr(cd))
    return cd.cpu().numpy()


def exact_fp4mm(a, as_, b, bs):
    """fp64 value of the block-scaled product (exact here: every term is a
    small integer times a power of two in the fp64 range)."""
    dec = np.array([oracle.e2m1_decode(i) for i in range(16)])
    A, B = dec[a], dec[b]
    out = np.zeros((32, 32))
    for blk in range(2):
        sa = 2.0 ** (as_[:, blk].astype(np.float64) - 127)
        sb = 2.0 ** (bs[:, blk].astype(np.float64) - 127)
        out += (A[:, 32 * blk:32 * blk + 32] @ B[:, 32 * blk:32 * blk + 32].T) * sa[:, None] * sb[None, :]
    return out


def test_mfma_fp4_layout_and_scales(P):
    # scales within 2^(+-3): every sum is exact in fp32, so any summation order gives the oracle's value
    a, as_, b, bs = fp4_case(8, 124, 131)
    ref, inexact = oracle.fp4mm(a, as_, b, bs, oracle.FMT_MX)
    ex = exact_fp4mm(a, as_, b, bs)
    assert inexact == 0 and np.array_equal(ex.astype(np.float32).astype(np.float64), ex)
    assert np.array_equal(gpu_fp4mm(P, a, as_, b, bs), ref)


def test_mfma_fp4_wide_scales_are_faithful(P):
    # scales 2^(-7..6) per operand: some sums of the two blocks need a rounding
    a, as_, b, bs = fp4_case(8, 120, 134)
    ex = exact_fp4mm(a, as_, b, bs)
    c = gpu_fp4mm(P, a, as_, b, bs).astype(np.float64)
    rne = ex.astype(np.float32).astype(np.float64)
    need = rne != ex
    assert need.sum() > 0
    assert np.array_equal(c[~need], ex[~need])
    lo = np.where(rne <= ex, rne, np.nextafter(rne.astype(np.float32), np.float32(-np.inf)).astype(np.float64))
    hi = np.where(rne >= ex, rne, np.nextafter(rne.astype(np.float32), np.float32(np.inf)).astype(np.float64))
    off = need & (c != rne)
    print(f"fp4 mfma: {need.sum()} sums need rounding, {off.sum()} differ from nearest-even;"
          f" toward zero {np.sum(off & (np.abs(c) < np.abs(ex)))}; max |err|/ulp"
          f" {np.max(np.abs(c - ex)[need] / (hi - lo)[need]):.3g}", flush=True)
    assert np.all((c == lo) | (c == hi)), "not faithfully rounded"


def test_mfma_int8_layout(P):
    torch = torch_dev()
    rng = np.random.default_rng(9)
    a = rng.integers(-127, 128, (32, 32)).astype(np.int8)
    b = rng.integers(-127, 128, (32, 32)).astype(np.int8)
    ad, bd_ = torch.from_numpy(a).cuda(), torch.from_numpy(b).cuda()
    cd = torch.empty((32, 32), dtype=torch.int32, device="cuda")
    run(P.sage_probe_mfma_i8, dptr(ad), dptr(bd_), dptr(cd))
    assert np.array_equal(cd.cpu().numpy(), a.astype(np.int64) @ b.astype(np.int64).T)


def test_mfma_bf16_layout(P):
    torch = torch_dev()
    rng = np.random.default_rng(10)
    a = wl.to_bits(rng.integers(-8, 9, (32, 16)).astype(np.float32) / 4, 1)   # small exact values
    b = wl.to_bits(rng.integers(-8, 9, (32, 16)).astype(np.float32) / 4, 1)
    ad = torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).cuda()
    bd_ = torch.from_numpy(np.ascontiguousarray(b).view(np.int16)).cuda()
    cd = torch.empty((32, 32), dtype=torch.float32, device="cuda")
    run(P.sage_probe_mfma_bf16, dptr(ad), dptr(bd_), dptr(cd))
    af, bf = wl.from_bits(a, 1).astype(np.float64), wl.from_bits(b, 1).astype(np.float64)
    assert np.array_equal(cd.cpu().numpy(), (af @ bf.T).astype(np.float32))


def e4m3_values():
    return np.array([oracle.e4m3_decode(c) for c in range(127)], dtype=np.float64)


def test_cvt_fp8_matches_the_e4m3_definition(P):
    """Every midpoint between neighbouring E4M3 values (and 3 ulp either side),
    a strided sweep of [2^-12, 460], zero and the saturation region [448, 460]:
    the hardware byte equals the oracle's encoder (nearest even, saturation at
    448); every code decodes to the oracle's value."""
    torch = torch_dev()
    vals = e4m3_values()
    xs = []
    for m in (vals[:-1] + vals[1:]) / 2:
        b = int(np.float32(m).view(np.uint32))
        xs.append((np.arange(-3, 4, dtype=np.int64) + b).astype(np.uint32).view(np.float32))
    lo, hi = int(np.float32(2.0 ** -12).view(np.uint32)), int(np.float32(460.0).view(np.uint32))
    xs.append(np.arange(lo, hi, 997, dtype=np.int64).astype(np.uint32).view(np.float32))
    xs.append(np.array([0.0, 448.0, 450.0, 459.0, 2.0 ** -10, 2.0 ** -11, 1e-30], dtype=np.float32))
    x = np.concatenate(xs)
    xd = torch.from_numpy(x).cuda()
    y = torch.zeros(x.size, dtype=torch.uint8, device="cuda:0")
    dec = torch.zeros(256, dtype=torch.float32, device="cuda:0")
    run(P.sage_probe_cvt_fp8, dptr(xd), dptr(y), x.size, dptr(dec))
    ref = np.array([oracle.e4m3_encode(float(v)) for v in x], dtype=np.uint8)
    got = y.cpu().numpy()
    bad = np.flatnonzero(got != ref)
    assert bad.size == 0, "x=%r: hardware %02x, oracle %02x" % (float(x[bad[0]]), got[bad[0]], ref[bad[0]])
    d = dec.cpu().numpy()[:127]
    assert np.array_equal(d, vals.astype(np.float32))


def test_cvt_bf16_fp4_applies_only_the_power_of_two_part_of_the_scale(P):
    torch = torch_dev()
    e2 = np.array([oracle.e2m1_decode(c) for c in range(16)])
    vals = e4m3_values()[1:]
    byte = np.tile(np.arange(256), vals.size).astype(np.uint8)
    sc = np.repeat(vals, 256).astype(np.float32)
    pow2 = 2.0 ** np.floor(np.log2(sc.astype(np.float64)))
    lo = (e2[byte & 15] * pow2).astype(np.float32).view(np.uint32) >> 16      # exact in bf16
    hi = (e2[byte >> 4] * pow2).astype(np.float32).view(np.uint32) >> 16
    y = torch.zeros(byte.size, dtype=torch.int32, device="cuda:0")
    bd_, sd = torch.from_numpy(byte).cuda(), torch.from_numpy(sc).cuda()      # held until the kernel has run
    run(P.sage_probe_cvt_bf16_fp4, dptr(bd_), dptr(sd), dptr(y), byte.size)
    got = y.cpu().numpy().view(np.uint32)
    assert np.array_equal(got, (lo | (hi << 16)).astype(np.uint32))


def test_cvt_f16_fp4_applies_the_power_of_two_scale_exactly(P):
    """v_cvt_scalef32_pk_f16_fp4 with power-of-two scales: E2M1 value times the
    scale, exact in f16 (the NV16 kernel splits an E4M3 scale into this power of
    two and an integer mantissa), nearest even into f16's subnormal range and to
    zero below it."""
    torch = torch_dev()
    e2 = np.array([oracle.e2m1_decode(c) for c in range(16)])
    exps = np.arange(-40, 6)
    byte = np.tile(np.arange(256), exps.size).astype(np.uint8)
    sc = np.repeat(2.0 ** exps, 256).astype(np.float32)
    lo = (e2[byte & 15] * sc.astype(np.float64)).astype(np.float16).view(np.uint16).astype(np.uint32)
    hi = (e2[byte >> 4] * sc.astype(np.float64)).astype(np.float16).view(np.uint16).astype(np.uint32)
    y = torch.zeros(byte.size, dtype=torch.int32, device="cuda:0")
    bd_, sd = torch.from_numpy(byte).cuda(), torch.from_numpy(sc).cuda()      # held until the kernel has run
    P.sage_probe_cvt_f16_fp4.argtypes = [ctypes.c_void_p] * 3 + [ctypes.c_int, ctypes.c_void_p]
    run(P.sage_probe_cvt_f16_fp4, dptr(bd_), dptr(sd), dptr(y), byte.size)
    got = y.cpu().numpy().view(np.uint32)
    exp = (lo | (hi << 16)).astype(np.uint32)
    bad = np.flatnonzero(got != exp)
    assert bad.size == 0, "byte %02x scale 2^%d: got %08x expected %08x" % (
        byte[bad[0]], int(np.log2(sc[bad[0]])), got[bad[0]], exp[bad[0]])
