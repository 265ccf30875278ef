#!/usr/bin/env python3
"""Benchmark: microscaled-FP4 attention forward on one MI355X.

One step = the whole hot path on one batch: smoothing-K mean, FP4 quantization
of Q, K and V (V transposed), and the FP4 attention kernel, through the C ABI
(sage_attn_fp4_fwd_ws, inputs resident in HBM, preallocated workspace).
Workload: B=1, H=32, N=32768, D=128 non-causal, bf16 inputs with 1% of Q and K
rows scaled by 20 (seeded synthetic data), MXFP4.

Throughput is attention TOPS = 4 B H N^2 D / t.  The JSON line also carries
the attention kernel's own rate (HIP events around repeated launches of the
kernel alone on the same stream) as a fraction of the MXFP4 dense MFMA peak,
the bf16-MFMA comparison kernel's rate when available, the 8-bit attention
forward of Algorithm 2 (its whole step and its INT8-MFMA kernel alone, with
its accuracy against exact attention) and the backward of Algorithm 3 on the
same inputs, and the CPU oracle
timed on a bounded sample of query rows on the host cores.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "FP4 attention fwd TOPS at D=128,N=32768; % of MI355X MXFP4 MFMA peak"
PEAK_FP4_TFLOPS = 10100.0      # MI355X dense MXFP4 MFMA, published
PEAK_BF16_TFLOPS = 2500.0      # MI355X dense bf16 MFMA, published
PEAK_INT8_TOPS = 5000.0        # MI355X dense int8 MFMA, published
PEAK_HBM_GBS = 8000.0
COUNTERS = os.path.join(ROOT, "profiles", "attn_fp4_mx_counters.json")
KERNEL_SRC = os.path.join(ROOT, "paper_2505_11594_amd", "csrc", "attn_fp4.hip")


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def warm(torch, fn, min_calls: int = 3, min_s: float = 0.1):
    """Run fn until at least min_calls launches and min_s seconds have passed, so
    that a timed block after host-side work (input generation, quantization)
    does not start on a GPU whose clocks are still ramping."""
    t0 = time.perf_counter()
    n = 0
    while n < min_calls or time.perf_counter() - t0 < min_s:
        fn()
        torch.cuda.synchronize()
        n += 1


def kernel_source_sha() -> str:
    return hashlib.sha256(open(KERNEL_SRC, "rb").read()).hexdigest()[:16]


def traffic_from_counters(variant: str = "default"):
    """HBM bytes per launch of the 256-key attention kernel on the bench
    workload ("default": 128-query workgroups, the library's shape without
    SAGE_WG256; "wg256": 256-query workgroups) from committed rocprofv3
    FETCH_SIZE/WRITE_SIZE runs scaled by the copy-kernel calibration, or None
    when the kernel source changed since they were taken."""
    if not os.path.exists(COUNTERS):
        return None
    c = json.load(open(COUNTERS))
    if c.get("source_sha") != kernel_source_sha() or variant not in c:
        return None
    return float(c[variant]["hbm_bytes_per_launch"])


def cpu_model() -> str:
    """The host CPU's model name, as /proc/cpuinfo gives it."""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(w, q, k, v, budget_s: float = 15.0):
    """The oracle, as is, on a bounded sample of query rows of head 0."""
    import oracle
    threads = oracle.default_threads()
    N, D = w.N, w.D
    rng = np.random.default_rng(0)
    # one query head's K/V are quantized once per call; take a small probe first
    q1, k1, v1 = (np.ascontiguousarray(x[:1, :1]) for x in (q, k, v))

    def run(nr):
        rows = np.sort(rng.choice(N, size=nr, replace=False)).astype(np.int64)
        t0 = time.perf_counter()
        oracle.attn(q1, k1, v1, w.in_dtype, w.causal, oracle.FMT_MX, w.bkv, rows=rows, nthreads=threads)
        return time.perf_counter() - t0

    # per-row cost from two probes (the head's K/V quantization is a fixed cost)
    t1, t2 = run(threads), run(4 * threads)
    per_row = max((t2 - t1) / (3 * threads), 1e-6)
    nrows = int(max(threads, min(N, (budget_s - t1) / per_row)))
    rows = np.sort(rng.choice(N, size=nrows, replace=False)).astype(np.int64)
    t0 = time.perf_counter()
    oracle.attn(q1, k1, v1, w.in_dtype, w.causal, oracle.FMT_MX, w.bkv, rows=rows, nthreads=threads)
    dt = time.perf_counter() - t0
    ops = 4.0 * nrows * N * D * (0.5 if w.causal else 1.0)
    return {"value": ops / dt / 1e12, "unit": "TOPS", "cores": threads, "cpu_model": cpu_model(), "kind": "oracle",
            "sample": "%d random query rows of head 0 (of %d x %d), K/V quantization of that head included, %.1f s"
                      % (nrows, w.B * w.H, N, dt)}


RATE_TESTS = [  # (name, what one loop iteration issues, instructions of the counted kind per iteration)
    ("fma", "32 v_fma_f32", 32), ("exp", "8 v_exp_f32", 8), ("cvt_fp4", "8 v_cvt_scalef32_pk_fp4_f32", 8),
    ("mfma_fp4", "4 v_mfma_scale_f32_32x32x64_f8f6f4 (FP4)", 4), ("mfma_fp4+fma", "4 FP4 MFMA + 32 v_fma_f32", 4),
    ("mfma_fp4+exp", "4 FP4 MFMA + 8 v_exp_f32", 4), ("mfma_bf16", "4 v_mfma_f32_32x32x16_bf16", 4),
    ("mfma_bf16+fma", "4 bf16 MFMA + 32 v_fma_f32", 4), ("mfma16_fp4", "8 v_mfma_scale_f32_16x16x128_f8f6f4 (FP4)", 8),
    ("mfma16_fp4+fma", "8 FP4 16x16x128 MFMA + 32 v_fma_f32", 8),
    ("split_unverified", "even HW wave slots: 4 FP4 MFMA; odd: 32 v_fma_f32 (placement unchecked)", None),
    ("exp+fma", "8 v_exp_f32 + 32 independent v_fma_f32", 8),
    ("cvt_fp4+fma", "8 v_cvt_scalef32_pk_fp4_f32 + 32 independent v_fma_f32", 8),
    ("chain", "8 x (v_fma_f32 -> v_exp_f32 -> v_add_f32) + 4 FP4 packs", 8),
    ("inter_fma", "4 x (1 FP4 MFMA, 8 v_fma_f32), order pinned", 4),
    ("inter_exp", "4 x (1 FP4 MFMA, 2 v_exp_f32), order pinned", 4),
    ("inter_chain", "4 x (1 FP4 MFMA, 2 chain links + 1 FP4 pack), order pinned", 4)]

SPLIT_OTHER = [("fma", "32 v_fma_f32"), ("exp", "8 v_exp_f32"), ("chain", "8 chain links + 4 FP4 packs")]


def split_rates(torch, lib, iters):
    """MFMA waves and VALU waves sharing each SIMD, placement verified: one
    workgroup per CU, waves ranked per SIMD from their HW_ID; the time is
    reported only when every SIMD holds W/2 waves of each role."""
    import ctypes
    import numpy as np
    lib.sage_rates_split.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                     ctypes.POINTER(ctypes.c_float)]
    stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    res = {}
    for w in (2, 4):
        nw = 4 * w
        out = torch.empty(256 * 64 * nw, dtype=torch.float32, device="cuda:0")
        place = torch.zeros(2 * 256 * nw, dtype=torch.int32, device="cuda:0")
        for o, (name, what) in enumerate(SPLIT_OTHER):
            ms = ctypes.c_float()
            rc = lib.sage_rates_split(o, w, ctypes.c_void_p(out.data_ptr()), ctypes.c_void_p(place.data_ptr()), stream,
                                      ctypes.byref(ms))
            if rc != 0:
                raise RuntimeError("sage_rates_split(%d, %d) failed: %d" % (o, w, rc))
            pl = place.cpu().numpy().view(np.uint32).reshape(256, nw, 2)
            simd = (pl[:, :, 0] >> 4) & 3
            ok = True
            for b in range(256):
                for sd in range(4):
                    roles = pl[b, simd[b] == sd, 1]
                    if roles.size != w or int(roles.sum()) != w // 2:
                        ok = False
            cyc = ms.value * 1e-3 * 2.4e9 / (iters * (w // 2))   # per (1 MFMA + 1 other) wave-iteration pair
            # how the SPI spreads a workgroup's waves: SIMD of wave i against i % 4
            rr = float(np.mean(simd == (np.arange(nw)[None, :] % 4)))
            res["split_%s@%d" % (name, w)] = dict(cycles=cyc, placement_verified=ok, simd_is_wave_mod_4=rr)
            log("waves/SIMD %d  split MFMA | %-30s %8.1f cycles per pair of iterations, placement %s"
                % (w, what, cyc, "verified" if ok else "NOT verified"))
    return res


def issue_rates(torch):
    """Cycles per wave64 instruction per SIMD (at the 2.4 GHz peak clock) of the
    instructions the FP4 attention kernel is made of, and how much VALU work
    hides under FP4 MFMAs.  Prints one JSON line."""
    import ctypes
    lib = ctypes.CDLL(os.path.join(ROOT, "paper_2505_11594_amd", "libsage_rates.so"))
    lib.sage_rates_run.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p,
                                   ctypes.POINTER(ctypes.c_float)]
    iters = lib.sage_rates_iterations()
    out = torch.empty(1024 * 8 * 64, dtype=torch.float32, device="cuda:0")
    stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    res = {}
    for w in (2, 4):
        for t, (name, what, _) in enumerate(RATE_TESTS):
            ms = ctypes.c_float()
            rc = lib.sage_rates_run(t, w, ctypes.c_void_p(out.data_ptr()), stream, ctypes.byref(ms))
            if rc != 0:
                raise RuntimeError("sage_rates_run(%d) failed: %d" % (t, rc))
            cyc = ms.value * 1e-3 * 2.4e9 / (iters * w)     # cycles per loop iteration per SIMD
            res["%s@%d" % (name, w)] = cyc
            log("waves/SIMD %d  %-16s %-52s %8.1f cycles/iteration" % (w, name, what, cyc))
    split = split_rates(torch, lib, iters)
    summary = {}
    for w in (2, 4):
        g = lambda k: res["%s@%d" % (k, w)]
        summary["w%d" % w] = {
            "fma_cycles": g("fma") / 32, "exp_cycles": g("exp") / 8, "cvt_fp4_cycles": g("cvt_fp4") / 8,
            "mfma_fp4_32x32x64_cycles": g("mfma_fp4") / 4, "mfma_bf16_32x32x16_cycles": g("mfma_bf16") / 4,
            "mfma_fp4_16x16x128_cycles": g("mfma16_fp4") / 8,
            "fp4_mfma_tflops": 4 * 2 * 32 * 32 * 64 * 1024 * 2.4e9 / g("mfma_fp4") / 1e12,
            # fraction of the VALU loop's time that disappears when it shares the wave with the MFMAs
            "fma_hidden_under_fp4_mfma": (g("mfma_fp4") + g("fma") - g("mfma_fp4+fma")) / g("fma"),
            "exp_hidden_under_fp4_mfma": (g("mfma_fp4") + g("exp") - g("mfma_fp4+exp")) / g("exp"),
            "fma_hidden_under_bf16_mfma": (g("mfma_bf16") + g("fma") - g("mfma_bf16+fma")) / g("fma"),
            "fma_hidden_under_fp4_16x16x128": (g("mfma16_fp4") + g("fma") - g("mfma16_fp4+fma")) / g("fma"),
            # transcendental / pack work against plain VALU work on independent registers
            "exp_hidden_under_fma": (g("fma") + g("exp") - g("exp+fma")) / g("exp"),
            "cvt_fp4_hidden_under_fma": (g("fma") + g("cvt_fp4") - g("cvt_fp4+fma")) / g("cvt_fp4"),
            # the attention kernel's per-score work (fma, exp, add, half a pack), as measured
            "chain_cycles_per_score": g("chain") / 8,
            "chain_vs_isolated_rates": g("chain") / (16 * g("fma") / 32 + g("exp") + 4 * g("cvt_fp4") / 8),
            # the same mixes with the interleave pinned (one MFMA, then its share of the other work)
            "fma_hidden_under_fp4_mfma_pinned": (g("mfma_fp4") + g("fma") - g("inter_fma")) / g("fma"),
            "exp_hidden_under_fp4_mfma_pinned": (g("mfma_fp4") + g("exp") - g("inter_exp")) / g("exp"),
            "chain_hidden_under_fp4_mfma_pinned": (g("mfma_fp4") + g("chain") - g("inter_chain")) / g("chain")}
        for name, _ in SPLIT_OTHER:
            sp = split["split_%s@%d" % (name, w)]
            other = g({"fma": "fma", "exp": "exp", "chain": "chain"}[name])
            summary["w%d" % w]["split_%s_hidden" % name] = (
                (g("mfma_fp4") + other - sp["cycles"]) / min(g("mfma_fp4"), other) if sp["placement_verified"] else None)
            summary["w%d" % w]["split_%s_vs_serial" % name] = (
                sp["cycles"] / (g("mfma_fp4") + other) if sp["placement_verified"] else None)
    print(json.dumps({"mode": "rates", "clock_assumed_ghz": 2.4, "iterations": iters,
                      "cycles_per_iteration": res, "split": split, "derived": summary}), flush=True)


def issue_ceilings(torch, kernel_ms: float, variant: str = "default"):
    """Ceilings of the 256-key FP4 kernel on the bench workload from instruction
    issue: the issue rates measured live (register-only loops, 2 waves per SIMD
    as in the kernel) times the kernel's instructions per tile-wave (one wave x
    one 256-key tile) from the committed SQ counters of the same source.  Each
    ceiling is the MFMA time per tile-wave at the spec peak (32 MFMAs x 32
    cycles) over the cycles that one kind of work, or a combination, needs; the
    achieved figure puts the measured kernel time in the same units at 2.4 GHz.
    None when the counters were taken on another kernel source."""
    import ctypes
    if not os.path.exists(COUNTERS):
        return None
    c = json.load(open(COUNTERS))
    if c.get("source_sha") != kernel_source_sha() or "sq_per_tile_wave" not in c.get(variant, {}):
        return None
    sq = c[variant]["sq_per_tile_wave"]
    n_mfma, n_exp, n_pack = sq["SQ_INSTS_MFMA"], sq["SQ_INSTS_VALU_TRANS_F32"], c["fp4_packs_per_tile_wave"]
    n_valu = sq["SQ_INSTS_VALU"] - n_mfma - n_exp - n_pack     # SQ_INSTS_VALU counts MFMA and transcendentals too
    lib = ctypes.CDLL(os.path.join(ROOT, "paper_2505_11594_amd", "libsage_rates.so"))
    lib.sage_rates_run.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p,
                                   ctypes.POINTER(ctypes.c_float)]
    iters = lib.sage_rates_iterations()
    out = torch.empty(1024 * 8 * 64, dtype=torch.float32, device="cuda:0")
    stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    names = [t[0] for t in RATE_TESTS]
    cyc = {}
    for name in ("fma", "exp", "cvt_fp4", "mfma_fp4"):
        ms = ctypes.c_float()
        for _ in range(2):                                  # the first launch warms the clocks
            rc = lib.sage_rates_run(names.index(name), 2, ctypes.c_void_p(out.data_ptr()), stream, ctypes.byref(ms))
            if rc != 0:
                raise RuntimeError("sage_rates_run(%s) failed: %d" % (name, rc))
        per_iter = ms.value * 1e-3 * 2.4e9 / (iters * 2)
        cyc[name] = per_iter / [t[2] for t in RATE_TESTS if t[0] == name][0]
    t_mfma, t_exp = n_mfma * cyc["mfma_fp4"], n_exp * cyc["exp"]
    t_valu = n_valu * cyc["fma"] + n_pack * cyc["cvt_fp4"]
    spec = n_mfma * 32.0
    tile_waves_per_simd = c["tile_waves_per_launch"] / 1024.0
    measured = kernel_ms * 1e-3 * 2.4e9 / tile_waves_per_simd
    return {"cycles_per_instruction": {k: round(v, 3) for k, v in cyc.items()},
            "per_tile_wave": {"mfma": n_mfma, "exp": n_exp, "fp4_pack": n_pack, "other_valu": round(n_valu, 1)},
            "cycles_per_tile_wave": {"mfma": round(t_mfma, 1), "exp": round(t_exp, 1), "valu_and_packs": round(t_valu, 1),
                                     "all_in_series": round(t_mfma + t_exp + t_valu, 1),
                                     "measured_at_2.4GHz": round(measured, 1)},
            "frac_of_peak": {"mfma_alone": spec / t_mfma, "exp_alone": spec / t_exp, "valu_alone": spec / t_valu,
                             "exp_hidden_under_mfma": spec / (t_valu + max(t_mfma, t_exp)),
                             "all_in_series": spec / (t_mfma + t_exp + t_valu), "achieved": spec / measured},
            "counters": "profiles/attn_fp4_mx_counters.json (rocprofv3 SQ counters; 64 FP4 packs per tile-wave from the code)"}


def accuracy_vs_exact(torch, q, k, v, o, w, nrows=512, seed=7):
    """CosSim, relative L1 and RMSE of an attention output against fp64 softmax(QK^T/sqrt(D))V
    (the paper's accuracy metrics), on a seeded sample of query rows of every head; the
    reference is plain torch fp64 on the GPU."""
    B, H, N, D = w.B, w.H, w.N, w.D
    g = torch.Generator().manual_seed(seed)
    rows = torch.randint(0, N, (nrows,), generator=g).to(q.device)
    ref, got = [], []
    for bh in range(B * H):
        b, h = divmod(bh, H)
        qs = q[b, h].index_select(0, rows).double()
        s = (qs @ k[b, h].double().T) / float(np.sqrt(D))
        if w.causal:
            s = s.masked_fill(torch.arange(N, device=q.device)[None, :] > rows[:, None], float("-inf"))
        ref.append(torch.softmax(s, dim=1) @ v[b, h].double())
        got.append(o[b, h].index_select(0, rows).double())
    a, c = torch.cat(ref).flatten(), torch.cat(got).flatten()
    return {"cossim": float((a * c).sum() / (a.norm() * c.norm())),
            "l1": float((a - c).abs().sum() / a.abs().sum()),
            "rmse": float(((a - c) ** 2).mean().sqrt()),
            "rows": "%d random query rows per head, all %d heads" % (nrows, B * H)}


def other_configs(torch, bd, wl, steps):
    """Attention kernel alone (quantized operands resident) on the other workloads: the small
    non-causal D=128 case, the causal case and the D=64 long-sequence case in both formats."""
    res = {}
    dev = torch.device("cuda:0")
    for ci in (1, 3, 4):
        w = wl.CONFIGS[ci]
        q, k, v = wl.generate(w)
        dt = torch.bfloat16 if w.in_dtype == wl.IN_BF16 else torch.float16
        to_dev = lambda a: torch.from_numpy(a.view(np.int16)).view(dt).to(dev)
        qd, kd, vd = to_dev(q), to_dev(k), to_dev(v)
        del q, k, v
        o = torch.empty((w.B, w.H, w.N, w.D), dtype=torch.float32, device=dev)
        for f in w.fmts:
            fmt = bd.SAGE_FMT_MXFP4 if f == wl.FMT_MX else bd.SAGE_FMT_NV16_E4M3
            qq, kq, vq = (bd.sage_quant_fp4(x, r, fmt) for x, r in ((qd, bd.SAGE_ROLE_Q), (kd, bd.SAGE_ROLE_K),
                                                                    (vd, bd.SAGE_ROLE_V)))
            fk = fmt | (bd.bkv_flag(w.bkv) if f == wl.FMT_MX else 0)
            run = lambda: bd.sage_attn_fp4_fwd_prequant(qq[:2], kq[:2], vq[:2], (w.B, w.H, w.N, w.D), causal=w.causal,
                                                         fmt=fk, out=o)
            warm(torch, run)
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            n = max(3, min(steps, 10))
            e0.record()
            for _ in range(n):
                run()
            e1.record()
            torch.cuda.synchronize()
            t = e0.elapsed_time(e1) / 1e3 / n
            name = "%s_%s" % (w.name, "mxfp4" if f == wl.FMT_MX else "nv16")
            res[name] = {"kernel_ms": t * 1e3, "tops": w.ops / t / 1e12, "frac_of_mxfp4_peak": w.ops / t / 1e12 / PEAK_FP4_TFLOPS}
            log("%s: attention kernel %.3f ms = %.1f TOPS" % (name, t * 1e3, w.ops / t / 1e12))
            del qq, kq, vq
        del qd, kd, vd, o
        torch.cuda.empty_cache()
    return res


def int8_forward(torch, bd, w, qd, kd, vd, o, steps):
    """Algorithm 2 on the bench inputs: the whole step (k-mean, INT8 quantization
    of Q, K, V, the INT8 attention kernel with L) and the kernel alone, both
    timed with HIP events on the launch stream, and its accuracy."""
    B, H, N, D = w.B, w.H, w.N, w.D
    flags = (bd.SAGE_IN_BF16 if w.in_dtype == 1 else 0) | bd.SAGE_OUT_F32
    ws = torch.empty(bd.attn_int8_workspace_size(B, H, N, D, flags), dtype=torch.uint8, device=qd.device)
    L = torch.empty((B, H, N), dtype=torch.float32, device=qd.device)
    step = lambda: bd.sage_attn_int8_fwd(qd, kd, vd, causal=w.causal, out=o, lse_out=L, workspace=ws)
    step()
    torch.cuda.synchronize()
    acc = accuracy_vs_exact(torch, qd, kd, vd, o, w)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    n = max(3, min(steps, 10))
    e0.record()
    for _ in range(n):
        step()
    e1.record()
    torch.cuda.synchronize()
    t_step = e0.elapsed_time(e1) / 1e3 / n
    qq = bd.sage_quant_int8(qd, bd.SAGE_ROLE_Q)
    kq = bd.sage_quant_int8(kd, bd.SAGE_ROLE_K)
    vq = bd.sage_quant_int8(vd, bd.SAGE_ROLE_V)
    run = lambda: bd.sage_attn_int8_fwd_prequant(qq[:2], kq[:2], vq[:2], (B, H, N, D), causal=w.causal)
    run()
    torch.cuda.synchronize()
    e0.record()
    for _ in range(n):
        run()
    e1.record()
    torch.cuda.synchronize()
    t_k = e0.elapsed_time(e1) / 1e3 / n
    tops = w.ops / t_k / 1e12
    log("int8 forward: step %.3f ms = %.1f TOPS; kernel %.3f ms = %.1f TOPS (%.1f%% of the int8 peak); cossim %.5f"
        % (t_step * 1e3, w.ops / t_step / 1e12, t_k * 1e3, tops, 100 * tops / PEAK_INT8_TOPS, acc["cossim"]))
    step()                                       # leave this step's O and L in o, L for the backward
    torch.cuda.synchronize()
    int8_forward.lse = L
    del ws, qq, kq, vq
    return {"step_ms": t_step * 1e3, "step_tops": w.ops / t_step / 1e12, "kernel": "attn_int8_kernel<128,128,false,0>",
            "kernel_ms": t_k * 1e3, "kernel_tops": tops, "peak": PEAK_INT8_TOPS, "frac_of_int8_peak": tops / PEAK_INT8_TOPS,
            "kv_tile": 128, "accuracy_vs_exact": acc}


def int8_backward(torch, bd, w, qd, kd, vd, o, L, steps):
    """Algorithm 3 on the bench inputs, from the 8-bit forward's O and L and a
    seeded dO: the whole step (INT8 psi of Q, K, dO and their transposed
    copies, D = rowsum(dO O), the dK/dV and dQ kernels) timed with HIP events.
    Algorithmic work: the five products, 10 B H N^2 D (halved when causal);
    its floor is four int8 products at the int8 peak plus dO V^T at the
    16-bit peak."""
    B, H, N, D = w.B, w.H, w.N, w.D
    g = torch.Generator(device=qd.device).manual_seed(11)
    dout = torch.randn((B, H, N, D), generator=g, device=qd.device, dtype=torch.float32).to(qd.dtype)
    flags = bd.SAGE_IN_BF16 if w.in_dtype == 1 else 0
    ws = torch.empty(bd.attn_int8_bwd_workspace_size(B, H, N, D, flags), dtype=torch.uint8, device=qd.device)
    grads = [torch.empty((B, H, N, D), dtype=torch.float32, device=qd.device) for _ in range(3)]
    run = lambda: bd.sage_attn_int8_bwd(qd, kd, vd, o, L, dout, causal=w.causal, workspace=ws, out=grads)
    run()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    n = max(2, min(steps, 3))
    e0.record()
    for _ in range(n):
        run()
    e1.record()
    torch.cuda.synchronize()
    t = e0.elapsed_time(e1) / 1e3 / n
    ops = 10.0 * B * H * N * N * D * (0.5 if w.causal else 1.0)
    floor = (0.8 * ops) / (PEAK_INT8_TOPS * 1e12) + (0.2 * ops) / (PEAK_BF16_TFLOPS * 1e12)
    log("int8 backward: step %.3f ms = %.1f TOPS (%.1f%% of its mixed int8/bf16 peak)" % (t * 1e3, ops / t / 1e12,
                                                                                      100 * floor / t))
    del ws, grads, dout
    return {"step_ms": t * 1e3, "tops": ops / t / 1e12, "ops": ops,
            # the recommended workspace stores dS^: dK writes it, dQ sums from it
            "kernels": ["i8_bwd_prep_kernel<128,true>", "attn_i8_bwd_dv_kernel<128,false>",
                        "attn_i8_bwd_dk_kernel<128,false,true,true>", "attn_i8_bwd_dq_ds_kernel<128,false>"],
            "frac_of_mixed_peak": floor / t,
            "peak_note": "8/10 of the work at the int8 peak (5000 TOPS), 2/10 (dO V^T) at the bf16 peak (2500 TFLOP/s)"}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-bf16", action="store_true")
    ap.add_argument("--no-configs", action="store_true", help="skip the attention-kernel timings of the other workloads")
    ap.add_argument("--no-int8", action="store_true", help="skip the 8-bit attention forward")
    ap.add_argument("--wg256", action="store_true", help="--mode attn: 256-query workgroups (SAGE_WG256)")
    ap.add_argument("--mode", choices=["full", "attn", "shapes", "attn_nv16", "attn_int8", "attn_int8_bwd", "copy",
                                       "rates"],
                    default="full",
                    help="attn: only the attention kernel (for counter runs); shapes: the step and the attention "
                         "kernel with 256- and 128-query workgroups, alternated in one process; "
                         "attn_nv16: only the NV16 kernel on "
                         "B1 H24 N76800 D64; attn_int8: only the 8-bit one; "
                         "attn_int8_bwd: only the 8-bit backward (after one 8-bit forward for O and L); "
                         "copy: a plain 1 GiB device copy (calibrates FETCH_SIZE / WRITE_SIZE); "
                         "rates: instruction issue-rate microbenchmarks behind the VALU co-bound")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py: this build runs on one GPU only (the per-head work needs no communication; "
              "see the sharding note in DESIGN.md); --gpus %d is not supported" % args.gpus, file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2505_11594_amd import binding as bd
    from paper_2505_11594_amd import workloads as wl

    if args.mode == "rates":
        issue_rates(torch)
        return

    if args.mode == "copy":
        nbytes = 1 << 30
        src = torch.empty(nbytes, dtype=torch.uint8, device="cuda:0").fill_(1)
        dst = torch.empty_like(src)
        for _ in range(args.warmup + args.steps):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"mode": "copy", "bytes_per_copy": nbytes, "copies": args.warmup + args.steps}))
        return

    if args.mode == "attn_nv16":
        w = wl.CONFIGS[4]
        assert wl.FMT_NV16 in w.fmts
        B, H, N, D = w.B, w.H, w.N, w.D
        dt = torch.bfloat16 if w.in_dtype == wl.IN_BF16 else torch.float16
        xs = [torch.from_numpy(a.view(np.int16)).view(dt).to("cuda:0") for a in wl.generate(w)]
        nv = bd.SAGE_FMT_NV16_E4M3
        qq, kq, vq = (bd.sage_quant_fp4(x, r, nv) for x, r in zip(xs, (bd.SAGE_ROLE_Q, bd.SAGE_ROLE_K, bd.SAGE_ROLE_V)))
        o = torch.empty((B, H, N, D), dtype=torch.float32, device="cuda:0")
        for _ in range(args.warmup + args.steps):
            bd.sage_attn_fp4_fwd_prequant(qq[:2], kq[:2], vq[:2], (B, H, N, D), causal=w.causal,
                                          fmt=nv | bd.bkv_flag(w.bkv), out=o)
        torch.cuda.synchronize()
        print(json.dumps({"mode": "attn_nv16", "workload": w.name, "launches": args.warmup + args.steps,
                          "ops_per_launch": w.ops}))
        return

    w = wl.CONFIGS[2]
    B, H, N, D = w.B, w.H, w.N, w.D
    log("generating inputs", w.name)
    q, k, v = wl.generate(w)
    dt = torch.bfloat16 if w.in_dtype == wl.IN_BF16 else torch.float16
    dev = torch.device("cuda:0")
    to_dev = lambda a: torch.from_numpy(a.view(np.int16)).view(dt).to(dev)
    qd, kd, vd = to_dev(q), to_dev(k), to_dev(v)
    tile = bd.bkv_flag(w.bkv)
    # 256-query workgroups where the kernel has them (256-key tiles, non-causal, no smoothing Q): each K^/V^T
    # tile in LDS then serves 8 waves, which halves the HBM fetches at the same or slightly lower time
    wg = w.bkv == 256 and not w.causal
    shape = tile | (bd.SAGE_WG256 if wg else 0)
    fmt = bd.SAGE_FMT_MXFP4 | shape | (bd.SAGE_IN_BF16 if w.in_dtype == wl.IN_BF16 else 0) | bd.SAGE_OUT_F32
    ws = torch.empty(bd.attn_fp4_workspace_size(B, H, N, D, fmt), dtype=torch.uint8, device=dev)
    o = torch.empty((B, H, N, D), dtype=torch.float32, device=dev)
    ops = w.ops

    def step():
        bd.sage_attn_fp4_fwd(qd, kd, vd, causal=w.causal, fmt=bd.SAGE_FMT_MXFP4 | shape, out_f32=True, out=o,
                             workspace=ws)

    if args.mode == "attn_int8":
        qq = bd.sage_quant_int8(qd, bd.SAGE_ROLE_Q)
        kq = bd.sage_quant_int8(kd, bd.SAGE_ROLE_K)
        vq = bd.sage_quant_int8(vd, bd.SAGE_ROLE_V)
        for _ in range(args.warmup + args.steps):
            bd.sage_attn_int8_fwd_prequant(qq[:2], kq[:2], vq[:2], (B, H, N, D), causal=w.causal)
        torch.cuda.synchronize()
        print(json.dumps({"mode": "attn_int8", "launches": args.warmup + args.steps, "ops_per_launch": ops}))
        return

    if args.mode == "attn_int8_bwd":
        o8, L8 = bd.sage_attn_int8_fwd(qd, kd, vd, causal=w.causal, out_f32=True)
        g = torch.Generator(device=dev).manual_seed(11)
        dout = torch.randn((B, H, N, D), generator=g, device=dev, dtype=torch.float32).to(dt)
        flags = bd.SAGE_IN_BF16 if w.in_dtype == wl.IN_BF16 else 0
        wsb = torch.empty(bd.attn_int8_bwd_workspace_size(B, H, N, D, flags), dtype=torch.uint8, device=dev)
        grads = [torch.empty((B, H, N, D), dtype=torch.float32, device=dev) for _ in range(3)]
        for _ in range(args.warmup + args.steps):
            bd.sage_attn_int8_bwd(qd, kd, vd, o8, L8, dout, causal=w.causal, workspace=wsb, out=grads)
        torch.cuda.synchronize()
        print(json.dumps({"mode": "attn_int8_bwd", "launches": args.warmup + args.steps,
                          "ops_per_launch": 10.0 * B * H * N * N * D * (0.5 if w.causal else 1.0)}))
        return

    if args.mode == "shapes":
        # the two workgroup shapes of the 256-key kernel, alternated args.warmup rounds (order swapped each
        # round), args.steps launches per timing: the whole step and the attention kernel alone
        qq = bd.sage_quant_fp4(qd, bd.SAGE_ROLE_Q)
        kq = bd.sage_quant_fp4(kd, bd.SAGE_ROLE_K)
        vq = bd.sage_quant_fp4(vd, bd.SAGE_ROLE_V)
        shapes = {"wg256": tile | bd.SAGE_WG256, "wg128": tile}
        wss = {n: torch.empty(bd.attn_fp4_workspace_size(B, H, N, D, fmt | f), dtype=torch.uint8, device=dev)
               for n, f in shapes.items()}
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)

        def timed(fn):
            e0.record()
            for _ in range(args.steps):
                fn()
            e1.record()
            torch.cuda.synchronize()
            return e0.elapsed_time(e1) / args.steps

        for n, f in shapes.items():
            warm(torch, lambda: bd.sage_attn_fp4_fwd(qd, kd, vd, causal=w.causal, fmt=bd.SAGE_FMT_MXFP4 | f,
                                                     out_f32=True, out=o, workspace=wss[n]))
        res = {"step_" + n: [] for n in shapes}
        res.update({"attn_" + n: [] for n in shapes})
        for r in range(max(2, args.warmup)):
            order = list(shapes) if r % 2 == 0 else list(shapes)[::-1]
            for n in order:
                f = shapes[n]
                res["step_" + n].append(timed(lambda: bd.sage_attn_fp4_fwd(
                    qd, kd, vd, causal=w.causal, fmt=bd.SAGE_FMT_MXFP4 | f, out_f32=True, out=o, workspace=wss[n])))
            for n in order:
                f = shapes[n]
                res["attn_" + n].append(timed(lambda: bd.sage_attn_fp4_fwd_prequant(
                    qq[:2], kq[:2], vq[:2], (B, H, N, D), causal=w.causal, fmt=f, out=o)))
            log("round %d: %s" % (r, ", ".join("%s %.4f ms" % (k_, v_[-1]) for k_, v_ in res.items())))
        print(json.dumps({"mode": "shapes", "workload": w.name, "launches_per_timing": args.steps,
                          "ms": res, "mean_ms": {k_: sum(v_) / len(v_) for k_, v_ in res.items()}}))
        return

    if args.mode == "attn":
        qq = bd.sage_quant_fp4(qd, bd.SAGE_ROLE_Q)
        kq = bd.sage_quant_fp4(kd, bd.SAGE_ROLE_K)
        vq = bd.sage_quant_fp4(vd, bd.SAGE_ROLE_V)
        fa = tile | (bd.SAGE_WG256 if args.wg256 else 0)
        for _ in range(args.warmup + args.steps):
            bd.sage_attn_fp4_fwd_prequant(qq[:2], kq[:2], vq[:2], (B, H, N, D), causal=w.causal, fmt=fa, out=o)
        torch.cuda.synchronize()
        print(json.dumps({"mode": "attn", "launches": args.warmup + args.steps, "ops_per_launch": ops}))
        return

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    t_step = (time.perf_counter() - t0) / args.steps
    log("step %.3f ms" % (t_step * 1e3))

    acc = accuracy_vs_exact(torch, qd, kd, vd, o, w)
    log("accuracy vs exact attention: cossim %.5f, l1 %.4f, rmse %.3g" % (acc["cossim"], acc["l1"], acc["rmse"]))

    # the attention kernel alone, timed with HIP events on the launch stream
    qq = bd.sage_quant_fp4(qd, bd.SAGE_ROLE_Q)
    kq = bd.sage_quant_fp4(kd, bd.SAGE_ROLE_K)
    vq = bd.sage_quant_fp4(vd, bd.SAGE_ROLE_V)

    def attn_only():
        bd.sage_attn_fp4_fwd_prequant(qq[:2], kq[:2], vq[:2], (B, H, N, D), causal=w.causal, fmt=shape, out=o)

    for _ in range(2):
        attn_only()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(args.steps):
        attn_only()
    e1.record()
    torch.cuda.synchronize()
    t_attn = e0.elapsed_time(e1) / 1e3 / args.steps
    attn_tflops = ops / t_attn / 1e12
    log("attention kernel %.3f ms = %.1f TFLOP/s (%.1f%% of MXFP4 peak)" % (t_attn * 1e3, attn_tflops,
                                                                        100 * attn_tflops / PEAK_FP4_TFLOPS))
    # quantization kernels alone (HBM-bound)
    e0.record()
    for _ in range(args.steps):
        bd.sage_quant_fp4(qd, bd.SAGE_ROLE_Q)
        bd.sage_quant_fp4(kd, bd.SAGE_ROLE_K)
        bd.sage_quant_fp4(vd, bd.SAGE_ROLE_V)
    e1.record()
    torch.cuda.synchronize()
    t_quant = e0.elapsed_time(e1) / 1e3 / args.steps
    n_el = B * H * N * D
    quant_bytes = n_el * (2 + 2 + 2 + 2) + 3 * n_el * (0.5 + 1.0 / 32)   # K read twice (mean + quantize)

    # the same kernel with 128-query workgroups (the shape without SAGE_WG256): same bits, twice the fetches
    wg128 = None
    if wg:
        run_wg = lambda: bd.sage_attn_fp4_fwd_prequant(qq[:2], kq[:2], vq[:2], (B, H, N, D), causal=w.causal,
                                                       fmt=tile, out=o)
        warm(torch, run_wg)
        e0.record()
        for _ in range(args.steps):
            run_wg()
        e1.record()
        torch.cuda.synchronize()
        t_wg = e0.elapsed_time(e1) / 1e3 / args.steps
        wg128 = {"kernel": "attn_fp4_mx256_kernel<%d,false,0,false,4>" % D, "kernel_ms": t_wg * 1e3,
                 "tops": ops / t_wg / 1e12, "frac_of_mxfp4_peak": ops / t_wg / 1e12 / PEAK_FP4_TFLOPS,
                 "traffic": traffic_from_counters("default")}
        log("attention kernel, 128-query workgroups %.3f ms = %.1f TFLOP/s" % (t_wg * 1e3, ops / t_wg / 1e12))

    bf16 = None
    if not args.no_bf16:
        try:
            bd.sage_attn_bf16_fwd(qd, kd, vd, causal=w.causal, out_f32=True, out=o)
            torch.cuda.synchronize()
            e0.record()
            for _ in range(args.steps):
                bd.sage_attn_bf16_fwd(qd, kd, vd, causal=w.causal, out_f32=True, out=o)
            e1.record()
            torch.cuda.synchronize()
            t_bf = e0.elapsed_time(e1) / 1e3 / args.steps
            bf16 = {"tops": ops / t_bf / 1e12, "ms": t_bf * 1e3,
                    "frac_of_bf16_peak": ops / t_bf / 1e12 / PEAK_BF16_TFLOPS,
                    "accuracy_vs_exact": accuracy_vs_exact(torch, qd, kd, vd, o, w)}
            log("bf16 kernel %.3f ms, cossim %.5f" % (t_bf * 1e3, bf16["accuracy_vs_exact"]["cossim"]))
        except bd.SageError as ex:
            log("bf16 kernel unavailable:", ex)

    others = None
    smooth_q = None
    if not args.no_configs:
        # the same step with smoothing Q (query-block means, their GEMV with K', the bias added to S)
        fmt_sq = bd.SAGE_FMT_MXFP4 | tile | bd.SAGE_SMOOTH_Q
        ws_sq = torch.empty(bd.attn_fp4_workspace_size(B, H, N, D, fmt_sq | bd.SAGE_IN_BF16 | bd.SAGE_OUT_F32),
                            dtype=torch.uint8, device=dev)
        step_sq = lambda: bd.sage_attn_fp4_fwd(qd, kd, vd, causal=w.causal, fmt=fmt_sq, out_f32=True, out=o,
                                               workspace=ws_sq)
        warm(torch, step_sq)
        n_sq = max(3, min(args.steps, 10))
        e0.record()
        for _ in range(n_sq):
            step_sq()
        e1.record()
        torch.cuda.synchronize()
        t_sq = e0.elapsed_time(e1) / 1e3 / n_sq
        smooth_q = {"step_ms": t_sq * 1e3, "tops": ops / t_sq / 1e12}
        log("step with smoothing Q %.3f ms = %.1f TOPS" % (t_sq * 1e3, ops / t_sq / 1e12))
        del ws_sq
        others = other_configs(torch, bd, wl, args.steps)

    int8 = None
    int8_bwd = None
    if not args.no_int8:
        int8 = int8_forward(torch, bd, w, qd, kd, vd, o, args.steps)
        int8_bwd = int8_backward(torch, bd, w, qd, kd, vd, o, int8_forward.lse, args.steps)

    ceilings = None
    if w.bkv == 256 and D == 128:
        ceilings = issue_ceilings(torch, t_attn * 1e3, "wg256" if wg else "default")
        if ceilings:
            log("issue ceilings (fraction of the MXFP4 peak): " +
                ", ".join("%s %.3f" % kv for kv in ceilings["frac_of_peak"].items()))

    cpu = None
    if not args.no_cpu_baseline:
        log("cpu baseline (oracle)")
        cpu = cpu_baseline(w, q, k, v)

    line = {
        "metric": METRIC,
        "value": ops / t_step / 1e12,
        "unit": "TOPS",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": t_step * 1e3,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "mxfp4",
        "data": "synthetic (seeded normal Q/K/V, 1% of Q and K rows x20)",
        "config": {"workload": w.name, "B": B, "H": H, "N": N, "D": D, "causal": w.causal,
                   "format": "MXFP4 (E2M1, 1x32 blocks, E8M0 scales)", "kv_tile": w.bkv, "parallelism": "none",
                   "step": "kmean + quantize Q/K/V + FP4 attention (sage_attn_fp4_fwd_ws)",
                   "query_workgroup": 256 if wg else 128},
        "roofline": {"bound": "mfma", "achieved": attn_tflops, "peak": PEAK_FP4_TFLOPS, "unit": "TFLOP/s",
                     "frac": attn_tflops / PEAK_FP4_TFLOPS,
                     "traffic": traffic_from_counters("wg256" if wg else "default") if w.bkv == 256 else None,
                     "kernel": ("attn_fp4_mx256_kernel<%d,false,0,false,%d>" % (D, 8 if wg else 4) if w.bkv == 256
                                else "attn_fp4_mx_kernel<%d,%d,false,0,false>" % (D, w.bkv)),
                     "kernel_ms": t_attn * 1e3,
                     "issue_ceilings": ceilings},
        "accuracy_vs_exact": acc,
        "quantize": {"ms": t_quant * 1e3, "algorithmic_GBs": quant_bytes / t_quant / 1e9,
                     "frac_of_hbm_peak": quant_bytes / t_quant / 1e9 / PEAK_HBM_GBS},
        "bf16_kernel": bf16,
        "attn_wg128": wg128,
        "smooth_q_step": smooth_q,
        "int8_fwd": int8,
        "int8_bwd": int8_bwd,
        "other_configs": others,
        "cpu_baseline": cpu,
    }
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
