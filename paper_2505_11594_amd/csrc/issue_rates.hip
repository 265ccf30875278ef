// Instruction issue-rate microbenchmarks for gfx950, built into a separate
// measurement library (not the attention library).  They ground the
// co-bound of the FP4 attention kernel: how many cycles the VALU, the
// transcendental unit, the FP4 pack convert and the block-scaled FP4 MFMA
// take per wave64 instruction, and how much VALU work runs while FP4 MFMAs
// execute.  Every wave runs register-only loops; nothing reads or writes
// memory except one store per lane at the end.
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

typedef int v8i __attribute__((ext_vector_type(8)));
typedef float v16f __attribute__((ext_vector_type(16)));
typedef float v4f __attribute__((ext_vector_type(4)));
typedef __bf16 v8bf __attribute__((ext_vector_type(8)));

constexpr int kIters = 1024;

enum Test {
  kFma = 0,          // 32 independent v_fma_f32
  kExp = 1,          // 8 v_exp_f32
  kCvtFp4 = 2,       // 8 v_cvt_scalef32_pk_fp4_f32
  kMfmaFp4 = 3,      // 4 v_mfma_scale_f32_32x32x64_f8f6f4 (FP4 x FP4, 4 accumulators)
  kMfmaFp4Fma = 4,   // the same 4 MFMAs + 32 independent v_fma_f32 in the same wave
  kMfmaFp4Exp = 5,   // the same 4 MFMAs + 8 v_exp_f32 in the same wave
  kMfmaBf16 = 6,     // 4 v_mfma_f32_32x32x16_bf16
  kMfmaBf16Fma = 7,  // the same + 32 v_fma_f32
  kMfma16Fp4 = 8,    // 8 v_mfma_scale_f32_16x16x128_f8f6f4 (the same MACs as test 3)
  kMfma16Fp4Fma = 9, // the same + 32 v_fma_f32
  kSplit = 10,       // waves on even SIMD slots: test 3; odd slots: 32 v_fma_f32
  kExpFma = 11,      // 8 v_exp_f32 + 32 v_fma_f32 on independent registers
  kCvtFma = 12,      // 8 v_cvt_scalef32_pk_fp4_f32 + 32 v_fma_f32 on independent registers
  kChain = 13,       // the attention kernel's per-score chain: 8 x (v_fma_f32 -> v_exp_f32 -> v_add_f32) + 4 FP4 packs
  kInterFma = 14,    // test 4 with the order pinned: 4 x (1 FP4 MFMA, 8 v_fma_f32)
  kInterExp = 15,    // test 5 with the order pinned: 4 x (1 FP4 MFMA, 2 v_exp_f32)
  kInterChain = 16,  // 4 x (1 FP4 MFMA, 2 chain links, 1 FP4 pack): the chain of test 13 under MFMAs
  kNumTests = 17
};

// sched_group_barrier masks (LLVM AMDGPU): VALU without transcendentals, MFMA, transcendental
constexpr int kSgValu = 0x002, kSgMfma = 0x008, kSgTrans = 0x400;

template <int T>
__global__ __launch_bounds__(64) void rate_kernel(float* out, float seed) {
  const int lane = threadIdx.x;
  float x[8], y[8], z[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) x[i] = seed + 0.001f * (lane + i);
#pragma unroll
  for (int i = 0; i < 8; ++i) y[i] = seed - 0.002f * (lane + i);
#pragma unroll
  for (int i = 0; i < 8; ++i) z[i] = 0.0f;
  unsigned w[8] = {0, 0, 0, 0, 0, 0, 0, 0};
  v16f acc[4] = {};
  v4f acc16[8] = {};
  const v8i a = v8i{lane, lane + 1, lane + 2, lane + 3, 0, 0, 0, 0};
  v8bf ab;
#pragma unroll
  for (int i = 0; i < 8; ++i) ab[i] = (__bf16)(0.01f * (lane + i));
  // hardware wave slot on this SIMD (HW_ID[3:0], a read-only register)
  const unsigned slot = __builtin_amdgcn_s_getreg((3 << 11) | (0 << 6) | 4) & 15u;
  const bool mfma_role = T != kSplit || (slot & 1u) == 0;
  for (int it = 0; it < kIters; ++it) {
    if (T == kMfmaFp4 || T == kMfmaFp4Fma || T == kMfmaFp4Exp || (T == kSplit && mfma_role)) {
#pragma unroll
      for (int i = 0; i < 4; ++i)
        acc[i] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a, a, acc[i], 4, 4, 0, 127, 0, 127);
    }
    if (T == kMfma16Fp4 || T == kMfma16Fp4Fma) {
#pragma unroll
      for (int i = 0; i < 8; ++i)
        acc16[i] = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(a, a, acc16[i], 4, 4, 0, 127, 0, 127);
    }
    if (T == kMfmaBf16 || T == kMfmaBf16Fma) {
#pragma unroll
      for (int i = 0; i < 4; ++i) acc[i] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ab, ab, acc[i], 0, 0, 0);
    }
    if (T == kFma || T == kMfmaFp4Fma || T == kMfmaBf16Fma || T == kMfma16Fp4Fma || (T == kSplit && !mfma_role)) {
#pragma unroll
      for (int r = 0; r < 4; ++r)
#pragma unroll
        for (int i = 0; i < 8; ++i) x[i] = __builtin_fmaf(x[i], 0.999f, 0.0001f);
    }
    if (T == kExpFma || T == kCvtFma) {
#pragma unroll
      for (int r = 0; r < 4; ++r)
#pragma unroll
        for (int i = 0; i < 8; ++i) y[i] = __builtin_fmaf(y[i], 0.999f, 0.0001f);
    }
    if (T == kExp || T == kMfmaFp4Exp || T == kExpFma) {
#pragma unroll
      for (int i = 0; i < 8; ++i) x[i] = __builtin_amdgcn_exp2f(-x[i]);
    }
    if (T == kChain) {
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const float p = __builtin_amdgcn_exp2f(__builtin_fmaf(x[i], 0.999f, -0.5f));
        z[i] += p;
        x[i] = p;
      }
#pragma unroll
      for (int i = 0; i < 4; ++i) w[i] = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(w[i], x[2 * i], x[2 * i + 1], 1.0f, 0);
    }
    if (T == kCvtFp4 || T == kCvtFma) {
#pragma unroll
      for (int i = 0; i < 8; ++i) w[i] = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(w[i], x[i], x[(i + 1) & 7], 1.0f, 0);
    }
    if (T == kInterFma || T == kInterExp || T == kInterChain) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        acc[i] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a, a, acc[i], 4, 4, 0, 127, 0, 127);
        if (T == kInterFma) {
#pragma unroll
          for (int j = 0; j < 8; ++j) x[j] = __builtin_fmaf(x[j], 0.999f, 0.0001f);
        } else if (T == kInterExp) {
          x[2 * i] = __builtin_amdgcn_exp2f(-x[2 * i]);
          x[2 * i + 1] = __builtin_amdgcn_exp2f(-x[2 * i + 1]);
        } else {
#pragma unroll
          for (int j = 2 * i; j < 2 * i + 2; ++j) {
            const float p = __builtin_amdgcn_exp2f(__builtin_fmaf(x[j], 0.999f, -0.5f));
            z[j] += p;
            x[j] = p;
          }
          w[i] = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(w[i], x[2 * i], x[2 * i + 1], 1.0f, 0);
        }
      }
      // pin the interleave: each MFMA followed by its share of the other work
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        __builtin_amdgcn_sched_group_barrier(kSgMfma, 1, 0);
        if (T == kInterFma) __builtin_amdgcn_sched_group_barrier(kSgValu, 8, 0);
        if (T == kInterExp) __builtin_amdgcn_sched_group_barrier(kSgTrans, 2, 0);
        if (T == kInterChain) {
          __builtin_amdgcn_sched_group_barrier(kSgValu, 1, 0);
          __builtin_amdgcn_sched_group_barrier(kSgTrans, 1, 0);
          __builtin_amdgcn_sched_group_barrier(kSgValu, 2, 0);
          __builtin_amdgcn_sched_group_barrier(kSgTrans, 1, 0);
          __builtin_amdgcn_sched_group_barrier(kSgValu, 2, 0);
        }
      }
    }
  }
  float s = 0.f;
#pragma unroll
  for (int i = 0; i < 8; ++i) s += x[i] + y[i] + z[i] + __uint_as_float(w[i] & 0x3fffffffu);
#pragma unroll
  for (int i = 0; i < 4; ++i) s += acc[i][lane & 15];
#pragma unroll
  for (int i = 0; i < 8; ++i) s += acc16[i][lane & 3];
  out[blockIdx.x * 64 + lane] = s;
}

template <int T>
hipError_t launch(float* out, int blocks, hipStream_t st) {
  hipLaunchKernelGGL(rate_kernel<T>, dim3((unsigned)blocks), dim3(64), 0, st, out, 0.5f);
  return hipGetLastError();
}

hipError_t launch_test(int test, float* out, int blocks, hipStream_t st) {
  switch (test) {
    case kFma: return launch<kFma>(out, blocks, st);
    case kExp: return launch<kExp>(out, blocks, st);
    case kCvtFp4: return launch<kCvtFp4>(out, blocks, st);
    case kMfmaFp4: return launch<kMfmaFp4>(out, blocks, st);
    case kMfmaFp4Fma: return launch<kMfmaFp4Fma>(out, blocks, st);
    case kMfmaFp4Exp: return launch<kMfmaFp4Exp>(out, blocks, st);
    case kMfmaBf16: return launch<kMfmaBf16>(out, blocks, st);
    case kMfmaBf16Fma: return launch<kMfmaBf16Fma>(out, blocks, st);
    case kMfma16Fp4: return launch<kMfma16Fp4>(out, blocks, st);
    case kMfma16Fp4Fma: return launch<kMfma16Fp4Fma>(out, blocks, st);
    case kSplit: return launch<kSplit>(out, blocks, st);
    case kExpFma: return launch<kExpFma>(out, blocks, st);
    case kCvtFma: return launch<kCvtFma>(out, blocks, st);
    case kChain: return launch<kChain>(out, blocks, st);
    case kInterFma: return launch<kInterFma>(out, blocks, st);
    case kInterExp: return launch<kInterExp>(out, blocks, st);
    case kInterChain: return launch<kInterChain>(out, blocks, st);
    default: return launch<kSplit>(out, blocks, st);
  }
}

// ---------------------------------------------------------------------------
// Cross-wave split with verified placement.  One workgroup per CU (its 96 KiB
// of LDS leave no room for a second), 4 W waves per workgroup.  Each wave
// reads its SIMD from HW_ID; waves are ranked among the workgroup's waves on
// the same SIMD, and even ranks run the FP4 MFMA loop of test 3, odd ranks
// the other role: 32 v_fma_f32 (OTHER = 0), 8 v_exp_f32 (1) or the chain of
// test 13 (2).  Every wave records HW_ID and its role, so the host can check
// that each SIMD holds W/2 waves of each role before it reports the time.
constexpr int kSplitLds = 96 * 1024;

template <int OTHER>
__global__ __launch_bounds__(1024) void split_kernel(float* out, unsigned* place, float seed) {
  __shared__ int lds[kSplitLds / 4];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, nw = blockDim.x >> 6;
  const unsigned hw = __builtin_amdgcn_s_getreg((31 << 11) | (0 << 6) | 4);   // HW_ID, 32 bits
  const int simd = (int)((hw >> 4) & 3u);
  if (lane == 0) lds[wave] = simd;
  __syncthreads();
  int rank = 0;
  for (int w = 0; w < wave; ++w) rank += lds[w] == simd;
  const bool mfma_role = (rank & 1) == 0;
  float x[8], z[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) { x[i] = seed + 0.001f * (lane + i); z[i] = 0.0f; }
  unsigned wd[4] = {0, 0, 0, 0};
  v16f acc[4] = {};
  const v8i a = v8i{lane, lane + 1, lane + 2, lane + 3, 0, 0, 0, 0};
  if (mfma_role) {
    for (int it = 0; it < kIters; ++it)
#pragma unroll
      for (int i = 0; i < 4; ++i)
        acc[i] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a, a, acc[i], 4, 4, 0, 127, 0, 127);
  } else {
    for (int it = 0; it < kIters; ++it) {
      if (OTHER == 0) {
#pragma unroll
        for (int r = 0; r < 4; ++r)
#pragma unroll
          for (int i = 0; i < 8; ++i) x[i] = __builtin_fmaf(x[i], 0.999f, 0.0001f);
      } else if (OTHER == 1) {
#pragma unroll
        for (int i = 0; i < 8; ++i) x[i] = __builtin_amdgcn_exp2f(-x[i]);
      } else {
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          const float p = __builtin_amdgcn_exp2f(__builtin_fmaf(x[i], 0.999f, -0.5f));
          z[i] += p;
          x[i] = p;
        }
#pragma unroll
        for (int i = 0; i < 4; ++i) wd[i] = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(wd[i], x[2 * i], x[2 * i + 1], 1.0f, 0);
      }
    }
  }
  float s = 0.f;
#pragma unroll
  for (int i = 0; i < 8; ++i) s += x[i] + z[i];
#pragma unroll
  for (int i = 0; i < 4; ++i) s += acc[i][lane & 15] + __uint_as_float(wd[i] & 0x3fffffffu);
  out[(size_t)blockIdx.x * blockDim.x + threadIdx.x] = s;
  if (lane == 0) {
    place[2 * ((size_t)blockIdx.x * nw + wave)] = hw;
    place[2 * ((size_t)blockIdx.x * nw + wave) + 1] = mfma_role ? 1u : 0u;
  }
}

template <int OTHER>
hipError_t launch_split(float* out, unsigned* place, int blocks, int waves, hipStream_t st) {
  hipLaunchKernelGGL(split_kernel<OTHER>, dim3((unsigned)blocks), dim3((unsigned)(64 * waves)), 0, st, out, place, 0.5f);
  return hipGetLastError();
}

hipError_t launch_split_any(int other, float* out, unsigned* place, int blocks, int waves, hipStream_t st) {
  if (other == 0) return launch_split<0>(out, place, blocks, waves, st);
  if (other == 1) return launch_split<1>(out, place, blocks, waves, st);
  return launch_split<2>(out, place, blocks, waves, st);
}

}  // namespace

extern "C" {

// Number of tests and loop iterations per wave (each iteration issues the
// instruction mix named in the test table above).
int sage_rates_num_tests(void) { return kNumTests; }
int sage_rates_iterations(void) { return kIters; }

// Runs test `test` with `waves_per_simd` one-wave workgroups per SIMD
// (1024 * waves_per_simd workgroups: 256 CUs x 4 SIMDs) and writes the mean
// duration of 5 launches after one warm-up launch, in milliseconds, to *ms.
// `out` is a device buffer of at least 1024 * waves_per_simd * 64 floats.
// Returns 0, 1 for bad arguments, 3 for a HIP error.  Synchronizes `stream`.
int sage_rates_run(int test, int waves_per_simd, float* out, hipStream_t stream, float* ms) {
  if (test < 0 || test >= kNumTests || waves_per_simd < 1 || waves_per_simd > 8 || !out || !ms) return 1;
  const int blocks = 1024 * waves_per_simd;
  hipEvent_t e0, e1;
  if (hipEventCreate(&e0) != hipSuccess) return 3;
  if (hipEventCreate(&e1) != hipSuccess) { (void)hipEventDestroy(e0); return 3; }
  int rc = 0;
  if (launch_test(test, out, blocks, stream) != hipSuccess || hipEventRecord(e0, stream) != hipSuccess) rc = 3;
  for (int r = 0; r < 5 && rc == 0; ++r)
    if (launch_test(test, out, blocks, stream) != hipSuccess) rc = 3;
  if (rc == 0 && (hipEventRecord(e1, stream) != hipSuccess || hipEventSynchronize(e1) != hipSuccess)) rc = 3;
  float t = 0.f;
  if (rc == 0 && hipEventElapsedTime(&t, e0, e1) != hipSuccess) rc = 3;
  *ms = t / 5.0f;
  (void)hipEventDestroy(e0);
  (void)hipEventDestroy(e1);
  return rc;
}

// The cross-wave split with verified placement: 256 workgroups (one per CU)
// of 4 * waves_per_simd waves (waves_per_simd 2 or 4); `other` picks the
// second role (0: 32 v_fma_f32, 1: 8 v_exp_f32, 2: the chain of test 13).
// `out` holds at least 256 * 64 * 4 * waves_per_simd floats, `place` at least
// 2 * 256 * 4 * waves_per_simd unsigned: per wave its HW_ID and role
// (1 = MFMA), from the last launch.  *ms: mean of 5 launches after a warm-up.
// Returns 0, 1 for bad arguments, 3 for a HIP error.  Synchronizes `stream`.
int sage_rates_split(int other, int waves_per_simd, float* out, unsigned* place, hipStream_t stream, float* ms) {
  if (other < 0 || other > 2 || (waves_per_simd != 2 && waves_per_simd != 4) || !out || !place || !ms) return 1;
  const int blocks = 256, waves = 4 * waves_per_simd;
  hipEvent_t e0, e1;
  if (hipEventCreate(&e0) != hipSuccess) return 3;
  if (hipEventCreate(&e1) != hipSuccess) { (void)hipEventDestroy(e0); return 3; }
  int rc = 0;
  if (launch_split_any(other, out, place, blocks, waves, stream) != hipSuccess || hipEventRecord(e0, stream) != hipSuccess) rc = 3;
  for (int r = 0; r < 5 && rc == 0; ++r)
    if (launch_split_any(other, out, place, blocks, waves, stream) != hipSuccess) rc = 3;
  if (rc == 0 && (hipEventRecord(e1, stream) != hipSuccess || hipEventSynchronize(e1) != hipSuccess)) rc = 3;
  float t = 0.f;
  if (rc == 0 && hipEventElapsedTime(&t, e0, e1) != hipSuccess) rc = 3;
  *ms = t / 5.0f;
  (void)hipEventDestroy(e0);
  (void)hipEventDestroy(e1);
  return rc;
}

}  // extern "C"
