// Hardware probes for gfx950, built into a separate library (not the
// attention library): the semantics the attention kernels rely on, exposed
// so that tests can check them against independent CPU definitions.
//   - v_cvt_scalef32_pk_fp4_f32: FP4 E2M1 rounding (nearest even), saturation
//     at +-6, the sign of zero, and division by the power-of-two scale;
//   - v_exp_f32: its error against the correctly rounded exp2;
//   - v_cvt_pk_u8_f32: its rounding (nearest even) and clamping to [0, 255];
//   - the register layouts of v_mfma_scale_f32_32x32x64_f8f6f4 (FP4 operands,
//     E8M0 scales), v_mfma_i32_32x32x32_i8 and v_mfma_f32_32x32x16_bf16: lane
//     l supplies row / column l%32 and a contiguous run of the reduction index
//     at (l/32) times the run length; lane l of the accumulator holds column
//     l%32 and rows 8g + 4(l/32) + r, g, r in 0..3, at register 4g + r.
// Every kernel is one or a few wave64 workgroups over caller buffers whose
// sizes the host checks.
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v8i __attribute__((ext_vector_type(8)));
typedef int v16i __attribute__((ext_vector_type(16)));
typedef float v16f __attribute__((ext_vector_type(16)));
typedef __bf16 v8bf __attribute__((ext_vector_type(8)));

// one byte per element: the E2M1 code of x[i] / 2^e (element pairs share a convert)
__global__ __launch_bounds__(256) void cvt_fp4_kernel(const float* __restrict__ x, uint8_t* __restrict__ codes, int npairs,
                                                      float scale) {
  const int p = blockIdx.x * blockDim.x + threadIdx.x;
  if (p >= npairs) return;
  const uint32_t b = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(0u, x[2 * p], x[2 * p + 1], scale, 0) & 0xFFu;
  codes[2 * p] = (uint8_t)(b & 0xF);
  codes[2 * p + 1] = (uint8_t)(b >> 4);
}

__global__ __launch_bounds__(256) void cvt_u8_kernel(const float* __restrict__ x, uint8_t* __restrict__ y, int n) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) y[i] = (uint8_t)(__builtin_amdgcn_cvt_pk_u8_f32(x[i], 0, 0u) & 0xFFu);
}

// the E4M3 byte v_cvt_pk_fp8_f32 makes of x[i], and v_cvt_f32_fp8 of every byte value
__global__ __launch_bounds__(256) void cvt_fp8_kernel(const float* __restrict__ x, uint8_t* __restrict__ y, int n,
                                                      float* __restrict__ dec) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) y[i] = (uint8_t)(__builtin_amdgcn_cvt_pk_fp8_f32(x[i], 0.0f, 0, false) & 0xFF);
  if (i < 256) dec[i] = __builtin_amdgcn_cvt_f32_fp8(i, 0);
}

// bf16 pairs of v_cvt_scalef32_pk_bf16_fp4: code byte c[i] (two E2M1 codes) times scale s[i]
__global__ __launch_bounds__(256) void cvt_bf16_fp4_kernel(const uint8_t* __restrict__ c, const float* __restrict__ s,
                                                           uint32_t* __restrict__ y, int n) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  const auto r = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4((uint32_t)c[i], s[i], 0);
  y[i] = __builtin_bit_cast(uint32_t, r);
}

// f16 pairs of v_cvt_scalef32_pk_f16_fp4: code byte c[i] (two E2M1 codes) times scale s[i]
__global__ __launch_bounds__(256) void cvt_f16_fp4_kernel(const uint8_t* __restrict__ c, const float* __restrict__ s,
                                                          uint32_t* __restrict__ y, int n) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  const auto r = __builtin_amdgcn_cvt_scalef32_pk_f16_fp4((uint32_t)c[i], s[i], 0);
  y[i] = __builtin_bit_cast(uint32_t, r);
}

__global__ __launch_bounds__(256) void exp2_kernel(const float* __restrict__ x, float* __restrict__ y, int n) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) y[i] = __builtin_amdgcn_exp2f(x[i]);
}

// C[32][32] = A[32][64] B[32][64]^T with FP4 codes (one byte per element, low
// nibble) and one E8M0 scale per row and 32-element block; C row-major fp32.
__global__ __launch_bounds__(64) void mfma_fp4_kernel(const uint8_t* __restrict__ a, const uint8_t* __restrict__ as,
                                                      const uint8_t* __restrict__ b, const uint8_t* __restrict__ bs,
                                                      float* __restrict__ c) {
  const int l = threadIdx.x, row = l & 31, h = l >> 5;
  uint32_t wa[4], wb[4];
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    uint32_t xa = 0, xb = 0;
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      xa |= (uint32_t)(a[row * 64 + 32 * h + 8 * w + k] & 0xF) << (4 * k);
      xb |= (uint32_t)(b[row * 64 + 32 * h + 8 * w + k] & 0xF) << (4 * k);
    }
    wa[w] = xa;
    wb[w] = xb;
  }
  const v8i A = v8i{(int)wa[0], (int)wa[1], (int)wa[2], (int)wa[3], 0, 0, 0, 0};
  const v8i B = v8i{(int)wb[0], (int)wb[1], (int)wb[2], (int)wb[3], 0, 0, 0, 0};
  const int sa = as[row * 2 + h], sb = bs[row * 2 + h];
  v16f acc = v16f{};
  acc = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(A, B, acc, 4, 4, 0, sa, 0, sb);
#pragma unroll
  for (int g = 0; g < 4; ++g)
#pragma unroll
    for (int r = 0; r < 4; ++r) c[(8 * g + 4 * h + r) * 32 + row] = acc[4 * g + r];
}

// C[32][32] = A[32][32] B[32][32]^T, int8 operands, int32 C row-major
__global__ __launch_bounds__(64) void mfma_i8_kernel(const int8_t* __restrict__ a, const int8_t* __restrict__ b,
                                                     int* __restrict__ c) {
  const int l = threadIdx.x, row = l & 31, h = l >> 5;
  const v4i A = *reinterpret_cast<const v4i*>(a + row * 32 + 16 * h);
  const v4i B = *reinterpret_cast<const v4i*>(b + row * 32 + 16 * h);
  v16i acc = v16i{};
  acc = __builtin_amdgcn_mfma_i32_32x32x32_i8(A, B, acc, 0, 0, 0);
#pragma unroll
  for (int g = 0; g < 4; ++g)
#pragma unroll
    for (int r = 0; r < 4; ++r) c[(8 * g + 4 * h + r) * 32 + row] = acc[4 * g + r];
}

// C[32][32] = A[32][16] B[32][16]^T, bf16 operands (bits), fp32 C row-major
__global__ __launch_bounds__(64) void mfma_bf16_kernel(const uint16_t* __restrict__ a, const uint16_t* __restrict__ b,
                                                       float* __restrict__ c) {
  const int l = threadIdx.x, row = l & 31, h = l >> 5;
  const v4i A = *reinterpret_cast<const v4i*>(a + row * 16 + 8 * h);
  const v4i B = *reinterpret_cast<const v4i*>(b + row * 16 + 8 * h);
  v16f acc = v16f{};
  acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(v8bf, A), __builtin_bit_cast(v8bf, B), acc, 0, 0, 0);
#pragma unroll
  for (int g = 0; g < 4; ++g)
#pragma unroll
    for (int r = 0; r < 4; ++r) c[(8 * g + 4 * h + r) * 32 + row] = acc[4 * g + r];
}

inline int st(hipError_t e) { return e == hipSuccess ? 0 : 3; }

}  // namespace

extern "C" {

// codes: n bytes (n even, n >= 2); scale: a power of two.  Returns 0, 1 (bad arguments) or 3 (HIP error).
int sage_probe_cvt_fp4(const float* x, uint8_t* codes, int n, float scale, hipStream_t stream) {
  if (!x || !codes || n < 2 || (n & 1)) return 1;
  const int np = n / 2;
  hipLaunchKernelGGL(cvt_fp4_kernel, dim3((unsigned)((np + 255) / 256)), dim3(256), 0, stream, x, codes, np, scale);
  return st(hipGetLastError());
}

// y: n bytes, the byte v_cvt_pk_u8_f32 makes of x[i]
int sage_probe_cvt_u8(const float* x, uint8_t* y, int n, hipStream_t stream) {
  if (!x || !y || n < 1) return 1;
  hipLaunchKernelGGL(cvt_u8_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, stream, x, y, n);
  return st(hipGetLastError());
}

// y: n bytes, the E4M3 byte of x[i]; dec: 256 floats, the decoded value of every byte
int sage_probe_cvt_fp8(const float* x, uint8_t* y, int n, float* dec, hipStream_t stream) {
  if (!x || !y || !dec || n < 256) return 1;
  hipLaunchKernelGGL(cvt_fp8_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, stream, x, y, n, dec);
  return st(hipGetLastError());
}

// y: n words, the two bf16 values (low half: low nibble of c[i]) scaled by s[i]
int sage_probe_cvt_bf16_fp4(const uint8_t* c, const float* s, uint32_t* y, int n, hipStream_t stream) {
  if (!c || !s || !y || n < 1) return 1;
  hipLaunchKernelGGL(cvt_bf16_fp4_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, stream, c, s, y, n);
  return st(hipGetLastError());
}

// y: n words, the two f16 values (low half: low nibble of c[i]) scaled by s[i]
int sage_probe_cvt_f16_fp4(const uint8_t* c, const float* s, uint32_t* y, int n, hipStream_t stream) {
  if (!c || !s || !y || n < 1) return 1;
  hipLaunchKernelGGL(cvt_f16_fp4_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, stream, c, s, y, n);
  return st(hipGetLastError());
}

int sage_probe_exp2(const float* x, float* y, int n, hipStream_t stream) {
  if (!x || !y || n < 1) return 1;
  hipLaunchKernelGGL(exp2_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, stream, x, y, n);
  return st(hipGetLastError());
}

// a, b: 32 x 64 codes (bytes); as, bs: 32 x 2 E8M0 bytes; c: 32 x 32 fp32
int sage_probe_mfma_fp4(const uint8_t* a, const uint8_t* as, const uint8_t* b, const uint8_t* bs, float* c,
                        hipStream_t stream) {
  if (!a || !as || !b || !bs || !c) return 1;
  hipLaunchKernelGGL(mfma_fp4_kernel, dim3(1), dim3(64), 0, stream, a, as, b, bs, c);
  return st(hipGetLastError());
}

// a, b: 32 x 32 int8 (16-byte aligned); c: 32 x 32 int32
int sage_probe_mfma_i8(const int8_t* a, const int8_t* b, int* c, hipStream_t stream) {
  if (!a || !b || !c || ((uintptr_t)a & 15) || ((uintptr_t)b & 15)) return 1;
  hipLaunchKernelGGL(mfma_i8_kernel, dim3(1), dim3(64), 0, stream, a, b, c);
  return st(hipGetLastError());
}

// a, b: 32 x 16 bf16 bits (16-byte aligned); c: 32 x 32 fp32
int sage_probe_mfma_bf16(const uint16_t* a, const uint16_t* b, float* c, hipStream_t stream) {
  if (!a || !b || !c || ((uintptr_t)a & 15) || ((uintptr_t)b & 15)) return 1;
  hipLaunchKernelGGL(mfma_bf16_kernel, dim3(1), dim3(64), 0, stream, a, b, c);
  return st(hipGetLastError());
}

}  // extern "C"
