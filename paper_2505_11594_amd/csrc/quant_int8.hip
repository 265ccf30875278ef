// INT8 per-block quantization psi for the 8-bit attention of SageBwd
// (Algorithms 2 and 3; Sec. 4.1, Eq. psi) on gfx950.
//
// One scale s = max|X| / 127 per block of R consecutive rows with all D
// channels -- R = 128 query rows for Q and dO (the attention kernels' query
// tile), the KV tile (128 or 64 rows) for K and V -- and codes round(x * fl32(1/s)) to the
// nearest integer, ties to even; an all-zero block gets s = 0 and zero codes.
// K is smoothed first: K' = fl32(K - mean_t K) with the exact mean of the
// FP4 path's k-mean kernels.
//
// Layouts: Q^ [BH, N, D] and K^ [BH, Np, D] token-major (rows >= N of K^ are
// zero); V^T [BH, D, Np] transposed, the tokens of every 32-token group
// stored in the order in which the int8 MFMA of P.V receives P from the
// accumulator of S^T = K^ Q^T: position 16h + 4g + r holds token 8g + 4h + r.
// The backward stores Q^, K^ and dO^ transposed the same way (the A operands
// of dK^T = Q^T dS^, dQ^T = K^T dS^T and dV^T = dO^T P^).
//
// One workgroup per block: each thread owns 8 channels of up to 8 rows (one
// 16-byte load each), the block max is reduced across the wave and through
// LDS, and the codes are formed by one add of 1.5 * 2^23, whose fp32 rounding
// is the round-to-nearest-even to an integer (the code is the low byte).
#include "sage_common.h"

namespace sage {

constexpr int I8Q_THREADS = 256;
constexpr float kRoundMagic = 12582912.0f;   // 1.5 * 2^23

// V^T storage position of token offset o inside its 32-token group
__device__ __forceinline__ int i8_v_pos(int o) {
  const int g = o >> 3, h = (o >> 2) & 1, r = o & 3;
  return (h << 4) | (g << 2) | r;
}

// the low bytes of four rounded values, packed (element 0 in the low byte)
__device__ __forceinline__ uint32_t pack_low_bytes(uint32_t a, uint32_t b, uint32_t c, uint32_t d) {
  const uint32_t ab = __builtin_amdgcn_perm(b, a, 0x0C0C0400u);   // [a.b0, b.b0, 0, 0]
  const uint32_t cd = __builtin_amdgcn_perm(d, c, 0x0C0C0400u);
  return __builtin_amdgcn_perm(cd, ab, 0x05040100u);              // [a, b, c, d]
}

// ROLE: 0 = Q, 1 = K, 2 = V (or any tensor stored transposed), 3 = K stored
// transposed (the backward's K^T).  Block b of head bh holds rows [b R, b R + R) of
// the input (rows >= N are zero); nb = blocks per head; Nout = rows of the
// Q^ / K^ output (N or Np), Np = columns of V^T.
template <int D, bool BF16, int ROLE>
__global__ __launch_bounds__(I8Q_THREADS) void quant_i8_kernel(const uint16_t* __restrict__ x,
                                                               const float* __restrict__ mu,
                                                               int8_t* __restrict__ codes, float* __restrict__ scales,
                                                               int N, int Nout, int R, int nb) {
  constexpr int UPR = D / 8;                      // 16-byte units per row
  constexpr int RSTEP = I8Q_THREADS / UPR;        // rows covered by one pass of the workgroup
  constexpr int MAXU = 128 / RSTEP;               // passes for R = 128
  const int b = blockIdx.x, bh = blockIdx.y, tid = threadIdx.x;
  const int cg = tid % UPR, rsub = tid / UPR;     // this thread's channels [8 cg, +8) and first row
  const int r0 = b * R;

  float m8[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) m8[i] = ((ROLE == 1 || ROLE == 3) && mu != nullptr) ? mu[(size_t)bh * D + cg * 8 + i] : 0.0f;

  float v[MAXU][8];
  float amax = 0.0f;
#pragma unroll
  for (int u = 0; u < MAXU; ++u) {
    const int row = rsub + u * RSTEP, t = r0 + row;
    if (row < R && t < N) {
      const uint4 raw = *reinterpret_cast<const uint4*>(x + ((size_t)bh * N + t) * D + cg * 8);
      const uint16_t* h = reinterpret_cast<const uint16_t*>(&raw);
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        float a = widen<BF16>(h[i]);
        if (ROLE == 1 || ROLE == 3) a = a - m8[i];
        v[u][i] = a;
        amax = __builtin_fmaxf(amax, __builtin_fabsf(a));
      }
    } else {
#pragma unroll
      for (int i = 0; i < 8; ++i) v[u][i] = 0.0f;
    }
  }
  // block max: across the wave, then across the 4 waves
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) amax = __builtin_fmaxf(amax, __shfl_xor(amax, off, 64));
  __shared__ float red[I8Q_THREADS / 64];
  if ((tid & 63) == 0) red[tid >> 6] = amax;
  __syncthreads();
  amax = __builtin_fmaxf(__builtin_fmaxf(red[0], red[1]), __builtin_fmaxf(red[2], red[3]));
  const float s = amax / 127.0f;                  // correctly rounded division
  const float r = amax > 0.0f ? 1.0f / s : 0.0f;  // a zero block: codes 0
  if (tid == 0) scales[(size_t)bh * nb + b] = s;

  if constexpr (ROLE == 0 || ROLE == 1) {
#pragma unroll
    for (int u = 0; u < MAXU; ++u) {
      const int row = rsub + u * RSTEP, t = r0 + row;
      if (row < R && t < Nout) {
        uint32_t w[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) w[i] = __float_as_uint(v[u][i] * r + kRoundMagic);
        const uint2 out = make_uint2(pack_low_bytes(w[0], w[1], w[2], w[3]), pack_low_bytes(w[4], w[5], w[6], w[7]));
        *reinterpret_cast<uint2*>(codes + ((size_t)bh * Nout + t) * D + cg * 8) = out;
      }
    }
  } else {
    // transpose through LDS: tr[c][position of the row]
    __shared__ __attribute__((aligned(16))) uint8_t tr[D][128];
#pragma unroll
    for (int u = 0; u < MAXU; ++u) {
      const int row = rsub + u * RSTEP;
      if (row < R) {
        const int p = (row & ~31) | i8_v_pos(row & 31);
#pragma unroll
        for (int i = 0; i < 8; ++i) tr[cg * 8 + i][p] = (uint8_t)__float_as_uint(v[u][i] * r + kRoundMagic);
      }
    }
    __syncthreads();
    const int chunks = R / 16;                    // 16-byte pieces per channel row
    for (int idx = tid; idx < D * chunks; idx += I8Q_THREADS) {
      const int c = idx / chunks, part = idx % chunks;
      *reinterpret_cast<uint4*>(codes + ((size_t)bh * D + c) * Nout + r0 + 16 * part) =
          *reinterpret_cast<const uint4*>(&tr[c][16 * part]);
    }
  }
}

// role: 0 Q (R must be 128, Nout = N), 1 K (Nout = Np), 2 V or any tensor
// transposed (Nout = Np, the row length of the transposed output), 3 K
// transposed.  nb = blocks per head: ceil(N / 128) for Q, Np / R otherwise.
hipError_t launch_quant_i8(const void* x, const float* mu, void* codes, float* scales, int BH, int N, int Nout,
                           int D, int R, int role, bool bf16, hipStream_t st) {
  const int nb = role == 0 ? (N + R - 1) / R : Nout / R;
  const dim3 grid((unsigned)nb, (unsigned)BH), block(I8Q_THREADS);
  const uint16_t* xp = static_cast<const uint16_t*>(x);
  int8_t* cp = static_cast<int8_t*>(codes);
#define SAGE_Q8(DD, BB, RR) \
  hipLaunchKernelGGL((quant_i8_kernel<DD, BB, RR>), grid, block, 0, st, xp, mu, cp, scales, N, Nout, R, nb)
#define SAGE_Q8R(DD, BB)                      \
  do {                                        \
    if (role == 0) SAGE_Q8(DD, BB, 0);        \
    else if (role == 1) SAGE_Q8(DD, BB, 1);   \
    else if (role == 2) SAGE_Q8(DD, BB, 2);   \
    else SAGE_Q8(DD, BB, 3);                  \
  } while (0)
  if (D == 128) { if (bf16) SAGE_Q8R(128, true); else SAGE_Q8R(128, false); }
  else { if (bf16) SAGE_Q8R(64, true); else SAGE_Q8R(64, false); }
#undef SAGE_Q8R
#undef SAGE_Q8
  return hipGetLastError();
}

}  // namespace sage
