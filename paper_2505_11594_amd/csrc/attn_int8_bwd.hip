// Backward pass of the 8-bit attention of SageBwd (Algorithm 3) for gfx950.
//
// Four of the five products run on v_mfma_i32_32x32x32_i8 with per-block INT8
// operands (psi, Sec. 4.1): S = MM(Q^, K^) s_Q s_K, dV += MM(P^T, dO^) s_P s_dO,
// dQ += MM(dS^, K^) s_dS s_K / sqrt(D) and dK += MM(dS^T, Q^) s_dS s_Q / sqrt(D);
// dP = MM(dO, V^T) stays in 16-bit inputs (v_mfma_f32_32x32x16_bf16 / _f16,
// fp32 accumulation).  P = exp(S/sqrt(D) - L) uses the forward's L, dS =
// P (dP - D) with D = rowsum(dO O), and dQ gets rowsum(dS) K_m / sqrt(D) for
// the smoothing of K.  psi of P and dS is per (128 query x 128 key) block,
// psi of dO per 128-row block, as the forward's Q^.
//
// Two deterministic kernels (no atomics):
//  - dK/dV: a workgroup owns 128 keys (4 waves x 32) and walks the query
//    blocks.  S = Q^ K^T puts a key in each lane's column and 16 queries in its
//    rows, so P^ and dS^ of a 32-query subtile are, as they stand, the B
//    operands of dV^T = dO^T P^ and dK^T = Q^T dS^ (A = dO^T / Q^T rows with
//    each 32-query group permuted as V^T in the forward).  The block scales
//    of P and dS need the block's maxima before any code is formed: P and dS
//    of the whole block stay in registers while the maxima are reduced across
//    the waves through LDS, then all codes are formed and each channel
//    block's two products run over the block's four subtiles.
//  - dQ: a workgroup owns 128 queries (4 waves x 32) and walks the KV blocks.
//    S^T = K^ Q^T puts a query in each lane's column; dS of the block stays in
//    registers while its maximum is reduced across the waves, and dS^ is the B
//    operand of dQ^T = K^T dS^T (A = K^T rows, permuted the same way).
// Both run one wave per SIMD (the int32 and fp32 accumulators of two
// products do not fit two waves' register budget).  Each workgroup stages the
// operands its four waves share -- a query block (Q^, dO, L, D and the
// transposed Q^, dO^) for dK/dV, a KV block (K^, V, K^T) for dQ -- in LDS in
// MFMA-operand order with global loads that write LDS, one block ahead of
// the block being computed.
#include "sage_common.h"

typedef int v16i __attribute__((ext_vector_type(16)));
typedef _Float16 v8h __attribute__((ext_vector_type(8)));

namespace sage {

constexpr int BW_Q = 128;    // query block (psi(Q), psi(dO), P and dS blocks)
constexpr int BW_K = 128;    // key block
constexpr float kBwRoundMagic = 12582912.0f;   // 1.5 * 2^23

template <bool BF16>
__device__ __forceinline__ v16f mfma16(const v4i a, const v4i b, v16f c) {
  if constexpr (BF16) return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(v8bf, a), __builtin_bit_cast(v8bf, b), c, 0, 0, 0);
  else return __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(v8h, a), __builtin_bit_cast(v8h, b), c, 0, 0, 0);
}

__device__ __forceinline__ int bw_pack4(float a, float b, float c, float d) {
  const uint32_t ab = __builtin_amdgcn_perm(__float_as_uint(b), __float_as_uint(a), 0x0C0C0400u);
  const uint32_t cd = __builtin_amdgcn_perm(__float_as_uint(d), __float_as_uint(c), 0x0C0C0400u);
  return (int)__builtin_amdgcn_perm(cd, ab, 0x05040100u);
}

// 16 values -> 16 int8 codes rint(x r) in value order (v = 4g + r -> byte v)
__device__ __forceinline__ v4i bw_codes(const float (&x)[16], float r) {
  int w[4];
#pragma unroll
  for (int g = 0; g < 4; ++g)
    w[g] = bw_pack4(x[4 * g] * r + kBwRoundMagic, x[4 * g + 1] * r + kBwRoundMagic,
                    x[4 * g + 2] * r + kBwRoundMagic, x[4 * g + 3] * r + kBwRoundMagic);
  return v4i{w[0], w[1], w[2], w[3]};
}

__device__ __forceinline__ float wave_max(float x) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) x = __builtin_fmaxf(x, __shfl_xor(x, off, 64));
  return x;
}

// ---------------------------------------------------------------------------
// D_q = sum_d dO[q,d] O[q,d] (fp32) and Lb_q = L_q log2(e), for q < N; rows
// [N, Np) get 0.  D/8 lanes per row, 8 elements each.
// ---------------------------------------------------------------------------
template <int D, bool BF16>
__global__ __launch_bounds__(256) void i8_bwd_prep_kernel(const uint16_t* __restrict__ dout, const float* __restrict__ o,
                                                          const float* __restrict__ lse, float* __restrict__ drow,
                                                          float* __restrict__ lb, int N, int Np, long long rows,
                                                          float log2e) {
  constexpr int LPR = D / 8;
  const long long t = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  const long long row = t / LPR;                   // (bh, q) over Np rows per head
  const int part = (int)(t % LPR);
  if (row >= rows) return;                         // whole rows: LPR divides the block size
  const long long bh = row / Np;
  const int q = (int)(row % Np);
  float s = 0.0f;
  if (q < N) {
    const size_t e = ((size_t)bh * N + q) * D + part * 8;
    const uint4 g = *reinterpret_cast<const uint4*>(dout + e);
    const uint16_t* gh = reinterpret_cast<const uint16_t*>(&g);
    const float4 o0 = *reinterpret_cast<const float4*>(o + e);
    const float4 o1 = *reinterpret_cast<const float4*>(o + e + 4);
    const float ov[8] = {o0.x, o0.y, o0.z, o0.w, o1.x, o1.y, o1.z, o1.w};
#pragma unroll
    for (int i = 0; i < 8; ++i) s = __builtin_fmaf(widen<BF16>(gh[i]), ov[i], s);
  }
#pragma unroll
  for (int off = LPR / 2; off >= 1; off >>= 1) s += __shfl_xor(s, off, 64);
  if (part == 0) {
    drow[row] = s;
    lb[row] = q < N ? lse[(size_t)bh * N + q] * log2e : 0.0f;
  }
}

__device__ __forceinline__ void bw_lds_load16(const void* src, void* dst) {
  __builtin_amdgcn_global_load_lds(src, (__attribute__((address_space(3))) void*)dst, 16, 0, 0);
}
__device__ __forceinline__ void bw_wait_all() { __builtin_amdgcn_s_waitcnt(0x0F70); }   // vmcnt(0)
// vmcnt(n) for the counts used below (n < 16: the low field of the immediate)
template <int N>
__device__ __forceinline__ void bw_wait_vm() {
  static_assert(N >= 0 && N < 16, "vmcnt field");
  __builtin_amdgcn_s_waitcnt(0x0F70 | N);
}

// LDS of the dK/dV kernel: per query block, in MFMA-operand order (1 KiB per
// 64-lane operand read, lane l's 16 bytes at 16 l):
//   A stage (double-buffered): Q^ operand blocks (u, s) -- rows q0 + 32u + col,
//   channels [32s + 16hi, +16) --, dO operand blocks (u, s16) -- channels
//   [16s16 + 8hi, +8) --, and the block's Lb and D (128 floats each);
//   T (single): Q^T and dO^T operand blocks (db, u) -- channel rows 32db +
//   col, queries [32u + 16hi, +16) of the block.
template <int D>
struct BwKvLds {
  static constexpr int NKS = D / 32, NKS16 = D / 16, NDB = D / 32;
  static constexpr int NQA = 4 * NKS, NGA = 4 * NKS16, NT = NDB * 4;
  static constexpr int QA_OFF = 0, GA_OFF = NQA * 1024, LD_OFF = GA_OFF + NGA * 1024, A_BYTES = LD_OFF + 1024;
  static constexpr int QT_OFF = 0, GT_OFF = NT * 1024, T_BYTES = 2 * NT * 1024;
  static constexpr int AJ = (NQA + NGA) / 4, TJ = 2 * NT / 4;   // loads per wave
  static_assert((NQA + NGA) % 4 == 0 && (2 * NT) % 4 == 0, "even split over 4 waves");
};

// ---------------------------------------------------------------------------
// dK, dV.  qc/kc: Q^, K^ row-major; qt, gt: Q^T, dO^T int8 [BH, D, Np] with
// each 32-query group permuted; qs, gs: s_Q, s_dO per 128 rows; ks: s_K per
// 128 keys; v, dout: 16-bit [BH, N, D]; drow, lb: [BH, Np].
// ---------------------------------------------------------------------------
template <int D, bool CAUSAL, bool BF16>
__global__ __launch_bounds__(256, 1) void attn_i8_bwd_dkdv_kernel(
    const int8_t* __restrict__ qc, const float* __restrict__ qs, const int8_t* __restrict__ qt,
    const int8_t* __restrict__ kc, const float* __restrict__ ks, const uint16_t* __restrict__ v,
    const uint16_t* __restrict__ dout, const int8_t* __restrict__ gt, const float* __restrict__ gs,
    const float* __restrict__ drow, const float* __restrict__ lb, float* __restrict__ dk, float* __restrict__ dv,
    int N, int Np, int nqb, float c2, float rsd) {
  using T = BwKvLds<D>;
  constexpr int NKS = T::NKS, NKS16 = T::NKS16, NDB = T::NDB;
  __shared__ __attribute__((aligned(16))) uint8_t ldsA[2][T::A_BYTES];
  __shared__ __attribute__((aligned(16))) uint8_t ldsT[T::T_BYTES];
  __shared__ float red[2][2][4];                   // [block parity][P, dS][wave]
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int col = lane & 31, hi = lane >> 5;
  const int kblk = blockIdx.x, bh = blockIdx.y;
  const int kb = kblk * BW_K, kw = kb + 32 * wave, key = kw + col;
  const float sK = ks[(size_t)bh * (Np / BW_K) + kblk];

  // B operands of this wave's 32 keys: K^ (channels [32s + 16hi, +16)) and V
  // (16-bit, channels [16s + 8hi, +8))
  v4i kreg[NKS], vreg[NKS16];
  {
    const int8_t* kr = kc + ((size_t)bh * Np + key) * D;
#pragma unroll
    for (int s = 0; s < NKS; ++s) kreg[s] = *reinterpret_cast<const v4i*>(kr + 32 * s + 16 * hi);
    const uint16_t* vr = v + ((size_t)bh * N + key) * D;
#pragma unroll
    for (int s = 0; s < NKS16; ++s)
      vreg[s] = key < N ? *reinterpret_cast<const v4i*>(vr + 16 * s + 8 * hi) : v4i{0, 0, 0, 0};
  }
  v16f dva[NDB], dka[NDB];
#pragma unroll
  for (int db = 0; db < NDB; ++db) { dva[db] = v16f{}; dka[db] = v16f{}; }

  // loads of query block i: wave w takes operand blocks w, w + 4, ...; rows
  // >= N read row N - 1 (those entries are masked)
  auto issue_A = [&](int i, int buf) {
    const int q0 = i * BW_Q;
    uint8_t* L = ldsA[buf];
#pragma unroll
    for (int k = 0; k < T::AJ; ++k) {
      const int b = wave + 4 * k;
      if (b < T::NQA) {
        const int u = b / NKS, s = b % NKS;
        const int q = min(q0 + 32 * u + col, N - 1);
        bw_lds_load16(qc + ((size_t)bh * N + q) * D + 32 * s + 16 * hi, L + T::QA_OFF + b * 1024);
      } else {
        const int g = b - T::NQA, u = g / NKS16, s = g % NKS16;
        const int q = min(q0 + 32 * u + col, N - 1);
        bw_lds_load16(dout + ((size_t)bh * N + q) * D + 16 * s + 8 * hi, L + T::GA_OFF + g * 1024);
      }
    }
  };
  auto issue_LD = [&](int i, int buf) {          // Lb and D of block i (wave 0)
    const int q0 = i * BW_Q;
    const float* src = (lane < 32 ? lb + (size_t)bh * Np + q0 + 4 * lane : drow + (size_t)bh * Np + q0 + 4 * (lane - 32));
    bw_lds_load16(src, ldsA[buf] + T::LD_OFF);
  };
  auto issue_T = [&](int i) {
    const int q0 = i * BW_Q;
#pragma unroll
    for (int k = 0; k < T::TJ; ++k) {
      const int b = wave + 4 * k, which = b / T::NT, t = b % T::NT, db = t / 4, u = t % 4;
      const size_t off = ((size_t)bh * D + 32 * db + col) * Np + q0 + 32 * u + 16 * hi;
      bw_lds_load16((which ? gt : qt) + off, ldsT + (which ? T::GT_OFF : T::QT_OFF) + t * 1024);
    }
  };

  const int i0 = CAUSAL ? kb / BW_Q : 0;
  if (wave == 0) issue_LD(i0, i0 & 1);
  issue_A(i0, i0 & 1);
  for (int i = i0; i < nqb; ++i) {
    const int q0 = i * BW_Q, a = i & 1;
    bw_wait_all();                                 // this wave's loads of block i have landed
    __syncthreads();                               // everyone's; every wave is done with block i - 1
    if (i + 1 < nqb && wave == 0) issue_LD(i + 1, a ^ 1);
    issue_T(i);
    if (i + 1 < nqb) issue_A(i + 1, a ^ 1);
    const uint8_t* L = ldsA[a];
    const float sQ = qs[(size_t)bh * nqb + i];
    const float ct = __builtin_fmaxf(sQ * sK * c2, 1.17549435e-38f);   // see the forward kernel
    const bool need_mask = (q0 + BW_Q > N) || (kb + BW_K > N) || (CAUSAL && q0 < kb + BW_K - 1);

    // S (exact int32) and dP (fp32) of one 32-query subtile
    auto products = [&](int u, v16i& sacc, v16f& dp) {
      sacc = v16i{};
#pragma unroll
      for (int s = 0; s < NKS; ++s)
        sacc = __builtin_amdgcn_mfma_i32_32x32x32_i8(
            *reinterpret_cast<const v4i*>(L + T::QA_OFF + (u * NKS + s) * 1024 + lane * 16), kreg[s], sacc, 0, 0, 0);
      dp = v16f{};
#pragma unroll
      for (int s = 0; s < NKS16; ++s)
        dp = mfma16<BF16>(*reinterpret_cast<const v4i*>(L + T::GA_OFF + (u * NKS16 + s) * 1024 + lane * 16), vreg[s], dp);
    };
    // P and dS of the subtile: element v is query q0 + 32u + 8(v>>2) + 4hi + (v&3)
    auto softmax_grad = [&](int u, const v16i& sacc, const v16f& dp, float (&P)[16], float (&dS)[16]) {
      const int qb4 = q0 + 32 * u + 4 * hi;
      const float* lbr = reinterpret_cast<const float*>(L + T::LD_OFF) + 32 * u + 4 * hi;
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const v4f l4 = *reinterpret_cast<const v4f*>(lbr + 8 * g);
        const v4f d4 = *reinterpret_cast<const v4f*>(lbr + 128 + 8 * g);
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int e = 4 * g + r;
          float arg = __builtin_fmaf((float)sacc[e], ct, -l4[r]);
          if (need_mask) {
            // visible iff q < N, key < N and (causal) key <= q: the three sign bits
            const int q = qb4 + 8 * g + r;
            int m = (q - N) & (key - N);
            if (CAUSAL) m &= ~(q - key);
            arg = __builtin_fminf(arg, __uint_as_float(0xFF800000u ^ ((uint32_t)m & 0x80000000u)));
          }
          const float p = __builtin_amdgcn_exp2f(arg);
          const float d = dp[e] - d4[r];
          P[e] = p;
          dS[e] = p * d;
        }
      }
    };

    // P and dS of the whole block stay in registers (4 subtiles x 16 values)
    // while the block maxima of P and |dS| are reduced across the waves; the
    // products of subtile u + 1 are issued before the softmax work of subtile u
    float P[BW_Q / 32][16], dS[BW_Q / 32][16];
    float pm = 0.0f, dm = 0.0f;
    v16i sacc[2];
    v16f dp[2];
    products(0, sacc[0], dp[0]);
#pragma unroll
    for (int u = 0; u < BW_Q / 32; ++u) {
      if (u + 1 < BW_Q / 32) products(u + 1, sacc[(u + 1) & 1], dp[(u + 1) & 1]);
      softmax_grad(u, sacc[u & 1], dp[u & 1], P[u], dS[u]);
#pragma unroll
      for (int e = 0; e < 16; ++e) { pm = __builtin_fmaxf(pm, P[u][e]); dm = __builtin_fmaxf(dm, __builtin_fabsf(dS[u][e])); }
      __builtin_amdgcn_sched_barrier(0);
    }
    pm = wave_max(pm);
    dm = wave_max(dm);
    if (lane == 0) { red[a][0][wave] = pm; red[a][1][wave] = dm; }
    // the T loads of this block were issued before the next block's A loads
    if (i + 1 < nqb) bw_wait_vm<T::AJ>();
    else bw_wait_all();
    __syncthreads();
    pm = __builtin_fmaxf(__builtin_fmaxf(red[a][0][0], red[a][0][1]), __builtin_fmaxf(red[a][0][2], red[a][0][3]));
    dm = __builtin_fmaxf(__builtin_fmaxf(red[a][1][0], red[a][1][1]), __builtin_fmaxf(red[a][1][2], red[a][1][3]));
    const float sP = pm / 127.0f, rP = pm > 0.0f ? 1.0f / sP : 0.0f;
    const float sdS = dm / 127.0f, rdS = dm > 0.0f ? 1.0f / sdS : 0.0f;

    // codes of the block, then per channel block the two int8 products over
    // its four subtiles (exact int32), folded into fp32 once per block
    v4i pc[BW_Q / 32], sc[BW_Q / 32];
#pragma unroll
    for (int u = 0; u < BW_Q / 32; ++u) { pc[u] = bw_codes(P[u], rP); sc[u] = bw_codes(dS[u], rdS); }
    const float fv = sP * gs[(size_t)bh * nqb + i];
    const float fk = (sdS * sQ) * rsd;
#pragma unroll
    for (int db = 0; db < NDB; ++db) {
      v16i dvi = v16i{}, dki = v16i{};
#pragma unroll
      for (int u = 0; u < BW_Q / 32; ++u) {
        const v4i ga = *reinterpret_cast<const v4i*>(ldsT + T::GT_OFF + (db * 4 + u) * 1024 + lane * 16);
        const v4i qa = *reinterpret_cast<const v4i*>(ldsT + T::QT_OFF + (db * 4 + u) * 1024 + lane * 16);
        dvi = __builtin_amdgcn_mfma_i32_32x32x32_i8(ga, pc[u], dvi, 0, 0, 0);
        dki = __builtin_amdgcn_mfma_i32_32x32x32_i8(qa, sc[u], dki, 0, 0, 0);
      }
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        dva[db][e] = __builtin_fmaf((float)dvi[e], fv, dva[db][e]);
        dka[db][e] = __builtin_fmaf((float)dki[e], fk, dka[db][e]);
      }
    }
  }

  // dV^T, dK^T: lane holds key kw + col and channels 32db + 8g + 4hi + r
  if (key < N) {
#pragma unroll
    for (int db = 0; db < NDB; ++db)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const size_t idx = ((size_t)bh * N + key) * D + 32 * db + 8 * g + 4 * hi;
        *reinterpret_cast<float4*>(dv + idx) = make_float4(dva[db][4 * g], dva[db][4 * g + 1], dva[db][4 * g + 2], dva[db][4 * g + 3]);
        *reinterpret_cast<float4*>(dk + idx) = make_float4(dka[db][4 * g], dka[db][4 * g + 1], dka[db][4 * g + 2], dka[db][4 * g + 3]);
      }
  }
}

// LDS of the dQ kernel: per KV block (double-buffered), in operand order:
// K^ blocks (t, s) -- key rows kb + 32t + col, channels [32s + 16hi, +16) --,
// V blocks (t, s16) -- channels [16s16 + 8hi, +8) --, K^T blocks (db, t) --
// channel rows 32db + col, keys [32t + 16hi, +16) of the block.
template <int D>
struct BwQLds {
  static constexpr int NKS = D / 32, NKS16 = D / 16, NDB = D / 32, NT = BW_K / 32;
  static constexpr int NKA = NT * NKS, NVA = NT * NKS16, NKT = NDB * NT;
  static constexpr int KA_OFF = 0, VA_OFF = NKA * 1024, KT_OFF = VA_OFF + NVA * 1024, BYTES = KT_OFF + NKT * 1024;
  static constexpr int J = (NKA + NVA + NKT) / 4;
  static_assert((NKA + NVA + NKT) % 4 == 0, "even split over 4 waves");
};

// ---------------------------------------------------------------------------
// dQ.  kt: K^T int8 [BH, D, Np] with each 32-key group permuted; kmean: K_m
// [BH, D] or null (no smoothing).
// ---------------------------------------------------------------------------
template <int D, bool CAUSAL, bool BF16>
__global__ __launch_bounds__(256, 1) void attn_i8_bwd_dq_kernel(
    const int8_t* __restrict__ qc, const float* __restrict__ qs, const int8_t* __restrict__ kc,
    const float* __restrict__ ks, const int8_t* __restrict__ kt, const uint16_t* __restrict__ v,
    const uint16_t* __restrict__ dout, const float* __restrict__ drow, const float* __restrict__ lb,
    const float* __restrict__ kmean, float* __restrict__ dq, int N, int Np, int nqb, float c2, float rsd) {
  using T = BwQLds<D>;
  constexpr int NKS = T::NKS, NKS16 = T::NKS16, NDB = T::NDB, NT = T::NT;
  __shared__ __attribute__((aligned(16))) uint8_t lds[2][T::BYTES];
  __shared__ __attribute__((aligned(16))) float kms[D];
  __shared__ float red[2][4];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int col = lane & 31, hi = lane >> 5;
  const int i = blockIdx.x, bh = blockIdx.y;
  const int q0 = i * BW_Q, qw = q0 + 32 * wave, qi = qw + col;
  const float sQ = qs[(size_t)bh * nqb + i];
  const float lbq = lb[(size_t)bh * Np + qi], dq_row = drow[(size_t)bh * Np + qi];
  if (tid < D) kms[tid] = kmean != nullptr ? kmean[(size_t)bh * D + tid] : 0.0f;

  v4i qreg[NKS], greg[NKS16];
  {
    const int8_t* qr = qc + ((size_t)bh * N + qi) * D;
    const uint16_t* gr = dout + ((size_t)bh * N + qi) * D;
#pragma unroll
    for (int s = 0; s < NKS; ++s) qreg[s] = qi < N ? *reinterpret_cast<const v4i*>(qr + 32 * s + 16 * hi) : v4i{0, 0, 0, 0};
#pragma unroll
    for (int s = 0; s < NKS16; ++s) greg[s] = qi < N ? *reinterpret_cast<const v4i*>(gr + 16 * s + 8 * hi) : v4i{0, 0, 0, 0};
  }
  v16f dqa[NDB];
#pragma unroll
  for (int db = 0; db < NDB; ++db) dqa[db] = v16f{};

  // loads of KV block j: wave w takes operand blocks w, w + 4, ...; V rows
  // >= N read row N - 1 (those keys are masked)
  auto issue = [&](int j, int buf) {
    const int kb = j * BW_K;
    uint8_t* L = lds[buf];
#pragma unroll
    for (int k = 0; k < T::J; ++k) {
      const int b = wave + 4 * k;
      if (b < T::NKA) {
        const int t = b / NKS, s = b % NKS;
        bw_lds_load16(kc + ((size_t)bh * Np + kb + 32 * t + col) * D + 32 * s + 16 * hi, L + T::KA_OFF + b * 1024);
      } else if (b < T::NKA + T::NVA) {
        const int g = b - T::NKA, t = g / NKS16, s = g % NKS16;
        const int kr = min(kb + 32 * t + col, N - 1);
        bw_lds_load16(v + ((size_t)bh * N + kr) * D + 16 * s + 8 * hi, L + T::VA_OFF + g * 1024);
      } else {
        const int g = b - T::NKA - T::NVA, db = g / NT, t = g % NT;
        bw_lds_load16(kt + ((size_t)bh * D + 32 * db + col) * Np + kb + 32 * t + 16 * hi, L + T::KT_OFF + g * 1024);
      }
    }
  };

  int nkb = (N + BW_K - 1) / BW_K;
  if (CAUSAL) nkb = min(nkb, min(q0 + BW_Q - 1, N - 1) / BW_K + 1);
  issue(0, 0);
  for (int j = 0; j < nkb; ++j) {
    const int kb = j * BW_K, buf = j & 1;
    bw_wait_all();
    __syncthreads();                               // block j has landed; every wave is done with block j - 1
    if (j + 1 < nkb) issue(j + 1, buf ^ 1);
    const uint8_t* L = lds[buf];
    const float sK = ks[(size_t)bh * (Np / BW_K) + j];
    const float ct = __builtin_fmaxf(sQ * sK * c2, 1.17549435e-38f);
    const bool need_mask = (q0 + BW_Q > N) || (kb + BW_K > N) || (CAUSAL && kb + BW_K - 1 > q0);
    float dS[NT][16];
    float dm = 0.0f, rs = 0.0f;
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      v16i sacc = v16i{};
#pragma unroll
      for (int s = 0; s < NKS; ++s)
        sacc = __builtin_amdgcn_mfma_i32_32x32x32_i8(
            *reinterpret_cast<const v4i*>(L + T::KA_OFF + (t * NKS + s) * 1024 + lane * 16), qreg[s], sacc, 0, 0, 0);
      v16f dp = v16f{};
#pragma unroll
      for (int s = 0; s < NKS16; ++s)
        dp = mfma16<BF16>(*reinterpret_cast<const v4i*>(L + T::VA_OFF + (t * NKS16 + s) * 1024 + lane * 16), greg[s], dp);
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        float arg = __builtin_fmaf((float)sacc[e], ct, -lbq);
        if (need_mask) {
          const int k = kb + 32 * t + 8 * (e >> 2) + 4 * hi + (e & 3);
          int m = (qi - N) & (k - N);
          if (CAUSAL) m &= ~(qi - k);
          arg = __builtin_fminf(arg, __uint_as_float(0xFF800000u ^ ((uint32_t)m & 0x80000000u)));
        }
        const float p = __builtin_amdgcn_exp2f(arg);
        const float d = dp[e] - dq_row;
        const float x = p * d;
        dS[t][e] = x;
        rs += x;
        dm = __builtin_fmaxf(dm, __builtin_fabsf(x));
      }
    }
    dm = wave_max(dm);
    if (lane == 0) red[buf][wave] = dm;
    __syncthreads();
    dm = __builtin_fmaxf(__builtin_fmaxf(red[buf][0], red[buf][1]), __builtin_fmaxf(red[buf][2], red[buf][3]));
    const float sdS = dm / 127.0f, rdS = dm > 0.0f ? 1.0f / sdS : 0.0f;
    v16i dqi[NDB];
#pragma unroll
    for (int db = 0; db < NDB; ++db) dqi[db] = v16i{};
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      const v4i sc = bw_codes(dS[t], rdS);
#pragma unroll
      for (int db = 0; db < NDB; ++db)
        dqi[db] = __builtin_amdgcn_mfma_i32_32x32x32_i8(
            *reinterpret_cast<const v4i*>(L + T::KT_OFF + (db * NT + t) * 1024 + lane * 16), sc, dqi[db], 0, 0, 0);
    }
    const float fq = (sdS * sK) * rsd;
    const float rr = (rs + __shfl_xor(rs, 32, 64)) * rsd;   // rowsum(dS) of this lane's query, / sqrt(D)
#pragma unroll
    for (int db = 0; db < NDB; ++db)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const v4f km = *reinterpret_cast<const v4f*>(kms + 32 * db + 8 * g + 4 * hi);
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int e = 4 * g + r;
          float x = __builtin_fmaf((float)dqi[db][e], fq, dqa[db][e]);
          if (kmean != nullptr) x = __builtin_fmaf(rr, km[r], x);
          dqa[db][e] = x;
        }
      }
  }
  if (qi < N) {
#pragma unroll
    for (int db = 0; db < NDB; ++db)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const size_t idx = ((size_t)bh * N + qi) * D + 32 * db + 8 * g + 4 * hi;
        *reinterpret_cast<float4*>(dq + idx) = make_float4(dqa[db][4 * g], dqa[db][4 * g + 1], dqa[db][4 * g + 2], dqa[db][4 * g + 3]);
      }
  }
}

hipError_t launch_i8_bwd_prep(const void* dout, const float* o, const float* lse, float* drow, float* lb, int BH,
                              int N, int Np, int D, bool bf16, hipStream_t st) {
  const long long rows = (long long)BH * Np;
  const long long threads = rows * (D / 8);
  const dim3 grid((unsigned)((threads + 255) / 256)), block(256);
  const float log2e = 1.44269504088896340736f;
  const uint16_t* g = static_cast<const uint16_t*>(dout);
  if (D == 128) {
    if (bf16) hipLaunchKernelGGL((i8_bwd_prep_kernel<128, true>), grid, block, 0, st, g, o, lse, drow, lb, N, Np, rows, log2e);
    else hipLaunchKernelGGL((i8_bwd_prep_kernel<128, false>), grid, block, 0, st, g, o, lse, drow, lb, N, Np, rows, log2e);
  } else {
    if (bf16) hipLaunchKernelGGL((i8_bwd_prep_kernel<64, true>), grid, block, 0, st, g, o, lse, drow, lb, N, Np, rows, log2e);
    else hipLaunchKernelGGL((i8_bwd_prep_kernel<64, false>), grid, block, 0, st, g, o, lse, drow, lb, N, Np, rows, log2e);
  }
  return hipGetLastError();
}

template <int D, bool CAUSAL, bool BF16>
static hipError_t launch_bwd_t(const int8_t* qc, const float* qs, const int8_t* qt, const int8_t* kc, const float* ks,
                               const int8_t* kt, const uint16_t* v, const uint16_t* dout, const int8_t* gt,
                               const float* gs, const float* drow, const float* lb, const float* kmean, float* dq,
                               float* dk, float* dv, int BH, int N, int Np, float c2, float rsd, hipStream_t st) {
  const int nqb = (N + BW_Q - 1) / BW_Q;
  hipLaunchKernelGGL((attn_i8_bwd_dkdv_kernel<D, CAUSAL, BF16>), dim3((unsigned)(Np / BW_K), (unsigned)BH), dim3(256), 0,
                     st, qc, qs, qt, kc, ks, v, dout, gt, gs, drow, lb, dk, dv, N, Np, nqb, c2, rsd);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((attn_i8_bwd_dq_kernel<D, CAUSAL, BF16>), dim3((unsigned)nqb, (unsigned)BH), dim3(256), 0, st, qc,
                     qs, kc, ks, kt, v, dout, drow, lb, kmean, dq, N, Np, nqb, c2, rsd);
  return hipGetLastError();
}

// Q^ [BH, N, D], K^ [BH, Np, D] row-major; Q^T, K^T, dO^T [BH, D, Np] permuted
// per 32 rows; scales per 128 rows; kmean null without smoothing.
hipError_t launch_attn_int8_bwd(const void* qc, const float* qs, const void* qt, const void* kc, const float* ks,
                                const void* kt, const void* v, const void* dout, const void* gt, const float* gs,
                                const float* drow, const float* lb, const float* kmean, float* dq, float* dk, float* dv,
                                int BH, int N, int Np, int D, bool causal, bool bf16, float c2, float rsd,
                                hipStream_t st) {
  const int8_t *a = (const int8_t*)qc, *b = (const int8_t*)qt, *c = (const int8_t*)kc, *d = (const int8_t*)kt,
               *g = (const int8_t*)gt;
  const uint16_t *vv = (const uint16_t*)v, *gg = (const uint16_t*)dout;
#define SAGE_BW(DD, CC, BB) \
  return launch_bwd_t<DD, CC, BB>(a, qs, b, c, ks, d, vv, gg, g, gs, drow, lb, kmean, dq, dk, dv, BH, N, Np, c2, rsd, st)
  if (D == 128) {
    if (causal) { if (bf16) SAGE_BW(128, true, true); else SAGE_BW(128, true, false); }
    else { if (bf16) SAGE_BW(128, false, true); else SAGE_BW(128, false, false); }
  } else {
    if (causal) { if (bf16) SAGE_BW(64, true, true); else SAGE_BW(64, true, false); }
    else { if (bf16) SAGE_BW(64, false, true); else SAGE_BW(64, false, false); }
  }
#undef SAGE_BW
}

}  // namespace sage
