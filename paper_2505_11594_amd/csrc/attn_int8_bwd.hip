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
// Three deterministic kernels (no atomics):
//  - dV and dK: a workgroup owns 128 keys (4 waves x 32) and walks the query
//    blocks.  S = Q^ K^T puts a key in each lane's column and 16 queries in its
//    rows, so P^ and dS^ of a 32-query subtile are, as they stand, the B
//    operands of dV^T = dO^T P^ and dK^T = Q^T dS^ (A = dO^T / Q^T rows with
//    each 32-query group permuted as V^T in the forward).  The block scales
//    of P and dS need the block's maxima before any code is formed: the
//    block's exp2 arguments (dV) or its dS (dK) stay in registers while the
//    maximum is reduced across the waves through LDS, then all codes are
//    formed and each channel block's product runs over the four subtiles.
//    Apart, the two kernels keep their fp32 state within the 256
//    architectural registers a wave has (together they would not), and dV
//    needs neither dP nor the 16-bit operands.
//  - dQ: a workgroup owns 128 queries (4 waves x 32) and walks the KV blocks.
//    S^T = K^ Q^T puts a query in each lane's column; dS of the block stays in
//    registers while its maximum is reduced across the waves, and dS^ is the B
//    operand of dQ^T = K^T dS^T (A = K^T rows, permuted the same way).
// Each workgroup stages the operands its four waves share -- a query block
// (Q^, dO, L, D and a transposed Q^ or dO^) for dV and dK, a KV block (K^, V,
// K^T) for dQ -- in LDS in MFMA-operand order with global loads that write
// LDS, one block ahead of the block being computed.
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

// 4 x 4 byte transpose inside each quad of lanes: lane 4m + j returns the
// bytes j of lanes 4m, 4m + 1, 4m + 2, 4m + 3 (in that order, low byte first).
__device__ __forceinline__ uint32_t quad_byte_transpose(uint32_t w, int lane) {
  const int j = lane & 3;
  const uint32_t p1 = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)w, 0xB1, 0xF, 0xF, true);    // quad_perm [1,0,3,2]
  const uint32_t x1 = __builtin_amdgcn_perm(p1, w, (j & 1) ? 0x03070105u : 0x06020400u);
  const uint32_t p2 = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x1, 0x4E, 0xF, 0xF, true);   // quad_perm [2,3,0,1]
  return __builtin_amdgcn_perm(p2, x1, (j & 2) ? 0x03020706u : 0x05040100u);
}

// One step of a butterfly reduction over lanes: each lane keeps one half of
// its 2H values (the upper half where `upper`), adds the partner lane's other
// half to it, the partner given by a DPP control (CTRL >= 0) or lane ^ 16.
template <int H, int CTRL>
__device__ __forceinline__ void bw_fold(float (&x)[16], bool upper) {
#pragma unroll
  for (int i = 0; i < H; ++i) {
    const float send = upper ? x[i] : x[i + H];
    const float keep = upper ? x[i + H] : x[i];
    float recv;
    if constexpr (CTRL < 0) recv = __shfl_xor(send, 16, 64);
    else recv = __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(send), CTRL, 0xF, 0xF, true));
    x[i] = keep + recv;
  }
}

// 16 values in [0, 127 (1 + 2^-20)] -> 16 codes rint(x r): v_cvt_pk_u8_f32
// rounds to nearest even (the same integer as the magic-number add above)
__device__ __forceinline__ v4i bw_codes_u(const float (&x)[16], float r) {
  int w[4];
#pragma unroll
  for (int g = 0; g < 4; ++g) {
    uint32_t t = __builtin_amdgcn_cvt_pk_u8_f32(x[4 * g] * r, 0, 0u);
    t = __builtin_amdgcn_cvt_pk_u8_f32(x[4 * g + 1] * r, 1, t);
    t = __builtin_amdgcn_cvt_pk_u8_f32(x[4 * g + 2] * r, 2, t);
    w[g] = (int)__builtin_amdgcn_cvt_pk_u8_f32(x[4 * g + 3] * r, 3, t);
  }
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

// The dV and dK kernels: a workgroup owns 128 keys (4 waves x 32) of one
// (b,h) and walks the query blocks; S = Q^ K^T puts a key in each lane's
// column and 16 queries in its rows.  LDS holds the query block's operands in
// MFMA-operand order (1 KiB per 64-lane operand read, lane l's 16 bytes at
// 16 l): Q^ operand blocks (u, s) -- rows q0 + 32u + col, channels
// [32s + 16hi, +16) --, dO operand blocks (u, s16) -- channels [16s16 + 8hi,
// +8) --, transposed operand blocks (db, u) -- channel rows 32db + col,
// queries [32u + 16hi, +16) of the block --, and the block's Lb and D (128
// floats each).  Query rows >= N read row N - 1 (those entries are masked).

// query-block loads shared by the two kernels (wave w takes operand blocks
// w, w + 4, ...)
template <int D>
__device__ __forceinline__ void bw_load_qa(const int8_t* qc, uint8_t* dst, int b, int bh, int N, int q0, int col,
                                           int hi) {
  constexpr int NKS = D / 32;
  const int u = b / NKS, s = b % NKS;
  const int q = min(q0 + 32 * u + col, N - 1);
  bw_lds_load16(qc + ((size_t)bh * N + q) * D + 32 * s + 16 * hi, dst);
}
template <int D>
__device__ __forceinline__ void bw_load_t(const int8_t* xt, uint8_t* dst, int t, int bh, int Np, int q0, int col,
                                          int hi) {
  const int db = t / 4, u = t % 4;
  bw_lds_load16(xt + ((size_t)bh * D + 32 * db + col) * Np + q0 + 32 * u + 16 * hi, dst);
}
// Lb and D of the query block (one wave: lanes 0-31 Lb, 32-63 D)
__device__ __forceinline__ void bw_load_ld(const float* lb, const float* drow, uint8_t* dst, int bh, int Np, int q0,
                                           int lane) {
  const float* src = lane < 32 ? lb + (size_t)bh * Np + q0 + 4 * lane : drow + (size_t)bh * Np + q0 + 4 * (lane - 32);
  bw_lds_load16(src, dst);
}

// visible iff q < N, key < N and (causal) key <= q: the three sign bits,
// applied to an exp2 argument as min(arg, bound)
template <bool CAUSAL>
__device__ __forceinline__ float bw_mask(float arg, int q, int key, int N) {
  int m = (q - N) & (key - N);
  if (CAUSAL) m &= ~(q - key);
  return smin(arg, __uint_as_float(0xFF800000u ^ ((uint32_t)m & 0x80000000u)));
}

// ---------------------------------------------------------------------------
// dV.  dV^T = dO^T P^ per query block: S = Q^ K^T, P = exp2(S c_t - Lb), psi
// of P per (128 x 128) block.  The block maximum of P is exp2 of the block
// maximum of its argument (exp2 is monotone), so the arguments of the whole
// block stay in registers while that maximum is reduced across the waves,
// and each P is formed once, right before its code.  No 16-bit operand
// takes part.  gt: dO^T int8 [BH, D, Np] permuted per 32 rows.
// ---------------------------------------------------------------------------
template <int D>
struct BwDvLds {
  static constexpr int NKS = D / 32, NDB = D / 32;
  static constexpr int NQA = 4 * NKS, NT = NDB * 4;
  static constexpr int QA_OFF = 0, GT_OFF = NQA * 1024, LD_OFF = GT_OFF + NT * 1024, BYTES = LD_OFF + 1024;
  static constexpr int J = (NQA + NT) / 4;
  static_assert((NQA + NT) % 4 == 0, "even split over 4 waves");
};

template <int D, bool CAUSAL>
__global__ __launch_bounds__(256, 2) void attn_i8_bwd_dv_kernel(
    const int8_t* __restrict__ qc, const float* __restrict__ qs, const int8_t* __restrict__ kc,
    const float* __restrict__ ks, const int8_t* __restrict__ gt, const float* __restrict__ gs,
    const float* __restrict__ drow, const float* __restrict__ lb, float* __restrict__ dv, int N, int Np, int nqb,
    float c2) {
  using T = BwDvLds<D>;
  constexpr int NKS = T::NKS, NDB = T::NDB, NU = BW_Q / 32;
  __shared__ __attribute__((aligned(16))) uint8_t lds[2][T::BYTES];
  __shared__ float red[2][4];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int col = lane & 31, hi = lane >> 5;
  const int kblk = blockIdx.x, bh = blockIdx.y;
  const int kb = kblk * BW_K, key = kb + 32 * wave + col;
  const float sK = ks[(size_t)bh * (Np / BW_K) + kblk];

  v4i kreg[NKS];   // B operand of S: this lane's key, channels [32s + 16hi, +16)
  {
    const int8_t* kr = kc + ((size_t)bh * Np + key) * D;
#pragma unroll
    for (int s = 0; s < NKS; ++s) kreg[s] = *reinterpret_cast<const v4i*>(kr + 32 * s + 16 * hi);
  }
  v16f dva[NDB];
#pragma unroll
  for (int db = 0; db < NDB; ++db) dva[db] = v16f{};

  auto issue = [&](int i, int buf) {
    const int q0 = i * BW_Q;
    uint8_t* L = lds[buf];
#pragma unroll
    for (int k = 0; k < T::J; ++k) {
      const int b = wave + 4 * k;
      if (b < T::NQA) bw_load_qa<D>(qc, L + T::QA_OFF + b * 1024, b, bh, N, q0, col, hi);
      else bw_load_t<D>(gt, L + T::GT_OFF + (b - T::NQA) * 1024, b - T::NQA, bh, Np, q0, col, hi);
    }
    if (wave == 0) bw_load_ld(lb, drow, L + T::LD_OFF, bh, Np, q0, lane);
  };

  const int i0 = CAUSAL ? kb / BW_Q : 0;
  issue(i0, i0 & 1);
  for (int i = i0; i < nqb; ++i) {
    const int q0 = i * BW_Q, a = i & 1;
    bw_wait_all();                                 // this wave's loads of block i have landed
    __syncthreads();                               // everyone's; every wave is done with block i - 1
    if (i + 1 < nqb) issue(i + 1, a ^ 1);
    const uint8_t* L = lds[a];
    const float sQ = qs[(size_t)bh * nqb + i];
    const float ct = __builtin_fmaxf(sQ * sK * c2, 1.17549435e-38f);   // see the forward kernel
    const bool need_mask = (q0 + BW_Q > N) || (kb + BW_K > N) || (CAUSAL && q0 < kb + BW_K - 1);

    // exp2 arguments of the block: element v of subtile u is query q0 + 32u + 8(v>>2) + 4hi + (v&3)
    float arg[NU][16];
    float am = -INFINITY;
#pragma unroll
    for (int u = 0; u < NU; ++u) {
      v16i sacc = v16i{};
#pragma unroll
      for (int s = 0; s < NKS; ++s)
        sacc = __builtin_amdgcn_mfma_i32_32x32x32_i8(
            *reinterpret_cast<const v4i*>(L + T::QA_OFF + (u * NKS + s) * 1024 + lane * 16), kreg[s], sacc, 0, 0, 0);
      const float* lbr = reinterpret_cast<const float*>(L + T::LD_OFF) + 32 * u + 4 * hi;
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const v4f l4 = *reinterpret_cast<const v4f*>(lbr + 8 * g);
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int e = 4 * g + r;
          float x = __builtin_fmaf((float)sacc[e], ct, -l4[r]);
          if (need_mask) x = bw_mask<CAUSAL>(x, q0 + 32 * u + 4 * hi + 8 * g + r, key, N);
          arg[u][e] = x;
          am = __builtin_fmaxf(am, x);
        }
      }
    }
    am = wave_max(am);
    if (lane == 0) red[a][wave] = am;
    __syncthreads();
    am = __builtin_fmaxf(__builtin_fmaxf(red[a][0], red[a][1]), __builtin_fmaxf(red[a][2], red[a][3]));
    const float pm = __builtin_amdgcn_exp2f(am);   // max P of the block (0 when it is fully masked)
    const float sP = pm / 127.0f, rP = pm > 0.0f ? 1.0f / sP : 0.0f;

    v4i pc[NU];
#pragma unroll
    for (int u = 0; u < NU; ++u) {
      float P[16];
#pragma unroll
      for (int e = 0; e < 16; ++e) P[e] = __builtin_amdgcn_exp2f(arg[u][e]);
      pc[u] = bw_codes_u(P, rP);
    }
    const float fv = sP * gs[(size_t)bh * nqb + i];
#pragma unroll
    for (int db = 0; db < NDB; ++db) {
      v16i dvi = v16i{};
#pragma unroll
      for (int u = 0; u < NU; ++u)
        dvi = __builtin_amdgcn_mfma_i32_32x32x32_i8(
            *reinterpret_cast<const v4i*>(L + T::GT_OFF + (db * 4 + u) * 1024 + lane * 16), pc[u], dvi, 0, 0, 0);
#pragma unroll
      for (int e = 0; e < 16; ++e) dva[db][e] = __builtin_fmaf((float)dvi[e], fv, dva[db][e]);
    }
  }

  // dV^T: lane holds key kb + 32 wave + col and channels 32db + 8g + 4hi + r
  if (key < N) {
#pragma unroll
    for (int db = 0; db < NDB; ++db)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const size_t idx = ((size_t)bh * N + key) * D + 32 * db + 8 * g + 4 * hi;
        *reinterpret_cast<float4*>(dv + idx) = make_float4(dva[db][4 * g], dva[db][4 * g + 1], dva[db][4 * g + 2], dva[db][4 * g + 3]);
      }
  }
}

// ---------------------------------------------------------------------------
// dK.  dK^T = Q^T dS^ per query block: S = Q^ K^T and dP = dO V^T of each
// 32-query subtile, P = exp2(S c_t - Lb), dS = P (dP - D); dS of the whole
// block stays in registers while its maximum is reduced across the waves,
// then psi of dS and the product.  Eight waves, two per 32-key group: wave
// (kg, qh) forms S, dP and dS of subtiles 2qh and 2qh + 1 for its keys, the
// waves swap their dS^ codes through LDS, and each wave then runs the product
// over all four subtiles for half of the channel blocks -- the int32 block
// products stay whole, and each wave holds half the fp32 accumulators, which
// lets two waves share a SIMD.  The query block's Q^ and dO (double-buffered)
// and Q^T (single: loaded after the block's first barrier, waited for before
// its second) are staged in LDS.  qt: Q^T int8 [BH, D, Np] permuted per 32
// rows.
// ---------------------------------------------------------------------------
constexpr int BW_DK_WAVES = 8;

template <int D>
struct BwDkLds {
  static constexpr int NKS = D / 32, NKS16 = D / 16, NDB = D / 32;
  static constexpr int NQA = 4 * NKS, NGA = 4 * NKS16, NT = NDB * 4;
  static constexpr int QA_OFF = 0, GA_OFF = NQA * 1024, LD_OFF = GA_OFF + NGA * 1024, A_BYTES = LD_OFF + 1024;
  static constexpr int T_BYTES = NT * 1024;
  static constexpr int AJ = (NQA + NGA) / BW_DK_WAVES, TJ = NT / BW_DK_WAVES;   // loads per wave
  static_assert((NQA + NGA) % BW_DK_WAVES == 0 && NT % BW_DK_WAVES == 0, "even split over the waves");
};

// STORE_DS: also write, for every (query block, KV block) pair, the dS^ codes
// in the operand order of the dQ kernel's product (query-block-major, 16
// operand blocks of 1 KiB: (query group w, key subtile t) -- lane l holds
// query 32w + l%32 and the 16 keys at positions [16 (l/32), +16) of subtile t,
// position 16h + 4g + r holding key 8g + 4h + r), s_dS of the pair, and the
// pair's row sums of the unquantized dS (one per query, [KV block][query]).
// The codes go through LDS (a byte transpose inside each quad of lanes, then
// dword writes in place) and leave with whole 16-byte vector stores; the row
// sums are reduced across lanes in registers.  Heads are
// bh0 + blockIdx.y; the stored arrays are indexed by blockIdx.y.
template <int D, bool CAUSAL, bool BF16, bool STORE_DS>
__global__ __launch_bounds__(64 * BW_DK_WAVES, 1) void attn_i8_bwd_dk_kernel(
    const int8_t* __restrict__ qc, const float* __restrict__ qs, const int8_t* __restrict__ qt,
    const int8_t* __restrict__ kc, const float* __restrict__ ks, const uint16_t* __restrict__ v,
    const uint16_t* __restrict__ dout, const float* __restrict__ drow, const float* __restrict__ lb,
    float* __restrict__ dk, int8_t* __restrict__ dsc, float* __restrict__ dss, float* __restrict__ drs, int N, int Np,
    int nqb, int bh0, float c2, float rsd) {
  using T = BwDkLds<D>;
  constexpr int NKS = T::NKS, NKS16 = T::NKS16, NDB = T::NDB, NU = BW_Q / 32, NH = NDB / 2;
  __shared__ __attribute__((aligned(16))) uint8_t ldsA[2][T::A_BYTES];
  __shared__ __attribute__((aligned(16))) uint8_t ldsT[T::T_BYTES];
  __shared__ __attribute__((aligned(16))) uint8_t cx[4 * NU * 1024];   // dS^ codes: (key group, subtile) blocks
  __shared__ __attribute__((aligned(16))) uint8_t dsl[STORE_DS ? 16 * 1024 : 16];
  __shared__ float red2[STORE_DS ? 4 * BW_Q : 1];
  __shared__ float red[2][BW_DK_WAVES];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int kg = wave & 3, qh = wave >> 2;          // key group; query half (subtiles 2qh, 2qh + 1); channel half
  const int col = lane & 31, hi = lane >> 5;
  const int kblk = blockIdx.x, lbh = blockIdx.y, bh = bh0 + lbh;
  const int nkb = Np / BW_K;
  const int kb = kblk * BW_K, key = kb + 32 * kg + col;
  const float sK = ks[(size_t)bh * (Np / BW_K) + kblk];

  // B operands of this lane's key: K^ (channels [32s + 16hi, +16)) and V
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
  v16f dka[NH];                                      // channel blocks qh NH + h
#pragma unroll
  for (int h = 0; h < NH; ++h) dka[h] = v16f{};

  auto issue_A = [&](int i, int buf) {
    const int q0 = i * BW_Q;
    uint8_t* L = ldsA[buf];
#pragma unroll
    for (int k = 0; k < T::AJ; ++k) {
      const int b = wave + BW_DK_WAVES * k;
      if (b < T::NQA) {
        bw_load_qa<D>(qc, L + T::QA_OFF + b * 1024, b, bh, N, q0, col, hi);
      } else {
        const int g = b - T::NQA, u = g / NKS16, s = g % NKS16;
        const int q = min(q0 + 32 * u + col, N - 1);
        bw_lds_load16(dout + ((size_t)bh * N + q) * D + 16 * s + 8 * hi, L + T::GA_OFF + g * 1024);
      }
    }
  };
  auto issue_T = [&](int i) {
#pragma unroll
    for (int k = 0; k < T::TJ; ++k) {
      const int t = wave + BW_DK_WAVES * k;
      bw_load_t<D>(qt, ldsT + t * 1024, t, bh, Np, i * BW_Q, col, hi);
    }
  };

  const int i0 = CAUSAL ? kb / BW_Q : 0;
  if (wave == 0) bw_load_ld(lb, drow, ldsA[i0 & 1] + T::LD_OFF, bh, Np, i0 * BW_Q, lane);
  issue_A(i0, i0 & 1);
  for (int i = i0; i < nqb; ++i) {
    const int q0 = i * BW_Q, a = i & 1;
    bw_wait_all();                                 // this wave's loads of block i have landed
    __syncthreads();                               // everyone's; every wave is done with block i - 1
    if (i + 1 < nqb && wave == 0) bw_load_ld(lb, drow, ldsA[a ^ 1] + T::LD_OFF, bh, Np, q0 + BW_Q, lane);
    issue_T(i);
    if (i + 1 < nqb) issue_A(i + 1, a ^ 1);
    const uint8_t* L = ldsA[a];
    const float sQ = qs[(size_t)bh * nqb + i];
    const float ct = __builtin_fmaxf(sQ * sK * c2, 1.17549435e-38f);   // see the forward kernel
    const bool need_mask = (q0 + BW_Q > N) || (kb + BW_K > N) || (CAUSAL && q0 < kb + BW_K - 1);

    // dS of this wave's two subtiles u = 2qh + uu: element v is query
    // q0 + 32u + 8(v>>2) + 4hi + (v&3); the masking choice is made per block
    float dS[2][16];
    float dm = 0.0f;
    auto phase1 = [&](auto MASK_) {
      constexpr bool MASK = decltype(MASK_)::value != 0;
#pragma unroll
      for (int uu = 0; uu < 2; ++uu) {
        const int u = 2 * qh + uu;
        v16i sacc = v16i{};
#pragma unroll
        for (int s = 0; s < NKS; ++s)
          sacc = __builtin_amdgcn_mfma_i32_32x32x32_i8(
              *reinterpret_cast<const v4i*>(L + T::QA_OFF + (u * NKS + s) * 1024 + lane * 16), kreg[s], sacc, 0, 0, 0);
        v16f dp = v16f{};
#pragma unroll
        for (int s = 0; s < NKS16; ++s)
          dp = mfma16<BF16>(*reinterpret_cast<const v4i*>(L + T::GA_OFF + (u * NKS16 + s) * 1024 + lane * 16), vreg[s], dp);
        const float* lbr = reinterpret_cast<const float*>(L + T::LD_OFF) + 32 * u + 4 * hi;
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const v4f l4 = *reinterpret_cast<const v4f*>(lbr + 8 * g);
          const v4f d4 = *reinterpret_cast<const v4f*>(lbr + 128 + 8 * g);
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int e = 4 * g + r;
            float x = __builtin_fmaf((float)sacc[e], ct, -l4[r]);
            if constexpr (MASK) x = bw_mask<CAUSAL>(x, q0 + 32 * u + 4 * hi + 8 * g + r, key, N);
            const float p = __builtin_amdgcn_exp2f(x);
            const float y = p * (dp[e] - d4[r]);
            dS[uu][e] = y;
            dm = __builtin_fmaxf(dm, __builtin_fabsf(y));
          }
        }
      }
    };
    if (need_mask) phase1(ic<1>{});
    else phase1(ic<0>{});
    dm = wave_max(dm);
    if (lane == 0) red[a][wave] = dm;
    // the T loads of this block were issued before the next block's A loads
    if (i + 1 < nqb) bw_wait_vm<T::AJ>();
    else bw_wait_all();
    __syncthreads();
    dm = 0.0f;
#pragma unroll
    for (int w = 0; w < BW_DK_WAVES; ++w) dm = __builtin_fmaxf(dm, red[a][w]);
    const float sdS = dm / 127.0f, rdS = dm > 0.0f ? 1.0f / sdS : 0.0f;

#pragma unroll
    for (int uu = 0; uu < 2; ++uu) {
      const int u = 2 * qh + uu;
      const v4i sc = bw_codes(dS[uu], rdS);
      *reinterpret_cast<v4i*>(cx + (kg * NU + u) * 1024 + lane * 16) = sc;
      if constexpr (STORE_DS) {
        // codes: byte e = 4g + r of sc is query 32u + 8g + 4hi + r and key
        // 32 kg + col; after the quad transpose this lane holds query
        // 32u + 8g + 4hi + (col & 3) for keys 4 (col >> 2) + [0, 4)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const uint32_t t = quad_byte_transpose((uint32_t)sc[g], lane);
          const int m = col >> 2, lq = 8 * g + 4 * hi + (col & 3) + 32 * (m & 1);
          *reinterpret_cast<uint32_t*>(dsl + (u * 4 + kg) * 1024 + lq * 16 + 4 * (m >> 1)) = t;
        }
        // row sums of dS over this wave's 32 keys: a butterfly over the 32
        // lanes that share hi (partners lane ^ 16, row rotation by 8, half-row
        // mirror, quad swaps), after which lanes 2e and 2e + 1 hold the sum of
        // element e
        float x[16];
#pragma unroll
        for (int e = 0; e < 16; ++e) x[e] = dS[uu][e];
        bw_fold<8, -1>(x, (col & 16) != 0);
        bw_fold<4, 0x128>(x, (col & 8) != 0);      // row_ror:8
        bw_fold<2, 0x141>(x, (col & 4) != 0);      // row_half_mirror
        bw_fold<1, 0x4E>(x, (col & 2) != 0);       // quad_perm [2,3,0,1]
        const float sum = x[0] + __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x[0]), 0xB1, 0xF, 0xF, true));
        if ((col & 1) == 0) {
          const int e = col >> 1;
          red2[kg * BW_Q + 32 * u + 8 * (e >> 2) + 4 * hi + (e & 3)] = sum;
        }
      }
    }
    __syncthreads();                               // every wave's codes (and, storing dS^, its staging) are in LDS
    v4i cs[NU];
#pragma unroll
    for (int u = 0; u < NU; ++u) cs[u] = *reinterpret_cast<const v4i*>(cx + (kg * NU + u) * 1024 + lane * 16);
    const float fk = (sdS * sQ) * rsd;
#pragma unroll
    for (int h = 0; h < NH; ++h) {
      const int db = qh * NH + h;
      v16i dki = v16i{};
#pragma unroll
      for (int u = 0; u < NU; ++u)
        dki = __builtin_amdgcn_mfma_i32_32x32x32_i8(*reinterpret_cast<const v4i*>(ldsT + (db * 4 + u) * 1024 + lane * 16),
                                                    cs[u], dki, 0, 0, 0);
#pragma unroll
      for (int e = 0; e < 16; ++e) dka[h][e] = __builtin_fmaf((float)dki[e], fk, dka[h][e]);
    }
    if constexpr (STORE_DS) {
      const size_t pair = ((size_t)lbh * nqb + i) * nkb + kblk;
#pragma unroll
      for (int b2 = 0; b2 < 16 / BW_DK_WAVES; ++b2) {
        const int b = wave * (16 / BW_DK_WAVES) + b2;
        *reinterpret_cast<v4i*>(dsc + (pair * 16 + b) * 1024 + lane * 16) =
            *reinterpret_cast<const v4i*>(dsl + b * 1024 + lane * 16);
      }
      if (tid < BW_Q) {
        const float x = (red2[tid] + red2[BW_Q + tid]) + (red2[2 * BW_Q + tid] + red2[3 * BW_Q + tid]);
        drs[((size_t)lbh * nkb + kblk) * Np + q0 + tid] = x;
      }
      if (tid == 0) dss[pair] = sdS;
    }
  }

  // dK^T: lane holds key kb + 32 kg + col and channels 32db + 8g + 4hi + r
  if (key < N) {
#pragma unroll
    for (int h = 0; h < NH; ++h)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const size_t idx = ((size_t)bh * N + key) * D + 32 * (qh * NH + h) + 8 * g + 4 * hi;
        *reinterpret_cast<float4*>(dk + idx) = make_float4(dka[h][4 * g], dka[h][4 * g + 1], dka[h][4 * g + 2], dka[h][4 * g + 3]);
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
    // S^T (exact int32) and dP^T (fp32) of one 32-key subtile
    auto products = [&](int t, v16i& sacc, v16f& dp) {
      sacc = v16i{};
#pragma unroll
      for (int s = 0; s < NKS; ++s)
        sacc = __builtin_amdgcn_mfma_i32_32x32x32_i8(
            *reinterpret_cast<const v4i*>(L + T::KA_OFF + (t * NKS + s) * 1024 + lane * 16), qreg[s], sacc, 0, 0, 0);
      dp = v16f{};
#pragma unroll
      for (int s = 0; s < NKS16; ++s)
        dp = mfma16<BF16>(*reinterpret_cast<const v4i*>(L + T::VA_OFF + (t * NKS16 + s) * 1024 + lane * 16), greg[s], dp);
    };
    // dS of the block stays in registers while its maximum is reduced across
    // the waves.  The products of subtile t + 1 are interleaved with the
    // softmax work of subtile t (one MFMA, then eight VALU instructions); the
    // masking choice is made per block.
    float dS[NT][16];
    float dm = 0.0f, rs = 0.0f;
    auto phase1 = [&](auto MASK_) {
      constexpr bool MASK = decltype(MASK_)::value != 0;
      v16i sacc[2];
      v16f dp[2];
      products(0, sacc[0], dp[0]);
      static_for<NT>([&](auto T_) {
        constexpr int t = decltype(T_)::value;
        if constexpr (t + 1 < NT) products(t + 1, sacc[(t + 1) & 1], dp[(t + 1) & 1]);
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          float arg = __builtin_fmaf((float)sacc[t & 1][e], ct, -lbq);
          if constexpr (MASK) arg = bw_mask<CAUSAL>(arg, qi, kb + 32 * t + 8 * (e >> 2) + 4 * hi + (e & 3), N);
          const float p = __builtin_amdgcn_exp2f(arg);
          const float x = p * (dp[t & 1][e] - dq_row);
          dS[t][e] = x;
          rs += x;
          dm = __builtin_fmaxf(dm, __builtin_fabsf(x));
        }
        if constexpr (t + 1 < NT) {
#pragma unroll
          for (int m = 0; m < NKS + NKS16; ++m) {
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
            __builtin_amdgcn_sched_group_barrier(0x002, 8, 0);
          }
        }
        __builtin_amdgcn_sched_barrier(0);
      });
    };
    if (need_mask) phase1(ic<1>{});
    else phase1(ic<0>{});
    dm = wave_max(dm);
    if (lane == 0) red[buf][wave] = dm;
    __syncthreads();
    dm = __builtin_fmaxf(__builtin_fmaxf(red[buf][0], red[buf][1]), __builtin_fmaxf(red[buf][2], red[buf][3]));
    const float sdS = dm / 127.0f, rdS = dm > 0.0f ? 1.0f / sdS : 0.0f;
    // codes of the block, then per channel block the product over its four
    // subtiles (exact int32), folded into fp32 once per block
    v4i sc[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) sc[t] = bw_codes(dS[t], rdS);
    const float fq = (sdS * sK) * rsd;
    const float rr = (rs + __shfl_xor(rs, 32, 64)) * rsd;   // rowsum(dS) of this lane's query, / sqrt(D)
#pragma unroll
    for (int db = 0; db < NDB; ++db) {
      v16i dqi = v16i{};
#pragma unroll
      for (int t = 0; t < NT; ++t)
        dqi = __builtin_amdgcn_mfma_i32_32x32x32_i8(
            *reinterpret_cast<const v4i*>(L + T::KT_OFF + (db * NT + t) * 1024 + lane * 16), sc[t], dqi, 0, 0, 0);
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const v4f km = *reinterpret_cast<const v4f*>(kms + 32 * db + 8 * g + 4 * hi);
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int e = 4 * g + r;
          float x = __builtin_fmaf((float)dqi[e], fq, dqa[db][e]);
          if (kmean != nullptr) x = __builtin_fmaf(rr, km[r], x);
          dqa[db][e] = x;
        }
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

// ---------------------------------------------------------------------------
// dQ from the stored dS^ of the dK kernel: per (query block, KV block) pair
// dQ^T += (K^T dS^T) s_dS s_K / sqrt(D) + rowsum(dS) K_m / sqrt(D), with the
// pair's codes, s_dS and row sums read back instead of recomputing S, dP and
// dS.  A workgroup owns 128 queries (4 waves x 32); each KV block's K^T
// operand blocks are staged in LDS one block ahead, and each wave loads its
// own four dS^ operand blocks (1 KiB each, contiguous) straight into
// registers one block ahead.  Heads are bh0 + blockIdx.y; the stored arrays
// are indexed by blockIdx.y.
// ---------------------------------------------------------------------------
template <int D>
struct BwQdsLds {
  static constexpr int NDB = D / 32, NT = BW_K / 32;
  static constexpr int NKT = NDB * NT;
  static constexpr int BYTES = NKT * 1024;
  static constexpr int J = NKT / 4;
  static_assert(NKT % 4 == 0, "even split over 4 waves");
};

template <int D, bool CAUSAL>
__global__ __launch_bounds__(256, 3) void attn_i8_bwd_dq_ds_kernel(
    const float* __restrict__ ks, const int8_t* __restrict__ kt, const int8_t* __restrict__ dsc,
    const float* __restrict__ dss, const float* __restrict__ drs, const float* __restrict__ kmean,
    float* __restrict__ dq, int N, int Np, int nqb, int bh0, float rsd) {
  using T = BwQdsLds<D>;
  constexpr int NDB = T::NDB, NT = T::NT;
  __shared__ __attribute__((aligned(16))) uint8_t lds[2][T::BYTES];
  __shared__ __attribute__((aligned(16))) float kms[D];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int col = lane & 31, hi = lane >> 5;
  const int i = blockIdx.x, lbh = blockIdx.y, bh = bh0 + lbh;
  const int nkbt = Np / BW_K;
  const int q0 = i * BW_Q, qi = q0 + 32 * wave + col;
  if (tid < D) kms[tid] = kmean != nullptr ? kmean[(size_t)bh * D + tid] : 0.0f;
  v16f dqa[NDB];
#pragma unroll
  for (int db = 0; db < NDB; ++db) dqa[db] = v16f{};

  auto issue = [&](int j, int buf) {
    const int kb = j * BW_K;
    uint8_t* L = lds[buf];
#pragma unroll
    for (int k = 0; k < T::J; ++k) {
      const int b = wave + 4 * k, db = b / NT, t = b % NT;
      bw_lds_load16(kt + ((size_t)bh * D + 32 * db + col) * Np + kb + 32 * t + 16 * hi, L + b * 1024);
    }
  };
  // this wave's dS^ operand blocks (query group `wave`, key subtiles 0..NT-1) of pair (i, j)
  auto load_ds = [&](int j, v4i (&d)[NT]) {
    const int8_t* p = dsc + ((((size_t)lbh * nqb + i) * nkbt + j) * (size_t)((BW_Q / 32) * NT) + wave * NT) * 1024 +
                      lane * 16;
#pragma unroll
    for (int t = 0; t < NT; ++t) d[t] = *reinterpret_cast<const v4i*>(p + t * 1024);
  };

  int nkb = nkbt;
  if (CAUSAL) nkb = min(nkb, min(q0 + BW_Q - 1, N - 1) / BW_K + 1);
  v4i dcur[NT], dnext[NT];
  issue(0, 0);
  load_ds(0, dcur);
  for (int j = 0; j < nkb; ++j) {
    const int buf = j & 1;
    bw_wait_all();
    __syncthreads();                               // block j has landed; every wave is done with block j - 1
    if (j + 1 < nkb) {
      issue(j + 1, buf ^ 1);
      load_ds(j + 1, dnext);
    }
    const uint8_t* L = lds[buf];
    const float sK = ks[(size_t)bh * nkbt + j];
    const float sdS = dss[((size_t)lbh * nqb + i) * nkbt + j];
    const float fq = (sdS * sK) * rsd;
    const float rr = drs[((size_t)lbh * nkbt + j) * Np + qi] * rsd;   // rowsum(dS) of this lane's query, / sqrt(D)
#pragma unroll
    for (int db = 0; db < NDB; ++db) {
      v16i dqi = v16i{};
#pragma unroll
      for (int t = 0; t < NT; ++t)
        dqi = __builtin_amdgcn_mfma_i32_32x32x32_i8(*reinterpret_cast<const v4i*>(L + (db * NT + t) * 1024 + lane * 16),
                                                    dcur[t], dqi, 0, 0, 0);
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const v4f km = *reinterpret_cast<const v4f*>(kms + 32 * db + 8 * g + 4 * hi);
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int e = 4 * g + r;
          float x = __builtin_fmaf((float)dqi[e], fq, dqa[db][e]);
          if (kmean != nullptr) x = __builtin_fmaf(rr, km[r], x);
          dqa[db][e] = x;
        }
      }
    }
#pragma unroll
    for (int t = 0; t < NT; ++t) dcur[t] = dnext[t];
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
                               float* dk, float* dv, int8_t* dsc, float* dss, float* drs, int G, int BH, int N, int Np,
                               float c2, float rsd, hipStream_t st) {
  const int nqb = (N + BW_Q - 1) / BW_Q, nkb = Np / BW_K;
  hipLaunchKernelGGL((attn_i8_bwd_dv_kernel<D, CAUSAL>), dim3((unsigned)nkb, (unsigned)BH), dim3(256), 0, st, qc, qs,
                     kc, ks, gt, gs, drow, lb, dv, N, Np, nqb, c2);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (G <= 0) {                                    // no room to store dS^: dQ recomputes it
    hipLaunchKernelGGL((attn_i8_bwd_dk_kernel<D, CAUSAL, BF16, false>), dim3((unsigned)nkb, (unsigned)BH),
                       dim3(64 * BW_DK_WAVES), 0,
                       st, qc, qs, qt, kc, ks, v, dout, drow, lb, dk, nullptr, nullptr, nullptr, N, Np, nqb, 0, c2, rsd);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL((attn_i8_bwd_dq_kernel<D, CAUSAL, BF16>), dim3((unsigned)nqb, (unsigned)BH), dim3(256), 0, st,
                       qc, qs, kc, ks, kt, v, dout, drow, lb, kmean, dq, N, Np, nqb, c2, rsd);
    return hipGetLastError();
  }
  for (int h0 = 0; h0 < BH; h0 += G) {             // groups of G heads share the stored dS^
    const int g = min(G, BH - h0);
    hipLaunchKernelGGL((attn_i8_bwd_dk_kernel<D, CAUSAL, BF16, true>), dim3((unsigned)nkb, (unsigned)g),
                       dim3(64 * BW_DK_WAVES), 0,
                       st, qc, qs, qt, kc, ks, v, dout, drow, lb, dk, dsc, dss, drs, N, Np, nqb, h0, c2, rsd);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL((attn_i8_bwd_dq_ds_kernel<D, CAUSAL>), dim3((unsigned)nqb, (unsigned)g), dim3(256), 0, st, ks, kt,
                       dsc, dss, drs, kmean, dq, N, Np, nqb, h0, rsd);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

// Bytes of stored dS^ state per head: codes (16 KiB per (query block, KV
// block) pair), s_dS per pair, and row sums [KV block][Np] fp32.
size_t i8_bwd_ds_bytes_per_head(int N) {
  const size_t Np = (size_t)((N + 127) / 128) * 128, nb = Np / 128;
  return nb * nb * 16384 + nb * nb * sizeof(float) + nb * Np * sizeof(float);
}

// Q^ [BH, N, D], K^ [BH, Np, D] row-major; Q^T, K^T, dO^T [BH, D, Np] permuted
// per 32 rows; scales per 128 rows; kmean null without smoothing.  dsc, dss,
// drs: the stored dS^ state of G heads (i8_bwd_ds_bytes_per_head each, in
// that order), or G = 0 to recompute dS^ in the dQ kernel.
hipError_t launch_attn_int8_bwd(const void* qc, const float* qs, const void* qt, const void* kc, const float* ks,
                                const void* kt, const void* v, const void* dout, const void* gt, const float* gs,
                                const float* drow, const float* lb, const float* kmean, float* dq, float* dk, float* dv,
                                void* ds_state, int G, int BH, int N, int Np, int D, bool causal, bool bf16, float c2,
                                float rsd, hipStream_t st) {
  const int8_t *a = (const int8_t*)qc, *b = (const int8_t*)qt, *c = (const int8_t*)kc, *d = (const int8_t*)kt,
               *g = (const int8_t*)gt;
  const uint16_t *vv = (const uint16_t*)v, *gg = (const uint16_t*)dout;
  const size_t nb = (size_t)Np / 128;
  int8_t* dsc = static_cast<int8_t*>(ds_state);
  float* dss = G > 0 ? reinterpret_cast<float*>(dsc + (size_t)G * nb * nb * 16384) : nullptr;
  float* drs = G > 0 ? dss + (size_t)G * nb * nb : nullptr;
#define SAGE_BW(DD, CC, BB)                                                                                          \
  return launch_bwd_t<DD, CC, BB>(a, qs, b, c, ks, d, vv, gg, g, gs, drow, lb, kmean, dq, dk, dv, dsc, dss, drs, G, BH, \
                                  N, Np, c2, rsd, st)
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
