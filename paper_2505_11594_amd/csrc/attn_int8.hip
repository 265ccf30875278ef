// 8-bit attention forward of SageBwd (Algorithm 2) for gfx950: per-block INT8
// Q, K, V (psi, Sec. 4.1), S = MM(Q^, K^) s_Q s_K on int8 MFMA, online
// softmax over KV tiles (128 or 64 keys), per-token INT8 quantization of P~ that reuses
// the row maxima (s_P = rowmax(P~)/127), O += MM(P^, V^) s_P s_V on int8
// MFMA, and the outputs O = O/l and L = m + log l.
//
// Work decomposition: one workgroup = 4 waves = 128 queries of one (b,h) --
// one block of psi(Q), so s_Q is uniform -- each wave owns 32 queries and
// walks all KV tiles.  Both products use v_mfma_i32_32x32x32_i8:
//   S^T (keys x queries) = K^ . Q^T    A = K^ tile (LDS), B = Q^ (registers)
//   O^T (dims x queries) += V^T . P^T  A = V^T tile (LDS), B = P^ (registers)
// Lane l supplies row/column l%32 and 16 bytes of the reduction index to
// each operand; the accumulator of lane l holds column l%32 (a query) and
// rows 8g + 4(l/32) + r (g, r in 0..3).  P^ for a 32-key subtile therefore
// sits in the lane that owns its query, as the 16 keys 8g + 4(l/32) + r in
// value order 4g + r; those 16 bytes are the lane's B operand of the P.V
// product directly, and V^T is stored with each 32-token group permuted so
// that the A operand's 16 bytes at offset 16(l/32) are the same keys.  S and
// P stay in registers; the row max needs one swap between the two lane
// halves that share a query.
//
// Scores are kept in the log2 domain u = fl32(acc) c_t, c_t =
// fl32(fl32(s_Q s_K) log2(e)/sqrt(D)), acc the exact int32 product: the tile
// max is taken on fl32(acc) (the rounding is monotone, so it is the max of
// u), P^ = rint(127 2^{u - t}) = rint(exp2(fma(acc, c_t, log2 127 - t)))
// with the rounding done by v_cvt_pk_u8_f32 (nearest even, packed a byte at
// a time), and the unquantized P~ = s_P P^ is summed into l.  Each tile's
// int32 P.V product is folded into the fp32 O with one fused multiply-add by
// s_P s_V after O is rescaled by alpha = 2^{m_old - m_new} (skipped when the
// whole wave has alpha = 1).
//
// Data movement: KV tiles go from HBM straight into LDS in MFMA-operand order
// (one 1 KiB block per 64-lane operand read), with the tile's two scales; two
// stages and one barrier per tile: after the barrier of tile j its loads
// have landed and every wave is done with tile j-1, whose stage the loads of
// tile j+1 then overwrite.  S^T is computed at the top of each tile.  (Issuing
// tile j+1's S^T under tile j's softmax, as the FP4 kernel does, measured
// slower here: the second set of int32 scores costs the register room of a
// third wave per SIMD at 64-key tiles and does not fit at 128.)
#include "sage_common.h"

typedef int v16i __attribute__((ext_vector_type(16)));

namespace sage {

constexpr int I8_AQ = 128;   // queries per workgroup (4 waves x 32)

__device__ __forceinline__ void i8_lds_load16(const void* src, void* dst) {
  __builtin_amdgcn_global_load_lds(src, (__attribute__((address_space(3))) void*)dst, 16, 0, 0);
}
__device__ __forceinline__ void i8_lds_load4(const void* src, void* dst) {
  __builtin_amdgcn_global_load_lds(src, (__attribute__((address_space(3))) void*)dst, 4, 0, 0);
}
__device__ __forceinline__ void i8_wait_loads() { __builtin_amdgcn_s_waitcnt(0x0F70); }   // vmcnt(0)

// rint of four values in [0, 255], packed (element 0 in the low byte):
// v_cvt_pk_u8_f32 rounds to nearest even and clamps to [0, 255]
__device__ __forceinline__ int i8_codes4(float a, float b, float c, float d) {
  uint32_t w = __builtin_amdgcn_cvt_pk_u8_f32(a, 0, 0u);
  w = __builtin_amdgcn_cvt_pk_u8_f32(b, 1, w);
  w = __builtin_amdgcn_cvt_pk_u8_f32(c, 2, w);
  return (int)__builtin_amdgcn_cvt_pk_u8_f32(d, 3, w);
}

template <int D, int BKV>
struct I8Stage {
  static constexpr int NSUB = BKV / 32;        // 32-key subtiles (S^T rows); K-steps of O^T += V^T P^T
  static constexpr int NKS = D / 32;           // K-steps of S^T = K^ Q^T
  static constexpr int NDB = D / 32;           // 32-dim blocks (O^T rows)
  static constexpr int NKB = NSUB * NKS;       // K^ operand blocks, 1 KiB each
  static constexpr int NVB = NDB * NSUB;       // V^T operand blocks, 1 KiB each
  static constexpr int KC_OFF = 0;
  static constexpr int VC_OFF = KC_OFF + NKB * 1024;
  static constexpr int SC_OFF = VC_OFF + NVB * 1024;   // s_K, s_V of the tile
  static constexpr int BYTES = SC_OFF + 16;
};

// OUT: 0 = fp32, 1 = bf16, 2 = fp16.
template <int D, int BKV, bool CAUSAL, int OUT>
__global__ __launch_bounds__(256, 2) void attn_int8_kernel(
    const int8_t* __restrict__ qc, const float* __restrict__ qs, const int8_t* __restrict__ kc,
    const float* __restrict__ ks, const int8_t* __restrict__ vc, const float* __restrict__ vs,
    void* __restrict__ o, float* __restrict__ lse, int BH, int N, int Np, int nqt, float c2, float log127) {
  using T = I8Stage<D, BKV>;
  constexpr int NSUB = T::NSUB, NKS = T::NKS, NDB = T::NDB;
  __shared__ __attribute__((aligned(16))) uint8_t lds[2][T::BYTES];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int col = lane & 31, hi = lane >> 5;

  // XCD-aware order, as in the FP4 kernel
  const int total = nqt * BH;
  int lin = blockIdx.x;
  if ((total & 7) == 0) lin = (blockIdx.x & 7) * (total >> 3) + (blockIdx.x >> 3);
  const long long bh = lin / nqt;
  int qt = lin % nqt;
  if (CAUSAL) qt = nqt - 1 - qt;
  const int q0 = qt * I8_AQ;
  const int qw = q0 + wave * 32;
  const int qi = qw + col;
  const float sQ = qs[(size_t)bh * nqt + qt];

  // Q^ fragment: 16 codes at channels [32 s + 16 hi, +16) per K-step s
  v4i qreg[NKS];
  if (qi < N) {
    const int8_t* qrow = qc + ((size_t)bh * N + qi) * D;
#pragma unroll
    for (int s = 0; s < NKS; ++s) qreg[s] = *reinterpret_cast<const v4i*>(qrow + 32 * s + 16 * hi);
  } else {
#pragma unroll
    for (int s = 0; s < NKS; ++s) qreg[s] = v4i{0, 0, 0, 0};
  }

  int ntiles = Np / BKV;
  {
    const int nt = (N + BKV - 1) / BKV;
    ntiles = nt < ntiles ? nt : ntiles;
  }
  if (CAUSAL) {
    const int qlast = min(q0 + I8_AQ - 1, N - 1);
    ntiles = min(ntiles, qlast / BKV + 1);
  }

  // ---- tile loads: HBM -> LDS ------------------------------------------
  // Wave w loads K^ operand blocks w, w + 4, ... (block b = (t, s): key row
  // 32t + col, channels [32s + 16hi, +16)) and V^T operand blocks w, w + 4, ...
  // (b = (db, u): dim row 32db + col, tile keys [32u + 16hi, +16)); wave 0's
  // lanes 0 and 1 load s_K and s_V of the tile.
  constexpr int KJ = (T::NKB + 3) / 4, VJ = (T::NVB + 3) / 4;
  const int8_t* kbase = kc + (size_t)bh * Np * D;
  const int8_t* vbase = vc + (size_t)bh * D * Np;
  const int nkt = Np / BKV;
  uint32_t ko[KJ], vo[VJ];
#pragma unroll
  for (int i = 0; i < KJ; ++i) {
    const int b = wave + 4 * i, t = b / NKS, s = b % NKS;
    ko[i] = (32 * t + col) * D + 32 * s + 16 * hi;
  }
#pragma unroll
  for (int i = 0; i < VJ; ++i) {
    const int b = wave + 4 * i, db = b / NSUB, u = b % NSUB;
    vo[i] = (32 * db + col) * Np + 32 * u + 16 * hi;
  }
  const float* sc_src = (lane == 0 ? ks : vs) + (size_t)bh * nkt;
  auto issue = [&](int j, int stage) {
    const int kb = j * BKV;
    uint8_t* L = lds[stage];
    const int8_t* kt = kbase + (size_t)kb * D;
    const int8_t* vt = vbase + kb;
#pragma unroll
    for (int i = 0; i < KJ; ++i)
      if (T::NKB % 4 == 0 || wave + 4 * i < T::NKB) i8_lds_load16(kt + ko[i], L + T::KC_OFF + (wave + 4 * i) * 1024);
#pragma unroll
    for (int i = 0; i < VJ; ++i)
      if (T::NVB % 4 == 0 || wave + 4 * i < T::NVB) i8_lds_load16(vt + vo[i], L + T::VC_OFF + (wave + 4 * i) * 1024);
    if (wave == 0 && lane < 2) i8_lds_load4(sc_src + j, L + T::SC_OFF);
  };

  v16f oacc[NDB];
#pragma unroll
  for (int db = 0; db < NDB; ++db) oacc[db] = v16f{};
  float m = -INFINITY, lsum = 0.0f;

  auto qk = [&](const uint8_t* L, v16i (&sacc)[NSUB]) {
#pragma unroll
    for (int t = 0; t < NSUB; ++t) {
      v16i acc = v16i{};
#pragma unroll
      for (int s = 0; s < NKS; ++s) {
        const v4i a = *reinterpret_cast<const v4i*>(L + T::KC_OFF + (t * NKS + s) * 1024 + lane * 16);
        acc = __builtin_amdgcn_mfma_i32_32x32x32_i8(a, qreg[s], acc, 0, 0, 0);
      }
      sacc[t] = acc;
    }
  };

  auto tile = [&](int j, int stage) {
    const uint8_t* L = lds[stage];
    const int kb = j * BKV;
    // kb < N always holds here; kept as a run-time test, it keeps the causal
    // variant inside the register budget (the compiler otherwise hoists work
    // across the tile boundary)
    const bool active = (!CAUSAL || kb <= qw + 31) && kb < N;
    float sf[NSUB][16];
    float ct = 0.f, bias = 0.f, alpha = 1.f, sP = 0.f;
    float ps[4] = {0.0f, 0.0f, 0.0f, 0.0f};
    if (active) {
      v16i sacc[NSUB];
      qk(L, sacc);
      const float sK = *reinterpret_cast<const float*>(L + T::SC_OFF);
#pragma unroll
      for (int u = 0; u < NSUB; ++u)
#pragma unroll
        for (int v = 0; v < 16; ++v) sf[u][v] = (float)sacc[u][v];   // exact: |acc| < 2^24
      const bool need_mask = (kb + BKV > N) || (CAUSAL && kb + BKV - 1 > qw);
      if (need_mask) {
        // element (u, v) is key kb + 32u + 8(v >> 2) + 4hi + (v & 3); kept iff
        // c = 32u + 8(v >> 2) + (v & 3) < rem (see the FP4 kernel)
        const int rem = (CAUSAL ? min(N, qi + 1) : N) - kb - 4 * hi;
#pragma unroll
        for (int u = 0; u < NSUB; ++u)
#pragma unroll
          for (int v = 0; v < 16; ++v) {
            const int c = 32 * u + 8 * (v >> 2) + (v & 3);
            const float bound = __uint_as_float(0xFF800000u ^ ((uint32_t)(c - rem) & 0x80000000u));
            sf[u][v] = smin(sf[u][v], bound);
          }
      }
      float x = sf[0][0];
#pragma unroll
      for (int u = 0; u < NSUB; ++u)
#pragma unroll
        for (int v = (u == 0 ? 1 : 0); v < 16; ++v) x = smax(x, sf[u][v]);
      const auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
      const float amax = smax(__uint_as_float(sw[0]), __uint_as_float(sw[1]));
      const float sqk = sQ * sK;
      // an all-zero Q or K block gives c_t = 0; the smallest normal fp32 in its
      // place keeps -inf scores at -inf and changes no P^ and no l (every
      // |u| is then below 2^-105, under half an ulp of log2 127)
      ct = __builtin_fmaxf(sqk * c2, 1.17549435e-38f);
      const float t = amax * ct;                       // tile max of u
      const float m_new = smax(m, t);
      alpha = __builtin_amdgcn_exp2f(m - m_new);       // 0 on the first tile (m = -inf)
      const float rho = __builtin_amdgcn_exp2f(t - m_new);
      sP = rho / 127.0f;                               // correctly rounded, as the oracle
      bias = log127 - t;
      m = m_new;
      // O <- alpha O, unless every query of the wave keeps its max
      if (__builtin_amdgcn_ballot_w64(alpha != 1.0f) != 0) {
#pragma unroll
        for (int db = 0; db < NDB; ++db)
#pragma unroll
          for (int v = 0; v < 16; ++v) oacc[db][v] *= alpha;
      }
    }

    if (active) {
      // P^ = rint(127 2^{u - t}) per element; the unquantized P~/s_P is summed
      v4i pw[NSUB];
#pragma unroll
      for (int u = 0; u < NSUB; ++u) {
        int w[4];
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          float p[4];
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            p[r] = __builtin_amdgcn_exp2f(__builtin_fmaf(sf[u][4 * g + r], ct, bias));
            ps[r] += p[r];
          }
          w[g] = i8_codes4(p[0], p[1], p[2], p[3]);
        }
        pw[u] = v4i{w[0], w[1], w[2], w[3]};
      }
      const float sV = *reinterpret_cast<const float*>(L + T::SC_OFF + 4);
      const float spv = sP * sV;
#pragma unroll
      for (int db = 0; db < NDB; ++db) {
        v16i acc = v16i{};
#pragma unroll
        for (int u = 0; u < NSUB; ++u) {
          const v4i a = *reinterpret_cast<const v4i*>(L + T::VC_OFF + (db * NSUB + u) * 1024 + lane * 16);
          acc = __builtin_amdgcn_mfma_i32_32x32x32_i8(a, pw[u], acc, 0, 0, 0);
        }
#pragma unroll
        for (int v = 0; v < 16; ++v) oacc[db][v] = __builtin_fmaf((float)acc[v], spv, oacc[db][v]);
      }
      const float psum = (ps[0] + ps[1]) + (ps[2] + ps[3]);
      lsum = lsum * alpha + sP * psum;
    }
  };

  issue(0, 0);
  for (int j = 0; j < ntiles; ++j) {
    i8_wait_loads();
    __syncthreads();
    if (j + 1 < ntiles) issue(j + 1, (j + 1) & 1);
    tile(j, j & 1);
  }

  // ---- epilogue: O = O^T / l stored row-major; L = ln 2 (m + log2 l) ----
  const float ltot = lsum + __shfl_xor(lsum, 32, 64);
  const float inv = 1.0f / ltot;
  if (qi < N) {
    if (lse != nullptr && hi == 0)
      lse[(size_t)bh * N + qi] = (m + __builtin_amdgcn_logf(ltot)) * 0.693147180559945309f;
    uint8_t* obase = reinterpret_cast<uint8_t*>(o);
#pragma unroll
    for (int db = 0; db < NDB; ++db)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int d0 = 32 * db + 8 * g + 4 * hi;
        const size_t idx = ((size_t)bh * N + qi) * D + d0;
        const float a0 = oacc[db][4 * g] * inv, a1 = oacc[db][4 * g + 1] * inv;
        const float a2 = oacc[db][4 * g + 2] * inv, a3 = oacc[db][4 * g + 3] * inv;
        if (OUT == 0) {
          *reinterpret_cast<float4*>(obase + idx * 4) = make_float4(a0, a1, a2, a3);
        } else {
          uint16_t h0, h1, h2, h3;
          if (OUT == 1) { h0 = f32_to_bf16_rne(a0); h1 = f32_to_bf16_rne(a1); h2 = f32_to_bf16_rne(a2); h3 = f32_to_bf16_rne(a3); }
          else { h0 = f32_to_fp16_rne(a0); h1 = f32_to_fp16_rne(a1); h2 = f32_to_fp16_rne(a2); h3 = f32_to_fp16_rne(a3); }
          *reinterpret_cast<uint2*>(obase + idx * 2) = make_uint2((uint32_t)h0 | ((uint32_t)h1 << 16), (uint32_t)h2 | ((uint32_t)h3 << 16));
        }
      }
  }
}

template <int D, int BKV, bool CAUSAL, int OUT>
static hipError_t launch_i8_t(const void* qc, const float* qs, const void* kc, const float* ks, const void* vc,
                              const float* vs, void* o, float* lse, int BH, int N, int Np, float c2, float log127,
                              hipStream_t st) {
  const int nqt = (N + I8_AQ - 1) / I8_AQ;
  hipLaunchKernelGGL((attn_int8_kernel<D, BKV, CAUSAL, OUT>), dim3((unsigned)(nqt * BH)), dim3(256), 0, st,
                     (const int8_t*)qc, qs, (const int8_t*)kc, ks, (const int8_t*)vc, vs, o, lse, BH, N, Np, nqt, c2,
                     log127);
  return hipGetLastError();
}

template <int D, int BKV, bool CAUSAL>
static hipError_t launch_i8_o(int out, const void* qc, const float* qs, const void* kc, const float* ks,
                              const void* vc, const float* vs, void* o, float* lse, int BH, int N, int Np, float c2,
                              float log127, hipStream_t st) {
  if (out == 0) return launch_i8_t<D, BKV, CAUSAL, 0>(qc, qs, kc, ks, vc, vs, o, lse, BH, N, Np, c2, log127, st);
  if (out == 1) return launch_i8_t<D, BKV, CAUSAL, 1>(qc, qs, kc, ks, vc, vs, o, lse, BH, N, Np, c2, log127, st);
  return launch_i8_t<D, BKV, CAUSAL, 2>(qc, qs, kc, ks, vc, vs, o, lse, BH, N, Np, c2, log127, st);
}

// KV tile (and K, V scale blocks) of bkv = 64 or 128 tokens; Q blocks of 128
// rows.  qs [BH, ceil(N/128)], ks and vs [BH, Np/bkv]; lse may be null.
hipError_t launch_attn_int8(const void* qc, const float* qs, const void* kc, const float* ks, const void* vc,
                            const float* vs, void* o, float* lse, int BH, int N, int Np, int D, int bkv, bool causal,
                            int out, float c2, float log127, hipStream_t st) {
#define SAGE_I8(DD, BB)                                                                                      \
  return causal ? launch_i8_o<DD, BB, true>(out, qc, qs, kc, ks, vc, vs, o, lse, BH, N, Np, c2, log127, st) \
                : launch_i8_o<DD, BB, false>(out, qc, qs, kc, ks, vc, vs, o, lse, BH, N, Np, c2, log127, st)
  if (D == 128) { if (bkv == 128) { SAGE_I8(128, 128); } else { SAGE_I8(128, 64); } }
  else { if (bkv == 128) { SAGE_I8(64, 128); } else { SAGE_I8(64, 64); } }
#undef SAGE_I8
}

}  // namespace sage
