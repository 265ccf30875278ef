// Microscaled-FP4 attention forward for gfx950 (SageAttention3, Algorithm 1
// without smoothing Q; two-level quantization of P~, Sec. 3.2).
//
// Work decomposition: one workgroup = 4 waves = 128 queries of one (b,h);
// each wave owns 32 queries and walks all KV tiles (BKV = 64 or 128 keys).
// Both products run on v_mfma_scale_f32_32x32x64_f8f6f4 with FP4 (E2M1)
// operands and E8M0 block scales:
//   S^T (keys x queries) = K^ . Q^T    A = K^ tile (LDS), B = Q^ (registers)
//   O^T (dims x queries) += V^T . P^T  A = V^T tile (LDS), B = P^ (registers)
// MFMA operand layout (32x32x64): lane l holds row/column l%32 and the 32
// consecutive K-indices [32*(l/32), +32) -- exactly one 32-element block and
// its scale byte.  The accumulator of lane l holds column l%32 and rows
// 8g + 4*(l/32) + r.  Because K^ is stored with its tokens permuted inside
// each 64-token group (quant.hip), the 32 scores a lane holds for one
// 64-key group are the original keys [32*(l/32), +32) of that group, in the
// order the B operand of the P.V product expects: S never leaves registers,
// the FP4 block of P is lane-local (its max needs no shuffle), and the row
// max over a tile needs one cross-half swap.
//
// Softmax state per query row (raw score domain): running max m, and the
// accumulator O^T and row sum kept in units of 6 * 2^-f_j of the true
// O_j, l_j, where 2^(delta_j) = 6 s_P1 = 2^{c2 (t_j - m_j)} is split into
// an integer part k_j (folded exactly into P's E8M0 scale) and a fraction
// f_j.  Each tile then rescales the accumulator once by
// gamma_j = 2^{c2 (m_{j-1} - m_j) + f_{j-1} - f_j}.
#include "sage_common.h"

namespace sage {

constexpr int AQ = 128;   // queries per workgroup (4 waves x 32)

// 16-byte-chunk XOR swizzle of LDS rows (64 or 32 bytes long).  An MFMA
// operand read has consecutive lanes on consecutive rows at one chunk; rows
// r and r + 4k must land in different chunks for 64 banks (16 lanes per pass)
// and rows r and r + 2k for 32 banks (8 lanes per pass).
template <int NCH>
__device__ __forceinline__ int swz(int row, int ch) { return ch ^ (((row >> 1) ^ (row >> 3)) & (NCH - 1)); }

template <int D, int BKV>
struct Fp4Tile {
  static constexpr int KROW = D / 2;          // bytes of one K^ row
  static constexpr int KCH = D / 32;          // 16-byte chunks per K^ row
  static constexpr int VROW = BKV / 2;        // bytes of one V^T row inside a tile
  static constexpr int VCH = BKV / 32;        // 16-byte chunks per V^T tile row
  static constexpr int KC_OFF = 0;
  static constexpr int KS_OFF = KC_OFF + BKV * KROW;
  static constexpr int VC_OFF = KS_OFF + BKV * 8;   // K scales: 2 dwords per key
  static constexpr int VS_OFF = VC_OFF + D * VROW;
  static constexpr int BYTES = VS_OFF + D * 8;      // V scales: 2 dwords per row
  static constexpr int KC_UNITS = BKV * KCH;  // 16-byte units
  static constexpr int VC_UNITS = D * VCH;
  static constexpr int KC_PER_T = (KC_UNITS + 255) / 256;
  static constexpr int VC_PER_T = (VC_UNITS + 255) / 256;
};

// Register staging of one KV tile: every thread issues the same fixed set of
// 16-byte global loads (no divergent branches, so the loads stay in flight
// while the current tile is computed) and later writes them to LDS.
template <int D, int BKV>
struct Stage {
  using T = Fp4Tile<D, BKV>;
  v4i kc[T::KC_PER_T];
  v4i vc[T::VC_PER_T];
  uint32_t ks, vs;

  __device__ __forceinline__ void load(const uint8_t* __restrict__ kcg, const uint8_t* __restrict__ ksg,
                                       const uint8_t* __restrict__ vcg, const uint8_t* __restrict__ vsg, long long bh,
                                       int Np, int kb, int tid) {
    const uint8_t* kbase = kcg + ((size_t)bh * Np + kb) * T::KROW;
#pragma unroll
    for (int i = 0; i < T::KC_PER_T; ++i) {
      const int u = (tid + 256 * i) % T::KC_UNITS;        // units beyond the tile repeat a valid one
      kc[i] = reinterpret_cast<const v4i*>(kbase)[u];
    }
#pragma unroll
    for (int i = 0; i < T::VC_PER_T; ++i) {
      const int u = (tid + 256 * i) % T::VC_UNITS;
      const int d = u / T::VCH, ch = u % T::VCH;
      vc[i] = *reinterpret_cast<const v4i*>(vcg + ((size_t)bh * D + d) * (Np / 2) + kb / 2 + ch * 16);
    }
    const int key = tid % BKV;
    const uint8_t* pk = ksg + ((size_t)bh * Np + kb + key) * (D / 32);
    ks = (D == 128) ? *reinterpret_cast<const uint32_t*>(pk) : (uint32_t)*reinterpret_cast<const uint16_t*>(pk);
    const int d = tid % D;
    const uint8_t* pv = vsg + ((size_t)bh * D + d) * (Np / 32) + kb / 32;
    vs = (BKV == 128) ? *reinterpret_cast<const uint32_t*>(pv) : (uint32_t)*reinterpret_cast<const uint16_t*>(pv);
  }

  __device__ __forceinline__ void store(uint8_t* lds, int tid) const {
#pragma unroll
    for (int i = 0; i < T::KC_PER_T; ++i) {
      const int u = (tid + 256 * i) % T::KC_UNITS;
      const int row = u / T::KCH, ch = u % T::KCH;
      *reinterpret_cast<v4i*>(lds + T::KC_OFF + row * T::KROW + swz<T::KCH>(row, ch) * 16) = kc[i];
    }
#pragma unroll
    for (int i = 0; i < T::VC_PER_T; ++i) {
      const int u = (tid + 256 * i) % T::VC_UNITS;
      const int row = u / T::VCH, ch = u % T::VCH;
      *reinterpret_cast<v4i*>(lds + T::VC_OFF + row * T::VROW + swz<T::VCH>(row, ch) * 16) = vc[i];
    }
    // Scale bytes of a row are split by lane half: the half-hi lanes of an
    // MFMA need bytes hi, hi+2 (blocks 2s + hi), so slot hi holds them as
    // bytes 0 and 1 and the MFMA op_sel picks byte s directly.  Duplicate
    // writers store identical values.
    const uint32_t k0 = (ks & 0xFFu) | ((ks >> 8) & 0xFF00u), k1 = ((ks >> 8) & 0xFFu) | ((ks >> 16) & 0xFF00u);
    const uint32_t v0 = (vs & 0xFFu) | ((vs >> 8) & 0xFF00u), v1 = ((vs >> 8) & 0xFFu) | ((vs >> 16) & 0xFF00u);
    *reinterpret_cast<uint2*>(lds + T::KS_OFF + (tid % BKV) * 8) = make_uint2(k0, k1);
    *reinterpret_cast<uint2*>(lds + T::VS_OFF + (tid % D) * 8) = make_uint2(v0, v1);
  }
};

__device__ __forceinline__ v8i as_op(const v4i x) { return v8i{x[0], x[1], x[2], x[3], 0, 0, 0, 0}; }

template <int D, int BKV, bool CAUSAL, int OUT>  // OUT: 0 = fp32, 1 = bf16, 2 = fp16
__global__ __launch_bounds__(256, 2) void attn_fp4_mx_kernel(
    const uint8_t* __restrict__ qc, const uint8_t* __restrict__ qs, const uint8_t* __restrict__ kc,
    const uint8_t* __restrict__ ks, const uint8_t* __restrict__ vc, const uint8_t* __restrict__ vs,
    void* __restrict__ o, int BH, int N, int Np, int nqt, float c2, float log6) {
  using T = Fp4Tile<D, BKV>;
  constexpr int NSUB = BKV / 32;   // 32-key subtiles of S^T
  constexpr int NG = BKV / 64;     // 64-key groups = PV K-steps
  constexpr int NKS = D / 64;      // QK K-steps
  constexpr int NDB = D / 32;      // 32-row blocks of O^T
  __shared__ __attribute__((aligned(16))) uint8_t lds[2][T::BYTES];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int col = lane & 31, hi = lane >> 5;

  // XCD-aware order: consecutive workgroups go round-robin over the 8 XCDs,
  // so give each XCD a contiguous range of (b,h, q-tile) work to keep one
  // head's K^/V^ in that XCD's L2.
  const int total = nqt * BH;
  int lin = blockIdx.x;
  if ((total & 7) == 0) lin = (blockIdx.x & 7) * (total >> 3) + (blockIdx.x >> 3);
  const long long bh = lin / nqt;
  int qt = lin % nqt;
  if (CAUSAL) qt = nqt - 1 - qt;            // longest rows first
  const int q0 = qt * AQ;
  const int qw = q0 + wave * 32;
  const int qi = qw + col;

  // Q^ fragment (B operand of S^T = K^ Q^T): 32 codes of block (2s + hi) per K-step s
  v4i qreg[NKS];
  uint32_t qsc = 0;
  if (qi < N) {
    const uint8_t* qrow = qc + ((size_t)bh * N + qi) * (D / 2);
#pragma unroll
    for (int s = 0; s < NKS; ++s) qreg[s] = *reinterpret_cast<const v4i*>(qrow + (2 * s + hi) * 16);
    const uint8_t* srow = qs + ((size_t)bh * N + qi) * (D / 32);
    qsc = (D == 128) ? *reinterpret_cast<const uint32_t*>(srow) : (uint32_t)*reinterpret_cast<const uint16_t*>(srow);
  } else {
#pragma unroll
    for (int s = 0; s < NKS; ++s) qreg[s] = v4i{0, 0, 0, 0};
  }
  qsc >>= 8 * hi;

  int ntiles = (N + BKV - 1) / BKV;
  if (CAUSAL) {
    const int qlast = min(q0 + AQ - 1, N - 1);
    ntiles = min(ntiles, qlast / BKV + 1);
  }

  v16f oacc[NDB];
#pragma unroll
  for (int db = 0; db < NDB; ++db) oacc[db] = v16f{};
  float m = -INFINITY, mc_old = -INFINITY, f_old = 0.0f, lsum_acc = 0.0f;

  // Per-lane LDS byte offsets, the same for every tile: A-operand chunk
  // (2s + hi) of row col (the swizzle depends on row bits 1..4 only, which
  // the 32-row subtile offset leaves unchanged).
  int koff[NKS], voff[NG];
#pragma unroll
  for (int s = 0; s < NKS; ++s) koff[s] = T::KC_OFF + col * T::KROW + swz<T::KCH>(col, 2 * s + hi) * 16;
#pragma unroll
  for (int g = 0; g < NG; ++g) voff[g] = T::VC_OFF + col * T::VROW + swz<T::VCH>(col, 2 * g + hi) * 16;
  const int ksoff = T::KS_OFF + col * 8 + hi * 4, vsoff = T::VS_OFF + col * 8 + hi * 4;

  Stage<D, BKV> stg;
  stg.load(kc, ks, vc, vs, bh, Np, 0, tid);
  stg.store(lds[0], tid);
  __syncthreads();

  auto tile = [&](auto BUF_, int j) {
    constexpr int buf = decltype(BUF_)::value;
    const uint8_t* L = lds[buf];
    const int kb = j * BKV;
    const bool more = j + 1 < ntiles;
    if (more) stg.load(kc, ks, vc, vs, bh, Np, kb + BKV, tid);

    const bool active = !CAUSAL || kb <= qw + 31;
    if (active) {
      // ---- S^T = K^ . Q^T ------------------------------------------------
      v16f sacc[NSUB];
#pragma unroll
      for (int t = 0; t < NSUB; ++t) {
        const uint32_t ksc = *reinterpret_cast<const uint32_t*>(L + ksoff + 32 * t * 8);
        v16f acc = v16f{};
        static_for<NKS>([&](auto S_) {
          constexpr int s = decltype(S_)::value;
          const v4i a = *reinterpret_cast<const v4i*>(L + koff[s] + 32 * t * T::KROW);
          acc = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(as_op(a), as_op(qreg[s]), acc, 4, 4, s, (int)ksc,
                                                                2 * s, (int)qsc);
        });
        sacc[t] = acc;
      }
      // ---- masking (tail keys >= N; causal keys > query) ---------------
      const bool need_mask = (kb + BKV > N) || (CAUSAL && kb + BKV - 1 > qw);
      if (need_mask) {
#pragma unroll
        for (int t = 0; t < NSUB; ++t)
#pragma unroll
          for (int v = 0; v < 16; ++v) {
            const int key = kb + 64 * (t >> 1) + 32 * hi + 16 * (t & 1) + v;
            const bool ok = key < N && (!CAUSAL || key <= qi);
            if (!ok) sacc[t][v] = -INFINITY;
          }
      }
      // ---- tile row max (raw scores); block max is lane-local ----------
      float bm[NG];
#pragma unroll
      for (int g = 0; g < NG; ++g) {
        // a serial chain: the compiler fuses it into v_max3 (a tree costs more)
        float x = sacc[2 * g][0];
#pragma unroll
        for (int v = 1; v < 16; ++v) x = __builtin_fmaxf(x, sacc[2 * g][v]);
#pragma unroll
        for (int v = 0; v < 16; ++v) x = __builtin_fmaxf(x, sacc[2 * g + 1][v]);
        bm[g] = x;
      }
      float tl = bm[0];
#pragma unroll
      for (int g = 1; g < NG; ++g) tl = __builtin_fmaxf(tl, bm[g]);
      // row max over the two lane halves that share a query
      const auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(tl), __float_as_uint(tl), false, false);
      const float t = __builtin_fmaxf(__uint_as_float(sw[0]), __uint_as_float(sw[1]));
      const float m_new = __builtin_fmaxf(m, t);
      const float tc = t * c2;
      const float mc = m_new * c2;
      const float delta = tc - mc;                       // c2 (t - m_new) <= 0
      const float kf = __builtin_floorf(delta);
      const float f = delta - kf;                        // in [0, 1)
      const float gam = __builtin_amdgcn_exp2f((mc_old - mc) + (f_old - f));
      const int kfold = (int)__builtin_fmaxf(kf, -300.0f);
      const float bias = log6 - tc;                      // P~2 = 2^{fma(S, c2, log2 6 - t c2)}

      // ---- P~2, unquantized row sum, FP4 pack with E8M0 block scales ----
      float ps[4] = {0.0f, 0.0f, 0.0f, 0.0f};            // independent partial row sums
      v4i pw[NG];
      int psb[NG];
#pragma unroll
      for (int g = 0; g < NG; ++g) {
        // smallest e with 6 2^e >= blockmax(P~2) = 6 2^{c2 (bm - t)}; a fully
        // masked block (bm = -inf) takes the floor -126
        const int e = (int)__builtin_fmaxf(__builtin_ceilf((bm[g] - t) * c2), -126.0f);
        const float escale = __builtin_ldexpf(1.0f, e);   // the convert divides by it exactly
        uint32_t w[4];
#pragma unroll
        for (int half = 0; half < 2; ++half) {
          const int tt = 2 * g + half;
#pragma unroll
          for (int q = 0; q < 2; ++q) {
            uint32_t word = 0;
            static_for<4>([&](auto I_) {
              constexpr int i = decltype(I_)::value;
              const float p0 = __builtin_amdgcn_exp2f(__builtin_fmaf(sacc[tt][8 * q + 2 * i], c2, bias));
              const float p1 = __builtin_amdgcn_exp2f(__builtin_fmaf(sacc[tt][8 * q + 2 * i + 1], c2, bias));
              ps[(2 * half + q) & 3] += p0;
              ps[(2 * half + q) & 3] += p1;
              word = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(word, p0, p1, escale, i);
            });
            w[2 * half + q] = word;
          }
        }
        pw[g] = v4i{(int)w[0], (int)w[1], (int)w[2], (int)w[3]};
        const int sb = e + kfold + 127;
        psb[g] = sb < 0 ? 0 : sb;
      }
      // ---- rescale and O^T += V^T . P^T ------------------------------------
#pragma unroll
      for (int db = 0; db < NDB; ++db)
#pragma unroll
        for (int v = 0; v < 16; ++v) oacc[db][v] *= gam;
      const float psum = (ps[0] + ps[1]) + (ps[2] + ps[3]);
      lsum_acc = lsum_acc * gam + __builtin_ldexpf(psum, kfold);
#pragma unroll
      for (int db = 0; db < NDB; ++db) {
        const uint32_t vsc = *reinterpret_cast<const uint32_t*>(L + vsoff + 32 * db * 8);
        static_for<NG>([&](auto G_) {
          constexpr int g = decltype(G_)::value;
          const v4i a = *reinterpret_cast<const v4i*>(L + voff[g] + 32 * db * T::VROW);
          oacc[db] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(as_op(a), as_op(pw[g]), oacc[db], 4, 4, g,
                                                                     (int)vsc, 0, psb[g]);
        });
      }
      m = m_new;
      mc_old = mc;
      f_old = f;
    }
    if (more) stg.store(lds[buf ^ 1], tid);
    __syncthreads();
  };

  for (int j = 0; j < ntiles; j += 2) {
    tile(ic<0>{}, j);
    if (j + 1 < ntiles) tile(ic<1>{}, j + 1);
  }

  // ---- epilogue: O = O^T / l, stored row-major ----------------------------
  const float ltot = lsum_acc + __shfl_xor(lsum_acc, 32, 64);
  const float inv = 1.0f / ltot;
  if (qi < N) {
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
static hipError_t launch_fp4_t(const void* qc, const void* qs, const void* kc, const void* ks, const void* vc,
                               const void* vs, void* o, int BH, int N, int Np, float c2, float log6, hipStream_t st) {
  const int nqt = (N + AQ - 1) / AQ;
  hipLaunchKernelGGL((attn_fp4_mx_kernel<D, BKV, CAUSAL, OUT>), dim3((unsigned)(nqt * BH)), dim3(256), 0, st,
                     (const uint8_t*)qc, (const uint8_t*)qs, (const uint8_t*)kc, (const uint8_t*)ks, (const uint8_t*)vc,
                     (const uint8_t*)vs, o, BH, N, Np, nqt, c2, log6);
  return hipGetLastError();
}

template <int D, int BKV, bool CAUSAL>
static hipError_t launch_fp4_o(int out, const void* qc, const void* qs, const void* kc, const void* ks, const void* vc,
                               const void* vs, void* o, int BH, int N, int Np, float c2, float log6, hipStream_t st) {
  if (out == 0) return launch_fp4_t<D, BKV, CAUSAL, 0>(qc, qs, kc, ks, vc, vs, o, BH, N, Np, c2, log6, st);
  if (out == 1) return launch_fp4_t<D, BKV, CAUSAL, 1>(qc, qs, kc, ks, vc, vs, o, BH, N, Np, c2, log6, st);
  return launch_fp4_t<D, BKV, CAUSAL, 2>(qc, qs, kc, ks, vc, vs, o, BH, N, Np, c2, log6, st);
}

hipError_t launch_attn_fp4_mx(const void* qc, const void* qs, const void* kc, const void* ks, const void* vc,
                              const void* vs, void* o, int BH, int N, int Np, int D, int bkv, bool causal, int out,
                              float c2, float log6, hipStream_t st) {
#define SAGE_A(DD, BB)                                                                              \
  return causal ? launch_fp4_o<DD, BB, true>(out, qc, qs, kc, ks, vc, vs, o, BH, N, Np, c2, log6, st) \
                : launch_fp4_o<DD, BB, false>(out, qc, qs, kc, ks, vc, vs, o, BH, N, Np, c2, log6, st)
  if (D == 128) { if (bkv == 128) { SAGE_A(128, 128); } else { SAGE_A(128, 64); } }
  else { if (bkv == 128) { SAGE_A(64, 128); } else { SAGE_A(64, 64); } }
#undef SAGE_A
}

}  // namespace sage
