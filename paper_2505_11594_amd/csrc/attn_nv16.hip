// NV16 (E2M1 codes, 16-element blocks, E4M3 scales -- the paper's NVFP4,
// Sec. 3.1) attention forward for gfx950.  The block-scaled MFMA only takes
// E8M0 scales at 32-element granularity, so this path dequantizes exactly to
// f16 and runs both products on v_mfma_f32_32x32x16_f16.  An E2M1 value times
// an E4M3 scale has at most 6 significant bits and lies in [2^-10, 2688], so
// f16 holds it exactly.  An E4M3 scale s is M * 2^X with an integer M < 16,
// so code * s is v_cvt_scalef32_pk_f16_fp4 (code * 2^X, exact) times M
// (v_pk_mul_f16, exact): one convert and one packed multiply per two values.
//   * Q^ is dequantized once into the B-operand registers;
//   * K^ and V^T are expanded once per call into f16 copies in HBM (the same
//     exact values), and each tile of them is copied into LDS with
//     direct-to-LDS loads a tile ahead: no per-workgroup dequantization;
//   * P~ gets the two-level quantization of Sec. 3.2 with R = 448 * 6 in
//     registers: the first level as in the MXFP4 kernel, the second level an
//     E4M3 scale s = M * 2^X per 16 keys (round to nearest even of
//     blockmax/6), E2M1 codes of P~2 / s with the division by M folded into
//     the exponent and the one by 2^X into the convert, and the dequantized
//     code * s * 2^k fed to the MFMA in f16.
//     This is exact unless the tile's max lies more than 9 / c2 below the
//     running max; then values under 2^-9 of the row's largest round into
//     f16's subnormal range (an absolute error below 2^-25 there), and a
//     tile with k < -31 contributes zero.
// K^ is stored with the tokens of every 32-token group permuted (offset
// 16h + 4g + r at position 8g + 4h + r), so the 16 scores a lane holds for one
// 32-key subtile are one 16-key block of original keys and, split in halves,
// exactly the P operand of two 16-key K-steps; V^T stays in natural order.
#include "sage_common.h"
#include "bf16_tile.h"

namespace sage {

constexpr int NQ = 128;   // queries per workgroup (4 waves x 32)

typedef _Float16 v2h __attribute__((ext_vector_type(2)));
typedef _Float16 v8h __attribute__((ext_vector_type(8)));
__device__ __forceinline__ v8h as_h(const v4i x) { return __builtin_bit_cast(v8h, x); }

// Direct-to-LDS 16-byte load: lane l's bytes land at dst + 16 l.
__device__ __forceinline__ void nv_lds_load16(const void* src, void* dst) {
  __builtin_amdgcn_global_load_lds(src, (__attribute__((address_space(3))) void*)dst, 16, 0, 0);
}
__device__ __forceinline__ void nv_wait_loads() { __builtin_amdgcn_s_waitcnt(0x0F70); }   // vmcnt(0)
// a workgroup-uniform address in scalar registers (scalar base + lane offset)
__device__ __forceinline__ const uint8_t* nv_sbase(const void* p) {
  const uint64_t v = reinterpret_cast<uint64_t>(p);
  const uint64_t lo = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)v);
  const uint64_t hi = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)(v >> 32));
  return reinterpret_cast<const uint8_t*>((hi << 32) | lo);
}

// Exact f16 expansion of K^ and V^T.  Both are flat arrays of 32-element
// units (16 code bytes, two E4M3 scale bytes, one per 16 elements); unit u of
// K^ (row-major [BH, Np, D]) and of V^T ([BH, D, Np]) expands to the 32 f16
// values at element 32 u of K~ / V~^T, so the token order of K^ is kept.
// code * s = v_cvt_scalef32_pk_f16_fp4(code, 2^X) * M (s = M * 2^X), both
// steps exact.  One thread per unit; K units first, then V units.
__global__ __launch_bounds__(256) void nv16_expand_kernel(const uint8_t* __restrict__ kc, const uint8_t* __restrict__ ks,
                                                          const uint8_t* __restrict__ vc, const uint8_t* __restrict__ vs,
                                                          uint8_t* __restrict__ kh, uint8_t* __restrict__ vth,
                                                          long long units) {
  __shared__ float ptab[128];
  __shared__ uint32_t mtab[128];
  const int tid = threadIdx.x;
  if (tid < 128) {
    const int E = tid >> 3, man = tid & 7;
    ptab[tid] = __builtin_ldexpf(1.0f, E ? E - 10 : -9);
    const _Float16 M = (_Float16)(E ? 8 + man : man);
    mtab[tid] = __builtin_bit_cast(uint32_t, v2h{M, M});
  }
  __syncthreads();
  long long u = (long long)blockIdx.x * 256 + tid;
  if (u >= 2 * units) return;
  const bool isv = u >= units;
  if (isv) u -= units;
  const uint8_t* c = (isv ? vc : kc) + 16 * u;
  const uint32_t sc2 = *reinterpret_cast<const uint16_t*>((isv ? vs : ks) + 2 * u);
  const v4i codes = *reinterpret_cast<const v4i*>(c);
  const uint32_t b0 = sc2 & 0x7Fu, b1 = (sc2 >> 8) & 0x7Fu;   // scales are non-negative E4M3 codes
  const float x0 = ptab[b0], x1 = ptab[b1];
  const v2h m0 = __builtin_bit_cast(v2h, mtab[b0]), m1 = __builtin_bit_cast(v2h, mtab[b1]);
  v4i* out = reinterpret_cast<v4i*>((isv ? vth : kh) + 64 * u);
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    const uint32_t word = (uint32_t)codes[w];
    uint32_t ov[4];
    static_for<4>([&](auto B_) {
      constexpr int b = decltype(B_)::value;
      const v2h h = __builtin_amdgcn_cvt_scalef32_pk_f16_fp4(word, w < 2 ? x0 : x1, b) * (w < 2 ? m0 : m1);
      ov[b] = __builtin_bit_cast(uint32_t, h);
    });
    out[w] = v4i{(int)ov[0], (int)ov[1], (int)ov[2], (int)ov[3]};
  }
}

// OUT: 0 = fp32, 1 = bf16, 2 = fp16.  SQ: smoothing Q -- S += qkb[bh, query
// block, key] (Algorithm 1's GEMV of the block mean with K'; one row of Np
// floats per 128-query block, this workgroup's query tile).
template <int D, int BKV, bool CAUSAL, int OUT, bool SQ>
__global__ __launch_bounds__(256, 2) void attn_nv16_kernel(
    const uint8_t* __restrict__ qc, const uint8_t* __restrict__ qs, const uint8_t* __restrict__ kh,
    const uint8_t* __restrict__ vth, const float* __restrict__ qkb, void* __restrict__ o, int BH, int N, int Np,
    int nqt, float c2, float logR) {
  using T = Bf16TileT<D, BKV>;
  constexpr int NSUB = BKV / 32;   // 32-key subtiles = P blocks per lane
  constexpr int NKS = D / 16;      // QK K-steps
  constexpr int NPK = BKV / 16;    // PV K-steps
  constexpr int NDB = D / 32;
  constexpr int BIAS_OFF = T::BYTES, LBYTES = T::BYTES + (SQ ? BKV * 4 : 0);   // bias of the tile's keys
  __shared__ __attribute__((aligned(16))) uint8_t lds[2][LBYTES];
  // per E4M3 code b (s = M * 2^X) of P's second level, one 16-byte record (one
  // LDS read): {2^X, M, fl32(log2 M), {M, M} in f16} -- M = 1 and log2 M = 0
  // for s = 0, whose codes are multiplied by the f16 M = 0 and whose values
  // still enter the row sum
  __shared__ float4 stab[128];
  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int col = lane & 31, hi = lane >> 5;

  const int total = nqt * BH;
  int lin = blockIdx.x;
  if ((total & 7) == 0) lin = (blockIdx.x & 7) * (total >> 3) + (blockIdx.x >> 3);
  const long long bh = lin / nqt;
  int qt = lin % nqt;
  if (CAUSAL) qt = nqt - 1 - qt;
  const int q0 = qt * NQ, qw = q0 + wave * 32, qi = qw + col;

  // Q^ dequantized into the B operand: K-step s holds dims [16s + 8hi, +8) (block s)
  v4i qreg[NKS];
  {
    const int qr = min(qi, N - 1);
    const uint8_t* crow = qc + ((size_t)bh * N + qr) * (D / 2);
    const uint8_t* srow = qs + ((size_t)bh * N + qr) * (D / 16);
#pragma unroll
    for (int s = 0; s < NKS; ++s) {
      const uint32_t word = *reinterpret_cast<const uint32_t*>(crow + 8 * s + 4 * hi);
      const float sc = (qi < N) ? e4m3_decode_hw<0>(srow[s]) : 0.0f;
      uint32_t w[4];
      static_for<4>([&](auto B_) {
        constexpr int b = decltype(B_)::value;
        const auto f = __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(word, 1.0f, b);
        const v2h ph = {(_Float16)(f[0] * sc), (_Float16)(f[1] * sc)};   // exact in f16
        w[b] = __builtin_bit_cast(uint32_t, ph);
      });
      qreg[s] = v4i{(int)w[0], (int)w[1], (int)w[2], (int)w[3]};
    }
  }
  int ntiles = (N + BKV - 1) / BKV;
  if (CAUSAL) ntiles = min(ntiles, min(q0 + NQ - 1, N - 1) / BKV + 1);

  int vo[NPK];   // V^T operand offsets: K-step (t, w) reads keys 32t + 16hi + 8w + [0, 8)
#pragma unroll
  for (int u = 0; u < NPK; ++u)
    vo[u] = T::V_OFF + col * T::VROW + bswz<T::VCH>(col, 4 * (u >> 1) + 2 * hi + (u & 1)) * 16;

  v16f oacc[NDB];
#pragma unroll
  for (int db = 0; db < NDB; ++db) oacc[db] = v16f{};
  float m = -INFINITY, mc_old = -INFINITY, f_old = 0.0f, lsum_acc = 0.0f;

  if (tid < 128) {
    const int E = tid >> 3, man = tid & 7;
    const int Mi = E ? 8 + man : man;
    const _Float16 M = (_Float16)(E ? 8 + man : man);
    stab[tid] = make_float4(__builtin_ldexpf(1.0f, E ? E - 10 : -9), (float)(Mi ? Mi : 1),
                            (float)log2((double)(Mi ? Mi : 1)), __builtin_bit_cast(float, v2h{M, M}));
  }
  __syncthreads();
  // Tile loads, direct to LDS in the swizzled f16 layout.  Job J of a tile
  // (1 KiB, wave J % 4) covers K~ rows J * KRJ .. + KRJ (V~^T rows J * VRJ ..);
  // lane l fills LDS chunk l of the job, which holds logical chunk
  // bswz(row, l % KCH) of its row.  For J = wave + 4 i that chunk and the
  // lane's row within the job do not depend on i, so every load is a uniform
  // base plus one fixed lane offset per operand.
  constexpr int KRJ = 1024 / T::KROW, VRJ = 1024 / T::VROW;
  constexpr int NKJ = BKV * T::KROW / 1024 / 4, NVJ = D * T::VROW / 1024 / 4;   // jobs per wave
  static_assert(BKV * T::KROW % 4096 == 0 && D * T::VROW % 4096 == 0, "jobs split evenly over 4 waves");
  uint32_t klo, vlo;
  {
    const int kr = wave * KRJ + lane / T::KCH, vr = wave * VRJ + lane / T::VCH;
    klo = (uint32_t)((lane / T::KCH) * (D * 2) + bswz<T::KCH>(kr, lane % T::KCH) * 16);
    vlo = (uint32_t)((lane / T::VCH) * (Np * 2) + bswz<T::VCH>(vr, lane % T::VCH) * 16);
  }
  const uint8_t* kbase = kh + ((size_t)bh * Np + wave * KRJ) * (D * 2);
  const uint8_t* vbase = vth + ((size_t)bh * D + wave * VRJ) * ((size_t)Np * 2);
  // smoothing Q: the tile's BKV bias entries, 16 bytes per lane of wave 0
  const float* brow = SQ ? qkb + ((size_t)bh * nqt + qt) * Np : nullptr;
  auto issue = [&](int kb, uint8_t* L) {
#pragma unroll
    for (int i = 0; i < NKJ; ++i)
      nv_lds_load16(nv_sbase(kbase + ((size_t)kb + (size_t)4 * KRJ * i) * (D * 2)) + klo,
                    L + T::K_OFF + (wave + 4 * i) * 1024);
#pragma unroll
    for (int i = 0; i < NVJ; ++i)
      nv_lds_load16(nv_sbase(vbase + (size_t)4 * VRJ * i * ((size_t)Np * 2) + (size_t)kb * 2) + vlo,
                    L + T::V_OFF + (wave + 4 * i) * 1024);
    if constexpr (SQ) {
      if (wave == 0 && lane < BKV / 4) nv_lds_load16(brow + kb + 4 * lane, L + BIAS_OFF);
    }
  };
  issue(0, lds[0]);

  auto tile = [&](auto BUF_, int j) {
    constexpr int buf = decltype(BUF_)::value;
    const uint8_t* L = lds[buf];
    const int kb = j * BKV;
    nv_wait_loads();                                   // this wave's loads of tile j have landed
    __syncthreads();                                   // everyone's; every wave is past tile j - 1
    if (j + 1 < ntiles) issue(kb + BKV, lds[buf ^ 1]);
    if (!CAUSAL || kb <= qw + 31) {
      v16f sacc[NSUB];
#pragma unroll
      for (int t = 0; t < NSUB; ++t) {
        const int row = 32 * t + col;
        v16f acc = v16f{};
#pragma unroll
        for (int s = 0; s < NKS; ++s) {
          const v4i a = *reinterpret_cast<const v4i*>(L + T::K_OFF + row * T::KROW + bswz<T::KCH>(row, 2 * s + hi) * 16);
          acc = __builtin_amdgcn_mfma_f32_32x32x16_f16(as_h(a), as_h(qreg[s]), acc, 0, 0, 0);
        }
        sacc[t] = acc;
      }
      if constexpr (SQ) {
        // S = fl32(S + bias); element (t, v) is key kb + 32 t + 16 hi + v
#pragma unroll
        for (int t = 0; t < NSUB; ++t) {
          const float* bp = reinterpret_cast<const float*>(L + BIAS_OFF) + 32 * t + 16 * hi;
#pragma unroll
          for (int w4 = 0; w4 < 4; ++w4) {
            const v4f b = *reinterpret_cast<const v4f*>(bp + 4 * w4);
#pragma unroll
            for (int r = 0; r < 4; ++r) sacc[t][4 * w4 + r] = sacc[t][4 * w4 + r] + b[r];
          }
        }
      }
      if ((kb + BKV > N) || (CAUSAL && kb + BKV - 1 > qw)) {
        // element (t, v) is key kb + 16 hi + c with c = 32 t + v, kept iff c < rem; the
        // sign bit of c - rem turns -inf into the bound +inf for kept keys (bit
        // arithmetic, so no per-element lane masks are formed)
        const int rem = (CAUSAL ? min(N, qi + 1) : N) - kb - 16 * hi;
#pragma unroll
        for (int t = 0; t < NSUB; ++t)
#pragma unroll
          for (int v = 0; v < 16; ++v) {
            const float bound = __uint_as_float(0xFF800000u ^ ((uint32_t)(32 * t + v - rem) & 0x80000000u));
            sacc[t][v] = smin(sacc[t][v], bound);
          }
      }
      float bm[NSUB];
#pragma unroll
      for (int t = 0; t < NSUB; ++t) {
        float x = sacc[t][0];
#pragma unroll
        for (int v = 1; v < 16; ++v) x = smax(x, sacc[t][v]);   // scores are finite or -inf
        bm[t] = x;
      }
      float tl = bm[0];
#pragma unroll
      for (int t = 1; t < NSUB; ++t) tl = smax(tl, bm[t]);
      const auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(tl), __float_as_uint(tl), false, false);
      const float tmax = smax(__uint_as_float(sw[0]), __uint_as_float(sw[1]));
      const float m_new = smax(m, tmax);
      const float tc = tmax * c2, mc = m_new * c2;
      const float delta = tc - mc;
      const float kf = __builtin_floorf(delta);
      const float f = delta - kf;
      const float gam = __builtin_amdgcn_exp2f((mc_old - mc) + (f_old - f));
      const int kfold = (int)__builtin_fmaxf(kf, -300.0f);
      const float bias = logR - tc;                    // P~2 = 2^{fma(S, c2, log2 R - t c2)}, R = 448 * 6
      // k_j folded into the power of two of the dequantized P; below 2^-31 the
      // tile's blocks are dropped (their f16 M becomes 0)
      const int kfl = kfold < -31 ? -31 : kfold;
      const uint32_t mkeep = kfold < -31 ? 0u : 0xFFFFFFFFu;
      float ps[2] = {0.0f, 0.0f};
      v4i pk[NPK];
#pragma unroll
      for (int t = 0; t < NSUB; ++t) {
        // second level: E4M3 scale s = M 2^X of this lane's 16-key block, from its largest P~2
        // tmax and so bias are finite (every row of a tile that is computed has
        // a key of it that is not masked), so a masked block's bm = -inf gives 0
        const float amax = __builtin_amdgcn_exp2f(__builtin_fmaf(bm[t], c2, bias));
        const uint32_t sb = e4m3_encode_hw(div6(amax));
        const float4 rec = stab[sb];
        // the division by s folded into the exponent: y = 2^{fma(S, c2, B - log2 M)} = P~2 / M,
        // codes E2M1(y 2^-X) (the convert divides by the power of two exactly), row sum M sum y
        const float bb = bias - rec.z;
        const float x2 = rec.x;
        const float x2k = __builtin_ldexpf(rec.x, kfl);
        const v2h m2 = __builtin_bit_cast(v2h, __builtin_bit_cast(uint32_t, rec.w) & mkeep);
        float bs[2] = {0.0f, 0.0f};
#pragma unroll
        for (int w = 0; w < 2; ++w) {
          uint32_t pw[4];
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const int v = 8 * w + 2 * i;
            const float y0 = __builtin_amdgcn_exp2f(__builtin_fmaf(sacc[t][v], c2, bb));
            const float y1 = __builtin_amdgcn_exp2f(__builtin_fmaf(sacc[t][v + 1], c2, bb));
            bs[i & 1] += y0;
            bs[i & 1] += y1;
            // byte 0 gets the two codes; the other bytes are never read
            const uint32_t code = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(__float_as_uint(y0), y0, y1, x2, 0);
            pw[i] = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_f16_fp4(code, x2k, 0) * m2);
          }
          pk[2 * t + w] = v4i{(int)pw[0], (int)pw[1], (int)pw[2], (int)pw[3]};
        }
        ps[t & 1] = __builtin_fmaf(bs[0] + bs[1], rec.y, ps[t & 1]);
      }
#pragma unroll
      for (int db = 0; db < NDB; ++db)
#pragma unroll
        for (int v = 0; v < 16; ++v) oacc[db][v] *= gam;
      lsum_acc = lsum_acc * gam + __builtin_ldexpf(ps[0] + ps[1], kfold);
#pragma unroll
      for (int db = 0; db < NDB; ++db)
#pragma unroll
        for (int u = 0; u < NPK; ++u) {
          const v4i a = *reinterpret_cast<const v4i*>(L + vo[u] + 32 * db * T::VROW);
          oacc[db] = __builtin_amdgcn_mfma_f32_32x32x16_f16(as_h(a), as_h(pk[u]), oacc[db], 0, 0, 0);
        }
      m = m_new;
      mc_old = mc;
      f_old = f;
    }
  };
  for (int j = 0; j < ntiles; j += 2) {
    tile(ic<0>{}, j);
    if (j + 1 < ntiles) tile(ic<1>{}, j + 1);
  }

  const float ltot = lsum_acc + __shfl_xor(lsum_acc, 32, 64);
  const float inv = 1.0f / ltot;
  if (qi < N) {
    uint8_t* ob = reinterpret_cast<uint8_t*>(o);
#pragma unroll
    for (int db = 0; db < NDB; ++db)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int d0 = 32 * db + 8 * g + 4 * hi;
        const size_t idx = ((size_t)bh * N + qi) * D + d0;
        const float a0 = oacc[db][4 * g] * inv, a1 = oacc[db][4 * g + 1] * inv;
        const float a2 = oacc[db][4 * g + 2] * inv, a3 = oacc[db][4 * g + 3] * inv;
        if (OUT == 0) {
          *reinterpret_cast<float4*>(ob + idx * 4) = make_float4(a0, a1, a2, a3);
        } else {
          uint16_t h0, h1, h2, h3;
          if (OUT == 1) { h0 = f32_to_bf16_rne(a0); h1 = f32_to_bf16_rne(a1); h2 = f32_to_bf16_rne(a2); h3 = f32_to_bf16_rne(a3); }
          else { h0 = f32_to_fp16_rne(a0); h1 = f32_to_fp16_rne(a1); h2 = f32_to_fp16_rne(a2); h3 = f32_to_fp16_rne(a3); }
          *reinterpret_cast<uint2*>(ob + idx * 2) = make_uint2((uint32_t)h0 | ((uint32_t)h1 << 16), (uint32_t)h2 | ((uint32_t)h3 << 16));
        }
      }
  }
}

template <int D, int BKV, bool CAUSAL, int OUT, bool SQ>
static hipError_t launch_nv16_t(const void* qc, const void* qs, const uint8_t* kh, const uint8_t* vth, const float* qkb,
                                void* o, int BH, int N, int Np, float c2, float logR, hipStream_t st) {
  const int nqt = (N + NQ - 1) / NQ;
  hipLaunchKernelGGL((attn_nv16_kernel<D, BKV, CAUSAL, OUT, SQ>), dim3((unsigned)(nqt * BH)), dim3(256), 0, st,
                     (const uint8_t*)qc, (const uint8_t*)qs, kh, vth, qkb, o, BH, N, Np, nqt, c2, logR);
  return hipGetLastError();
}

template <int D, int BKV, bool CAUSAL, bool SQ>
static hipError_t launch_nv16_o(int out, const void* qc, const void* qs, const uint8_t* kh, const uint8_t* vth,
                                const float* qkb, void* o, int BH, int N, int Np, float c2, float logR, hipStream_t st) {
  if (out == 0) return launch_nv16_t<D, BKV, CAUSAL, 0, SQ>(qc, qs, kh, vth, qkb, o, BH, N, Np, c2, logR, st);
  if (out == 1) return launch_nv16_t<D, BKV, CAUSAL, 1, SQ>(qc, qs, kh, vth, qkb, o, BH, N, Np, c2, logR, st);
  return launch_nv16_t<D, BKV, CAUSAL, 2, SQ>(qc, qs, kh, vth, qkb, o, BH, N, Np, c2, logR, st);
}

template <int D, int BKV, bool CAUSAL>
static hipError_t launch_nv16_s(int out, const void* qc, const void* qs, const uint8_t* kh, const uint8_t* vth,
                                const float* qkb, void* o, int BH, int N, int Np, float c2, float logR, hipStream_t st) {
  return qkb ? launch_nv16_o<D, BKV, CAUSAL, true>(out, qc, qs, kh, vth, qkb, o, BH, N, Np, c2, logR, st)
             : launch_nv16_o<D, BKV, CAUSAL, false>(out, qc, qs, kh, vth, qkb, o, BH, N, Np, c2, logR, st);
}

size_t nv16_expand_bytes(int BH, int Np, int D) { return 2 * (size_t)BH * Np * D * sizeof(uint16_t); }

// kv16: nv16_expand_bytes(BH, Np, D) bytes of device memory (256-byte aligned)
// for the f16 expansion of K^ (first half) and V^T (second half).
// qkb: smoothing-Q bias [BH, ceil(N/128), Np] fp32, or null without smoothing Q.
hipError_t launch_attn_nv16(const void* qc, const void* qs, const void* kc, const void* ks, const void* vc,
                            const void* vs, void* kv16, const float* qkb, void* o, int BH, int N, int Np, int D,
                            int bkv, bool causal, int out, float c2, float logR, hipStream_t st) {
  const long long units = (long long)BH * Np * (D / 32);   // 32-element units of K^, and of V^T
  uint8_t* kh = static_cast<uint8_t*>(kv16);
  uint8_t* vth = kh + nv16_expand_bytes(BH, Np, D) / 2;
  hipLaunchKernelGGL(nv16_expand_kernel, dim3((unsigned)((2 * units + 255) / 256)), dim3(256), 0, st,
                     (const uint8_t*)kc, (const uint8_t*)ks, (const uint8_t*)vc, (const uint8_t*)vs, kh, vth, units);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
#define SAGE_N(DD, BB)                                                                              \
  return causal ? launch_nv16_s<DD, BB, true>(out, qc, qs, kh, vth, qkb, o, BH, N, Np, c2, logR, st) \
                : launch_nv16_s<DD, BB, false>(out, qc, qs, kh, vth, qkb, o, BH, N, Np, c2, logR, st)
  if (D == 128) { if (bkv == 128) { SAGE_N(128, 128); } else { SAGE_N(128, 64); } }
  else { if (bkv == 128) { SAGE_N(64, 128); } else { SAGE_N(64, 64); } }
#undef SAGE_N
}

}  // namespace sage
