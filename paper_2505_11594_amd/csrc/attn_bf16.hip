// bf16-MFMA comparison kernel for gfx950: FlashAttention forward (Sec. 2)
// with the same work decomposition as the FP4 kernel -- 4 waves x 32
// queries per workgroup, K and V^T tiles double-buffered in LDS, online
// softmax in registers -- on v_mfma_f32_32x32x16_bf16:
//   S^T (keys x queries) = K . Q^T     A = K tile (LDS), B = Q (registers)
//   O^T (dims x queries) += V^T . P^T  A = V^T tile (LDS), B = P in bf16
// S is fp32, the softmax is fp32, P is rounded to bf16 (nearest even) for the
// second product.  Layout (32x32x16): lane l holds row/column l%32 and
// K-indices [8*(l/32), +8); the accumulator of lane l holds column l%32 and
// rows 8g + 4*(l/32) + r.  The V^T pre-pass stores the tokens of every
// 16-token group with offset bits 2 and 3 swapped, so the 8 scores a lane
// holds for one 16-key K-step are exactly the keys its P operand slots need.
#include "sage_common.h"
#include "bf16_tile.h"

namespace sage {

constexpr int BQ = 128;        // queries per workgroup
constexpr int BK = 64;         // keys per tile
template <int D> using Bf16Tile = Bf16TileT<D, BK>;

__device__ __forceinline__ int vt_pos(int t) {
  // offset bits (b3 b2) swapped inside each 16-token group (an involution)
  return (t & ~12) | ((t & 4) << 1) | ((t & 8) >> 1);
}

// V [bh, N, D] -> V^T [bh, D, Np] (bf16), tokens permuted by vt_pos, tail zero.
template <int D>
__global__ __launch_bounds__(256) void transpose_v_kernel(const uint16_t* __restrict__ v, uint16_t* __restrict__ vt,
                                                          int N, int Np) {
  __shared__ uint16_t tile[64][D + 2];
  const int t0 = blockIdx.x * 64, bh = blockIdx.y, tid = threadIdx.x;
  const uint16_t* vb = v + (size_t)bh * N * D;
  constexpr int UPR = D / 8;
  for (int i = tid; i < 64 * UPR; i += 256) {
    const int r = i / UPR, cu = i % UPR;
    uint4 raw = make_uint4(0, 0, 0, 0);
    if (t0 + r < N) raw = *reinterpret_cast<const uint4*>(vb + (size_t)(t0 + r) * D + cu * 8);
    const uint16_t* h = reinterpret_cast<const uint16_t*>(&raw);
#pragma unroll
    for (int j = 0; j < 8; ++j) tile[r][cu * 8 + j] = h[j];
  }
  __syncthreads();
  // thread -> (channel d, 8 consecutive stored positions): one 16-byte store
  for (int i = tid; i < D * 8; i += 256) {
    const int d = i / 8, p0 = (i % 8) * 8;
    uint16_t o[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) o[j] = tile[vt_pos(p0 + j)][d];
    uint4 w;
    w.x = o[0] | ((uint32_t)o[1] << 16); w.y = o[2] | ((uint32_t)o[3] << 16);
    w.z = o[4] | ((uint32_t)o[5] << 16); w.w = o[6] | ((uint32_t)o[7] << 16);
    *reinterpret_cast<uint4*>(vt + ((size_t)bh * D + d) * Np + t0 + p0) = w;
  }
}

template <int D>
struct Bf16Stage {
  using T = Bf16Tile<D>;
  v4i k[T::KPT], v[T::VPT];
  __device__ __forceinline__ void load(const uint16_t* __restrict__ kg, const uint16_t* __restrict__ vtg, long long bh,
                                       int N, int Np, int kb, int tid) {
#pragma unroll
    for (int i = 0; i < T::KPT; ++i) {
      const int u = tid + 256 * i;
      const int row = u / T::KCH, ch = u % T::KCH;
      const int key = min(kb + row, N - 1);          // rows past N repeat a valid key (masked later)
      k[i] = *reinterpret_cast<const v4i*>(kg + ((size_t)bh * N + key) * D + ch * 8);
    }
#pragma unroll
    for (int i = 0; i < T::VPT; ++i) {
      const int u = tid + 256 * i;
      const int d = u / T::VCH, ch = u % T::VCH;
      v[i] = *reinterpret_cast<const v4i*>(vtg + ((size_t)bh * D + d) * Np + kb + ch * 8);
    }
  }
  __device__ __forceinline__ void store(uint8_t* lds, int tid) const {
#pragma unroll
    for (int i = 0; i < T::KPT; ++i) {
      const int u = tid + 256 * i;
      const int row = u / T::KCH, ch = u % T::KCH;
      *reinterpret_cast<v4i*>(lds + T::K_OFF + row * T::KROW + bswz<T::KCH>(row, ch) * 16) = k[i];
    }
#pragma unroll
    for (int i = 0; i < T::VPT; ++i) {
      const int u = tid + 256 * i;
      const int row = u / T::VCH, ch = u % T::VCH;
      *reinterpret_cast<v4i*>(lds + T::V_OFF + row * T::VROW + bswz<T::VCH>(row, ch) * 16) = v[i];
    }
  }
};


template <int D, bool CAUSAL, bool OUT_F32>
__global__ __launch_bounds__(256, 2) void attn_bf16_kernel(const uint16_t* __restrict__ q, const uint16_t* __restrict__ k,
                                                           const uint16_t* __restrict__ vt, void* __restrict__ o,
                                                           int BH, int N, int Np, int nqt, float c2) {
  using T = Bf16Tile<D>;
  constexpr int NSUB = BK / 32;    // 2 key subtiles
  constexpr int NKS = D / 16;      // QK K-steps
  constexpr int NPK = BK / 16;     // PV K-steps
  constexpr int NDB = D / 32;
  __shared__ __attribute__((aligned(16))) uint8_t lds[2][T::BYTES];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int col = lane & 31, hi = lane >> 5;

  const int total = nqt * BH;
  int lin = blockIdx.x;
  if ((total & 7) == 0) lin = (blockIdx.x & 7) * (total >> 3) + (blockIdx.x >> 3);
  const long long bh = lin / nqt;
  int qt = lin % nqt;
  if (CAUSAL) qt = nqt - 1 - qt;
  const int q0 = qt * BQ, qw = q0 + wave * 32, qi = qw + col;

  v4i qreg[NKS];
  {
    const int qr = min(qi, N - 1);
    const uint16_t* qrow = q + ((size_t)bh * N + qr) * D;
#pragma unroll
    for (int s = 0; s < NKS; ++s) qreg[s] = *reinterpret_cast<const v4i*>(qrow + 16 * s + 8 * hi);
  }
  int ntiles = (N + BK - 1) / BK;
  if (CAUSAL) ntiles = min(ntiles, min(q0 + BQ - 1, N - 1) / BK + 1);

  // per-lane V^T operand offsets (row col of each 32-row block, chunk 2u + hi)
  int vo[NPK];
#pragma unroll
  for (int u = 0; u < NPK; ++u) vo[u] = T::V_OFF + col * T::VROW + bswz<T::VCH>(col, 2 * u + hi) * 16;

  v16f oacc[NDB];
#pragma unroll
  for (int db = 0; db < NDB; ++db) oacc[db] = v16f{};
  float m = -INFINITY, l = 0.0f;

  Bf16Stage<D> stg;
  stg.load(k, vt, bh, N, Np, 0, tid);
  stg.store(lds[0], tid);
  __syncthreads();

  auto tile = [&](auto BUF_, int j) {
    constexpr int buf = decltype(BUF_)::value;
    const uint8_t* L = lds[buf];
    const int kb = j * BK;
    const bool more = j + 1 < ntiles;
    if (more) stg.load(k, vt, bh, N, Np, kb + BK, tid);
    if (!CAUSAL || kb <= qw + 31) {
      v16f sacc[NSUB];
#pragma unroll
      for (int t = 0; t < NSUB; ++t) {
        const int row = 32 * t + col;
        v16f acc = v16f{};
#pragma unroll
        for (int s = 0; s < NKS; ++s) {
          const v4i a = *reinterpret_cast<const v4i*>(L + T::K_OFF + row * T::KROW + bswz<T::KCH>(row, 2 * s + hi) * 16);
          acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf(a), as_bf(qreg[s]), acc, 0, 0, 0);
        }
        sacc[t] = acc;
      }
      if ((kb + BK > N) || (CAUSAL && kb + BK - 1 > qw)) {
#pragma unroll
        for (int t = 0; t < NSUB; ++t)
#pragma unroll
          for (int v = 0; v < 16; ++v) {
            const int key = kb + 32 * t + 8 * (v >> 2) + 4 * hi + (v & 3);
            if (!(key < N && (!CAUSAL || key <= qi))) sacc[t][v] = -INFINITY;
          }
      }
      float x = sacc[0][0];
#pragma unroll
      for (int t = 0; t < NSUB; ++t)
#pragma unroll
        for (int v = 0; v < 16; ++v) x = __builtin_fmaxf(x, sacc[t][v]);
      const auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
      const float tmax = __builtin_fmaxf(__uint_as_float(sw[0]), __uint_as_float(sw[1]));
      const float m_new = __builtin_fmaxf(m, tmax);
      const float mc = m_new * c2;
      const float alpha = __builtin_amdgcn_exp2f(m * c2 - mc);      // 0 on the first tile
      float ps[2] = {0.0f, 0.0f};
      v4i pk[NPK];
#pragma unroll
      for (int u = 0; u < NPK; ++u) {
        const int t = u >> 1, base = 8 * (u & 1);
        uint32_t w[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const float p0 = __builtin_amdgcn_exp2f(__builtin_fmaf(sacc[t][base + 2 * i], c2, -mc));
          const float p1 = __builtin_amdgcn_exp2f(__builtin_fmaf(sacc[t][base + 2 * i + 1], c2, -mc));
          ps[i & 1] += p0;
          ps[i & 1] += p1;
          typedef __bf16 v2bf __attribute__((ext_vector_type(2)));
          const v2bf pb = {(__bf16)p0, (__bf16)p1};
          w[i] = __builtin_bit_cast(uint32_t, pb);
        }
        pk[u] = v4i{(int)w[0], (int)w[1], (int)w[2], (int)w[3]};
      }
      l = l * alpha + (ps[0] + ps[1]);
      // rescale only when some row's max moved (alpha == 1 is an exact no-op)
      if (__ballot(alpha != 1.0f) != 0) {
#pragma unroll
        for (int db = 0; db < NDB; ++db)
#pragma unroll
          for (int v = 0; v < 16; ++v) oacc[db][v] *= alpha;
      }
#pragma unroll
      for (int db = 0; db < NDB; ++db)
#pragma unroll
        for (int u = 0; u < NPK; ++u) {
          const v4i a = *reinterpret_cast<const v4i*>(L + vo[u] + 32 * db * T::VROW);
          oacc[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf(a), as_bf(pk[u]), oacc[db], 0, 0, 0);
        }
      m = m_new;
    }
    if (more) stg.store(lds[buf ^ 1], tid);
    __syncthreads();
  };
  for (int j = 0; j < ntiles; j += 2) {
    tile(ic<0>{}, j);
    if (j + 1 < ntiles) tile(ic<1>{}, j + 1);
  }

  const float ltot = l + __shfl_xor(l, 32, 64);
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
        if (OUT_F32) *reinterpret_cast<float4*>(ob + idx * 4) = make_float4(a0, a1, a2, a3);
        else
          *reinterpret_cast<uint2*>(ob + idx * 2) =
              make_uint2((uint32_t)f32_to_bf16_rne(a0) | ((uint32_t)f32_to_bf16_rne(a1) << 16),
                         (uint32_t)f32_to_bf16_rne(a2) | ((uint32_t)f32_to_bf16_rne(a3) << 16));
      }
  }
}

hipError_t launch_transpose_v_bf16(const void* v, void* vt, int BH, int N, int Np, int D, hipStream_t st) {
  if (D == 128)
    hipLaunchKernelGGL((transpose_v_kernel<128>), dim3(Np / 64, BH), dim3(256), 0, st, (const uint16_t*)v, (uint16_t*)vt, N, Np);
  else
    hipLaunchKernelGGL((transpose_v_kernel<64>), dim3(Np / 64, BH), dim3(256), 0, st, (const uint16_t*)v, (uint16_t*)vt, N, Np);
  return hipGetLastError();
}

template <int D, bool CAUSAL, bool OUT_F32>
static hipError_t launch_bf16_t(const void* q, const void* k, const void* vt, void* o, int BH, int N, int Np, float c2,
                                hipStream_t st) {
  const int nqt = (N + BQ - 1) / BQ;
  hipLaunchKernelGGL((attn_bf16_kernel<D, CAUSAL, OUT_F32>), dim3((unsigned)(nqt * BH)), dim3(256), 0, st,
                     (const uint16_t*)q, (const uint16_t*)k, (const uint16_t*)vt, o, BH, N, Np, nqt, c2);
  return hipGetLastError();
}

hipError_t launch_attn_bf16(const void* q, const void* k, const void* vt, void* o, int BH, int N, int Np, int D,
                            bool causal, bool out_f32, float c2, hipStream_t st) {
#define SAGE_B(DD)                                                                                        \
  if (causal) return out_f32 ? launch_bf16_t<DD, true, true>(q, k, vt, o, BH, N, Np, c2, st)              \
                             : launch_bf16_t<DD, true, false>(q, k, vt, o, BH, N, Np, c2, st);            \
  return out_f32 ? launch_bf16_t<DD, false, true>(q, k, vt, o, BH, N, Np, c2, st)                         \
                 : launch_bf16_t<DD, false, false>(q, k, vt, o, BH, N, Np, c2, st)
  if (D == 128) { SAGE_B(128); }
  SAGE_B(64);
#undef SAGE_B
}

}  // namespace sage
