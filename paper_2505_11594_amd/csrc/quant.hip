// Quantization kernels for gfx950: smoothing-K mean, FP4 microscaling of Q and
// K along the head dimension, and of V along tokens with the transpose fused in.
//
// phi (Sec. 3.1, Eq. microscaling): per 1 x n block, s = max|x| / 6 stored as
// E8M0 (MXFP4, n = 32: the smallest power of two with 6 s >= max) or E4M3
// (n = 16, round to nearest even, saturating at 448); codes are FP4 E2M1
// round-to-nearest-even of x / s.  Smoothing K (Algorithm 1 preprocessing)
// subtracts the per-(b,h) channel mean first, smoothing Q (Algorithm 1) the
// mean of each block of QB query rows; the V transpose is fused into its
// quantization (Appendix, "Transposing V").  For smoothing Q the GEMV of the
// block means with K' is computed here as well.
//
// All three kernels are HBM-bound: each element is read once as 16 bits
// (twice for K, which the mean also reads) and written as 4 bits plus 8 bits
// per block.
#include <climits>

#include "sage_common.h"

namespace sage {

// ---------------------------------------------------------------------------
// Smoothing K, pass 1: per-chunk fp64 column sums.  Block (chunk, bh) sums
// tokens [chunk * KM_CHUNK, ...) of K[bh] for every channel.  Every value is a
// 16-bit float, so the fp64 partial sums are exact for the token counts used
// here and the final mean does not depend on the summation order.
// ---------------------------------------------------------------------------
constexpr int KM_CHUNK = 512;
constexpr int KM_THREADS = 256;

template <int D, bool BF16>
__global__ __launch_bounds__(KM_THREADS) void kmean_partial_kernel(const uint16_t* __restrict__ k,
                                                                   double* __restrict__ part, int N,
                                                                   int nchunk) {
  constexpr int CG = D / 8;                  // 8-channel groups per row (16 bytes)
  constexpr int RS = KM_THREADS / CG;        // rows handled in parallel
  const int chunk = blockIdx.x, bh = blockIdx.y;
  const int tid = threadIdx.x;
  const int cg = tid % CG, rsub = tid / CG;
  const int t0 = chunk * KM_CHUNK;
  const int t1 = min(N, t0 + KM_CHUNK);
  const uint16_t* kb = k + (size_t)bh * N * D;
  double acc[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) acc[i] = 0.0;
  for (int t = t0 + rsub; t < t1; t += RS) {
    uint4 raw = *reinterpret_cast<const uint4*>(kb + (size_t)t * D + cg * 8);
    const uint16_t* h = reinterpret_cast<const uint16_t*>(&raw);
#pragma unroll
    for (int i = 0; i < 8; ++i) acc[i] += (double)widen<BF16>(h[i]);
  }
  __shared__ double red[KM_THREADS][9];      // padded against bank conflicts
#pragma unroll
  for (int i = 0; i < 8; ++i) red[tid][i] = acc[i];
  __syncthreads();
  if (tid < D) {
    const int c = tid, g = c / 8, i = c % 8;
    double s = 0.0;
    for (int r = 0; r < RS; ++r) s += red[r * CG + g][i];
    part[((size_t)bh * nchunk + chunk) * D + c] = s;
  }
}

// Pass 2: mu = fl32(fl64(sum) / N).  One workgroup per (b,h): 256 / D
// threads per channel sum strided chunks, then one of them adds the partial
// sums (exact in fp64, so the order does not matter).
template <int D>
__global__ __launch_bounds__(256) void kmean_final_kernel(const double* __restrict__ part, float* __restrict__ mu,
                                                          int N, int nchunk) {
  constexpr int TPC = 256 / D;
  const int bh = blockIdx.x, tid = threadIdx.x, c = tid % D, k = tid / D;
  double s = 0.0;
  for (int j = k; j < nchunk; j += TPC) s += part[((size_t)bh * nchunk + j) * D + c];
  __shared__ double red[256];
  red[tid] = s;
  __syncthreads();
  if (k == 0) {
    double t = 0.0;
#pragma unroll
    for (int i = 0; i < TPC; ++i) t += red[i * D + c];
    mu[(size_t)bh * D + c] = (float)(t / (double)N);
  }
}

// ---------------------------------------------------------------------------
// Smoothing Q (Algorithm 1): qbar[bh, b, c] = mean of Q[bh, t, c] over the QB
// rows t of query block b (the last block holds the remaining rows), an fp64
// sum -- exact for 16-bit inputs, so the order does not matter -- divided by
// the row count and rounded once to fp32.  One workgroup per (block, bh).
// ---------------------------------------------------------------------------
constexpr int QB = 128;   // query rows per smoothing block (= the attention kernel's query tile)

template <int D, bool BF16>
__global__ __launch_bounds__(KM_THREADS) void qmean_kernel(const uint16_t* __restrict__ q, float* __restrict__ qbar,
                                                           int N, int nqb) {
  constexpr int CG = D / 8, RS = KM_THREADS / CG;
  const int b = blockIdx.x, bh = blockIdx.y, tid = threadIdx.x;
  const int cg = tid % CG, rsub = tid / CG;
  const int t0 = b * QB, t1 = min(N, t0 + QB);
  const uint16_t* qh = q + (size_t)bh * N * D;
  double acc[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) acc[i] = 0.0;
  for (int t = t0 + rsub; t < t1; t += RS) {
    uint4 raw = *reinterpret_cast<const uint4*>(qh + (size_t)t * D + cg * 8);
    const uint16_t* h = reinterpret_cast<const uint16_t*>(&raw);
#pragma unroll
    for (int i = 0; i < 8; ++i) acc[i] += (double)widen<BF16>(h[i]);
  }
  __shared__ double red[KM_THREADS][9];
#pragma unroll
  for (int i = 0; i < 8; ++i) red[tid][i] = acc[i];
  __syncthreads();
  if (tid < D) {
    const int c = tid, g = c / 8, i = c % 8;
    double s = 0.0;
    for (int r = 0; r < RS; ++r) s += red[r * CG + g][i];
    qbar[((size_t)bh * nqb + b) * D + c] = (float)(s / (double)(t1 - t0));
  }
}

// GEMV of smoothing Q: bias[bh, b, k] = qbar[bh, b, :] . K'[bh, k, :] with
// K' = fl32(K - mu) (K itself without smoothing K), as a chain of fp32 fused
// multiply-adds in order of the channel from 0; keys k >= N get 0.  One
// thread per key keeps K' in registers; the workgroup stages the means of QBG
// query blocks at a time in LDS as [channel][block] (double-buffered), so a
// thread reads the QBG values of one channel with two broadcast 16-byte LDS
// reads and runs QBG independent chains.
constexpr int QBG = 8;
constexpr int QB_THREADS = 256;

template <int D, bool BF16>
__global__ __launch_bounds__(QB_THREADS) void qk_bias_kernel(const uint16_t* __restrict__ k, const float* __restrict__ mu,
                                                             const float* __restrict__ qbar, float* __restrict__ bias,
                                                             int N, int Np, int nqb) {
  static_assert(D * QBG == 4 * QB_THREADS || D * QBG == 2 * QB_THREADS, "one or two staged means per thread");
  constexpr int PER_T = D * QBG / QB_THREADS;      // means staged per thread per group
  __shared__ __attribute__((aligned(16))) float qs[2][D][QBG];
  const int bh = blockIdx.y, tid = threadIdx.x;
  const int key = blockIdx.x * QB_THREADS + tid;   // the grid covers Np (a multiple of 128) rounded up
  const bool valid = key < N;
  float kv[D];
  if (valid) {
    const uint16_t* kr = k + ((size_t)bh * N + key) * D;
#pragma unroll
    for (int c8 = 0; c8 < D / 8; ++c8) {
      uint4 raw = *reinterpret_cast<const uint4*>(kr + c8 * 8);
      const uint16_t* h = reinterpret_cast<const uint16_t*>(&raw);
#pragma unroll
      for (int i = 0; i < 8; ++i) kv[c8 * 8 + i] = widen<BF16>(h[i]);
    }
    if (mu != nullptr) {
#pragma unroll
      for (int c = 0; c < D; ++c) kv[c] = kv[c] - mu[(size_t)bh * D + c];
    }
  } else {
#pragma unroll
    for (int c = 0; c < D; ++c) kv[c] = 0.0f;
  }
  const float* qm = qbar + (size_t)bh * nqb * D;
  // stage the means of blocks [b0, b0 + QBG) (zero past nqb), transposed to [channel][block]
  auto stage = [&](int b0, int buf) {
#pragma unroll
    for (int e = 0; e < PER_T; ++e) {
      const int idx = tid * PER_T + e, i = idx / D, c = idx % D;   // block i, channel c
      qs[buf][c][i] = (b0 + i < nqb) ? qm[(size_t)(b0 + i) * D + c] : 0.0f;
    }
  };
  const int ngroups = (nqb + QBG - 1) / QBG;
  stage(0, 0);
  __syncthreads();
  for (int gi = 0; gi < ngroups; ++gi) {
    const int b0 = gi * QBG, buf = gi & 1;
    if (gi + 1 < ngroups) stage(b0 + QBG, buf ^ 1);   // the other buffer was last read before the barrier below
    float acc[QBG];
#pragma unroll
    for (int i = 0; i < QBG; ++i) acc[i] = 0.0f;
#pragma unroll
    for (int c = 0; c < D; ++c) {
      const v4f m0 = *reinterpret_cast<const v4f*>(&qs[buf][c][0]);
      const v4f m1 = *reinterpret_cast<const v4f*>(&qs[buf][c][4]);
#pragma unroll
      for (int i = 0; i < 4; ++i) acc[i] = __builtin_fmaf(m0[i], kv[c], acc[i]);
#pragma unroll
      for (int i = 0; i < 4; ++i) acc[4 + i] = __builtin_fmaf(m1[i], kv[c], acc[4 + i]);
    }
    // materialize every chain here: otherwise the compiler sinks each chain into
    // its guarded store below and keeps all the staged means it reads live
#pragma unroll
    for (int i = 0; i < QBG; ++i) asm volatile("" : "+v"(acc[i]));
    if (key < Np) {
      float* out = bias + ((size_t)bh * nqb + b0) * Np + key;
#pragma unroll
      for (int i = 0; i < QBG; ++i)
        if (b0 + i < nqb) out[(size_t)i * Np] = valid ? acc[i] : 0.0f;
    }
    __syncthreads();
  }
}

// ---------------------------------------------------------------------------
// Row quantizer for Q and K (blocks along D).  One lane owns 8 consecutive
// channels (a 16-byte load); the 4 (MXFP4) or 2 (NV16) lanes of a block
// reduce their absolute maxima with cross-lane swaps.  A lane writes its 8
// codes as one 32-bit word.  A mean, when given, is subtracted first: row t
// of head bh uses mu[(bh * nmb + (t >> mshift)) * D + c] (role K: one mean
// per head; role Q with smoothing: one per QB-row block).  Role K stores each
// token at its permuted position inside its group.
// ---------------------------------------------------------------------------
// Stored row of K token t.  MXFP4 (32x32x64 block-scaled MFMA): inside each
// 64-token group, offset o = 32h + 16t' + 4g + r goes to 32t' + 8g + 4h + r.
// NV16 (32x32x16 bf16 MFMA after dequantization): inside each 32-token group,
// o = 16h + 4g + r goes to 8g + 4h + r.
template <int FMT>
__device__ __forceinline__ int k_stored_pos(int t) {
  if constexpr (FMT == kFmtMX) {
    const int o = t & 63;
    const int h = o >> 5, tt = (o >> 4) & 1, g = (o >> 2) & 3, r = o & 3;
    return (t & ~63) | (tt << 5) | (g << 3) | (h << 2) | r;
  } else {
    const int o = t & 31;
    const int h = o >> 4, g = (o >> 2) & 3, r = o & 3;
    return (t & ~31) | (g << 3) | (h << 2) | r;
  }
}

// Units (8 channels of one row) per thread of the row quantizer: role K reads
// the mean beside each unit, and four units per thread, their loads issued
// together, keep more bytes in flight (K 82 -> 67 us on B1 H32 N32768 D128);
// Q is fastest with one (four: +4%).
template <bool IS_K>
constexpr int rows_units() { return IS_K ? 4 : 1; }

template <int D, bool BF16, int FMT, bool IS_K>
__global__ __launch_bounds__(256) void quant_rows_kernel(const uint16_t* __restrict__ x, const float* __restrict__ mu,
                                                         int mshift, int nmb, uint8_t* __restrict__ codes,
                                                         uint8_t* __restrict__ scales, int N, int Nout,
                                                         long long total_units) {
  constexpr int NB = (FMT == kFmtMX) ? 32 : 16;     // block size
  constexpr int LPB = NB / 8;                       // lanes per block
  constexpr int UPR = D / 8;                        // units (lanes) per row
  constexpr int U = rows_units<IS_K>();
  // a workgroup of 256 threads takes U x 256 consecutive units, 256 per step
  // (each load coalesced across the wave), all loads issued before the first
  // is used
  const long long nsb = (total_units + 256 * U - 1) / (256 * U);
  for (long long sb = blockIdx.x; sb < nsb; sb += gridDim.x) {
    const long long u0 = sb * (256 * U) + threadIdx.x;
    uint4 raws[U];
#pragma unroll
    for (int k = 0; k < U; ++k) {
      const long long u = u0 + 256 * k;
      raws[k] = (u < total_units) ? *reinterpret_cast<const uint4*>(x + (size_t)u * 8) : make_uint4(0, 0, 0, 0);
    }
#pragma unroll
    for (int k = 0; k < U; ++k) {
      const long long u = u0 + 256 * k;
      if (u >= total_units) break;                    // whole rows, so whole blocks of lanes, leave together
      const long long row = u / UPR;                  // (bh, t) flattened over the N input rows
      const int cu = (int)(u % UPR);
      const long long bh = row / N;
      const int t = (int)(row % N);
      const uint16_t* hv = reinterpret_cast<const uint16_t*>(&raws[k]);
      float v[8];
#pragma unroll
      for (int i = 0; i < 8; ++i) v[i] = widen<BF16>(hv[i]);
      if (mu != nullptr) {
        const float* m = mu + ((size_t)bh * nmb + (t >> mshift)) * D + cu * 8;
#pragma unroll
        for (int i = 0; i < 8; ++i) v[i] = v[i] - m[i];
      }
      float am = 0.0f;
#pragma unroll
      for (int i = 0; i < 8; ++i) am = __builtin_fmaxf(am, __builtin_fabsf(v[i]));
#pragma unroll
      for (int off = 1; off < LPB; off <<= 1) am = __builtin_fmaxf(am, __shfl_xor(am, off, 64));
      uint32_t sbyte;
      float y[8];
      if (FMT == kFmtMX) {
        const int e = e8m0_exponent(am);
        sbyte = (uint32_t)(e + 127);
#pragma unroll
        for (int i = 0; i < 8; ++i) y[i] = __builtin_ldexpf(v[i], -e);   // exact power-of-two scaling
      } else {
        sbyte = e4m3_encode(am / 6.0f);
        const float s = e4m3_decode(sbyte);
        if (s == 0.0f) {
#pragma unroll
          for (int i = 0; i < 8; ++i) y[i] = 0.0f;
        } else {
          const float r = 1.0f / s;
#pragma unroll
          for (int i = 0; i < 8; ++i) y[i] = v[i] * r;
        }
      }
      uint32_t word = 0;
#pragma unroll
      for (int i = 0; i < 4; ++i) word |= cvt_fp4x2(y[2 * i], y[2 * i + 1]) << (8 * i);
      const long long orow = bh * Nout + (IS_K ? k_stored_pos<FMT>(t) : t);
      *reinterpret_cast<uint32_t*>(codes + (size_t)orow * (D / 2) + cu * 4) = word;
      if ((cu % LPB) == 0) scales[(size_t)orow * (D / NB) + cu / LPB] = (uint8_t)sbyte;
    }
  }
}

// Zero codes (and unit scales) of K's padded tail tokens N .. Np-1.
template <int D, int FMT>
__global__ void k_tail_kernel(uint8_t* __restrict__ codes, uint8_t* __restrict__ scales, int N, int Np) {
  constexpr int NB = (FMT == kFmtMX) ? 32 : 16;
  const int bh = blockIdx.y;
  const int ntail = Np - N;
  for (int i = threadIdx.x + blockIdx.x * blockDim.x; i < ntail * (D / 2); i += gridDim.x * blockDim.x) {
    const int t = N + i / (D / 2), b = i % (D / 2);
    const long long orow = (long long)bh * Np + k_stored_pos<FMT>(t);
    codes[(size_t)orow * (D / 2) + b] = 0;
    if (b < D / NB) scales[(size_t)orow * (D / NB) + b] = (FMT == kFmtMX) ? 127 : 0;
  }
}

// ---------------------------------------------------------------------------
// V quantizer with the transpose fused in.  A block of 256 threads stages a
// 128-token x D tile in LDS (coalesced 16-byte loads), then each thread
// quantizes whole token blocks of one channel and writes them contiguously
// into V^T [bh, d, Np/2].  Tokens >= N are zero.  Each block walks a
// contiguous range of per_wg (bh, tile) pairs and keeps the loads of the next
// two tiles in registers while it quantizes the current one.
// ---------------------------------------------------------------------------
constexpr int VT = 128;       // tokens per tile (a V^T row segment of 64 bytes)
// One workgroup per CU, two tiles in flight: 79.7 us on B1 H32 N32768 D128,
// against 96 us for one tile per workgroup and, with the same loop, 92 us at
// two workgroups per CU (one tile ahead: 83.5 us at one per CU, 87, 96 and
// 101 us at two, three and four); with the scale bytes staged, 71.4 us.
constexpr int V_WG_PER_CU = 1;

template <int D, bool BF16, int FMT>
__global__ __launch_bounds__(256) void quant_v_kernel(const uint16_t* __restrict__ v, uint8_t* __restrict__ codes,
                                                      uint8_t* __restrict__ scales, int N, int Np, int total,
                                                      int per_wg) {
  constexpr int NB = (FMT == kFmtMX) ? 32 : 16;
  // all lanes of a wave read one row (consecutive channels): no padding needed
  __shared__ uint16_t tile[VT][D];
  // The scale bytes of up to ST_TILES consecutive tiles of one head, per
  // V^T row: one 128-byte segment of the row, stored whole (written one byte
  // per block as they come, a row's line would fill over the workgroup's
  // whole range and partly leave L2 before it is complete).  Rows are 132
  // bytes apart, so the byte writes of a wave's channels fall in different banks.
  constexpr int SPT = VT / NB, ST_TILES = 128 / SPT, ST_ROW = 132;
  __shared__ __attribute__((aligned(16))) uint8_t sst[D * ST_ROW];
  const int ntt = (Np + VT - 1) / VT;
  // Workgroups are dealt round-robin to the 8 XCDs; give each XCD a contiguous
  // range of (bh, tile), so the two 64-byte halves of every 128-byte V^T line
  // are written through the same L2, mostly by one workgroup, one tile apart.
  int w = blockIdx.x;
  if ((gridDim.x & 7) == 0) w = (blockIdx.x & 7) * (gridDim.x >> 3) + (blockIdx.x >> 3);
  const int first = w * per_wg, last = min(total, first + per_wg);
  const int tid = threadIdx.x;
  constexpr int UPR = D / 8, LPT = VT * UPR / 256;   // 16-byte units per row, per thread
  static_assert(LPT * 256 == VT * UPR, "tile loads split evenly");
  uint4 ra[LPT], rb[LPT];
  auto load = [&](int lin, uint4 (&raw)[LPT]) {
    const int t0 = (lin % ntt) * VT;
    const uint16_t* vb = v + (size_t)(lin / ntt) * N * D;
#pragma unroll
    for (int k = 0; k < LPT; ++k) {
      const int i = tid + 256 * k, t = t0 + i / UPR;
      raw[k] = (t < N) ? *reinterpret_cast<const uint4*>(vb + (size_t)t * D + (i % UPR) * 8) : make_uint4(0, 0, 0, 0);
    }
  };
  if (first < last) load(first, ra);
  if (first + 1 < last) load(first + 1, rb);
  // each thread quantizes CPT adjacent channels of BPT token blocks (one
  // 32-bit LDS read per token for two channels)
  constexpr int CPT = (D == 128) ? 2 : 1;
  constexpr int TPG = 256 / (D / CPT);       // threads per channel group
  constexpr int BPT = VT / NB / TPG;         // token blocks per thread
  static_assert(BPT >= 1 && TPG * (D / CPT) == 256, "tile shape");
  const int c0 = (tid % (D / CPT)) * CPT, part = tid / (D / CPT);
  int nst = 0;                               // tiles staged in sst (consecutive, one head)
  auto flush = [&](int lin_last) {           // workgroup-uniform
    __syncthreads();                         // every staged byte is written
    const int lin0 = lin_last - nst + 1;
    const int t0 = (lin0 % ntt) * VT;
    const size_t bh = (size_t)(lin0 / ntt);
    const int ndw = nst * SPT / 4;           // dwords per row (SPT is 4 or 8)
    for (int e = tid; e < D * ndw; e += 256) {
      const int c = e / ndw, i = e % ndw;
      *reinterpret_cast<uint32_t*>(scales + (bh * D + c) * (Np / NB) + t0 / NB + 4 * i) =
          *reinterpret_cast<const uint32_t*>(&sst[c * ST_ROW + 4 * i]);
    }
    nst = 0;                                 // sst is written again only after the next tile's barriers
  };
  auto step = [&](int lin, uint4 (&raw)[LPT]) {
    __syncthreads();                         // every thread is done with the previous tile in LDS
#pragma unroll
    for (int k = 0; k < LPT; ++k) {
      const int i = tid + 256 * k;
      *reinterpret_cast<uint4*>(&tile[i / UPR][(i % UPR) * 8]) = raw[k];
    }
    __syncthreads();
    if (lin + 2 < last) load(lin + 2, raw);  // two tiles in flight while this one is quantized
    const int t0 = (lin % ntt) * VT;
    const size_t bh = (size_t)(lin / ntt);
#pragma unroll
    for (int bb = 0; bb < BPT; ++bb) {
      const int blk = part * BPT + bb;         // token block inside the tile
      if (t0 + blk * NB >= Np) break;          // the last tile may end at Np (a multiple of 128)
      float x[CPT][NB];
      float am[CPT];
#pragma unroll
      for (int k = 0; k < CPT; ++k) am[k] = 0.0f;
#pragma unroll
      for (int j = 0; j < NB; ++j) {
        const int r = blk * NB + j;
        const bool in = t0 + r < N;
        if constexpr (CPT == 2) {
          const uint32_t two = *reinterpret_cast<const uint32_t*>(&tile[r][c0]);
          x[0][j] = in ? widen<BF16>((uint16_t)(two & 0xFFFFu)) : 0.0f;
          x[1][j] = in ? widen<BF16>((uint16_t)(two >> 16)) : 0.0f;
        } else {
          x[0][j] = in ? widen<BF16>(tile[r][c0]) : 0.0f;
        }
#pragma unroll
        for (int k = 0; k < CPT; ++k) am[k] = __builtin_fmaxf(am[k], __builtin_fabsf(x[k][j]));
      }
#pragma unroll
      for (int k = 0; k < CPT; ++k) {
        uint32_t sbyte;
        if (FMT == kFmtMX) {
          const int e = e8m0_exponent(am[k]);
          sbyte = (uint32_t)(e + 127);
#pragma unroll
          for (int j = 0; j < NB; ++j) x[k][j] = __builtin_ldexpf(x[k][j], -e);
        } else {
          sbyte = e4m3_encode(am[k] / 6.0f);
          const float s = e4m3_decode(sbyte);
          const float r = (s == 0.0f) ? 0.0f : 1.0f / s;
#pragma unroll
          for (int j = 0; j < NB; ++j) x[k][j] = (s == 0.0f) ? 0.0f : x[k][j] * r;
        }
        uint32_t wd[NB / 8];
#pragma unroll
        for (int q = 0; q < NB / 8; ++q) {
          wd[q] = 0;
#pragma unroll
          for (int i = 0; i < 4; ++i) wd[q] |= cvt_fp4x2(x[k][8 * q + 2 * i], x[k][8 * q + 2 * i + 1]) << (8 * i);
        }
        const int c = c0 + k;
        uint8_t* dst = codes + (bh * D + c) * (Np / 2) + (t0 + blk * NB) / 2;
        if (NB == 32) *reinterpret_cast<uint4*>(dst) = make_uint4(wd[0], wd[1], wd[2], wd[3]);
        else *reinterpret_cast<uint2*>(dst) = make_uint2(wd[0], wd[1]);
        sst[c * ST_ROW + nst * SPT + blk] = (uint8_t)sbyte;
      }
    }
    ++nst;
    if (nst == ST_TILES || lin + 1 >= last || (lin + 1) / ntt != lin / ntt) flush(lin);
  };
  for (int lin = first; lin < last; lin += 2) {
    step(lin, ra);
    if (lin + 1 < last) step(lin + 1, rb);
  }
}

// ---------------------------------------------------------------------------
// Host-side launchers (called by the C ABI in sage_abi.hip).
// ---------------------------------------------------------------------------
int kmean_chunks(int N) { return (N + KM_CHUNK - 1) / KM_CHUNK; }

template <int D, bool BF16>
static hipError_t launch_kmean_t(const void* k, double* part, float* mu, int BH, int N, hipStream_t st) {
  const int nchunk = kmean_chunks(N);
  hipLaunchKernelGGL((kmean_partial_kernel<D, BF16>), dim3(nchunk, BH), dim3(KM_THREADS), 0, st,
                     (const uint16_t*)k, part, N, nchunk);
  hipLaunchKernelGGL((kmean_final_kernel<D>), dim3(BH), dim3(256), 0, st, (const double*)part, mu, N, nchunk);
  return hipGetLastError();
}

hipError_t launch_kmean(const void* k, double* part, float* mu, int BH, int N, int D, bool bf16, hipStream_t st) {
  if (D == 128) return bf16 ? launch_kmean_t<128, true>(k, part, mu, BH, N, st) : launch_kmean_t<128, false>(k, part, mu, BH, N, st);
  return bf16 ? launch_kmean_t<64, true>(k, part, mu, BH, N, st) : launch_kmean_t<64, false>(k, part, mu, BH, N, st);
}

template <int D, bool BF16, int FMT, bool IS_K>
static hipError_t launch_rows_t(const void* x, const float* mu, int mshift, int nmb, void* codes, void* scales, int BH,
                                int N, int Nout, hipStream_t st) {
  const long long units = (long long)BH * N * (D / 8);
  constexpr int U = rows_units<IS_K>();
  long long blocks = (units + 256 * U - 1) / (256 * U);
  if (blocks > 65536) blocks = 65536;
  hipLaunchKernelGGL((quant_rows_kernel<D, BF16, FMT, IS_K>), dim3((unsigned)blocks), dim3(256), 0, st,
                     (const uint16_t*)x, mu, mshift, nmb, (uint8_t*)codes, (uint8_t*)scales, N, Nout, units);
  if (IS_K && Nout > N) {
    hipLaunchKernelGGL((k_tail_kernel<D, FMT>), dim3(1, BH), dim3(256), 0, st, (uint8_t*)codes, (uint8_t*)scales, N, Nout);
  }
  return hipGetLastError();
}

template <int D, int FMT, bool IS_K>
static hipError_t launch_rows_d(const void* x, const float* mu, int mshift, int nmb, void* codes, void* scales, int BH,
                                int N, int Nout, bool bf16, hipStream_t st) {
  return bf16 ? launch_rows_t<D, true, FMT, IS_K>(x, mu, mshift, nmb, codes, scales, BH, N, Nout, st)
              : launch_rows_t<D, false, FMT, IS_K>(x, mu, mshift, nmb, codes, scales, BH, N, Nout, st);
}

// mu: role K one mean per head (or null); role Q with smoothing one per QB-row block (or null).
hipError_t launch_quant_rows(const void* x, const float* mu, void* codes, void* scales, int BH, int N, int Nout, int D,
                             int fmt, bool is_k, bool bf16, hipStream_t st) {
  const int mshift = is_k ? 30 : 7, nmb = is_k ? 1 : (N + QB - 1) / QB;
  static_assert(QB == (1 << 7), "query smoothing blocks are 128 rows");
#define SAGE_ROWS(DD, FF)                                                                                   \
  return is_k ? launch_rows_d<DD, FF, true>(x, mu, mshift, nmb, codes, scales, BH, N, Nout, bf16, st)      \
              : launch_rows_d<DD, FF, false>(x, mu, mshift, nmb, codes, scales, BH, N, Nout, bf16, st)
  if (D == 128) { if (fmt == kFmtMX) { SAGE_ROWS(128, kFmtMX); } else { SAGE_ROWS(128, kFmtNV16); } }
  else { if (fmt == kFmtMX) { SAGE_ROWS(64, kFmtMX); } else { SAGE_ROWS(64, kFmtNV16); } }
#undef SAGE_ROWS
}

int qmean_blocks(int N) { return (N + QB - 1) / QB; }

hipError_t launch_qmean(const void* q, float* qbar, int BH, int N, int D, bool bf16, hipStream_t st) {
  const dim3 grid((unsigned)qmean_blocks(N), (unsigned)BH);
#define SAGE_QM(DD, BB) hipLaunchKernelGGL((qmean_kernel<DD, BB>), grid, dim3(KM_THREADS), 0, st, (const uint16_t*)q, \
                                           qbar, N, qmean_blocks(N))
  if (D == 128) { if (bf16) { SAGE_QM(128, true); } else { SAGE_QM(128, false); } }
  else { if (bf16) { SAGE_QM(64, true); } else { SAGE_QM(64, false); } }
#undef SAGE_QM
  return hipGetLastError();
}

// bias [BH, nqb, Np] fp32; Np is a multiple of 128
hipError_t launch_qk_bias(const void* k, const float* mu, const float* qbar, float* bias, int BH, int N, int Np, int D,
                          bool bf16, hipStream_t st) {
  const dim3 grid((unsigned)((Np + QB_THREADS - 1) / QB_THREADS), (unsigned)BH);
  const int nqb = qmean_blocks(N);
#define SAGE_QB(DD, BB) hipLaunchKernelGGL((qk_bias_kernel<DD, BB>), grid, dim3(QB_THREADS), 0, st, (const uint16_t*)k, \
                                           mu, qbar, bias, N, Np, nqb)
  if (D == 128) { if (bf16) { SAGE_QB(128, true); } else { SAGE_QB(128, false); } }
  else { if (bf16) { SAGE_QB(64, true); } else { SAGE_QB(64, false); } }
#undef SAGE_QB
  return hipGetLastError();
}

template <int D, bool BF16, int FMT>
static hipError_t launch_v_t(const void* v, void* codes, void* scales, int BH, int N, int Np, hipStream_t st) {
  // Np is a multiple of 128; a last half tile is handled by the tile-range guard
  const long long total = (long long)((Np + VT - 1) / VT) * BH;
  if (total == 0) return hipSuccess;
  if (total > INT_MAX) return hipErrorInvalidValue;
  int dev = 0, ncu = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e == hipSuccess) e = hipDeviceGetAttribute(&ncu, hipDeviceAttributeMultiprocessorCount, dev);
  if (e != hipSuccess) return e;
  const long long slots = (long long)(ncu > 0 ? ncu : 1) * V_WG_PER_CU;
  const int per_wg = (int)((total + slots - 1) / slots);
  const int grid = (int)((total + per_wg - 1) / per_wg);
  hipLaunchKernelGGL((quant_v_kernel<D, BF16, FMT>), dim3(grid), dim3(256), 0, st, (const uint16_t*)v,
                     (uint8_t*)codes, (uint8_t*)scales, N, Np, (int)total, per_wg);
  return hipGetLastError();
}

hipError_t launch_quant_v(const void* v, void* codes, void* scales, int BH, int N, int Np, int D, int fmt, bool bf16,
                          hipStream_t st) {
#define SAGE_V(DD, FF) return bf16 ? launch_v_t<DD, true, FF>(v, codes, scales, BH, N, Np, st) \
                                   : launch_v_t<DD, false, FF>(v, codes, scales, BH, N, Np, st)
  if (D == 128) { if (fmt == kFmtMX) { SAGE_V(128, kFmtMX); } else { SAGE_V(128, kFmtNV16); } }
  else { if (fmt == kFmtMX) { SAGE_V(64, kFmtMX); } else { SAGE_V(64, kFmtNV16); } }
#undef SAGE_V
}

}  // namespace sage
