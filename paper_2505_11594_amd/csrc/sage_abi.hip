// C ABI of the gfx950 microscaled-FP4 attention library.  Argument checks run
// on the host before any HIP call; kernels are enqueued on the caller's stream.
#include <algorithm>
#include <cmath>
#include <cstdint>
#include <cstring>
#include <mutex>

#include "sage_common.h"
#include "sage_mi355x.h"

namespace sage {
hipError_t launch_kmean(const void* k, double* part, float* mu, int BH, int N, int D, bool bf16, hipStream_t st);
int kmean_chunks(int N);
hipError_t launch_quant_rows(const void* x, const float* mu, void* codes, void* scales, int BH, int N, int Nout, int D,
                             int fmt, bool is_k, bool bf16, hipStream_t st);
hipError_t launch_quant_v(const void* v, void* codes, void* scales, int BH, int N, int Np, int D, int fmt, bool bf16,
                          hipStream_t st);
hipError_t launch_qmean(const void* q, float* qbar, int BH, int N, int D, bool bf16, hipStream_t st);
int qmean_blocks(int N);
hipError_t launch_qk_bias(const void* k, const float* mu, const float* qbar, float* bias, int BH, int N, int Np, int D,
                          bool bf16, hipStream_t st);
hipError_t launch_attn_fp4_mx(const void* qc, const void* qs, const void* kc, const void* ks, const void* vc,
                              const void* vs, const float* qkb, void* o, int BH, int N, int Np, int D, int bkv,
                              bool causal, int out, float c2, float log6, bool wg256, hipStream_t st);
hipError_t launch_attn_nv16(const void* qc, const void* qs, const void* kc, const void* ks, const void* vc,
                            const void* vs, void* kv16, const float* qkb, void* o, int BH, int N, int Np, int D,
                            int bkv, bool causal, int out, float c2, float logR, hipStream_t st);
size_t nv16_expand_bytes(int BH, int Np, int D);
hipError_t launch_attn_bf16(const void* q, const void* k, const void* vt, void* o, int BH, int N, int Np, int D,
                            bool causal, bool out_f32, float c2, hipStream_t st);
hipError_t launch_transpose_v_bf16(const void* v, void* vt, int BH, int N, int Np, int D, hipStream_t st);
hipError_t launch_quant_i8(const void* x, const float* mu, void* codes, float* scales, int BH, int N, int Nout,
                           int D, int R, int role, bool bf16, hipStream_t st);
hipError_t launch_attn_int8(const void* qc, const float* qs, const void* kc, const float* ks, const void* vc,
                            const float* vs, void* o, float* lse, int BH, int N, int Np, int D, int bkv, bool causal,
                            int out, float c2, float log127, hipStream_t st);
hipError_t launch_i8_bwd_prep(const void* dout, const float* o, const float* lse, float* drow, float* lb, int BH,
                              int N, int Np, int D, bool bf16, hipStream_t st);
hipError_t launch_attn_int8_bwd(const void* qc, const float* qs, const void* qt, const void* kc, const float* ks,
                                const void* kt, const void* v, const void* dout, const void* gt, const float* gs,
                                const float* drow, const float* lb, const float* kmean, float* dq, float* dk, float* dv,
                                void* ds_state, int G, int BH, int N, int Np, int D, bool causal, bool bf16, float c2,
                                float rsd, hipStream_t st);
size_t i8_bwd_ds_bytes_per_head(int N);
}  // namespace sage

// the scratch of sage_attn_fp4_fwd_noalloc (see the no-allocation entry point below)
__device__ __align__(256) uint8_t sage_noalloc_scratch[SAGE_NOALLOC_SCRATCH_BYTES];

namespace {

constexpr long long kMaxElems = 1LL << 40;   // bound on B*H*N*D (keeps every offset in 64-bit range)

inline bool aligned(const void* p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) & (a - 1)) == 0; }
inline int fmt_of(unsigned f) { return (int)(f & SAGE_FMT_MASK); }
inline int blk_of(unsigned f) { return fmt_of(f) == SAGE_FMT_MXFP4 ? 32 : 16; }
inline int pad128(int N) { return (N + 127) / 128 * 128; }
inline size_t up256(size_t x) { return (x + 255) & ~(size_t)255; }

int check_shape(int B, int H, int N, int D, unsigned fmt) {
  if (B <= 0 || H <= 0 || N <= 0) return SAGE_ERR_INVALID_ARG;
  if (D != 64 && D != 128) return SAGE_ERR_INVALID_ARG;
  if (fmt & ~SAGE_FMT_ALL_BITS) return SAGE_ERR_INVALID_ARG;
  if ((fmt & SAGE_BKV64) && (fmt & SAGE_BKV256)) return SAGE_ERR_INVALID_ARG;
  const int f = fmt_of(fmt);
  if (f != SAGE_FMT_MXFP4 && f != SAGE_FMT_NV16_E4M3) return SAGE_ERR_INVALID_ARG;
  if ((long long)B * H > (1LL << 30)) return SAGE_ERR_INVALID_ARG;
  if (N > (1 << 30) - 128) return SAGE_ERR_INVALID_ARG;
  // one head's tensors are indexed with 32-bit offsets (row * Np, key * D)
  if ((long long)pad128(N) * D > (1LL << 31)) return SAGE_ERR_INVALID_ARG;
  if ((long long)B * H * (long long)pad128(N) * D > kMaxElems) return SAGE_ERR_INVALID_ARG;
  return SAGE_OK;
}

// smoothing Q in the attention: both formats
inline bool smooth_q_supported(unsigned) { return true; }

void sizes(int role, int B, int H, int N, int D, unsigned fmt, size_t* cb, size_t* sb) {
  const size_t BH = (size_t)B * H;
  const size_t n = blk_of(fmt);
  const size_t rows = (role == SAGE_ROLE_K) ? (size_t)pad128(N) : (size_t)N;
  if (role == SAGE_ROLE_V) {
    const size_t Np = pad128(N);
    *cb = BH * D * Np / 2;
    *sb = BH * D * Np / n;
  } else {
    *cb = BH * rows * D / 2;
    *sb = BH * rows * D / n;
  }
}

size_t kmean_ws_bytes(int B, int H, int N, int D) {
  return (size_t)B * H * (size_t)sage::kmean_chunks(N) * D * sizeof(double);
}

struct AttnWs {
  size_t qc, qs, kc, ks, vc, vs, mu, part, qbar, bias, kv16, total;
};

AttnWs attn_ws_layout(int B, int H, int N, int D, unsigned fmt) {
  AttnWs w;
  size_t c, s, off = 0;
  sizes(SAGE_ROLE_Q, B, H, N, D, fmt, &c, &s);
  w.qc = off; off += up256(c); w.qs = off; off += up256(s);
  sizes(SAGE_ROLE_K, B, H, N, D, fmt, &c, &s);
  w.kc = off; off += up256(c); w.ks = off; off += up256(s);
  sizes(SAGE_ROLE_V, B, H, N, D, fmt, &c, &s);
  w.vc = off; off += up256(c); w.vs = off; off += up256(s);
  w.mu = off; off += up256((size_t)B * H * D * sizeof(float));
  w.part = off; off += up256(kmean_ws_bytes(B, H, N, D));
  const size_t nqb = (fmt & SAGE_SMOOTH_Q) ? (size_t)sage::qmean_blocks(N) : 0;
  w.qbar = off; off += up256((size_t)B * H * nqb * D * sizeof(float));
  w.bias = off; off += up256((size_t)B * H * nqb * pad128(N) * sizeof(float));
  // NV16: the exact f16 expansion of K^ and V^T that the attention kernel reads
  w.kv16 = off;
  if (fmt_of(fmt) == SAGE_FMT_NV16_E4M3) off += up256(sage::nv16_expand_bytes(B * H, pad128(N), D));
  w.total = off;
  return w;
}

inline int hip_status(hipError_t e) { return e == hipSuccess ? SAGE_OK : SAGE_ERR_HIP; }

int quant_impl(const void* x, int role, int B, int H, int N, int D, unsigned fmt, void* codes, void* scales,
               float* kmean, void* ws, hipStream_t st) {
  const bool bf16 = (fmt & SAGE_IN_BF16) != 0;
  const int BH = B * H, f = fmt_of(fmt);
  hipError_t e = hipSuccess;
  if (role == SAGE_ROLE_Q) {
    const bool smooth = (fmt & SAGE_SMOOTH_Q) != 0;     // kmean receives the block means
    if (smooth) {
      e = sage::launch_qmean(x, kmean, BH, N, D, bf16, st);
      if (e != hipSuccess) return SAGE_ERR_HIP;
    }
    e = sage::launch_quant_rows(x, smooth ? kmean : nullptr, codes, scales, BH, N, N, D, f, false, bf16, st);
  } else if (role == SAGE_ROLE_K) {
    const bool smooth = !(fmt & SAGE_NO_SMOOTH_K);
    if (smooth) {
      e = sage::launch_kmean(x, static_cast<double*>(ws), kmean, BH, N, D, bf16, st);
      if (e != hipSuccess) return SAGE_ERR_HIP;
    }
    e = sage::launch_quant_rows(x, smooth ? kmean : nullptr, codes, scales, BH, N, pad128(N), D, f, true, bf16, st);
  } else {
    e = sage::launch_quant_v(x, codes, scales, BH, N, pad128(N), D, f, bf16, st);
  }
  return hip_status(e);
}

int attn_args(const void* q, const void* k, const void* v, const void* o, int B, int H, int N, int D, int causal,
              unsigned fmt) {
  int rc = check_shape(B, H, N, D, fmt);
  if (rc != SAGE_OK) return rc;
  if ((fmt & SAGE_BKV256) && fmt_of(fmt) != SAGE_FMT_MXFP4) return SAGE_ERR_UNSUPPORTED;
  if ((fmt & SAGE_WG256) && (!(fmt & SAGE_BKV256) || causal || (fmt & SAGE_SMOOTH_Q))) return SAGE_ERR_UNSUPPORTED;
  if (!q || !k || !v || !o) return SAGE_ERR_INVALID_ARG;
  if (!aligned(q, 16) || !aligned(k, 16) || !aligned(v, 16) || !aligned(o, 16)) return SAGE_ERR_INVALID_ARG;
  if (causal != 0 && causal != 1) return SAGE_ERR_INVALID_ARG;
  return SAGE_OK;
}

inline float softmax_c2(int D) { return (float)(1.0 / (std::log(2.0) * std::sqrt((double)D))); }
inline float log2_of_6() { return (float)std::log2(6.0); }
inline float log2_of_2688() { return (float)std::log2(448.0 * 6.0); }
inline int out_kind(unsigned fmt) { return (fmt & SAGE_OUT_F32) ? 0 : ((fmt & SAGE_IN_BF16) ? 1 : 2); }

// kv16: for NV16, device memory of nv16_expand_bytes() for the f16 expansion of
// K^ and V^T, or null to take it from hipMallocAsync on st for this call.
int attn_prequant_impl(const void* qc, const void* qs, const void* kc, const void* ks, const void* vc, const void* vs,
                       void* kv16, const float* qkb, void* o, int B, int H, int N, int D, int causal, unsigned fmt,
                       hipStream_t st) {
  const int bkv = (fmt & SAGE_BKV64) ? 64 : ((fmt & SAGE_BKV256) ? 256 : 128);
  if (fmt_of(fmt) == SAGE_FMT_NV16_E4M3) {
    if (bkv == 256) return SAGE_ERR_UNSUPPORTED;
    void* own = nullptr;
    if (!kv16) {
      if (hipMallocAsync(&own, sage::nv16_expand_bytes(B * H, pad128(N), D), st) != hipSuccess) return SAGE_ERR_HIP;
      kv16 = own;
    }
    int rc = hip_status(sage::launch_attn_nv16(qc, qs, kc, ks, vc, vs, kv16, qkb, o, B * H, N, pad128(N), D, bkv,
                                               causal != 0, out_kind(fmt), softmax_c2(D), log2_of_2688(), st));
    if (own && hipFreeAsync(own, st) != hipSuccess && rc == SAGE_OK) rc = SAGE_ERR_HIP;
    return rc;
  }
  return hip_status(sage::launch_attn_fp4_mx(qc, qs, kc, ks, vc, vs, qkb, o, B * H, N, pad128(N), D, bkv,
                                             causal != 0, out_kind(fmt), softmax_c2(D), log2_of_6(),
                                             (fmt & SAGE_WG256) != 0, st));
}

int attn_ws_impl(const void* q, const void* k, const void* v, void* o, int B, int H, int N, int D, int causal,
                 unsigned fmt, void* ws, hipStream_t st) {
  const AttnWs w = attn_ws_layout(B, H, N, D, fmt);
  uint8_t* base = static_cast<uint8_t*>(ws);
  float* mu = reinterpret_cast<float*>(base + w.mu);
  const bool smooth_q = (fmt & SAGE_SMOOTH_Q) != 0, smooth_k = !(fmt & SAGE_NO_SMOOTH_K);
  float* qbar = smooth_q ? reinterpret_cast<float*>(base + w.qbar) : nullptr;
  float* bias = smooth_q ? reinterpret_cast<float*>(base + w.bias) : nullptr;
  int rc = quant_impl(q, SAGE_ROLE_Q, B, H, N, D, fmt, base + w.qc, base + w.qs, qbar, nullptr, st);
  if (rc == SAGE_OK) rc = quant_impl(k, SAGE_ROLE_K, B, H, N, D, fmt, base + w.kc, base + w.ks, mu, base + w.part, st);
  if (rc == SAGE_OK) rc = quant_impl(v, SAGE_ROLE_V, B, H, N, D, fmt, base + w.vc, base + w.vs, nullptr, nullptr, st);
  if (rc == SAGE_OK && smooth_q)   // GEMV(qbar_i, K'^T) of every query block, over K' = K - mean(K)
    rc = hip_status(sage::launch_qk_bias(k, smooth_k ? mu : nullptr, qbar, bias, B * H, N, pad128(N), D,
                                         (fmt & SAGE_IN_BF16) != 0, st));
  if (rc == SAGE_OK)
    rc = attn_prequant_impl(base + w.qc, base + w.qs, base + w.kc, base + w.ks, base + w.vc, base + w.vs, base + w.kv16,
                            bias, o, B, H, N, D, causal, fmt, st);
  return rc;
}

// ---- the no-allocation entry point -----------------------------------------
// sage_attn_fp4_fwd_noalloc runs attn_ws_impl on a fixed scratch: a file-scope
// device array, one copy per GPU, held until the process ends.  Host code never
// passes the array's name to a kernel (on the host it is a stand-in, not a
// device address): the address comes from hipGetSymbolAddress, once per
// device with that device current, and is kept per device.  Every call on a
// GPU shares that GPU's scratch, so calls that overlap on one GPU (two streams,
// two host threads) race.  Nothing in it needs to start at zero: every byte
// attn_ws_impl reads is written earlier in the same call.
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices];   // device address of sage_noalloc_scratch, per device

// ---- 8-bit attention (Algorithm 2) ----------------------------------------
constexpr unsigned kI8Flags = SAGE_IN_BF16 | SAGE_OUT_F32 | SAGE_NO_SMOOTH_K | SAGE_BKV64;
constexpr int kI8Bq = 128;
inline int i8_bkv(unsigned flags) { return (flags & SAGE_BKV64) ? 64 : 128; }   // KV tile = K, V scale block

int check_i8(int B, int H, int N, int D, unsigned flags) {
  if (flags & ~kI8Flags) return SAGE_ERR_INVALID_ARG;
  return check_shape(B, H, N, D, flags & (SAGE_IN_BF16 | SAGE_OUT_F32));
}

void sizes_i8(int role, int B, int H, int N, int D, unsigned flags, size_t* cb, size_t* sb) {
  const size_t BH = (size_t)B * H, Np = pad128(N);
  if (role == SAGE_ROLE_Q) {
    *cb = BH * N * D;
    *sb = BH * ((N + kI8Bq - 1) / kI8Bq) * sizeof(float);
  } else {
    *cb = BH * Np * D;
    *sb = BH * (Np / i8_bkv(flags)) * sizeof(float);
  }
}

struct I8Ws {
  size_t qc, qs, kc, ks, vc, vs, mu, part, total;
};

I8Ws i8_ws_layout(int B, int H, int N, int D, unsigned flags) {
  I8Ws w;
  size_t c, s, off = 0;
  sizes_i8(SAGE_ROLE_Q, B, H, N, D, flags, &c, &s);
  w.qc = off; off += up256(c); w.qs = off; off += up256(s);
  sizes_i8(SAGE_ROLE_K, B, H, N, D, flags, &c, &s);
  w.kc = off; off += up256(c); w.ks = off; off += up256(s);
  sizes_i8(SAGE_ROLE_V, B, H, N, D, flags, &c, &s);
  w.vc = off; off += up256(c); w.vs = off; off += up256(s);
  w.mu = off; off += up256((size_t)B * H * D * sizeof(float));
  w.part = off; off += up256(kmean_ws_bytes(B, H, N, D));
  w.total = off;
  return w;
}

int quant_i8_impl(const void* x, int role, int B, int H, int N, int D, unsigned flags, void* codes, float* scales,
                  float* kmean, void* ws, hipStream_t st) {
  const bool bf16 = (flags & SAGE_IN_BF16) != 0;
  const int BH = B * H;
  hipError_t e = hipSuccess;
  if (role == SAGE_ROLE_Q) {
    e = sage::launch_quant_i8(x, nullptr, codes, scales, BH, N, N, D, kI8Bq, 0, bf16, st);
  } else if (role == SAGE_ROLE_K) {
    const bool smooth = !(flags & SAGE_NO_SMOOTH_K);
    if (smooth) {
      e = sage::launch_kmean(x, static_cast<double*>(ws), kmean, BH, N, D, bf16, st);
      if (e != hipSuccess) return SAGE_ERR_HIP;
    }
    e = sage::launch_quant_i8(x, smooth ? kmean : nullptr, codes, scales, BH, N, pad128(N), D, i8_bkv(flags), 1,
                              bf16, st);
  } else {
    e = sage::launch_quant_i8(x, nullptr, codes, scales, BH, N, pad128(N), D, i8_bkv(flags), 2, bf16, st);
  }
  return hip_status(e);
}

inline float log2_of_127() { return (float)std::log2(127.0); }

int attn_i8_prequant_impl(const void* qc, const float* qs, const void* kc, const float* ks, const void* vc,
                          const float* vs, void* o, float* lse, int B, int H, int N, int D, int causal,
                          unsigned flags, hipStream_t st) {
  return hip_status(sage::launch_attn_int8(qc, qs, kc, ks, vc, vs, o, lse, B * H, N, pad128(N), D, i8_bkv(flags),
                                           causal != 0, out_kind(flags), softmax_c2(D), log2_of_127(), st));
}

int attn_i8_ws_impl(const void* q, const void* k, const void* v, void* o, float* lse, int B, int H, int N, int D,
                    int causal, unsigned flags, void* ws, hipStream_t st) {
  const I8Ws w = i8_ws_layout(B, H, N, D, flags);
  uint8_t* base = static_cast<uint8_t*>(ws);
  float* qs = reinterpret_cast<float*>(base + w.qs);
  float* ks = reinterpret_cast<float*>(base + w.ks);
  float* vs = reinterpret_cast<float*>(base + w.vs);
  float* mu = reinterpret_cast<float*>(base + w.mu);
  int rc = quant_i8_impl(q, SAGE_ROLE_Q, B, H, N, D, flags, base + w.qc, qs, nullptr, nullptr, st);
  if (rc == SAGE_OK) rc = quant_i8_impl(k, SAGE_ROLE_K, B, H, N, D, flags, base + w.kc, ks, mu, base + w.part, st);
  if (rc == SAGE_OK) rc = quant_i8_impl(v, SAGE_ROLE_V, B, H, N, D, flags, base + w.vc, vs, nullptr, nullptr, st);
  if (rc == SAGE_OK)
    rc = attn_i8_prequant_impl(base + w.qc, qs, base + w.kc, ks, base + w.vc, vs, o, lse, B, H, N, D, causal, flags,
                               st);
  return rc;
}

int attn_i8_args(const void* q, const void* k, const void* v, const void* o, const float* lse, int B, int H, int N,
                 int D, int causal, unsigned flags) {
  int rc = check_i8(B, H, N, D, flags);
  if (rc != SAGE_OK) return rc;
  if (!q || !k || !v || !o) return SAGE_ERR_INVALID_ARG;
  if (!aligned(q, 16) || !aligned(k, 16) || !aligned(v, 16) || !aligned(o, 16)) return SAGE_ERR_INVALID_ARG;
  if (lse && !aligned(lse, 4)) return SAGE_ERR_INVALID_ARG;
  if (causal != 0 && causal != 1) return SAGE_ERR_INVALID_ARG;
  return SAGE_OK;
}

// ---- 8-bit attention backward (Algorithm 3) -------------------------------
constexpr unsigned kI8BwdFlags = SAGE_IN_BF16 | SAGE_OUT_F32 | SAGE_NO_SMOOTH_K | SAGE_BKV64;

// Stored dS^ state of the backward (the dK kernel writes it, the dQ kernel
// reads it back instead of recomputing S, dP and dS) is capped at this many
// bytes in the recommended workspace: heads are processed in groups that fit.
constexpr size_t kI8BwdDsCap = size_t(64) << 30;

struct I8BwdWs {
  size_t qc, qs, qt, kc, ks, kt, mu, part, gt, gs, drow, lb, ds, total;   // total: without the dS^ state
};

I8BwdWs i8_bwd_ws_layout(int B, int H, int N, int D) {
  I8BwdWs w;
  const size_t BH = (size_t)B * H, Np = pad128(N), nb = Np / 128, off0 = 0;
  size_t off = off0;
  w.qc = off; off += up256(BH * N * D);
  w.qs = off; off += up256(BH * nb * sizeof(float));
  w.qt = off; off += up256(BH * D * Np);
  w.kc = off; off += up256(BH * Np * D);
  w.ks = off; off += up256(BH * nb * sizeof(float));
  w.kt = off; off += up256(BH * D * Np);
  w.mu = off; off += up256(BH * D * sizeof(float));
  w.part = off; off += up256(kmean_ws_bytes(B, H, N, D));
  w.gt = off; off += up256(BH * D * Np);
  w.gs = off; off += up256(BH * nb * sizeof(float));
  w.drow = off; off += up256(BH * Np * sizeof(float));
  w.lb = off; off += up256(BH * Np * sizeof(float));
  w.ds = off;
  w.total = off;
  return w;
}

// heads whose dS^ state fits in `bytes` of workspace (0: the dQ kernel recomputes dS^)
int i8_bwd_ds_heads(int B, int H, int N, int D, size_t bytes) {
  const I8BwdWs w = i8_bwd_ws_layout(B, H, N, D);
  if (bytes <= w.ds) return 0;
  const size_t fit = (bytes - w.ds) / sage::i8_bwd_ds_bytes_per_head(N);
  return (int)std::min<size_t>(fit, (size_t)B * H);
}

size_t i8_bwd_recommended_bytes(int B, int H, int N, int D) {
  const I8BwdWs w = i8_bwd_ws_layout(B, H, N, D);
  const size_t per = sage::i8_bwd_ds_bytes_per_head(N);
  const size_t heads = std::min<size_t>((size_t)B * H, kI8BwdDsCap / per);
  return w.ds + heads * per;
}

int attn_i8_bwd_ws_impl(const void* q, const void* k, const void* v, const float* o, const float* lse,
                        const void* dout, float* dq, float* dk, float* dv, int B, int H, int N, int D, int causal,
                        unsigned flags, void* ws, size_t ws_bytes, hipStream_t st) {
  const I8BwdWs w = i8_bwd_ws_layout(B, H, N, D);
  const int G = i8_bwd_ds_heads(B, H, N, D, ws_bytes);
  uint8_t* base = static_cast<uint8_t*>(ws);
  const bool bf16 = (flags & SAGE_IN_BF16) != 0, smooth = !(flags & SAGE_NO_SMOOTH_K);
  const int BH = B * H, Np = pad128(N);
  float* qs = reinterpret_cast<float*>(base + w.qs);
  float* ks = reinterpret_cast<float*>(base + w.ks);
  float* gs = reinterpret_cast<float*>(base + w.gs);
  float* mu = reinterpret_cast<float*>(base + w.mu);
  float* drow = reinterpret_cast<float*>(base + w.drow);
  float* lb = reinterpret_cast<float*>(base + w.lb);
  // psi of Q (row-major and transposed), K' (both), dO (transposed): blocks of 128 rows
  hipError_t e = sage::launch_quant_i8(q, nullptr, base + w.qc, qs, BH, N, N, D, 128, 0, bf16, st);
  if (e == hipSuccess) e = sage::launch_quant_i8(q, nullptr, base + w.qt, qs, BH, N, Np, D, 128, 2, bf16, st);
  if (e == hipSuccess && smooth) e = sage::launch_kmean(k, reinterpret_cast<double*>(base + w.part), mu, BH, N, D, bf16, st);
  const float* mup = smooth ? mu : nullptr;
  if (e == hipSuccess) e = sage::launch_quant_i8(k, mup, base + w.kc, ks, BH, N, Np, D, 128, 1, bf16, st);
  if (e == hipSuccess) e = sage::launch_quant_i8(k, mup, base + w.kt, ks, BH, N, Np, D, 128, 3, bf16, st);
  if (e == hipSuccess) e = sage::launch_quant_i8(dout, nullptr, base + w.gt, gs, BH, N, Np, D, 128, 2, bf16, st);
  if (e == hipSuccess) e = sage::launch_i8_bwd_prep(dout, o, lse, drow, lb, BH, N, Np, D, bf16, st);
  if (e == hipSuccess)
    e = sage::launch_attn_int8_bwd(base + w.qc, qs, base + w.qt, base + w.kc, ks, base + w.kt, v, dout, base + w.gt, gs,
                                   drow, lb, mup, dq, dk, dv, base + w.ds, G, BH, N, Np, D, causal != 0, bf16,
                                   softmax_c2(D), (float)(1.0 / std::sqrt((double)D)), st);
  return hip_status(e);
}

int attn_i8_bwd_args(const void* q, const void* k, const void* v, const float* o, const float* lse, const void* dout,
                     const float* dq, const float* dk, const float* dv, int B, int H, int N, int D, int causal,
                     unsigned flags) {
  if (flags & ~kI8BwdFlags) return SAGE_ERR_INVALID_ARG;
  int rc = check_shape(B, H, N, D, flags & SAGE_IN_BF16);
  if (rc != SAGE_OK) return rc;
  if (!q || !k || !v || !o || !lse || !dout || !dq || !dk || !dv) return SAGE_ERR_INVALID_ARG;
  for (const void* p : {q, k, v, (const void*)o, dout, (const void*)dq, (const void*)dk, (const void*)dv})
    if (!aligned(p, 16)) return SAGE_ERR_INVALID_ARG;
  if (!aligned(lse, 4)) return SAGE_ERR_INVALID_ARG;
  if (causal != 0 && causal != 1) return SAGE_ERR_INVALID_ARG;
  if (flags & SAGE_BKV64) return SAGE_ERR_UNSUPPORTED;     // the backward's KV blocks are 128 keys
  return SAGE_OK;
}

}  // namespace

extern "C" {

int sage_quant_sizes(int role, int B, int H, int N, int D, unsigned fmt, size_t* codes_bytes, size_t* scales_bytes) {
  if (!codes_bytes || !scales_bytes) return SAGE_ERR_INVALID_ARG;
  if (role != SAGE_ROLE_Q && role != SAGE_ROLE_K && role != SAGE_ROLE_V) return SAGE_ERR_INVALID_ARG;
  const int rc = check_shape(B, H, N, D, fmt);
  if (rc != SAGE_OK) return rc;
  sizes(role, B, H, N, D, fmt, codes_bytes, scales_bytes);
  return SAGE_OK;
}

size_t sage_quant_workspace_size(int role, int B, int H, int N, int D, unsigned fmt) {
  if (role != SAGE_ROLE_K || (fmt & SAGE_NO_SMOOTH_K) || check_shape(B, H, N, D, fmt) != SAGE_OK) return 0;
  return kmean_ws_bytes(B, H, N, D);
}

int sage_quant_fp4(const void* x, int role, int B, int H, int N, int D, unsigned fmt, void* codes, void* scales,
                   float* kmean, void* workspace, size_t workspace_bytes, hipStream_t stream) {
  if (role != SAGE_ROLE_Q && role != SAGE_ROLE_K && role != SAGE_ROLE_V) return SAGE_ERR_INVALID_ARG;
  int rc = check_shape(B, H, N, D, fmt);
  if (rc != SAGE_OK) return rc;
  if (!x || !codes || !scales) return SAGE_ERR_INVALID_ARG;
  if (!aligned(x, 16) || !aligned(codes, 16) || !aligned(scales, 4)) return SAGE_ERR_INVALID_ARG;
  const bool smooth = role == SAGE_ROLE_K && !(fmt & SAGE_NO_SMOOTH_K);
  const bool smooth_q = role == SAGE_ROLE_Q && (fmt & SAGE_SMOOTH_Q);
  if (smooth) {
    if (!kmean || !aligned(kmean, 4) || !workspace || !aligned(workspace, 8)) return SAGE_ERR_INVALID_ARG;
    if (workspace_bytes < kmean_ws_bytes(B, H, N, D)) return SAGE_ERR_WORKSPACE;
  } else if (smooth_q) {
    if (!kmean || !aligned(kmean, 4)) return SAGE_ERR_INVALID_ARG;
  } else if (kmean) {
    return SAGE_ERR_INVALID_ARG;
  }
  return quant_impl(x, role, B, H, N, D, fmt, codes, scales, kmean, workspace, stream);
}

size_t sage_attn_fp4_workspace_size(int B, int H, int N, int D, unsigned fmt) {
  if (check_shape(B, H, N, D, fmt) != SAGE_OK || !smooth_q_supported(fmt)) return 0;
  return attn_ws_layout(B, H, N, D, fmt).total;
}

int sage_attn_fp4_fwd_ws(const void* q, const void* k, const void* v, void* o, int B, int H, int N, int D, int causal,
                         unsigned fmt, void* workspace, size_t workspace_bytes, hipStream_t stream) {
  int rc = attn_args(q, k, v, o, B, H, N, D, causal, fmt);
  if (rc != SAGE_OK) return rc;
  if (!smooth_q_supported(fmt)) return SAGE_ERR_UNSUPPORTED;
  if (!workspace || !aligned(workspace, 256)) return SAGE_ERR_INVALID_ARG;
  if (workspace_bytes < attn_ws_layout(B, H, N, D, fmt).total) return SAGE_ERR_WORKSPACE;
  return attn_ws_impl(q, k, v, o, B, H, N, D, causal, fmt, workspace, stream);
}

int sage_attn_fp4_fwd(const void* q, const void* k, const void* v, void* o, int B, int H, int N, int D, int causal,
                      unsigned fmt, hipStream_t stream) {
  int rc = attn_args(q, k, v, o, B, H, N, D, causal, fmt);
  if (rc != SAGE_OK) return rc;
  if (!smooth_q_supported(fmt)) return SAGE_ERR_UNSUPPORTED;
  const size_t bytes = attn_ws_layout(B, H, N, D, fmt).total;
  void* ws = nullptr;
  if (hipMallocAsync(&ws, bytes, stream) != hipSuccess) return SAGE_ERR_HIP;
  rc = attn_ws_impl(q, k, v, o, B, H, N, D, causal, fmt, ws, stream);
  if (hipFreeAsync(ws, stream) != hipSuccess && rc == SAGE_OK) rc = SAGE_ERR_HIP;
  return rc;
}

int sage_attn_fp4_fwd_noalloc(const void* q, const void* k, const void* v, void* o, int B, int H, int N, int D,
                              int causal, unsigned fmt, hipStream_t stream) {
  int rc = attn_args(q, k, v, o, B, H, N, D, causal, fmt);
  if (rc != SAGE_OK) return rc;
  if (!smooth_q_supported(fmt)) return SAGE_ERR_UNSUPPORTED;
  if (attn_ws_layout(B, H, N, D, fmt).total > (size_t)SAGE_NOALLOC_SCRATCH_BYTES) return SAGE_ERR_WORKSPACE;
  int dev = -1;
  hipDevice_t sdev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0) return SAGE_ERR_HIP;
  if (hipStreamGetDevice(stream, &sdev) != hipSuccess) return SAGE_ERR_HIP;
  if (sdev != dev || dev >= kMaxDevices) return SAGE_ERR_INVALID_ARG;   // the stream must be on the current device
  void* ws = nullptr;
  {
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
      void* p = nullptr;
      if (hipGetSymbolAddress(&p, HIP_SYMBOL(sage_noalloc_scratch)) != hipSuccess || !p) return SAGE_ERR_HIP;
      g_scratch_ptr[dev] = p;
    }
    ws = g_scratch_ptr[dev];
  }
  return attn_ws_impl(q, k, v, o, B, H, N, D, causal, fmt, ws, stream);
}

int sage_attn_fp4_fwd_prequant(const void* q_codes, const void* q_scales, const void* k_codes, const void* k_scales,
                               const void* vt_codes, const void* vt_scales, void* o, int B, int H, int N, int D,
                               int causal, unsigned fmt, hipStream_t stream) {
  int rc = check_shape(B, H, N, D, fmt);
  if (rc != SAGE_OK) return rc;
  if (!q_codes || !q_scales || !k_codes || !k_scales || !vt_codes || !vt_scales || !o) return SAGE_ERR_INVALID_ARG;
  if (!aligned(q_codes, 16) || !aligned(k_codes, 16) || !aligned(vt_codes, 16) || !aligned(o, 16)) return SAGE_ERR_INVALID_ARG;
  if (!aligned(q_scales, 4) || !aligned(k_scales, 4) || !aligned(vt_scales, 4)) return SAGE_ERR_INVALID_ARG;
  if (causal != 0 && causal != 1) return SAGE_ERR_INVALID_ARG;
  if (fmt & SAGE_SMOOTH_Q) return SAGE_ERR_UNSUPPORTED;   // the GEMV bias is not an input of this entry point
  if ((fmt & SAGE_WG256) && (!(fmt & SAGE_BKV256) || fmt_of(fmt) != SAGE_FMT_MXFP4 || causal))
    return SAGE_ERR_UNSUPPORTED;
  return attn_prequant_impl(q_codes, q_scales, k_codes, k_scales, vt_codes, vt_scales, nullptr, nullptr, o, B, H, N, D,
                            causal, fmt, stream);
}

int sage_attn_bf16_fwd(const void* q, const void* k, const void* v, void* o, int B, int H, int N, int D, int causal,
                       unsigned flags, hipStream_t stream) {
  if (flags & ~(unsigned)(SAGE_IN_BF16 | SAGE_OUT_F32)) return SAGE_ERR_INVALID_ARG;
  if (!(flags & SAGE_IN_BF16)) return SAGE_ERR_INVALID_ARG;
  int rc = attn_args(q, k, v, o, B, H, N, D, causal, flags);
  if (rc != SAGE_OK) return rc;
  const int Np = pad128(N);
  const size_t bytes = (size_t)B * H * D * Np * 2;
  void* vt = nullptr;
  if (hipMallocAsync(&vt, bytes, stream) != hipSuccess) return SAGE_ERR_HIP;
  hipError_t e = sage::launch_transpose_v_bf16(v, vt, B * H, N, Np, D, stream);
  if (e == hipSuccess)
    e = sage::launch_attn_bf16(q, k, vt, o, B * H, N, Np, D, causal != 0, (flags & SAGE_OUT_F32) != 0, softmax_c2(D),
                               stream);
  rc = hip_status(e);
  if (hipFreeAsync(vt, stream) != hipSuccess && rc == SAGE_OK) rc = SAGE_ERR_HIP;
  return rc;
}

int sage_quant_int8_sizes(int role, int B, int H, int N, int D, unsigned flags, size_t* codes_bytes,
                          size_t* scales_bytes) {
  if (!codes_bytes || !scales_bytes) return SAGE_ERR_INVALID_ARG;
  if (role != SAGE_ROLE_Q && role != SAGE_ROLE_K && role != SAGE_ROLE_V) return SAGE_ERR_INVALID_ARG;
  const int rc = check_i8(B, H, N, D, flags);
  if (rc != SAGE_OK) return rc;
  sizes_i8(role, B, H, N, D, flags, codes_bytes, scales_bytes);
  return SAGE_OK;
}

int sage_quant_int8(const void* x, int role, int B, int H, int N, int D, unsigned flags, void* codes, float* scales,
                    float* kmean, void* workspace, size_t workspace_bytes, hipStream_t stream) {
  if (role != SAGE_ROLE_Q && role != SAGE_ROLE_K && role != SAGE_ROLE_V) return SAGE_ERR_INVALID_ARG;
  int rc = check_i8(B, H, N, D, flags);
  if (rc != SAGE_OK) return rc;
  if (!x || !codes || !scales) return SAGE_ERR_INVALID_ARG;
  if (!aligned(x, 16) || !aligned(codes, 16) || !aligned(scales, 4)) return SAGE_ERR_INVALID_ARG;
  const bool smooth = role == SAGE_ROLE_K && !(flags & SAGE_NO_SMOOTH_K);
  if (smooth) {
    if (!kmean || !aligned(kmean, 4) || !workspace || !aligned(workspace, 8)) return SAGE_ERR_INVALID_ARG;
    if (workspace_bytes < kmean_ws_bytes(B, H, N, D)) return SAGE_ERR_WORKSPACE;
  } else if (kmean) {
    return SAGE_ERR_INVALID_ARG;
  }
  return quant_i8_impl(x, role, B, H, N, D, flags, codes, scales, kmean, workspace, stream);
}

size_t sage_attn_int8_workspace_size(int B, int H, int N, int D, unsigned flags) {
  if (check_i8(B, H, N, D, flags) != SAGE_OK) return 0;
  return i8_ws_layout(B, H, N, D, flags).total;
}

int sage_attn_int8_fwd_ws(const void* q, const void* k, const void* v, void* o, float* lse, int B, int H, int N,
                          int D, int causal, unsigned flags, void* workspace, size_t workspace_bytes,
                          hipStream_t stream) {
  int rc = attn_i8_args(q, k, v, o, lse, B, H, N, D, causal, flags);
  if (rc != SAGE_OK) return rc;
  if (!workspace || !aligned(workspace, 256)) return SAGE_ERR_INVALID_ARG;
  if (workspace_bytes < i8_ws_layout(B, H, N, D, flags).total) return SAGE_ERR_WORKSPACE;
  return attn_i8_ws_impl(q, k, v, o, lse, B, H, N, D, causal, flags, workspace, stream);
}

int sage_attn_int8_fwd(const void* q, const void* k, const void* v, void* o, float* lse, int B, int H, int N, int D,
                       int causal, unsigned flags, hipStream_t stream) {
  int rc = attn_i8_args(q, k, v, o, lse, B, H, N, D, causal, flags);
  if (rc != SAGE_OK) return rc;
  const size_t bytes = i8_ws_layout(B, H, N, D, flags).total;
  void* ws = nullptr;
  if (hipMallocAsync(&ws, bytes, stream) != hipSuccess) return SAGE_ERR_HIP;
  rc = attn_i8_ws_impl(q, k, v, o, lse, B, H, N, D, causal, flags, ws, stream);
  if (hipFreeAsync(ws, stream) != hipSuccess && rc == SAGE_OK) rc = SAGE_ERR_HIP;
  return rc;
}

int sage_attn_int8_fwd_prequant(const void* q_codes, const float* q_scales, const void* k_codes,
                                const float* k_scales, const void* vt_codes, const float* vt_scales, void* o,
                                float* lse, int B, int H, int N, int D, int causal, unsigned flags,
                                hipStream_t stream) {
  int rc = check_i8(B, H, N, D, flags);
  if (rc != SAGE_OK) return rc;
  if (!q_codes || !q_scales || !k_codes || !k_scales || !vt_codes || !vt_scales || !o) return SAGE_ERR_INVALID_ARG;
  if (!aligned(q_codes, 16) || !aligned(k_codes, 16) || !aligned(vt_codes, 16) || !aligned(o, 16))
    return SAGE_ERR_INVALID_ARG;
  if (!aligned(q_scales, 4) || !aligned(k_scales, 4) || !aligned(vt_scales, 4)) return SAGE_ERR_INVALID_ARG;
  if (lse && !aligned(lse, 4)) return SAGE_ERR_INVALID_ARG;
  if (causal != 0 && causal != 1) return SAGE_ERR_INVALID_ARG;
  return attn_i8_prequant_impl(q_codes, q_scales, k_codes, k_scales, vt_codes, vt_scales, o, lse, B, H, N, D, causal,
                               flags, stream);
}

size_t sage_attn_int8_bwd_workspace_size(int B, int H, int N, int D, unsigned flags) {
  if ((flags & ~kI8BwdFlags) || (flags & SAGE_BKV64) || check_shape(B, H, N, D, flags & SAGE_IN_BF16) != SAGE_OK)
    return 0;
  return i8_bwd_recommended_bytes(B, H, N, D);
}

size_t sage_attn_int8_bwd_min_workspace_size(int B, int H, int N, int D, unsigned flags) {
  if ((flags & ~kI8BwdFlags) || (flags & SAGE_BKV64) || check_shape(B, H, N, D, flags & SAGE_IN_BF16) != SAGE_OK)
    return 0;
  return i8_bwd_ws_layout(B, H, N, D).total;
}

int sage_attn_int8_bwd_ws(const void* q, const void* k, const void* v, const float* o, const float* lse,
                          const void* dout, float* dq, float* dk, float* dv, int B, int H, int N, int D, int causal,
                          unsigned flags, void* workspace, size_t workspace_bytes, hipStream_t stream) {
  int rc = attn_i8_bwd_args(q, k, v, o, lse, dout, dq, dk, dv, B, H, N, D, causal, flags);
  if (rc != SAGE_OK) return rc;
  if (!workspace || !aligned(workspace, 256)) return SAGE_ERR_INVALID_ARG;
  if (workspace_bytes < i8_bwd_ws_layout(B, H, N, D).total) return SAGE_ERR_WORKSPACE;
  return attn_i8_bwd_ws_impl(q, k, v, o, lse, dout, dq, dk, dv, B, H, N, D, causal, flags, workspace, workspace_bytes,
                             stream);
}

int sage_attn_int8_bwd(const void* q, const void* k, const void* v, const float* o, const float* lse, const void* dout,
                       float* dq, float* dk, float* dv, int B, int H, int N, int D, int causal, unsigned flags,
                       hipStream_t stream) {
  int rc = attn_i8_bwd_args(q, k, v, o, lse, dout, dq, dk, dv, B, H, N, D, causal, flags);
  if (rc != SAGE_OK) return rc;
  const size_t bytes = i8_bwd_recommended_bytes(B, H, N, D);
  void* ws = nullptr;
  if (hipMallocAsync(&ws, bytes, stream) != hipSuccess) return SAGE_ERR_HIP;
  rc = attn_i8_bwd_ws_impl(q, k, v, o, lse, dout, dq, dk, dv, B, H, N, D, causal, flags, ws, bytes, stream);
  if (hipFreeAsync(ws, stream) != hipSuccess && rc == SAGE_OK) rc = SAGE_ERR_HIP;
  return rc;
}

const char* sage_status_string(int status) {
  switch (status) {
    case SAGE_OK: return "SAGE_OK";
    case SAGE_ERR_INVALID_ARG: return "SAGE_ERR_INVALID_ARG";
    case SAGE_ERR_UNSUPPORTED: return "SAGE_ERR_UNSUPPORTED";
    case SAGE_ERR_HIP: return "SAGE_ERR_HIP";
    case SAGE_ERR_WORKSPACE: return "SAGE_ERR_WORKSPACE";
    default: return "SAGE_ERR_UNKNOWN";
  }
}

const char* sage_version(void) { return "sage-mi355x 0.1 (gfx950)"; }

}  // extern "C"
