/*
 * sage_mi355x.h -- C ABI of the MI355X (gfx950) microscaled-FP4 attention
 * forward of SageAttention3 (arXiv 2505.11594), and of the paper's 8-bit
 * attention (SageBwd: the forward of Algorithm 2, the backward of Algorithm 3).
 *
 * Every function returns an int status (sage_status).  Arguments are checked
 * on the host before any HIP call, so invalid calls fail without touching the
 * GPU.  All GPU work is enqueued asynchronously on the caller's stream; no
 * function synchronizes.  The library never frees caller memory.  Pointers
 * are device pointers unless stated otherwise; tensors are contiguous.
 *
 * Inputs Q, K, V are 16-bit (fp16 or bf16) [B, H, N, D] tensors: the problem
 * statement of Algorithm 1 (N x d matrices per head, FP16 inputs) with the
 * FlashAttention tiling of Sec. 2.  Inputs must be finite.
 */
#ifndef SAGE_MI355X_H
#define SAGE_MI355X_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  SAGE_OK = 0,
  SAGE_ERR_INVALID_ARG = 1,  /* null pointer, bad size, misalignment, unknown flag bits */
  SAGE_ERR_UNSUPPORTED = 2,  /* a valid request this build does not implement          */
  SAGE_ERR_HIP = 3,          /* a HIP runtime call or kernel launch failed              */
  SAGE_ERR_WORKSPACE = 4     /* caller workspace smaller than the size query returned   */
} sage_status;

/* ---- shapes ------------------------------------------------------------ */
/* Every entry point takes B, H, N, D with B, H, N >= 1 and D in {64, 128}. */
/* Np = N rounded up to 128.  Per head, Np * D <= 2^31 (N <= 2^24 at        */
/* D = 128, 2^25 at D = 64); in total, B * H * Np * D <= 2^40.  Larger      */
/* shapes return SAGE_ERR_INVALID_ARG.                                      */

/* ---- fmt bitfield ----------------------------------------------------- */
/* Microscaling format (Sec. 3.1, "Data type determination"):              */
#define SAGE_FMT_MXFP4      0x0u  /* E2M1 codes, 1x32 blocks, E8M0 scales (gfx950 native) */
#define SAGE_FMT_NV16_E4M3  0x1u  /* E2M1 codes, 1x16 blocks, E4M3 scales (paper's NVFP4)  */
#define SAGE_FMT_MASK       0x3u
/* Input dtype of q, k, v (and of o unless SAGE_OUT_F32):                  */
#define SAGE_IN_FP16        0x0u
#define SAGE_IN_BF16        0x4u
#define SAGE_OUT_F32        0x8u  /* o is fp32; otherwise o has the input dtype           */
#define SAGE_NO_SMOOTH_K    0x10u /* ablation: skip K <- K - mean(K) (Algorithm 1)         */
#define SAGE_SMOOTH_Q       0x20u /* smoothing Q (Algorithm 1), see below                   */
#define SAGE_BKV64          0x40u /* KV tile of 64 tokens instead of 128                   */
#define SAGE_BKV256         0x80u /* KV tile of 256 tokens (MXFP4 attention only)          */
#define SAGE_WG256          0x100u /* 256 queries per workgroup instead of 128: each K^/V^T
                                      tile is fetched from L2 once per 256 queries (about
                                      half the fetch traffic) for about 1% more time.  Only
                                      with SAGE_BKV256, non-causal, without SAGE_SMOOTH_Q;
                                      otherwise SAGE_ERR_UNSUPPORTED.  Same results.      */
#define SAGE_FMT_ALL_BITS   0x1FFu

/* ---- quantization roles ------------------------------------------------ */
#define SAGE_ROLE_Q 0
#define SAGE_ROLE_K 1
#define SAGE_ROLE_V 2

/*
 * Physical layout of quantized tensors (n = 32 for MXFP4, 16 for NV16;
 * Np = N rounded up to 128).  Codes are E2M1, two per byte, element 2i in the
 * low nibble.  Scale bytes are E8M0 (2^(b-127)) or E4M3FN.
 *   Q^  codes [B,H,N,D/2],  scales [B,H,N,D/n]      blocks along D
 *   K^  codes [B,H,Np,D/2], scales [B,H,Np,D/n]     blocks along D, of
 *       K' = fl32(K - mean_t K) (smoothing K), tokens permuted so the MFMA
 *       accumulator of S^T = K^ Q^T is laid out as the B operand of the P.V
 *       product (the CDNA form of the paper's "Permutation for K", Sec. 3.3):
 *       MXFP4: inside every 64-token group the token with offset
 *       o = 32h + 16t + 4g + r (h,t in {0,1}; g,r in {0..3}) is stored at
 *       position 32t + 8g + 4h + r;  NV16: inside every 32-token group the
 *       offset o = 16h + 4g + r goes to position 8g + 4h + r.
 *       Tokens >= N have zero codes.
 *   V^T codes [B,H,D,Np/2], scales [B,H,D,Np/n]     blocks along tokens, V
 *       transposed (Appendix, "Transposing V"), natural token order, tokens
 *       >= N are zero.
 * kmean: fp32 [B,H,D], the per-(b,h) channel mean of K over the N tokens,
 * computed as an exact fp64 sum divided by N and rounded to fp32.
 *
 * Smoothing Q (SAGE_SMOOTH_Q; Algorithm 1, "Smoothing Q of SageAttention2"):
 * Q is split into blocks of 128 consecutive rows (the last block holds the
 * rest); qbar[b,h,i,:] is the mean of block i (exact fp64 sum / rows, rounded
 * to fp32) and Q^ = phi(fl32(Q - qbar)).  The attention adds the GEMV
 * qbar_i . K'_k to every score of block i, with K' = fl32(K - kmean) (K when
 * SAGE_NO_SMOOTH_K) and the dot product evaluated as a chain of fp32 fused
 * multiply-adds in order of the channel: S = fl32(FP4MM + GEMV).
 */

/* Byte sizes of the codes and scales buffers for one role.  Host only. */
int sage_quant_sizes(int role, int B, int H, int N, int D, unsigned fmt,
                     size_t* codes_bytes, size_t* scales_bytes);

/* Workspace bytes sage_quant_fp4 needs for role K with smoothing (the
 * per-chunk partial sums of the mean); 0 otherwise.  Host only. */
size_t sage_quant_workspace_size(int role, int B, int H, int N, int D, unsigned fmt);

/*
 * sage_quant_fp4 -- microscaling FP4 quantization phi (Sec. 3.1, Eq.
 * microscaling): s = max|block|/6 stored as E8M0 (smallest power of two with
 * 6 s >= max, no clipping) or E4M3 (round to nearest even, saturating at
 * 448); codes = FP4 round-to-nearest-even of x/s, saturating at +-6, sign
 * kept.  Role K first subtracts the channel mean (smoothing K) and stores
 * the tokens permuted as described above; role V writes V^T.
 *  x        : 16-bit input [B,H,N,D], 16-byte aligned
 *  codes    : output, sage_quant_sizes() bytes, 16-byte aligned
 *  scales   : output, sage_quant_sizes() bytes, 4-byte aligned
 *  kmean    : role K: output fp32 [B,H,D] (required unless SAGE_NO_SMOOTH_K);
 *             role Q with SAGE_SMOOTH_Q: output qbar fp32 [B,H,ceil(N/128),D]
 *             (required); otherwise must be NULL
 *  workspace: role K with smoothing: device buffer of at least
 *             sage_quant_workspace_size() bytes, 8-byte aligned; else may be NULL
 * D must be 64 or 128; N >= 1.
 */
int sage_quant_fp4(const void* x, int role, int B, int H, int N, int D, unsigned fmt,
                   void* codes, void* scales, float* kmean,
                   void* workspace, size_t workspace_bytes, hipStream_t stream);

/* Workspace bytes for sage_attn_fp4_fwd_ws (quantized Q, K, V, the mean and
 * its partial sums; with SAGE_SMOOTH_Q also the query-block means and the
 * GEMV term, B*H*ceil(N/128)*(D + Np)*4 bytes; with NV16 also the exact f16
 * expansion of K^ and V^T the attention kernel reads, 4*B*H*Np*D bytes).
 * 0 for invalid arguments.  Host only. */
size_t sage_attn_fp4_workspace_size(int B, int H, int N, int D, unsigned fmt);

/*
 * sage_attn_fp4_fwd -- the microscaling FP4 attention forward, Algorithm 1
 * without smoothing Q: smoothing K, phi(Q), phi(K), phi(V) (V blocked along
 * tokens), S = FP4MM(Q^, K^) on block-scaled MFMA, online softmax over KV
 * tiles with the two-level quantization of P~ (Sec. 3.2: s_P1 = rowmax/R
 * per row and tile, then phi of P~/s_P1 with R = 6 for E8M0 scales and
 * 448*6 for E4M3 scales) and O += FP4MM(P^, V^) * s_P1; O = O / l.
 * MXFP4 runs on block-scaled FP4 MFMA; NV16 (whose E4M3 scales at 16-element
 * granularity the MFMA cannot take) expands K^ and V^T exactly to f16 once
 * per call, dequantizes Q^ and P^ exactly to f16 in registers, and runs on
 * f16 MFMA.
 * With SAGE_SMOOTH_Q the scores get the smoothing-Q GEMV term described above
 * (both formats).
 * KV tiles (the granularity of s_P1) are 128 keys; SAGE_BKV64 takes 64,
 * SAGE_BKV256 takes 256 (MXFP4 only: SAGE_ERR_UNSUPPORTED with NV16; both
 * tile flags together are SAGE_ERR_INVALID_ARG).  The tile changes only the
 * rounding of P (per-tile row maxima), not the quantized layouts.
 * Softmax scale is 1/sqrt(D).  causal = 1 keeps key j for query i iff j <= i.
 *  q, k, v  : 16-bit [B,H,N,D], 16-byte aligned
 *  o        : [B,H,N,D] fp32 (SAGE_OUT_F32) or input dtype, 16-byte aligned
 * The internal workspace comes from hipMallocAsync on `stream` and is freed
 * with hipFreeAsync on the same stream.
 */
int sage_attn_fp4_fwd(const void* q, const void* k, const void* v, void* o,
                      int B, int H, int N, int D, int causal, unsigned fmt, hipStream_t stream);

/* Same, with a caller-provided workspace of at least
 * sage_attn_fp4_workspace_size() bytes (256-byte aligned). */
int sage_attn_fp4_fwd_ws(const void* q, const void* k, const void* v, void* o,
                         int B, int H, int N, int D, int causal, unsigned fmt,
                         void* workspace, size_t workspace_bytes, hipStream_t stream);

/*
 * sage_attn_fp4_fwd_noalloc -- sage_attn_fp4_fwd for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc): the same arguments, kernels and results
 * as sage_attn_fp4_fwd, with no hipMalloc, hipFree or allocating library call.
 * Its workspace is a fixed scratch of SAGE_NOALLOC_SCRATCH_BYTES inside the
 * library, one per GPU, held until the process ends; shapes whose
 * sage_attn_fp4_workspace_size() exceeds it return SAGE_ERR_WORKSPACE before
 * any HIP call (256 MiB holds B = 1, H = 32, N = 32768, D = 128 in MXFP4;
 * NV16 also needs the f16 expansion of K^ and V^T, 4*B*H*Np*D bytes).
 * `stream` must belong to the current device (else SAGE_ERR_INVALID_ARG).
 * All calls on one GPU share its scratch: calls that overlap on one GPU
 * (other streams, other host threads) race and must be serialized by the
 * caller; consecutive calls on one stream are safe.
 */
#define SAGE_NOALLOC_SCRATCH_BYTES (256ull << 20)
int sage_attn_fp4_fwd_noalloc(const void* q, const void* k, const void* v, void* o,
                              int B, int H, int N, int D, int causal, unsigned fmt, hipStream_t stream);

/*
 * sage_attn_fp4_fwd_prequant -- the attention kernel alone, on tensors
 * produced by sage_quant_fp4 (layouts above).  kmean is not needed: the
 * smoothing is already inside K^ (softmax is invariant to it).  SAGE_SMOOTH_Q
 * returns SAGE_ERR_UNSUPPORTED (its GEMV term is not an input here).  With
 * NV16 the f16 expansion of K^ and V^T (4*B*H*Np*D bytes) comes from
 * hipMallocAsync on `stream` and is freed with hipFreeAsync on it.
 */
int sage_attn_fp4_fwd_prequant(const void* q_codes, const void* q_scales,
                               const void* k_codes, const void* k_scales,
                               const void* vt_codes, const void* vt_scales,
                               void* o, int B, int H, int N, int D, int causal,
                               unsigned fmt, hipStream_t stream);

/*
 * sage_attn_bf16_fwd -- comparison kernel with the same tiling on bf16 MFMA:
 * S = Q K^T in fp32, online softmax in fp32, P rounded to bf16, O += P V
 * (FlashAttention forward, Sec. 2).  q, k, v must be bf16 (flags must
 * contain SAGE_IN_BF16); o is fp32 with SAGE_OUT_F32, else bf16.  Only
 * SAGE_IN_BF16 and SAGE_OUT_F32 are accepted in flags (the kernel uses
 * 64-key tiles).  The V transpose goes to a hipMallocAsync workspace on
 * `stream`.
 */
int sage_attn_bf16_fwd(const void* q, const void* k, const void* v, void* o,
                       int B, int H, int N, int D, int causal, unsigned flags, hipStream_t stream);

/* ======================================================================== */
/* 8-bit attention forward of SageBwd (Algorithm 2, Sec. 4.1).             */
/*                                                                          */
/* Accepted flags: SAGE_IN_BF16, SAGE_OUT_F32, SAGE_NO_SMOOTH_K and        */
/* SAGE_BKV64; any other bit is SAGE_ERR_INVALID_ARG.  The KV tile, which   */
/* is also the block of psi(K) and psi(V), is bkv = 128 tokens, or 64 with  */
/* SAGE_BKV64 (the flag must then be passed to every call that touches the  */
/* quantized tensors).  D must be 64 or 128; N >= 1.                         */
/*                                                                          */
/* psi (Eq. psi): one fp32 scale s = max|X|/127 per block of rows -- 128    */
/* query rows for Q (the last block holds the rest), bkv rows for K and V -- */
/* and int8 codes round(x * fl32(1/s)), nearest, ties to even; an all-zero  */
/* block has s = 0 and zero codes.  K is first smoothed, K' = fl32(K -       */
/* kmean), unless SAGE_NO_SMOOTH_K.  Physical layout (Np = N rounded up to  */
/* 128):                                                                    */
/*   Q^  int8 [B,H,N,D],  s_Q fp32 [B,H,ceil(N/128)]                        */
/*   K^  int8 [B,H,Np,D], s_K fp32 [B,H,Np/bkv] (rows >= N are zero)        */
/*   V^T int8 [B,H,D,Np], s_V fp32 [B,H,Np/bkv] V transposed; inside every  */
/*       32-token group, position 16h + 4g + r (h in {0,1}; g, r in 0..3)   */
/*       holds token 8g + 4h + r (the order in which the int8 MFMA receives */
/*       P from the accumulator of S^T); tokens >= N are zero.              */
/* ======================================================================== */

/* Byte sizes of the codes and scales buffers for one role.  Host only. */
int sage_quant_int8_sizes(int role, int B, int H, int N, int D, unsigned flags,
                          size_t* codes_bytes, size_t* scales_bytes);

/*
 * sage_quant_int8 -- psi for one role (layouts above).
 *  x        : 16-bit input [B,H,N,D], 16-byte aligned
 *  codes    : output, sage_quant_int8_sizes() bytes, 16-byte aligned
 *  scales   : output fp32, sage_quant_int8_sizes() bytes, 4-byte aligned
 *  kmean    : role K with smoothing: output fp32 [B,H,D] (the exact mean,
 *             as for sage_quant_fp4); otherwise must be NULL
 *  workspace: role K with smoothing: at least
 *             sage_quant_workspace_size(SAGE_ROLE_K, B, H, N, D, 0) bytes,
 *             8-byte aligned; otherwise may be NULL
 */
int sage_quant_int8(const void* x, int role, int B, int H, int N, int D, unsigned flags,
                    void* codes, float* scales, float* kmean,
                    void* workspace, size_t workspace_bytes, hipStream_t stream);

/* Workspace bytes for sage_attn_int8_fwd_ws (quantized Q, K, V, their
 * scales, the mean and its partial sums); 0 for invalid arguments.  Host
 * only. */
size_t sage_attn_int8_workspace_size(int B, int H, int N, int D, unsigned flags);

/*
 * sage_attn_int8_fwd -- Algorithm 2: smoothing K, psi(Q), psi(K), psi(V),
 * S = MM(Q^, K^) s_Q s_K on int8 MFMA (exact int32 products), online softmax
 * over bkv-key tiles with the running max m, per-token quantization of P~
 * reusing the maxima (s_P = rowmax_tile(P~)/127, P^ = rint(P~/s_P)),
 * O = diag(e^{m_old - m_new}) O + MM(P^, V^) s_P s_V on int8 MFMA, O = O/l.
 * Softmax scale 1/sqrt(D); causal = 1 keeps key j for query i iff j <= i.
 *  q, k, v : 16-bit [B,H,N,D], 16-byte aligned
 *  o       : [B,H,N,D] fp32 (SAGE_OUT_F32) or input dtype, 16-byte aligned
 *  lse     : fp32 [B,H,N] or NULL: L = m + log(l), the natural-log
 *            log-sum-exp of the scaled scores S/sqrt(D) of each query row
 *            (the value the backward pass of Algorithm 3 consumes)
 * The internal workspace comes from hipMallocAsync on `stream` and is freed
 * with hipFreeAsync on the same stream.
 */
int sage_attn_int8_fwd(const void* q, const void* k, const void* v, void* o, float* lse,
                       int B, int H, int N, int D, int causal, unsigned flags, hipStream_t stream);

/* Same, with a caller-provided workspace of at least
 * sage_attn_int8_workspace_size() bytes (256-byte aligned). */
int sage_attn_int8_fwd_ws(const void* q, const void* k, const void* v, void* o, float* lse,
                          int B, int H, int N, int D, int causal, unsigned flags,
                          void* workspace, size_t workspace_bytes, hipStream_t stream);

/* The 8-bit attention kernel alone, on tensors produced by sage_quant_int8
 * (layouts above; kmean is not needed, the smoothing is inside K^).  flags:
 * SAGE_OUT_F32, SAGE_IN_BF16 (the dtype of a 16-bit o) and SAGE_BKV64 (as
 * given to sage_quant_int8). */
int sage_attn_int8_fwd_prequant(const void* q_codes, const float* q_scales,
                                const void* k_codes, const float* k_scales,
                                const void* vt_codes, const float* vt_scales,
                                void* o, float* lse, int B, int H, int N, int D, int causal,
                                unsigned flags, hipStream_t stream);

/*
 * sage_attn_int8_bwd -- the backward pass of the 8-bit attention (Algorithm
 * 3): D = rowsum(dO o O); per KV block j and query block i (128 x 128):
 * S = MM(Q^, K^) s_Q s_K, P = exp(S/sqrt(D) - L), psi(P), psi(dO) (per 128
 * rows), dV_j += MM(P^T, dO^) s_P s_dO, dP = MM(dO, V^T) in the 16-bit input
 * type with fp32 accumulation, dS = P o (dP - D), psi(dS), dQ_i +=
 * MM(dS^, K^) s_dS s_K / sqrt(D) + rowsum(dS) K_m / sqrt(D) (the smoothing
 * of K), dK_j += MM(dS^T, Q^) s_dS s_Q / sqrt(D).  Q^, K^ and K_m are
 * recomputed exactly as the forward computes them (psi blocks of 128 rows).
 *  q, k, v, dout: 16-bit [B,H,N,D] (dO has the input dtype), 16-byte aligned
 *  o    : the forward's output, fp32 [B,H,N,D], 16-byte aligned
 *  lse  : the forward's L, fp32 [B,H,N], 4-byte aligned
 *  dq, dk, dv: outputs, fp32 [B,H,N,D], 16-byte aligned
 * flags: SAGE_IN_BF16, SAGE_NO_SMOOTH_K (as given to the forward); SAGE_OUT_F32
 * is accepted and changes nothing (gradients are fp32); SAGE_BKV64 returns
 * SAGE_ERR_UNSUPPORTED (the backward's KV blocks are 128 keys).  The
 * internal workspace (sage_attn_int8_bwd_workspace_size bytes) comes from
 * hipMallocAsync on `stream`.
 */
int sage_attn_int8_bwd(const void* q, const void* k, const void* v, const float* o, const float* lse,
                       const void* dout, float* dq, float* dk, float* dv,
                       int B, int H, int N, int D, int causal, unsigned flags, hipStream_t stream);

/* Recommended workspace bytes for sage_attn_int8_bwd_ws (the size
 * sage_attn_int8_bwd allocates); 0 for invalid or unsupported arguments.
 * Beyond the minimum it holds the stored dS^ state of up to B*H heads
 * (sage_attn_int8_bwd_min_workspace_size explains it), capped at 64 GiB of
 * that state: about N^2 + 4 N^2 / 128 bytes per head.  Host only. */
size_t sage_attn_int8_bwd_workspace_size(int B, int H, int N, int D, unsigned flags);

/* Smallest workspace sage_attn_int8_bwd_ws accepts; 0 for invalid or
 * unsupported arguments.  Host only.  With it the dQ kernel recomputes S, dP
 * and dS; every head whose stored dS^ state (its codes, s_dS per block pair
 * and per-pair row sums of dS, which the dK kernel writes) also fits lets the
 * dQ kernel read them back instead, heads processed in groups of that many.
 * The result does not depend on the workspace size beyond rounding order of
 * the row-sum term of the smoothing of K. */
size_t sage_attn_int8_bwd_min_workspace_size(int B, int H, int N, int D, unsigned flags);

/* Same as sage_attn_int8_bwd, with a caller-provided workspace of at least
 * sage_attn_int8_bwd_min_workspace_size() bytes (256-byte aligned). */
int sage_attn_int8_bwd_ws(const void* q, const void* k, const void* v, const float* o, const float* lse,
                          const void* dout, float* dq, float* dk, float* dv,
                          int B, int H, int N, int D, int causal, unsigned flags,
                          void* workspace, size_t workspace_bytes, hipStream_t stream);

/* Human-readable status name; never NULL. */
const char* sage_status_string(int status);

/* Library version string. */
const char* sage_version(void);

#ifdef __cplusplus
}
#endif
#endif /* SAGE_MI355X_H */
