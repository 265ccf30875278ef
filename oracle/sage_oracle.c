/*
 * sage_oracle.c -- plain, slow CPU oracle for microscaled-FP4 attention
 * (SageAttention3 forward, arXiv 2505.11594).
 *
 * TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the
 * benchmark's CPU-baseline leg may load this library.  It shares no source
 * with the HIP path and the HIP path never calls it.
 *
 * What it follows (paper sections / equations):
 *   - FP4 microscaling quantization phi and dequantization phi^-1:
 *     Sec. 3.1, Eq. (microscaling): s = max|X_block| / 6, X^ = round_FP4(X / s).
 *   - FP4MM: the product of the two dequantized operands (Sec. 3.1, Eq. FP4MM),
 *     evaluated exactly and rounded once to fp32.
 *   - Data types NVFP4 (E2M1 codes, 1x16 blocks, E4M3 scales) and MXFP4
 *     (E2M1, 1x32 blocks, E8M0 scales): Sec. 3.1 "Data type determination".
 *   - Algorithm 1 (microscaling FP4 attention) without smoothing Q:
 *     smoothing K (preprocessing), FlashAttention tiling with online softmax,
 *     two-level quantization of P~ (Sec. 3.2, Eq. two-level), and the output
 *     update O = diag(e^{m_old-m_new}) O + FP4MM(P^, s_P2, V^, s_V) * s_P1.
 *   - Accuracy metrics (Appendix, "Accuracy metrics") are computed in Python.
 *
 * Readings of points the paper leaves open are listed next to the code that
 * takes them.  Floating-point steps the paper fixes to fp32 (P~, P~2, s_P1,
 * the softmax state) are done in fp32 with explicit roundings; everything
 * else that has an exact value (FP4MM, the smoothing mean) is computed exactly.
 *
 * Build: gcc -O2 -fPIC -shared -ffp-contract=off -fno-fast-math -pthread -lm
 *
 * Parity pins (tests without a GPU) cover: every E2M1 code and tie, the E4M3
 * table and the paper's value counts (35 / 127 / 8 / 280 / 1016), the E8M0
 * rule, FP4MM against brute force, the identity-quantizer attention against
 * textbook softmax attention, closed forms (Q = 0, one-hot scores),
 * key/value permutation invariance and the FP4 error bound vs exact attention.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#include <pthread.h>

#define ORC_FMT_MX 0     /* MXFP4: E2M1 codes, blocks of 32, E8M0 scales      */
#define ORC_FMT_NV16 1   /* NVFP4-style: E2M1 codes, blocks of 16, E4M3 scales */
#define ORC_FMT_NONE 2   /* identity quantizer (pins the attention machinery)  */

#define ORC_IN_FP16 0
#define ORC_IN_BF16 1

#define ORC_ROLE_Q 0
#define ORC_ROLE_K 1
#define ORC_ROLE_V 2

/* attention flags */
#define ORC_NO_SMOOTH_K 1u   /* ablation: skip K <- K - mean(K)                  */
#define ORC_DIRECT_P 2u      /* ablation: quantize P~ directly (no first level) */
#define ORC_R_LITERAL 4u     /* ablation: first-level constant 448*6 with E8M0  */
#define ORC_SMOOTH_Q 8u      /* smoothing Q (Algorithm 1): quantize Q_i - mean(Q_i)
                                over each block of B_q rows and add the GEMV
                                mean(Q_i) . K_j^T to S                          */
#define ORC_OCP_SCALE 16u    /* ablation (MX only): E8M0 block scales by the floor
                                rule 2^(floor(log2 amax) - 2) for Q, K, V and the
                                second level of P, values above 6 s clip to 6    */

/* ------------------------------------------------------------------------ */
/* 16-bit input widening (exact)                                             */
/* ------------------------------------------------------------------------ */
static float widen_fp16(uint16_t h) {
  int s = (h >> 15) & 1, e = (h >> 10) & 31, m = h & 1023;
  float v;
  if (e == 0) v = ldexpf((float)m, -24);
  else if (e == 31) v = m ? NAN : INFINITY;
  else v = ldexpf((float)(1024 + m), e - 25);
  return s ? -v : v;
}
static float widen_bf16(uint16_t b) {
  uint32_t u = (uint32_t)b << 16;
  float v;
  memcpy(&v, &u, 4);
  return v;
}
float orc_widen(uint16_t x, int in_dtype) {
  return in_dtype == ORC_IN_BF16 ? widen_bf16(x) : widen_fp16(x);
}

/* ------------------------------------------------------------------------ */
/* E2M1 (FP4) codec.  Codes 0..7 are {0, .5, 1, 1.5, 2, 3, 4, 6}; bit 3 is    */
/* the sign.  Rounding "FP4 rounding" (Sec. 3.1) is read as round to nearest, */
/* ties to the even mantissa bit (even code index), saturating at +-6; the    */
/* sign of the input is kept, so small negatives give 0x8 (-0).               */
/* ------------------------------------------------------------------------ */
static const float E2M1_VAL[8] = {0.0f, 0.5f, 1.0f, 1.5f, 2.0f, 3.0f, 4.0f, 6.0f};

uint8_t orc_e2m1_encode(float y) {
  uint8_t sign = signbit(y) ? 8 : 0;
  float a = fabsf(y);
  for (int i = 0; i < 7; ++i) {
    float mid = 0.5f * (E2M1_VAL[i] + E2M1_VAL[i + 1]); /* exact */
    if (a < mid) return sign | (uint8_t)i;
    if (a == mid) return sign | (uint8_t)((i & 1) ? i + 1 : i);
  }
  return sign | 7; /* a > 5 rounds to 6; a >= 6 saturates to 6 */
}
float orc_e2m1_decode(uint8_t c) {
  float v = E2M1_VAL[c & 7];
  return (c & 8) ? -v : v;
}

/* ------------------------------------------------------------------------ */
/* E4M3 (FN variant, bias 7, no infinities, 0x7F = NaN, max 448) codec.       */
/* Conversion of a scale to E4M3 (Sec. 3.2) is read as round to nearest even */
/* with saturation at 448.  Only non-negative inputs occur (scales).          */
/* ------------------------------------------------------------------------ */
float orc_e4m3_decode(uint8_t b) {
  int s = b >> 7, e = (b >> 3) & 15, m = b & 7;
  float v;
  if (e == 15 && m == 7) return NAN;
  if (e == 0) v = ldexpf((float)m, -9);          /* m/8 * 2^-6 */
  else v = ldexpf((float)(8 + m), e - 10);       /* (1+m/8) * 2^(e-7) */
  return s ? -v : v;
}
uint8_t orc_e4m3_encode(float s) {
  /* nearest of the 127 non-negative finite values, ties to even code */
  if (!(s > 0.0f)) return 0;
  if (s >= 448.0f) return 0x7E;
  int best = 0;
  for (int c = 1; c <= 0x7E; ++c) {
    float v = orc_e4m3_decode((uint8_t)c);
    if (v <= s) best = c; else break;          /* values increase with code */
  }
  if (best == 0x7E) return 0x7E;
  float lo = orc_e4m3_decode((uint8_t)best), hi = orc_e4m3_decode((uint8_t)(best + 1));
  double dl = (double)s - lo, dh = (double)hi - s; /* exact in fp64 */
  if (dl < dh) return (uint8_t)best;
  if (dh < dl) return (uint8_t)(best + 1);
  return (uint8_t)((best & 1) ? best + 1 : best);
}

/* ------------------------------------------------------------------------ */
/* E8M0 scale (MXFP4).  The paper gives s = max|X|/6 (Sec. 3.1); E8M0 holds   */
/* only powers of two.  Reading: the smallest power of two 2^e with           */
/* 6 * 2^e >= amax, so that the block max still maps to at most 6 and        */
/* nothing clips; amax = 0 gives e = -127.  e is clamped to [-127, 127] and   */
/* stored with bias 127 (0xFF, NaN, is never produced).                       */
/* ------------------------------------------------------------------------ */
int orc_e8m0_exponent(float amax) {
  if (!(amax > 0.0f)) return -127;
  int E;
  double m = frexp((double)amax, &E);           /* amax = m 2^E, m in [.5,1) */
  int e = (m <= 0.75) ? E - 3 : E - 2;
  if (e < -127) e = -127;
  if (e > 127) e = 127;
  return e;
}
float orc_e8m0_decode(uint8_t b) { return ldexpf(1.0f, (int)b - 127); }

/* The alternative E8M0 rule (ablation ORC_OCP_SCALE): 2^e with e =          */
/* floor(log2 amax) - 2, the exponent of amax less that of the largest FP4    */
/* value's binade (6 = 1.5 * 2^2).  Block values in (6, 8) 2^e exceed the FP4 */
/* range and saturate to 6; in exchange the scale is half the default one    */
/* for blocks whose max lies in (6, 8) 2^e.  amax = 0 gives -127.             */
int orc_e8m0_exponent_floor(float amax) {
  if (!(amax > 0.0f)) return -127;
  int E;
  frexp((double)amax, &E);                      /* amax in [2^(E-1), 2^E) */
  int e = (E - 1) - 2;
  if (e < -127) e = -127;
  if (e > 127) e = 127;
  return e;
}

/* ------------------------------------------------------------------------ */
/* phi on one block of n values (Sec. 3.1, Eq. microscaling).                */
/* codes: n bytes, one code per byte.  Returns the scale byte.               */
/*  MX:   e = E8M0 exponent of amax; code_k = E2M1(x_k * 2^-e) (exact scale). */
/*  NV16: s = E4M3(fl32(amax / 6)); s = 0 -> all codes 0; otherwise          */
/*        code_k = E2M1(fl32(x_k * fl32(1 / s))).  Division by s is read as    */
/*        multiplication by the fp32 reciprocal of the stored scale.          */
/* ------------------------------------------------------------------------ */
uint8_t orc_phi_block(const float* x, int n, int fmt, uint8_t* codes) {
  float amax = 0.0f;
  for (int k = 0; k < n; ++k) { float a = fabsf(x[k]); if (a > amax) amax = a; }
  if (fmt == ORC_FMT_MX) {
    int e = orc_e8m0_exponent(amax);
    for (int k = 0; k < n; ++k) codes[k] = orc_e2m1_encode(ldexpf(x[k], -e));
    return (uint8_t)(e + 127);
  } else {
    volatile float q = amax / 6.0f;
    uint8_t sb = orc_e4m3_encode(q);
    float s = orc_e4m3_decode(sb);
    if (s == 0.0f) { for (int k = 0; k < n; ++k) codes[k] = 0; return sb; }
    volatile float r = 1.0f / s;
    for (int k = 0; k < n; ++k) { volatile float y = x[k] * r; codes[k] = orc_e2m1_encode(y); }
    return sb;
  }
}
/* phi with the attention flags: ORC_OCP_SCALE selects the floor rule for MX */
uint8_t orc_phi_block_ex(const float* x, int n, int fmt, unsigned flags, uint8_t* codes) {
  if (fmt != ORC_FMT_MX || !(flags & ORC_OCP_SCALE)) return orc_phi_block(x, n, fmt, codes);
  float amax = 0.0f;
  for (int k = 0; k < n; ++k) { float a = fabsf(x[k]); if (a > amax) amax = a; }
  int e = orc_e8m0_exponent_floor(amax);
  for (int k = 0; k < n; ++k) codes[k] = orc_e2m1_encode(ldexpf(x[k], -e));
  return (uint8_t)(e + 127);
}
static float scale_value(uint8_t sb, int fmt) {
  return fmt == ORC_FMT_MX ? orc_e8m0_decode(sb) : orc_e4m3_decode(sb);
}
static int block_of(int fmt) { return fmt == ORC_FMT_MX ? 32 : 16; }

/* ------------------------------------------------------------------------ */
/* Smoothing K (Algorithm 1, preprocessing): mu[b,h,c] = mean over the N      */
/* tokens of K[b,h,:,c].  The sum is accumulated in fp64 with an error-free   */
/* transformation (TwoSum) so that its exactness is checked; mu is the fp64   */
/* quotient sum/N rounded to fp32.  Returns the number of (b,h,c) columns     */
/* whose fp64 sum was not exact (0 for every workload used here).            */
/* ------------------------------------------------------------------------ */
long orc_kmean(const uint16_t* k, int in_dtype, int B, int H, int N, int D, float* mu) {
  /* Returns the number of columns whose sum is not provably exact in every
     summation order: all values are integer multiples of 2^lsb, so any order
     is exact when sum |x| < 2^(53 + lsb).  The sequential sum itself is also
     checked with TwoSum. */
  long inexact = 0;
  for (long bh = 0; bh < (long)B * H; ++bh) {
    const uint16_t* kb = k + bh * (long)N * D;
    for (int c = 0; c < D; ++c) {
      double s = 0.0, err = 0.0, sabs = 0.0;
      int lsb = 1 << 30;
      for (int t = 0; t < N; ++t) {
        double a = (double)orc_widen(kb[(long)t * D + c], in_dtype);
        if (a != 0.0) {
          /* exponent of the lowest set bit of the fp32 value */
          float af = (float)a;
          uint32_t u;
          memcpy(&u, &af, 4);
          int be = (int)((u >> 23) & 255);
          uint32_t man = u & 0x7FFFFFu;
          if (be) man |= 0x800000u;
          int lb = (be ? be : 1) - 127 - 23 + __builtin_ctz(man);
          if (lb < lsb) lsb = lb;
        }
        sabs += fabs(a);
        double sn = s + a, bb = sn - s;
        err += (s - (sn - bb)) + (a - bb);
        s = sn;
      }
      if (err != 0.0 || (sabs > 0.0 && !(sabs < ldexp(1.0, 53 + lsb)))) inexact++;
      mu[bh * D + c] = (float)(s / (double)N);
    }
  }
  return inexact;
}

/* ------------------------------------------------------------------------ */
/* Quantize one tensor in the LOGICAL layout (one code per byte):             */
/*  Q:  codes [B,H,N,D],    scales [B,H,N,D/n]   (blocks along D)            */
/*  K:  K' = fl32(K - mu);  same layout as Q      (blocks along D)            */
/*  V:  codes [B,H,D,Np],   scales [B,H,D,Np/n]  (blocks along tokens; V is   */
/*      transposed, Np = N rounded up to n, tail tokens are zero)            */
/* Block axes are read as each GEMM's reduction dimension (Q, K along D; V   */
/* along tokens), which is what FP4MM needs (Appendix, "Transposing V").     */
/* mu: role K with smoothing -> output [B,H,D] (else may be NULL).           */
/* fmt NONE is not valid here.  Returns the kmean inexact count (role K).    */
/* ------------------------------------------------------------------------ */
long orc_quant(const uint16_t* x, int in_dtype, int role, int B, int H, int N, int D,
               int fmt, int smooth_k, uint8_t* codes, uint8_t* scales, float* mu) {
  int n = block_of(fmt);
  long inexact = 0;
  float* work = (float*)malloc(sizeof(float) * (size_t)(n > D ? n : D));
  if (role == ORC_ROLE_K && smooth_k) inexact = orc_kmean(x, in_dtype, B, H, N, D, mu);
  for (long bh = 0; bh < (long)B * H; ++bh) {
    const uint16_t* xb = x + bh * (long)N * D;
    if (role == ORC_ROLE_Q || role == ORC_ROLE_K) {
      for (int t = 0; t < N; ++t) {
        for (int c = 0; c < D; ++c) {
          float v = orc_widen(xb[(long)t * D + c], in_dtype);
          if (role == ORC_ROLE_K && smooth_k) { volatile float d = v - mu[bh * D + c]; v = d; }
          work[c] = v;
        }
        for (int blk = 0; blk < D / n; ++blk) {
          uint8_t* cp = codes + ((bh * N + t) * (long)D) + blk * n;
          scales[(bh * N + t) * (long)(D / n) + blk] = orc_phi_block(work + blk * n, n, fmt, cp);
        }
      }
    } else {
      long Np = ((long)N + n - 1) / n * n;
      for (int c = 0; c < D; ++c) {
        for (long t0 = 0; t0 < Np; t0 += n) {
          for (int k = 0; k < n; ++k) {
            long t = t0 + k;
            work[k] = t < N ? orc_widen(xb[t * D + c], in_dtype) : 0.0f;
          }
          uint8_t* cp = codes + (bh * D + c) * Np + t0;
          scales[(bh * D + c) * (Np / n) + t0 / n] = orc_phi_block(work, n, fmt, cp);
        }
      }
    }
  }
  free(work);
  return inexact;
}

/* ------------------------------------------------------------------------ */
/* Smoothing Q (Algorithm 1, first step of the loop over query blocks):      */
/* qbar_i = mean of the rows of block Q_i (B_q consecutive rows; the last    */
/* block holds the remaining rows).  The sum is accumulated in fp64, where   */
/* it is exact for 16-bit inputs and B_q <= 2^20 rows, and the quotient is   */
/* rounded once to fp32.  qbar: [nqb][D] for one head.                       */
/* ------------------------------------------------------------------------ */
static void qmean_head(const uint16_t* qh, int in_dtype, int N, int D, int bq, float* qbar) {
  const int nqb = (N + bq - 1) / bq;
  for (int b = 0; b < nqb; ++b) {
    const int r0 = b * bq, r1 = (r0 + bq < N) ? r0 + bq : N;
    for (int c = 0; c < D; ++c) {
      double s = 0.0;
      for (int t = r0; t < r1; ++t) s += (double)orc_widen(qh[(long)t * D + c], in_dtype);
      qbar[(long)b * D + c] = (float)(s / (double)(r1 - r0));
    }
  }
}

/* phi(Q_i - qbar_i) along D for every row (logical layout as orc_quant),    */
/* and qbar [B,H,ceil(N/bq),D].                                              */
void orc_quant_smooth_q(const uint16_t* q, int in_dtype, int B, int H, int N, int D, int bq, int fmt,
                        uint8_t* codes, uint8_t* scales, float* qbar) {
  const int n = block_of(fmt), nqb = (N + bq - 1) / bq;
  float* work = (float*)malloc(sizeof(float) * (size_t)D);
  for (long bh = 0; bh < (long)B * H; ++bh) {
    const uint16_t* qh = q + bh * (long)N * D;
    float* qm = qbar + bh * (long)nqb * D;
    qmean_head(qh, in_dtype, N, D, bq, qm);
    for (int t = 0; t < N; ++t) {
      for (int c = 0; c < D; ++c) {
        volatile float d = orc_widen(qh[(long)t * D + c], in_dtype) - qm[(long)(t / bq) * D + c];
        work[c] = d;
      }
      for (int blk = 0; blk < D / n; ++blk)
        scales[(bh * N + t) * (long)(D / n) + blk] =
            orc_phi_block(work + blk * n, n, fmt, codes + (bh * N + t) * (long)D + blk * n);
    }
  }
  free(work);
}

/* ------------------------------------------------------------------------ */
/* Exact sums.  FP4MM (Sec. 3.1) equals the matmul of the dequantized        */
/* operands.  With codes c (2c is an integer in [-12,12]) and scales s, a     */
/* block's contribution is (sum_k (2c_a)(2c_b)) * s_a s_b / 4 -- an integer   */
/* times a product of two scales, exact in fp64.  Block contributions are     */
/* added in fp64 with TwoSum so that any rounding is detected and counted.   */
/* ------------------------------------------------------------------------ */
typedef struct { double s, err; } xsum_t;
static void xsum_add(xsum_t* a, double v) {
  double sn = a->s + v, bb = sn - a->s;
  a->err += (a->s - (sn - bb)) + (v - bb);
  a->s = sn;
}

/* ------------------------------------------------------------------------ */
/* Per-head quantized operands.                                              */
/* ------------------------------------------------------------------------ */
typedef struct {
  int N, D, Np, n, fmt;
  int8_t* kc2;     /* [N][D]   2*code value of K^ (integer)     (fmt != NONE) */
  float* ks;       /* [N][D/n] scale value of K^                              */
  int8_t* vc2;     /* [D][Np]  2*code value of V^T                            */
  float* vs;       /* [D][Np/n]                                               */
  float* kf;       /* [N][D]   fp32 K' (fmt NONE, or smoothing Q: the GEMV)   */
  float* vf;       /* [N][D]   fp32 V  (fmt NONE)                             */
  double vabs_max; /* max |deq(V^)| (for the tie-tolerance bound)             */
} head_t;

typedef struct {
  const uint16_t *q, *k, *v;
  int in_dtype, B, H, N, D, causal, fmt, bkv, bq;
  unsigned flags;
  const int64_t* rows;
  int64_t nrows;
  float* out;        /* [nrows][D] */
  float* tie_tol;    /* [nrows] extra tolerance from tie-ambiguous P codes, or NULL */
  int64_t* counters; /* [4]: inexact S sums, inexact O sums, ambiguous P codes, skipped tiles */
  head_t* heads;     /* [B*H], only the ones used are filled */
  char* head_used;
  int64_t next;
  pthread_mutex_t mu;
  int64_t cnt[4];
} attn_job_t;

static void two_code(float v, int* c2) {
  /* 2 * decoded E2M1 value as an integer */
  *c2 = (int)(2.0f * v);
}

static void build_head(attn_job_t* J, long bh) {
  head_t* h = &J->heads[bh];
  int N = J->N, D = J->D, fmt = J->fmt;
  h->N = N; h->D = D; h->fmt = fmt;
  const uint16_t* kb = J->k + bh * (long)N * D;
  const uint16_t* vb = J->v + bh * (long)N * D;
  int smooth = !(J->flags & ORC_NO_SMOOTH_K);
  float* mu = (float*)calloc(D, sizeof(float));
  if (smooth) {
    /* same definition as orc_kmean, for this head only */
    orc_kmean(kb, J->in_dtype, 1, 1, N, D, mu);
  }
  if (fmt == ORC_FMT_NONE) {
    h->n = 1; h->Np = N;
    h->kf = (float*)malloc(sizeof(float) * (size_t)N * D);
    h->vf = (float*)malloc(sizeof(float) * (size_t)N * D);
    double vm = 0;
    for (long i = 0; i < (long)N * D; ++i) {
      float kv = orc_widen(kb[i], J->in_dtype);
      if (smooth) { volatile float d = kv - mu[i % D]; kv = d; }
      h->kf[i] = kv;
      h->vf[i] = orc_widen(vb[i], J->in_dtype);
      if (fabs(h->vf[i]) > vm) vm = fabs(h->vf[i]);
    }
    h->vabs_max = vm;
    free(mu);
    return;
  }
  int n = block_of(fmt);
  h->n = n;
  h->Np = (N + n - 1) / n * n;
  uint8_t* codes = (uint8_t*)malloc((size_t)N * D);
  uint8_t* sc = (uint8_t*)malloc((size_t)N * (D / n));
  /* K' along D */
  float* work = (float*)malloc(sizeof(float) * (size_t)(D > n ? D : n));
  h->kc2 = (int8_t*)malloc((size_t)N * D);
  h->ks = (float*)malloc(sizeof(float) * (size_t)N * (D / n));
  if (J->flags & ORC_SMOOTH_Q) h->kf = (float*)malloc(sizeof(float) * (size_t)N * D);
  for (int t = 0; t < N; ++t) {
    for (int c = 0; c < D; ++c) {
      float kv = orc_widen(kb[(long)t * D + c], J->in_dtype);
      if (smooth) { volatile float d = kv - mu[c]; kv = d; }
      work[c] = kv;
      if (h->kf) h->kf[(long)t * D + c] = kv;
    }
    for (int blk = 0; blk < D / n; ++blk) {
      uint8_t sb = orc_phi_block_ex(work + blk * n, n, fmt, J->flags, codes + (long)t * D + blk * n);
      h->ks[(long)t * (D / n) + blk] = scale_value(sb, fmt);
    }
    for (int c = 0; c < D; ++c) { int c2; two_code(orc_e2m1_decode(codes[(long)t * D + c]), &c2); h->kc2[(long)t * D + c] = (int8_t)c2; }
  }
  /* V^T along tokens */
  int Np = h->Np;
  h->vc2 = (int8_t*)malloc((size_t)D * Np);
  h->vs = (float*)malloc(sizeof(float) * (size_t)D * (Np / n));
  uint8_t cb[32];
  double vm = 0;
  for (int c = 0; c < D; ++c) {
    for (int t0 = 0; t0 < Np; t0 += n) {
      for (int kk = 0; kk < n; ++kk) {
        int t = t0 + kk;
        work[kk] = t < N ? orc_widen(vb[(long)t * D + c], J->in_dtype) : 0.0f;
      }
      uint8_t sb = orc_phi_block_ex(work, n, fmt, J->flags, cb);
      float s = scale_value(sb, fmt);
      h->vs[(long)c * (Np / n) + t0 / n] = s;
      for (int kk = 0; kk < n; ++kk) {
        int c2; float dv = orc_e2m1_decode(cb[kk]);
        two_code(dv, &c2);
        h->vc2[(long)c * Np + t0 + kk] = (int8_t)c2;
        double a = fabs((double)dv * s);
        if (a > vm) vm = a;
      }
    }
  }
  h->vabs_max = vm;
  free(work); free(codes); free(sc); free(mu);
}

static void free_head(head_t* h) {
  free(h->kc2); free(h->ks); free(h->vc2); free(h->vs); free(h->kf); free(h->vf);
  memset(h, 0, sizeof(*h));
}

/* correctly rounded (to fp32) exp2: the fp64 exp2 rounded once */
static float exp2_f32(float x) { return (float)exp2((double)x); }

/* ------------------------------------------------------------------------ */
/* One query row of Algorithm 1 (smoothing Q optional, flag ORC_SMOOTH_Q).   */
/*                                                                           */
/* Readings (the paper does not fix these):                                  */
/*  - smoothing Q: the block mean qbar_i is taken over the B_q rows of the   */
/*    row's query block; the GEMV(qbar_i, K_j^T) uses the unquantized K' of  */
/*    the smoothing-K step in fp32, as a chain of fp32 fused multiply-adds   */
/*    in order of d starting from 0, and is added to the fp32 FP4MM result:  */
/*    S = fl32(fl32(FP4MM) + GEMV).                                          */
/*  - softmax scale 1/sqrt(D) is applied and exp is taken base 2:            */
/*    P~_k = 2^{c2 (S_k - m)} with c2 = fl32(log2(e)/sqrt(D)).                */
/*  - running max m and tile max t are kept in the raw score domain S.        */
/*  - two-level (Sec. 3.2): s_P1 = rowmax(P~)/R, P~2 = P~ / s_P1.  Since      */
/*    rowmax(P~) = 2^{c2 (t - m)}, P~2_k = R 2^{c2 (S_k - t)}; it is computed  */
/*    in fp32 as exp2(fma(S_k, c2, fl32(log2 R - fl32(t c2)))).  R = 448*6    */
/*    for E4M3 scales; with E8M0 scales R = 6 (maps the tile row max onto    */
/*    the largest FP4 value; ORC_R_LITERAL keeps 448*6 as an ablation).       */
/*  - the second level is phi over each n-key block of P~2.  For MX the      */
/*    block's E8M0 exponent is the smallest e with 6 2^e >= blockmax(P~2),    */
/*    where blockmax(P~2) = 6 2^{c2 (bm - t)} (bm = block max of S) is read   */
/*    in the score domain: e = ceil(fl32(fl32(bm - t) c2)) (for R = 6), so    */
/*    the decision does not depend on the exp implementation.  Values that    */
/*    round above 6 2^e saturate to code 6 (E2M1 saturation).                */
/*  - l accumulates the unquantized P~ (Algorithm 1): the tile's            */
/*    rowsum(P~) is fl32(s_P1 * sum_k P~2_k) with a sequential fp32 sum.      */
/*  - O_new = fl32(fl32(alpha O) + fl32(FP4MM(P^2, V^) s_P1)),               */
/*    alpha = 2^{c2 (m_old - m_new)} (0 on the first visited tile).          */
/*  - the final O = fl32(O / l).                                             */
/*  - causal: key k is visible to query i iff k <= i; fully masked tiles are  */
/*    skipped; keys >= N are masked.                                         */
/* tie_tol: the bound on |O| change if any P code whose pre-rounding value   */
/* lies within TIE_REL of an E2M1 rounding boundary took the other            */
/* neighbouring code (both are valid results when exp is evaluated in fp32   */
/* to within a few ulp, which the paper leaves unspecified).                  */
/* ------------------------------------------------------------------------ */
#define TIE_REL (1.0 / 1048576.0) /* 8 ulp of fp32 */

static int e2m1_tie_step(float y, double* step) {
  /* y >= 0: if y lies within TIE_REL (relative) of a rounding midpoint,
     return 1 and the distance between the two neighbouring grid values */
  for (int i = 0; i < 7; ++i) {
    double mid = 0.5 * ((double)E2M1_VAL[i] + E2M1_VAL[i + 1]);
    if (fabs((double)y - mid) <= TIE_REL * mid) { *step = (double)E2M1_VAL[i + 1] - E2M1_VAL[i]; return 1; }
  }
  return 0;
}

static int e4m3_tie(float s) {
  /* s > 0: within TIE_REL of a midpoint between two adjacent E4M3 values */
  if (!(s > 0.0f) || s >= 448.0f) return 0;
  for (int c = 0; c < 0x7E; ++c) {
    double lo = orc_e4m3_decode((uint8_t)c), hi = orc_e4m3_decode((uint8_t)(c + 1));
    double mid = 0.5 * (lo + hi);
    if (fabs((double)s - mid) <= TIE_REL * mid) return 1;
    if (hi > s * 2.0) break;
  }
  return 0;
}

/* ------------------------------------------------------------------------ */
/* orc_p_tile: online-softmax update and two-level quantization of P~ for    */
/* one query row and one KV tile (Algorithm 1; Sec. 3.2, Eq. two-level).     */
/*  S[bkv]  : the tile's scores (fp32), -inf for masked keys; at least one    */
/*            key is unmasked                                                */
/*  m_old   : running max (raw score domain), -inf before the first tile      */
/* outputs:                                                                  */
/*  m_new, alpha = 2^{c2 (m_old - m_new)} (0 on the first tile),              */
/*  s1 = rowmax(P~)/R (1 for direct quantization), rowsum = rowsum(P~),       */
/*  p2[bkv] = P~2 (fp32), codes[bkv] (one per byte), sbytes[bkv/n] scale      */
/*  bytes, tie_step[bkv] (0, or the grid step if the code is tie-ambiguous),  */
/*  scale_tie[bkv/n] (NV16: the block scale is tie-ambiguous).               */
/* fmt NONE: codes/sbytes untouched, p2 holds P~2 unquantized.               */
/* ------------------------------------------------------------------------ */
int orc_p_tile(const float* S, int bkv, float m_old, int D, int fmt, unsigned flags,
               float* m_new_out, float* alpha_out, float* s1_out, float* rowsum_out,
               float* p2, uint8_t* codes, uint8_t* sbytes, double* tie_step, uint8_t* scale_tie) {
  const int n = (fmt == ORC_FMT_NONE) ? 1 : block_of(fmt);
  const int direct = (flags & ORC_DIRECT_P) != 0;
  const float c2 = (float)(1.0 / (log(2.0) * sqrt((double)D)));
  const float R = (fmt == ORC_FMT_NV16 || (flags & ORC_R_LITERAL)) ? 448.0f * 6.0f : 6.0f;
  const float logR = (float)log2((double)R);

  float t = -INFINITY;
  for (int kk = 0; kk < bkv; ++kk) if (S[kk] > t) t = S[kk];
  if (t == -INFINITY) return -1;
  const float m_new = m_old > t ? m_old : t;
  volatile float tc = t * c2;
  volatile float mc_new = m_new * c2;
  float alpha = 0.0f;
  if (m_old != -INFINITY) { volatile float mc_old = m_old * c2; volatile float d = mc_old - mc_new; alpha = exp2_f32(d); }

  /* first level: s_P1 = rowmax(P~)/R with rowmax(P~) = 2^{c2 (t - m_new)} */
  float s1;
  volatile float bias;
  if (direct) { s1 = 1.0f; bias = -mc_new; }
  else {
    volatile float dt = tc - mc_new;
    float rho = exp2_f32(dt);
    volatile float q = rho / R;
    s1 = q;
    bias = logR - tc;
  }
  /* P~2 = R 2^{c2 (S - t)}, and the unquantized row sum */
  float psum = 0.0f;
  for (int kk = 0; kk < bkv; ++kk) {
    p2[kk] = (S[kk] == -INFINITY) ? 0.0f : exp2_f32(fmaf(S[kk], c2, bias));
    psum += p2[kk];
    if (tie_step) tie_step[kk] = 0.0;
  }
  volatile float rs = s1 * psum;
  *m_new_out = m_new; *alpha_out = alpha; *s1_out = s1; *rowsum_out = rs;
  if (fmt == ORC_FMT_NONE) return 0;

  /* second level: (s_P2, P^2) = phi(P~2) over n-key blocks */
  for (int b0 = 0; b0 < bkv; b0 += n) {
    const int blk = b0 / n;
    if (scale_tie) scale_tie[blk] = 0;
    if (fmt == ORC_FMT_MX) {
      float bm = -INFINITY;
      for (int kk = b0; kk < b0 + n; ++kk) if (S[kk] > bm) bm = S[kk];
      int e;
      if (bm == -INFINITY) e = -126;
      else if (direct || (flags & (ORC_R_LITERAL | ORC_OCP_SCALE))) {
        float am = 0.0f;
        for (int kk = b0; kk < b0 + n; ++kk) if (p2[kk] > am) am = p2[kk];
        e = (flags & ORC_OCP_SCALE) ? orc_e8m0_exponent_floor(am) : orc_e8m0_exponent(am);
      } else {
        /* blockmax(P~2) = 6 2^{c2 (bm - t)}; smallest e with 6 2^e >= it */
        volatile float dd = bm - t;
        volatile float d2 = dd * c2;
        e = (int)ceilf(d2);
      }
      /* P scales stay in the normal fp32 range: blocks below 2^-126 of the
         tile max hold values that vanish next to it */
      if (e < -126) e = -126;
      sbytes[blk] = (uint8_t)(e + 127);
      for (int kk = b0; kk < b0 + n; ++kk) {
        float y = ldexpf(p2[kk], -e);
        codes[kk] = orc_e2m1_encode(y);
        double step;
        if (tie_step && e2m1_tie_step(y, &step)) tie_step[kk] = step;
      }
    } else {
      uint8_t sb = orc_phi_block(p2 + b0, n, fmt, codes + b0);
      sbytes[blk] = sb;
      float scale = orc_e4m3_decode(sb);
      float am = 0.0f;
      for (int kk = b0; kk < b0 + n; ++kk) if (p2[kk] > am) am = p2[kk];
      volatile float q6 = am / 6.0f;
      if (scale_tie && e4m3_tie(q6)) scale_tie[blk] = 1;
      if (tie_step && scale > 0.0f) {
        volatile float r = 1.0f / scale;
        for (int kk = b0; kk < b0 + n; ++kk) {
          volatile float y = p2[kk] * r;
          double step;
          if (e2m1_tie_step(y, &step)) tie_step[kk] = step;
        }
      }
    }
  }
  return 0;
}

/* ------------------------------------------------------------------------ */
/* One query row of Algorithm 1 (smoothing Q optional, flag ORC_SMOOTH_Q).   */
/*                                                                           */
/* Readings (the paper does not fix these):                                  */
/*  - smoothing Q: the block mean qbar_i is taken over the B_q rows of the   */
/*    row's query block; the GEMV(qbar_i, K_j^T) uses the unquantized K' of  */
/*    the smoothing-K step in fp32, as a chain of fp32 fused multiply-adds   */
/*    in order of d starting from 0, and is added to the fp32 FP4MM result:  */
/*    S = fl32(fl32(FP4MM) + GEMV).                                          */
/*  - softmax scale 1/sqrt(D) is applied and exp is taken base 2:            */
/*    P~_k = 2^{c2 (S_k - m)} with c2 = fl32(log2(e)/sqrt(D)).                */
/*  - running max m and tile max t are kept in the raw score domain S.        */
/*  - two-level (Sec. 3.2): s_P1 = rowmax(P~)/R, P~2 = P~ / s_P1.  Since      */
/*    rowmax(P~) = 2^{c2 (t - m)}, P~2_k = R 2^{c2 (S_k - t)}; it is computed  */
/*    in fp32 as exp2(fma(S_k, c2, fl32(log2 R - fl32(t c2)))).  R = 448*6    */
/*    for E4M3 scales; with E8M0 scales R = 6 (maps the tile row max onto    */
/*    the largest FP4 value; ORC_R_LITERAL keeps 448*6 as an ablation).       */
/*  - the second level is phi over each n-key block of P~2.  For MX the      */
/*    block's E8M0 exponent is the smallest e with 6 2^e >= blockmax(P~2),    */
/*    where blockmax(P~2) = 6 2^{c2 (bm - t)} (bm = block max of S) is read   */
/*    in the score domain: e = ceil(fl32(fl32(bm - t) c2)) (for R = 6), so    */
/*    the decision does not depend on the exp implementation.  Values that    */
/*    round above 6 2^e saturate to code 6 (E2M1 saturation).                */
/*  - l accumulates the unquantized P~ (Algorithm 1): the tile's            */
/*    rowsum(P~) is fl32(s_P1 * sum_k P~2_k) with a sequential fp32 sum.      */
/*  - O_new = fl32(fl32(alpha O) + fl32(FP4MM(P^2, V^) s_P1)),               */
/*    alpha = 2^{c2 (m_old - m_new)} (0 on the first visited tile).          */
/*  - the final O = fl32(O / l).                                             */
/*  - causal: key k is visible to query i iff k <= i; fully masked tiles are  */
/*    skipped; keys >= N are masked.                                         */
/* tie_tol: the bound on |O| change if any P code whose pre-rounding value   */
/* lies within TIE_REL of an E2M1 rounding boundary took the other            */
/* neighbouring code (both are valid results when exp is evaluated in fp32   */
/* to within a few ulp, which the paper leaves unspecified), or if an NV16   */
/* block scale is itself tie-ambiguous.                                      */
/* ------------------------------------------------------------------------ */
static void attn_row(attn_job_t* J, long bh, int i, float* out, float* tol_out, int64_t* cnt) {
  head_t* h = &J->heads[bh];
  const int N = J->N, D = J->D, fmt = J->fmt, bkv = J->bkv;
  const int n = (fmt == ORC_FMT_NONE) ? 1 : block_of(fmt);
  const int nblk = bkv / n;
  const uint16_t* qb = J->q + (bh * (long)N + i) * D;

  /* phi(Q_i) along D; with smoothing Q, phi(Q_i - qbar_i) (Algorithm 1) */
  float* qf = (float*)malloc(sizeof(float) * D);
  int* qc2 = (int*)malloc(sizeof(int) * D);
  float* qs = (float*)malloc(sizeof(float) * (D / n + 1));
  float* qbar = NULL;
  for (int c = 0; c < D; ++c) qf[c] = orc_widen(qb[c], J->in_dtype);
  if (J->flags & ORC_SMOOTH_Q) {
    const int bq = J->bq, blk0 = (i / bq) * bq;
    const int rows = (blk0 + bq < N) ? bq : N - blk0;
    qbar = (float*)malloc(sizeof(float) * D);
    /* the mean of this row's block only (same definition as qmean_head) */
    qmean_head(J->q + (bh * (long)N + blk0) * D, J->in_dtype, rows, D, bq, qbar);
    for (int c = 0; c < D; ++c) { volatile float d = qf[c] - qbar[c]; qf[c] = d; }
  }
  if (fmt != ORC_FMT_NONE) {
    uint8_t cb[32];
    for (int blk = 0; blk < D / n; ++blk) {
      uint8_t sb = orc_phi_block_ex(qf + blk * n, n, fmt, J->flags, cb);
      qs[blk] = scale_value(sb, fmt);
      for (int kk = 0; kk < n; ++kk) { int c2; two_code(orc_e2m1_decode(cb[kk]), &c2); qc2[blk * n + kk] = c2; }
    }
  }

  float* S = (float*)malloc(sizeof(float) * bkv);
  float* P2 = (float*)malloc(sizeof(float) * bkv);
  uint8_t* pc = (uint8_t*)malloc((size_t)bkv);
  uint8_t* psb = (uint8_t*)malloc((size_t)nblk + 1);
  uint8_t* stie = (uint8_t*)malloc((size_t)nblk + 1);
  double* tstep = (double*)malloc(sizeof(double) * bkv);
  float* O = (float*)calloc(D, sizeof(float));
  double tol = 0.0;
  float m = -INFINITY, l = 0.0f;

  const int ntiles = (N + bkv - 1) / bkv;
  for (int j = 0; j < ntiles; ++j) {
    const int k0 = j * bkv;
    if (J->causal && k0 > i) { cnt[3]++; continue; }
    /* S_ij = FP4MM(Q^_i, s_Q, K^_j, s_K): exact, rounded once to fp32 */
    int nvalid = 0;
    for (int kk = 0; kk < bkv; ++kk) {
      const int k = k0 + kk;
      if (k >= N || (J->causal && k > i)) { S[kk] = -INFINITY; continue; }
      nvalid++;
      xsum_t acc = {0.0, 0.0};
      if (fmt == ORC_FMT_NONE) {
        for (int c = 0; c < D; ++c) xsum_add(&acc, (double)qf[c] * (double)h->kf[(long)k * D + c]);
      } else {
        for (int blk = 0; blk < D / n; ++blk) {
          long isum = 0;
          for (int c = blk * n; c < blk * n + n; ++c) isum += (long)qc2[c] * h->kc2[(long)k * D + c];
          xsum_add(&acc, (double)isum * ((double)qs[blk] * (double)h->ks[(long)k * (D / n) + blk]) * 0.25);
        }
      }
      if (acc.err != 0.0) cnt[0]++;
      S[kk] = (float)acc.s;
      if (qbar) {
        /* + GEMV(qbar_i, K_j^T) in fp32: a chain of fused multiply-adds in
           order of d from 0, then added to the fp32 score */
        float g = 0.0f;
        for (int c = 0; c < D; ++c) g = fmaf(qbar[c], h->kf[(long)k * D + c], g);
        volatile float sb = S[kk] + g;
        S[kk] = sb;
      }
    }
    if (nvalid == 0) { cnt[3]++; continue; }

    float m_new, alpha, s1, rowsum;
    orc_p_tile(S, bkv, m, D, fmt, J->flags, &m_new, &alpha, &s1, &rowsum, P2, pc, psb,
               tol_out ? tstep : NULL, tol_out ? stie : NULL);
    volatile float al = alpha * l;
    l = al + rowsum;
    tol = (double)alpha * tol;

    if (fmt != ORC_FMT_NONE && tol_out) {
      for (int blk = 0; blk < nblk; ++blk) {
        double sc = fmt == ORC_FMT_MX ? orc_e8m0_decode(psb[blk]) : orc_e4m3_decode(psb[blk]);
        if (fmt == ORC_FMT_NV16 && stie[blk]) {
          cnt[2]++;
          double sc2 = orc_e4m3_decode(psb[blk] < 0x7E ? psb[blk] + 1 : psb[blk]);
          tol += (double)n * 2.0 * sc2 * (double)s1 * h->vabs_max;
          continue;
        }
        for (int kk = blk * n; kk < blk * n + n; ++kk)
          if (tstep[kk] != 0.0) { cnt[2]++; tol += tstep[kk] * sc * (double)s1 * h->vabs_max; }
      }
    }

    /* O = diag(alpha) O + FP4MM(P^2, s_P2, V^, s_V) * s_P1 */
    for (int c = 0; c < D; ++c) {
      xsum_t acc = {0.0, 0.0};
      if (fmt == ORC_FMT_NONE) {
        for (int kk = 0; kk < bkv && k0 + kk < N; ++kk)
          xsum_add(&acc, (double)P2[kk] * (double)h->vf[(long)(k0 + kk) * D + c]);
      } else {
        for (int blk = 0; blk < nblk; ++blk) {
          const int b0 = blk * n;
          if (k0 + b0 >= h->Np) break;                 /* past the zero-padded tail */
          long isum = 0;
          for (int kk = b0; kk < b0 + n; ++kk) {
            int p2i;
            two_code(orc_e2m1_decode(pc[kk]), &p2i);
            isum += (long)p2i * h->vc2[(long)c * h->Np + k0 + kk];
          }
          double ps = scale_value(psb[blk], fmt);
          xsum_add(&acc, (double)isum * (ps * (double)h->vs[(long)c * (h->Np / n) + (k0 + b0) / n]) * 0.25);
        }
      }
      if (acc.err != 0.0) cnt[1]++;
      volatile float T = (float)acc.s;
      volatile float Ts = T * s1;
      volatile float aO = alpha * O[c];
      O[c] = aO + Ts;
    }
    m = m_new;
  }
  for (int c = 0; c < D; ++c) { volatile float o = O[c] / l; out[c] = o; }
  if (tol_out) *tol_out = (float)(tol / (double)l);
  free(qf); free(qc2); free(qs); free(qbar); free(S); free(P2); free(pc); free(psb); free(stie); free(tstep); free(O);
}

static void* attn_worker(void* arg) {
  attn_job_t* J = (attn_job_t*)arg;
  int64_t cnt[4] = {0, 0, 0, 0};
  for (;;) {
    pthread_mutex_lock(&J->mu);
    int64_t r = J->next++;
    pthread_mutex_unlock(&J->mu);
    if (r >= J->nrows) break;
    int64_t flat = J->rows[r];
    long bh = (long)(flat / J->N);
    int i = (int)(flat % J->N);
    attn_row(J, bh, i, J->out + r * J->D, J->tie_tol ? J->tie_tol + r : NULL, cnt);
  }
  pthread_mutex_lock(&J->mu);
  for (int c = 0; c < 4; ++c) J->cnt[c] += cnt[c];
  pthread_mutex_unlock(&J->mu);
  return NULL;
}

typedef struct { attn_job_t* J; long* list; long nlist; long next; pthread_mutex_t mu; } head_job_t;
static void* head_worker(void* arg) {
  head_job_t* HJ = (head_job_t*)arg;
  for (;;) {
    pthread_mutex_lock(&HJ->mu);
    long idx = HJ->next++;
    pthread_mutex_unlock(&HJ->mu);
    if (idx >= HJ->nlist) break;
    build_head(HJ->J, HJ->list[idx]);
  }
  return NULL;
}

/* ------------------------------------------------------------------------ */
/* orc_attn2: Algorithm 1 for a list of query rows; smoothing Q (flag        */
/* ORC_SMOOTH_Q) uses query blocks of bq rows.  orc_attn: bq = 128.          */
/*  q, k, v : 16-bit [B,H,N,D] host arrays (in_dtype fp16/bf16)              */
/*  rows    : flat row ids ((b*H + h)*N + i), nrows of them                   */
/*  out     : [nrows][D] fp32;  tie_tol: [nrows] or NULL;                     */
/*  counters: [4] or NULL (inexact S sums, inexact O sums, tie-ambiguous P    */
/*            codes, skipped tiles)                                          */
/* Returns 0, or -1 for invalid arguments.                                   */
/* ------------------------------------------------------------------------ */
int orc_attn2(const uint16_t* q, const uint16_t* k, const uint16_t* v, int in_dtype,
              int B, int H, int N, int D, int causal, int fmt, int bkv, int bq, unsigned flags,
              const int64_t* rows, int64_t nrows, float* out, float* tie_tol,
              int64_t* counters, int nthreads) {
  if (B <= 0 || H <= 0 || N <= 0 || D <= 0 || bkv <= 0 || bq <= 0) return -1;
  if (fmt != ORC_FMT_NONE && (D % block_of(fmt) || bkv % block_of(fmt))) return -1;
  attn_job_t J;
  memset(&J, 0, sizeof(J));
  J.q = q; J.k = k; J.v = v; J.in_dtype = in_dtype; J.B = B; J.H = H; J.N = N; J.D = D;
  J.causal = causal; J.fmt = fmt; J.bkv = bkv; J.bq = bq; J.flags = flags; J.rows = rows; J.nrows = nrows;
  J.out = out; J.tie_tol = tie_tol;
  J.heads = (head_t*)calloc((size_t)B * H, sizeof(head_t));
  J.head_used = (char*)calloc((size_t)B * H, 1);
  pthread_mutex_init(&J.mu, NULL);
  for (int64_t r = 0; r < nrows; ++r) {
    int64_t bh = rows[r] / N;
    if (rows[r] < 0 || bh >= (int64_t)B * H) { free(J.heads); free(J.head_used); return -1; }
    J.head_used[bh] = 1;
  }
  if (nthreads < 1) nthreads = 1;
  if (nthreads > 256) nthreads = 256;
  pthread_t th[256];
  head_job_t HJ;
  memset(&HJ, 0, sizeof(HJ));
  HJ.J = &J;
  HJ.list = (long*)malloc(sizeof(long) * (size_t)B * H);
  for (long bh = 0; bh < (long)B * H; ++bh) if (J.head_used[bh]) HJ.list[HJ.nlist++] = bh;
  pthread_mutex_init(&HJ.mu, NULL);
  for (int t = 0; t < nthreads; ++t) pthread_create(&th[t], NULL, head_worker, &HJ);
  for (int t = 0; t < nthreads; ++t) pthread_join(th[t], NULL);
  for (int t = 0; t < nthreads; ++t) pthread_create(&th[t], NULL, attn_worker, &J);
  for (int t = 0; t < nthreads; ++t) pthread_join(th[t], NULL);
  if (counters) for (int c = 0; c < 4; ++c) counters[c] = J.cnt[c];
  for (long i = 0; i < HJ.nlist; ++i) free_head(&J.heads[HJ.list[i]]);
  free(HJ.list); free(J.heads); free(J.head_used);
  pthread_mutex_destroy(&J.mu); pthread_mutex_destroy(&HJ.mu);
  return 0;
}

int orc_attn(const uint16_t* q, const uint16_t* k, const uint16_t* v, int in_dtype,
             int B, int H, int N, int D, int causal, int fmt, int bkv, unsigned flags,
             const int64_t* rows, int64_t nrows, float* out, float* tie_tol,
             int64_t* counters, int nthreads) {
  return orc_attn2(q, k, v, in_dtype, B, H, N, D, causal, fmt, bkv, 128, flags, rows, nrows, out, tie_tol,
                   counters, nthreads);
}

/* ------------------------------------------------------------------------ */
/* Exact attention (fp64): softmax(Q K^T / sqrt(D)) V on the unquantized     */
/* inputs (Sec. 2, FlashAttention definition), for the accuracy metrics.     */
/* causal uses the same mask as orc_attn.                                    */
/* ------------------------------------------------------------------------ */
typedef struct {
  const uint16_t *q, *k, *v; int in_dtype, N, D, causal;
  const int64_t* rows; int64_t nrows; double* out;
  int64_t next; pthread_mutex_t mu;
} exact_job_t;

static void* exact_worker(void* arg) {
  exact_job_t* J = (exact_job_t*)arg;
  int N = J->N, D = J->D;
  double* s = (double*)malloc(sizeof(double) * N);
  double* qd = (double*)malloc(sizeof(double) * D);
  for (;;) {
    pthread_mutex_lock(&J->mu);
    int64_t r = J->next++;
    pthread_mutex_unlock(&J->mu);
    if (r >= J->nrows) break;
    long bh = (long)(J->rows[r] / N);
    int i = (int)(J->rows[r] % N);
    const uint16_t* kb = J->k + bh * (long)N * D;
    const uint16_t* vb = J->v + bh * (long)N * D;
    for (int c = 0; c < D; ++c) qd[c] = orc_widen(J->q[(bh * (long)N + i) * D + c], J->in_dtype);
    double mx = -INFINITY;
    int kend = J->causal ? i + 1 : N;
    for (int kk = 0; kk < kend; ++kk) {
      double a = 0;
      for (int c = 0; c < D; ++c) a += qd[c] * (double)orc_widen(kb[(long)kk * D + c], J->in_dtype);
      s[kk] = a / sqrt((double)D);
      if (s[kk] > mx) mx = s[kk];
    }
    double den = 0;
    for (int kk = 0; kk < kend; ++kk) { s[kk] = exp(s[kk] - mx); den += s[kk]; }
    double* o = J->out + r * D;
    for (int c = 0; c < D; ++c) o[c] = 0;
    for (int kk = 0; kk < kend; ++kk) {
      double w = s[kk] / den;
      for (int c = 0; c < D; ++c) o[c] += w * (double)orc_widen(vb[(long)kk * D + c], J->in_dtype);
    }
  }
  free(s); free(qd);
  return NULL;
}

int orc_exact_attn(const uint16_t* q, const uint16_t* k, const uint16_t* v, int in_dtype,
                   int B, int H, int N, int D, int causal, const int64_t* rows, int64_t nrows,
                   double* out, int nthreads) {
  if (B <= 0 || H <= 0 || N <= 0 || D <= 0) return -1;
  exact_job_t J;
  memset(&J, 0, sizeof(J));
  J.q = q; J.k = k; J.v = v; J.in_dtype = in_dtype; J.N = N; J.D = D; J.causal = causal;
  J.rows = rows; J.nrows = nrows; J.out = out;
  pthread_mutex_init(&J.mu, NULL);
  if (nthreads < 1) nthreads = 1;
  if (nthreads > 256) nthreads = 256;
  pthread_t th[256];
  for (int t = 0; t < nthreads; ++t) pthread_create(&th[t], NULL, exact_worker, &J);
  for (int t = 0; t < nthreads; ++t) pthread_join(th[t], NULL);
  pthread_mutex_destroy(&J.mu);
  return 0;
}

/* FP4MM on explicit operands (for the brute-force pin): C[i][j] =
 * fl32(exact sum_k deq(A)[i][k] deq(B)[j][k]); codes one per byte, scales as
 * bytes in the given format, blocks of n along k.  Returns the number of
 * sums that were not exact in fp64. */
long orc_fp4mm(const uint8_t* ac, const uint8_t* as, const uint8_t* bc, const uint8_t* bs,
               int M, int Nn, int K, int fmt, float* C) {
  int n = block_of(fmt);
  long inexact = 0;
  for (int i = 0; i < M; ++i)
    for (int j = 0; j < Nn; ++j) {
      xsum_t acc = {0, 0};
      for (int blk = 0; blk < K / n; ++blk) {
        long isum = 0;
        for (int kk = 0; kk < n; ++kk) {
          int a2, b2;
          two_code(orc_e2m1_decode(ac[(long)i * K + blk * n + kk]), &a2);
          two_code(orc_e2m1_decode(bc[(long)j * K + blk * n + kk]), &b2);
          isum += (long)a2 * b2;
        }
        double sa = scale_value(as[(long)i * (K / n) + blk], fmt), sb = scale_value(bs[(long)j * (K / n) + blk], fmt);
        xsum_add(&acc, (double)isum * (sa * sb) * 0.25);
      }
      if (acc.err != 0.0) inexact++;
      C[(long)i * Nn + j] = (float)acc.s;
    }
  return inexact;
}
