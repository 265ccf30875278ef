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
#define ORC_FUSED_P 256u     /* P~2 in the fused order a GPU evaluates it (for the
                                test that bounds its differences; orc_p_tile)     */

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
  int64_t* counters; /* [5]: inexact S sums, inexact O sums, ambiguous P codes, skipped tiles,
                        P blocks with another accepted scale */
  head_t* heads;     /* [B*H], only the ones used are filled */
  char* head_used;
  int64_t next;
  pthread_mutex_t mu;
  int64_t cnt[5];
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

/* half an fp32 ulp at magnitude |x|: the largest error of one fp32 rounding
   to a result of that size (subnormal results: half the smallest step) */
static double hulp32(double x) {
  x = fabs(x);
  if (x < 0x1p-126) return 0x1p-150;
  int e;
  frexp(x, &e);                      /* x = f 2^e, f in [0.5, 1): ulp = 2^(e-24) */
  return ldexp(1.0, e - 25);
}

/* ------------------------------------------------------------------------ */
/* orc_p_tile: one KV tile of one query row -- the online-softmax step and   */
/* the two-level quantization of P~ (Algorithm 1; Sec. 3.2, Eq. two-level),  */
/* evaluated in the order the paper writes them:                             */
/*                                                                           */
/*   m_new = max(m_old, rowmax(S))                                           */
/*   P~_k  = exp(S_k - m_new)        base 2 with the softmax scale (R7):     */
/*           fl32(exp2(fl32(fl32(S_k c2) - fl32(m_new c2))))                  */
/*   rowsum(P~) = sequential fp32 sum of the P~_k (l takes it unquantized)   */
/*   alpha = exp(m_old - m_new) = fl32(exp2(fl32(fl32(m_old c2) - fl32(m_new c2)))), */
/*           0 on the first visited tile                                     */
/*   rho   = rowmax(P~) over the tile (R9)                                   */
/*   s_P1  = fl32(rho / R)                                                   */
/*   P~2_k = P~_k / s_P1, read as fl32(P~_k fl32(1/s_P1)) (R4)               */
/*   (s_P2, P^2) = phi(P~2) over the n-key blocks of the tile (Sec. 3.1):    */
/*           MX: e = smallest e with 6 2^e >= max of the block's P~2 values, */
/*               clamped to [-127, 127] (R2); codes E2M1(P~2 2^-e);          */
/*           NV16: s = E4M3(fl32(amax/6)), codes E2M1(fl32(P~2 fl32(1/s)))   */
/*   s_P1 < 2^-126 (below the normal fp32 range, its reciprocal would       */
/*           overflow) -> the tile adds nothing to O: s_P1 = 0, P^ = 0.      */
/*                                                                           */
/* R = 6 with E8M0 scales, 448*6 with E4M3 scales (R8); ORC_R_LITERAL keeps  */
/* 448*6 with E8M0 (ablation).  ORC_DIRECT_P quantizes P~ itself (s_P1 = 1,  */
/* ablation of Table 1(b)).                                                  */
/*                                                                           */
/* ORC_FUSED_P evaluates the same quantities in the fused order a GPU uses:  */
/* P~2_k = exp2(fma(S_k, c2, fl32(fl32(log2 R) - fl32(t c2)))), the MX block */
/* exponent from scores, e = max(ceil(fl32(fl32(bm - t) c2)), -126) with bm  */
/* the block's largest score, s_P1 = fl32(exp2(fl32(t c2) - fl32(m c2))/R),  */
/* rowsum = fl32(s_P1 sum P~2).  NV16 takes the block scale s = M 2^X from   */
/* the fused P~2 values as above, and folds the division by s into the      */
/* exponent: y_k = exp2(fma(S_k, c2, fl32(B - fl32(log2 M)))), codes         */
/* E2M1(y_k 2^-X) (exact), the row sum s_P1 sum over blocks of M sum y_k (a  */
/* block with s = 0 keeps its P~2 values in the row sum and gets zero codes).*/
/* Equal in exact arithmetic; it exists so that a test can show every       */
/* difference it makes lies inside the set of results the intervals below   */
/* accept.                                                                   */
/*                                                                           */
/* Acceptance intervals (the paper fixes no fp32 evaluation order).  For     */
/* each key, [lo, hi] holds every P~2 value that either evaluation can       */
/* produce: the plain value above, and the fused value, whose log2 differs   */
/* from the exact log2 R + c2 (S_k - t) (fp64 here) by at most               */
/*   W_k = h(log2 R) + h(t c2) + h(B) + h(arg_k) + 2^-22/ln 2,               */
/* h = half an fp32 ulp of each rounded intermediate (B = fl32(log2 R - t c2),*/
/* arg_k = fl32(fma(S_k, c2, B))), the last term a 1-ulp exp2 plus its own   */
/* rounding.  NV16 adds the roundings of the folded division (log2 M with   */
/* M <= 15 to within an ulp, B - log2 M, and the fma at that argument), each */
/* bounded by half an ulp at |B| + 4 or |arg_k| + 4, or an ulp at 4.          */
/* [sb_lo, sb_hi] holds every block scale byte either evaluation             */
/* can choose: MX -- the plain exponent and ceil of the score-domain         */
/* exponent c2 (bm - t) within its two roundings; NV16 -- E4M3 of amax/6 for */
/* amax anywhere in the block max's interval (and the plain one).  The       */
/* block holding the tile max has c2 (bm - t) = 0 exactly, so the fused      */
/* choice there is 2^0, while the plain P~2 of that key lands within an ulp  */
/* of 6 on either side: when it lands above, the plain rule takes 2^1 and    */
/* both bytes are in the range.                                              */
/* cont_out: sum over keys of (hi - lo), the bound on the move of the tile's */
/* unquantized row sum between the two evaluations (in P~2 units).           */
/* ------------------------------------------------------------------------ */
int orc_p_tile(const float* S, int bkv, float m_old, int D, int fmt, unsigned flags,
               float* m_new_out, float* alpha_out, float* s1_out, float* rowsum_out,
               float* p2, uint8_t* codes, uint8_t* sbytes, double* lo, double* hi,
               uint8_t* sb_lo, uint8_t* sb_hi, double* cont_out) {
  const int n = (fmt == ORC_FMT_NONE) ? 1 : block_of(fmt);
  const int direct = (flags & ORC_DIRECT_P) != 0, fused = (flags & ORC_FUSED_P) != 0;
  const float c2 = (float)(1.0 / (log(2.0) * sqrt((double)D)));
  const float R = (fmt == ORC_FMT_NV16 || (flags & ORC_R_LITERAL)) ? 448.0f * 6.0f : 6.0f;
  const float logR = (float)log2((double)R);

  float t = -INFINITY;                                  /* rowmax(S) of the tile */
  for (int kk = 0; kk < bkv; ++kk) if (S[kk] > t) t = S[kk];
  if (t == -INFINITY) return -1;
  const float m_new = m_old > t ? m_old : t;
  volatile float tc = t * c2;                           /* u = S c2 is monotone in S */
  volatile float mc_new = m_new * c2;
  float alpha = 0.0f;
  if (m_old != -INFINITY) { volatile float mc_old = m_old * c2; volatile float d = mc_old - mc_new; alpha = exp2_f32(d); }

  float s1, psum = 0.0f, rowsum;
  if (fused) {
    volatile float bias;
    if (direct) { s1 = 1.0f; bias = -mc_new; }
    else { volatile float dt = tc - mc_new; volatile float q = exp2_f32(dt) / R; s1 = q; bias = logR - tc; }
    for (int kk = 0; kk < bkv; ++kk) {
      p2[kk] = (S[kk] == -INFINITY) ? 0.0f : exp2_f32(fmaf(S[kk], c2, bias));
      psum += p2[kk];
    }
    volatile float rs = s1 * psum;
    rowsum = rs;                          /* NV16 without DIRECT_P: replaced below */
  } else {
    /* P~ = exp(S - m_new), its row sum and its row max */
    float rho = 0.0f;
    for (int kk = 0; kk < bkv; ++kk) {
      float p = 0.0f;
      if (S[kk] != -INFINITY) { volatile float u = S[kk] * c2; volatile float d = u - mc_new; p = exp2_f32(d); }
      p2[kk] = p;
      psum += p;
      if (p > rho) rho = p;
    }
    rowsum = psum;
    if (direct) s1 = 1.0f;
    else {
      /* s_P1 = rowmax(P~)/R; P~2 = P~/s_P1 */
      volatile float q = rho / R;
      s1 = q;
    }
    if (!direct && s1 < 0x1p-126f) {
      /* s_P1 below the normal fp32 range (P~ underflows, or the tile lies
         more than 126 binades under the running max): 1/s_P1 would overflow,
         and the tile adds nothing to O */
      s1 = 0.0f;
      for (int kk = 0; kk < bkv; ++kk) p2[kk] = 0.0f;
    } else if (!direct) {
      volatile float r = 1.0f / s1;
      for (int kk = 0; kk < bkv; ++kk) { volatile float y = p2[kk] * r; p2[kk] = y; }
    }
  }
  *m_new_out = m_new; *alpha_out = alpha; *s1_out = s1; *rowsum_out = rowsum;
  if (cont_out) *cont_out = 0.0;

  /* acceptance intervals of the P~2 values */
  if (lo) {
    volatile float B = logR - tc;
    const double wfix = hulp32(logR) + hulp32(tc) + hulp32(B) + 0x1p-22 / log(2.0);
    double cont = 0.0;
    for (int kk = 0; kk < bkv; ++kk) {
      if (S[kk] == -INFINITY) { lo[kk] = hi[kk] = 0.0; continue; }
      if (direct) { lo[kk] = hi[kk] = p2[kk]; continue; }
      const double pex = (double)R * exp2((double)c2 * ((double)S[kk] - (double)t));
      const float arg = fmaf(S[kk], c2, B);
      double W = wfix + hulp32(arg);
      if (fmt == ORC_FMT_NV16) W += hulp32(4.0) + hulp32(fabs((double)B) + 4.0) + hulp32(fabs((double)arg) + 4.0);
      double flo = pex * exp2(-W), fhi = pex * exp2(W);
      if (fhi < 0x1p-120) { flo = 0.0; fhi += 0x1p-147; } /* fp32 flushes or rounds to subnormal steps there */
      lo[kk] = flo < p2[kk] ? flo : p2[kk];
      hi[kk] = fhi > p2[kk] ? fhi : p2[kk];
      cont += hi[kk] - lo[kk];
    }
    if (cont_out) *cont_out = cont;
  }
  if (fmt == ORC_FMT_NONE) return 0;

  /* second level: (s_P2, P^2) = phi(P~2) over n-key blocks */
  float fsum_nv = 0.0f;                 /* NV16, fused order: sum over blocks of M sum y */
  for (int b0 = 0; b0 < bkv; b0 += n) {
    const int blk = b0 / n;
    float am = 0.0f, bm = -INFINITY;
    for (int kk = b0; kk < b0 + n; ++kk) { if (p2[kk] > am) am = p2[kk]; if (S[kk] > bm) bm = S[kk]; }
    if (fmt == ORC_FMT_MX) {
      int e;
      if (fused && !direct && !(flags & (ORC_R_LITERAL | ORC_OCP_SCALE))) {
        if (bm == -INFINITY) e = -126;
        else { volatile float dd = bm - t; volatile float d2 = dd * c2; e = (int)ceilf(d2); }
        if (e < -126) e = -126;
      } else {
        e = (flags & ORC_OCP_SCALE) ? orc_e8m0_exponent_floor(am) : orc_e8m0_exponent(am);
      }
      sbytes[blk] = (uint8_t)(e + 127);
      for (int kk = b0; kk < b0 + n; ++kk) codes[kk] = orc_e2m1_encode(ldexpf(p2[kk], -e));
      if (sb_lo) {
        int elo = e, ehi = e;
        if (!direct && bm != -INFINITY && !(flags & (ORC_R_LITERAL | ORC_OCP_SCALE))) {
          /* the score-domain exponent: c2 (bm - t) after the roundings of
             bm - t and of the product */
          volatile float dd = bm - t;
          const double x = (double)c2 * ((double)bm - (double)t);
          /* bm = t (the block holding the tile max): both roundings are exact */
          const double w = dd == 0.0f ? 0.0 : hulp32(dd) * (double)c2 + hulp32((double)dd * c2);
          int a = (int)ceil(x - w), b = (int)ceil(x + w);
          if (a < -126) a = -126;
          if (b < -126) b = -126;
          if (a < elo) elo = a;
          if (b > ehi) ehi = b;
        } else if (!direct && bm != -INFINITY) {
          /* ablation rules on the value maximum: any value in the block max's interval */
          double hm = 0.0, lm = 0.0;
          for (int kk = b0; kk < b0 + n; ++kk) { if (hi[kk] > hm) hm = hi[kk]; if (lo[kk] > lm) lm = lo[kk]; }
          int a = (flags & ORC_OCP_SCALE) ? orc_e8m0_exponent_floor((float)lm) : orc_e8m0_exponent((float)lm);
          int b = (flags & ORC_OCP_SCALE) ? orc_e8m0_exponent_floor((float)hm) : orc_e8m0_exponent((float)hm);
          if (a < elo) elo = a;
          if (b > ehi) ehi = b;
        }
        sb_lo[blk] = (uint8_t)(elo + 127);
        sb_hi[blk] = (uint8_t)(ehi + 127);
      }
    } else {
      uint8_t sb = orc_phi_block(p2 + b0, n, fmt, codes + b0);
      sbytes[blk] = sb;
      if (fused && !direct) {
        /* the division by s = M 2^X folded into the exponent (see above) */
        const int E = sb >> 3, man = sb & 7;
        const int M = E ? 8 + man : man, X = E ? E - 10 : -9;
        const float lgm = M ? (float)log2((double)M) : 0.0f;
        volatile float Bf = logR - tc;
        volatile float bb = Bf - lgm;
        float ys = 0.0f;
        for (int kk = b0; kk < b0 + n; ++kk) {
          const float y = (S[kk] == -INFINITY) ? 0.0f : exp2_f32(fmaf(S[kk], c2, bb));
          ys += y;
          codes[kk] = M ? orc_e2m1_encode(ldexpf(y, -X)) : 0;
        }
        volatile float wsum = (float)(M ? M : 1) * ys;
        fsum_nv += wsum;
      }
      if (sb_lo) {
        /* E4M3(fl32(amax/6)) for amax anywhere in the block max's interval;
           the division's own rounding widens it by an ulp */
        double hm = 0.0, lm = 0.0;
        for (int kk = b0; kk < b0 + n; ++kk) { if (hi[kk] > hm) hm = hi[kk]; if (lo[kk] > lm) lm = lo[kk]; }
        uint8_t a = orc_e4m3_encode((float)(lm / 6.0 * (1.0 - 0x1p-23)));
        uint8_t b = orc_e4m3_encode((float)(hm / 6.0 * (1.0 + 0x1p-23)));
        sb_lo[blk] = a < sb ? a : sb;
        sb_hi[blk] = b > sb ? b : sb;
      }
    }
  }
  if (fused && !direct && fmt == ORC_FMT_NV16) { volatile float rs = s1 * fsum_nv; *rowsum_out = rs; }
  return 0;
}

/* dequantized V^ of key k, channel c (zero past the padded tail) */
static double vhat(const head_t* h, int c, int k) {
  if (k >= h->Np) return 0.0;
  return 0.5 * (double)h->vc2[(long)c * h->Np + k] * (double)h->vs[(long)c * (h->Np / h->n) + k / h->n];
}

/* the E2M1 code of a P~2 value at block scale byte sb: MX divides by the
   power of two exactly, NV16 multiplies by fl32(1/s) (R4) */
static uint8_t p_code(float y, uint8_t sb, int fmt) {
  if (fmt == ORC_FMT_MX) return orc_e2m1_encode(ldexpf(y, -((int)sb - 127)));
  const float s = orc_e4m3_decode(sb);
  if (!(s > 0.0f)) return 0;
  volatile float r = 1.0f / s;
  volatile float q = y * r;
  return orc_e2m1_encode(q);
}

/* largest change of a code's value (times the scale sc) when its P~2 value
   is anywhere in [lo, hi], against the code c; the interval is widened by
   2^-21 so that the rounding of y/sc to fp32 and of NV16's reciprocal never
   narrows it */
static double code_dev(double lo, double hi, double sc, uint8_t c) {
  if (!(sc > 0.0)) return 0.0;
  const double v = orc_e2m1_decode(c);
  const double a = orc_e2m1_decode(orc_e2m1_encode((float)(lo * (1.0 - 0x1p-21) / sc)));
  const double b = orc_e2m1_decode(orc_e2m1_encode((float)(hi * (1.0 + 0x1p-21) / sc)));
  const double d = fabs(a - v) > fabs(b - v) ? fabs(a - v) : fabs(b - v);
  return d * sc;
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
/*  - the softmax step and the two-level quantization of each tile follow    */
/*    Algorithm 1's order (orc_p_tile): P~, its row sum and row max, s_P1,   */
/*    P~2 = P~/s_P1, phi(P~2).                                               */
/*  - l = fl32(fl32(alpha l) + rowsum(P~)), over the unquantized P~.         */
/*  - O_new = fl32(fl32(alpha O) + fl32(FP4MM(P^2, V^) s_P1)).               */
/*  - the final O = fl32(O / l).                                             */
/*  - causal: key k is visible to query i iff k <= i; fully masked tiles are  */
/*    skipped; keys >= N are masked.                                         */
/* tie_tol: a bound on |O_c| - over the channels c - of the change between  */
/* this result and any other accepted evaluation of the P step (orc_p_tile's */
/* intervals).  Per tile and block it takes the larger of (a) the codes that */
/* any value in a key's interval maps to at the block's own scale, and (b)   */
/* for every other accepted block scale, the exact change of that block's    */
/* contribution to O_c when its codes are re-derived at that scale, plus     */
/* (a) at that scale; both weigh |V^_kc| and are scaled by s_P1, carried    */
/* through alpha like O and divided by l at the end.  The row sum moves by   */
/* at most s_P1 sum_k (hi - lo) per tile between evaluations (plus 2^-20 of  */
/* the tile's row sum for the fp32 roundings of s_P1 and alpha); that moves  */
/* O by at most max|V^| times it over l.  Tiles whose s_P1 lies below     */
/* 2^-126 add a bound of bkv 2^-110 max|V^| (R 2^-126 per key, both ways).  */
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
  double* plo = (double*)malloc(sizeof(double) * bkv);
  double* phi = (double*)malloc(sizeof(double) * bkv);
  uint8_t* sblo = (uint8_t*)malloc((size_t)nblk + 1);
  uint8_t* sbhi = (uint8_t*)malloc((size_t)nblk + 1);
  double* tolc = (double*)calloc(D, sizeof(double));
  double* blkc = (double*)calloc(D, sizeof(double));
  double tolcont = 0.0;
  float* O = (float*)calloc(D, sizeof(float));
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
    double cont = 0.0;
    orc_p_tile(S, bkv, m, D, fmt, J->flags, &m_new, &alpha, &s1, &rowsum, P2, pc, psb,
               tol_out ? plo : NULL, tol_out ? phi : NULL, tol_out ? sblo : NULL, tol_out ? sbhi : NULL, &cont);
    volatile float al = alpha * l;
    l = al + rowsum;

    if (fmt != ORC_FMT_NONE && tol_out) {
      for (int c = 0; c < D; ++c) tolc[c] *= (double)alpha;
      tolcont = (double)alpha * tolcont + (double)s1 * cont + (double)rowsum * 0x1p-20 +
                (s1 == 0.0f ? (double)bkv * 0x1p-110 : 0.0);
      for (int blk = 0; blk < nblk && s1 > 0.0f; ++blk) {
        const int b0 = blk * n;
        if (k0 + b0 >= h->Np) break;                   /* V^ is zero past the padded tail */
        if (fmt == ORC_FMT_MX && sbhi[blk] < 127 - 120) {
          /* every accepted scale is below 2^-120: bound the block's whole
             contribution instead of enumerating it */
          const double bnd = (double)s1 * n * 6.0 * ldexp(1.0, (int)sbhi[blk] - 127) * h->vabs_max;
          for (int c = 0; c < D; ++c) tolc[c] += bnd;
          continue;
        }
        const double sc = scale_value(psb[blk], fmt);
        /* (a) at the block's own scale */
        for (int c = 0; c < D; ++c) blkc[c] = 0.0;
        for (int kk = b0; kk < b0 + n; ++kk) {
          const double dv = code_dev(plo[kk], phi[kk], sc, pc[kk]);
          if (dv == 0.0) continue;
          cnt[2]++;
          for (int c = 0; c < D; ++c) blkc[c] += dv * fabs(vhat(h, c, k0 + kk));
        }
        /* (b) every other accepted block scale */
        for (int sb = sblo[blk]; sb <= sbhi[blk]; ++sb) {
          if (sb == psb[blk]) continue;
          cnt[4]++;
          const double sa = scale_value((uint8_t)sb, fmt);
          uint8_t ca[32];
          double dva[32];
          for (int kk = b0; kk < b0 + n; ++kk) {
            ca[kk - b0] = p_code(P2[kk], (uint8_t)sb, fmt);
            dva[kk - b0] = code_dev(plo[kk], phi[kk], sa, ca[kk - b0]);
          }
          for (int c = 0; c < D; ++c) {
            double d = 0.0, w = 0.0;
            for (int kk = b0; kk < b0 + n; ++kk) {
              const double v = vhat(h, c, k0 + kk);
              d += ((double)orc_e2m1_decode(ca[kk - b0]) * sa - (double)orc_e2m1_decode(pc[kk]) * sc) * v;
              w += dva[kk - b0] * fabs(v);
            }
            if (fabs(d) + w > blkc[c]) blkc[c] = fabs(d) + w;
          }
        }
        for (int c = 0; c < D; ++c) tolc[c] += (double)s1 * blkc[c];
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
  if (tol_out) {
    double tmax = 0.0;
    for (int c = 0; c < D; ++c) if (tolc[c] > tmax) tmax = tolc[c];
    *tol_out = (float)((tmax + h->vabs_max * tolcont) / (double)l);
  }
  free(qf); free(qc2); free(qs); free(qbar); free(S); free(P2); free(pc); free(psb); free(O);
  free(plo); free(phi); free(sblo); free(sbhi); free(tolc); free(blkc);
}

static void* attn_worker(void* arg) {
  attn_job_t* J = (attn_job_t*)arg;
  int64_t cnt[5] = {0, 0, 0, 0, 0};
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
  for (int c = 0; c < 5; ++c) J->cnt[c] += cnt[c];
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
/*  counters: [5] or NULL (inexact S sums, inexact O sums, P codes with an   */
/*            accepted alternative, skipped tiles, P blocks with an accepted */
/*            alternative scale)                                             */
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
  if (counters) for (int c = 0; c < 5; ++c) counters[c] = J.cnt[c];
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
