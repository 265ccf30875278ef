/*
 * sage_oracle_int8.c -- plain, slow CPU oracle for the 8-bit attention of
 * SageBwd (arXiv 2505.11594): the forward (Algorithm 2) and the backward
 * (Algorithm 3, further below).
 *
 * TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the
 * benchmark's CPU-baseline leg may load this library.  It shares no source
 * with the HIP path and the HIP path never calls it.
 *
 * What it follows (paper sections / equations):
 *   - smoothing K: K <- K - mean(K) over the tokens (Algorithm 2, first
 *     step; the mean is the same exact fp64 quotient as the FP4 oracle's);
 *   - per-block INT8 quantization psi (Sec. 4.1, Eq. psi): s = max|X|/127,
 *     X^ = X/s, for Q blocks of B_q rows and K, V blocks of B_kv rows;
 *   - S = MM(Q^, K^) * s_Q * s_K, online softmax over KV tiles (FlashAttention
 *     tiling), per-token quantization of P~ reusing the row maxima:
 *     s_P = exp(rowmax(S_ij) - m_ij)/127, P^ = P~/s_P, and
 *     O = diag(e^{m_old-m_new}) O + MM(P^, V^) * s_P * s_V;
 *   - the outputs O = O/l and L = m + log(l).
 *
 * Readings of points Algorithm 2 leaves open (the kernels implement the same):
 *   - rounding of X/s: X/s is read as x * fl32(1/s) with s = fl32(amax/127),
 *     rounded to the nearest integer, ties to even (|code| <= 127 then holds);
 *     a block of zeros gets s = 0 and zero codes.
 *   - softmax scale 1/sqrt(D), exp taken base 2 (as in the FP4 oracle): the
 *     scores are kept in the log2 domain u = fl32(fl32(acc) * c_t) with
 *     c_t = fl32(fl32(s_Q s_K) c2), c2 = fl32(log2(e)/sqrt(D)), acc the exact
 *     integer product of the codes (|acc| < 2^24 for D <= 128, so fl32(acc)
 *     is exact).  The running max m and the tile max t are in this domain.
 *   - the per-token quantization of P~ in Algorithm 2's order:
 *     P~_k = fl32(exp2(fl32(u_k - m_new))), s_P = fl32(exp(rowmax(S) - m)/127)
 *     = fl32(fl32(exp2(fl32(t - m_new)))/127), P^_k = P~_k/s_P read as
 *     rint(fl32(P~_k fl32(1/s_P))) (ties to even, at most 127).  A tile whose
 *     s_P lies below the normal fp32 range adds nothing (1/s_P would overflow).
 *   - l accumulates the unquantized P~ as Algorithm 2 writes it:
 *     l = fl32(fl32(alpha l) + rowsum(P~)), the row sum sequential in fp32;
 *     alpha = 2^{m_old - m_new}, 0 on the first visited tile (the running max
 *     starts at -inf).
 *   - tolerance: a GPU may evaluate P^ in the fused order
 *     exp2(fma(fl32(acc), c_t, fl32(log2 127 - t))); per key, [lo, hi] holds
 *     every value either order can reach before rounding -- the plain value
 *     and 127 2^{acc c_t - t} (fp64) within the fused order's roundings,
 *     W = h(log2 127) + h(t) + h(B) + h(arg) + 2^-22/ln 2 in log2 units
 *     (h = half an fp32 ulp of each rounded intermediate).  Every code that
 *     [lo, hi] reaches adds its distance to the plain code times s_P s_V
 *     max|V^ row|, and the row sum's move s_P sum (hi - lo) adds max|V^|
 *     times it; both are carried through alpha and divided by l.
 *   - O = fma(fl32(MM(P^, V^)), fl32(s_P s_V), fl32(alpha O)) per tile, the
 *     integer product exact; O = fl32(O / l) at the end.
 *   - L is the natural-log log-sum-exp of the scaled scores S/sqrt(D):
 *     L = fl32(fl32(m + log2(l)) * fl32(ln 2)).
 *   - causal: key j visible to query i iff j <= i; fully masked tiles are
 *     skipped; keys >= N are masked; the last K and V blocks hold the
 *     remaining rows.
 *
 * Flags: ORC_NO_SMOOTH_K (1) skips smoothing K; ORC_I8_STATIC_P (32) is the
 * ablation the paper argues against: P~ = 2^{u - m} quantized with the static
 * scale 1/127; ORC_I8_IDENTITY (64) skips every quantization (pins the
 * tiling, the online softmax and L against textbook attention);
 * ORC_I8_FUSED_P (512) evaluates P^ in the fused order (a test shows the
 * difference stays inside the tolerance).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#include <pthread.h>

float orc_widen(uint16_t bits, int in_dtype);
long orc_kmean(const uint16_t* k, int in_dtype, int B, int H, int N, int D, float* mu);

#define ORC_NO_SMOOTH_K 1u
#define ORC_I8_STATIC_P 32u
#define ORC_I8_IDENTITY 64u
#define ORC_I8_FUSED_P 512u   /* P^ in the fused order a GPU evaluates it (for the test
                                 that bounds its differences): rint(exp2(fma(fl32(acc),
                                 c_t, fl32(log2 127 - t)))), l += fl32(s_P sum of them) */

#define ORC_ROLE_Q 0
#define ORC_ROLE_K 1
#define ORC_ROLE_V 2


/* ------------------------------------------------------------------------ */
/* psi on one block of n values (Eq. psi).  Returns the scale.               */
/* ------------------------------------------------------------------------ */
float orc_psi_block(const float* x, long n, int8_t* codes) {
  float amax = 0.0f;
  for (long k = 0; k < n; ++k) { float a = fabsf(x[k]); if (a > amax) amax = a; }
  if (!(amax > 0.0f)) { memset(codes, 0, (size_t)n); return 0.0f; }
  volatile float s = amax / 127.0f;
  volatile float r = 1.0f / s;
  for (long k = 0; k < n; ++k) {
    volatile float y = x[k] * r;
    float c = rintf(y);                       /* nearest, ties to even */
    if (c > 127.0f) c = 127.0f;
    if (c < -127.0f) c = -127.0f;
    codes[k] = (int8_t)c;
  }
  return s;
}

/* ------------------------------------------------------------------------ */
/* Quantize one tensor, logical layout.  Role Q: blocks of blk rows of Q;    */
/* role K: of K' = fl32(K - mu) (mu: output [B,H,D], the smoothing mean,     */
/* unless smooth_k = 0); role V: of V.  codes [B,H,N,D] int8, scales          */
/* [B,H,ceil(N/blk)] fp32.  Returns the k-mean inexact count (role K).        */
/* ------------------------------------------------------------------------ */
long orc_quant_int8(const uint16_t* x, int in_dtype, int role, int B, int H, int N, int D, int blk, int smooth_k,
                    int8_t* codes, float* scales, float* mu) {
  long inexact = 0;
  const int nb = (N + blk - 1) / blk;
  if (role == ORC_ROLE_K && smooth_k) inexact = orc_kmean(x, in_dtype, B, H, N, D, mu);
  float* work = (float*)malloc(sizeof(float) * (size_t)blk * D);
  for (long bh = 0; bh < (long)B * H; ++bh) {
    const uint16_t* xb = x + bh * (long)N * D;
    for (int b = 0; b < nb; ++b) {
      const int r0 = b * blk, r1 = (r0 + blk < N) ? r0 + blk : N;
      for (int t = r0; t < r1; ++t)
        for (int c = 0; c < D; ++c) {
          float v = orc_widen(xb[(long)t * D + c], in_dtype);
          if (role == ORC_ROLE_K && smooth_k) { volatile float d = v - mu[bh * D + c]; v = d; }
          work[(long)(t - r0) * D + c] = v;
        }
      scales[bh * nb + b] = orc_psi_block(work, (long)(r1 - r0) * D, codes + (bh * (long)N + r0) * D);
    }
  }
  free(work);
  return inexact;
}

/* ------------------------------------------------------------------------ */
/* Per-head operands.                                                        */
/* ------------------------------------------------------------------------ */
typedef struct {
  int8_t *qc, *kc, *vc;       /* [N][D] codes                               */
  float *qs, *ks, *vs;        /* block scales                               */
  int* vrow_max;              /* [N] max_d |V^[k,d]| (tie bound)            */
  float *qf, *kf, *vf;        /* identity mode: Q, K', V in fp32            */
  double vabs_max;            /* max |V| (identity), max |deq(V^)| otherwise */
} i8head_t;

typedef struct {
  const uint16_t *q, *k, *v;
  int in_dtype, B, H, N, D, causal, bq, bkv;
  unsigned flags;
  const int64_t* rows;
  int64_t nrows;
  float *out, *lse, *tie_tol;
  i8head_t* heads;
  int64_t next;
  pthread_mutex_t mu;
  int64_t cnt[2];             /* tie-ambiguous P codes, skipped tiles */
} i8job_t;

static void i8_build_head(i8job_t* J, long bh) {
  i8head_t* h = &J->heads[bh];
  const int N = J->N, D = J->D;
  const long ND = (long)N * D;
  const uint16_t *qb = J->q + bh * ND, *kb = J->k + bh * ND, *vb = J->v + bh * ND;
  const int smooth = !(J->flags & ORC_NO_SMOOTH_K);
  if (J->flags & ORC_I8_IDENTITY) {
    float* mu = (float*)calloc(D, sizeof(float));
    if (smooth) orc_kmean(kb, J->in_dtype, 1, 1, N, D, mu);
    h->qf = (float*)malloc(sizeof(float) * ND);
    h->kf = (float*)malloc(sizeof(float) * ND);
    h->vf = (float*)malloc(sizeof(float) * ND);
    double vm = 0.0;
    for (long e = 0; e < ND; ++e) {
      h->qf[e] = orc_widen(qb[e], J->in_dtype);
      float kv = orc_widen(kb[e], J->in_dtype);
      if (smooth) { volatile float d = kv - mu[e % D]; kv = d; }
      h->kf[e] = kv;
      h->vf[e] = orc_widen(vb[e], J->in_dtype);
      if (fabs(h->vf[e]) > vm) vm = fabs(h->vf[e]);
    }
    h->vabs_max = vm;
    free(mu);
    return;
  }
  const int nqb = (N + J->bq - 1) / J->bq, nkb = (N + J->bkv - 1) / J->bkv;
  float* mu = (float*)calloc(D, sizeof(float));
  h->qc = (int8_t*)malloc(ND); h->kc = (int8_t*)malloc(ND); h->vc = (int8_t*)malloc(ND);
  h->qs = (float*)malloc(sizeof(float) * nqb);
  h->ks = (float*)malloc(sizeof(float) * nkb);
  h->vs = (float*)malloc(sizeof(float) * nkb);
  orc_quant_int8(qb, J->in_dtype, ORC_ROLE_Q, 1, 1, N, D, J->bq, 0, h->qc, h->qs, NULL);
  orc_quant_int8(kb, J->in_dtype, ORC_ROLE_K, 1, 1, N, D, J->bkv, smooth, h->kc, h->ks, mu);
  orc_quant_int8(vb, J->in_dtype, ORC_ROLE_V, 1, 1, N, D, J->bkv, 0, h->vc, h->vs, NULL);
  h->vrow_max = (int*)malloc(sizeof(int) * N);
  h->vabs_max = 0.0;
  for (int k = 0; k < N; ++k) {
    int m = 0;
    for (int c = 0; c < D; ++c) { int a = abs(h->vc[(long)k * D + c]); if (a > m) m = a; }
    h->vrow_max[k] = m;
    const double a = (double)m * h->vs[k / J->bkv];
    if (a > h->vabs_max) h->vabs_max = a;
  }
  free(mu);
}

static void i8_free_head(i8head_t* h) {
  free(h->qc); free(h->kc); free(h->vc); free(h->qs); free(h->ks); free(h->vs); free(h->vrow_max);
  free(h->qf); free(h->kf); free(h->vf);
  memset(h, 0, sizeof(*h));
}

static float exp2_cr(float x) { return (float)exp2((double)x); }   /* correctly rounded fp32 exp2 */
static float log2_cr(float x) { return (float)log2((double)x); }

/* half an fp32 ulp at magnitude |x| (subnormal results: half the smallest step) */
static double i8_hulp(double x) {
  x = fabs(x);
  if (x < 0x1p-126) return 0x1p-150;
  int e;
  frexp(x, &e);
  return ldexp(1.0, e - 25);
}

/* rint clamped to the code range [0, 127] of P^ */
static double i8_pcode(double y) { double c = rint(y); return c > 127.0 ? 127.0 : c; }

/* One query row of Algorithm 2. */
static void i8_row(i8job_t* J, long bh, int i, float* out, float* lse, float* tol_out, int64_t* cnt) {
  const i8head_t* h = &J->heads[bh];
  const int N = J->N, D = J->D, bkv = J->bkv;
  const int ident = (J->flags & ORC_I8_IDENTITY) != 0, stat = (J->flags & ORC_I8_STATIC_P) != 0;
  const float c2 = (float)(1.0 / (log(2.0) * sqrt((double)D)));
  const float log127 = (float)log2(127.0);
  const float sQ = ident ? 1.0f : h->qs[i / J->bq];
  float* accf = (float*)malloc(sizeof(float) * bkv);
  float* ub = (float*)malloc(sizeof(float) * bkv);      /* u = fl32(acc) c_t */
  float* pt = (float*)malloc(sizeof(float) * bkv);      /* P~ */
  float* code = (float*)malloc(sizeof(float) * bkv);    /* P^ (identity: P~/s_P unrounded) */
  char* valid = (char*)malloc((size_t)bkv);
  float* O = (float*)calloc(D, sizeof(float));
  double tol = 0.0, tolcont = 0.0;
  float m = -INFINITY, l = 0.0f;

  const int ntiles = (N + bkv - 1) / bkv;
  for (int j = 0; j < ntiles; ++j) {
    const int k0 = j * bkv;
    if (J->causal && k0 > i) { cnt[1]++; continue; }
    const float sK = ident ? 1.0f : h->ks[j];
    volatile float sqk = sQ * sK;
    volatile float ct = sqk * c2;
    /* S_ij = MM(Q^_i, K^_j) s_Q s_K, in the log2 domain u = fl32(acc) c_t */
    float t = -INFINITY;
    for (int kk = 0; kk < bkv; ++kk) {
      const int k = k0 + kk;
      valid[kk] = !(k >= N || (J->causal && k > i));
      if (!valid[kk]) continue;
      if (ident) {
        double a = 0.0;
        for (int c = 0; c < D; ++c) a += (double)h->qf[(long)i * D + c] * (double)h->kf[(long)k * D + c];
        accf[kk] = (float)a;
      } else {
        long a = 0;
        for (int c = 0; c < D; ++c) a += (long)h->qc[(long)i * D + c] * h->kc[(long)k * D + c];
        accf[kk] = (float)a;                 /* exact: |a| <= 127^2 D < 2^24 */
      }
      volatile float u = accf[kk] * ct;
      ub[kk] = u;
      if (u > t) t = u;
    }
    if (t == -INFINITY) { cnt[1]++; continue; }
    const float m_new = m > t ? m : t;
    float alpha = 0.0f;
    if (m != -INFINITY) { volatile float d = m - m_new; alpha = exp2_cr(d); }
    /* P~ = exp(S - m_new) and its row sum */
    float psum = 0.0f;
    for (int kk = 0; kk < bkv; ++kk) {
      float p = 0.0f;
      if (valid[kk]) { volatile float d = ub[kk] - m_new; p = exp2_cr(d); }
      pt[kk] = p;
      psum += p;
    }
    /* per-token scale of P~ from the reused maxima: s_P = exp(rowmax(S) - m)/127 */
    float sP, r;
    if (stat) { sP = 1.0f / 127.0f; r = 127.0f; }
    else { volatile float d = t - m_new; volatile float q = exp2_cr(d) / 127.0f; sP = q; volatile float rr = 1.0f / sP; r = rr; }
    if (!stat && sP < 0x1p-126f) { sP = 0.0f; r = 0.0f; }   /* the tile adds nothing to O */
    /* P^ = P~/s_P */
    for (int kk = 0; kk < bkv; ++kk) {
      volatile float y = pt[kk] * r;
      code[kk] = ident ? y : (float)i8_pcode(y);
    }
    if ((J->flags & ORC_I8_FUSED_P) && !stat && !ident && sP > 0.0f) {
      volatile float B = log127 - t;
      float ys = 0.0f;
      for (int kk = 0; kk < bkv; ++kk) {
        const float y = valid[kk] ? exp2_cr(fmaf(accf[kk], ct, B)) : 0.0f;
        ys += y;
        code[kk] = (float)i8_pcode(y);
      }
      volatile float rs = sP * ys;
      psum = rs;
    }
    volatile float al = alpha * l;
    l = al + psum;
    const float sV = ident ? 1.0f : h->vs[j];
    volatile float spv = sP * sV;
    tol = (double)alpha * tol;
    tolcont = (double)alpha * tolcont;
    if (!ident && tol_out) {
      if (!stat) {
        /* values the fused order reaches: 127 2^{acc c_t - t} within W */
        volatile float B = log127 - t;
        const double wfix = i8_hulp(log127) + i8_hulp(t) + i8_hulp(B) + 0x1p-22 / log(2.0);
        double cont = 0.0;
        for (int kk = 0; kk < bkv; ++kk) {
          if (!valid[kk]) continue;
          const double y = (double)pt[kk] * (double)r;
          const double pex = 127.0 * exp2((double)accf[kk] * (double)ct - (double)t);
          const double W = wfix + i8_hulp(fmaf(accf[kk], ct, B));
          double flo = pex * exp2(-W), fhi = pex * exp2(W);
          if (fhi < 0x1p-120) { flo = 0.0; fhi += 0x1p-147; }
          const double lo = flo < y ? flo : y, hi = fhi > y ? fhi : y;
          cont += hi - lo;
          const double c0 = code[kk], d1 = fabs(i8_pcode(lo) - c0), d2 = fabs(i8_pcode(hi) - c0);
          const double dv = d1 > d2 ? d1 : d2;
          if (dv > 0.0) { cnt[0]++; tol += dv * (double)spv * h->vrow_max[k0 + kk]; }
        }
        tolcont += (double)sP * cont;
        if (sP == 0.0f) tolcont += (double)bkv * 0x1p-110;
      } else {
        for (int kk = 0; kk < bkv; ++kk) {
          if (!valid[kk]) continue;
          const double y = (double)pt[kk] * 127.0;
          const double mid = floor(y) + 0.5;
          if (fabs(y - mid) <= mid * 0x1p-20) { cnt[0]++; tol += (double)spv * h->vrow_max[k0 + kk]; }
        }
      }
      tolcont += (double)psum * 0x1p-20;
    }
    /* O = diag(alpha) O + MM(P^, V^) s_P s_V */
    for (int c = 0; c < D; ++c) {
      float pv;
      if (ident) {
        double a = 0.0;
        for (int kk = 0; kk < bkv; ++kk) if (valid[kk]) a += (double)code[kk] * (double)h->vf[(long)(k0 + kk) * D + c];
        pv = (float)a;
      } else {
        long a = 0;
        for (int kk = 0; kk < bkv; ++kk) if (valid[kk]) a += (long)code[kk] * h->vc[(long)(k0 + kk) * D + c];
        pv = (float)a;                       /* exact: |a| <= 127^2 B_kv < 2^24 */
      }
      volatile float aO = alpha * O[c];
      O[c] = fmaf(pv, spv, aO);
    }
    m = m_new;
  }
  for (int c = 0; c < D; ++c) { volatile float o = O[c] / l; out[c] = o; }
  volatile float ml = m + log2_cr(l);
  volatile float L = ml * (float)log(2.0);
  *lse = L;
  if (tol_out) *tol_out = (float)((tol + h->vabs_max * tolcont) / (double)l);
  free(accf); free(ub); free(pt); free(code); free(valid); free(O);
}

static void* i8_worker(void* arg) {
  i8job_t* J = (i8job_t*)arg;
  int64_t cnt[2] = {0, 0};
  for (;;) {
    pthread_mutex_lock(&J->mu);
    int64_t r = J->next++;
    pthread_mutex_unlock(&J->mu);
    if (r >= J->nrows) break;
    const int64_t flat = J->rows[r];
    i8_row(J, (long)(flat / J->N), (int)(flat % J->N), J->out + r * J->D, J->lse + r,
           J->tie_tol ? J->tie_tol + r : NULL, cnt);
  }
  pthread_mutex_lock(&J->mu);
  J->cnt[0] += cnt[0]; J->cnt[1] += cnt[1];
  pthread_mutex_unlock(&J->mu);
  return NULL;
}

/* ------------------------------------------------------------------------ */
/* orc_attn_int8: Algorithm 2 for a list of query rows.                      */
/*  q, k, v : 16-bit [B,H,N,D] host arrays                                   */
/*  bq, bkv : the query block of psi(Q) and the KV tile (block of psi(K),     */
/*            psi(V) and of the online softmax)                              */
/*  rows    : flat row ids ((b*H + h)*N + i)                                 */
/*  out [nrows][D], lse [nrows]; tie_tol [nrows] or NULL; counters [2] or    */
/*  NULL (tie-ambiguous P codes, skipped tiles).  Returns 0, or -1.          */
/* ------------------------------------------------------------------------ */
int orc_attn_int8(const uint16_t* q, const uint16_t* k, const uint16_t* v, int in_dtype, int B, int H, int N, int D,
                  int causal, int bq, int bkv, unsigned flags, const int64_t* rows, int64_t nrows, float* out,
                  float* lse, float* tie_tol, int64_t* counters, int nthreads) {
  if (B <= 0 || H <= 0 || N <= 0 || D <= 0 || D > 128 || bq <= 0 || bkv <= 0 || bkv > 1024) return -1;
  i8job_t J;
  memset(&J, 0, sizeof(J));
  J.q = q; J.k = k; J.v = v; J.in_dtype = in_dtype; J.B = B; J.H = H; J.N = N; J.D = D; J.causal = causal;
  J.bq = bq; J.bkv = bkv; J.flags = flags; J.rows = rows; J.nrows = nrows; J.out = out; J.lse = lse;
  J.tie_tol = tie_tol;
  J.heads = (i8head_t*)calloc((size_t)B * H, sizeof(i8head_t));
  char* used = (char*)calloc((size_t)B * H, 1);
  for (int64_t r = 0; r < nrows; ++r) {
    if (rows[r] < 0 || rows[r] >= (int64_t)B * H * N) { free(J.heads); free(used); return -1; }
    used[rows[r] / N] = 1;
  }
  for (long bh = 0; bh < (long)B * H; ++bh) if (used[bh]) i8_build_head(&J, bh);
  pthread_mutex_init(&J.mu, NULL);
  if (nthreads < 1) nthreads = 1;
  pthread_t* th = (pthread_t*)malloc(sizeof(pthread_t) * (size_t)nthreads);
  for (int t = 0; t < nthreads; ++t) pthread_create(&th[t], NULL, i8_worker, &J);
  for (int t = 0; t < nthreads; ++t) pthread_join(th[t], NULL);
  free(th);
  pthread_mutex_destroy(&J.mu);
  if (counters) { counters[0] = J.cnt[0]; counters[1] = J.cnt[1]; }
  for (long bh = 0; bh < (long)B * H; ++bh) if (used[bh]) i8_free_head(&J.heads[bh]);
  free(J.heads); free(used);
  return 0;
}

/* ======================================================================== */
/* Backward pass of the 8-bit attention (Algorithm 3).                      */
/*                                                                          */
/* Readings (the kernels implement the same):                               */
/*  - inputs: Q, K, V, dO 16-bit, O fp32 and L fp32 from the forward; Q^,   */
/*    K^ (and K_m) are psi of the forward's blocks (B_q = 128 rows of Q,    */
/*    B_kv rows of K' = fl32(K - K_m)); V enters only dP = MM(dO, V^T),     */
/*    which stays in 16-bit inputs with fp32 accumulation ("keep in FP16"): */
/*    dP = fl32 of the exact dot product.                                   */
/*  - D_q = fl32(sum_d dO[q,d] O[q,d]) (exact sum, rounded once).           */
/*  - scores as in the forward: u = fl32(fl32(acc) c_t) in the log2 domain; */
/*    P = exp(S/sqrt(D) - L) in Algorithm 3's order: fl32(exp2(fl32(u -    */
/*    Lb))), Lb = fl32(L fl32(log2 e)); masked entries have P = 0.  A GPU   */
/*    may fuse it as exp2(fma(fl32(acc), c_t, -Lb)) (flag ORC_I8_FUSED_BWD  */
/*    evaluates that order); the two differ by at most a relative          */
/*    e_P = ln 2 (h(u) + h(u - Lb) + h(fused argument)) + 2^-22 (h = half  */
/*    an fp32 ulp of each rounded intermediate; the last term the two exp2 */
/*    evaluations, one correctly rounded, one within 1 ulp).                */
/*  - psi of P, dO and dS per (B_q x B_kv) block, (B_q x D) block and      */
/*    (B_q x B_kv) block, as psi of the forward (s = fl32(max|x|/127),      */
/*    codes rint(fl32(x fl32(1/s)))).  A block with no visible entry is     */
/*    skipped.                                                              */
/*  - dS = fl32(P fl32(dP - D)); the softmax scale enters dQ and dK: with   */
/*    rsd = fl32(1/sqrt(D)),                                                */
/*      dV_j = fma(fl32(MM(P^T, dO^)), fl32(s_P s_dO), dV_j)                */
/*      dK_j = fma(fl32(MM(dS^T, Q^)), fl32(fl32(s_dS s_Q) rsd), dK_j)      */
/*      dQ_i = fma(fl32(MM(dS^, K^)), fl32(fl32(s_dS s_K) rsd), dQ_i)       */
/*             then + fl32(fl32(rowsum(dS) rsd) K_m) (smoothing K; the     */
/*             rowsum sequential in fp32 over the block's keys),            */
/*    accumulated in the order of Algorithm 3 (KV block j outer, query      */
/*    block i inner).                                                       */
/*  - tolerance: a code of P^ or dS^ whose pre-rounding value lies within a */
/*    window of a rounding midpoint may take either neighbour on a GPU      */
/*    (exp2 to 1 ulp; dP and D summed in another order); each such code     */
/*    adds the size of its effect to the per-element tolerance of dV, dK,   */
/*    dQ.  The window: for P^ a relative e_P of the value plus the block's */
/*    largest e_P (it bounds the move of s_P) plus 8 ulp; for dS^ the bound */
/*    |P| (e_dP + e_D) + |dP - D| |P| (2^-21 + e_P) (e_x = 2^-17 times the  */
/*    sum of |terms| of x) over s_dS, plus 8 ulp; block scales that move by */
/*    an ulp shift every code by a relative 2^-22, also inside it.  The     */
/*    move of s_P reaches dV continuously, and the                          */
/*    same dS error reaches dQ and dK continuously -- through s_dS          */
/*    (its bound is the largest element bound over 127: every code's value */
/*    and the fold factor move with it) and through rowsum(dS) in the       */
/*    smoothing-K term -- and is added to their tolerance.                  */
/* Flags: ORC_NO_SMOOTH_K, ORC_I8_IDENTITY (no psi anywhere: the exact      */
/* gradients of softmax attention up to fp32 rounding), ORC_I8_DP_INT8      */
/* (ablation, Table 1(c): dP = MM(dO^, V^) with per-block INT8 dO and V),    */
/* ORC_I8_FUSED_BWD (P in the fused order, for the test that bounds it).     */
/* ======================================================================== */
#define ORC_I8_DP_INT8 128u
#define ORC_I8_FUSED_BWD 1024u

typedef struct {
  const uint16_t *q, *k, *v, *dout;
  const float *o, *lse;
  int in_dtype, B, H, N, D, causal, bq, bkv;
  unsigned flags;
  float *dq, *dk, *dv, *tq, *tk, *tv;
  long next;
  pthread_mutex_t mu;
} i8bwd_t;

static double mid_dist(float y) {
  /* distance of |y| to the nearest rounding midpoint k + 1/2 */
  double a = fabs((double)y);
  return fabs(a - (floor(a) + 0.5));
}

static void i8_bwd_head(i8bwd_t* J, long bh) {
  const int N = J->N, D = J->D, bq = J->bq, bkv = J->bkv;
  const long ND = (long)N * D;
  const int ident = (J->flags & ORC_I8_IDENTITY) != 0, smooth = !(J->flags & ORC_NO_SMOOTH_K);
  const int dp8 = (J->flags & ORC_I8_DP_INT8) != 0;
  const uint16_t *qb = J->q + bh * ND, *kb = J->k + bh * ND, *vb = J->v + bh * ND, *gb = J->dout + bh * ND;
  const float *ob = J->o + bh * ND, *lb = J->lse + bh * (long)N;
  float *dq = J->dq + bh * ND, *dk = J->dk + bh * ND, *dv = J->dv + bh * ND;
  float *tq = J->tq ? J->tq + bh * ND : NULL, *tk = J->tk ? J->tk + bh * ND : NULL, *tv = J->tv ? J->tv + bh * ND : NULL;
  const int nqb = (N + bq - 1) / bq, nkb = (N + bkv - 1) / bkv;
  const float c2 = (float)(1.0 / (log(2.0) * sqrt((double)D)));
  const float rsd = (float)(1.0 / sqrt((double)D));
  const float log2e = (float)(1.0 / log(2.0));

  float* mu = (float*)calloc(D, sizeof(float));
  int8_t *qc = (int8_t*)calloc(ND, 1), *kc = (int8_t*)calloc(ND, 1), *gc = (int8_t*)calloc(ND, 1);
  int8_t *vc8 = (int8_t*)calloc(ND, 1);
  float *qs = (float*)calloc(nqb, sizeof(float)), *ks = (float*)calloc(nkb, sizeof(float));
  float *gs = (float*)calloc(nqb, sizeof(float)), *vs8 = (float*)calloc(nkb, sizeof(float));
  float *qf = (float*)malloc(sizeof(float) * ND), *kf = (float*)malloc(sizeof(float) * ND);
  float *vf = (float*)malloc(sizeof(float) * ND), *gf = (float*)malloc(sizeof(float) * ND);
  if (smooth) orc_kmean(kb, J->in_dtype, 1, 1, N, D, mu);
  for (long e = 0; e < ND; ++e) {
    qf[e] = orc_widen(qb[e], J->in_dtype);
    float kv = orc_widen(kb[e], J->in_dtype);
    if (smooth) { volatile float d = kv - mu[e % D]; kv = d; }
    kf[e] = kv;
    vf[e] = orc_widen(vb[e], J->in_dtype);
    gf[e] = orc_widen(gb[e], J->in_dtype);
  }
  if (!ident) {
    orc_quant_int8(qb, J->in_dtype, ORC_ROLE_Q, 1, 1, N, D, bq, 0, qc, qs, NULL);
    float* mu2 = (float*)calloc(D, sizeof(float));
    orc_quant_int8(kb, J->in_dtype, ORC_ROLE_K, 1, 1, N, D, bkv, smooth, kc, ks, mu2);
    free(mu2);
    orc_quant_int8(gb, J->in_dtype, ORC_ROLE_Q, 1, 1, N, D, bq, 0, gc, gs, NULL);
    if (dp8) orc_quant_int8(vb, J->in_dtype, ORC_ROLE_V, 1, 1, N, D, bkv, 0, vc8, vs8, NULL);
  }
  /* D_q and Lb_q */
  float* Dr = (float*)malloc(sizeof(float) * N);
  float* Lb = (float*)malloc(sizeof(float) * N);
  double* Dabs = (double*)malloc(sizeof(double) * N);
  for (int q = 0; q < N; ++q) {
    double s = 0.0, a = 0.0;
    for (int c = 0; c < D; ++c) { double t = (double)gf[(long)q * D + c] * (double)ob[(long)q * D + c]; s += t; a += fabs(t); }
    Dr[q] = (float)s; Dabs[q] = a;
    volatile float l2 = lb[q] * log2e;
    Lb[q] = l2;
  }
  memset(dq, 0, sizeof(float) * ND); memset(dk, 0, sizeof(float) * ND); memset(dv, 0, sizeof(float) * ND);
  if (tq) { memset(tq, 0, sizeof(float) * ND); memset(tk, 0, sizeof(float) * ND); memset(tv, 0, sizeof(float) * ND); }

  float* P = (float*)malloc(sizeof(float) * (size_t)bq * bkv);
  float* dS = (float*)malloc(sizeof(float) * (size_t)bq * bkv);
  float* Pc = (float*)malloc(sizeof(float) * (size_t)bq * bkv);     /* P^ (identity: P)  */
  float* Sc = (float*)malloc(sizeof(float) * (size_t)bq * bkv);     /* dS^ (identity: dS) */
  double* win = (double*)malloc(sizeof(double) * (size_t)bq * bkv);
  double* eP = (double*)calloc((size_t)bq * bkv, sizeof(double));     /* relative window of P */
  char* vis = (char*)malloc((size_t)bq * bkv);
  double* acc = (double*)malloc(sizeof(double) * (size_t)(bq > bkv ? bq : bkv) * D);

  for (int j = 0; j < nkb; ++j) {
    const int k0 = j * bkv, k1 = (k0 + bkv < N) ? k0 + bkv : N, nk = k1 - k0;
    for (int i = 0; i < nqb; ++i) {
      const int q0 = i * bq, q1 = (q0 + bq < N) ? q0 + bq : N, nq = q1 - q0;
      int any = 0;
      memset(vis, 0, (size_t)bq * bkv);
      memset(P, 0, sizeof(float) * (size_t)bq * bkv);
      memset(dS, 0, sizeof(float) * (size_t)bq * bkv);
      for (int a = 0; a < nq; ++a)
        for (int b = 0; b < nk; ++b) {
          const int vv = !(J->causal && k0 + b > q0 + a);
          vis[a * bkv + b] = (char)vv;
          any |= vv;
        }
      if (!any) continue;
      const float sQ = ident ? 1.0f : qs[i], sK = ident ? 1.0f : ks[j];
      volatile float sqk = sQ * sK;
      volatile float ct = sqk * c2;
      /* P = exp(S - L) and dS = P (dP - D) */
      float pmax = 0.0f;
      double ePmax = 0.0;                     /* largest relative window of P in the block */
      for (int a = 0; a < nq; ++a)
        for (int b = 0; b < nk; ++b) {
          const int q = q0 + a, k = k0 + b, e = a * bkv + b;
          if (!vis[e]) { P[e] = 0.0f; dS[e] = 0.0f; continue; }
          float accf;
          if (ident) {
            double s = 0.0;
            for (int c = 0; c < D; ++c) s += (double)qf[(long)q * D + c] * (double)kf[(long)k * D + c];
            accf = (float)s;
          } else {
            long s = 0;
            for (int c = 0; c < D; ++c) s += (long)qc[(long)q * D + c] * kc[(long)k * D + c];
            accf = (float)s;
          }
          volatile float u = accf * ct;
          volatile float d = u - Lb[q];
          P[e] = (J->flags & ORC_I8_FUSED_BWD) ? exp2_cr(fmaf(accf, ct, -Lb[q])) : exp2_cr(d);
          eP[e] = log(2.0) * (i8_hulp(u) + i8_hulp(d) + i8_hulp(fmaf(accf, ct, -Lb[q]))) + 0x1p-22;
          if (P[e] > pmax) pmax = P[e];
          if (eP[e] > ePmax) ePmax = eP[e];     /* bounds the move of the block max */
        }
      float dsmax = 0.0f;
      for (int a = 0; a < nq; ++a)
        for (int b = 0; b < nk; ++b) {
          const int q = q0 + a, k = k0 + b, e = a * bkv + b;
          win[e] = 0.0;
          if (!vis[e]) continue;
          double s = 0.0, sa = 0.0;
          if (dp8) {
            long si = 0;
            for (int c = 0; c < D; ++c) si += (long)gc[(long)q * D + c] * vc8[(long)k * D + c];
            s = (double)(float)si * (double)(float)(gs[i] * vs8[j]);
            sa = fabs(s);
          } else {
            for (int c = 0; c < D; ++c) { double t = (double)gf[(long)q * D + c] * (double)vf[(long)k * D + c]; s += t; sa += fabs(t); }
          }
          const float dP = (float)s;
          volatile float d = dP - Dr[q];
          volatile float ds = P[e] * d;
          dS[e] = ds;
          if (fabsf(ds) > dsmax) dsmax = fabsf(ds);
          /* error window of dS from the GPU's other summation orders and exp2 */
          win[e] = fabs((double)P[e]) * (ldexp(sa, -17) + ldexp(Dabs[q], -17)) +
                   fabs((double)d) * fabs((double)P[e]) * (ldexp(1.0, -21) + eP[e]);
        }
      /* psi(P) over the block, psi(dS) over the block */
      float sP = 1.0f, sdS = 1.0f;
      double es = 0.0;                        /* bound on the move of s_dS */
      for (int e = 0; e < bq * bkv; ++e) if (win[e] > es) es = win[e];
      es /= 127.0;
      if (!ident) {
        volatile float s1 = pmax / 127.0f; sP = s1;
        volatile float r1 = pmax > 0.0f ? 1.0f / sP : 0.0f;
        volatile float s2 = dsmax / 127.0f; sdS = s2;
        volatile float r2 = dsmax > 0.0f ? 1.0f / sdS : 0.0f;
        for (int e = 0; e < bq * bkv; ++e) {
          volatile float y1 = P[e] * r1;
          volatile float y2 = dS[e] * r2;
          Pc[e] = rintf(y1);
          Sc[e] = rintf(y2);
          if (tq) {
            /* flag codes near a midpoint; the effect goes into the tolerance */
            const double w1 = fabs((double)y1) * (eP[e] + ePmax + ldexp(1.0, -20)) + ldexp(1.0, -20);
            const double w2 = win[e] * (double)r2 + fabs((double)y2) * (es * (double)r2 + ldexp(1.0, -20)) +
                              ldexp(1.0, -20);
            const int a = e / bkv, b = e % bkv;
            if (vis[e] && a < nq && b < nk) {
              const int q = q0 + a, k = k0 + b;
              if (mid_dist(y1) <= w1) {
                const double f = (double)sP * gs[i];
                for (int c = 0; c < D; ++c) tv[(long)k * D + c] += (float)(f * abs(gc[(long)q * D + c]));
              }
              if (mid_dist(y2) <= w2) {
                const double fk = (double)sdS * qs[i] * rsd, fq = (double)sdS * ks[j] * rsd;
                for (int c = 0; c < D; ++c) {
                  tk[(long)k * D + c] += (float)(fk * abs(qc[(long)q * D + c]));
                  tq[(long)q * D + c] += (float)(fq * abs(kc[(long)k * D + c]));
                }
              }
            }
          }
        }
      } else {
        for (int e = 0; e < bq * bkv; ++e) { Pc[e] = P[e]; Sc[e] = dS[e]; }
      }
      /* dV_j += MM(P^T, dO^) s_P s_dO */
      {
        volatile float f = sP * (ident ? 1.0f : gs[i]);
        for (int b = 0; b < nk; ++b)
          for (int c = 0; c < D; ++c) {
            double s = 0.0;
            for (int a = 0; a < nq; ++a)
              s += (double)Pc[a * bkv + b] * (ident ? (double)gf[(long)(q0 + a) * D + c] : (double)gc[(long)(q0 + a) * D + c]);
            const long o = (long)(k0 + b) * D + c;
            dv[o] = fmaf((float)s, f, dv[o]);
            /* s_P moves with the block max by at most ePmax (relative) */
            if (tv && !ident) tv[o] += (float)(fabs(s) * (double)f * ePmax);
          }
      }
      /* dK_j += MM(dS^T, Q^) s_dS s_Q / sqrt(D) */
      {
        volatile float f0 = sdS * sQ;
        volatile float f = f0 * rsd;
        for (int b = 0; b < nk; ++b)
          for (int c = 0; c < D; ++c) {
            double s = 0.0;
            for (int a = 0; a < nq; ++a)
              s += (double)Sc[a * bkv + b] * (ident ? (double)qf[(long)(q0 + a) * D + c] : (double)qc[(long)(q0 + a) * D + c]);
            const long o = (long)(k0 + b) * D + c;
            dk[o] = fmaf((float)s, f, dk[o]);
            if (tk && !ident) tk[o] += (float)(fabs(s) * es * sQ * rsd);
          }
      }
      /* dQ_i += MM(dS^, K^) s_dS s_K / sqrt(D) + rowsum(dS) K_m / sqrt(D) */
      {
        volatile float f0 = sdS * sK;
        volatile float f = f0 * rsd;
        for (int a = 0; a < nq; ++a) {
          float rs = 0.0f;
          double rse = 0.0;                   /* bound on the error of rowsum(dS) */
          for (int b = 0; b < nk; ++b) { rs += dS[a * bkv + b]; rse += win[a * bkv + b]; }
          volatile float rr = rs * rsd;
          for (int c = 0; c < D; ++c) {
            double s = 0.0;
            for (int b = 0; b < nk; ++b)
              s += (double)Sc[a * bkv + b] * (ident ? (double)kf[(long)(k0 + b) * D + c] : (double)kc[(long)(k0 + b) * D + c]);
            const long o = (long)(q0 + a) * D + c;
            float x = fmaf((float)s, f, dq[o]);
            if (smooth) x = fmaf(rr, mu[c], x);
            dq[o] = x;
            if (tq && !ident)
              tq[o] += (float)(fabs(s) * es * sK * rsd + (smooth ? rse * rsd * fabs((double)mu[c]) : 0.0));
          }
        }
      }
    }
  }
  free(mu); free(qc); free(kc); free(gc); free(vc8); free(qs); free(ks); free(gs); free(vs8);
  free(qf); free(kf); free(vf); free(gf); free(Dr); free(Lb); free(Dabs);
  free(P); free(dS); free(Pc); free(Sc); free(win); free(eP); free(vis); free(acc);
}

static void* i8_bwd_worker(void* arg) {
  i8bwd_t* J = (i8bwd_t*)arg;
  for (;;) {
    pthread_mutex_lock(&J->mu);
    long bh = J->next++;
    pthread_mutex_unlock(&J->mu);
    if (bh >= (long)J->B * J->H) break;
    i8_bwd_head(J, bh);
  }
  return NULL;
}

/* ------------------------------------------------------------------------ */
/* orc_attn_int8_bwd: Algorithm 3 for every head.                            */
/*  q, k, v, dout: 16-bit [B,H,N,D]; o fp32 [B,H,N,D]; lse fp32 [B,H,N]     */
/*  dq, dk, dv: fp32 [B,H,N,D] outputs; tq, tk, tv: per-element tolerances  */
/*  (same shape) or all NULL.  Returns 0, or -1 for invalid arguments.      */
/* ------------------------------------------------------------------------ */
int orc_attn_int8_bwd(const uint16_t* q, const uint16_t* k, const uint16_t* v, const uint16_t* dout,
                      const float* o, const float* lse, int in_dtype, int B, int H, int N, int D, int causal,
                      int bq, int bkv, unsigned flags, float* dq, float* dk, float* dv, float* tq, float* tk,
                      float* tv, int nthreads) {
  if (B <= 0 || H <= 0 || N <= 0 || D <= 0 || D > 128 || bq <= 0 || bkv <= 0) return -1;
  if ((tq == NULL) != (tk == NULL) || (tq == NULL) != (tv == NULL)) return -1;
  i8bwd_t J;
  memset(&J, 0, sizeof(J));
  J.q = q; J.k = k; J.v = v; J.dout = dout; J.o = o; J.lse = lse; J.in_dtype = in_dtype;
  J.B = B; J.H = H; J.N = N; J.D = D; J.causal = causal; J.bq = bq; J.bkv = bkv; J.flags = flags;
  J.dq = dq; J.dk = dk; J.dv = dv; J.tq = tq; J.tk = tk; J.tv = tv;
  pthread_mutex_init(&J.mu, NULL);
  if (nthreads < 1) nthreads = 1;
  pthread_t* th = (pthread_t*)malloc(sizeof(pthread_t) * (size_t)nthreads);
  for (int t = 0; t < nthreads; ++t) pthread_create(&th[t], NULL, i8_bwd_worker, &J);
  for (int t = 0; t < nthreads; ++t) pthread_join(th[t], NULL);
  free(th);
  pthread_mutex_destroy(&J.mu);
  return 0;
}
