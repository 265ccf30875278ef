/*
 * sage_oracle_int8.c -- plain, slow CPU oracle for the 8-bit attention
 * forward of SageBwd (arXiv 2505.11594, Algorithm 2).
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
 *   - P^ = P~/s_P = 127 * 2^{u - t}, evaluated as
 *     exp2(fma(fl32(acc), c_t, fl32(log2 127 - t))) and rounded to the
 *     nearest integer (ties to even); s_P = fl32(2^{t - m}/127).
 *   - l accumulates the unquantized P~ as Algorithm 2 writes it:
 *     l = fl32(fl32(alpha l) + fl32(s_P sum_k P~_k/s_P)), the sum sequential
 *     in fp32; alpha = 2^{m_old - m_new}, 0 on the first visited tile (the
 *     running max starts at -inf).
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
 * tiling, the online softmax and L against textbook attention).
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

#define ORC_ROLE_Q 0
#define ORC_ROLE_K 1
#define ORC_ROLE_V 2

#define I8_TIE_REL (1.0 / 1048576.0) /* 8 ulp of fp32, as for the FP4 codes of P */

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
  double vabs_max;            /* identity mode: max |V|                     */
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
  for (int k = 0; k < N; ++k) {
    int m = 0;
    for (int c = 0; c < D; ++c) { int a = abs(h->vc[(long)k * D + c]); if (a > m) m = a; }
    h->vrow_max[k] = m;
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

/* One query row of Algorithm 2. */
static void i8_row(i8job_t* J, long bh, int i, float* out, float* lse, float* tol_out, int64_t* cnt) {
  const i8head_t* h = &J->heads[bh];
  const int N = J->N, D = J->D, bkv = J->bkv;
  const int ident = (J->flags & ORC_I8_IDENTITY) != 0, stat = (J->flags & ORC_I8_STATIC_P) != 0;
  const float c2 = (float)(1.0 / (log(2.0) * sqrt((double)D)));
  const float log127 = (float)log2(127.0);
  const float sQ = ident ? 1.0f : h->qs[i / J->bq];
  float* accf = (float*)malloc(sizeof(float) * bkv);
  float* code = (float*)malloc(sizeof(float) * bkv);    /* P^ (identity: P~/s_P unrounded) */
  char* valid = (char*)malloc((size_t)bkv);
  char* tie = (char*)malloc((size_t)bkv);
  float* O = (float*)calloc(D, sizeof(float));
  double tol = 0.0;
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
      if (u > t) t = u;
    }
    if (t == -INFINITY) { cnt[1]++; continue; }
    const float m_new = m > t ? m : t;
    float alpha = 0.0f;
    if (m != -INFINITY) { volatile float d = m - m_new; alpha = exp2_cr(d); }
    /* per-token scale of P~ from the reused maxima: s_P = rowmax(P~)/127 */
    float sP;
    volatile float bias;
    if (stat) { sP = 1.0f / 127.0f; bias = log127 - m_new; }
    else { volatile float d = t - m_new; float rho = exp2_cr(d); volatile float q = rho / 127.0f; sP = q; bias = log127 - t; }
    float psum = 0.0f;
    for (int kk = 0; kk < bkv; ++kk) {
      tie[kk] = 0;
      if (!valid[kk]) { code[kk] = 0.0f; continue; }
      const float p = exp2_cr(fmaf(accf[kk], ct, bias));
      psum += p;
      if (ident) { code[kk] = p; continue; }
      float c = rintf(p);
      if (c > 127.0f) c = 127.0f;
      code[kk] = c;
      const double mid = floor((double)p) + 0.5;
      if (fabs((double)p - mid) <= I8_TIE_REL * mid) tie[kk] = 1;
    }
    volatile float rs = sP * psum;
    volatile float al = alpha * l;
    l = al + rs;
    const float sV = ident ? 1.0f : h->vs[j];
    volatile float spv = sP * sV;
    tol = (double)alpha * tol;
    if (!ident && tol_out)
      for (int kk = 0; kk < bkv; ++kk)
        if (tie[kk]) { cnt[0]++; tol += (double)spv * h->vrow_max[k0 + kk]; }
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
  if (tol_out) *tol_out = (float)(tol / (double)l);
  free(accf); free(code); free(valid); free(tie); free(O);
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
