/*
 * kf_oracle.c -- plain CPU oracle for the K-Forcing joint next-k-token decode.
 *
 * TEST INFRASTRUCTURE ONLY.  Only tests/, __graft_entry__.smoke() and the
 * cpu_baseline leg of bench.py may load this code.  It shares no source,
 * header, table or helper with the HIP library.
 *
 * What it computes (paper: Sec. 3.1 formulation of the push-forward LM,
 * Sec. 3.3 "fully causal" architecture, Appendix C.1 algorithm "K-Forcing
 * Inference with KV Cache"):
 *
 *   One forward pass of a pre-LayerNorm causal Transformer over a block of new
 *   rows appended to a per-sequence KV cache of committed context.  A block
 *   holds nr real-token rows followed by k noise rows.  Real row i carries a
 *   token id at absolute position C+i; noise row j carries a scalar
 *   u_j in [0,1) encoded by a sinusoid + two-layer GELU MLP (Sec. 3.3 and the
 *   model table of Appendix D) at position C+nr+j.  Attention is causal over
 *   the concatenation [cache, real rows, noise rows] (fully causal design:
 *   the j-th output sees the context and z_1..z_j only).  Outputs:
 *     - k > 0: logits of the k noise rows through the final norm and the tied
 *       head (the algorithm takes the argmax over the last k outputs);
 *     - k = 0: logits of the last real row (ordinary AR decoding).
 *   Only the real rows' K/V are appended to the cache; noise K/V are dropped
 *   (Appendix C.1, cache-commit rule).
 *
 * Compiled twice: -DREAL=double (the parity oracle) and -DREAL=float (timed
 * as the CPU baseline).  Each instantiation's symbols carry a suffix.
 *
 * Readings of points the paper leaves open (listed in the design notes):
 *   - backbone: LayerNorm (eps 1e-5, affine) pre-norm, learned absolute
 *     positions added at the embedding, GELU in tanh form, tied head, no head
 *     bias, final norm before the head;
 *   - noise row j sits at the position of the token it emits;
 *   - sinusoid of u: a_i = 1000 * u * 10000^(-i/(d/2)), e = [cos a, sin a];
 *   - noise MLP: Linear(d -> 4d), GELU, Linear(4d -> d); no token embedding
 *     on noise rows;
 *   - weights: 2-D tensors are rounded to bf16 (round-to-nearest-even) for
 *     bf16 models, 1-D tensors stay as given;
 *   - the paper's own backbone (Appendix D model table: RMSNorm pre-norm,
 *     RoPE with d_rot = 64), for blobs whose header word 9 has bit 1 set:
 *     every norm is RMSNorm x / sqrt(mean(x^2) + 1e-5) * g (the shift
 *     tensors are ignored), there are no learned positions (the position
 *     table is ignored), and q and k of every row are rotated at the row's
 *     position p by RoFormer's rotary map on the first d_rot = min(64, d_head)
 *     dimensions of each head: pairs (2i, 2i+1) turned by p * 10000^(-2i/d_rot);
 *   - temperature conditioning (Sec. 3.3 "Temperature-controlled generation",
 *     Appendix C.2 "Temperature control at inference"): a model whose blob
 *     carries the temperature encoder maps each sequence's tau through the
 *     same sinusoid and Linear(d -> d), GELU, Linear(d -> d), and adds the
 *     result to every noise row of that sequence.  With the noise MLP this
 *     gives the encoder 10 d^2 + 7 d parameters (5.9 M at d = 768, the size
 *     the paper's model table lists for the noise encoder).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#ifndef REAL
#define REAL double
#endif
#ifndef SFX
#define SFX _f64
#endif
#define CAT2(a, b) a##b
#define CAT(a, b) CAT2(a, b)
#define SYM(name) CAT(name, SFX)

#define ORC_MAGIC 0x4B465731
#define ORC_HDR 16
#define ORC_FLAG_TEMPERATURE 1 /* header word 9 */
#define ORC_FLAG_RMS_ROPE 2    /* header word 9: RMSNorm + rotary positions */

typedef struct {
  REAL *ln1_g, *ln1_b, *wqkv, *bqkv, *wo, *bo, *ln2_g, *ln2_b, *w1, *b1, *w2, *b2;
} orc_layer;

typedef struct {
  int L, d, H, f, V, T, dtype, temp, rope;
  REAL *tok, *pos, *nw1, *nb1, *nw2, *nb2, *lnf_g, *lnf_b;
  REAL *tw1, *tb1, *tw2, *tb2; /* temperature encoder (temp != 0) */
  orc_layer *layer;
  REAL *store;
} orc_model;

typedef struct {
  const orc_model *m;
  int C;        /* committed context length */
  REAL *K, *Vc; /* [L][T][d] committed keys / values */
  REAL *temb;   /* [d] temperature embedding added to noise rows, or NULL */
} orc_seq;

/* ---------------------------------------------------------------- helpers */

/* bf16 round-to-nearest-even of an fp32 value (NaN is not expected here). */
static float round_bf16(float x) {
  uint32_t u;
  memcpy(&u, &x, 4);
  uint32_t lsb = (u >> 16) & 1u;
  u = (u + 0x7FFFu + lsb) & 0xFFFF0000u;
  float y;
  memcpy(&y, &u, 4);
  return y;
}

/* y[o] = b[o] + sum_i W[o][i] x[i]   (W stored [out][in]) */
static void linear(const REAL *x, const REAL *W, const REAL *b, int in, int out, REAL *y) {
  for (int o = 0; o < out; ++o) {
    const REAL *w = W + (size_t)o * in;
    REAL s = 0;
    for (int i = 0; i < in; ++i) s += w[i] * x[i];
    y[o] = (b ? b[o] : (REAL)0) + s;
  }
}

/* LayerNorm: (x - mean) / sqrt(var + 1e-5) * g + b, biased variance. */
static void layernorm(const REAL *x, const REAL *g, const REAL *b, int d, REAL *y) {
  REAL mean = 0;
  for (int i = 0; i < d; ++i) mean += x[i];
  mean /= d;
  REAL var = 0;
  for (int i = 0; i < d; ++i) var += (x[i] - mean) * (x[i] - mean);
  var /= d;
  REAL r = (REAL)1 / (REAL)sqrt((double)(var + (REAL)1e-5));
  for (int i = 0; i < d; ++i) y[i] = (x[i] - mean) * r * g[i] + b[i];
}

/* RMSNorm: x / sqrt(mean(x^2) + 1e-5) * g. */
static void rmsnorm(const REAL *x, const REAL *g, int d, REAL *y) {
  REAL ms = 0;
  for (int i = 0; i < d; ++i) ms += x[i] * x[i];
  ms /= d;
  REAL r = (REAL)1 / (REAL)sqrt((double)(ms + (REAL)1e-5));
  for (int i = 0; i < d; ++i) y[i] = x[i] * r * g[i];
}

/* The model's pre-norm: LayerNorm, or RMSNorm for the rotary backbone. */
static void norm(const orc_model *m, const REAL *x, const REAL *g, const REAL *b, REAL *y) {
  if (m->rope) rmsnorm(x, g, m->d, y);
  else layernorm(x, g, b, m->d, y);
}

/* Rotary positions (RoFormer): in each head of x [H][dh], the pairs
 * (2i, 2i+1), i < d_rot/2, turned by the angle p * 10000^(-2i/d_rot). */
static void rope(REAL *x, int H, int dh, int p) {
  const int dr = dh < 64 ? dh : 64;
  for (int h = 0; h < H; ++h)
    for (int i = 0; i < dr / 2; ++i) {
      const double a = (double)p * pow(10000.0, -2.0 * i / (double)dr);
      const double c = cos(a), sn = sin(a);
      REAL *e = x + (size_t)h * dh + 2 * i;
      const double x0 = (double)e[0], x1 = (double)e[1];
      e[0] = (REAL)(x0 * c - x1 * sn);
      e[1] = (REAL)(x0 * sn + x1 * c);
    }
}

/* GELU, tanh form: 0.5 x (1 + tanh(sqrt(2/pi) (x + 0.044715 x^3))). */
static REAL gelu(REAL x) {
  const double c = 0.7978845608028654; /* sqrt(2/pi) */
  double xd = (double)x;
  return (REAL)(0.5 * xd * (1.0 + tanh(c * (xd + 0.044715 * xd * xd * xd))));
}

/* Sinusoidal encoding of the scalar u into d features: cos half, then sin half. */
static void sinusoid(double u, int d, REAL *e) {
  int h = d / 2;
  for (int i = 0; i < h; ++i) {
    double w = pow(10000.0, -(double)i / (double)h);
    double a = 1000.0 * u * w;
    e[i] = (REAL)cos(a);
    e[i + h] = (REAL)sin(a);
  }
}

/*
 * One attention head for one query: scores q.k_t * scale over the nk visible
 * keys, softmax with the maximum subtracted, weighted sum of the values.
 * Keys and values are given by pointer so that committed cache rows and the
 * block's new rows can be visited in position order.  P is scratch of nk
 * entries.  Returns the sum of the normalised weights.
 */
static REAL attend(const REAL *q, const REAL *const *kp, const REAL *const *vp, int nk, int dh,
                   REAL scale, REAL *P, REAL *o) {
  REAL mx = -INFINITY;
  for (int t = 0; t < nk; ++t) {
    REAL sc = 0;
    for (int e = 0; e < dh; ++e) sc += q[e] * kp[t][e];
    P[t] = sc * scale;
    if (P[t] > mx) mx = P[t];
  }
  REAL den = 0;
  for (int t = 0; t < nk; ++t) {
    P[t] = (REAL)exp((double)(P[t] - mx));
    den += P[t];
  }
  REAL psum = 0;
  for (int t = 0; t < nk; ++t) {
    P[t] /= den;
    psum += P[t];
  }
  for (int e = 0; e < dh; ++e) o[e] = 0;
  for (int t = 0; t < nk; ++t)
    for (int e = 0; e < dh; ++e) o[e] += P[t] * vp[t][e];
  return psum;
}

/* ------------------------------------------------------------------ model */

static long model_params(int L, int d, int f, int V, int T) {
  long per = 2L * d + 3L * d * d + 3L * d + (long)d * d + d + 2L * d + (long)f * d + f +
             (long)d * f + d;
  return (long)V * d + (long)T * d + 4L * d * d + 4L * d + 4L * d * d + d + L * per + 2L * d;
}

static long temp_params(int d) { return 2L * d * d + 2L * d; }

long SYM(orc_blob_floats)(const int32_t *hdr) {
  if (hdr[0] != ORC_MAGIC) return -1;
  return ORC_HDR + model_params(hdr[2], hdr[3], hdr[5], hdr[6], hdr[7]) +
         ((hdr[9] & ORC_FLAG_TEMPERATURE) ? temp_params(hdr[3]) : 0);
}

/* Copy n floats into REAL storage, rounding to bf16 when asked. */
static REAL *take(REAL **cur, const float **src, long n, int to_bf16) {
  REAL *dst = *cur;
  for (long i = 0; i < n; ++i) {
    float v = (*src)[i];
    dst[i] = (REAL)(to_bf16 ? round_bf16(v) : v);
  }
  *cur += n;
  *src += n;
  return dst;
}

orc_model *SYM(orc_model_new)(const float *blob, long n_floats) {
  int32_t hdr[ORC_HDR];
  memcpy(hdr, blob, sizeof(hdr));
  if (hdr[0] != ORC_MAGIC || hdr[1] != 1) return NULL;
  int L = hdr[2], d = hdr[3], H = hdr[4], f = hdr[5], V = hdr[6], T = hdr[7], dt = hdr[8];
  if (L < 1 || d < 2 || H < 1 || d % H || d % 2 || f < 1 || V < 1 || T < 1) return NULL;
  if (hdr[9] & ~(ORC_FLAG_TEMPERATURE | ORC_FLAG_RMS_ROPE)) return NULL;
  const int temp = (hdr[9] & ORC_FLAG_TEMPERATURE) != 0;
  long np = model_params(L, d, f, V, T) + (temp ? temp_params(d) : 0);
  if (n_floats != ORC_HDR + np) return NULL;
  orc_model *m = (orc_model *)calloc(1, sizeof(orc_model));
  m->L = L; m->d = d; m->H = H; m->f = f; m->V = V; m->T = T; m->dtype = dt; m->temp = temp;
  m->rope = (hdr[9] & ORC_FLAG_RMS_ROPE) != 0;
  m->store = (REAL *)malloc(sizeof(REAL) * (size_t)np);
  m->layer = (orc_layer *)calloc((size_t)L, sizeof(orc_layer));
  REAL *cur = m->store;
  const float *src = blob + ORC_HDR;
  int mb = (dt == 1); /* matrices in bf16 */
  m->tok = take(&cur, &src, (long)V * d, mb);
  m->pos = take(&cur, &src, (long)T * d, mb);
  m->nw1 = take(&cur, &src, 4L * d * d, mb);
  m->nb1 = take(&cur, &src, 4L * d, 0);
  m->nw2 = take(&cur, &src, 4L * d * d, mb);
  m->nb2 = take(&cur, &src, d, 0);
  for (int l = 0; l < L; ++l) {
    orc_layer *y = &m->layer[l];
    y->ln1_g = take(&cur, &src, d, 0);
    y->ln1_b = take(&cur, &src, d, 0);
    y->wqkv = take(&cur, &src, 3L * d * d, mb);
    y->bqkv = take(&cur, &src, 3L * d, 0);
    y->wo = take(&cur, &src, (long)d * d, mb);
    y->bo = take(&cur, &src, d, 0);
    y->ln2_g = take(&cur, &src, d, 0);
    y->ln2_b = take(&cur, &src, d, 0);
    y->w1 = take(&cur, &src, (long)f * d, mb);
    y->b1 = take(&cur, &src, f, 0);
    y->w2 = take(&cur, &src, (long)d * f, mb);
    y->b2 = take(&cur, &src, d, 0);
  }
  m->lnf_g = take(&cur, &src, d, 0);
  m->lnf_b = take(&cur, &src, d, 0);
  if (temp) {
    m->tw1 = take(&cur, &src, (long)d * d, mb);
    m->tb1 = take(&cur, &src, d, 0);
    m->tw2 = take(&cur, &src, (long)d * d, mb);
    m->tb2 = take(&cur, &src, d, 0);
  }
  return m;
}

void SYM(orc_model_free)(orc_model *m) {
  if (!m) return;
  free(m->store);
  free(m->layer);
  free(m);
}

orc_seq *SYM(orc_seq_new)(const orc_model *m) {
  orc_seq *s = (orc_seq *)calloc(1, sizeof(orc_seq));
  s->m = m;
  s->C = 0;
  size_t n = (size_t)m->L * m->T * m->d;
  s->K = (REAL *)calloc(n, sizeof(REAL));
  s->Vc = (REAL *)calloc(n, sizeof(REAL));
  return s;
}

void SYM(orc_seq_free)(orc_seq *s) {
  if (!s) return;
  free(s->K);
  free(s->Vc);
  free(s->temb);
  free(s);
}

/* Temperature of the sequence: its embedding W_t2 GELU(W_t1 sin(tau) + b_t1) + b_t2
 * is added to every later noise row.  -1 when the model has no temperature
 * encoder. */
int SYM(orc_seq_set_temperature)(orc_seq *s, double tau) {
  const orc_model *m = s->m;
  if (!m->temp) return -1;
  const int d = m->d;
  REAL *e = (REAL *)malloc(sizeof(REAL) * (size_t)d);
  REAL *h = (REAL *)malloc(sizeof(REAL) * (size_t)d);
  if (!s->temb) s->temb = (REAL *)malloc(sizeof(REAL) * (size_t)d);
  sinusoid(tau, d, e);
  linear(e, m->tw1, m->tb1, d, d, h);
  for (int i = 0; i < d; ++i) h[i] = gelu(h[i]);
  linear(h, m->tw2, m->tb2, d, d, s->temb);
  free(e);
  free(h);
  return 0;
}

int SYM(orc_seq_len)(const orc_seq *s) { return s->C; }

/* Make dst hold src's committed context (keys, values, length, temperature
 * embedding); both sequences must belong to the same model.  Returns -1 on a
 * model mismatch. */
int SYM(orc_seq_copy)(orc_seq *dst, const orc_seq *src) {
  const orc_model *m = src->m;
  if (dst->m != m) return -1;
  size_t n = (size_t)m->L * m->T * m->d;
  memcpy(dst->K, src->K, sizeof(REAL) * n);
  memcpy(dst->Vc, src->Vc, sizeof(REAL) * n);
  dst->C = src->C;
  if (src->temb) {
    if (!dst->temb) dst->temb = (REAL *)malloc(sizeof(REAL) * (size_t)m->d);
    memcpy(dst->temb, src->temb, sizeof(REAL) * (size_t)m->d);
  } else {
    free(dst->temb);
    dst->temb = NULL;
  }
  return 0;
}

/* Copy committed K or V of layer l, positions [0, C), into out[C][d] (as double). */
void SYM(orc_seq_kv)(const orc_seq *s, int l, int which, double *out) {
  const orc_model *m = s->m;
  const REAL *src = (which ? s->Vc : s->K) + (size_t)l * m->T * m->d;
  for (long i = 0; i < (long)s->C * m->d; ++i) out[i] = (double)src[i];
}

/* ------------------------------------------------------------------- step */

/*
 * One forward pass over nr real rows (tokens toks[0..nr)) and k noise rows
 * (u[0..k)) appended to the sequence's committed cache of length C.
 *
 *   logits  : [(k > 0 ? k : 1)][V] head outputs (see file header); may be NULL
 *   hidden  : optional [nr + k][d] final residual stream of every new row
 *   commit  : when nonzero, append the real rows' K/V and advance C by nr
 *   softmax_dev : optional, receives max |sum of attention weights - 1|
 *
 * Returns the number of head rows, or -1 on a bad argument (state unchanged).
 */
int SYM(orc_step)(orc_seq *s, int nr, const int32_t *toks, int k, const double *u, int commit,
                  double *logits, double *hidden, double *softmax_dev) {
  const orc_model *m = s->m;
  const int d = m->d, H = m->H, dh = d / H, f = m->f, V = m->V, L = m->L;
  const int C = s->C, n = nr + k;
  if (nr < 0 || k < 0 || n < 1 || C + n > m->T) return -1;
  if (k == 0 && nr < 1) return -1;
  if (k > 0 && m->temp && !s->temb) return -1; /* the model needs each sequence's tau */
  for (int i = 0; i < nr; ++i)
    if (toks[i] < 0 || toks[i] >= V) return -1;

  /* Rows are independent inside each loop below (a row's dot products, norm
   * and attention read only earlier results), so the row loops run over
   * OpenMP threads; every row is computed in the same order as a serial run,
   * so the results do not depend on the thread count.  Called from inside
   * orc_step_batch's parallel region, these regions are inactive (serial). */
  REAL *X = (REAL *)malloc(sizeof(REAL) * (size_t)n * d);
  REAL *Q = (REAL *)malloc(sizeof(REAL) * (size_t)n * d);
  REAL *Kn = (REAL *)malloc(sizeof(REAL) * (size_t)L * n * d);
  REAL *Vn = (REAL *)malloc(sizeof(REAL) * (size_t)L * n * d);
  REAL *O = (REAL *)malloc(sizeof(REAL) * (size_t)n * d);
  const size_t wide = (size_t)(f > 4 * d ? f : 4 * d);
  double dev = 0;

  /* Embedding (algorithm: Embed for real rows, NoiseEnc for noise rows). */
#pragma omp parallel
  {
    REAL *A = (REAL *)malloc(sizeof(REAL) * (size_t)d);
    REAL *Y = (REAL *)malloc(sizeof(REAL) * wide);
    REAL *Z = (REAL *)malloc(sizeof(REAL) * (size_t)d);
#pragma omp for schedule(static)
    for (int r = 0; r < n; ++r) {
      REAL *x = X + (size_t)r * d;
      const REAL *pe = m->pos + (size_t)(C + r) * d;
      if (r < nr) {
        const REAL *te = m->tok + (size_t)toks[r] * d;
        for (int i = 0; i < d; ++i) x[i] = te[i] + (m->rope ? (REAL)0 : pe[i]);
      } else {
        sinusoid(u[r - nr], d, A);
        linear(A, m->nw1, m->nb1, d, 4 * d, Y);
        for (int i = 0; i < 4 * d; ++i) Y[i] = gelu(Y[i]);
        linear(Y, m->nw2, m->nb2, 4 * d, d, Z);
        for (int i = 0; i < d; ++i) x[i] = Z[i] + (m->rope ? (REAL)0 : pe[i]);
        if (s->temb)
          for (int i = 0; i < d; ++i) x[i] += s->temb[i];
      }
    }
    free(A); free(Y); free(Z);
  }

  const REAL scale = (REAL)(1.0 / sqrt((double)dh));
  for (int l = 0; l < L; ++l) {
    const orc_layer *y = &m->layer[l];
    REAL *kn = Kn + (size_t)l * n * d, *vn = Vn + (size_t)l * n * d;
    const REAL *kc = s->K + (size_t)l * m->T * d, *vc = s->Vc + (size_t)l * m->T * d;
    /* q, k, v of every new row */
#pragma omp parallel
    {
      REAL *A = (REAL *)malloc(sizeof(REAL) * (size_t)d);
      REAL *QKV = (REAL *)malloc(sizeof(REAL) * 3 * (size_t)d);
#pragma omp for schedule(static)
      for (int r = 0; r < n; ++r) {
        norm(m, X + (size_t)r * d, y->ln1_g, y->ln1_b, A);
        linear(A, y->wqkv, y->bqkv, d, 3 * d, QKV);
        if (m->rope) { /* row r sits at position C + r */
          rope(QKV, H, dh, C + r);
          rope(QKV + d, H, dh, C + r);
        }
        memcpy(Q + (size_t)r * d, QKV, sizeof(REAL) * d);
        memcpy(kn + (size_t)r * d, QKV + d, sizeof(REAL) * d);
        memcpy(vn + (size_t)r * d, QKV + 2 * d, sizeof(REAL) * d);
      }
      free(A); free(QKV);
    }
    /* causal attention: row r sees cache [0, C) then new rows [0, r] */
#pragma omp parallel
    {
      REAL *P = (REAL *)malloc(sizeof(REAL) * (size_t)(C + n));
      const REAL **kp = (const REAL **)malloc(sizeof(REAL *) * (size_t)(C + n));
      const REAL **vp = (const REAL **)malloc(sizeof(REAL *) * (size_t)(C + n));
      double tdev = 0;
#pragma omp for schedule(dynamic, 1)
      for (int rh = 0; rh < n * H; ++rh) {
        const int r = rh / H, h = rh % H;
        const int nk = C + r + 1;
        for (int t = 0; t < nk; ++t) {
          kp[t] = (t < C) ? kc + (size_t)t * d + h * dh : kn + (size_t)(t - C) * d + h * dh;
          vp[t] = (t < C) ? vc + (size_t)t * d + h * dh : vn + (size_t)(t - C) * d + h * dh;
        }
        REAL psum = attend(Q + (size_t)r * d + h * dh, kp, vp, nk, dh, scale, P, O + (size_t)r * d + h * dh);
        double dv = fabs((double)psum - 1.0);
        if (dv > tdev) tdev = dv;
      }
#pragma omp critical
      if (tdev > dev) dev = tdev;
      free(P); free(kp); free(vp);
    }
    /* attention output projection + residual, then the MLP sub-block */
#pragma omp parallel
    {
      REAL *A = (REAL *)malloc(sizeof(REAL) * (size_t)d);
      REAL *Y = (REAL *)malloc(sizeof(REAL) * wide);
      REAL *Z = (REAL *)malloc(sizeof(REAL) * (size_t)d);
#pragma omp for schedule(static)
      for (int r = 0; r < n; ++r) {
        REAL *x = X + (size_t)r * d;
        linear(O + (size_t)r * d, y->wo, y->bo, d, d, Z);
        for (int i = 0; i < d; ++i) x[i] += Z[i];
        norm(m, x, y->ln2_g, y->ln2_b, A);
        linear(A, y->w1, y->b1, d, f, Y);
        for (int i = 0; i < f; ++i) Y[i] = gelu(Y[i]);
        linear(Y, y->w2, y->b2, f, d, Z);
        for (int i = 0; i < d; ++i) x[i] += Z[i];
      }
      free(A); free(Y); free(Z);
    }
  }

  if (hidden)
    for (long i = 0; i < (long)n * d; ++i) hidden[i] = (double)X[i];

  /* head: final norm, tied token table */
  int nh = k > 0 ? k : 1;
  int r0 = k > 0 ? nr : nr - 1;
  if (logits) {
    REAL *A = (REAL *)malloc(sizeof(REAL) * (size_t)d);
    for (int j = 0; j < nh; ++j) {
      norm(m, X + (size_t)(r0 + j) * d, m->lnf_g, m->lnf_b, A);
#pragma omp parallel for schedule(static)
      for (int v = 0; v < V; ++v) {
        const REAL *w = m->tok + (size_t)v * d;
        REAL sc = 0;
        for (int i = 0; i < d; ++i) sc += w[i] * A[i];
        logits[(size_t)j * V + v] = (double)sc;
      }
    }
    free(A);
  }

  /* cache commit: keep the real rows' K/V only */
  if (commit) {
    for (int l = 0; l < L; ++l) {
      REAL *kc = s->K + (size_t)l * m->T * d, *vc = s->Vc + (size_t)l * m->T * d;
      memcpy(kc + (size_t)C * d, Kn + (size_t)l * n * d, sizeof(REAL) * (size_t)nr * d);
      memcpy(vc + (size_t)C * d, Vn + (size_t)l * n * d, sizeof(REAL) * (size_t)nr * d);
    }
    s->C = C + nr;
  }
  if (softmax_dev) *softmax_dev = dev;

  free(X); free(Q); free(Kn); free(Vn); free(O);
  return nh;
}

/* The same step over B independent sequences (OpenMP over sequences). */
int SYM(orc_step_batch)(orc_seq **seqs, int B, int nr, const int32_t *toks, int k, const double *u,
                        int commit, double *logits) {
  int err = 0;
  int nh = k > 0 ? k : 1;
  long V = B > 0 ? seqs[0]->m->V : 0;
#pragma omp parallel for schedule(dynamic, 1) reduction(| : err)
  for (int b = 0; b < B; ++b) {
    int rc = SYM(orc_step)(seqs[b], nr, toks ? toks + (size_t)b * nr : NULL, k,
                           u ? u + (size_t)b * k : NULL, commit,
                           logits ? logits + (size_t)b * nh * V : NULL, NULL, NULL);
    if (rc < 0) err |= 1;
  }
  return err ? -1 : 0;
}

/* ------------------------------------------------------- token decisions */

/* Greedy head decoding: argmax over v, exact ties to the lowest id. */
int SYM(orc_argmax)(const double *logits, int V) {
  int best = 0;
  for (int v = 1; v < V; ++v)
    if (logits[v] > logits[best]) best = v;
  return best;
}

/*
 * Inverse-CDF map (Appendix B, CDF and inverse-CDF equations): with the
 * vocabulary in id order and F_m = q_1 + ... + q_m, return the smallest m with
 * F_m > z.  If rounding leaves F_V <= z, return the largest m with q_m > 0.
 * q is a probability vector; z in [0, 1).
 */
int SYM(orc_icdf)(const double *q, int V, double z) {
  double F = 0;
  for (int m = 0; m < V; ++m) {
    F += q[m];
    if (F > z) return m;
  }
  for (int m = V - 1; m >= 0; --m)
    if (q[m] > 0) return m;
  return V - 1;
}

/* Softmax over logits (max subtracted) into q; returns the sum before normalising. */
double SYM(orc_softmax)(const double *logits, int V, double *q) {
  double mx = logits[0];
  for (int v = 1; v < V; ++v)
    if (logits[v] > mx) mx = logits[v];
  double s = 0;
  for (int v = 0; v < V; ++v) {
    q[v] = exp(logits[v] - mx);
    s += q[v];
  }
  for (int v = 0; v < V; ++v) q[v] /= s;
  return s;
}

/* ---------------------------------------------- component entry points */

double SYM(orc_gelu)(double x) { return (double)gelu((REAL)x); }

void SYM(orc_rmsnorm)(const double *x, const double *g, int d, double *y) {
  REAL *xr = (REAL *)malloc(sizeof(REAL) * 3 * (size_t)d);
  for (int i = 0; i < d; ++i) { xr[i] = (REAL)x[i]; xr[d + i] = (REAL)g[i]; }
  rmsnorm(xr, xr + d, d, xr + 2 * d);
  for (int i = 0; i < d; ++i) y[i] = (double)xr[2 * d + i];
  free(xr);
}

void SYM(orc_rope)(double *x, int H, int dh, int p) {
  REAL *xr = (REAL *)malloc(sizeof(REAL) * (size_t)H * dh);
  for (int i = 0; i < H * dh; ++i) xr[i] = (REAL)x[i];
  rope(xr, H, dh, p);
  for (int i = 0; i < H * dh; ++i) x[i] = (double)xr[i];
  free(xr);
}

void SYM(orc_layernorm)(const double *x, const double *g, const double *b, int d, double *y) {
  REAL *xr = (REAL *)calloc(3 * (size_t)d, sizeof(REAL)), *yr = (REAL *)calloc((size_t)d, sizeof(REAL));
  for (int i = 0; i < d; ++i) { xr[i] = (REAL)x[i]; xr[d + i] = (REAL)g[i]; xr[2 * d + i] = (REAL)b[i]; }
  layernorm(xr, xr + d, xr + 2 * d, d, yr);
  for (int i = 0; i < d; ++i) y[i] = (double)yr[i];
  free(xr); free(yr);
}

void SYM(orc_sinusoid)(double u, int d, double *e) {
  REAL *er = (REAL *)malloc(sizeof(REAL) * (size_t)d);
  sinusoid(u, d, er);
  for (int i = 0; i < d; ++i) e[i] = (double)er[i];
  free(er);
}

/* One head over n contiguous keys/values [n][dh]; returns the weight sum. */
double SYM(orc_attend)(const double *q, const double *K, const double *Vv, int n, int dh, double *o) {
  REAL *buf = (REAL *)malloc(sizeof(REAL) * ((size_t)2 * n * dh + 2 * (size_t)dh + n));
  const REAL **kp = (const REAL **)malloc(sizeof(REAL *) * (size_t)n);
  const REAL **vp = (const REAL **)malloc(sizeof(REAL *) * (size_t)n);
  REAL *kr = buf, *vr = buf + (size_t)n * dh, *qr = vr + (size_t)n * dh, *orr = qr + dh, *P = orr + dh;
  for (long i = 0; i < (long)n * dh; ++i) { kr[i] = (REAL)K[i]; vr[i] = (REAL)Vv[i]; }
  for (int e = 0; e < dh; ++e) qr[e] = (REAL)q[e];
  for (int t = 0; t < n; ++t) { kp[t] = kr + (size_t)t * dh; vp[t] = vr + (size_t)t * dh; }
  REAL ps = attend(qr, kp, vp, n, dh, (REAL)(1.0 / sqrt((double)dh)), P, orr);
  for (int e = 0; e < dh; ++e) o[e] = (double)orr[e];
  free(buf); free(kp); free(vp);
  return (double)ps;
}

float SYM(orc_round_bf16)(float x) { return round_bf16(x); }
