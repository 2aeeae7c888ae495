/*
 * CPU oracle for the batched speculative-verification step of WISP
 * (arXiv 2601.11652).  TEST INFRASTRUCTURE ONLY: the test suite, the package's
 * smoke check and the benchmark's CPU-baseline leg are its only users; the
 * product library neither links nor calls it, and it shares no code with it.
 *
 * Plain, slow and meant to be checked by eye against the paper:
 *   - forward pass (Sec. 4.5, "batched one-step verification"): each request's
 *     gamma+1 new rows [root, y_1..y_gamma] are forwarded on top of its cached
 *     prefix KV, stored in fixed-size pages (paged KV, Sec. 4.5), and the new
 *     rows' K/V are written in place at positions ctx_len .. ctx_len+gamma.
 *     Arithmetic is fp64; in bf16 mode values are rounded to bf16 at the
 *     points where the GPU path stores bf16 (GEMM inputs, q/k/v, KV pages).
 *     A second mode (acc32) accumulates every sum in fp32 in natural index
 *     order instead -- one more correct rounding order, used to measure how far
 *     two correct accumulation orders drift apart through the bf16 rounding
 *     points (the floor any other fp32-accumulating implementation lands on).
 *   - acceptance (Sec. 2.4, Eq. (1)-(3), with the residual distribution of
 *     Leviathan et al. that the paper relies on for losslessness): fp32, the
 *     precision in which the GPU path takes the same decisions.
 *   - Philox4x32-10 (Salmon et al., SC'11) for the method's random draws.
 *
 * Build: gcc -std=c11 -O2 -fopenmp -shared -fPIC (no fast-math, no contraction).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define ORC_PAGE 16
#define TAG_ACCEPT 1u
#define TAG_RACE 2u

/* ------------------------------------------------------------------------------------ */
/* bf16 storage helpers                                                                  */
/* ------------------------------------------------------------------------------------ */
static double bf16_to_double(uint16_t b) {
  uint32_t u = (uint32_t)b << 16;
  float f;
  memcpy(&f, &u, 4);
  return (double)f;
}

/* Round a double to the nearest bf16 value (8 significant bits), ties to even,
 * directly from double (no intermediate float rounding). */
static double round_bf16(double x) {
  if (x == 0.0 || !isfinite(x)) return x;
  int e;
  double m = frexp(x, &e);                  /* x = m * 2^e, 0.5 <= |m| < 1 */
  int q = e - 8;                            /* quantum exponent for 8 significant bits */
  if (q < -133) q = -133;                   /* bf16 subnormal quantum is 2^-133 */
  double r = nearbyint(ldexp(x, -q));       /* default rounding mode: to nearest, ties even */
  double y = ldexp(r, q);
  if (fabs(y) > 3.3895313892515355e38) y = copysign(INFINITY, x);  /* beyond bf16 max */
  return y;
}

static uint16_t double_to_bf16_bits(double x) {
  float f = (float)round_bf16(x);           /* exact: the value has <= 8 significant bits */
  uint32_t u;
  memcpy(&u, &f, 4);
  return (uint16_t)(u >> 16);
}

int orc_round_bf16_array(const double *x, double *y, int64_t n) {
  for (int64_t i = 0; i < n; i++) y[i] = round_bf16(x[i]);
  return 0;
}

/* ------------------------------------------------------------------------------------ */
/* Philox4x32-10, from Salmon, Moraes, Dror, Shaw, "Parallel random numbers: as easy as  */
/* 1, 2, 3", SC'11: ten rounds of two 32x32->64 multiplies with a Weyl key schedule.    */
/* ------------------------------------------------------------------------------------ */
void orc_philox4x32_10(const uint32_t ctr[4], const uint32_t key[2], uint32_t out[4]) {
  const uint32_t M0 = 0xD2511F53u, M1 = 0xCD9E8D57u;
  const uint32_t W0 = 0x9E3779B9u, W1 = 0xBB67AE85u;
  uint32_t c0 = ctr[0], c1 = ctr[1], c2 = ctr[2], c3 = ctr[3];
  uint32_t k0 = key[0], k1 = key[1];
  for (int round = 0; round < 10; round++) {
    if (round > 0) {
      k0 += W0;
      k1 += W1;
    }
    uint64_t p0 = (uint64_t)M0 * c0;
    uint64_t p1 = (uint64_t)M1 * c2;
    uint32_t hi0 = (uint32_t)(p0 >> 32), lo0 = (uint32_t)p0;
    uint32_t hi1 = (uint32_t)(p1 >> 32), lo1 = (uint32_t)p1;
    uint32_t n0 = hi1 ^ c1 ^ k0;
    uint32_t n2 = hi0 ^ c3 ^ k1;
    c0 = n0;
    c1 = lo1;
    c2 = n2;
    c3 = lo0;
  }
  out[0] = c0;
  out[1] = c1;
  out[2] = c2;
  out[3] = c3;
}

/* One 32-bit word of the verification RNG: key = seed, counter = (idx/4, row, req, tag). */
static uint32_t rng_word(uint64_t seed, uint32_t req_id, uint32_t tag, uint32_t row, uint32_t idx) {
  uint32_t key[2] = {(uint32_t)seed, (uint32_t)(seed >> 32)};
  uint32_t ctr[4] = {idx >> 2, row, req_id, tag};
  uint32_t out[4];
  orc_philox4x32_10(ctr, key, out);
  return out[idx & 3u];
}

/* Uniform in (0,1) on the midpoint grid of 2^23 cells: (2 * (w >> 9) + 1) * 2^-24.
 * The odd numerator is below 2^24, so the value is exact in fp32 and never 0 or 1. */
static float uniform_from_word(uint32_t w) {
  return (float)(((w >> 9) << 1) | 1u) * 5.9604644775390625e-8f;
}

float orc_uniform(uint64_t seed, uint32_t req_id, uint32_t tag, uint32_t row, uint32_t idx) {
  return uniform_from_word(rng_word(seed, req_id, tag, row, idx));
}

void orc_uniform_array(uint64_t seed, uint32_t req_id, uint32_t tag, uint32_t row, uint32_t n, float *out) {
  for (uint32_t i = 0; i < n; i++) out[i] = orc_uniform(seed, req_id, tag, row, i);
}

/* ------------------------------------------------------------------------------------ */
/* acceptance: Sec. 2.4, Eq. (1)-(3)                                                     */
/* ------------------------------------------------------------------------------------ */
typedef struct {
  int32_t R;           /* first rejected draft (1-based), gamma+1 when all accepted      */
  int32_t degenerate;  /* rejection whose residual max(0, p - q) had no positive entry    */
  float race_key1;     /* winning race key                                               */
  float race_key2;     /* runner-up race key (-inf when there is none)                   */
} orc_accept_info;

/* Target probabilities of one logits row at temperature T > 0:
 * z = l / T, m = max z, S = sum exp(z - m) (accumulated in fp64, rounded to fp32),
 * p(k) = exp(z_k - m) / S. */
static void row_softmax_stats(const float *l, int V, float T, float *m_out, float *S_out) {
  float m = -INFINITY;
  for (int k = 0; k < V; k++) {
    float z = l[k] / T;
    if (z > m) m = z;
  }
  double s = 0.0;
  for (int k = 0; k < V; k++) s += (double)expf(l[k] / T - m);
  *m_out = m;
  *S_out = (float)s;
}

static float prob_at(const float *l, float T, float m, float S, int k) {
  return expf(l[k] / T - m) / S;
}

static int argmax_first(const float *l, int V) {
  int best = 0;
  for (int k = 1; k < V; k++)
    if (l[k] > l[best]) best = k;
  return best;
}

/* Gumbel-max / exponential race: argmax_k [score_k - ln(-ln u_k)], smallest k on ties.
 * Entries with score = -inf never win. */
static int race(const float *score, int V, uint64_t seed, uint32_t req_id, uint32_t row,
                float *key1, float *key2) {
  int best = -1;
  float b1 = -INFINITY, b2 = -INFINITY;
  for (int k = 0; k < V; k++) {
    if (score[k] == -INFINITY) continue;
    float u = orc_uniform(seed, req_id, TAG_RACE, row, (uint32_t)k);
    float key = score[k] - logf(-logf(u));
    if (best < 0 || key > b1) {
      b2 = b1;
      b1 = key;
      best = k;
    } else if (key > b2) {
      b2 = key;
    }
  }
  *key1 = b1;
  *key2 = b2;
  return best;
}

/* One request.  logits: (gamma+1) rows of V; tok: [root, y_1..y_gamma]; q: gamma rows
 * (row j-1 holds q_j); out: gamma+1 slots filled with y_1..y_L, extra token, then -1.
 * u_inject (gamma values or NULL) replaces the Philox acceptance draws.
 * acc_u / acc_a (gamma slots or NULL) receive the draws and ratios of decisions taken. */
int orc_accept_one(int V, int gamma, const float *logits, const int32_t *tok, const float *q,
                   float T, uint64_t seed, uint32_t req_id, const float *u_inject,
                   int32_t *out, float *acc_u, float *acc_a, orc_accept_info *info) {
  int R = gamma + 1;
  float *work = (float *)malloc(sizeof(float) * (size_t)V);
  orc_accept_info inf = {0, 0, -INFINITY, -INFINITY};
  for (int j = 0; j <= gamma; j++) out[j] = -1;

  if (T == 0.0f) {                                   /* greedy: the T -> 0 limit */
    for (int j = 1; j <= gamma; j++) {
      int g = argmax_first(logits + (size_t)(j - 1) * V, V);
      if (acc_u) acc_u[j - 1] = 0.5f;
      if (acc_a) acc_a[j - 1] = (tok[j] == g) ? 1.0f : 0.0f;
      if (tok[j] != g) {
        R = j;
        break;
      }
    }
    for (int j = 1; j < R; j++) out[j - 1] = tok[j];
    out[R - 1] = argmax_first(logits + (size_t)(R - 1) * V, V);
    inf.R = R;
    if (info) *info = inf;
    free(work);
    return R - 1;
  }

  /* Eq. (1): a_j = min(1, p(y_j | x, y_<j) / q(y_j | x, y_<j)), accept iff u_j <= a_j. */
  for (int j = 1; j <= gamma; j++) {
    const float *l = logits + (size_t)(j - 1) * V;
    float m, S;
    row_softmax_stats(l, V, T, &m, &S);
    int y = tok[j];
    float P = prob_at(l, T, m, S, y);
    float Q = q[(size_t)(j - 1) * V + y];
    float a = (Q > 0.0f) ? fminf(1.0f, P / Q) : (P > 0.0f ? 1.0f : 0.0f);
    float u = u_inject ? u_inject[j - 1] : orc_uniform(seed, req_id, TAG_ACCEPT, (uint32_t)j, 0u);
    if (acc_u) acc_u[j - 1] = u;
    if (acc_a) acc_a[j - 1] = a;
    if (!(u <= a)) {                                  /* Eq. (2): R = first rejection */
      R = j;
      break;
    }
  }
  int L = R - 1;
  for (int j = 1; j <= L; j++) out[j - 1] = tok[j];

  /* Eq. (3) and the residual: after a rejection the extra token follows
   * norm(max(0, p_R - q_R)); after a fully accepted block it follows p. */
  int r = R - 1;                                     /* logits row that scores position R */
  const float *l = logits + (size_t)r * V;
  float m, S;
  row_softmax_stats(l, V, T, &m, &S);
  int extra;
  if (R <= gamma) {
    const float *qr = q + (size_t)(R - 1) * V;
    int any = 0;
    for (int k = 0; k < V; k++) {
      float w = prob_at(l, T, m, S, k) - qr[k];
      if (w > 0.0f) {
        work[k] = logf(w);
        any = 1;
      } else {
        work[k] = -INFINITY;
      }
    }
    if (!any) {                                      /* zero residual mass: sample p */
      inf.degenerate = 1;
      for (int k = 0; k < V; k++) work[k] = l[k] / T;
    }
  } else {
    for (int k = 0; k < V; k++) work[k] = l[k] / T;
  }
  extra = race(work, V, seed, req_id, (uint32_t)r, &inf.race_key1, &inf.race_key2);
  out[L] = extra;
  inf.R = R;
  if (info) *info = inf;
  free(work);
  return L;
}

/* Batch of requests laid out as in the step: request i owns rows off_i .. off_i+gamma_i
 * of logits/tokens/out and rows doff_i .. doff_i+gamma_i-1 of q (off, doff prefix sums). */
int orc_accept_batch(int B, int V, const int32_t *gamma, const uint32_t *req_id,
                     const float *logits, const int32_t *tokens, const float *q, float T,
                     uint64_t seed, const float *u_inject, int32_t *accept_len, int32_t *out,
                     float *acc_u, float *acc_a, int32_t *R_out, int32_t *degenerate,
                     float *race_key1, float *race_key2) {
  int64_t *off = (int64_t *)malloc(sizeof(int64_t) * (size_t)(B + 1));
  int64_t *doff = (int64_t *)malloc(sizeof(int64_t) * (size_t)(B + 1));
  off[0] = doff[0] = 0;
  for (int i = 0; i < B; i++) {
    off[i + 1] = off[i] + gamma[i] + 1;
    doff[i + 1] = doff[i] + gamma[i];
  }
#pragma omp parallel for schedule(dynamic, 64)
  for (int i = 0; i < B; i++) {
    orc_accept_info inf;
    accept_len[i] = orc_accept_one(
        V, gamma[i], logits + off[i] * V, tokens + off[i], q + doff[i] * V, T, seed,
        req_id ? req_id[i] : (uint32_t)i, u_inject ? u_inject + doff[i] : NULL, out + off[i],
        acc_u ? acc_u + doff[i] : NULL, acc_a ? acc_a + doff[i] : NULL, &inf);
    if (R_out) R_out[i] = inf.R;
    if (degenerate) degenerate[i] = inf.degenerate;
    if (race_key1) race_key1[i] = inf.race_key1;
    if (race_key2) race_key2[i] = inf.race_key2;
  }
  free(off);
  free(doff);
  return 0;
}

/* Ordinary (non-speculative) decoding of one logits row: a sample from p at temperature
 * T (Gumbel-max over the same RNG stream as a race on that row), or argmax when T = 0. */
int32_t orc_plain_decode(int V, const float *l, float T, uint64_t seed, uint32_t req_id, uint32_t row) {
  if (T == 0.0f) {
    int best = 0;
    for (int k = 1; k < V; k++)
      if (l[k] > l[best]) best = k;
    return best;
  }
  int best = -1;
  float bk = 0.0f;
  for (int k = 0; k < V; k++) {
    float g = -logf(-logf(orc_uniform(seed, req_id, TAG_RACE, row, (uint32_t)k)));
    float key = l[k] / T + g;
    if (best < 0 || key > bk) {
      bk = key;
      best = k;
    }
  }
  return best;
}

/* ------------------------------------------------------------------------------------ */
/* forward pass                                                                          */
/* ------------------------------------------------------------------------------------ */
typedef struct {
  int32_t n_layers, d, n_q, n_kv, hd, F, V;
  int32_t bf16;          /* 0: fp32 storage, no rounding; 1: bf16 storage and rounding     */
  int32_t acc32;         /* 0: sums in fp64; 1: sums in fp32, natural index order          */
  double eps, rope_base;
  const void *embed;     /* [V][d]                                                       */
  const void *lm_head;   /* [V][d]                                                       */
  const void *final_norm;/* [d]                                                          */
  const void *const *attn_norm, *const *wq, *const *wk, *const *wv, *const *wo;
  const void *const *mlp_norm, *const *w_gate, *const *w_up, *const *w_down;
} orc_model;

static double wval(const orc_model *m, const void *p, int64_t i) {
  return m->bf16 ? bf16_to_double(((const uint16_t *)p)[i]) : (double)((const float *)p)[i];
}

static double act_round(const orc_model *m, double x) { return m->bf16 ? round_bf16(x) : x; }

/* y[r][n] = sum_k x[r][k] * W[n][k] for all rows r (W natural [out][in] layout).
 * acc32: the products of the fp32 operands are summed in fp32, k = 0, 1, ... */
static void linear(const orc_model *m, const void *W, const double *x, double *y, int rows,
                   int in, int outn) {
#pragma omp parallel for schedule(static)
  for (int n = 0; n < outn; n++) {
    for (int r = 0; r < rows; r++) {
      const double *xr = x + (int64_t)r * in;
      if (m->acc32) {
        float acc = 0.0f;
        for (int k = 0; k < in; k++) acc += (float)xr[k] * (float)wval(m, W, (int64_t)n * in + k);
        y[(int64_t)r * outn + n] = acc;
      } else {
        double acc = 0.0;
        for (int k = 0; k < in; k++) acc += xr[k] * wval(m, W, (int64_t)n * in + k);
        y[(int64_t)r * outn + n] = acc;
      }
    }
  }
}

/* The residual update h += t; acc32 keeps the residual stream in fp32. */
static void residual_add(const orc_model *m, double *h, const double *t, int64_t n) {
  for (int64_t e = 0; e < n; e++) h[e] = m->acc32 ? (double)((float)h[e] + (float)t[e]) : h[e] + t[e];
}

/* RMSNorm: x * g / sqrt(mean(x^2) + eps); acc32 sums the squares in fp32. */
static void rmsnorm(const orc_model *m, const void *g, const double *h, double *x, int rows) {
  int d = m->d;
  for (int r = 0; r < rows; r++) {
    double ss = 0.0;
    float ss32 = 0.0f;
    for (int k = 0; k < d; k++) {
      const double v = h[(int64_t)r * d + k];
      ss += v * v;
      ss32 += (float)v * (float)v;
    }
    if (m->acc32) ss = ss32;
    double inv = 1.0 / sqrt(ss / d + m->eps);
    for (int k = 0; k < d; k++)
      x[(int64_t)r * d + k] = act_round(m, h[(int64_t)r * d + k] * inv * wval(m, g, k));
  }
}

/* Rotary embedding, rotate-half pairing (i, i + hd/2), angle pos * base^(-2i/hd). */
static void rope(double *v, int hd, int pos, double base) {
  int h2 = hd / 2;
  for (int i = 0; i < h2; i++) {
    double inv_freq = pow(base, -2.0 * i / hd);
    double ang = (double)pos * inv_freq;
    double c = cos(ang), s = sin(ang);
    double x1 = v[i], x2 = v[i + h2];
    v[i] = x1 * c - x2 * s;
    v[i + h2] = x2 * c + x1 * s;
  }
}

/* KV pool of one layer: [n_blocks][n_kv][16][hd], a page holding 16 slots of hd values
 * each, slot-major.  Token t of request i lives in block page_table[i][t / 16], slot t % 16. */
static double kv_get(int bf16, const void *pool, int64_t idx) {
  return bf16 ? bf16_to_double(((const uint16_t *)pool)[idx]) : (double)((const float *)pool)[idx];
}

static void kv_put(int bf16, void *pool, int64_t idx, double v) {
  if (bf16)
    ((uint16_t *)pool)[idx] = double_to_bf16_bits(v);
  else
    ((float *)pool)[idx] = (float)v;
}

static int64_t kv_index(int n_kv, int hd, int block, int kvh, int slot, int dim) {
  return (((int64_t)block * n_kv + kvh) * ORC_PAGE + slot) * hd + dim;
}

/* Causal attention of the new rows over each request's paged KV (one layer).
 * q: [M][n_q][hd]; out: [M][n_q][hd].  Row j of request i sits at position
 * ctx_len[i] + j and sees keys 0 .. ctx_len[i] + j.  acc32: the dot products, the
 * softmax denominator and the weighted sum of values accumulate in fp32, and in bf16
 * mode the weights exp(s - max) are rounded to bf16 first (the operand precision of a
 * bf16 matrix-core product of weights and values), the denominator summing the rounded
 * weights. */
int orc_paged_attention(int n_q, int n_kv, int hd, int bf16, int acc32, const void *k_pool,
                        const void *v_pool, const int32_t *page_table, int pt_stride, int B,
                        const int32_t *ctx_len, const int32_t *n_new, const double *q, double *out) {
  int G = n_q / n_kv;
  int64_t *off = (int64_t *)malloc(sizeof(int64_t) * (size_t)(B + 1));
  off[0] = 0;
  for (int i = 0; i < B; i++) off[i + 1] = off[i] + n_new[i];
  int64_t M = off[B];
  double scale = 1.0 / sqrt((double)hd);
#pragma omp parallel for schedule(dynamic, 1)
  for (int64_t rh = 0; rh < M * n_q; rh++) {
    int64_t r = rh / n_q;
    int hq = (int)(rh % n_q);
    int i = 0;
    while (off[i + 1] <= r) i++;
    int pos = ctx_len[i] + (int)(r - off[i]);
    int kvh = hq / G;
    const double *qv = q + (r * n_q + hq) * hd;
    double *s = (double *)malloc(sizeof(double) * (size_t)(pos + 1));
    double mx = -INFINITY;
    for (int t = 0; t <= pos; t++) {
      int blk = page_table[(int64_t)i * pt_stride + t / ORC_PAGE];
      double dot = 0.0;
      float dot32 = 0.0f;
      for (int e = 0; e < hd; e++) {
        const double kk = kv_get(bf16, k_pool, kv_index(n_kv, hd, blk, kvh, t % ORC_PAGE, e));
        if (acc32)
          dot32 += (float)qv[e] * (float)kk;
        else
          dot += qv[e] * kk;
      }
      s[t] = (acc32 ? (double)dot32 : dot) * scale;
      if (s[t] > mx) mx = s[t];
    }
    double den = 0.0;
    float den32 = 0.0f;
    for (int t = 0; t <= pos; t++) {
      s[t] = exp(s[t] - mx);
      if (acc32 && bf16) s[t] = round_bf16(s[t]);
      den += s[t];
      den32 += (float)s[t];
    }
    if (acc32) den = den32;
    double *o = out + (r * n_q + hq) * hd;
    for (int e = 0; e < hd; e++) o[e] = 0.0;
    for (int t = 0; t <= pos; t++) {
      int blk = page_table[(int64_t)i * pt_stride + t / ORC_PAGE];
      double w = s[t] / den;
      for (int e = 0; e < hd; e++) {
        const double vv = kv_get(bf16, v_pool, kv_index(n_kv, hd, blk, kvh, t % ORC_PAGE, e));
        o[e] = acc32 ? (double)((float)o[e] + (float)w * (float)vv) : o[e] + w * vv;
      }
    }
    free(s);
  }
  free(off);
  return 0;
}

/* Forward the new rows of every request; writes their K/V into the pools (all layers,
 * pools laid out [n_layers][n_blocks]...) and returns fp32 logits [M][V]. */
int orc_forward(const orc_model *m, void *k_pool, void *v_pool, int n_blocks, int B,
                const int32_t *ctx_len, const int32_t *n_new, const int32_t *page_table,
                int pt_stride, const int32_t *tokens, float *logits) {
  int d = m->d, hd = m->hd, nq = m->n_q, nkv = m->n_kv, F = m->F;
  int64_t M = 0;
  for (int i = 0; i < B; i++) M += n_new[i];
  if (M == 0) return 0;
  int *pos = (int *)malloc(sizeof(int) * (size_t)M);
  int *req = (int *)malloc(sizeof(int) * (size_t)M);
  {
    int64_t r = 0;
    for (int i = 0; i < B; i++)
      for (int j = 0; j < n_new[i]; j++, r++) {
        pos[r] = ctx_len[i] + j;
        req[r] = i;
      }
  }
  int qd = nq * hd, kd = nkv * hd;
  double *h = (double *)calloc((size_t)(M * d), sizeof(double));
  double *x = (double *)malloc(sizeof(double) * (size_t)(M * d));
  double *qb = (double *)malloc(sizeof(double) * (size_t)(M * qd));
  double *kb = (double *)malloc(sizeof(double) * (size_t)(M * kd));
  double *vb = (double *)malloc(sizeof(double) * (size_t)(M * kd));
  double *ob = (double *)malloc(sizeof(double) * (size_t)(M * qd));
  double *gb = (double *)malloc(sizeof(double) * (size_t)(M * F));
  double *ub = (double *)malloc(sizeof(double) * (size_t)(M * F));
  double *tmp = (double *)malloc(sizeof(double) * (size_t)(M * d));
  int64_t layer_k = (int64_t)n_blocks * nkv * ORC_PAGE * hd;   /* elements per layer */
  int esz = m->bf16 ? 2 : 4;

  for (int64_t r = 0; r < M; r++)
    for (int k = 0; k < d; k++) h[r * d + k] = wval(m, m->embed, (int64_t)tokens[r] * d + k);

  for (int l = 0; l < m->n_layers; l++) {
    char *kl = (char *)k_pool + (size_t)(l * layer_k) * esz;
    char *vl = (char *)v_pool + (size_t)(l * layer_k) * esz;
    rmsnorm(m, m->attn_norm[l], h, x, (int)M);
    linear(m, m->wq[l], x, qb, (int)M, d, qd);
    linear(m, m->wk[l], x, kb, (int)M, d, kd);
    linear(m, m->wv[l], x, vb, (int)M, d, kd);
    for (int64_t r = 0; r < M; r++) {
      for (int hh = 0; hh < nq; hh++) rope(qb + r * qd + hh * hd, hd, pos[r], m->rope_base);
      for (int hh = 0; hh < nkv; hh++) rope(kb + r * kd + hh * hd, hd, pos[r], m->rope_base);
      for (int e = 0; e < qd; e++) qb[r * qd + e] = act_round(m, qb[r * qd + e]);
      /* append k, v at this row's position (the store rounds to the pool dtype) */
      int blk = page_table[(int64_t)req[r] * pt_stride + pos[r] / ORC_PAGE];
      int slot = pos[r] % ORC_PAGE;
      for (int hh = 0; hh < nkv; hh++)
        for (int e = 0; e < hd; e++) {
          kv_put(m->bf16, kl, kv_index(nkv, hd, blk, hh, slot, e), kb[r * kd + hh * hd + e]);
          kv_put(m->bf16, vl, kv_index(nkv, hd, blk, hh, slot, e), vb[r * kd + hh * hd + e]);
        }
    }
    orc_paged_attention(nq, nkv, hd, m->bf16, m->acc32, kl, vl, page_table, pt_stride, B, ctx_len,
                        n_new, qb, ob);
    for (int64_t e = 0; e < M * qd; e++) ob[e] = act_round(m, ob[e]);
    linear(m, m->wo[l], ob, tmp, (int)M, qd, d);
    residual_add(m, h, tmp, M * d);

    rmsnorm(m, m->mlp_norm[l], h, x, (int)M);
    linear(m, m->w_gate[l], x, gb, (int)M, d, F);
    linear(m, m->w_up[l], x, ub, (int)M, d, F);
    for (int64_t e = 0; e < M * F; e++) {
      double g = gb[e];
      gb[e] = act_round(m, g / (1.0 + exp(-g)) * ub[e]);   /* SwiGLU: silu(gate) * up */
    }
    linear(m, m->w_down[l], gb, tmp, (int)M, F, d);
    residual_add(m, h, tmp, M * d);
  }
  rmsnorm(m, m->final_norm, h, x, (int)M);
  {
    int V = m->V;
    double *lg = (double *)malloc(sizeof(double) * (size_t)(M * V));
    linear(m, m->lm_head, x, lg, (int)M, d, V);
    for (int64_t e = 0; e < M * V; e++) logits[e] = (float)lg[e];
    free(lg);
  }
  free(pos);
  free(req);
  free(h);
  free(x);
  free(qb);
  free(kb);
  free(vb);
  free(ob);
  free(gb);
  free(ub);
  free(tmp);
  return 0;
}

/* ------------------------------------------------------------------------------------ */
/* small pieces exposed for the pin tests                                                */
/* ------------------------------------------------------------------------------------ */
/* Target distribution of one logits row at temperature T > 0, as the acceptance uses it. */
int orc_row_probs(const float *l, int V, float T, float *p) {
  float m, S;
  row_softmax_stats(l, V, T, &m, &S);
  for (int k = 0; k < V; k++) p[k] = prob_at(l, T, m, S, k);
  return 0;
}

/* One projection y = x W^T as the forward computes it (fp64, or fp32 sums with acc32);
 * W holds fp32 values, x rows of `in` values. */
int orc_linear_apply(const float *W, const double *x, double *y, int rows, int in, int outn, int acc32) {
  orc_model m;
  memset(&m, 0, sizeof(m));
  m.acc32 = acc32;
  linear(&m, W, x, y, rows, in, outn);
  return 0;
}

int orc_rope_apply(double *v, int hd, int pos, double base) {
  rope(v, hd, pos, base);
  return 0;
}

int orc_rmsnorm_apply(const double *h, double *x, int rows, int d, double eps, int bf16) {
  orc_model m;
  memset(&m, 0, sizeof(m));
  m.d = d;
  m.eps = eps;
  m.bf16 = bf16;
  float *gf = (float *)malloc(sizeof(float) * (size_t)d);
  for (int k = 0; k < d; k++) gf[k] = 1.0f;
  m.bf16 = 0;                       /* gains read as fp32 ones */
  rmsnorm(&m, gf, h, x, rows);
  if (bf16)
    for (int64_t e = 0; e < (int64_t)rows * d; e++) x[e] = round_bf16(x[e]);
  free(gf);
  return 0;
}
