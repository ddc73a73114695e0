/*
 * ssref.c -- plain CPU oracle for the fused LLM sampling pipeline.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path may link, load or
 * call this file; only the tests, the smoke check and the CPU-baseline leg of
 * the benchmark do.  It shares no code, header, table or constant with the
 * HIP implementation.
 *
 * What it computes (SonicSampler, arXiv 2607.20475):
 *   - the logit-processing prologue in the paper's order (Alg. 8 "Stage 1",
 *     prologue steps; equations of Appendix C.1): grammar bit-mask,
 *     multiplicative repetition penalty, frequency and presence penalties,
 *     logit bias.  Each step is one IEEE float32 operation per element, as a
 *     float32 kernel computes it (build with -ffp-contract=off);
 *   - a full sort of the valid tokens (value descending, index ascending:
 *     the paper's index-complement packing in Section 3.4 makes the lower
 *     index win ties);
 *   - truncation in Alg. 11 order (top-k, then top-p on the top-k-renormalised
 *     distribution, then min-p in the logit domain, eq. "min_p_trick",
 *     Appendix C.2), temperature entering only the probabilities; requests
 *     without a top-k cut either bounded to the k_cap leading tokens
 *     (Section 3.3's bounded candidate set) or, in the full-row form, with
 *     top-p over the whole row's distribution (Appendix C.2) whenever the
 *     kept set fits the bound;
 *   - categorical selection by inverse CDF over the kept prefix, with a
 *     uniform from Philox4x32-10 keyed by (seed, request, position); or by
 *     Gumbel-max over the kept set with caller-drawn noise g = ln z,
 *     z ~ Exp(1) (Appendix C.3; the Stage-2 selection subtracts g at the kept
 *     ids);
 *   - speculative verification (Section 3.1 "Speculative Verification",
 *     Appendix C.4): accept when u*q(d) <= p(d), else resample from
 *     normalize(max(0, p - q)); a bonus token after full acceptance; the
 *     draft distribution q either dense over the vocabulary or sparse, as the
 *     (id, probability) list a singular-mode draft step emits over its
 *     candidate set (Section 3.2), every unlisted id having q = 0; and, for
 *     one path through a draft tree, a map from the path's positions to the
 *     target rows computed for the tree (the draft-to-target mapping of
 *     Appendix C.4);
 *   - top-k log-probabilities (indicator bit 0x400 of the bit-level encoding
 *     table, Section 3.5): the leading tokens of the canonical order with
 *     their log-probabilities under the untruncated distribution of the row.
 *
 * Probabilities, sums and every decision taken on them are in double
 * precision.  Readings of points the paper leaves open are listed in the
 * design notes; the ones that change results are repeated where they apply.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

/* Per-request indicator bits: the paper's bit-level encoding table (Section 3.5). */
enum {
  R_GRAMMAR = 0x001, R_REP = 0x002, R_FREQ = 0x004, R_PRES = 0x008,
  R_BIAS = 0x010, R_TEMP = 0x020, R_GREEDY = 0x040, R_TOPK = 0x080,
  R_TOPP = 0x100, R_MINP = 0x200, R_LOGPROBS = 0x400
};
/* Per-row result flags. */
enum { RF_EMPTY = 1, RF_KCAP = 8 };

/* ------------------------------------------------------------------------- */
/* Philox4x32-10 (Salmon, Moraes, Dror, Shaw, SC'11), written from its        */
/* published definition: 10 rounds of two 32x32->64 multiplies with a Weyl    */
/* key schedule.                                                              */
/* ------------------------------------------------------------------------- */
void ssref_philox4x32_10(const uint32_t ctr_in[4], const uint32_t key_in[2], uint32_t out[4]) {
  uint32_t c0 = ctr_in[0], c1 = ctr_in[1], c2 = ctr_in[2], c3 = ctr_in[3];
  uint32_t k0 = key_in[0], k1 = key_in[1];
  for (int round = 0; round < 10; ++round) {
    uint64_t p0 = (uint64_t)0xD2511F53u * (uint64_t)c0;
    uint64_t p1 = (uint64_t)0xCD9E8D57u * (uint64_t)c2;
    uint32_t hi0 = (uint32_t)(p0 >> 32), lo0 = (uint32_t)p0;
    uint32_t hi1 = (uint32_t)(p1 >> 32), lo1 = (uint32_t)p1;
    uint32_t n0 = hi1 ^ c1 ^ k0;
    uint32_t n1 = lo1;
    uint32_t n2 = hi0 ^ c3 ^ k1;
    uint32_t n3 = lo0;
    c0 = n0; c1 = n1; c2 = n2; c3 = n3;
    k0 += 0x9E3779B9u;
    k1 += 0xBB67AE85u;
  }
  out[0] = c0; out[1] = c1; out[2] = c2; out[3] = c3;
}

/* Uniform in (0,1) for (seed, request, position); `word` 0 drives token draws,
 * word 1 the acceptance test.  u = (w + 1/2) * 2^-32, exact in double. */
double ssref_uniform(uint64_t seed, uint32_t request, int64_t position, int word) {
  uint32_t ctr[4] = {request, (uint32_t)((uint64_t)position & 0xFFFFFFFFu),
                     (uint32_t)((uint64_t)position >> 32), 0u};
  uint32_t key[2] = {(uint32_t)(seed & 0xFFFFFFFFu), (uint32_t)(seed >> 32)};
  uint32_t o[4];
  ssref_philox4x32_10(ctr, key, o);
  return ((double)o[word & 3] + 0.5) * (1.0 / 4294967296.0);
}

/* ------------------------------------------------------------------------- */
/* Logit load: bf16 widens exactly to float32.  NaN -> -inf, -0 -> +0.         */
/* ------------------------------------------------------------------------- */
static float load_logit(const void *x, int dtype, int64_t i) {
  float v;
  if (dtype == 1) {
    uint32_t u = ((uint32_t)((const uint16_t *)x)[i]) << 16;
    memcpy(&v, &u, 4);
  } else {
    v = ((const float *)x)[i];
  }
  if (isnan(v)) return -INFINITY;
  if (v == 0.0f) return 0.0f;
  return v;
}

/* ------------------------------------------------------------------------- */
/* Prologue for one row (Alg. 8 prologue order; Appendix C.1 equations).       */
/*   hist/nhist  : decoded token ids so far (multiplicity = count c_i)         */
/*   extra/nextra: further decoded ids (accepted drafts during verification)   */
/*   bias        : (id, value) entries, summed per id in list order            */
/*   mask_row    : allow bits, bit (i & 31) of word (i >> 5); NULL = no mask    */
/* ------------------------------------------------------------------------- */
void ssref_process_row(const void *x, int dtype, int V, uint32_t mode,
                       float rep, float freq, float pres,
                       const int32_t *hist, int nhist, const int32_t *extra, int nextra,
                       const int32_t *bias_ids, const float *bias_vals, int nbias,
                       const uint32_t *mask_row, float *y) {
  for (int i = 0; i < V; ++i) y[i] = load_logit(x, dtype, i);

  /* Grammar bit-masking: x_i <- -inf where m_i = 0. */
  if ((mode & R_GRAMMAR) && mask_row) {
    for (int i = 0; i < V; ++i)
      if (((mask_row[i >> 5] >> (i & 31)) & 1u) == 0u) y[i] = -INFINITY;
  }

  /* Repetition penalties: c_i = occurrences of i in the decoded sequence. */
  if (mode & (R_REP | R_FREQ | R_PRES)) {
    int32_t *c = (int32_t *)calloc((size_t)V, sizeof(int32_t));
    for (int h = 0; h < nhist; ++h)
      if (hist[h] >= 0 && hist[h] < V) c[hist[h]]++;
    for (int h = 0; h < nextra; ++h)
      if (extra[h] >= 0 && extra[h] < V) c[extra[h]]++;
    for (int i = 0; i < V; ++i) {
      if (c[i] == 0) continue;
      float v = y[i];
      if (mode & R_REP) v = (v > 0.0f) ? v / rep : v * rep;   /* multiplicative */
      if (mode & R_FREQ) { float t = freq * (float)c[i]; v = v - t; }  /* - beta*c_i */
      if (mode & R_PRES) v = v - pres;                         /* - gamma*1[c_i>0] */
      y[i] = v;
    }
    free(c);
  }

  /* Logit bias: x_i <- x_i + b_i, b_i the float32 sum of the row's entries for i. */
  if ((mode & R_BIAS) && nbias > 0) {
    float *b = (float *)calloc((size_t)V, sizeof(float));
    unsigned char *has = (unsigned char *)calloc((size_t)V, 1);
    for (int e = 0; e < nbias; ++e) {
      int id = bias_ids[e];
      if (id < 0 || id >= V) continue;
      b[id] = b[id] + bias_vals[e];
      has[id] = 1;
    }
    for (int i = 0; i < V; ++i)
      if (has[i]) y[i] = y[i] + b[i];
    free(b);
    free(has);
  }
}

/* ------------------------------------------------------------------------- */
/* Canonical order: valid tokens (y > -inf) by value descending, then index    */
/* ascending.  A full sort; the comparator is a total order.                   */
/* ------------------------------------------------------------------------- */
typedef struct { float y; int32_t i; } vi_t;

static int cmp_vi(const void *a, const void *b) {
  const vi_t *p = (const vi_t *)a, *q = (const vi_t *)b;
  if (p->y > q->y) return -1;
  if (p->y < q->y) return 1;
  return (p->i < q->i) ? -1 : (p->i > q->i);
}

int ssref_order(const float *y, int V, int32_t *order) {
  vi_t *a = (vi_t *)malloc(sizeof(vi_t) * (size_t)(V > 0 ? V : 1));
  int n = 0;
  for (int i = 0; i < V; ++i)
    if (y[i] > -INFINITY) { a[n].y = y[i]; a[n].i = i; ++n; }
  qsort(a, (size_t)n, sizeof(vi_t), cmp_vi);
  for (int r = 0; r < n; ++r) order[r] = a[r].i;
  free(a);
  return n;
}

/* ------------------------------------------------------------------------- */
/* Truncated distribution of one row (Alg. 11 epilogue order).                 */
/* ------------------------------------------------------------------------- */
typedef struct {
  int greedy;      /* 1: greedy row (argmax, no distribution)              */
  int n_valid;     /* tokens with y > -inf                                 */
  int n_k, n_p, n_m, n_s;
  double M, tau, Z_k, Z_s;
  double margin_p; /* relative distance of the top-p comparisons to p*Z_k  */
  double margin_m; /* distance of the min-p comparisons to ln(theta)       */
  int ns_lo, ns_hi; /* admissible kept-set sizes (see ssref_near below)     */
  int flags;
} dist_t;

/* Near-boundary band.  A data-dependent comparison whose two sides differ by
 * less than this (relative to the row's normaliser for masses, absolute in
 * the logit domain for min-p) may go either way in a float32 / fixed-point
 * implementation; the oracle then admits both outcomes.  Every other
 * comparison must come out exactly as here. */
#define SSREF_NEAR 1e-6
double ssref_near(void) { return SSREF_NEAR; }

static double weight_of(double yr, double M, double tau) {
  if (yr == M) return 1.0;               /* also covers y = M = +inf */
  return exp((yr - M) / tau);
}

/* Fills w[0..n_s) (unnormalised weights in canonical order) and `d`. */
static void row_distribution(const float *y, const int32_t *order, int n_valid, uint32_t mode,
                             float temperature, int32_t top_k, float top_p, float min_p,
                             int k_cap, double *w, dist_t *d) {
  memset(d, 0, sizeof(*d));
  d->n_valid = n_valid;
  d->margin_p = INFINITY;
  d->margin_m = INFINITY;
  if (n_valid == 0) { d->flags |= RF_EMPTY; return; }
  d->greedy = (mode & R_GREEDY) || ((mode & R_TEMP) && temperature <= 0.0f);
  d->M = (double)y[order[0]];
  if (d->greedy) {
    d->n_k = d->n_p = d->n_m = d->n_s = d->ns_lo = d->ns_hi = 1;
    d->Z_k = d->Z_s = 1.0;
    w[0] = 1.0;
    return;
  }
  d->tau = (mode & R_TEMP) ? (double)temperature : 1.0;

  /* Top-k: the k highest logits.  Bounded by the candidate capacity k_cap
   * (the paper's bounded candidate set, Section 3.3). */
  int64_t k_req = ((mode & R_TOPK) && top_k >= 1) ? (int64_t)top_k : INT64_MAX;
  int64_t nk = k_req;
  if (nk > k_cap) nk = k_cap;
  if (nk > n_valid) nk = n_valid;
  if (k_req > k_cap) d->flags |= RF_KCAP;  /* request wants more than the bound */
  d->n_k = (int)nk;

  double Zk = 0.0;
  for (int r = 0; r < d->n_k; ++r) {
    w[r] = weight_of((double)y[order[r]], d->M, d->tau);
    Zk += w[r];
  }
  d->Z_k = Zk;

  /* Top-p on the top-k renormalised distribution: keep rank r while the mass
   * strictly before it is below p (minimal prefix with mass >= p). */
  d->n_p = d->n_k;
  int p_lo = d->n_k, p_hi = d->n_k;
  if ((mode & R_TOPP) && top_p < 1.0f) {
    double thr = (double)top_p * Zk;
    double excl = 0.0;
    int cnt = 0, stopped = 0;
    p_lo = -1;
    p_hi = -1;
    for (int r = 0; r < d->n_k; ++r) {
      double m = fabs(excl - thr) / Zk;
      int keep = excl < thr, near = m < SSREF_NEAR;
      if (m < d->margin_p) d->margin_p = m;
      /* admissible cut: the first rank that may stop, the first that must */
      if (p_lo < 0 && (!keep || near)) p_lo = r;
      if (p_hi < 0 && !keep && !near) p_hi = r;
      if (!stopped) {
        if (keep) cnt = r + 1; else stopped = 1;
      }
      if (stopped && p_hi >= 0) break;
      excl += w[r];
    }
    if (p_lo < 0) p_lo = d->n_k;
    if (p_hi < 0) p_hi = d->n_k;
    if (cnt < 1) cnt = 1;
    if (p_lo < 1) p_lo = 1;
    if (p_hi < 1) p_hi = 1;
    d->n_p = cnt;
  }

  /* Min-p in the logit domain: keep r when (y_r - M)/tau >= ln(theta);
   * rank 0 is always kept. */
  d->n_m = d->n_k;
  int m_lo = d->n_k, m_hi = d->n_k;
  if ((mode & R_MINP) && min_p > 0.0f) {
    double lt = log((double)min_p);
    int cnt = 1, stopped = 0;
    m_lo = -1;
    m_hi = -1;
    for (int r = 1; r < d->n_k; ++r) {
      double yr = (double)y[order[r]];
      double l = (yr == d->M) ? 0.0 : (yr - d->M) / d->tau;
      double m = fabs(l - lt);
      int keep = l >= lt, near = m < SSREF_NEAR;
      if (m < d->margin_m) d->margin_m = m;
      if (m_lo < 0 && (!keep || near)) m_lo = r;
      if (m_hi < 0 && !keep && !near) m_hi = r;
      if (!stopped) {
        if (keep) cnt = r + 1; else stopped = 1;
      }
      if (stopped && m_hi >= 0) break;
    }
    if (m_lo < 0) m_lo = d->n_k;
    if (m_hi < 0) m_hi = d->n_k;
    d->n_m = cnt;
  }

  int ns = d->n_k;
  if (d->n_p < ns) ns = d->n_p;
  if (d->n_m < ns) ns = d->n_m;
  d->n_s = ns;
  /* every min(n_k, a, b) with a, b in the admissible top-p / min-p ranges */
  d->ns_lo = d->n_k < p_lo ? d->n_k : p_lo;
  if (m_lo < d->ns_lo) d->ns_lo = m_lo;
  d->ns_hi = d->n_k < p_hi ? d->n_k : p_hi;
  if (m_hi < d->ns_hi) d->ns_hi = m_hi;
  double Zs = 0.0;
  for (int r = 0; r < ns; ++r) Zs += w[r];
  d->Z_s = Zs;
}

/* Inverse CDF over weights w[0..n): first r with sum_{s<=r} w_s > u*Z. */
static int draw_index(const double *w, int n, double Z, double u, double *margin) {
  double target = u * Z;
  double cum = 0.0, prev = 0.0;
  int pick = n - 1;
  for (int r = 0; r < n; ++r) {
    prev = cum;
    cum += w[r];
    if (cum > target) { pick = r; break; }
  }
  if (margin) {
    double m = fabs(cum - target);
    if (pick > 0 && fabs(prev - target) < m) m = fabs(prev - target);
    *margin = (Z > 0.0) ? m / Z : 0.0;
  }
  return pick;
}

/* Ranks an inverse-CDF draw over w[0..n) may return when a prefix sum within
 * `band` of the target u*Z may compare either way: rank r is admissible when
 * "sum_{s<r} w_s <= target" and "sum_{s<=r} w_s > target" may both hold
 * (the last rank takes every overshoot).  The draw's own pick comes first in
 * out[]; returns the count (at most max). */
static int draw_admissible(const double *w, int n, double Z, double u, double band, int *out, int max) {
  if (n <= 0 || max <= 0) return 0;
  const int pick = draw_index(w, n, Z, u, NULL);
  const double target = u * Z;
  int cnt = 0;
  out[cnt++] = pick;
  double prev = 0.0, cum = 0.0;
  for (int r = 0; r < n && cnt < max; ++r) {
    prev = cum;
    cum += w[r];
    int before = prev <= target || fabs(prev - target) < band;
    int after = cum > target || fabs(cum - target) < band || r == n - 1;
    if (!before) break;
    if (after && r != pick) out[cnt++] = r;
  }
  return cnt;
}

static double prefix_sum(const double *w, int n) {
  double z = 0.0;
  for (int r = 0; r < n; ++r) z += w[r];
  return z;
}

/* ------------------------------------------------------------------------- */
/* Parameter bundle (NULL arrays disable the matching mode bits).              */
/* ------------------------------------------------------------------------- */
typedef struct {
  int B, V;
  const uint32_t *mode;
  const float *temperature, *top_p, *min_p, *rep, *freq, *pres;
  const int32_t *top_k;
  const int32_t *hist_off, *hist_ids;
  const int32_t *bias_off, *bias_ids;
  const float *bias_vals;
  const uint32_t *bitmask;
  int64_t mask_ld;
  const uint64_t *seed;
  const int64_t *position;
  int k_cap;
} ssref_params;

static uint32_t effective_mode(const ssref_params *p, int b) {
  uint32_t m = p->mode ? p->mode[b] : 0u;
  if (!p->temperature) m &= ~(uint32_t)R_TEMP;
  if (!p->top_k) m &= ~(uint32_t)R_TOPK;
  if (!p->top_p) m &= ~(uint32_t)R_TOPP;
  if (!p->min_p) m &= ~(uint32_t)R_MINP;
  if (!p->rep) m &= ~(uint32_t)R_REP;
  if (!p->freq) m &= ~(uint32_t)R_FREQ;
  if (!p->pres) m &= ~(uint32_t)R_PRES;
  if (!p->hist_off || !p->hist_ids) m &= ~(uint32_t)(R_REP | R_FREQ | R_PRES);
  if (!p->bias_off || !p->bias_ids || !p->bias_vals) m &= ~(uint32_t)R_BIAS;
  if (!p->bitmask) m &= ~(uint32_t)R_GRAMMAR;
  return m;
}

static float pf(const float *a, int b, float dflt) { return a ? a[b] : dflt; }

static void process_one(const void *x, int dtype, int64_t row_off, const ssref_params *p, int b,
                        const int32_t *extra, int nextra, int64_t mask_row, float *y) {
  uint32_t mode = effective_mode(p, b);
  const int32_t *hist = NULL; int nh = 0;
  if (mode & (R_REP | R_FREQ | R_PRES)) { hist = p->hist_ids + p->hist_off[b]; nh = p->hist_off[b + 1] - p->hist_off[b]; }
  const int32_t *bid = NULL; const float *bval = NULL; int nb = 0;
  if (mode & R_BIAS) { bid = p->bias_ids + p->bias_off[b]; bval = p->bias_vals + p->bias_off[b]; nb = p->bias_off[b + 1] - p->bias_off[b]; }
  const uint32_t *mrow = (mode & R_GRAMMAR) ? p->bitmask + mask_row * p->mask_ld : NULL;
  const void *xr = (dtype == 1) ? (const void *)((const uint16_t *)x + row_off)
                                : (const void *)((const float *)x + row_off);
  ssref_process_row(xr, dtype, p->V, mode, pf(p->rep, b, 1.0f), pf(p->freq, b, 0.0f),
                    pf(p->pres, b, 0.0f), hist, nh, extra, nextra, bid, bval, nb, mrow, y);
}

/* ------------------------------------------------------------------------- */
/* Batched entry points (OpenMP over rows; rows are independent).              */
/* ------------------------------------------------------------------------- */

/* Singular-mode sampling.
 *   margin[b]   smallest relative distance of any data-dependent comparison
 *               (draw, top-p, min-p) to its boundary;
 *   adm_tok / adm_lp [B, SSREF_ADM]: the admissible outcomes -- every
 *               (token, log-probability) the row can produce when each
 *               comparison within SSREF_NEAR of its boundary may go either
 *               way; entry 0 is the oracle's own outcome, -1 pads;
 *   n_adm[b]    number of admissible outcomes (1 unless a comparison is near). */
#define SSREF_ADM 16
int ssref_adm_max(void) { return SSREF_ADM; }

int ssref_sample(const void *x, int dtype, int64_t ld, const ssref_params *p,
                 int32_t *out_token, float *out_logprob, int32_t *flags,
                 double *margin, int32_t *n_kept, int32_t *adm_tok, float *adm_lp,
                 int32_t *n_adm, int nthreads) {
  int B = p->B, V = p->V;
#ifdef _OPENMP
  if (nthreads > 0) omp_set_num_threads(nthreads);
#pragma omp parallel for schedule(dynamic, 1)
#endif
  for (int b = 0; b < B; ++b) {
    float *y = (float *)malloc(sizeof(float) * (size_t)V);
    int32_t *order = (int32_t *)malloc(sizeof(int32_t) * (size_t)V);
    double *w = (double *)malloc(sizeof(double) * (size_t)(p->k_cap > 0 ? p->k_cap : 1) + 8);
    process_one(x, dtype, (int64_t)b * ld, p, b, NULL, 0, b, y);
    int nv = ssref_order(y, V, order);
    uint32_t mode = effective_mode(p, b);
    dist_t d;
    row_distribution(y, order, nv, mode, pf(p->temperature, b, 1.0f), p->top_k ? p->top_k[b] : 0,
                     pf(p->top_p, b, 1.0f), pf(p->min_p, b, 0.0f), p->k_cap, w, &d);
    double mg = INFINITY;
    int tok = -1;
    float lp = 0.0f;
    int32_t at[SSREF_ADM];
    float al[SSREF_ADM];
    int na = 0;
    if (nv > 0) {
      if (d.greedy) {
        tok = order[0];
      } else {
        double u = ssref_uniform(p->seed[b], (uint32_t)b, p->position[b], 0);
        double md;
        int r = draw_index(w, d.n_s, d.Z_s, u, &md);
        tok = order[r];
        lp = (float)log(w[r] / d.Z_s);
        mg = md;
        if (d.margin_p < mg) mg = d.margin_p;
        if (d.margin_m < mg) mg = d.margin_m;
        /* admissible outcomes: the own kept-set size first, then the others */
        at[na] = tok;
        al[na] = lp;
        ++na;
        for (int pass = 0; pass < 2; ++pass) {
          for (int ns = d.ns_lo; ns <= d.ns_hi && na < SSREF_ADM; ++ns) {
            if ((pass == 0) != (ns == d.n_s)) continue;
            double Z = prefix_sum(w, ns);
            int ranks[SSREF_ADM];
            int nr = draw_admissible(w, ns, Z, u, SSREF_NEAR * Z, ranks, SSREF_ADM);
            for (int j = 0; j < nr && na < SSREF_ADM; ++j) {
              int32_t t = order[ranks[j]];
              float l = (float)log(w[ranks[j]] / Z);
              int dup = 0;
              for (int e = 0; e < na; ++e) dup |= (at[e] == t && al[e] == l);
              if (!dup) { at[na] = t; al[na] = l; ++na; }
            }
          }
        }
      }
    }
    if (na == 0) { at[0] = tok; al[0] = lp; na = 1; }
    out_token[b] = tok;
    if (out_logprob) out_logprob[b] = lp;
    if (flags) flags[b] = d.flags;
    if (margin) margin[b] = mg;
    if (n_kept) n_kept[b] = d.n_s;
    if (adm_tok) {
      for (int e = 0; e < SSREF_ADM; ++e) {
        adm_tok[(int64_t)b * SSREF_ADM + e] = e < na ? at[e] : -1;
        if (adm_lp) adm_lp[(int64_t)b * SSREF_ADM + e] = e < na ? al[e] : 0.0f;
      }
    }
    if (n_adm) n_adm[b] = na;
    free(y); free(order); free(w);
  }
  return 0;
}

/* Gumbel-max selection over the kept prefix (Appendix C.3): the rank whose
 * score (y - M)/tau - g[id] is largest, the lower token id on equal scores.
 * The score is formed in double exactly in this order (y == M gives 0). */
static int gumbel_pick(const float *y, const int32_t *order, int ns, double M, double tau, const float *g) {
  int best = -1;
  double bs = 0.0;
  for (int r = 0; r < ns; ++r) {
    double yr = (double)y[order[r]];
    double sc = ((yr == M) ? 0.0 : (yr - M) / tau) - (double)g[order[r]];
    if (best < 0 || sc > bs || (sc == bs && order[r] < order[best])) { best = r; bs = sc; }
  }
  return best;
}

/* Sampling with the Gumbel-max draw: as ssref_sample, the token chosen by
 * gumbel_pick with noise g [B, ld_g] (read at the kept ids only).  The
 * admissible outcomes are the picks over every admissible kept-set size. */
int ssref_sample_gumbel(const void *x, int dtype, int64_t ld, const ssref_params *p, const float *g,
                        int64_t ld_g, int32_t *out_token, float *out_logprob, int32_t *flags,
                        int32_t *n_kept, int32_t *adm_tok, float *adm_lp, int32_t *n_adm, int nthreads) {
  int B = p->B, V = p->V;
#ifdef _OPENMP
  if (nthreads > 0) omp_set_num_threads(nthreads);
#pragma omp parallel for schedule(dynamic, 1)
#endif
  for (int b = 0; b < B; ++b) {
    float *y = (float *)malloc(sizeof(float) * (size_t)V);
    int32_t *order = (int32_t *)malloc(sizeof(int32_t) * (size_t)V);
    double *w = (double *)malloc(sizeof(double) * (size_t)(p->k_cap > 0 ? p->k_cap : 1) + 8);
    process_one(x, dtype, (int64_t)b * ld, p, b, NULL, 0, b, y);
    int nv = ssref_order(y, V, order);
    uint32_t mode = effective_mode(p, b);
    dist_t d;
    row_distribution(y, order, nv, mode, pf(p->temperature, b, 1.0f), p->top_k ? p->top_k[b] : 0,
                     pf(p->top_p, b, 1.0f), pf(p->min_p, b, 0.0f), p->k_cap, w, &d);
    int tok = -1;
    float lp = 0.0f;
    int32_t at[SSREF_ADM];
    float al[SSREF_ADM];
    int na = 0;
    if (nv > 0) {
      if (d.greedy) {
        tok = order[0];
      } else {
        const float *gr = g + (int64_t)b * ld_g;
        for (int pass = 0; pass < 2; ++pass) {
          for (int ns = d.ns_lo; ns <= d.ns_hi && na < SSREF_ADM; ++ns) {
            if ((pass == 0) != (ns == d.n_s)) continue;
            int r = gumbel_pick(y, order, ns, d.M, d.tau, gr);
            int32_t t = order[r];
            float l = (float)log(w[r] / prefix_sum(w, ns));
            if (pass == 0) { tok = t; lp = l; }
            int dup = 0;
            for (int e = 0; e < na; ++e) dup |= (at[e] == t && al[e] == l);
            if (!dup) { at[na] = t; al[na] = l; ++na; }
          }
        }
      }
    }
    if (na == 0) { at[0] = tok; al[0] = lp; na = 1; }
    out_token[b] = tok;
    if (out_logprob) out_logprob[b] = lp;
    if (flags) flags[b] = d.flags;
    if (n_kept) n_kept[b] = d.n_s;
    if (adm_tok) {
      for (int e = 0; e < SSREF_ADM; ++e) {
        adm_tok[(int64_t)b * SSREF_ADM + e] = e < na ? at[e] : -1;
        if (adm_lp) adm_lp[(int64_t)b * SSREF_ADM + e] = e < na ? al[e] : 0.0f;
      }
    }
    if (n_adm) n_adm[b] = na;
    free(y); free(order); free(w);
  }
  return 0;
}

/* Sampling with full-row truncation for requests without a top-k cut (top-k
 * bit off or k <= 0; not greedy): top-p and min-p over every valid token of
 * the row (the Appendix C.2 definitions), used when the kept set fits the
 * candidate bound, i.e. holds fewer than k_cap tokens; otherwise the bounded
 * result of ssref_sample with RF_KCAP (the same tokens when the row has at
 * most k_cap valid tokens: the bounded set is then the whole row).  Other
 * requests are sampled exactly as by ssref_sample.  Outputs as ssref_sample;
 * the admissible outcomes cover both sides of the fit test when a kept-set
 * size within the band changes it. */
static int full_fits(int ns, int k_cap) { return ns < k_cap; }

/* adds the admissible draws over w[0..ns) to the outcome list (no duplicates) */
static void add_draws(const double *w, int ns, const int32_t *order, double u, int32_t *at, float *al, int *na) {
  double Z = prefix_sum(w, ns);
  int ranks[SSREF_ADM];
  int nr = draw_admissible(w, ns, Z, u, SSREF_NEAR * Z, ranks, SSREF_ADM);
  for (int j = 0; j < nr && *na < SSREF_ADM; ++j) {
    int32_t t = order[ranks[j]];
    float l = (float)log(w[ranks[j]] / Z);
    int dup = 0;
    for (int e = 0; e < *na; ++e) dup |= (at[e] == t && al[e] == l);
    if (!dup) { at[*na] = t; al[*na] = l; ++*na; }
  }
}

int ssref_sample_full(const void *x, int dtype, int64_t ld, const ssref_params *p, int32_t *out_token,
                      float *out_logprob, int32_t *flags, int32_t *n_kept, int32_t *adm_tok, float *adm_lp,
                      int32_t *n_adm, int nthreads) {
  int B = p->B, V = p->V;
#ifdef _OPENMP
  if (nthreads > 0) omp_set_num_threads(nthreads);
#pragma omp parallel for schedule(dynamic, 1)
#endif
  for (int b = 0; b < B; ++b) {
    float *y = (float *)malloc(sizeof(float) * (size_t)V);
    int32_t *order = (int32_t *)malloc(sizeof(int32_t) * (size_t)V);
    double *wf = (double *)malloc(sizeof(double) * (size_t)V + 8);
    double *wb = (double *)malloc(sizeof(double) * (size_t)(p->k_cap > 0 ? p->k_cap : 1) + 8);
    process_one(x, dtype, (int64_t)b * ld, p, b, NULL, 0, b, y);
    int nv = ssref_order(y, V, order);
    uint32_t mode = effective_mode(p, b);
    const float tmp = pf(p->temperature, b, 1.0f), tp = pf(p->top_p, b, 1.0f), mp = pf(p->min_p, b, 0.0f);
    const int32_t tk = p->top_k ? p->top_k[b] : 0;
    const int cap = p->k_cap;
    dist_t db, df;
    row_distribution(y, order, nv, mode, tmp, tk, tp, mp, cap, wb, &db);
    const int full = nv > 0 && !db.greedy && !((mode & R_TOPK) && tk >= 1);
    if (full) row_distribution(y, order, nv, mode, tmp, tk, tp, mp, nv, wf, &df);
    int tok = -1, ns_own = db.n_s, fl = db.flags;
    float lp = 0.0f;
    int32_t at[SSREF_ADM];
    float al[SSREF_ADM];
    int na = 0;
    if (nv > 0 && db.greedy) {
      tok = order[0];
    } else if (nv > 0) {
      const double u = ssref_uniform(p->seed[b], (uint32_t)b, p->position[b], 0);
      const int own_full = full && full_fits(df.n_s, cap);
      const double *wo = own_full ? wf : wb;
      const int no = own_full ? df.n_s : db.n_s;
      const double Zo = prefix_sum(wo, no);
      const int r = draw_index(wo, no, Zo, u, NULL);
      tok = order[r];
      lp = (float)log(wo[r] / Zo);
      ns_own = no;
      if (full) fl = (df.flags & ~RF_KCAP) | (own_full ? 0 : RF_KCAP);
      at[na] = tok; al[na] = lp; ++na;
      /* every admissible kept-set size (the own one first): a full-row size
       * that fits gives its own draws, one that does not gives the bounded
       * distribution's */
      const dist_t *d0 = full ? &df : &db;
      for (int pass = 0; pass < 2; ++pass) {
        for (int m = d0->ns_lo; m <= d0->ns_hi; ++m) {
          if ((pass == 0) != (m == d0->n_s)) continue;
          if (full && full_fits(m, cap)) {
            add_draws(wf, m, order, u, at, al, &na);
          } else {
            for (int q = 0; q < 2; ++q)
              for (int nb = db.ns_lo; nb <= db.ns_hi; ++nb)
                if ((q == 0) == (nb == db.n_s)) add_draws(wb, nb, order, u, at, al, &na);
          }
        }
      }
    }
    out_token[b] = tok;
    if (out_logprob) out_logprob[b] = lp;
    if (flags) flags[b] = fl;
    if (n_kept) n_kept[b] = ns_own;
    if (na == 0) { at[0] = tok; al[0] = lp; na = 1; }
    if (adm_tok) {
      for (int e = 0; e < SSREF_ADM; ++e) {
        adm_tok[(int64_t)b * SSREF_ADM + e] = e < na ? at[e] : -1;
        if (adm_lp) adm_lp[(int64_t)b * SSREF_ADM + e] = e < na ? al[e] : 0.0f;
      }
    }
    if (n_adm) n_adm[b] = na;
    free(y); free(order); free(wf); free(wb);
  }
  return 0;
}

/* Materialised processed logits y [B,V] (float32, pre-temperature) and the
 * final truncated distribution P [B,V] (double; zero outside the kept set,
 * one-hot at the argmax for greedy rows).
 *   ns_range [B,2] or NULL: admissible kept-set sizes (lowest, highest);
 *   force_ns [B] or NULL:   a kept-set size to use instead of the oracle's own
 *                           when it lies in the admissible range (values
 *                           outside it are ignored). */
int ssref_process_logits(const void *x, int dtype, int64_t ld, const ssref_params *p,
                         float *out_y, double *out_p, int32_t *flags, int32_t *ns_range,
                         const int32_t *force_ns, int nthreads) {
  int B = p->B, V = p->V;
#ifdef _OPENMP
  if (nthreads > 0) omp_set_num_threads(nthreads);
#pragma omp parallel for schedule(dynamic, 1)
#endif
  for (int b = 0; b < B; ++b) {
    float *y = out_y ? out_y + (int64_t)b * V : (float *)malloc(sizeof(float) * (size_t)V);
    int32_t *order = (int32_t *)malloc(sizeof(int32_t) * (size_t)V);
    double *w = (double *)malloc(sizeof(double) * (size_t)(p->k_cap > 0 ? p->k_cap : 1) + 8);
    process_one(x, dtype, (int64_t)b * ld, p, b, NULL, 0, b, y);
    int nv = ssref_order(y, V, order);
    dist_t d;
    row_distribution(y, order, nv, effective_mode(p, b), pf(p->temperature, b, 1.0f),
                     p->top_k ? p->top_k[b] : 0, pf(p->top_p, b, 1.0f), pf(p->min_p, b, 0.0f),
                     p->k_cap, w, &d);
    int ns = d.n_s;
    double Z = d.Z_s;
    if (force_ns && !d.greedy && nv > 0 && force_ns[b] >= d.ns_lo && force_ns[b] <= d.ns_hi) {
      ns = force_ns[b];
      Z = prefix_sum(w, ns);
    }
    if (out_p) {
      double *P = out_p + (int64_t)b * V;
      for (int i = 0; i < V; ++i) P[i] = 0.0;
      if (nv > 0) {
        if (d.greedy) P[order[0]] = 1.0;
        else for (int r = 0; r < ns; ++r) P[order[r]] = w[r] / Z;
      }
    }
    if (ns_range) {
      ns_range[2 * (int64_t)b] = d.ns_lo;
      ns_range[2 * (int64_t)b + 1] = d.ns_hi;
    }
    if (flags) flags[b] = d.flags;
    if (!out_y) free(y);
    free(order); free(w);
  }
  return 0;
}

/* Standalone top-k on raw values (no prologue): the first min(k_b, k_max,
 * n_valid) entries of the canonical order, padded with (-inf, -1).
 * k == NULL means k_b = k_max for every row; k_b <= 0 selects nothing. */
int ssref_topk(const void *x, int dtype, int B, int V, int64_t ld, const int32_t *k, int k_max,
               float *out_val, int32_t *out_idx, int nthreads) {
#ifdef _OPENMP
  if (nthreads > 0) omp_set_num_threads(nthreads);
#pragma omp parallel for schedule(dynamic, 1)
#endif
  for (int b = 0; b < B; ++b) {
    float *y = (float *)malloc(sizeof(float) * (size_t)V);
    int32_t *order = (int32_t *)malloc(sizeof(int32_t) * (size_t)V);
    const void *xr = (dtype == 1) ? (const void *)((const uint16_t *)x + (int64_t)b * ld)
                                  : (const void *)((const float *)x + (int64_t)b * ld);
    for (int i = 0; i < V; ++i) y[i] = load_logit(xr, dtype, i);
    int nv = ssref_order(y, V, order);
    int kb = k ? k[b] : k_max;
    if (kb < 0) kb = 0;
    if (kb > k_max) kb = k_max;
    if (kb > nv) kb = nv;
    for (int r = 0; r < k_max; ++r) {
      out_val[(int64_t)b * k_max + r] = (r < kb) ? y[order[r]] : -INFINITY;
      out_idx[(int64_t)b * k_max + r] = (r < kb) ? order[r] : -1;
    }
    free(y); free(order);
  }
  return 0;
}

/* Top-k log-probabilities (indicator bit 0x400, Section 3.5; the log-
 * probability output of Alg. 11).  For a row with the bit: the first
 * min(n_lp, n_valid) tokens of the canonical order of the processed logits y
 * (value descending, lower index first) and their log-probabilities under the
 * untruncated distribution softmax(y / tau) over every valid token:
 *   lp_i = (y_i - M) / tau - ln sum_j exp((y_j - M) / tau),   M = max_j y_j,
 * tau the row's temperature when its bit is on, tau > 0 and the row is not
 * greedy, else 1 (a greedy row reports the untempered distribution).  Top-k,
 * top-p and min-p do not apply.  Rows without the bit, and entries beyond the
 * valid tokens, hold (-1, -inf). */
int ssref_logprobs(const void *x, int dtype, int64_t ld, const ssref_params *p, int n_lp,
                   int32_t *out_idx, float *out_lp, int nthreads) {
  int B = p->B, V = p->V;
#ifdef _OPENMP
  if (nthreads > 0) omp_set_num_threads(nthreads);
#pragma omp parallel for schedule(dynamic, 1)
#endif
  for (int b = 0; b < B; ++b) {
    int32_t *oi = out_idx + (int64_t)b * n_lp;
    float *ol = out_lp + (int64_t)b * n_lp;
    for (int r = 0; r < n_lp; ++r) { oi[r] = -1; ol[r] = -INFINITY; }
    uint32_t mode = p->mode ? p->mode[b] : 0u;
    if (!(mode & R_LOGPROBS)) continue;
    float *y = (float *)malloc(sizeof(float) * (size_t)V);
    int32_t *order = (int32_t *)malloc(sizeof(int32_t) * (size_t)V);
    process_one(x, dtype, (int64_t)b * ld, p, b, NULL, 0, b, y);
    int nv = ssref_order(y, V, order);
    if (nv > 0) {
      uint32_t em = effective_mode(p, b);
      double tau = 1.0;
      if ((em & R_TEMP) && !(em & R_GREEDY) && p->temperature[b] > 0.0f) tau = (double)p->temperature[b];
      double M = (double)y[order[0]];
      double Z = 0.0;
      for (int r = 0; r < nv; ++r) Z += exp(((double)y[order[r]] - M) / tau);
      double lz = log(Z);
      int n = n_lp < nv ? n_lp : nv;
      for (int r = 0; r < n; ++r) {
        oi[r] = order[r];
        ol[r] = (float)(((double)y[order[r]] - M) / tau - lz);
      }
    }
    free(y); free(order);
  }
  return 0;
}

/* Multistep speculative verification over target rows [B, L+1, V].
 * Row l (0-based) is the target distribution for draft position l+1; its
 * penalty history is the request history plus accepted drafts d_1..d_l.
 * Draft ids outside [0, V) end the draft (q = 0 there: the position then
 * samples from the target distribution).  Outputs out_tokens [B, L+1]
 * (-1 padded) and n_acc [B].
 *
 * Admissible outcomes: every (out_tokens, n_acc) the request can produce
 * when each comparison within SSREF_NEAR of its boundary (top-p, min-p,
 * acceptance u*q(d) <= P(d), the draws; masses relative to the row's
 * normaliser, the residual draw absolute in probability units) may go either
 * way.  adm_seq [B, SSREF_ADM, L+1] and adm_nacc [B, SSREF_ADM] hold them,
 * entry 0 being the oracle's own outcome; n_adm[b] counts them. */
typedef struct {
  int ready, nv;
  dist_t d;
  float *y;
  int32_t *order;
  double *w;
} vrow_t;

typedef struct {
  const void *x;
  int dtype;
  int64_t ld_row;
  const float *q;     /* dense q [B, L, ld_q], or NULL when sparse */
  int64_t ld_q;
  const int32_t *qi;  /* sparse q: ids [B, L, kq] */
  const float *qv;    /*           probabilities [B, L, kq] */
  int kq;
  const int32_t *rmap; /* path position -> target row of the request [B, L+1], or NULL */
  int Lt;              /* target rows per request (L+1 without a map) */
  const int32_t *dr;  /* this request's drafts [L] */
  int L, b, V;
  const ssref_params *p;
  uint32_t mode;
  vrow_t *rows;       /* [L+1], computed when first reached */
  double *res;
  int32_t *seq;       /* [SSREF_ADM, L+1] */
  int32_t *nacc;      /* [SSREF_ADM] */
  int nseq;
  int fl;
  double mg;
} vctx_t;

/* Draft probability q_l(id) at draft position l (1-based).  Sparse lists: the
 * sum, in double and in list order, of the entries naming id (ids outside
 * [0, V) are padding); an unlisted id has q = 0. */
static double qget(const vctx_t *c, int l, int id) {
  if (c->kq <= 0) return (double)c->q[(int64_t)c->b * c->L * c->ld_q + (int64_t)(l - 1) * c->ld_q + id];
  const int64_t o = ((int64_t)c->b * c->L + (l - 1)) * c->kq;
  double s = 0.0;
  for (int i = 0; i < c->kq; ++i)
    if (c->qi[o + i] == id) s += (double)c->qv[o + i];
  return s;
}

static vrow_t *vrow_get(vctx_t *c, int l) {
  vrow_t *r = &c->rows[l - 1];
  if (r->ready) return r;
  int64_t row = (int64_t)c->b * (c->L + 1) + (l - 1);  /* path row: its grammar mask row */
  int64_t src = (int64_t)c->b * c->Lt + (l - 1);
  int dead = 0;
  if (c->rmap) {
    int32_t t = c->rmap[row];
    if (t >= 0 && t < c->Lt) src = (int64_t)c->b * c->Lt + t;
    else dead = 1;
  }
  if (dead) {  /* a map entry outside [0, Lt): every token of the row is masked */
    for (int v = 0; v < c->V; ++v) r->y[v] = -INFINITY;
  } else {
    process_one(c->x, c->dtype, src * c->ld_row, c->p, c->b, c->dr, l - 1, row, r->y);
  }
  r->nv = ssref_order(r->y, c->V, r->order);
  row_distribution(r->y, r->order, r->nv, c->mode, pf(c->p->temperature, c->b, 1.0f),
                   c->p->top_k ? c->p->top_k[c->b] : 0, pf(c->p->top_p, c->b, 1.0f),
                   pf(c->p->min_p, c->b, 0.0f), c->p->k_cap, r->w, &r->d);
  c->fl |= r->d.flags;
  if (!r->d.greedy) {
    if (r->d.margin_p < c->mg) c->mg = r->d.margin_p;
    if (r->d.margin_m < c->mg) c->mg = r->d.margin_m;
  }
  r->ready = 1;
  return r;
}

/* records the outcome "drafts 1..l-1 accepted, `emit` at position l" */
static void vterminal(vctx_t *c, int l, int32_t emit) {
  int L = c->L;
  if (c->nseq >= SSREF_ADM) return;
  int32_t *s = c->seq + (int64_t)c->nseq * (L + 1);
  for (int j = 0; j <= L; ++j) s[j] = -1;
  for (int j = 0; j < l - 1; ++j) s[j] = c->dr[j];
  s[l - 1] = emit;
  for (int e = 0; e < c->nseq; ++e) {
    if (c->nacc[e] != l - 1) continue;
    if (memcmp(c->seq + (int64_t)e * (L + 1), s, sizeof(int32_t) * (size_t)(L + 1)) == 0) return;
  }
  c->nacc[c->nseq] = l - 1;
  c->nseq++;
}

/* draws at position l over the first ns weights (own pick first) */
static void vdraw(vctx_t *c, int l, const vrow_t *r, const double *w, int ns, double total, double band, double u) {
  int ranks[SSREF_ADM];
  int nr = draw_admissible(w, ns, total, u, band, ranks, SSREF_ADM);
  for (int j = 0; j < nr; ++j) vterminal(c, l, r->order[ranks[j]]);
}

static void vexplore(vctx_t *c, int l) {
  vrow_t *r = vrow_get(c, l);
  const int L = c->L, b = c->b;
  const int64_t pos = c->p->position[b] + (l - 1);
  const int has_draft = (l <= L) && c->dr[l - 1] >= 0 && c->dr[l - 1] < c->V;
  if (r->nv == 0) {  /* empty target row: rejected, no correction token */
    vterminal(c, l, -1);
    return;
  }
  if (r->d.greedy) {
    if (has_draft && c->dr[l - 1] == r->order[0]) vexplore(c, l + 1);
    else vterminal(c, l, r->order[0]);
    return;
  }
  const double u0 = ssref_uniform(c->p->seed[b], (uint32_t)b, pos, 0);
  if (!has_draft) {
    double md;
    (void)draw_index(r->w, r->d.n_s, r->d.Z_s, u0, &md);
    if (md < c->mg) c->mg = md;
    for (int pass = 0; pass < 2; ++pass)
      for (int ns = r->d.ns_lo; ns <= r->d.ns_hi; ++ns) {
        if ((pass == 0) != (ns == r->d.n_s)) continue;
        double Z = prefix_sum(r->w, ns);
        vdraw(c, l, r, r->w, ns, Z, SSREF_NEAR * Z, u0);
      }
    return;
  }
  const int dl = c->dr[l - 1];
  const double qd = qget(c, l, dl);
  const double a = ssref_uniform(c->p->seed[b], (uint32_t)b, pos, 1);
  const double lhs = a * qd;
  int rd = -1;  /* rank of the draft token in the canonical order (top-k range) */
  for (int k = 0; k < r->d.n_k; ++k)
    if (r->order[k] == dl) { rd = k; break; }
  int accept_done = 0;
  for (int pass = 0; pass < 2; ++pass) {
    for (int ns = r->d.ns_lo; ns <= r->d.ns_hi; ++ns) {
      if ((pass == 0) != (ns == r->d.n_s)) continue;
      double Z = prefix_sum(r->w, ns);
      double Pd = (rd >= 0 && rd < ns) ? r->w[rd] / Z : 0.0;
      int acc = Pd > 0.0 && lhs <= Pd;
      int near = 0;
      if (Pd > 0.0) {
        double den = Pd > qd ? Pd : qd;
        double m = fabs(lhs - Pd) / den;
        if (m < c->mg) c->mg = m;
        near = m < SSREF_NEAR;
      }
      for (int branch = 0; branch < 2; ++branch) {
        int take_accept = (branch == 0) ? acc : !acc;
        if (branch == 1 && !near) break;  /* the other branch only near the boundary */
        if (take_accept) {
          if (!accept_done) { accept_done = 1; vexplore(c, l + 1); }
          continue;
        }
        /* residual max(0, P - q) over the kept set, canonical order */
        double R = 0.0;
        for (int k = 0; k < ns; ++k) {
          double P = r->w[k] / Z;
          double v = P - qget(c, l, r->order[k]);
          c->res[k] = v > 0.0 ? v : 0.0;
          R += c->res[k];
        }
        double md;
        if (R > 0.0) {
          (void)draw_index(c->res, ns, R, u0, &md);
          if (ns == r->d.n_s && md < c->mg) c->mg = md;
          vdraw(c, l, r, c->res, ns, R, SSREF_NEAR, u0);
        }
        if (R < SSREF_NEAR) vdraw(c, l, r, r->w, ns, Z, SSREF_NEAR * Z, u0);
      }
    }
  }
}

static int verify_all(const void *x, int dtype, int64_t ld_row, int Lt, const int32_t *row_map,
                      const float *draft_probs, int64_t ld_q, const int32_t *q_idx, const float *q_val, int kq,
                      const int32_t *draft_tokens, int L, const ssref_params *p, int32_t *out_tokens,
                      int32_t *n_acc, int32_t *flags, double *margin, int32_t *adm_seq, int32_t *adm_nacc,
                      int32_t *n_adm, int nthreads) {
  int B = p->B, V = p->V;
#ifdef _OPENMP
  if (nthreads > 0) omp_set_num_threads(nthreads);
#pragma omp parallel for schedule(dynamic, 1)
#endif
  for (int b = 0; b < B; ++b) {
    int cap = p->k_cap > 0 ? p->k_cap : 1;
    vctx_t c;
    memset(&c, 0, sizeof(c));
    c.x = x; c.dtype = dtype; c.ld_row = ld_row; c.q = draft_probs; c.ld_q = ld_q;
    c.qi = q_idx; c.qv = q_val; c.kq = kq;
    c.rmap = row_map; c.Lt = Lt;
    c.dr = draft_tokens + (int64_t)b * L; c.L = L; c.b = b; c.V = V; c.p = p;
    c.mode = effective_mode(p, b);
    c.mg = INFINITY;
    c.rows = (vrow_t *)calloc((size_t)(L + 1), sizeof(vrow_t));
    for (int l = 0; l <= L; ++l) {
      c.rows[l].y = (float *)malloc(sizeof(float) * (size_t)V);
      c.rows[l].order = (int32_t *)malloc(sizeof(int32_t) * (size_t)V);
      c.rows[l].w = (double *)malloc(sizeof(double) * (size_t)cap + 8);
    }
    c.res = (double *)malloc(sizeof(double) * (size_t)cap + 8);
    c.seq = (int32_t *)malloc(sizeof(int32_t) * (size_t)SSREF_ADM * (size_t)(L + 1));
    c.nacc = (int32_t *)malloc(sizeof(int32_t) * SSREF_ADM);
    vexplore(&c, 1);
    for (int l = 0; l <= L; ++l) out_tokens[(int64_t)b * (L + 1) + l] = c.seq[l];
    n_acc[b] = c.nacc[0];
    if (flags) flags[b] = c.fl;
    if (margin) margin[b] = c.mg;
    if (adm_seq) {
      for (int e = 0; e < SSREF_ADM; ++e)
        for (int l = 0; l <= L; ++l)
          adm_seq[((int64_t)b * SSREF_ADM + e) * (L + 1) + l] = e < c.nseq ? c.seq[(int64_t)e * (L + 1) + l] : -1;
    }
    if (adm_nacc)
      for (int e = 0; e < SSREF_ADM; ++e) adm_nacc[(int64_t)b * SSREF_ADM + e] = e < c.nseq ? c.nacc[e] : -1;
    if (n_adm) n_adm[b] = c.nseq;
    for (int l = 0; l <= L; ++l) { free(c.rows[l].y); free(c.rows[l].order); free(c.rows[l].w); }
    free(c.rows); free(c.res); free(c.seq); free(c.nacc);
  }
  return 0;
}

/* Verification against a dense draft distribution q [B, L, ld_q]. */
int ssref_verify(const void *x, int dtype, int64_t ld_row, const float *draft_probs,
                 int64_t ld_q, const int32_t *draft_tokens, int L, const ssref_params *p,
                 int32_t *out_tokens, int32_t *n_acc, int32_t *flags, double *margin,
                 int32_t *adm_seq, int32_t *adm_nacc, int32_t *n_adm, int nthreads) {
  return verify_all(x, dtype, ld_row, L + 1, NULL, draft_probs, ld_q, NULL, NULL, 0, draft_tokens, L, p,
                    out_tokens, n_acc, flags, margin, adm_seq, adm_nacc, n_adm, nthreads);
}

/* Verification against sparse draft distributions: kq (id, probability)
 * entries per draft position, [B, L, kq] each (qget gives their meaning). */
int ssref_verify_sparse(const void *x, int dtype, int64_t ld_row, const int32_t *q_idx, const float *q_val,
                        int kq, const int32_t *draft_tokens, int L, const ssref_params *p,
                        int32_t *out_tokens, int32_t *n_acc, int32_t *flags, double *margin,
                        int32_t *adm_seq, int32_t *adm_nacc, int32_t *n_adm, int nthreads) {
  if (kq < 1) return -1;
  return verify_all(x, dtype, ld_row, L + 1, NULL, NULL, 0, q_idx, q_val, kq, draft_tokens, L, p, out_tokens,
                    n_acc, flags, margin, adm_seq, adm_nacc, n_adm, nthreads);
}

/* Verification of one path through a draft tree (draft-to-target mapping,
 * Appendix C.4): the target computed Lt rows per request (x [B, Lt, ld_row]);
 * path position l (0-based; l = L is the bonus position) is verified against
 * target row row_map[b, l], an entry outside [0, Lt) giving a row with every
 * token masked.  Draft lists are sparse (as ssref_verify_sparse); the
 * penalty history and the grammar rows follow the path. */
int ssref_verify_tree(const void *x, int dtype, int64_t ld_row, int Lt, const int32_t *row_map,
                      const int32_t *q_idx, const float *q_val, int kq, const int32_t *draft_tokens, int L,
                      const ssref_params *p, int32_t *out_tokens, int32_t *n_acc, int32_t *flags,
                      double *margin, int32_t *adm_seq, int32_t *adm_nacc, int32_t *n_adm, int nthreads) {
  if (kq < 1 || Lt < 1 || !row_map) return -1;
  return verify_all(x, dtype, ld_row, Lt, row_map, NULL, 0, q_idx, q_val, kq, draft_tokens, L, p, out_tokens,
                    n_acc, flags, margin, adm_seq, adm_nacc, n_adm, nthreads);
}

/* One row's truncated distribution, for pin tests: fills order[0..n_valid),
 * P[0..n_s) (normalised, canonical order) and the counts/normalisers. */
int ssref_row_distribution(const float *y, int V, uint32_t mode, float temperature, int32_t top_k,
                           float top_p, float min_p, int k_cap, int32_t *order, double *P,
                           int32_t *counts /* n_valid,n_k,n_p,n_m,n_s,greedy,flags,ns_lo,ns_hi */,
                           double *sums /* M, tau, Z_k, Z_s, margin_p, margin_m */) {
  int nv = ssref_order(y, V, order);
  double *w = (double *)malloc(sizeof(double) * (size_t)(k_cap > 0 ? k_cap : 1) + 8);
  dist_t d;
  row_distribution(y, order, nv, mode, temperature, top_k, top_p, min_p, k_cap, w, &d);
  for (int r = 0; r < d.n_s; ++r) P[r] = w[r] / d.Z_s;
  counts[0] = d.n_valid; counts[1] = d.n_k; counts[2] = d.n_p; counts[3] = d.n_m;
  counts[4] = d.n_s; counts[5] = d.greedy; counts[6] = d.flags;
  counts[7] = d.ns_lo; counts[8] = d.ns_hi;
  sums[0] = d.M; sums[1] = d.tau; sums[2] = d.Z_k; sums[3] = d.Z_s;
  sums[4] = d.margin_p; sums[5] = d.margin_m;
  free(w);
  return nv;
}

/* Inverse-CDF draw over given weights (exposed for pin tests). */
int ssref_draw(const double *w, int n, double u) {
  double Z = 0.0;
  for (int r = 0; r < n; ++r) Z += w[r];
  return draw_index(w, n, Z, u, NULL);
}

/* The same draw with its boundary distance (relative to sum w) and its
 * admissible ranks (band SSREF_NEAR relative to sum w; own pick first). */
int ssref_draw_ex(const double *w, int n, double u, double *margin, int32_t *adm, int max, int32_t *n_adm) {
  double Z = prefix_sum(w, n);
  int pick = draw_index(w, n, Z, u, margin);
  int ranks[SSREF_ADM];
  if (max > SSREF_ADM) max = SSREF_ADM;
  int nr = draw_admissible(w, n, Z, u, SSREF_NEAR * Z, ranks, max);
  for (int j = 0; j < nr; ++j) adm[j] = ranks[j];
  *n_adm = nr;
  return pick;
}
