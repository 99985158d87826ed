/*
 * ETA decode oracle -- TEST INFRASTRUCTURE ONLY.
 *
 * A plain, slow, fp64 CPU reference of the Elastic Threshold Attention
 * inference decode path.  Only the test suite, the smoke check and the
 * benchmark's CPU-baseline leg may load it.  The GPU library never calls it
 * and it never calls the GPU library; the two share no source.
 *
 * Every quantity is computed in double precision from inputs that are upcast
 * exactly from their stored type (fp32, or bf16 given as raw 16-bit words).
 *
 * What it follows (paper sections / equations / algorithms):
 *   - block summaries mu_B, sigma_B, M_B:
 *       Sec. "Block-Based Scanning via Dual Metadata Caching" (definitions
 *       of the Dual Probabilistic-Geometric Block Index); population
 *       variance (divide by b), the standard deviation being what is stored
 *       (App. "GQA-Grouped Execution and Compact Metadata Layout").
 *   - threshold predictor: Eq. (tau_pred), tau = concat(q_1..q_H) W + b.
 *   - gate: Eq. (soft_mask) and Eq. (mult_attn): S~ = S * sigmoid(beta (S - tau)),
 *       the diagonal (the query's own key) ungated.
 *   - bound: Eq. (dual_bound_eq), (1/sqrt d) min(<q,mu> + z sqrt(sum q_i^2 sigma_i^2), |q| M).
 *   - selection, top-1 rescue, tail: Alg. "Hardware-Aligned Block-Sparse
 *       Decoding (Inference)" and App. "Top-1 Rescue, Tail Handling, and
 *       Kernel Validation"; slack tau_eff = tau - a for screening and gate
 *       (same algorithm); pinning of the most recent blocks
 *       (App. sub-block envelope paragraph, "lwb").
 *   - half-precision index records: the fp16 centroid / standard deviation
 *       of App. "GQA-Grouped Execution and Compact Metadata Layout",
 *       modelled by rounding the fp64 statistics to the nearest IEEE 754
 *       binary16 value (ties to even) before the bound uses them.
 *   - offline density-matched calibration of static thresholds: App.
 *       "Offline Threshold Calibration via 1/t-Weighted Histograms" and Alg.
 *       "Density-Matched Offline Threshold Calibration": 1/t-weighted score
 *       histogram, target density of the dynamic gates, bisection of the
 *       histogram's density function.
 *   - gated prefill / training forward: App. "Hardware-Aligned Forward
 *       Kernel" (Alg. fwd_kernel) -- causal scores, gates sigmoid(beta (S -
 *       tau_i)) and their row sums R_i, multiplicative (S sigma) or additive
 *       (S + C sigma - C) masking with the diagonal ungated, softmax output
 *       and log-sum-exp, from the definitions (no blocking).
 *   - softmax over the attended set: the plain definition (Sec.
 *       "Elastic Threshold Attention", dense attention output), which the
 *       chunked two-stage reduction of the paper reaches exactly.
 *
 * Readings where the paper is silent or ambiguous:
 *   - a block survives iff bound >= tau_eff (the algorithm's comparison).
 *   - rescue window: blocks [0, min(c, N)); rescue fires iff no block in the
 *     window is selected (threshold or pin); the rescued block is the first
 *     index attaining the maximum bound (strict '>' scan over the window).
 *     A bound that is NaN is never selected and never rescued.
 *   - T < b: no full blocks, no rescue, only the tail is attended.
 *   - T = 0 or nothing attended (rescue disabled, nothing selected, no tail):
 *     the output is the zero vector and the log-sum-exp is -inf.
 *   - tau = -inf: the gate is identically 1 (S~ = S).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#include <omp.h>

#define OR_F32 0
#define OR_BF16 1

static double ld(const void* p, int dt, int64_t i) {
  if (dt == OR_F32) return (double)((const float*)p)[i];
  uint32_t u = ((uint32_t)((const uint16_t*)p)[i]) << 16;
  float f;
  memcpy(&f, &u, 4);
  return (double)f;
}

/* sigmoid, evaluated without overflow for either sign of x. */
static double sigmoid(double x) {
  if (x >= 0.0) return 1.0 / (1.0 + exp(-x));
  double e = exp(x);
  return e / (1.0 + e);
}

/* Eq. (soft_mask) x Eq. (mult_attn): the gated score S * sigma(beta (S - tau)). */
double eta_oracle_gate(double S, double tau, double beta) {
  if (isinf(tau) && tau < 0) return S;
  return S * sigmoid(beta * (S - tau));
}

/*
 * Block summaries for one (sequence, kv head): rows k[t * row_stride + i],
 * t in [0, T).  N = floor(T / b) full blocks; outputs mu[N][d], sigma[N][d],
 * maxnorm[N].  Population statistics, two passes (mean, then deviations).
 */
void eta_oracle_summaries(const void* k, int dt, int64_t row_stride, int64_t T, int d, int b,
                          double* mu, double* sigma, double* maxnorm) {
  int64_t N = T / b;
  for (int64_t j = 0; j < N; ++j) {
    double* m = mu + j * d;
    double* s = sigma + j * d;
    for (int i = 0; i < d; ++i) { m[i] = 0.0; s[i] = 0.0; }
    double best = 0.0;
    for (int t = 0; t < b; ++t) {
      int64_t row = (j * b + t) * row_stride;
      double n2 = 0.0;
      for (int i = 0; i < d; ++i) {
        double x = ld(k, dt, row + i);
        m[i] += x;
        n2 += x * x;
      }
      double n = sqrt(n2);
      if (n > best) best = n;
    }
    for (int i = 0; i < d; ++i) m[i] /= (double)b;
    for (int t = 0; t < b; ++t) {
      int64_t row = (j * b + t) * row_stride;
      for (int i = 0; i < d; ++i) {
        double dv = ld(k, dt, row + i) - m[i];
        s[i] += dv * dv;
      }
    }
    for (int i = 0; i < d; ++i) s[i] = sqrt(s[i] / (double)b);
    maxnorm[j] = best;
  }
}

/*
 * Sub-block envelope variant of sigma (App. "Sub-Block Variance Envelope",
 * Eq. subblock_envelope_appx): per coordinate, the largest over contiguous
 * sub-blocks of b_sub tokens of sqrt(mean over the sub-block of (k_i - mu_i)^2),
 * with mu the full-block centroid.  Same layout as eta_oracle_summaries.
 */
/*
 * Nearest IEEE 754 binary16 value to x, ties to even, returned as a double:
 * 11 significant bits, binades 2^-14 .. 2^15, fixed spacing 2^-24 below 2^-14
 * (subnormals), largest finite 65504; magnitudes of 65520 and above round to
 * infinity.  NaN, infinities and zeros pass through.
 */
double eta_oracle_round_f16(double x) {
  if (isnan(x) || isinf(x) || x == 0.0) return x;
  const double a = fabs(x);
  double r;
  if (a >= 65520.0) {
    r = INFINITY;
  } else {
    int e;
    frexp(a, &e);              /* a in [2^(e-1), 2^e) */
    int ex = e - 1;
    if (ex < -14) ex = -14;    /* subnormal range: the spacing of the lowest binade */
    const double ulp = ldexp(1.0, ex - 10);
    r = nearbyint(a / ulp) * ulp;   /* a / ulp is exact; default mode rounds half to even */
  }
  return copysign(r, x);
}

void eta_oracle_round_f16_array(const double* in, double* out, int64_t n) {
  for (int64_t i = 0; i < n; ++i) out[i] = eta_oracle_round_f16(in[i]);
}

/*
 * Nearest 8-bit E4M3 value to x (1 sign, 4 exponent bits with bias 7, 3
 * fraction bits; the OCP "e4m3fn" format), ties to even, returned as a double:
 * 4 significant bits, binades 2^-6 .. 2^8, fixed spacing 2^-9 below 2^-6
 * (subnormals), largest finite 448.  The format has no infinity; magnitudes
 * of 464 (the tie between 448 and the next step) and above saturate to 448.
 * NaN and zeros pass through.  The FP8 index records (Sec. "Limitations and
 * Conclusion" names FP8 metadata quantisation as a way to cut screening
 * traffic).
 */
double eta_oracle_round_e4m3(double x) {
  if (isnan(x) || x == 0.0) return x;
  const double a = fabs(x);
  double r;
  if (a >= 464.0) {
    r = 448.0;
  } else {
    int e;
    frexp(a, &e);              /* a in [2^(e-1), 2^e) */
    int ex = e - 1;
    if (ex < -6) ex = -6;      /* subnormal range: the spacing of the lowest binade */
    const double ulp = ldexp(1.0, ex - 3);
    r = nearbyint(a / ulp) * ulp;   /* a / ulp is exact; default mode rounds half to even */
  }
  return copysign(r, x);
}

void eta_oracle_round_e4m3_array(const double* in, double* out, int64_t n) {
  for (int64_t i = 0; i < n; ++i) out[i] = eta_oracle_round_e4m3(in[i]);
}

void eta_oracle_envelope(const void* k, int dt, int64_t row_stride, int64_t T, int d, int b,
                         int b_sub, const double* mu, double* env) {
  int64_t N = T / b;
  int nsub = b / b_sub;
  for (int64_t j = 0; j < N; ++j) {
    const double* m = mu + j * d;
    double* e = env + j * d;
    for (int i = 0; i < d; ++i) e[i] = 0.0;
    for (int sb = 0; sb < nsub; ++sb) {
      for (int i = 0; i < d; ++i) {
        double acc = 0.0;
        for (int t = 0; t < b_sub; ++t) {
          int64_t row = (j * b + (int64_t)sb * b_sub + t) * row_stride;
          double dv = ld(k, dt, row + i) - m[i];
          acc += dv * dv;
        }
        double sd = sqrt(acc / (double)b_sub);
        if (sd > e[i]) e[i] = sd;
      }
    }
  }
}

/* Eq. (dual_bound_eq) for one query head and one block. */
double eta_oracle_bound(const double* q, const double* mu, const double* sigma, double M, int d,
                        double z) {
  double dot = 0.0, var = 0.0, qn2 = 0.0;
  for (int i = 0; i < d; ++i) {
    dot += q[i] * mu[i];
    var += q[i] * q[i] * sigma[i] * sigma[i];
    qn2 += q[i] * q[i];
  }
  double gauss = dot + z * sqrt(var);
  double spher = sqrt(qn2) * M;
  double lo = gauss < spher ? gauss : spher;
  if (isnan(gauss) || isnan(spher)) lo = NAN;
  return lo / sqrt((double)d);
}

/* Eq. (tau_pred): tau[b][h] = sum_j qbar[b][j] W[j][h] + bias[h]; W == NULL -> tau = bias. */
void eta_oracle_predict(const void* q, int dt, int B, int Hq, int d, const float* W,
                        const float* bias, double* tau) {
  int64_t J = (int64_t)Hq * d;
  for (int bb = 0; bb < B; ++bb) {
    for (int h = 0; h < Hq; ++h) {
      double acc = bias ? (double)bias[h] : 0.0;
      if (W) {
        for (int64_t j = 0; j < J; ++j) acc += ld(q, dt, (int64_t)bb * J + j) * (double)W[j * Hq + h];
      }
      tau[(int64_t)bb * Hq + h] = acc;
    }
  }
}

/*
 * Block selection for one head: threshold, pins, top-1 rescue.
 * Returns the rescued block index, or -1 when rescue did not fire.
 */
int64_t eta_oracle_select(const double* bound, int64_t N, double tau_eff, int c, int lwb,
                          int screen_all, uint8_t* sel) {
  for (int64_t j = 0; j < N; ++j) sel[j] = (screen_all || bound[j] >= tau_eff) ? 1 : 0;
  for (int64_t j = N - lwb; j < N; ++j)
    if (j >= 0) sel[j] = 1;
  int64_t Wn = c < N ? c : N;
  if (Wn < 1) return -1;
  for (int64_t j = 0; j < Wn; ++j)
    if (sel[j]) return -1;
  double best = -INFINITY;
  int64_t arg = -1;
  for (int64_t j = 0; j < Wn; ++j) {
    if (isnan(bound[j])) continue;
    if (arg < 0 || bound[j] > best) { best = bound[j]; arg = j; }
  }
  if (arg >= 0) sel[arg] = 1;
  return arg;
}

/*
 * Gated softmax attention of one query head over the tokens of the selected
 * full blocks, plus the tail [N b, T) when use_tail.  K, V rows are
 * k[t * row_stride + i].  gate_off = 1 gives plain softmax attention (the dense
 * baseline).  Writes o[d], the log-sum-exp of the gated scores and the number of
 * attended tokens.
 */
void eta_oracle_attend(const double* q, const void* k, const void* v, int dt, int64_t row_stride,
                       int64_t T, int d, int b, const uint8_t* sel, int use_tail, double tau_eff,
                       double beta, int self_ungated, int gate_off, double* o, double* lse,
                       int64_t* count) {
  int64_t N = T / b;
  double scale = 1.0 / sqrt((double)d);
  /* pass 1: gated scores of the attended set and their maximum */
  double* st = (double*)malloc(sizeof(double) * (size_t)(T > 0 ? T : 1));
  uint8_t* in = (uint8_t*)malloc((size_t)(T > 0 ? T : 1));
  double m = -INFINITY;
  int64_t cnt = 0;
  for (int64_t t = 0; t < T; ++t) {
    int64_t j = t / b;
    in[t] = (j < N) ? sel[j] : (uint8_t)(use_tail ? 1 : 0);
    if (!in[t]) continue;
    double S = 0.0;
    for (int i = 0; i < d; ++i) S += q[i] * ld(k, dt, t * row_stride + i);
    S *= scale;
    double Sg = (gate_off || (self_ungated && t == T - 1)) ? S : eta_oracle_gate(S, tau_eff, beta);
    st[t] = Sg;
    if (Sg > m) m = Sg;
    ++cnt;
  }
  for (int i = 0; i < d; ++i) o[i] = 0.0;
  if (cnt == 0) {
    *lse = -INFINITY;
    *count = 0;
    free(st);
    free(in);
    return;
  }
  /* pass 2: normalised weights and the weighted value sum */
  double Z = 0.0;
  for (int64_t t = 0; t < T; ++t) {
    if (!in[t]) continue;
    double w = exp(st[t] - m);
    Z += w;
    for (int i = 0; i < d; ++i) o[i] += w * ld(v, dt, t * row_stride + i);
  }
  for (int i = 0; i < d; ++i) o[i] /= Z;
  *lse = m + log(Z);
  *count = cnt;
  free(st);
  free(in);
}

/*
 * Screening-quality diagnostics of one head (Tab. "index_quality" in App. "GQA
 * Union Loading and Variance Dilution at Coarse Block Sizes"; the block false
 * negatives and recall of above-threshold keys discussed in Sec. "Block
 * Granularity and GQA Union Loading").  From the brute-force scores
 * S_t = <q, k_t> / sqrt(d) of every key:
 *   blockmax[j]  max over block j's keys of S_t (full blocks j < N)
 *   qual[0]  positive blocks:  blockmax[j] >= tau_eff
 *   qual[1]  false negatives:  positive and not selected
 *   qual[2]  false positives:  selected and not positive
 *   qual[3]  selected blocks
 *   qual[4]  above-threshold keys of the full blocks: S_t >= tau_eff
 *   qual[5]  those among them that are attended (their block is selected)
 *   missed  the softmax mass of the rejected full blocks under gated attention
 *           over every key (the no-screening distribution of Sec. "Elastic
 *           Threshold Attention": sum over rejected keys of exp(S~_t) / sum over
 *           all T keys), S~ gated with tau_eff as in eta_oracle_attend
 * The tail [N b, T) is never screened, so it enters only the denominator of the
 * missed mass.  blockmax may be NULL.
 */
void eta_oracle_screen_quality(const double* q, const void* k, int dt, int64_t row_stride,
                               int64_t T, int d, int b, const uint8_t* sel, double tau_eff,
                               double beta, int self_ungated, int gate_off, double* blockmax,
                               int64_t* qual, double* missed) {
  int64_t N = T / b;
  double scale = 1.0 / sqrt((double)d);
  for (int f = 0; f < 6; ++f) qual[f] = 0;
  *missed = 0.0;
  if (T <= 0) return;
  double* sg = (double*)malloc(sizeof(double) * (size_t)T);
  double m = -INFINITY;
  for (int64_t j = 0; j <= N; ++j) {
    int64_t t0 = j * b, t1 = j < N ? t0 + b : T;
    double bmax = -INFINITY;
    int64_t above = 0;
    for (int64_t t = t0; t < t1; ++t) {
      double S = 0.0;
      for (int i = 0; i < d; ++i) S += q[i] * ld(k, dt, t * row_stride + i);
      S *= scale;
      if (S > bmax) bmax = S;
      if (S >= tau_eff) ++above;
      double Sg = (gate_off || (self_ungated && t == T - 1)) ? S : eta_oracle_gate(S, tau_eff, beta);
      sg[t] = Sg;
      if (Sg > m) m = Sg;
    }
    if (j == N) break;
    int positive = bmax >= tau_eff;
    if (blockmax) blockmax[j] = bmax;
    qual[0] += positive;
    qual[1] += positive && !sel[j];
    qual[2] += !positive && sel[j];
    qual[3] += sel[j] != 0;
    qual[4] += above;
    qual[5] += sel[j] ? above : 0;
  }
  double Z = 0.0, Zrej = 0.0;
  for (int64_t t = 0; t < T; ++t) {
    double w = exp(sg[t] - m);
    Z += w;
    if (t < N * b && !sel[t / b]) Zrej += w;
  }
  *missed = Z > 0.0 ? Zrej / Z : 0.0;
  free(sg);
}

/* ---------------------------------------------------------------- batched */

typedef struct {
  int32_t B, Hq, Hkv, d, b;
  int64_t T_cap;               /* rows per (sequence, kv head) in K and V */
  int32_t q_dtype, kv_dtype;   /* OR_F32 / OR_BF16 */
  const void* q;               /* [B][Hq][d] */
  const void* k;               /* [B][Hkv][T_cap][d] */
  const void* v;               /* [B][Hkv][T_cap][d] */
  const int32_t* seq_lens;     /* [B] */
  const double* tau;           /* [B][Hq] predicted or constant threshold */
  double beta, z, a;           /* gate temperature, z-score, slack (tau_eff = tau - a) */
  int32_t c;                   /* rescue window in blocks (0 disables rescue) */
  int32_t lwb;                 /* pinned most-recent full blocks */
  int32_t self_ungated;        /* key T-1 keeps S~ = S */
  int32_t screen_all;          /* every full block selected */
  int32_t gate_off;            /* plain softmax (dense baseline) */
  int32_t bounds_only;         /* stop after the bounds (no selection, no attention) */
  /* optional precomputed summaries [B][Hkv][N_cap][d], [B][Hkv][N_cap]; NULL -> computed here */
  const double* mu;
  const double* sigma;
  const double* maxnorm;
  /* optional external block mask [B][Hq][N_cap] replacing bounds + selection */
  const uint8_t* sel_in;
  /* optional subset of rows (b * Hq + h); NULL -> every row */
  const int32_t* rows;
  int32_t n_rows;
  int32_t n_threads;           /* <= 0: OpenMP default */
  /* outputs (any may be NULL except o) */
  double* o;                   /* [B][Hq][d] */
  uint8_t* sel;                /* [B][Hq][N_cap] */
  double* bounds;              /* [B][Hq][N_cap] (NaN beyond N_b) */
  int64_t* counts;             /* [B][Hq] attended tokens */
  double* lse;                 /* [B][Hq] */
  int64_t* rescued;            /* [B][Hq] rescued block or -1 */
  /* optional screening-quality diagnostics (eta_oracle_screen_quality); NULL: skipped */
  double* blockmax;            /* [B][Hq][N_cap] brute-force block maxima (NaN beyond N_b) */
  int64_t* quality;            /* [B][Hq][6] */
  double* missed;              /* [B][Hq] */
} eta_oracle_problem;

static const void* off(const void* p, int dt, int64_t elems) {
  return (const char*)p + elems * (dt == OR_F32 ? 4 : 2);
}

int eta_oracle_decode(const eta_oracle_problem* P) {
  if (P->Hkv <= 0 || P->Hq % P->Hkv || P->b <= 0 || P->d <= 0) return 1;
  const int64_t Ncap = P->T_cap / P->b;
  const int G = P->Hq / P->Hkv;
  const int d = P->d;
  const int64_t nrows = P->rows ? P->n_rows : (int64_t)P->B * P->Hq;
  const int64_t nbg = (int64_t)P->B * P->Hkv;
  const int nthr = P->n_threads > 0 ? P->n_threads : omp_get_max_threads();

  /* block summaries of the (sequence, kv head) pairs the requested rows use */
  uint8_t* need = (uint8_t*)calloc((size_t)nbg, 1);
  for (int64_t r = 0; r < nrows; ++r) {
    int32_t row = P->rows ? P->rows[r] : (int32_t)r;
    need[(row / P->Hq) * P->Hkv + (row % P->Hq) / G] = 1;
  }
  const double* mu = P->mu;
  const double* sg = P->sigma;
  const double* mx = P->maxnorm;
  double *own_mu = NULL, *own_sg = NULL, *own_mx = NULL;
  if (mu == NULL && P->sel_in == NULL) {
    own_mu = (double*)malloc(sizeof(double) * (size_t)(nbg * Ncap * d + 1));
    own_sg = (double*)malloc(sizeof(double) * (size_t)(nbg * Ncap * d + 1));
    own_mx = (double*)malloc(sizeof(double) * (size_t)(nbg * Ncap + 1));
#pragma omp parallel for schedule(dynamic, 1) num_threads(nthr)
    for (int64_t bg = 0; bg < nbg; ++bg) {
      if (!need[bg]) continue;
      int64_t T = P->seq_lens[bg / P->Hkv];
      if (T > P->T_cap) T = P->T_cap;
      if (T < 0) T = 0;
      eta_oracle_summaries(off(P->k, P->kv_dtype, bg * P->T_cap * d), P->kv_dtype, d, T, d, P->b,
                           own_mu + bg * Ncap * d, own_sg + bg * Ncap * d, own_mx + bg * Ncap);
    }
    mu = own_mu;
    sg = own_sg;
    mx = own_mx;
  }

  /* per query head: bounds -> selection -> rescue -> gated attention */
#pragma omp parallel for schedule(dynamic, 1) num_threads(nthr)
  for (int64_t r = 0; r < nrows; ++r) {
    int32_t row = P->rows ? P->rows[r] : (int32_t)r;
    int bb = row / P->Hq, h = row % P->Hq, g = h / G;
    int64_t bg = (int64_t)bb * P->Hkv + g;
    int64_t T = P->seq_lens[bb];
    if (T > P->T_cap) T = P->T_cap;
    if (T < 0) T = 0;
    int64_t N = T / P->b;
    double* qh = (double*)malloc(sizeof(double) * (size_t)d);
    for (int i = 0; i < d; ++i) qh[i] = ld(P->q, P->q_dtype, (int64_t)row * d + i);
    double tau_eff = P->tau[row] - P->a;
    uint8_t* sel = (uint8_t*)calloc((size_t)(Ncap + 1), 1);
    int64_t resc = -1;
    if (P->sel_in) {
      memcpy(sel, P->sel_in + (int64_t)row * Ncap, (size_t)N);
    } else {
      double* bnd = (double*)malloc(sizeof(double) * (size_t)(N + 1));
      for (int64_t j = 0; j < N; ++j)
        bnd[j] = eta_oracle_bound(qh, mu + (bg * Ncap + j) * d, sg + (bg * Ncap + j) * d,
                                  mx[bg * Ncap + j], d, P->z);
      if (!P->bounds_only) resc = eta_oracle_select(bnd, N, tau_eff, P->c, P->lwb, P->screen_all, sel);
      if (P->bounds) {
        for (int64_t j = 0; j < Ncap; ++j) P->bounds[(int64_t)row * Ncap + j] = j < N ? bnd[j] : NAN;
      }
      free(bnd);
    }
    if (P->bounds_only) {
      free(sel);
      free(qh);
      continue;
    }
    double lse;
    int64_t cnt;
    const int64_t kvoff = bg * P->T_cap * d;
    eta_oracle_attend(qh, off(P->k, P->kv_dtype, kvoff), off(P->v, P->kv_dtype, kvoff), P->kv_dtype,
                      d, T, d, P->b, sel, 1, tau_eff, P->beta, P->self_ungated, P->gate_off,
                      P->o + (int64_t)row * d, &lse, &cnt);
    if (P->sel) memcpy(P->sel + (int64_t)row * Ncap, sel, (size_t)Ncap);
    if (P->counts) P->counts[row] = cnt;
    if (P->lse) P->lse[row] = lse;
    if (P->quality) {
      double* bm = P->blockmax ? P->blockmax + (int64_t)row * Ncap : NULL;
      if (bm)
        for (int64_t j = 0; j < Ncap; ++j) bm[j] = NAN;
      eta_oracle_screen_quality(qh, off(P->k, P->kv_dtype, kvoff), P->kv_dtype, d, T, d, P->b, sel,
                                tau_eff, P->beta, P->self_ungated, P->gate_off, bm,
                                P->quality + (int64_t)row * 6, P->missed + row);
    }
    if (P->rescued) P->rescued[row] = resc;
    free(sel);
    free(qh);
  }
  free(own_mu);
  free(own_sg);
  free(own_mx);
  free(need);
  return 0;
}

/*
 * Offline calibration, accumulation (App. "Offline Threshold Calibration via
 * 1/t-Weighted Histograms"; Alg. "Density-Matched Offline Threshold
 * Calibration").  Every calibration sequence x has T steps; at step t
 * (0-based) the query q_t of head h sees the t + 1 causal keys k_0..k_t of kv
 * head h / G, and each causal pair weighs 1 / (t + 1) (the paper's 1/t with
 * steps counted from one).  For each pair:
 *   S   = <q_t, k_s> / sqrt(d)                       raw score
 *   bin = floor((S - lo) / w), w = (hi - lo) / nb     clamped to [0, nb)
 *   hist[h][bin] += 1 / (t + 1);  dens[h] += sigmoid(beta (S - tau[x][h][t])) / (t + 1)
 * and total[h] sums the weights (N T).  hist_lo / hist_hi (may be NULL) bin
 * the same pairs at S - delta and S + delta, delta = gamma * sum_i |q_ti k_si|
 * / sqrt(d) + eps_abs: the interval any computation of S within that error
 * bound falls into.  Layouts: q [N][Hq][T][d], k [N][Hkv][T][d] (fp32 or bf16
 * words), tau [N][Hq][T]; outputs [Hq][nb] and [Hq].
 */
static int calib_bin(double S, double lo, double w, int nb) {
  double f = floor((S - lo) / w);
  if (!(f >= 0.0)) return 0;            /* also NaN */
  if (f >= (double)nb) return nb - 1;
  return (int)f;
}

void eta_oracle_calib_hist(const void* q, const void* k, int dt, const double* tau, int N, int Hq,
                           int Hkv, int T, int d, double beta, double lo, double hi, int nb,
                           double gamma, double eps_abs, double* hist, double* hist_lo,
                           double* hist_hi, double* dens, double* total) {
  const int G = Hq / Hkv;
  const double w = (hi - lo) / (double)nb;
  const double scale = 1.0 / sqrt((double)d);
#pragma omp parallel for schedule(dynamic, 1)
  for (int h = 0; h < Hq; ++h) {
    double* H = hist + (int64_t)h * nb;
    double* HL = hist_lo ? hist_lo + (int64_t)h * nb : NULL;
    double* HH = hist_hi ? hist_hi + (int64_t)h * nb : NULL;
    for (int b = 0; b < nb; ++b) {
      H[b] = 0.0;
      if (HL) HL[b] = 0.0;
      if (HH) HH[b] = 0.0;
    }
    double dsum = 0.0, wsum = 0.0;
    for (int x = 0; x < N; ++x) {
      const int64_t qb = (((int64_t)x * Hq + h) * T) * d;
      const int64_t kb = (((int64_t)x * Hkv + h / G) * T) * d;
      for (int t = 0; t < T; ++t) {
        const double wt = 1.0 / (double)(t + 1);
        const double tau_t = tau[((int64_t)x * Hq + h) * T + t];
        for (int s2 = 0; s2 <= t; ++s2) {
          double dot = 0.0, mag = 0.0;
          for (int i = 0; i < d; ++i) {
            const double a = ld(q, dt, qb + (int64_t)t * d + i);
            const double c = ld(k, dt, kb + (int64_t)s2 * d + i);
            dot += a * c;
            mag += fabs(a * c);
          }
          const double S = dot * scale;
          H[calib_bin(S, lo, w, nb)] += wt;
          if (HL || HH) {
            const double delta = gamma * mag * scale + eps_abs;
            if (HL) HL[calib_bin(S - delta, lo, w, nb)] += wt;
            if (HH) HH[calib_bin(S + delta, lo, w, nb)] += wt;
          }
          dsum += sigmoid(beta * (S - tau_t)) * wt;
          wsum += wt;
        }
      }
    }
    dens[h] = dsum;
    total[h] = wsum;
  }
}

/*
 * The histogram's density function g(c) = sum_b H_b sigmoid(beta (s_b - c)),
 * H normalised to sum one, s_b = lo + (b + 1/2) w the bin centres.
 */
double eta_oracle_calib_g(const double* hist, int nb, double lo, double hi, double beta, double c) {
  const double w = (hi - lo) / (double)nb;
  double tot = 0.0, g = 0.0;
  for (int b = 0; b < nb; ++b) tot += hist[b];
  for (int b = 0; b < nb; ++b) g += hist[b] * sigmoid(beta * (lo + ((double)b + 0.5) * w - c));
  return g / tot;
}

/*
 * Static threshold c with g(c) = target by bisection (g falls strictly from
 * one to zero, beta > 0).  Bracket [lo - 60 / beta, hi + 60 / beta]; halves
 * until the midpoint equals an end; a target outside g's range on the bracket
 * gives the nearer end.
 */
double eta_oracle_calib_solve(const double* hist, int nb, double lo, double hi, double beta,
                              double target) {
  double a = lo - 60.0 / beta, b = hi + 60.0 / beta;
  for (int it = 0; it < 4096; ++it) {
    const double m = 0.5 * (a + b);
    if (m <= a || m >= b) break;
    if (eta_oracle_calib_g(hist, nb, lo, hi, beta, m) > target) a = m; else b = m;
  }
  return 0.5 * (a + b);
}

/*
 * Gated prefill / training forward (App. "Hardware-Aligned Forward Kernel"):
 * for every sequence b, query head h (kv head h / G) and position i < T_b,
 * over the causal keys j <= i:
 *   S_ij     = s <q_i, k_j>,  s = 1 / sqrt(d)
 *   sigma_ij = sigmoid(beta (S_ij - tau_i)),     R_i = sum_{j <= i} sigma_ij
 *   S~_ij    = S_ij sigma_ij (multiplicative) or S_ij + C sigma_ij - C
 *              (additive); S~_ii = S_ii (the diagonal is never gated)
 *   O_i      = sum_j exp(S~_ij - L_i) v_j,  L_i = log sum_j exp(S~_ij)
 * Layouts q, O [B][Hq][T][d], k, v [B][Hkv][T][d] (fp32 or bf16 words),
 * tau, R, L [B][Hq][T].  Rows i >= T_b: O = 0, R = 0, L = -inf.
 */
/* One row (b, h, i) of the above; st is scratch of at least i + 1 doubles. */
static void prefill_row(const void* q, const void* k, const void* v, int dt, const double* tau,
                        const int32_t* seq_lens, int Hq, int Hkv, int T, int d, double beta,
                        int additive, double C, int b, int h, int i, double* o, double* R_out,
                        double* L_out, double* st) {
  const int G = Hq / Hkv;
  const double scale = 1.0 / sqrt((double)d);
  const int Tb = seq_lens[b] < 0 ? 0 : (seq_lens[b] > T ? T : seq_lens[b]);
  const int64_t qb = (((int64_t)b * Hq + h) * T) * d;
  const int64_t kb = (((int64_t)b * Hkv + h / G) * T) * d;
  const int64_t row = ((int64_t)b * Hq + h) * T + i;
  for (int c = 0; c < d; ++c) o[c] = 0.0;
  if (i >= Tb) {
    *R_out = 0.0;
    *L_out = -INFINITY;
    return;
  }
  double rsum = 0.0, m = -INFINITY;
  for (int j = 0; j <= i; ++j) {
    double dot = 0.0;
    for (int c = 0; c < d; ++c)
      dot += ld(q, dt, qb + (int64_t)i * d + c) * ld(k, dt, kb + (int64_t)j * d + c);
    const double S = dot * scale;
    const double g = sigmoid(beta * (S - tau[row]));
    rsum += g;
    double Sg = additive ? S + C * g - C : S * g;
    if (j == i) Sg = S;
    st[j] = Sg;
    if (Sg > m) m = Sg;
  }
  double l = 0.0;
  for (int j = 0; j <= i; ++j) {
    const double w = exp(st[j] - m);
    l += w;
    for (int c = 0; c < d; ++c) o[c] += w * ld(v, dt, kb + (int64_t)j * d + c);
  }
  for (int c = 0; c < d; ++c) o[c] /= l;
  *R_out = rsum;
  *L_out = m + log(l);
}

void eta_oracle_prefill(const void* q, const void* k, const void* v, int dt, const double* tau,
                        const int32_t* seq_lens, int B, int Hq, int Hkv, int T, int d, double beta,
                        int additive, double C, double* O, double* R, double* L) {
#pragma omp parallel for collapse(2) schedule(dynamic, 1)
  for (int b = 0; b < B; ++b) {
    for (int h = 0; h < Hq; ++h) {
      double* st = (double*)malloc(sizeof(double) * (size_t)(T > 0 ? T : 1));
      for (int i = 0; i < T; ++i) {
        const int64_t row = ((int64_t)b * Hq + h) * T + i;
        prefill_row(q, k, v, dt, tau, seq_lens, Hq, Hkv, T, d, beta, additive, C, b, h, i,
                    O + row * d, R + row, L + row, st);
      }
      free(st);
    }
  }
}

/*
 * The same outputs for n selected rows only: rows[3 r .. 3 r + 2] = (b, h, i);
 * O [n][d], R, L [n].  For checking long sequences on a sample of rows.
 */
void eta_oracle_prefill_rows(const void* q, const void* k, const void* v, int dt,
                             const double* tau, const int32_t* seq_lens, int B, int Hq, int Hkv,
                             int T, int d, double beta, int additive, double C,
                             const int32_t* rows, int n, double* O, double* R, double* L) {
  (void)B;
#pragma omp parallel for schedule(dynamic, 1)
  for (int r = 0; r < n; ++r) {
    double* st = (double*)malloc(sizeof(double) * (size_t)(T > 0 ? T : 1));
    prefill_row(q, k, v, dt, tau, seq_lens, Hq, Hkv, T, d, beta, additive, C, rows[3 * r],
                rows[3 * r + 1], rows[3 * r + 2], O + (int64_t)r * d, R + r, L + r, st);
    free(st);
  }
}
