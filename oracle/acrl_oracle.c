/*
 * acrl_oracle.c -- plain CPU oracle for the ACRL scoring / discrepancy path.
 *
 * TEST INFRASTRUCTURE ONLY (tests, the smoke check and the benchmark's CPU
 * baseline may use it; the product path never does).  Written from the
 * definitions in the ACRL paper, slow on purpose: straight loops, fp64
 * arithmetic, no blocking, no fusion, no reordering beyond what the
 * definitions state.  Parallelism is only across independent tokens / rows.
 *
 * Build: gcc -O2 -std=c11 -fopenmp -fPIC -shared (no -ffast-math; x86-64 SSE
 * arithmetic, FLT_EVAL_METHOD == 0, so float operations round to float).
 *
 * Readings of passages the paper leaves open are the ones listed in the
 * design notes of this repository; each function states the one it takes.
 */
#include "acrl_oracle.h"

#include <float.h>
#include <math.h>
#include <stdlib.h>
#include <string.h>

#if FLT_EVAL_METHOD != 0
#error "the oracle needs float arithmetic evaluated in float (SSE)"
#endif

/* ------------------------------------------------------------------ */
/* Number formats                                                       */
/* ------------------------------------------------------------------ */

/* bfloat16 is the upper half of an IEEE binary32. */
float acrl_ref_bf16_to_float(uint16_t bits) {
  uint32_t u = (uint32_t)bits << 16;
  float f;
  memcpy(&f, &u, sizeof f);
  return f;
}

/* Round a non-negative double that is exact (no prior rounding) to an
 * integer: nearest with ties to even, or toward zero. */
static double round_integer(double v, int rounding) {
  if (rounding == REF_ROUND_TOWARD_ZERO) return trunc(v);
  return nearbyint(v); /* default environment: round-to-nearest-even */
}

/*
 * OCP 8-bit floating point, E4M3 variant (the FP8 of the paper's inference
 * engine, Sec. 2.1 / 5.1): 1 sign bit, 4 exponent bits with bias 7, 3
 * mantissa bits; no infinities; S.1111.111 is NaN; largest finite 448.
 *   normal    (E in 1..15): (1 + m/8) * 2^(E-7)
 *   subnormal (E == 0)    : (m/8) * 2^-6 = m * 2^-9
 * Encoding (the reading taken for "nearest-around" FP8): round |x| to the
 * nearest representable value, ties to the even mantissa; results at or
 * above 448 saturate to 448 (so do infinities); NaN maps to S.1111.111.
 * Toward-zero (the stress test's trunc(x/S)) truncates the magnitude.
 */
uint8_t acrl_ref_e4m3_encode(float x, int rounding) {
  uint32_t bits;
  memcpy(&bits, &x, sizeof bits);
  const uint8_t sign = (bits >> 31) ? 0x80u : 0x00u;
  if (isnan(x)) return (uint8_t)(sign | 0x7Fu);
  const double a = fabs((double)x);
  if (a >= 448.0) return (uint8_t)(sign | 0x7Eu); /* saturate (incl. inf) */

  if (a < ldexp(1.0, -6)) {
    /* subnormal band: a = m * 2^-9 with m real in [0, 8) */
    const double m = round_integer(a * 512.0, rounding); /* exact scaling */
    /* m == 8 is the carry into the smallest normal, code 0x08 */
    return (uint8_t)(sign | (uint8_t)m);
  }
  int e2;
  (void)frexp(a, &e2);          /* a = f * 2^e2, f in [0.5, 1) */
  int E = e2 - 1;               /* a in [2^E, 2^(E+1)), E in [-6, 8] */
  const double frac = (a / ldexp(1.0, E) - 1.0) * 8.0; /* exact, in [0, 8) */
  double m = round_integer(frac, rounding);
  if (m == 8.0) { /* mantissa overflow carries into the exponent */
    m = 0.0;
    E += 1;
  }
  /* a < 448 guarantees (E, m) <= (8, 6) here */
  return (uint8_t)(sign | (uint8_t)((E + 7) << 3) | (uint8_t)m);
}

double acrl_ref_e4m3_decode(uint8_t code) {
  const int s = code >> 7;
  const int E = (code >> 3) & 0xF;
  const int m = code & 0x7;
  if (E == 15 && m == 7) return NAN;
  const double mag = (E == 0) ? ldexp((double)m, -9) : ldexp(8.0 + m, E - 10);
  return s ? -mag : mag;
}

/* OCP E8M0: an unsigned power-of-two exponent with bias 127; 0xFF is NaN. */
double acrl_ref_e8m0_decode(uint8_t code) {
  if (code == 0xFF) return NAN;
  return ldexp(1.0, (int)code - 127);
}

void acrl_ref_e4m3_encode_array(const float* x, int64_t n, int rounding, uint8_t* out) {
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < n; ++i) out[i] = acrl_ref_e4m3_encode(x[i], rounding);
}

/* ------------------------------------------------------------------ */
/* a1 / a2: FP8 quantization                                            */
/* ------------------------------------------------------------------ */

/* Largest magnitude over n bf16 values with stride 1 (NaNs are skipped). */
static float amax_bf16(const uint16_t* x, int64_t n) {
  float amax = 0.0f;
  for (int64_t k = 0; k < n; ++k) {
    const float v = fabsf(acrl_ref_bf16_to_float(x[k]));
    if (v > amax) amax = v;
  }
  return amax;
}

/* Scale of a per-tensor / per-row group (Sec. 5.1, per-token activations and
 * per-channel weights): s = amax / 448 in fp32, so that the largest
 * magnitude maps to the largest e4m3 value; an all-zero group takes s = 1.
 * Elements are encoded from the fp32 quotient x / s (correctly rounded
 * divide, then the e4m3 rounding). */
static float fp8_group_scale(float amax) {
  return (amax == 0.0f) ? 1.0f : amax / 448.0f;
}

/* MX shared scale of one 32-element block (OCP Microscaling v1.0 rule, the
 * reading taken for the paper's MXFP8): X = 2^(floor(log2 amax) - 8), where
 * 8 is the exponent of e4m3's largest power of two; stored as E8M0
 * (biased by 127, clamped to [0, 254]); an all-zero block stores 0. */
static uint8_t mx_block_scale(float amax) {
  if (amax == 0.0f) return 0;
  int e2;
  (void)frexp((double)amax, &e2); /* amax = f * 2^e2, f in [0.5, 1) */
  const int floor_log2 = e2 - 1;
  int code = floor_log2 - 8 + 127;
  if (code < 0) code = 0;
  if (code > 254) code = 254;
  return (uint8_t)code;
}

int acrl_ref_quantize_fp8(const uint16_t* x, int64_t rows, int64_t cols, int64_t ld,
                          int scaling, int rounding, uint8_t* q, void* scales) {
  if (!x || !q || !scales || rows < 0 || cols < 0 || ld < cols) return -1;
  if (rounding != REF_ROUND_NEAREST_EVEN && rounding != REF_ROUND_TOWARD_ZERO) return -1;

  if (scaling == REF_PER_TENSOR) {
    float amax = 0.0f;
    for (int64_t r = 0; r < rows; ++r) {
      const float a = amax_bf16(x + r * ld, cols);
      if (a > amax) amax = a;
    }
    const float s = fp8_group_scale(amax);
    ((float*)scales)[0] = s;
    for (int64_t r = 0; r < rows; ++r)
      for (int64_t k = 0; k < cols; ++k)
        q[r * cols + k] = acrl_ref_e4m3_encode(acrl_ref_bf16_to_float(x[r * ld + k]) / s, rounding);
    return 0;
  }
  if (scaling == REF_PER_ROW) {
    for (int64_t r = 0; r < rows; ++r) {
      const float s = fp8_group_scale(amax_bf16(x + r * ld, cols));
      ((float*)scales)[r] = s;
      for (int64_t k = 0; k < cols; ++k)
        q[r * cols + k] = acrl_ref_e4m3_encode(acrl_ref_bf16_to_float(x[r * ld + k]) / s, rounding);
    }
    return 0;
  }
  if (scaling == REF_MX32) {
    if (cols % 32 != 0) return -1;
    const int64_t nb = cols / 32;
    uint8_t* sc = (uint8_t*)scales;
    for (int64_t r = 0; r < rows; ++r) {
      for (int64_t b = 0; b < nb; ++b) {
        const uint16_t* blk = x + r * ld + 32 * b;
        const uint8_t code = mx_block_scale(amax_bf16(blk, 32));
        sc[r * nb + b] = code;
        /* element = x / X with X = 2^(code-127): an exact power-of-two scaling */
        for (int k = 0; k < 32; ++k) {
          const float v = ldexpf(acrl_ref_bf16_to_float(blk[k]), 127 - (int)code);
          q[r * cols + 32 * b + k] = acrl_ref_e4m3_encode(v, rounding);
        }
      }
    }
    return 0;
  }
  return -1;
}

/* ------------------------------------------------------------------ */
/* a3 / a4: logits                                                      */
/* ------------------------------------------------------------------ */

/* Training policy pi in BF16: z_v = (sum_k h_k W[v,k]) / tau, with the exact
 * bf16 values summed in double.  W is the LM head [V, d], row v = vocab v. */
int acrl_ref_logits_pi(const uint16_t* h_row, const uint16_t* w, int64_t d, int64_t V,
                       double inv_temperature, double* z) {
  if (!h_row || !w || !z || d <= 0 || V <= 0) return -1;
  double* h = (double*)malloc((size_t)d * sizeof(double));
  if (!h) return -1;
  for (int64_t k = 0; k < d; ++k) h[k] = acrl_ref_bf16_to_float(h_row[k]);
  for (int64_t v = 0; v < V; ++v) {
    const uint16_t* wr = w + v * d;
    double acc = 0.0;
    for (int64_t k = 0; k < d; ++k) acc += h[k] * (double)acrl_ref_bf16_to_float(wr[k]);
    z[v] = acc * inv_temperature;
  }
  free(h);
  return 0;
}

/* Inference policy mu with FP8 operands:
 *   per-tensor / per-row: z_v = s_a * s_w[v] * (sum_k qa_k * qw[v,k]) / tau
 *   MX32:                 z_v = sum_b 2^(ea_b-127) 2^(ew[v,b]-127) (sum_{k in b} qa_k qw[v,k]) / tau
 * where qa, qw are the decoded e4m3 values; every product and every block
 * sum is exact in double. */
int acrl_ref_logits_mu(const uint8_t* hq_row, const void* row_scale, const uint8_t* wq,
                       const void* wq_scales, int scaling, int64_t d, int64_t V,
                       double inv_temperature, double* z) {
  if (!hq_row || !row_scale || !wq || !wq_scales || !z || d <= 0 || V <= 0) return -1;
  if (scaling == REF_MX32 && d % 32 != 0) return -1;
  if (scaling != REF_PER_TENSOR && scaling != REF_PER_ROW && scaling != REF_MX32) return -1;
  /* value of every code, from the decoder above (a table only saves calls) */
  double dec[256];
  for (int c = 0; c < 256; ++c) dec[c] = acrl_ref_e4m3_decode((uint8_t)c);
  double* a = (double*)malloc((size_t)d * sizeof(double));
  if (!a) return -1;
  for (int64_t k = 0; k < d; ++k) a[k] = dec[hq_row[k]];

  if (scaling == REF_PER_TENSOR || scaling == REF_PER_ROW) {
    const double s_a = *(const float*)row_scale;
    for (int64_t v = 0; v < V; ++v) {
      const double s_w = (scaling == REF_PER_TENSOR) ? ((const float*)wq_scales)[0]
                                                     : ((const float*)wq_scales)[v];
      const uint8_t* wr = wq + v * d;
      double acc = 0.0;
      for (int64_t k = 0; k < d; ++k) acc += a[k] * dec[wr[k]];
      z[v] = s_a * s_w * acc * inv_temperature;
    }
  } else {
    const int64_t nb = d / 32;
    const uint8_t* ea = (const uint8_t*)row_scale;
    const uint8_t* ew = (const uint8_t*)wq_scales;
    for (int64_t v = 0; v < V; ++v) {
      const uint8_t* wr = wq + v * d;
      double acc = 0.0;
      for (int64_t b = 0; b < nb; ++b) {
        double blk = 0.0;
        for (int64_t k = 32 * b; k < 32 * b + 32; ++k) blk += a[k] * dec[wr[k]];
        acc += acrl_ref_e8m0_decode(ea[b]) * acrl_ref_e8m0_decode(ew[v * nb + b]) * blk;
      }
      z[v] = acc * inv_temperature;
    }
  }
  free(a);
  return 0;
}

/* ------------------------------------------------------------------ */
/* Log-softmax statistics of one token                                  */
/* ------------------------------------------------------------------ */

/* For logits z over the vocabulary and the sampled token id:
 *   lse = log sum_v exp(z_v)            (two passes: max, then shifted sum)
 *   logp = z_id - lse                   = log pi(a_t) (or log mu(a_t))
 *   entropy = sum_v p_v (lse - z_v),  p_v = exp(z_v - lse)   (-sum p log p) */
void acrl_ref_token_stats(const double* z, int64_t V, int32_t id,
                          double* lse, double* logp, double* entropy) {
  double m = -INFINITY;
  for (int64_t v = 0; v < V; ++v)
    if (z[v] > m) m = z[v];
  double s = 0.0;
  for (int64_t v = 0; v < V; ++v) s += exp(z[v] - m);
  const double l = m + log(s);
  double h = 0.0;
  for (int64_t v = 0; v < V; ++v) h += exp(z[v] - l) * (l - z[v]);
  if (lse) *lse = l;
  if (logp) *logp = (id >= 0 && id < V) ? z[id] - l : NAN;
  if (entropy) *entropy = h;
}

/* Scale of row r of the quantized activations, as passed to logits_mu. */
static const void* row_scale_ptr(const void* hq_scales, int scaling, int64_t r, int64_t d) {
  if (scaling == REF_PER_TENSOR) return hq_scales;
  if (scaling == REF_PER_ROW) return (const float*)hq_scales + r;
  return (const uint8_t*)hq_scales + r * (d / 32);
}

static double ref_lse(const double* z, int64_t V) {
  double m = z[0];
  for (int64_t v = 1; v < V; ++v)
    if (z[v] > m) m = z[v];
  double s = 0.0;
  for (int64_t v = 0; v < V; ++v) s += exp(z[v] - m);
  return m + log(s);
}

void acrl_ref_token_divergence(const double* z_pi, const double* z_mu, int64_t V,
                               double* kl_pi_mu, double* kl_mu_pi, double* l2) {
  const double lp = ref_lse(z_pi, V), lm = ref_lse(z_mu, V);
  double a = 0.0, b = 0.0, c = 0.0;
  for (int64_t v = 0; v < V; ++v) {
    const double log_p = z_pi[v] - lp, log_q = z_mu[v] - lm;
    const double p = exp(log_p), q = exp(log_q);
    a += p * (log_p - log_q);
    b += q * (log_q - log_p);
    c += (p - q) * (p - q);
  }
  if (kl_pi_mu) *kl_pi_mu = a;
  if (kl_mu_pi) *kl_mu_pi = b;
  if (l2) *l2 = sqrt(c);
}

int acrl_ref_score(int64_t n_rows, int64_t d, int64_t V,
                   const uint16_t* h, const uint16_t* w,
                   const uint8_t* hq, const void* hq_scales,
                   const uint8_t* wq, const void* wq_scales, int scaling,
                   const int32_t* ids, const uint8_t* mask, double inv_temperature,
                   double* logp_pi, double* logp_mu, double* ent_pi, double* ent_mu,
                   double* lse_pi, double* lse_mu, double* z_pi, double* z_mu) {
  if (n_rows < 0 || d <= 0 || V <= 0 || !h || !w || !hq || !hq_scales || !wq || !wq_scales ||
      !ids || !logp_pi || !logp_mu)
    return -1;
  if (scaling != REF_PER_TENSOR && scaling != REF_PER_ROW && scaling != REF_MX32) return -1;
  if (scaling == REF_MX32 && d % 32 != 0) return -1;
  int bad = 0;
#pragma omp parallel reduction(| : bad)
  {
    double* zp = (double*)malloc((size_t)V * sizeof(double));
    double* zm = (double*)malloc((size_t)V * sizeof(double));
    if (!zp || !zm) bad = 1;
#pragma omp for schedule(dynamic, 1)
    for (int64_t r = 0; r < n_rows; ++r) {
      if (bad) continue;
      double lp_p = 0, lp_m = 0, hp = 0, hm = 0, lsp = 0, lsm = 0, zap = 0, zam = 0;
      const int valid = mask ? (mask[r] != 0) : 1;
      if (valid) {
        if (acrl_ref_logits_pi(h + r * d, w, d, V, inv_temperature, zp) ||
            acrl_ref_logits_mu(hq + r * d, row_scale_ptr(hq_scales, scaling, r, d), wq, wq_scales,
                               scaling, d, V, inv_temperature, zm)) {
          bad = 1;
          continue;
        }
        acrl_ref_token_stats(zp, V, ids[r], &lsp, &lp_p, &hp);
        acrl_ref_token_stats(zm, V, ids[r], &lsm, &lp_m, &hm);
        zap = (ids[r] >= 0 && ids[r] < V) ? zp[ids[r]] : NAN;
        zam = (ids[r] >= 0 && ids[r] < V) ? zm[ids[r]] : NAN;
      }
      logp_pi[r] = lp_p;
      logp_mu[r] = lp_m;
      if (ent_pi) ent_pi[r] = hp;
      if (ent_mu) ent_mu[r] = hm;
      if (lse_pi) lse_pi[r] = lsp;
      if (lse_mu) lse_mu[r] = lsm;
      if (z_pi) z_pi[r] = zap;
      if (z_mu) z_mu[r] = zam;
    }
    free(zp);
    free(zm);
  }
  return bad ? -1 : 0;
}

/* ------------------------------------------------------------------ */
/* a6 / a7: discrepancy and segmented reductions                        */
/* ------------------------------------------------------------------ */

/*
 * Per token (Eq. distance_metric): d = |pi(a_t) - mu(a_t)| on probabilities,
 * pi(a_t) = exp(logp_pi); the log-ratio log(pi/mu) = logp_pi - logp_mu is the
 * log of the TIS ratio rho (Sec. 2.2); its per-sequence sum is log rho_i of MIS.
 * Per sequence i: n_i = number of valid tokens (|a_i|), sum of d, sum of
 * log-ratios, mean d = (1/|a_i|) sum_t d.
 * Per group g (the G responses of one prompt; the formula for Y and the inner
 * term of X in Sec. 4.1): Y_g = (1/G_g) sum_{i in g} mean_d_i, over the G_g
 * sequences of the group that have at least one valid token.
 * Batch: Y_batch = mean over non-empty groups of Y_g (the outer 1/n sum of X);
 * token-level mean / max / population std of d, mean entropies, mean
 * log-ratio, counts.
 */
int acrl_ref_discrepancy_reduce(int64_t B, int64_t L,
                                const double* logp_pi, const double* logp_mu,
                                const double* ent_pi, const double* ent_mu,
                                const uint8_t* mask, const int32_t* group_of_seq, int64_t n_groups,
                                double* d_tok, int32_t* seq_len, double* seq_sum_d,
                                double* seq_sum_logratio, double* seq_mean_d,
                                double* group_y, int32_t* group_nseq, double* stats) {
  if (B < 0 || L < 0 || n_groups < 0 || !logp_pi || !logp_mu || !mask || !group_of_seq) return -1;
  for (int64_t i = 0; i < B; ++i)
    if (group_of_seq[i] < 0 || group_of_seq[i] >= n_groups) return -1;

  double* sd = (double*)calloc((size_t)(B ? B : 1), sizeof(double));
  double* sl = (double*)calloc((size_t)(B ? B : 1), sizeof(double));
  int64_t* n = (int64_t*)calloc((size_t)(B ? B : 1), sizeof(int64_t));
  double* gsum = (double*)calloc((size_t)(n_groups ? n_groups : 1), sizeof(double));
  int64_t* gcnt = (int64_t*)calloc((size_t)(n_groups ? n_groups : 1), sizeof(int64_t));
  if (!sd || !sl || !n || !gsum || !gcnt) {
    free(sd); free(sl); free(n); free(gsum); free(gcnt);
    return -1;
  }

  double tok_n = 0, tok_sum_d = 0, tok_max_d = 0, tok_sum_hp = 0, tok_sum_hm = 0, tok_sum_lr = 0;
  for (int64_t i = 0; i < B; ++i) {
    for (int64_t j = 0; j < L; ++j) {
      const int64_t t = i * L + j;
      double dv = 0.0;
      if (mask[t]) {
        dv = fabs(exp(logp_pi[t]) - exp(logp_mu[t]));
        const double lr = logp_pi[t] - logp_mu[t];
        n[i] += 1;
        sd[i] += dv;
        sl[i] += lr;
        tok_n += 1;
        tok_sum_d += dv;
        tok_sum_lr += lr;
        if (dv > tok_max_d) tok_max_d = dv;
        if (ent_pi) tok_sum_hp += ent_pi[t];
        if (ent_mu) tok_sum_hm += ent_mu[t];
      }
      if (d_tok) d_tok[t] = dv;
    }
  }
  const double tok_mean_d = tok_n > 0 ? tok_sum_d / tok_n : 0.0;
  double tok_ss = 0.0; /* second pass: sum of squared deviations */
  for (int64_t t = 0; t < B * L; ++t)
    if (mask[t]) {
      const double dv = fabs(exp(logp_pi[t]) - exp(logp_mu[t]));
      tok_ss += (dv - tok_mean_d) * (dv - tok_mean_d);
    }

  int64_t n_seqs = 0;
  for (int64_t i = 0; i < B; ++i) {
    const double mean_d = n[i] > 0 ? sd[i] / (double)n[i] : 0.0;
    if (seq_len) seq_len[i] = (int32_t)n[i];
    if (seq_sum_d) seq_sum_d[i] = sd[i];
    if (seq_sum_logratio) seq_sum_logratio[i] = sl[i];
    if (seq_mean_d) seq_mean_d[i] = mean_d;
    if (n[i] > 0) {
      gsum[group_of_seq[i]] += mean_d;
      gcnt[group_of_seq[i]] += 1;
      n_seqs += 1;
    }
  }
  double ysum = 0.0;
  int64_t ng = 0;
  for (int64_t g = 0; g < n_groups; ++g) {
    const double yg = gcnt[g] > 0 ? gsum[g] / (double)gcnt[g] : 0.0;
    if (group_y) group_y[g] = yg;
    if (group_nseq) group_nseq[g] = (int32_t)gcnt[g];
    if (gcnt[g] > 0) {
      ysum += yg;
      ng += 1;
    }
  }
  if (stats) {
    stats[REF_STAT_Y_BATCH] = ng > 0 ? ysum / (double)ng : 0.0;
    stats[REF_STAT_TOK_MEAN_D] = tok_mean_d;
    stats[REF_STAT_TOK_MAX_D] = tok_max_d;
    stats[REF_STAT_TOK_STD_D] = tok_n > 0 ? sqrt(tok_ss / tok_n) : 0.0;
    stats[REF_STAT_MEAN_H_PI] = tok_n > 0 ? tok_sum_hp / tok_n : 0.0;
    stats[REF_STAT_MEAN_H_MU] = tok_n > 0 ? tok_sum_hm / tok_n : 0.0;
    stats[REF_STAT_N_TOKENS] = tok_n;
    stats[REF_STAT_N_GROUPS] = (double)ng;
    stats[REF_STAT_TOK_MEAN_LOGRATIO] = tok_n > 0 ? tok_sum_lr / tok_n : 0.0;
    stats[REF_STAT_N_SEQS] = (double)n_seqs;
  }
  free(sd); free(sl); free(n); free(gsum); free(gcnt);
  return 0;
}

/* ------------------------------------------------------------------ */
/* a8: controller                                                       */
/* ------------------------------------------------------------------ */

static double sign_of(double a) { return (a > 0) - (a < 0); }

/*
 * Eq. ACRL and the definitions after it (Sec. 4.1):
 *   rho_{i,t} = (pi(a_t) / mu(a_t))^alpha,  alpha = gamma * sign(A_{i,t}) * (1 - Y/X),
 * with gamma > 0, C > 1, and the per-token weight min(rho_{i,t}, C) that
 * multiplies the clipped surrogate's gradient.  pi/mu = exp(logp_pi - logp_mu).
 */
int acrl_ref_controller_step(int64_t B, int64_t L, const uint8_t* mask,
                             const int32_t* group_of_seq, int64_t n_groups,
                             const double* logp_pi, const double* logp_mu,
                             const double* adv, int adv_per_token, int y_level,
                             const double* seq_mean_d, const double* group_y,
                             const double* stats, double X, double gamma, double C,
                             int mode, double k, double* alpha, double* weight) {
  if (B < 0 || L < 0 || !mask || !logp_pi || !logp_mu || !adv || !weight) return -1;
  if (!(X > 0.0) || !(gamma > 0.0) || !(C > 1.0)) return -1;
  if (mode < REF_CTRL_ACRL || mode > REF_CTRL_FALLBACK) return -1;
  if (mode == REF_CTRL_CONTINUOUS && !(k > 0.0)) return -1;
  for (int64_t i = 0; i < B; ++i) {
    double Y;
    if (y_level == REF_Y_SEQUENCE) {
      if (!seq_mean_d) return -1;
      Y = seq_mean_d[i];
    } else if (y_level == REF_Y_GROUP) {
      if (!group_y || !group_of_seq) return -1;
      /* a response outside every group has no Y */
      Y = (group_of_seq[i] >= 0 && group_of_seq[i] < n_groups) ? group_y[group_of_seq[i]] : NAN;
    } else if (y_level == REF_Y_BATCH) {
      if (!stats) return -1;
      Y = stats[REF_STAT_Y_BATCH];
    } else {
      return -1;
    }
    /* Eq. mis_objective: the sequence's probability ratio pi(a_i)/mu(a_i),
     * the product of its token ratios */
    double rho_seq = 1.0;
    if (mode == REF_CTRL_MIS)
      for (int64_t j = 0; j < L; ++j)
        if (mask[i * L + j]) rho_seq *= exp(logp_pi[i * L + j] - logp_mu[i * L + j]);
    for (int64_t j = 0; j < L; ++j) {
      const int64_t t = i * L + j;
      double a = 0.0, wt = 0.0;
      if (mask[t]) {
        const double A = adv_per_token ? adv[t] : adv[i];
        const double ratio = exp(logp_pi[t] - logp_mu[t]); /* pi / mu */
        /* min(x, C) of an undefined x is undefined: NaN stays NaN */
        if (mode == REF_CTRL_TIS) {
          a = 1.0;
          wt = isnan(ratio) ? NAN : (ratio < C ? ratio : C);
        } else if (mode == REF_CTRL_MIS) {
          a = 1.0;
          wt = isnan(rho_seq) ? NAN : (rho_seq <= C ? rho_seq : 0.0);
        } else if (mode == REF_CTRL_FALLBACK && Y < X) {
          a = 0.0;
          wt = 1.0;
        } else {
          if (mode == REF_CTRL_CONTINUOUS) a = -k * sign_of(A);
          else a = gamma * sign_of(A) * (1.0 - Y / X);
          /* (pi/mu)^alpha; pow() would give 1 for a NaN ratio at alpha = 0 */
          const double rho = (isnan(ratio) || isnan(a)) ? NAN : pow(ratio, a);
          wt = isnan(rho) ? NAN : (rho < C ? rho : C);
        }
      }
      if (alpha) alpha[t] = a;
      weight[t] = wt;
    }
  }
  return 0;
}

/* Reference X (Sec. 4.1): X = (1/n) sum_j (1/G) sum_i (1/|a_i|) sum_t d, i.e.
 * the mean of the per-group discrepancy over the n prompts of step 0. */
int acrl_ref_reference_x(const double* group_y, const int32_t* group_nseq, int64_t n_groups,
                         double* X) {
  if (!group_y || !group_nseq || !X || n_groups < 0) return -1;
  double s = 0.0;
  int64_t n = 0;
  for (int64_t g = 0; g < n_groups; ++g)
    if (group_nseq[g] > 0) {
      s += group_y[g];
      n += 1;
    }
  if (n == 0) return -1;
  *X = s / (double)n;
  return 0;
}

/* ------------------------------------------------------------------ */
/* Fixture helper: sampling ids from a softmax                          */
/* ------------------------------------------------------------------ */

int acrl_ref_sample_inverse_cdf(const double* z, int64_t n_rows, int64_t V,
                                const double* u, int32_t* ids) {
  if (!z || !u || !ids || V <= 0 || n_rows < 0) return -1;
  for (int64_t r = 0; r < n_rows; ++r) {
    const double* zr = z + r * V;
    double lse;
    acrl_ref_token_stats(zr, V, 0, &lse, NULL, NULL);
    double c = 0.0;
    int32_t pick = (int32_t)(V - 1);
    for (int64_t v = 0; v < V; ++v) {
      c += exp(zr[v] - lse);
      if (c > u[r]) {
        pick = (int32_t)v;
        break;
      }
    }
    ids[r] = pick;
  }
  return 0;
}

/* ------------------------------------------------------------------ */
/* Gumbel-max sampling from mu                                          */
/* ------------------------------------------------------------------ */

/* Philox4x32-10: each round multiplies words 0 and 2 by the two round
 * constants, mixes the high halves with the other words and the key, and
 * the key advances by the two Weyl constants between rounds. */
void acrl_ref_philox4x32_10(const uint32_t ctr[4], const uint32_t key[2], uint32_t out[4]) {
  const uint32_t M0 = 0xD2511F53u, M1 = 0xCD9E8D57u, W0 = 0x9E3779B9u, W1 = 0xBB67AE85u;
  uint32_t c0 = ctr[0], c1 = ctr[1], c2 = ctr[2], c3 = ctr[3];
  uint32_t k0 = key[0], k1 = key[1];
  for (int round = 0; round < 10; ++round) {
    const uint64_t p0 = (uint64_t)M0 * c0, p1 = (uint64_t)M1 * c2;
    const uint32_t hi0 = (uint32_t)(p0 >> 32), lo0 = (uint32_t)p0;
    const uint32_t hi1 = (uint32_t)(p1 >> 32), lo1 = (uint32_t)p1;
    const uint32_t n0 = hi1 ^ c1 ^ k0, n1 = lo1, n2 = hi0 ^ c3 ^ k1, n3 = lo0;
    c0 = n0; c1 = n1; c2 = n2; c3 = n3;
    k0 += W0;
    k1 += W1;
  }
  out[0] = c0; out[1] = c1; out[2] = c2; out[3] = c3;
}

double acrl_ref_sample_uniform(uint64_t seed, int64_t t, int64_t v) {
  const uint32_t ctr[4] = {(uint32_t)(v / 4), (uint32_t)t, 0u, 0u};
  const uint32_t key[2] = {(uint32_t)seed, (uint32_t)(seed >> 32)};
  uint32_t w[4];
  acrl_ref_philox4x32_10(ctr, key, w);
  return ((double)(w[v % 4] >> 9) + 0.5) / 8388608.0;
}

int acrl_ref_gumbel_sample(const double* z, int64_t n_rows, int64_t V, uint64_t seed,
                           int64_t row_offset, int32_t* ids, double* key_out) {
  if (!z || !ids || V <= 0 || n_rows < 0) return -1;
  for (int64_t r = 0; r < n_rows; ++r) {
    double best = -INFINITY;
    int32_t pick = 0;
    for (int64_t v = 0; v < V; ++v) {
      const double u = acrl_ref_sample_uniform(seed, row_offset + r, v);
      const double key = z[r * V + v] - log(-log(u));
      if (key > best) {
        best = key;
        pick = (int32_t)v;
      }
    }
    ids[r] = pick;
    if (key_out) key_out[r] = best;
  }
  return 0;
}

/* Blockwise Gumbel-max: the same draw from softmax(z) with two uniforms per
 * block of vocabulary rows instead of one per row.  The vocabulary is cut
 * into blocks of 16 rows: row v lies in block k(v) = 2 floor(v/32) +
 * (floor(v/4) mod 2), i.e. block k holds rows 32 floor(k/2) + 8q + 4 (k mod 2)
 * + j, q, j in 0..3 (fewer at the end of the vocabulary).  Two facts make it
 * exact.  First, the largest of z_v + G_v over a block is distributed as
 * lse_k + G with one Gumbel G (the Gumbel family is max-stable).  Second,
 * which row attains it is independent of that value and has probability
 * exp(z_v - lse_k).  So the block is drawn by Gumbel-max over the keys
 * lse_k - ln(-ln u_k), and the row inside it by inverse CDF with a second
 * uniform u'_k.
 * Uniforms: Philox4x32-10 on counter (floor(v/64), row_offset + r,
 * k mod 2, 0) under key (seed low, seed high); e = floor(k/2) mod 2 picks
 * words 2e (u_k) and 2e+1 (u'_k); u = (w >> 9 + 1/2) 2^-23.  Ties between
 * block keys go to the smaller block; inside the block the first row (in
 * increasing v) whose cumulative probability exceeds u'_k, else the block's
 * last row of nonzero probability. */
static void block_uniforms(uint64_t seed, int64_t t, int64_t k, double* u_key, double* u_pick) {
  const int64_t v0 = 32 * (k / 2) + 4 * (k % 2); /* first row of block k */
  const uint32_t ctr[4] = {(uint32_t)(v0 / 64), (uint32_t)t, (uint32_t)(k % 2), 0u};
  const uint32_t key[2] = {(uint32_t)seed, (uint32_t)(seed >> 32)};
  uint32_t w[4];
  acrl_ref_philox4x32_10(ctr, key, w);
  const int e = (int)((k / 2) % 2);
  *u_key = ((double)(w[2 * e] >> 9) + 0.5) / 8388608.0;
  *u_pick = ((double)(w[2 * e + 1] >> 9) + 0.5) / 8388608.0;
}

/* Row of slot q (0..15) of block k, or -1 past the vocabulary. */
static int64_t block_row(int64_t k, int q, int64_t V) {
  const int64_t v = 32 * (k / 2) + 8 * (q / 4) + 4 * (k % 2) + (q % 4);
  return v < V ? v : -1;
}

/* Key of every block of one token's logits zr (n_blocks = 2 ceil(V/32)):
 * lse of the block's rows - ln(-ln u_k); -inf for a block past V. */
int acrl_ref_block_gumbel_keys(const double* zr, int64_t V, uint64_t seed, int64_t t, double* keys) {
  if (!zr || !keys || V <= 0) return -1;
  const int64_t n_blocks = 2 * ((V + 31) / 32);
  for (int64_t k = 0; k < n_blocks; ++k) {
    double m = -INFINITY;
    for (int q = 0; q < 16; ++q) {
      const int64_t v = block_row(k, q, V);
      if (v >= 0 && zr[v] > m) m = zr[v];
    }
    if (m == -INFINITY) {
      keys[k] = -INFINITY;
      continue;
    }
    double sum = 0.0;
    for (int q = 0; q < 16; ++q) {
      const int64_t v = block_row(k, q, V);
      if (v >= 0) sum += exp(zr[v] - m);
    }
    double u_key, u_pick;
    block_uniforms(seed, t, k, &u_key, &u_pick);
    keys[k] = m + log(sum) - log(-log(u_key));
  }
  return 0;
}

/* The row block k gives token t: the first row (in increasing v) whose
 * cumulative softmax probability within the block exceeds u'_k, else the
 * block's last row of nonzero probability.  cum (nullable, 16 entries): the
 * cumulative probabilities after each slot (NaN past V); u_pick (nullable):
 * u'_k. */
int64_t acrl_ref_block_pick(const double* zr, int64_t V, uint64_t seed, int64_t t, int64_t k, double* cum,
                            double* u_pick_out) {
  double u_key, u_pick;
  block_uniforms(seed, t, k, &u_key, &u_pick);
  double m = -INFINITY;
  for (int q = 0; q < 16; ++q) {
    const int64_t v = block_row(k, q, V);
    if (v >= 0 && zr[v] > m) m = zr[v];
  }
  double total = 0.0;
  int64_t last = -1;
  for (int q = 0; q < 16; ++q) {
    const int64_t v = block_row(k, q, V);
    if (v < 0) continue;
    const double e = exp(zr[v] - m);
    total += e;
    if (e > 0.0) last = v;
  }
  int64_t pick = last;
  int found = 0;
  double c = 0.0;
  for (int q = 0; q < 16; ++q) {
    const int64_t v = block_row(k, q, V);
    if (v < 0) {
      if (cum) cum[q] = NAN;
      continue;
    }
    c += exp(zr[v] - m);
    if (cum) cum[q] = c / total;
    if (!found && c > u_pick * total) {
      pick = v;
      found = 1;
    }
  }
  if (u_pick_out) *u_pick_out = u_pick;
  return pick;
}

int acrl_ref_block_gumbel_sample(const double* z, int64_t n_rows, int64_t V, uint64_t seed,
                                 int64_t row_offset, int32_t* ids, double* key_out,
                                 int64_t* block_out) {
  if (!z || !ids || V <= 0 || n_rows < 0) return -1;
  const int64_t n_blocks = 2 * ((V + 31) / 32);
  double* keys = (double*)malloc((size_t)n_blocks * sizeof(double));
  if (!keys) return -1;
  for (int64_t r = 0; r < n_rows; ++r) {
    const double* zr = z + r * V;
    acrl_ref_block_gumbel_keys(zr, V, seed, row_offset + r, keys);
    /* the block of the largest key (the smaller block on a tie) */
    double best = -INFINITY;
    int64_t best_k = -1;
    for (int64_t k = 0; k < n_blocks; ++k)
      if (keys[k] > best) {
        best = keys[k];
        best_k = k;
      }
    ids[r] = (int32_t)acrl_ref_block_pick(zr, V, seed, row_offset + r, best_k, NULL, NULL);
    if (key_out) key_out[r] = best;
    if (block_out) block_out[r] = best_k;
  }
  free(keys);
  return 0;
}

/* ------------------------------------------------------------------ */
/* The ACRL-weighted surrogate (Eq. ACRL) and its LM-head backward      */
/* ------------------------------------------------------------------ */

int acrl_ref_surrogate(int64_t B, int64_t L, const uint8_t* mask, const int32_t* group_of_seq,
                       int64_t n_groups, const double* logp_new, const double* logp_old,
                       const double* adv, int adv_per_token, const double* weight,
                       double eps_low, double eps_high, double* coef, double* loss) {
  if (B < 0 || L < 0 || n_groups < 0 || !mask || !group_of_seq || !logp_new || !logp_old ||
      !adv || !coef || !loss)
    return -1;
  if (!(eps_low >= 0.0) || !(eps_high >= 0.0)) return -1;
  for (int64_t i = 0; i < B; ++i)
    if (group_of_seq[i] < 0 || group_of_seq[i] >= n_groups) return -1;
  /* |a_i|, then the non-empty responses of each prompt, then the prompts */
  int64_t* n = (int64_t*)calloc((size_t)(B > 0 ? B : 1), sizeof(int64_t));
  int64_t* G = (int64_t*)calloc((size_t)(n_groups > 0 ? n_groups : 1), sizeof(int64_t));
  if (!n || !G) {
    free(n);
    free(G);
    return -1;
  }
  for (int64_t i = 0; i < B; ++i)
    for (int64_t j = 0; j < L; ++j) n[i] += mask[i * L + j] != 0;
  for (int64_t i = 0; i < B; ++i)
    if (n[i] > 0) G[group_of_seq[i]] += 1;
  int64_t prompts = 0;
  for (int64_t g = 0; g < n_groups; ++g) prompts += G[g] > 0;
  double J = 0.0;
  for (int64_t i = 0; i < B; ++i) {
    for (int64_t j = 0; j < L; ++j) {
      const int64_t t = i * L + j;
      coef[t] = 0.0;
      if (!mask[t]) continue;
      const double c = 1.0 / ((double)prompts * (double)G[group_of_seq[i]] * (double)n[i]);
      const double A = adv_per_token ? adv[t] : adv[i];
      const double wt = weight ? weight[t] : 1.0;
      const double r = exp(logp_new[t] - logp_old[t]);
      double rc = r;
      if (rc < 1.0 - eps_low) rc = 1.0 - eps_low;
      if (rc > 1.0 + eps_high) rc = 1.0 + eps_high;
      const double unclipped = r * A, clipped = rc * A;
      const double m = unclipped <= clipped ? unclipped : clipped;
      J += c * wt * m;
      /* d(r A)/d logp_new = r A; the clipped term is constant in logp_new */
      if (unclipped <= clipped) coef[t] = -c * wt * r * A;
    }
  }
  *loss = -J;
  free(n);
  free(G);
  return 0;
}

int acrl_ref_lm_head_backward(int64_t n_rows, int64_t d, int64_t V, const uint16_t* h,
                              const uint16_t* w, const int32_t* ids, const double* coef,
                              double inv_temperature, int64_t n_hrows, const int64_t* hrows,
                              double* dh, double* dh_abs, int64_t n_wrows, const int64_t* wrows,
                              double* dw, double* dw_abs) {
  if (n_rows < 0 || d <= 0 || V <= 0 || !h || !w || !ids || !coef) return -1;
  if ((n_hrows > 0 && (!hrows || !dh)) || (n_wrows > 0 && (!wrows || !dw))) return -1;
  for (int64_t t = 0; t < n_rows; ++t)
    if (ids[t] < 0 || ids[t] >= V) return -1;
  for (int64_t i = 0; i < n_hrows; ++i)
    if (hrows[i] < 0 || hrows[i] >= n_rows) return -1;
  for (int64_t j = 0; j < n_wrows; ++j)
    if (wrows[j] < 0 || wrows[j] >= V) return -1;
  /* dZ of every token, one row at a time: the logits, their log-sum-exp,
   * then coef (delta - p) / tau */
  double* dz = (double*)malloc((size_t)(n_rows > 0 ? n_rows : 1) * (size_t)V * sizeof(double));
  if (!dz) return -1;
  int bad = 0;
#pragma omp parallel for schedule(dynamic, 1) reduction(| : bad)
  for (int64_t t = 0; t < n_rows; ++t) {
    double* z = dz + t * V;
    if (acrl_ref_logits_pi(h + t * d, w, d, V, inv_temperature, z)) {
      bad = 1;
      continue;
    }
    double lse;
    acrl_ref_token_stats(z, V, ids[t], &lse, NULL, NULL);
    for (int64_t v = 0; v < V; ++v) {
      const double p = exp(z[v] - lse);
      z[v] = coef[t] * ((v == ids[t] ? 1.0 : 0.0) - p) * inv_temperature;
    }
  }
  if (bad) {
    free(dz);
    return -1;
  }
  /* dH[t, k] = sum_v dZ[t, v] W[v, k]  (v ascending; the row of W is the
   * inner loop only so that memory is walked in order) */
#pragma omp parallel for schedule(dynamic, 1)
  for (int64_t i = 0; i < n_hrows; ++i) {
    const double* zr = dz + hrows[i] * V;
    double* s = dh + i * d;
    for (int64_t k = 0; k < d; ++k) {
      s[k] = 0.0;
      if (dh_abs) dh_abs[i * d + k] = 0.0;
    }
    for (int64_t v = 0; v < V; ++v)
      for (int64_t k = 0; k < d; ++k) {
        const double wv = acrl_ref_bf16_to_float(w[v * d + k]);
        s[k] += zr[v] * wv;
        if (dh_abs) dh_abs[i * d + k] += fabs(zr[v]) * fabs(wv);
      }
  }
  /* dW[v, k] = sum_t dZ[t, v] H[t, k]  (t ascending) */
#pragma omp parallel for schedule(dynamic, 1)
  for (int64_t j = 0; j < n_wrows; ++j) {
    const int64_t v = wrows[j];
    double* s = dw + j * d;
    for (int64_t k = 0; k < d; ++k) {
      s[k] = 0.0;
      if (dw_abs) dw_abs[j * d + k] = 0.0;
    }
    for (int64_t t = 0; t < n_rows; ++t)
      for (int64_t k = 0; k < d; ++k) {
        const double hv = acrl_ref_bf16_to_float(h[t * d + k]);
        s[k] += dz[t * V + v] * hv;
        if (dw_abs) dw_abs[j * d + k] += fabs(dz[t * V + v]) * fabs(hv);
      }
  }
  free(dz);
  return 0;
}

int acrl_ref_divergence(int64_t n_rows, int64_t d, int64_t V, const uint16_t* h, const uint16_t* w,
                        const uint8_t* hq, const void* hq_scales, const uint8_t* wq,
                        const void* wq_scales, int scaling, const uint8_t* mask,
                        double inv_temperature, double* kl_pi_mu, double* kl_mu_pi, double* l2) {
  if (n_rows < 0 || d <= 0 || V <= 0 || !h || !w || !hq || !hq_scales || !wq || !wq_scales)
    return -1;
  if (scaling != REF_PER_TENSOR && scaling != REF_PER_ROW && scaling != REF_MX32) return -1;
  if (scaling == REF_MX32 && d % 32 != 0) return -1;
  int bad = 0;
#pragma omp parallel reduction(| : bad)
  {
    double* zp = (double*)malloc((size_t)V * sizeof(double));
    double* zm = (double*)malloc((size_t)V * sizeof(double));
    if (!zp || !zm) bad = 1;
#pragma omp for schedule(dynamic, 1)
    for (int64_t r = 0; r < n_rows; ++r) {
      if (bad) continue;
      double a = 0.0, b = 0.0, c = 0.0;
      if (!mask || mask[r]) {
        if (acrl_ref_logits_pi(h + r * d, w, d, V, inv_temperature, zp) ||
            acrl_ref_logits_mu(hq + r * d, row_scale_ptr(hq_scales, scaling, r, d), wq, wq_scales,
                               scaling, d, V, inv_temperature, zm)) {
          bad = 1;
          continue;
        }
        acrl_ref_token_divergence(zp, zm, V, &a, &b, &c);
      }
      if (kl_pi_mu) kl_pi_mu[r] = a;
      if (kl_mu_pi) kl_mu_pi[r] = b;
      if (l2) l2[r] = c;
    }
    free(zp);
    free(zm);
  }
  return bad ? -1 : 0;
}
