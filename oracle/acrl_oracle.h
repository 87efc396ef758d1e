/*
 * acrl_oracle.h -- CPU oracle for the ACRL scoring / discrepancy path.
 *
 * TEST INFRASTRUCTURE ONLY.  This library is the slow, plain, fp64 statement
 * of what the GPU path must compute.  Only the test suite, the smoke check and
 * the benchmark's CPU-baseline leg may load it.  It shares no code, header,
 * table or helper with the HIP library; the two are independent on purpose.
 *
 * Every array argument is a HOST pointer.  Floating point is double unless
 * the definition being followed fixes fp32 (the quantizer's scale and divide).
 * Return value of the int functions: 0 on success, -1 on a bad argument.
 *
 * Citations name the section / equation of the ACRL paper
 * ("Adaptive Control of Training-Inference Discrepancy for Stable RL").
 */
#ifndef ACRL_ORACLE_H
#define ACRL_ORACLE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Scaling granularity of the FP8 inference policy mu (Sec. 5.1 setup: per-token
 * activations, per-channel weights; Sec. 5.2 / 5.4: MXFP8).                  */
enum { REF_PER_TENSOR = 0, REF_PER_ROW = 1, REF_MX32 = 2 };
/* Rounding of the FP8 encoder: nearest (Sec. 5.1 "nearest-around") or the
 * truncation used in the stress test, Q(x) = trunc(x/S) (Sec. 5.3).          */
enum { REF_ROUND_NEAREST_EVEN = 0, REF_ROUND_TOWARD_ZERO = 1 };
/* Granularity of Y in alpha = gamma*sign(A)*(1 - Y/X) (Sec. 4.1).            */
enum { REF_Y_GROUP = 0, REF_Y_SEQUENCE = 1, REF_Y_BATCH = 2 };
/* Weighting rule of the controller step: the paper's ACRL (Eq. ACRL), the
 * token-level TIS it builds on (Eq. tis_objective), sequence-level MIS
 * (Eq. mis_objective), and the two one-sided ablations of Sec. 5
 * ("continuous reduction", "fallback to GRPO"). */
enum { REF_CTRL_ACRL = 0, REF_CTRL_TIS = 1, REF_CTRL_MIS = 2, REF_CTRL_CONTINUOUS = 3, REF_CTRL_FALLBACK = 4 };

/* Indices into the batch statistics vector written by the reduce. */
enum {
  REF_STAT_Y_BATCH = 0,        /* mean over non-empty groups of Y_g            */
  REF_STAT_TOK_MEAN_D = 1,     /* token-level mean of d over valid tokens      */
  REF_STAT_TOK_MAX_D = 2,      /* token-level max of d                         */
  REF_STAT_TOK_STD_D = 3,      /* token-level population std of d              */
  REF_STAT_MEAN_H_PI = 4,      /* mean entropy of pi over valid tokens         */
  REF_STAT_MEAN_H_MU = 5,      /* mean entropy of mu over valid tokens         */
  REF_STAT_N_TOKENS = 6,       /* number of valid tokens                       */
  REF_STAT_N_GROUPS = 7,       /* number of non-empty groups                   */
  REF_STAT_TOK_MEAN_LOGRATIO = 8, /* token-level mean of log(pi/mu)            */
  REF_STAT_N_SEQS = 9,         /* number of non-empty sequences                */
  REF_N_STATS = 10
};

/* ---- number formats -------------------------------------------------- */
float   acrl_ref_bf16_to_float(uint16_t bits);
/* OCP FP8 E4M3 ("fn": bias 7, max 448, S.1111.111 = NaN, no infinities).
 * Nearest-even or toward-zero; magnitudes >= 448 (and infinities) saturate
 * to +-448; NaN -> 0x7F with the input's sign.                              */
uint8_t acrl_ref_e4m3_encode(float x, int rounding);
double  acrl_ref_e4m3_decode(uint8_t code);
/* OCP E8M0 shared scale: 2^(code-127); code 255 is NaN.                     */
double  acrl_ref_e8m0_decode(uint8_t code);
void    acrl_ref_e4m3_encode_array(const float* x, int64_t n, int rounding, uint8_t* out);

/* ---- a1/a2: FP8 quantization of a bf16 matrix ------------------------- *
 * x: bf16 bits [rows, ld] (cols used).  q: [rows, cols] codes.
 * scales: float[1] (PER_TENSOR), float[rows] (PER_ROW),
 *         uint8 e8m0 [rows, cols/32] (MX32, cols % 32 == 0).               */
int acrl_ref_quantize_fp8(const uint16_t* x, int64_t rows, int64_t cols, int64_t ld,
                          int scaling, int rounding, uint8_t* q, void* scales);

/* ---- a3/a4: logits of one token over the whole vocabulary -------------- */
int acrl_ref_logits_pi(const uint16_t* h_row, const uint16_t* w, int64_t d, int64_t V,
                       double inv_temperature, double* z);
/* hq_row: codes of the token; row_scale: pointer to this token's scale
 * (float for PER_TENSOR/PER_ROW, d/32 e8m0 bytes for MX32).  wq_scales is the
 * weight scale array as produced by acrl_ref_quantize_fp8 for W.            */
int acrl_ref_logits_mu(const uint8_t* hq_row, const void* row_scale, const uint8_t* wq,
                       const void* wq_scales, int scaling, int64_t d, int64_t V,
                       double inv_temperature, double* z);

/* ---- a3..a5: log-softmax statistics of one token ---------------------- */
void acrl_ref_token_stats(const double* z, int64_t V, int32_t id,
                          double* lse, double* logp, double* entropy);

/* ---- a3..a5 for many rows: both policies ----------------------------- *
 * Row r of h / hq is scored with sampled id ids[r].  Rows with mask[r]==0
 * (mask may be NULL = all valid) get all outputs 0.  Outputs are [n_rows]
 * doubles; every output pointer except logp_pi/logp_mu may be NULL.
 * hq_scales: float[1] / float[n_rows] / uint8 [n_rows, d/32].              */
int acrl_ref_score(int64_t n_rows, int64_t d, int64_t V,
                   const uint16_t* h, const uint16_t* w,
                   const uint8_t* hq, const void* hq_scales,
                   const uint8_t* wq, const void* wq_scales, int scaling,
                   const int32_t* ids, const uint8_t* mask, double inv_temperature,
                   double* logp_pi, double* logp_mu, double* ent_pi, double* ent_mu,
                   double* lse_pi, double* lse_mu, double* z_pi, double* z_mu);

/* ---- Full-vocabulary discrepancy between the two policies --------------- *
 * The paper measures the discrepancy on the sampled token's probabilities
 * (Eq. distance_metric) and names the KL divergence and the Euclidean
 * distance as other measures (remark after Eq. distance_metric; Sec. 7).
 * Over the whole vocabulary, with p = softmax(z_pi), q = softmax(z_mu):
 *   kl_pi_mu = sum_v p_v (log p_v - log q_v)    (KL(pi || mu))
 *   kl_mu_pi = sum_v q_v (log q_v - log p_v)    (KL(mu || pi))
 *   l2       = sqrt(sum_v (p_v - q_v)^2)         (Euclidean distance)
 * in double: the two log-sum-exps first, then the sums over v.  Any output
 * may be NULL.                                                              */
void acrl_ref_token_divergence(const double* z_pi, const double* z_mu, int64_t V,
                               double* kl_pi_mu, double* kl_mu_pi, double* l2);
/* The same for every row, from the logits of acrl_ref_score (same operands
 * and arguments); rows with mask[r] == 0 get 0.                            */
int acrl_ref_divergence(int64_t n_rows, int64_t d, int64_t V, const uint16_t* h, const uint16_t* w,
                        const uint8_t* hq, const void* hq_scales, const uint8_t* wq,
                        const void* wq_scales, int scaling, const uint8_t* mask,
                        double inv_temperature, double* kl_pi_mu, double* kl_mu_pi, double* l2);

/* ---- a6/a7: per-token discrepancy and the segmented masked reduce ------ *
 * Slot (i, j) = i*L + j.  ent_pi/ent_mu may be NULL (means reported as 0).
 * Outputs: d_tok[B*L] (0 where masked), seq_len[B], seq_sum_d[B],
 * seq_sum_logratio[B], seq_mean_d[B] (0 for empty sequences),
 * group_y[n_groups] (0 for empty groups), group_nseq[n_groups] (non-empty
 * sequences per group), stats[REF_N_STATS].  Any output may be NULL.       */
int acrl_ref_discrepancy_reduce(int64_t B, int64_t L,
                                const double* logp_pi, const double* logp_mu,
                                const double* ent_pi, const double* ent_mu,
                                const uint8_t* mask, const int32_t* group_of_seq, int64_t n_groups,
                                double* d_tok, int32_t* seq_len, double* seq_sum_d,
                                double* seq_sum_logratio, double* seq_mean_d,
                                double* group_y, int32_t* group_nseq, double* stats);

/* ---- a8: the ACRL controller step ------------------------------------ *
 * adv: [B] (one advantage per response, GRPO) or [B*L] (adv_per_token=1).
 * Y is read from seq_mean_d[i], group_y[group_of_seq[i]] or stats[0]
 * according to y_level.  Outputs alpha, weight [B*L]; masked slots -> 0.
 * mode (REF_CTRL_*), per valid token t of sequence i, rho_t = pi/mu:
 *   ACRL:       alpha = gamma sign(A) (1 - Y/X), weight = min(rho_t^alpha, C)
 *   TIS:        alpha = 1,                       weight = min(rho_t, C)
 *   MIS:        alpha = 1, weight = rho_i if rho_i <= C else 0, with
 *               rho_i = product of rho_t over the valid tokens of i
 *   CONTINUOUS: alpha = -k sign(A),              weight = min(rho_t^alpha, C)
 *   FALLBACK:   Y < X: alpha = 0, weight = 1 (plain GRPO); else as ACRL
 * Requires X > 0, gamma > 0, C > 1, k > 0 (k is read in CONTINUOUS only).
 * An undefined input gives an undefined weight (NaN), never the clip C: a
 * NaN log-prob (the scorer's mark of an invalid token id), a NaN ratio, or
 * a response whose group id lies outside [0, n_groups) (its Y is undefined;
 * its alpha is NaN as well).                                               */
int acrl_ref_controller_step(int64_t B, int64_t L, const uint8_t* mask,
                             const int32_t* group_of_seq, int64_t n_groups,
                             const double* logp_pi, const double* logp_mu,
                             const double* adv, int adv_per_token, int y_level,
                             const double* seq_mean_d, const double* group_y,
                             const double* stats, double X, double gamma, double C,
                             int mode, double k, double* alpha, double* weight);

/* Reference X (Sec. 4.1): mean of the per-group discrepancy over the
 * non-empty groups (group_nseq > 0) of the step-0 batches.                 */
int acrl_ref_reference_x(const double* group_y, const int32_t* group_nseq, int64_t n_groups,
                         double* X);

/* ---- Sampling from mu by the Gumbel-max trick ------------------------ *
 * Counter-based random numbers: Philox4x32-10 (Salmon, Moraes, Dror, Shaw,
 * "Parallel random numbers: as easy as 1, 2, 3", SC 2011): 10 rounds on a
 * 128-bit counter under a 64-bit key.                                       */
void acrl_ref_philox4x32_10(const uint32_t ctr[4], const uint32_t key[2], uint32_t out[4]);

/* The uniform of vocabulary entry v of token t (global token index) under
 * seed: word (v mod 4) of Philox4x32-10 on counter (v / 4, t, 0, 0) and key
 * (seed low 32 bits, seed high 32 bits); u = (word >> 9 + 1/2) 2^-23, in
 * (0, 1) and exact in fp32.                                                  */
double acrl_ref_sample_uniform(uint64_t seed, int64_t t, int64_t v);

/* Gumbel-max sampling: ids[r] = argmax_v z[r, v] - ln(-ln u(seed, row_offset
 * + r, v)) over the logits z (natural units, temperature applied); a draw
 * from softmax(z).  key_out[r] (nullable) = the winning key.  Ties go to the
 * smaller v.                                                                */
int acrl_ref_gumbel_sample(const double* z, int64_t n_rows, int64_t V, uint64_t seed,
                           int64_t row_offset, int32_t* ids, double* key_out);

/* ---- fixture helper (not part of the method): inverse-CDF sampling ----- *
 * Samples one id per row from softmax(z_row) using the supplied uniform
 * u[r] in [0,1): the smallest v whose cumulative probability exceeds u.     */
/* Blockwise Gumbel-max: blocks of 16 vocabulary rows (row v in block
 * 2 floor(v/32) + (floor(v/4) mod 2)); one Gumbel key lse_k - ln(-ln u_k)
 * per block, then the row inside the winning block by inverse CDF with
 * u'_k; u_k, u'_k from Philox4x32-10 on (floor(v/64), row_offset + r,
 * k mod 2, 0), words 2e and 2e+1 with e = floor(k/2) mod 2.  A draw from
 * softmax(z).  key_out / block_out (nullable): the winning key and block. */
int acrl_ref_block_gumbel_sample(const double* z, int64_t n_rows, int64_t V, uint64_t seed,
                                 int64_t row_offset, int32_t* ids, double* key_out,
                                 int64_t* block_out);
/* The pieces of it: every block's key for token t, and the row block k
 * gives (cum: its 16 cumulative probabilities, u_pick: u'_k; nullable). */
int acrl_ref_block_gumbel_keys(const double* zr, int64_t V, uint64_t seed, int64_t t, double* keys);
int64_t acrl_ref_block_pick(const double* zr, int64_t V, uint64_t seed, int64_t t, int64_t k, double* cum,
                            double* u_pick_out);
int acrl_ref_sample_inverse_cdf(const double* z, int64_t n_rows, int64_t V,
                                const double* u, int32_t* ids);

/* ---- The ACRL-weighted surrogate and its LM-head backward ------------- *
 * Eq. ACRL (Sec. 4.1), which extends Eq. grpo_objective (Sec. 2): the
 * objective of a batch is
 *   J = mean over prompts of (1/G) sum_i (1/|a_i|) sum_t w_t min(r_t A_t, clip(r_t) A_t),
 * r_t = pi_theta(a_t) / pi_theta_old(a_t) = exp(logp_new - logp_old),
 * clip(r) = min(max(r, 1 - eps_low), 1 + eps_high) (eps_low = eps_high = eps
 * in the paper), w_t = min(rho_t, C) the controller weight (held constant).
 * Readings: the prompts averaged are the groups with a non-empty response,
 * G is the count of the group's non-empty responses (as for Y), an empty
 * response contributes nothing; loss = -J.
 * coef[t] = d loss / d logp_new[t] = -c_t w_t r_t A_t when the unclipped term
 * is the minimum (r A <= clip(r) A; a tie counts as unclipped), else 0;
 * c_t = 1 / (n_prompts * G_g * |a_i|).  Masked slots: coef 0.
 * weight NULL means w = 1 (plain GRPO).                                    */
int acrl_ref_surrogate(int64_t B, int64_t L, const uint8_t* mask, const int32_t* group_of_seq,
                       int64_t n_groups, const double* logp_new, const double* logp_old,
                       const double* adv, int adv_per_token, const double* weight,
                       double eps_low, double eps_high, double* coef, double* loss);

/* Gradient of Phi(H, W) = sum_t coef_t log softmax(W h_t / tau)[a_t] with
 * respect to H [n_rows, d] and W [V, d] (bf16 bit patterns), by the chain
 * rule through the surrogate: dZ[t, v] = coef_t (delta(v, a_t) - p_tv) / tau,
 * p_t = softmax(W h_t / tau); dH = dZ W, dW = dZ^T H, all in double.
 * Only the requested rows are formed: dh[i, :] = dH[hrows[i], :],
 * dw[j, :] = dW[wrows[j], :].  dh_abs / dw_abs (nullable) receive
 * sum_v |dZ[t, v]| |W[v, k]| and sum_t |dZ[t, v]| |H[t, k]|, the magnitude a
 * rounding error of each product is relative to.  ids must lie in [0, V).   */
int acrl_ref_lm_head_backward(int64_t n_rows, int64_t d, int64_t V, const uint16_t* h,
                              const uint16_t* w, const int32_t* ids, const double* coef,
                              double inv_temperature, int64_t n_hrows, const int64_t* hrows,
                              double* dh, double* dh_abs, int64_t n_wrows, const int64_t* wrows,
                              double* dw, double* dw_abs);

#ifdef __cplusplus
}
#endif
#endif
