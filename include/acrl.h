/*
 * acrl.h -- C ABI of libacrl, the MI355X (gfx950) scoring and discrepancy path
 * of ACRL ("Adaptive Control of Training-Inference Discrepancy for Stable RL").
 *
 * The library scores every rollout token under the BF16 training policy pi and
 * the FP8 / MXFP8 inference policy mu, reduces the training-inference
 * discrepancy per sequence, group and batch, and applies the ACRL controller.
 *
 * Conventions shared by every entry point:
 *  - Array arguments are DEVICE pointers (memory of the current HIP device)
 *    unless the comment says "host".  The caller owns all memory; the library
 *    allocates nothing, keeps no per-call state, and writes only the outputs
 *    and the workspace it is given.
 *  - `stream` is a hipStream_t passed as void* (NULL = the legacy default
 *    stream).  Arguments are validated on the host, synchronously; on success
 *    the kernels are enqueued on `stream` and the call returns; results are
 *    ready when the stream has been synchronized.
 *  - Every call returns an acrl_status.  No exception crosses the ABI and the
 *    library never aborts.  acrl_last_error() gives a thread-local message for
 *    the last failing call of the calling thread.
 *  - Calls that share a workspace must not overlap in time.
 *  - Only gfx950 devices are supported (ACRL_ERR_UNSUPPORTED otherwise).
 *  - bf16 tensors are passed as their 16-bit patterns; FP8 tensors are OCP
 *    E4M3 ("fn": bias 7, largest finite 448) bytes; MX scales are OCP E8M0
 *    bytes (value 2^(code-127)).
 *  - Row-major layouts; pointers 16-byte aligned.
 */
#ifndef ACRL_H
#define ACRL_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define ACRL_ABI_VERSION 6

typedef int acrl_status;
enum {
  ACRL_OK = 0,
  ACRL_ERR_INVALID_ARG = 1,   /* a pointer, size or hyper-parameter is out of contract */
  ACRL_ERR_UNSUPPORTED = 2,   /* device is not gfx950, or an unsupported option       */
  ACRL_ERR_WORKSPACE = 3,     /* workspace missing or smaller than the query returns  */
  ACRL_ERR_HIP = 4            /* the HIP runtime reported an error                    */
};

/* Scaling granularity of the FP8 inference policy mu.  The paper's engine
 * quantizes activations per token and weights per channel (Sec. 5.1), and
 * runs MXFP8 for the larger models (Sec. 5.2, 5.4).                          */
typedef enum {
  ACRL_SCALE_PER_TENSOR = 0,  /* one fp32 scale for the whole matrix               */
  ACRL_SCALE_PER_ROW = 1,     /* one fp32 scale per row (token / vocabulary row)    */
  ACRL_SCALE_MX32 = 2         /* one E8M0 scale per 32 consecutive elements of a row */
} acrl_scaling;

/* FP8 rounding: nearest-even (the "nearest-around" quantization of Sec. 5.1)
 * or toward zero (the truncated FP8 of the stress test, Sec. 5.3).          */
typedef enum { ACRL_ROUND_NEAREST_EVEN = 0, ACRL_ROUND_TOWARD_ZERO = 1 } acrl_rounding;

/* Which discrepancy Y enters alpha = gamma*sign(A)*(1 - Y/X) (Sec. 4.1).    */
typedef enum {
  ACRL_Y_GROUP = 0,           /* Y of the response's prompt group (the formula)     */
  ACRL_Y_SEQUENCE = 1,        /* Y of the response itself                           */
  ACRL_Y_BATCH = 2            /* Y of the whole batch                               */
} acrl_y_level;

/* Weighting rule of acrl_controller_step. */
typedef enum {
  ACRL_CTRL_ACRL = 0,         /* Eq. ACRL: rho = (pi/mu)^alpha, alpha = gamma sign(A)(1 - Y/X) */
  ACRL_CTRL_TIS = 1,          /* Eq. tis_objective: token-level min(pi/mu, C)                  */
  ACRL_CTRL_MIS = 2,          /* Eq. mis_objective: the sequence ratio, 0 where it exceeds C   */
  ACRL_CTRL_CONTINUOUS = 3,   /* Sec. 5 ablation "continuous reduction": alpha = -k sign(A)    */
  ACRL_CTRL_FALLBACK = 4      /* Sec. 5 ablation "fallback to GRPO": weight 1 when Y < X       */
} acrl_ctrl_mode;

/* Which policies one acrl_score_pi_mu call scores (acrl_score_desc.policies). */
enum {
  ACRL_POLICY_BOTH = 0,       /* pi and mu (the default)                            */
  ACRL_POLICY_PI = 1,         /* pi only: the mu operands and outputs are not read   */
  ACRL_POLICY_MU = 2          /* mu only: the pi operands and outputs are not read   */
};

/* Slots of the batch statistics vector (double[ACRL_N_STATS]). */
enum {
  ACRL_STAT_Y_BATCH = 0,      /* mean over non-empty groups of Y_g                  */
  ACRL_STAT_TOK_MEAN_D = 1,   /* mean of d over valid tokens                        */
  ACRL_STAT_TOK_MAX_D = 2,    /* max of d over valid tokens                         */
  ACRL_STAT_TOK_STD_D = 3,    /* population standard deviation of d                */
  ACRL_STAT_MEAN_H_PI = 4,    /* mean entropy of pi over valid tokens (0 if absent)  */
  ACRL_STAT_MEAN_H_MU = 5,    /* mean entropy of mu over valid tokens (0 if absent)  */
  ACRL_STAT_N_TOKENS = 6,     /* number of valid tokens                             */
  ACRL_STAT_N_GROUPS = 7,     /* number of groups with a non-empty response         */
  ACRL_STAT_TOK_MEAN_LOGRATIO = 8, /* mean of log(pi/mu) over valid tokens          */
  ACRL_STAT_N_SEQS = 9,       /* number of non-empty responses                      */
  ACRL_N_STATS = 10
};

const char* acrl_status_string(acrl_status status);
const char* acrl_last_error(void);
int acrl_abi_version(void);
/* sizeof of the descriptor structs as compiled into the library (host);
 * bindings compare them with their own layout.  Any pointer may be NULL.    */
void acrl_abi_struct_sizes(size_t* score_desc, size_t* reduce_desc, size_t* controller_desc,
                           size_t* sample_desc, size_t* surrogate_desc, size_t* backward_desc);

/* ======================================================================== */
/* a1/a2  acrl_quantize_fp8 -- FP8 quantization of a bf16 matrix            */
/* ======================================================================== *
 * Quantizes the LM head W (rows = V) for mu once per weight version, and the
 * hidden states H (rows = tokens) every step (Sec. 5.1: per-channel weights,
 * per-token activations; MXFP8 per Sec. 5.2).
 *   x      bf16 [rows, ld], columns [0, cols) are used.  (device)
 *   q      uint8 [rows, cols], dense; E4M3 codes.                  (device, out)
 *   scales PER_TENSOR: float[1]; PER_ROW: float[rows];
 *          MX32: uint8 E8M0 [rows, cols/32].                       (device, out)
 * Definition.  PER_TENSOR / PER_ROW: amax = max |x| over the group, fp32;
 * s = amax / 448 (fp32, correctly rounded; s = 1 if amax == 0);
 * q = e4m3(x / s) with a correctly rounded fp32 divide.  MX32 (OCP MX v1.0):
 * per 32-element block, code = clamp(floor(log2 amax) - 8 + 127, 0, 254)
 * (0 for an all-zero block), q = e4m3(x * 2^(127 - code)).  e4m3() rounds as
 * `rounding` says and saturates magnitudes >= 448 to 448; NaN -> 0x7F|sign.
 * Requirements: rows >= 0, cols > 0 and a multiple of 32, ld >= cols and a
 * multiple of 8.  PER_TENSOR needs a workspace of
 * acrl_quantize_workspace_size() bytes; the others need none (may be NULL).
 */
acrl_status acrl_quantize_workspace_size(int64_t rows, int64_t cols, int scaling, size_t* bytes);
acrl_status acrl_quantize_fp8(const void* x, int64_t rows, int64_t cols, int64_t ld,
                              int scaling, int rounding, void* q, void* scales,
                              void* workspace, size_t workspace_bytes, void* stream);

/* Element-wise fp32 -> E4M3 encoder with the rounding and saturation above
 * (x: float[n], q: uint8[n], device).  A building block and a test hook for
 * the encoder used by acrl_quantize_fp8.                                   */
acrl_status acrl_fp8_encode(const float* x, int64_t n, int rounding, void* q, void* stream);

/* ======================================================================== */
/* a3/a4/a5  acrl_score_pi_mu -- sampled-token log-probs under pi and mu    */
/* ======================================================================== *
 * For every row r (a token with hidden state h_r and sampled id a_r) and both
 * policies: z = (h W^T) / tau over the whole vocabulary, lse = log sum exp z,
 * logp = z[a_r] - lse (= log pi(a_t) or log mu(a_t), the quantities of
 * Eq. distance_metric and of rho in Sec. 4.1), entropy = -sum p log p.
 *   pi: z = (h . W_v) / tau with bf16 operands, fp32 accumulation.
 *   mu: z = s_a s_w[v] (hq . Wq_v) / tau (PER_TENSOR / PER_ROW), or
 *       sum_b 2^(ea_b-127) 2^(ew_vb-127) (hq_b . Wq_vb) / tau (MX32),
 *       with E4M3 operands from acrl_quantize_fp8 and fp32 accumulation.
 * The [rows, V] logits never reach memory: the softmax statistics are reduced
 * inside the GEMM.  Outputs of row r go to slot out_slot[r] (or r if
 * out_slot is NULL); rows with mask[r] == 0 write 0 to their slot; slots not
 * named by any row are not touched.
 * Requirements: n_rows >= 0; d > 0 and d % 128 == 0; V > 0 and V < 2^31;
 * for rows = V and rows = n_rows: (rows rounded up to 256) * d / 8 < 2^32;
 * token ids in [0, V) (else the row's outputs are NaN and *error_flag, if
 * given, becomes nonzero; the flag is never cleared by the library).
 * The workspace holds a tiled copy of W, h, Wq and hq and of the E8M0 scales
 * of Wq and hq (about (3 + 1/32) (V + n_rows) d bytes) besides the per-strip
 * partial states and the work-queue counters of the persistent launches
 * (cleared by the call itself); with packed_weights (acrl_pack_weights) the
 * copies of W and Wq come from there and the workspace holds only the
 * activations' (acrl_score_workspace_query).
 * policies = ACRL_POLICY_PI scores pi only (h, w, logp_pi required; the mu
 * fields are not read and the mu outputs not written), ACRL_POLICY_MU mu only;
 * the full-vocabulary measures need both.
 *
 * Full-vocabulary measures (optional; the paper's measure is the absolute
 * distance on the sampled token, Eq. distance_metric, and it names the KL
 * divergence and the Euclidean distance as the others): with p = softmax of
 * pi's logits and q = softmax of mu's over the whole vocabulary,
 *   kl_pi_mu = sum_v p_v log(p_v / q_v),  kl_mu_pi = sum_v q_v log(q_v / p_v),
 *   l2 = sqrt(sum_v (p_v - q_v)^2),
 * per row (0 for masked rows).  When any of the three is non-NULL, rows are
 * scored in passes of at most div_chunk rows (0 = 16384; the passes that
 * needs share the rows evenly): mu's logits of a pass are kept in the
 * workspace (4 bytes per logit, so V * 4 bytes per row of a pass; larger
 * passes leave fewer partly idle grid ends), and the pi kernel that follows
 * reads them back and accumulates the three measures against mu's lse; the
 * workspace must have acrl_score_div_workspace_size() bytes.  The terms are
 * formed in fp32 relative to mu's lse: rows where |lse_pi - lse_mu| > 32
 * get NaN measures (such policies have nothing in common numerically), and
 * l2 is NaN where its terms cancel so far that its error could exceed ~1e-4
 * (lse_pi several nats above lse_mu; policies that differ by quantization
 * stay far inside).
 */
typedef struct acrl_score_desc {
  int64_t n_rows;               /* rows scored by this call (a chunk of the batch is fine) */
  int64_t d;                    /* hidden size                                              */
  int64_t V;                    /* vocabulary size                                          */
  const void* h;                /* bf16 [n_rows, d]  hidden states (pi input)               */
  const void* w;                /* bf16 [V, d]       LM head of theta_old (pi)              */
  const void* hq;               /* e4m3 [n_rows, d]  quantized hidden states (mu)           */
  const void* hq_scales;        /* scales of hq, layout per mu_scaling                      */
  const void* wq;               /* e4m3 [V, d]       quantized LM head (mu)                 */
  const void* wq_scales;        /* scales of wq, layout per mu_scaling                      */
  int32_t mu_scaling;           /* acrl_scaling used for BOTH hq and wq                     */
  float inv_temperature;        /* 1/tau applied to both policies' logits (> 0)             */
  const int32_t* token_ids;     /* [n_rows] sampled ids a_t                                 */
  const uint8_t* mask;          /* [n_rows] 1 = score this row; NULL = all rows             */
  const int32_t* out_slot;      /* [n_rows] output slot of each row; NULL = identity        */
  float* logp_pi;               /* [slots] out                                              */
  float* logp_mu;               /* [slots] out                                              */
  float* entropy_pi;            /* [slots] out, nullable                                    */
  float* entropy_mu;            /* [slots] out, nullable                                    */
  float* lse_pi;                /* [slots] out, nullable                                    */
  float* lse_mu;                /* [slots] out, nullable                                    */
  float* logit_pi;              /* [slots] out, nullable: z[a_t] under pi                    */
  float* logit_mu;              /* [slots] out, nullable: z[a_t] under mu                    */
  int32_t* error_flag;          /* device int, nullable                                     */
  void* workspace;              /* acrl_score_workspace_size() bytes, device                */
  size_t workspace_bytes;
  float* kl_pi_mu;              /* [slots] out, nullable: KL(pi || mu) over the vocabulary   */
  float* kl_mu_pi;              /* [slots] out, nullable: KL(mu || pi)                       */
  float* l2;                    /* [slots] out, nullable: Euclidean distance of p and q      */
  int64_t div_chunk;            /* rows per pass of the three measures (0 = 16384)           */
  int32_t policies;             /* ACRL_POLICY_*: both (0), pi only or mu only               */
  const void* packed_weights;   /* nullable: W and Wq as acrl_pack_weights laid them out     */
  size_t packed_weights_bytes;  /* acrl_packed_weights_size() bytes when packed_weights set   */
} acrl_score_desc;

acrl_status acrl_score_workspace_size(int64_t n_rows, int64_t d, int64_t V, int mu_scaling,
                                      size_t* bytes);
/* Workspace of the call the descriptor describes (reads n_rows, d, V,
 * mu_scaling, the full-vocabulary outputs, div_chunk and whether
 * packed_weights is set; the pointers are not dereferenced).              */
acrl_status acrl_score_workspace_query(const acrl_score_desc* desc, size_t* bytes);
/* Workspace of a call that also asks for the full-vocabulary measures.      */
acrl_status acrl_score_div_workspace_size(int64_t n_rows, int64_t d, int64_t V, int mu_scaling,
                                          int64_t div_chunk, size_t* bytes);
acrl_status acrl_score_pi_mu(const acrl_score_desc* desc, void* stream);

/* ======================================================================== */
/* Sampling from mu (the step before scoring: the rollout's token draw)      */
/* ======================================================================== *
 For every row r, a draw a_r from softmax(z), with z the mu logits (as in
 * acrl_score_pi_mu, 1/tau applied), by blockwise Gumbel-max.  The vocabulary
 * is cut into blocks of 16 rows: row v lies in block k = 2 floor(v/32) +
 * (floor(v/4) mod 2).  The step runs in three parts.
 *  1. Each block gets one key, lse_k - ln(-ln u_k), with lse_k the
 *     log-sum-exp of its logits.
 *  2. The block of the largest key wins.
 *  3. Inside the winning block, a_r is the first row (in increasing v) whose
 *     cumulative softmax probability within the block exceeds u'_k.
 * This is exactly a draw from softmax(z): the maximum of z_v + Gumbel over a
 * block is lse_k + Gumbel, and the row attaining it has probability
 * exp(z_v - lse_k), independently.  u_k and u'_k are words 2e and 2e+1,
 * with e = floor(k/2) mod 2, of Philox4x32-10 (Salmon et al., SC 2011) on
 * counter (floor(v/64), row_offset + r, k mod 2, 0) under key (seed low,
 * seed high 32 bits), as (w >> 9 + 1/2) 2^-23.  The draw is fused into the
 * mu kernel's epilogue: the logits never reach memory, and one generator
 * call serves 32 logits.  logp_mu[r] (nullable) = log mu(a_r).  The draw
 * depends only on (seed, row_offset + r), so chunked calls reproduce one
 * call.
 * Requirements: as acrl_score_pi_mu for n_rows, d, V, mu_scaling and the
 * operands; workspace of acrl_score_workspace_size() bytes (with
 * packed_weights, what acrl_score_workspace_query gives for a descriptor with
 * the same sizes and packed_weights set suffices).
 */
typedef struct acrl_sample_desc {
  int64_t n_rows;
  int64_t d;
  int64_t V;
  const void* hq;               /* e4m3 [n_rows, d]                                         */
  const void* hq_scales;
  const void* wq;               /* e4m3 [V, d]                                              */
  const void* wq_scales;
  int32_t mu_scaling;
  float inv_temperature;        /* 1/tau (> 0)                                              */
  uint64_t seed;
  int64_t row_offset;           /* global token index of row 0 (>= 0)                       */
  int32_t* ids;                 /* [n_rows] out: sampled vocabulary rows                    */
  float* logp_mu;               /* [n_rows] out, nullable                                   */
  void* workspace;
  size_t workspace_bytes;
  const void* packed_weights;   /* nullable: from acrl_pack_weights (W's part is not read)   */
  size_t packed_weights_bytes;
} acrl_sample_desc;

acrl_status acrl_sample_mu(const acrl_sample_desc* desc, void* stream);

/* Packed LM head (once per weight version).  The scorers stream their
 * operands from a tiled copy: per 256-row tile and 64-byte K chunk, one
 * contiguous 16 KiB image of the tile's rows, each row's four 16-byte pieces
 * at positions c ^ ((row / 4) mod 4), rows past V repeating row V-1; for MX32
 * also the E8M0 scales of Wq per tile and chunk.  acrl_pack_weights writes
 * that copy of W and Wq (and Wq's MX scales) into caller-owned device memory
 * of acrl_packed_weights_size() bytes; passing it as packed_weights to
 * acrl_score_pi_mu / acrl_sample_mu skips their own packing of W and Wq, so
 * the per-step calls pack only the activations.  Valid as long as W, Wq and
 * their scales do not change (the weights of theta_old are quantized once
 * per weight version, Sec. 5.1).  w, wq, wq_scales: as acrl_score_pi_mu's;
 * same requirements on V, d and the alignment.                              */
acrl_status acrl_packed_weights_size(int64_t V, int64_t d, int mu_scaling, size_t* bytes);
acrl_status acrl_pack_weights(const void* w, const void* wq, const void* wq_scales, int64_t V, int64_t d,
                              int mu_scaling, void* packed, size_t packed_bytes, void* stream);

/* ======================================================================== */
/* a6/a7  acrl_discrepancy_reduce -- per-token d, segmented reductions       */
/* ======================================================================== *
 * Slots are [B, L] (slot of response i, position j is i*L + j).  For valid
 * slots (mask != 0): d = |exp(logp_pi) - exp(logp_mu)| (Eq. distance_metric,
 * on probabilities) and the log-ratio log(pi/mu) = logp_pi - logp_mu.
 * Per response i: |a_i| = valid count, sums of d and of the log-ratio (the
 * latter is log rho_i of sequence-level MIS, Sec. 2.2), mean d.
 * Per group g (the G responses of one prompt): Y_g = mean over the group's
 * non-empty responses of their mean d (the formula for Y in Sec. 4.1).
 * Batch: mean over non-empty groups of Y_g (the outer mean of X, Sec. 4.1) and
 * the token-level statistics of ACRL_STAT_*.  Sums are accumulated in fp64;
 * the standard deviation merges per-piece squared deviations pairwise
 * (Chan, Golub and LeVeque), so every slot is read once.  Results are
 * deterministic (fixed reduction trees, no floating-point atomics).
 * Requirements: B, L, n_groups >= 0 (n_groups > 0 when B > 0);
 * group_of_seq[i] in [0, n_groups) (device data, not checked: a response
 * with another id belongs to no group and enters no batch statistic).
 * Grouping the responses of a prompt together (non-decreasing group_of_seq)
 * lets each group find its responses by binary search instead of a scan.
 */
typedef struct acrl_reduce_desc {
  int64_t B;                    /* responses                                                */
  int64_t L;                    /* slots per response                                       */
  int64_t n_groups;             /* prompts                                                  */
  const float* logp_pi;         /* [B*L]                                                    */
  const float* logp_mu;         /* [B*L]                                                    */
  const float* entropy_pi;      /* [B*L], nullable                                          */
  const float* entropy_mu;      /* [B*L], nullable                                          */
  const uint8_t* mask;          /* [B*L]                                                    */
  const int32_t* group_of_seq;  /* [B] prompt index of each response                        */
  float* d_tok;                 /* [B*L] out, nullable: d (0 where masked)                  */
  int32_t* seq_len;             /* [B] out, nullable                                        */
  double* seq_sum_d;            /* [B] out, nullable                                        */
  double* seq_sum_logratio;     /* [B] out, nullable                                        */
  float* seq_mean_d;            /* [B] out (0 for an empty response)                        */
  float* group_y;               /* [n_groups] out (0 for an empty group)                    */
  int32_t* group_nseq;          /* [n_groups] out, nullable: non-empty responses per group  */
  double* stats;                /* [ACRL_N_STATS] out                                       */
  void* workspace;              /* acrl_reduce_workspace_size() bytes, device               */
  size_t workspace_bytes;
} acrl_reduce_desc;

acrl_status acrl_reduce_workspace_size(int64_t B, int64_t L, int64_t n_groups, size_t* bytes);
acrl_status acrl_discrepancy_reduce(const acrl_reduce_desc* desc, void* stream);

/* acrl_discrepancy_reduce_noalloc -- the same reduce for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc).  It computes exactly what
 * acrl_discrepancy_reduce computes, with the same kernels, but takes its
 * intermediate records from a fixed device array of ACRL_REDUCE_SCRATCH_BYTES
 * that the library holds on each device it runs on, for the life of the
 * process; desc->workspace and desc->workspace_bytes are ignored.  It calls
 * no hipMalloc / hipFree and allocates nothing.
 * Limit: acrl_reduce_workspace_size(B, L, n_groups) (64 bytes per response,
 * 144 per group, plus alignment) must not exceed ACRL_REDUCE_SCRATCH_BYTES
 * (4 MiB: e.g. 49152 responses in 4096 groups); larger batches get
 * ACRL_ERR_WORKSPACE.
 * Every call on a device shares that device's array, which keeps the last
 * call's contents (each call clears what it needs): calls that overlap in
 * time on one device (different streams or threads) race and must be
 * serialized by the caller.  Other requirements and errors as
 * acrl_discrepancy_reduce.                                                  */
#define ACRL_REDUCE_SCRATCH_BYTES (4u << 20)
acrl_status acrl_discrepancy_reduce_noalloc(const acrl_reduce_desc* desc, void* stream);

/* ======================================================================== */
/* a8  acrl_controller_step -- ACRL per-token weights                       */
/* ======================================================================== *
 * Eq. ACRL (mode ACRL_CTRL_ACRL): the clipped surrogate of every valid token
 * is weighted by min(rho, C) with rho = (pi(a_t)/mu(a_t))^alpha and
 * alpha = gamma * sign(A) * (1 - Y/X) (sign(0) = 0).  Computed as
 * weight = exp(min(alpha * (logp_pi - logp_mu), ln C)), which equals
 * min(rho, C).  Masked slots get alpha = 0 and weight = 0.
 * Y comes from seq_mean_d[i], group_y[group_of_seq[i]] or
 * stats[ACRL_STAT_Y_BATCH] per y_level (outputs of acrl_discrepancy_reduce).
 * Other modes (alpha output in parentheses):
 *   ACRL_CTRL_TIS        weight = min(pi/mu, C)                     (1)
 *   ACRL_CTRL_MIS        weight = rho_i if rho_i <= C, else 0, for every valid
 *                        token of sequence i, rho_i = exp(seq_sum_logratio[i])
 *                        (the output of acrl_discrepancy_reduce)       (1)
 *   ACRL_CTRL_CONTINUOUS alpha = -k sign(A), weight = min((pi/mu)^alpha, C)
 *   ACRL_CTRL_FALLBACK   Y < X: weight = 1 (plain GRPO)             (0);
 *                        otherwise as ACRL_CTRL_ACRL
 * Requirements: X > 0, gamma > 0, C > 1 (Sec. 4.1); k > 0 for CONTINUOUS;
 * seq_sum_logratio non-NULL for MIS; the arrays y_level reads non-NULL for
 * ACRL and FALLBACK.
 * Undefined inputs give NaN, never the clip C: a valid slot whose log-prob is
 * NaN (acrl_score_pi_mu's mark of an invalid token id) gets weight NaN, and a
 * response whose group id lies outside [0, n_groups) gets alpha = NaN and
 * weight = NaN under ACRL_Y_GROUP (ACRL and FALLBACK modes).
 */
typedef struct acrl_controller_desc {
  int64_t B;
  int64_t L;
  int64_t n_groups;             /* prompts; group ids outside [0, n_groups) give NaN        */
  const uint8_t* mask;          /* [B*L]                                                    */
  const int32_t* group_of_seq;  /* [B] (needed for ACRL_Y_GROUP)                            */
  const float* logp_pi;         /* [B*L]                                                    */
  const float* logp_mu;         /* [B*L]                                                    */
  const float* adv;             /* [B] or [B*L] advantages A                                */
  int32_t adv_per_token;        /* 0: adv is [B] (GRPO); 1: adv is [B*L] (PPO)              */
  int32_t y_level;              /* acrl_y_level                                             */
  const float* seq_mean_d;      /* [B]                                                      */
  const float* group_y;         /* [n_groups]                                               */
  const double* stats;          /* [ACRL_N_STATS]                                           */
  float X;                      /* reference discrepancy, > 0                               */
  float gamma;                  /* control strength, > 0                                    */
  float C;                      /* clip, > 1                                                */
  float* alpha;                 /* [B*L] out, nullable                                      */
  float* weight;                /* [B*L] out                                                */
  int32_t mode;                 /* acrl_ctrl_mode (0 = ACRL)                                 */
  float k;                      /* |alpha| of ACRL_CTRL_CONTINUOUS, > 0                     */
  const double* seq_sum_logratio; /* [B] (ACRL_CTRL_MIS)                                    */
} acrl_controller_desc;

acrl_status acrl_controller_step(const acrl_controller_desc* desc, void* stream);

/* ======================================================================== */
/* acrl_surrogate -- the ACRL-weighted clipped surrogate and d loss/d logp   */
/* ======================================================================== *
 * Eq. ACRL (Sec. 4.1) weights the clipped objective of Eq. grpo_objective
 * (Sec. 2) token by token with w_t = min(rho_t, C):
 *   J = (1/P) sum_g (1/G_g) sum_{i in g} (1/|a_i|) sum_t w_t min(r_t A_t, clip(r_t) A_t),
 *   r_t = exp(logp_new - logp_old), clip(r) = min(max(r, 1 - eps_low), 1 + eps_high),
 * over the valid slots (mask != 0); G_g counts the non-empty responses of
 * prompt g and P the prompts with at least one (empty responses contribute
 * nothing).  loss[0] = -J (fp64).  coef[t] = d loss / d logp_new[t] =
 * -w_t r_t A_t / (P G_g |a_i|) where the unclipped term is the minimum (a tie
 * counts as unclipped), 0 where the clipped term is, 0 for masked slots,
 * NaN for a response whose group id lies outside [0, n_groups).  w_t is held
 * constant (it is the controller's output for the behaviour policy);
 * weight == NULL means w = 1 (plain GRPO).  r, the clip and the sums are
 * evaluated in fp64 from the fp32 inputs.
 * Requirements: B, L, n_groups >= 0 (n_groups > 0 if B > 0);
 * eps_low in [0, 1), eps_high >= 0; workspace of
 * acrl_surrogate_workspace_size() bytes.                                    */
typedef struct acrl_surrogate_desc {
  int64_t B;
  int64_t L;
  int64_t n_groups;
  const uint8_t* mask;          /* [B*L]                                                    */
  const int32_t* group_of_seq;  /* [B]                                                      */
  const float* logp_new;        /* [B*L] log pi_theta(a_t) of the policy being trained       */
  const float* logp_old;        /* [B*L] log pi_theta_old(a_t)                              */
  const float* adv;             /* [B] or [B*L] advantages A                                */
  int32_t adv_per_token;        /* 0: adv is [B]; 1: adv is [B*L]                           */
  float eps_low;                /* clip range of r: [1 - eps_low, 1 + eps_high]             */
  float eps_high;
  const float* weight;          /* [B*L] w_t = min(rho, C) (acrl_controller_step), nullable */
  float* coef;                  /* [B*L] out: d loss / d logp_new                           */
  double* loss;                 /* [1] out: -J                                              */
  void* workspace;
  size_t workspace_bytes;
} acrl_surrogate_desc;

acrl_status acrl_surrogate_workspace_size(int64_t B, int64_t n_groups, size_t* bytes);
acrl_status acrl_surrogate(const acrl_surrogate_desc* desc, void* stream);

/* ======================================================================== */
/* acrl_lm_head_backward -- gradient of the surrogate w.r.t. H and W        */
/* ======================================================================== *
 * With z_t = (W h_t) / tau (bf16 operands, fp32 accumulation) and
 * p_t = softmax(z_t), the loss depends on H and W through
 * logp_new[t] = z_t[a_t] - lse_t, so by the chain rule
 *   dZ[t, v] = coef_t (delta(v, a_t) - p_tv) / tau,
 *   dH = dZ W  ([n_rows, d]),   dW = dZ^T H  ([V, d]).
 * p is recomputed from the logits and the row's lse (acrl_score_pi_mu's
 * lse_pi output for the same h, W, tau); dZ is rounded to bf16 and lives only
 * in the workspace (one pass of token_chunk rows at a time); dH and dW are
 * the products of the bf16 operands accumulated in fp32.  Rows with coef 0
 * (masked slots) contribute nothing.  An id outside [0, V) contributes no
 * one-hot term.
 *   coef, lse  slot arrays: row r reads slot row_slot[r] (r if row_slot is NULL).
 *   dh         [n_rows, d] fp32 out, nullable (not computed).
 *   dw         [V, d] fp32 out, nullable; dw = dW, or dw += dW with
 *              accumulate_dw = 1 (chunked calls).
 * Requirements: n_rows >= 0; d > 0, d % 128 == 0; 0 < V < 2^23;
 * (V rounded up to 256) * d / 8 < 2^32; token_chunk >= 0 (0 = 16384; rounded
 * up to a multiple of 256; at most 2^23); workspace of
 * acrl_backward_workspace_size() bytes (packed W, W^T, one chunk of H, H^T
 * and two bf16 copies of its dZ: about 4 V d + 4 c d + 4 c V bytes for a
 * chunk of c rows; plus the products' work-queue counters, cleared by the
 * call).                                                                    */
typedef struct acrl_backward_desc {
  int64_t n_rows;
  int64_t d;
  int64_t V;
  const void* h;                /* bf16 [n_rows, d]                                         */
  const void* w;                /* bf16 [V, d]                                              */
  const int32_t* token_ids;     /* [n_rows] a_t                                             */
  const int32_t* row_slot;      /* [n_rows] slot of each row in coef / lse; NULL = identity */
  const float* coef;            /* [slots] d loss / d logp_new (acrl_surrogate)             */
  const float* lse;             /* [slots] log-sum-exp of pi's logits (natural units)       */
  float inv_temperature;        /* 1/tau (> 0), as in the forward pass                      */
  float* dh;                    /* [n_rows, d] out, nullable                                */
  float* dw;                    /* [V, d] out, nullable                                     */
  int32_t accumulate_dw;        /* 1: dw += dW                                              */
  int64_t token_chunk;          /* rows per internal pass (0 = default)                     */
  void* workspace;
  size_t workspace_bytes;
} acrl_backward_desc;

acrl_status acrl_backward_workspace_size(int64_t n_rows, int64_t d, int64_t V, int64_t token_chunk,
                                         size_t* bytes);
acrl_status acrl_lm_head_backward(const acrl_backward_desc* desc, void* stream);

/* Host helper (host pointers): the reference discrepancy X of Sec. 4.1 is the
 * mean of Y_g over the non-empty groups (group_nseq > 0) of the step-0
 * batches.  Returns ACRL_ERR_INVALID_ARG if no group is non-empty.          */
acrl_status acrl_reference_from_groups(const float* group_y, const int32_t* group_nseq,
                                       int64_t n_groups, float* X_out);

#ifdef __cplusplus
}
#endif
#endif /* ACRL_H */
