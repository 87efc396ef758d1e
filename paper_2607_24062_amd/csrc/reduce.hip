// reduce.hip -- per-token training-inference discrepancy, its segmented
// masked reductions, and the ACRL controller step.
//
//  * d = |pi(a_t) - mu(a_t)| on probabilities (Eq. distance_metric) and the
//    log-ratio log(pi/mu) (the log of rho in Sec. 2.2 / 4.1).
//  * Per response: |a_i|, sum d, sum log-ratio (log rho_i of sequence-level
//    MIS), mean d.  Per group (the G responses of a prompt): Y_g, the formula
//    of Y in Sec. 4.1.  Batch: mean of Y_g (the outer mean of X) and token
//    statistics (mean / max / population std of d, mean entropies).
//  * Controller (Eq. ACRL): weight = min((pi/mu)^alpha, C),
//    alpha = gamma sign(A) (1 - Y/X).
//
// Layout: slots [B, L] row-major, the usual right-padded response layout.
// One workgroup per response reads its L contiguous slots with coalesced
// loads; all sums are fp64 and combined by fixed-shape tree reductions, so
// results are deterministic (no floating-point atomics).  These kernels are
// HBM / latency bound; the controller is a plain grid-stride stream.
#include "acrl_internal.h"

namespace acrl {
namespace {

constexpr int kRedThreads = 256;

// Per-response intermediate record in the workspace.
struct SeqRec {
  double n, sum_d, sum_lr, sum_hp, sum_hm, max_d, m2;  // m2 = sum (d - mean_i)^2
  double pad;
};

__device__ __forceinline__ double block_sum(double v, double* sh) {
  v = wave_sum(v);
  const int w = threadIdx.x >> 6;
  __syncthreads();
  if ((threadIdx.x & 63) == 0) sh[w] = v;
  __syncthreads();
  double t = 0.0;
  for (int k = 0; k < (int)(blockDim.x >> 6); ++k) t += sh[k];
  return t;
}

__device__ __forceinline__ double block_max(double v, double* sh) {
#pragma unroll
  for (int m = 1; m < 64; m <<= 1) v = fmax(v, __shfl_xor(v, m));
  const int w = threadIdx.x >> 6;
  __syncthreads();
  if ((threadIdx.x & 63) == 0) sh[w] = v;
  __syncthreads();
  double t = sh[0];
  for (int k = 1; k < (int)(blockDim.x >> 6); ++k) t = fmax(t, sh[k]);
  return t;
}

__device__ __forceinline__ double token_distance(float lp_pi, float lp_mu) {
  return fabs(exp((double)lp_pi) - exp((double)lp_mu));
}

// One workgroup per response.
__global__ __launch_bounds__(kRedThreads) void reduce_seq_kernel(acrl_reduce_desc p, SeqRec* rec) {
  __shared__ double sh[kRedThreads / 64];
  const int64_t i = blockIdx.x;
  const int64_t base = i * p.L;
  double n = 0, sd = 0, sl = 0, shp = 0, shm = 0, mx = 0;
  for (int64_t j = threadIdx.x; j < p.L; j += kRedThreads) {
    const int64_t t = base + j;
    float dtok = 0.0f;
    if (p.mask[t]) {
      const float a = p.logp_pi[t], b = p.logp_mu[t];
      const double dv = token_distance(a, b);
      n += 1.0;
      sd += dv;
      sl += (double)a - (double)b;
      if (p.entropy_pi) shp += p.entropy_pi[t];
      if (p.entropy_mu) shm += p.entropy_mu[t];
      mx = fmax(mx, dv);
      dtok = (float)dv;
    }
    if (p.d_tok) p.d_tok[t] = dtok;
  }
  n = block_sum(n, sh);
  sd = block_sum(sd, sh);
  sl = block_sum(sl, sh);
  shp = block_sum(shp, sh);
  shm = block_sum(shm, sh);
  mx = block_max(mx, sh);
  const double mean = n > 0 ? sd / n : 0.0;
  double m2 = 0.0;  // second pass over the (cached) slots: squared deviations
  for (int64_t j = threadIdx.x; j < p.L; j += kRedThreads) {
    const int64_t t = base + j;
    if (p.mask[t]) {
      const double dv = token_distance(p.logp_pi[t], p.logp_mu[t]) - mean;
      m2 += dv * dv;
    }
  }
  m2 = block_sum(m2, sh);
  if (threadIdx.x == 0) {
    SeqRec r;
    r.n = n; r.sum_d = sd; r.sum_lr = sl; r.sum_hp = shp; r.sum_hm = shm; r.max_d = mx; r.m2 = m2;
    r.pad = 0;
    rec[i] = r;
    if (p.seq_len) p.seq_len[i] = (int32_t)n;
    if (p.seq_sum_d) p.seq_sum_d[i] = sd;
    if (p.seq_sum_logratio) p.seq_sum_logratio[i] = sl;
    p.seq_mean_d[i] = (float)mean;
  }
}

// One workgroup per group: Y_g over the group's non-empty responses.
__global__ __launch_bounds__(kRedThreads) void reduce_group_kernel(acrl_reduce_desc p,
                                                                   const SeqRec* rec,
                                                                   double* gy, double* gcount) {
  __shared__ double sh[kRedThreads / 64];
  const int g = blockIdx.x;
  double s = 0, c = 0;
  for (int64_t i = threadIdx.x; i < p.B; i += kRedThreads) {
    if (p.group_of_seq[i] == g && rec[i].n > 0) {
      s += rec[i].sum_d / rec[i].n;
      c += 1.0;
    }
  }
  s = block_sum(s, sh);
  c = block_sum(c, sh);
  if (threadIdx.x == 0) {
    const double y = c > 0 ? s / c : 0.0;
    gy[g] = y;
    gcount[g] = c;
    p.group_y[g] = (float)y;
    if (p.group_nseq) p.group_nseq[g] = (int32_t)c;
  }
}

// One workgroup: batch statistics.
__global__ __launch_bounds__(kRedThreads) void reduce_batch_kernel(acrl_reduce_desc p,
                                                                   const SeqRec* rec,
                                                                   const double* gy,
                                                                   const double* gcount) {
  __shared__ double sh[kRedThreads / 64];
  double n = 0, sd = 0, sl = 0, shp = 0, shm = 0, mx = 0, ns = 0;
  for (int64_t i = threadIdx.x; i < p.B; i += kRedThreads) {
    const SeqRec r = rec[i];
    n += r.n; sd += r.sum_d; sl += r.sum_lr; shp += r.sum_hp; shm += r.sum_hm;
    mx = fmax(mx, r.max_d);
    ns += r.n > 0 ? 1.0 : 0.0;
  }
  n = block_sum(n, sh);
  sd = block_sum(sd, sh);
  sl = block_sum(sl, sh);
  shp = block_sum(shp, sh);
  shm = block_sum(shm, sh);
  mx = block_max(mx, sh);
  ns = block_sum(ns, sh);
  const double mean = n > 0 ? sd / n : 0.0;
  // total squared deviation from the per-response ones (parallel-variance merge)
  double m2 = 0;
  for (int64_t i = threadIdx.x; i < p.B; i += kRedThreads) {
    const SeqRec r = rec[i];
    if (r.n > 0) {
      const double dm = r.sum_d / r.n - mean;
      m2 += r.m2 + r.n * dm * dm;
    }
  }
  m2 = block_sum(m2, sh);
  double ys = 0, ng = 0;
  for (int64_t g = threadIdx.x; g < p.n_groups; g += kRedThreads) {
    if (gcount[g] > 0) {
      ys += gy[g];
      ng += 1.0;
    }
  }
  ys = block_sum(ys, sh);
  ng = block_sum(ng, sh);
  if (threadIdx.x == 0) {
    double* st = p.stats;
    st[ACRL_STAT_Y_BATCH] = ng > 0 ? ys / ng : 0.0;
    st[ACRL_STAT_TOK_MEAN_D] = mean;
    st[ACRL_STAT_TOK_MAX_D] = mx;
    st[ACRL_STAT_TOK_STD_D] = n > 0 ? sqrt(m2 / n) : 0.0;
    st[ACRL_STAT_MEAN_H_PI] = n > 0 ? shp / n : 0.0;
    st[ACRL_STAT_MEAN_H_MU] = n > 0 ? shm / n : 0.0;
    st[ACRL_STAT_N_TOKENS] = n;
    st[ACRL_STAT_N_GROUPS] = ng;
    st[ACRL_STAT_TOK_MEAN_LOGRATIO] = n > 0 ? sl / n : 0.0;
    st[ACRL_STAT_N_SEQS] = ns;
  }
}

// Element-wise controller.  alpha and the weight are evaluated in fp64 from
// the fp32 inputs (exact conversions), then rounded to fp32 once.  Modes:
// Eq. ACRL, token-level TIS (Eq. tis_objective), sequence-level MIS (Eq.
// mis_objective, from the fp64 per-sequence log-ratio sums of the reduce),
// and the continuous-reduction / fallback-to-GRPO ablations of Sec. 5.
__global__ __launch_bounds__(256) void controller_kernel(acrl_controller_desc p) {
  const int64_t n = p.B * p.L;
  const double X = p.X, gamma = p.gamma, lnC = log((double)p.C), C = p.C;
  for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < n;
       t += (int64_t)gridDim.x * blockDim.x) {
    float a_out = 0.0f, w_out = 0.0f;
    if (p.mask[t]) {
      const int64_t i = t / p.L;
      const double A = p.adv_per_token ? p.adv[t] : p.adv[i];
      const double sg = (A > 0) - (A < 0);
      const double lr = (double)p.logp_pi[t] - (double)p.logp_mu[t];  // ln(pi/mu)
      if (p.mode == ACRL_CTRL_MIS) {
        const double s = p.seq_sum_logratio[i];  // ln rho_i
        a_out = 1.0f;
        w_out = s <= lnC ? (float)exp(s) : 0.0f;
      } else if (p.mode == ACRL_CTRL_TIS) {
        a_out = 1.0f;
        w_out = (float)(lr < lnC ? exp(lr) : C);
      } else {
        double alpha;
        bool grpo = false;
        if (p.mode == ACRL_CTRL_CONTINUOUS) {
          alpha = -(double)p.k * sg;
        } else {
          double Y;
          if (p.y_level == ACRL_Y_SEQUENCE) Y = p.seq_mean_d[i];
          else if (p.y_level == ACRL_Y_GROUP) {
            const int32_t g = p.group_of_seq[i];
            Y = (g >= 0 && g < p.n_groups) ? (double)p.group_y[g] : __builtin_nan("");
          }
          else Y = p.stats[ACRL_STAT_Y_BATCH];
          grpo = p.mode == ACRL_CTRL_FALLBACK && Y < X;
          alpha = gamma * sg * (1.0 - Y / X);
        }
        if (grpo) {
          a_out = 0.0f;
          w_out = 1.0f;
        } else {
          const double e = alpha * lr;  // ln rho
          a_out = (float)alpha;
          w_out = (float)(e < lnC ? exp(e) : C);
        }
      }
    }
    if (p.alpha) p.alpha[t] = a_out;
    p.weight[t] = w_out;
  }
}

// ------------------------------------------------------------------ surrogate
// The ACRL-weighted clipped surrogate (Eq. ACRL on top of the GRPO objective
// of Sec. 2): J = mean over prompts of (1/G) sum_i (1/|a_i|) sum_t
// w_t min(r_t A_t, clip(r_t) A_t), r_t = exp(logp_new - logp_old); the
// prompts averaged are those with a non-empty response and G counts a
// prompt's non-empty responses.  loss = -J, coef_t = d loss / d logp_new_t.

struct SurrSeq {
  double n, J;  // |a_i| and sum_t w_t min(r A, clip(r) A)
};

// r A, clip(r) A and whether the unclipped term is the minimum (a tie counts
// as unclipped), in fp64 from the fp32 inputs.
__device__ __forceinline__ void surr_terms(const acrl_surrogate_desc& p, int64_t t, int64_t i, double& r,
                                           double& A, double& m, bool& unclipped) {
  A = p.adv_per_token ? p.adv[t] : p.adv[i];
  r = exp((double)p.logp_new[t] - (double)p.logp_old[t]);
  const double rc = fmin(fmax(r, 1.0 - (double)p.eps_low), 1.0 + (double)p.eps_high);
  const double u = r * A, c = rc * A;
  unclipped = u <= c;
  m = unclipped ? u : c;
}

// One workgroup per response.
__global__ __launch_bounds__(kRedThreads) void surr_seq_kernel(acrl_surrogate_desc p, SurrSeq* rec) {
  __shared__ double sh[kRedThreads / 64];
  const int64_t i = blockIdx.x;
  double n = 0, J = 0;
  for (int64_t j = threadIdx.x; j < p.L; j += kRedThreads) {
    const int64_t t = i * p.L + j;
    if (!p.mask[t]) continue;
    double r, A, m;
    bool unc;
    surr_terms(p, t, i, r, A, m, unc);
    n += 1.0;
    J += (p.weight ? (double)p.weight[t] : 1.0) * m;
  }
  n = block_sum(n, sh);
  J = block_sum(J, sh);
  if (threadIdx.x == 0) rec[i] = SurrSeq{n, J};
}

// One workgroup per group: G_g and the group's sum of per-response means.
__global__ __launch_bounds__(kRedThreads) void surr_group_kernel(acrl_surrogate_desc p, const SurrSeq* rec,
                                                                 double* gG, double* gJ) {
  __shared__ double sh[kRedThreads / 64];
  const int g = blockIdx.x;
  double G = 0, J = 0;
  for (int64_t i = threadIdx.x; i < p.B; i += kRedThreads)
    if (p.group_of_seq[i] == g && rec[i].n > 0) {
      G += 1.0;
      J += rec[i].J / rec[i].n;
    }
  G = block_sum(G, sh);
  J = block_sum(J, sh);
  if (threadIdx.x == 0) {
    gG[g] = G;
    gJ[g] = J;
  }
}

// One workgroup: the number of prompts and the loss.
__global__ __launch_bounds__(kRedThreads) void surr_batch_kernel(acrl_surrogate_desc p, const double* gG,
                                                                 const double* gJ, double* prompts) {
  __shared__ double sh[kRedThreads / 64];
  double np = 0, J = 0;
  for (int64_t g = threadIdx.x; g < p.n_groups; g += kRedThreads)
    if (gG[g] > 0) {
      np += 1.0;
      J += gJ[g] / gG[g];
    }
  np = block_sum(np, sh);
  J = block_sum(J, sh);
  if (threadIdx.x == 0) {
    prompts[0] = np;
    p.loss[0] = np > 0 ? -J / np : 0.0;
  }
}

// Element-wise: coef_t = -w_t r_t A_t / (prompts G_g |a_i|) where the
// unclipped term is the minimum, else 0 (the clipped term does not depend on
// logp_new); masked slots 0; a group id outside [0, n_groups) gives NaN.
__global__ __launch_bounds__(256) void surr_coef_kernel(acrl_surrogate_desc p, const SurrSeq* rec, const double* gG,
                                                        const double* prompts) {
  const int64_t n = p.B * p.L;
  for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < n; t += (int64_t)gridDim.x * blockDim.x) {
    float out = 0.0f;
    if (p.mask[t]) {
      const int64_t i = t / p.L;
      const int32_t g = p.group_of_seq[i];
      if (g < 0 || g >= p.n_groups) {
        out = __builtin_nanf("");
      } else {
        double r, A, m;
        bool unc;
        surr_terms(p, t, i, r, A, m, unc);
        if (unc) {
          const double c = 1.0 / (prompts[0] * gG[g] * rec[i].n);
          out = (float)(-c * (p.weight ? (double)p.weight[t] : 1.0) * r * A);
        }
      }
    }
    p.coef[t] = out;
  }
}

inline size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

}  // namespace

size_t surrogate_workspace_bytes(int64_t B, int64_t n_groups) {
  return align_up((size_t)B * sizeof(SurrSeq), 256) + 2 * align_up((size_t)n_groups * sizeof(double), 256) + 256;
}

hipError_t launch_surrogate(const acrl_surrogate_desc& p, hipStream_t s) {
  uint8_t* ws = static_cast<uint8_t*>(p.workspace);
  SurrSeq* rec = reinterpret_cast<SurrSeq*>(ws);
  size_t off = align_up((size_t)p.B * sizeof(SurrSeq), 256);
  double* gG = reinterpret_cast<double*>(ws + off);
  off += align_up((size_t)p.n_groups * sizeof(double), 256);
  double* gJ = reinterpret_cast<double*>(ws + off);
  off += align_up((size_t)p.n_groups * sizeof(double), 256);
  double* prompts = reinterpret_cast<double*>(ws + off);
  if (p.B > 0)
    hipLaunchKernelGGL(surr_seq_kernel, dim3((unsigned)p.B), dim3(kRedThreads), 0, s, p, rec);
  if (p.n_groups > 0)
    hipLaunchKernelGGL(surr_group_kernel, dim3((unsigned)p.n_groups), dim3(kRedThreads), 0, s, p,
                       (const SurrSeq*)rec, gG, gJ);
  hipLaunchKernelGGL(surr_batch_kernel, dim3(1), dim3(kRedThreads), 0, s, p, (const double*)gG, (const double*)gJ,
                     prompts);
  const int64_t n = p.B * p.L;
  if (n > 0) {
    int64_t g = (n + 255) / 256;
    if (g > 8192) g = 8192;
    hipLaunchKernelGGL(surr_coef_kernel, dim3((unsigned)g), dim3(256), 0, s, p, (const SurrSeq*)rec,
                       (const double*)gG, (const double*)prompts);
  }
  return hipGetLastError();
}

size_t reduce_workspace_bytes(int64_t B, int64_t L, int64_t n_groups) {
  (void)L;
  return align_up((size_t)B * sizeof(SeqRec), 256) + 2 * align_up((size_t)n_groups * sizeof(double), 256);
}

hipError_t launch_reduce(const acrl_reduce_desc& p, hipStream_t s) {
  uint8_t* ws = static_cast<uint8_t*>(p.workspace);
  SeqRec* rec = reinterpret_cast<SeqRec*>(ws);
  double* gy = reinterpret_cast<double*>(ws + align_up((size_t)p.B * sizeof(SeqRec), 256));
  double* gc = gy + align_up((size_t)p.n_groups * sizeof(double), 256) / sizeof(double);
  if (p.B > 0)
    hipLaunchKernelGGL(reduce_seq_kernel, dim3((unsigned)p.B), dim3(kRedThreads), 0, s, p, rec);
  if (p.n_groups > 0)
    hipLaunchKernelGGL(reduce_group_kernel, dim3((unsigned)p.n_groups), dim3(kRedThreads), 0, s, p,
                       (const SeqRec*)rec, gy, gc);
  hipLaunchKernelGGL(reduce_batch_kernel, dim3(1), dim3(kRedThreads), 0, s, p, (const SeqRec*)rec,
                     (const double*)gy, (const double*)gc);
  return hipGetLastError();
}

hipError_t launch_controller(const acrl_controller_desc& p, hipStream_t s) {
  const int64_t n = p.B * p.L;
  if (n == 0) return hipSuccess;
  int64_t g = (n + 255) / 256;
  if (g > 8192) g = 8192;
  hipLaunchKernelGGL(controller_kernel, dim3((unsigned)g), dim3(256), 0, s, p);
  return hipGetLastError();
}

}  // namespace acrl
