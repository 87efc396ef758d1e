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
#include <mutex>

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

// Count, mean and sum of squared deviations of a set of values; two sets
// combine exactly in real arithmetic (the pairwise update of Chan, Golub and
// LeVeque), so the squared deviations need no second pass over the slots.
struct Var {
  double n, mu, m2;
};
__device__ __forceinline__ Var var_merge(const Var& a, const Var& b) {
  if (b.n == 0.0) return a;
  if (a.n == 0.0) return b;
  const double n = a.n + b.n, d = b.mu - a.mu, f = b.n / n;
  return Var{n, a.mu + d * f, a.m2 + b.m2 + d * d * a.n * f};
}

// Block-wide sums of NS values, their maximum and the merge of the threads'
// Vars, with one barrier: shuffle trees inside each wavefront, then every
// thread combines the wavefronts' results in wavefront order, so all threads
// hold the (deterministic) totals.  A second call on the same shared memory
// needs a barrier in between.
template <int NS, int NT = kRedThreads>
struct BlockShared {
  double s[NT / 64][NS];
  double mx[NT / 64];
  Var var[NT / 64];
};
template <int NS, int NT = kRedThreads>
__device__ __forceinline__ void block_stats(double (&v)[NS], double& mx, Var& var, BlockShared<NS, NT>& sh) {
  const int w = threadIdx.x >> 6;
#pragma unroll
  for (int k = 0; k < NS; ++k) v[k] = wave_sum(v[k]);
#pragma unroll
  for (int m = 1; m < 64; m <<= 1) {
    mx = fmax(mx, __shfl_xor(mx, m));
    var = var_merge(var, Var{__shfl_xor(var.n, m), __shfl_xor(var.mu, m), __shfl_xor(var.m2, m)});
  }
  if ((threadIdx.x & 63) == 0) {
#pragma unroll
    for (int k = 0; k < NS; ++k) sh.s[w][k] = v[k];
    sh.mx[w] = mx;
    sh.var[w] = var;
  }
  __syncthreads();
#pragma unroll
  for (int k = 0; k < NS; ++k) {
    double t = 0.0;
#pragma unroll 1
    for (int q = 0; q < NT / 64; ++q) t += sh.s[q][k];
    v[k] = t;
  }
  mx = sh.mx[0];
  var = sh.var[0];
#pragma unroll 1
  for (int q = 1; q < NT / 64; ++q) {
    mx = fmax(mx, sh.mx[q]);
    var = var_merge(var, sh.var[q]);
  }
}

__device__ __forceinline__ double token_distance(float lp_pi, float lp_mu) {
  return fabs(exp((double)lp_pi) - exp((double)lp_mu));
}

// VEC consecutive slots of one thread: 16-byte loads for VEC = 4.
template <int VEC>
struct Slots {
  float a[VEC], b[VEC], hp[VEC], hm[VEC];
  uint8_t m[VEC];
};
template <int VEC>
__device__ __forceinline__ void load_slots(const acrl_reduce_desc& p, int64_t t, bool ent, Slots<VEC>& v) {
  if constexpr (VEC == 4) {
    const float4 a = *reinterpret_cast<const float4*>(p.logp_pi + t);
    const float4 b = *reinterpret_cast<const float4*>(p.logp_mu + t);
    const uchar4 m = *reinterpret_cast<const uchar4*>(p.mask + t);
    v.a[0] = a.x; v.a[1] = a.y; v.a[2] = a.z; v.a[3] = a.w;
    v.b[0] = b.x; v.b[1] = b.y; v.b[2] = b.z; v.b[3] = b.w;
    v.m[0] = m.x; v.m[1] = m.y; v.m[2] = m.z; v.m[3] = m.w;
    if (ent) {
      const float4 hp = p.entropy_pi ? *reinterpret_cast<const float4*>(p.entropy_pi + t) : float4{};
      const float4 hm = p.entropy_mu ? *reinterpret_cast<const float4*>(p.entropy_mu + t) : float4{};
      v.hp[0] = hp.x; v.hp[1] = hp.y; v.hp[2] = hp.z; v.hp[3] = hp.w;
      v.hm[0] = hm.x; v.hm[1] = hm.y; v.hm[2] = hm.z; v.hm[3] = hm.w;
    }
  } else {
    v.a[0] = p.logp_pi[t];
    v.b[0] = p.logp_mu[t];
    v.m[0] = p.mask[t];
    if (ent) {
      v.hp[0] = p.entropy_pi ? p.entropy_pi[t] : 0.0f;
      v.hm[0] = p.entropy_mu ? p.entropy_mu[t] : 0.0f;
    }
  }
}

// One workgroup per response; thread k takes the VEC-slot pieces k, k + 256,
// ... of the response's L slots.  Every slot is loaded (masked ones too: no
// load waits on the mask).  The sums are plain fp64 sums in piece order; the
// squared deviations of each piece (about its own mean) merge into the
// thread's running Var, and the threads' Vars merge in a fixed tree.
template <int VEC>
__global__ __launch_bounds__(kRedThreads) void reduce_seq_kernel(acrl_reduce_desc p, SeqRec* rec,
                                                                 uint32_t* unsorted) {
  __shared__ BlockShared<5> sh;
  const int64_t i = blockIdx.x;
  const int64_t base = i * p.L;
  const bool ent = p.entropy_pi || p.entropy_mu;
  constexpr int kStride = kRedThreads * VEC;
  double n = 0, sd = 0, sl = 0, shp = 0, shm = 0, mx = 0;
  Var var{0.0, 0.0, 0.0};
#pragma unroll 2
  for (int64_t j = (int64_t)threadIdx.x * VEC; j < p.L; j += kStride) {
    Slots<VEC> v;
    load_slots<VEC>(p, base + j, ent, v);
    double dv[VEC];
    float dt[VEC];
    double pn = 0.0, ps = 0.0;
#pragma unroll
    for (int k = 0; k < VEC; ++k) {
      dt[k] = 0.0f;
      dv[k] = 0.0;
      if (v.m[k]) {
        dv[k] = token_distance(v.a[k], v.b[k]);
        n += 1.0;
        sd += dv[k];
        sl += (double)v.a[k] - (double)v.b[k];
        if (ent) {
          shp += v.hp[k];
          shm += v.hm[k];
        }
        mx = fmax(mx, dv[k]);
        dt[k] = (float)dv[k];
        pn += 1.0;
        ps += dv[k];
      }
    }
    if (pn > 0.0) {
      const double pm = ps / pn;
      double pm2 = 0.0;
#pragma unroll
      for (int k = 0; k < VEC; ++k)
        if (v.m[k]) pm2 += (dv[k] - pm) * (dv[k] - pm);
      var = var_merge(var, Var{pn, pm, pm2});
    }
    if (p.d_tok) {
      if constexpr (VEC == 4) *reinterpret_cast<float4*>(p.d_tok + base + j) = make_float4(dt[0], dt[1], dt[2], dt[3]);
      else p.d_tok[base + j] = dt[0];
    }
  }
  double v[5] = {n, sd, sl, shp, shm};
  block_stats<5>(v, mx, var, sh);
  n = v[0];
  sd = v[1];
  sl = v[2];
  shp = v[3];
  shm = v[4];
  if (threadIdx.x == 0) {
    const double mean = n > 0 ? sd / n : 0.0;
    SeqRec r;
    r.n = n; r.sum_d = sd; r.sum_lr = sl; r.sum_hp = shp; r.sum_hm = shm; r.max_d = mx; r.m2 = var.m2;
    r.pad = 0;
    rec[i] = r;
    if (p.seq_len) p.seq_len[i] = (int32_t)n;
    if (p.seq_sum_d) p.seq_sum_d[i] = sd;
    if (p.seq_sum_logratio) p.seq_sum_logratio[i] = sl;
    p.seq_mean_d[i] = (float)mean;
    if (i + 1 < p.B && p.group_of_seq[i] > p.group_of_seq[i + 1]) atomicOr(unsorted, 1u);
  }
}

__global__ void clear_flag_kernel(uint32_t* f) { *f = 0u; }

// Per-group partial record (the groups partition the responses, so the
// batch statistics come from these).
struct GroupRec {
  double n, sum_d, sum_lr, sum_hp, sum_hm, max_d, nseq, mu, m2;
  double pad[7];
};

// One workgroup per group: Y_g over the group's non-empty responses, and the
// group's share of the batch statistics.  When group_of_seq is non-decreasing
// (flag unsorted == 0, set by the per-response kernel) the group's responses are
// the range found by binary search; otherwise every response is scanned.
__global__ __launch_bounds__(kRedThreads) void reduce_group_kernel(acrl_reduce_desc p, const SeqRec* rec,
                                                                   const uint32_t* unsorted, double* gy,
                                                                   double* gcount, GroupRec* grec) {
  __shared__ BlockShared<7> sh;
  __shared__ int64_t range[2];
  const int g = blockIdx.x;
  const bool sorted = *unsorted == 0u;
  int64_t lo = 0, hi = p.B;
  if (sorted) {
    if (threadIdx.x == 0) {
      int64_t a = 0, b = p.B;
      while (a < b) {  // first response with group >= g
        const int64_t m = (a + b) >> 1;
        if (p.group_of_seq[m] < g) a = m + 1;
        else b = m;
      }
      range[0] = a;
      b = p.B;
      while (a < b) {  // first response with group > g
        const int64_t m = (a + b) >> 1;
        if (p.group_of_seq[m] <= g) a = m + 1;
        else b = m;
      }
      range[1] = a;
    }
    __syncthreads();
    lo = range[0];
    hi = range[1];
  }
  double v[7] = {0, 0, 0, 0, 0, 0, 0};  // sum of means, responses, n, sum d, sum log-ratio, sum H_pi, sum H_mu
  double mx = 0.0;
  Var var{0.0, 0.0, 0.0};
  for (int64_t i = lo + threadIdx.x; i < hi; i += kRedThreads) {
    if (sorted || p.group_of_seq[i] == g) {
      const SeqRec r = rec[i];
      if (r.n > 0) {
        const double mean = r.sum_d / r.n;
        v[0] += mean;
        v[1] += 1.0;
        v[2] += r.n;
        v[3] += r.sum_d;
        v[4] += r.sum_lr;
        v[5] += r.sum_hp;
        v[6] += r.sum_hm;
        mx = fmax(mx, r.max_d);
        var = var_merge(var, Var{r.n, mean, r.m2});
      }
    }
  }
  block_stats<7>(v, mx, var, sh);
  if (threadIdx.x == 0) {
    const double c = v[1];
    const double y = c > 0 ? v[0] / c : 0.0;
    gy[g] = y;
    gcount[g] = c;
    p.group_y[g] = (float)y;
    if (p.group_nseq) p.group_nseq[g] = (int32_t)c;
    GroupRec r;
    r.n = v[2]; r.sum_d = v[3]; r.sum_lr = v[4]; r.sum_hp = v[5]; r.sum_hm = v[6]; r.max_d = mx; r.nseq = c;
    r.mu = var.mu; r.m2 = var.m2;
    for (int k = 0; k < 7; ++k) r.pad[k] = 0.0;
    grec[g] = r;
  }
}

// One workgroup of kBatchThreads: batch statistics from the group records.
constexpr int kBatchThreads = 1024;
__global__ __launch_bounds__(kBatchThreads) void reduce_batch_kernel(acrl_reduce_desc p, const GroupRec* grec,
                                                                     const double* gy, const double* gcount) {
  __shared__ BlockShared<8, kBatchThreads> sh;
  double v[8] = {0, 0, 0, 0, 0, 0, 0, 0};  // n, sum d, sum log-ratio, sum H_pi, sum H_mu, responses, sum Y_g, groups
  double mx = 0.0;
  Var var{0.0, 0.0, 0.0};
  for (int64_t g = threadIdx.x; g < p.n_groups; g += kBatchThreads) {
    const GroupRec r = grec[g];
    v[0] += r.n;
    v[1] += r.sum_d;
    v[2] += r.sum_lr;
    v[3] += r.sum_hp;
    v[4] += r.sum_hm;
    v[5] += r.nseq;
    if (gcount[g] > 0) {
      v[6] += gy[g];
      v[7] += 1.0;
    }
    mx = fmax(mx, r.max_d);
    var = var_merge(var, Var{r.n, r.mu, r.m2});
  }
  block_stats<8, kBatchThreads>(v, mx, var, sh);
  if (threadIdx.x == 0) {
    const double n = v[0], ng = v[7];
    double* st = p.stats;
    st[ACRL_STAT_Y_BATCH] = ng > 0 ? v[6] / ng : 0.0;
    st[ACRL_STAT_TOK_MEAN_D] = n > 0 ? v[1] / n : 0.0;
    st[ACRL_STAT_TOK_MAX_D] = mx;
    st[ACRL_STAT_TOK_STD_D] = n > 0 ? sqrt(var.m2 / n) : 0.0;
    st[ACRL_STAT_MEAN_H_PI] = n > 0 ? v[3] / n : 0.0;
    st[ACRL_STAT_MEAN_H_MU] = n > 0 ? v[4] / n : 0.0;
    st[ACRL_STAT_N_TOKENS] = n;
    st[ACRL_STAT_N_GROUPS] = ng;
    st[ACRL_STAT_TOK_MEAN_LOGRATIO] = n > 0 ? v[2] / n : 0.0;
    st[ACRL_STAT_N_SEQS] = v[5];
  }
}


// Element-wise controller.  alpha and the weight are evaluated in fp64 from
// the fp32 inputs (exact conversions), then rounded to fp32 once.  Modes:
// Eq. ACRL, token-level TIS (Eq. tis_objective), sequence-level MIS (Eq.
// mis_objective, from the fp64 per-sequence log-ratio sums of the reduce),
// and the continuous-reduction / fallback-to-GRPO ablations of Sec. 5.
// min(x, C) of an undefined x is undefined: a NaN log-ratio (an invalid
// token id) or a NaN Y (a group id outside [0, n_groups)) gives weight NaN,
// not the clip C.
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
        w_out = isnan(s) ? __builtin_nanf("") : (s <= lnC ? (float)exp(s) : 0.0f);
      } else if (p.mode == ACRL_CTRL_TIS) {
        a_out = 1.0f;
        w_out = isnan(lr) ? __builtin_nanf("") : (float)(lr < lnC ? exp(lr) : C);
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
          const double e = alpha * lr;  // ln rho (NaN if alpha or lr is)
          a_out = (float)alpha;
          w_out = isnan(e) ? __builtin_nanf("") : (float)(e < lnC ? exp(e) : C);
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
  return align_up((size_t)B * sizeof(SeqRec), 256) + 2 * align_up((size_t)n_groups * sizeof(double), 256) +
         align_up((size_t)n_groups * sizeof(GroupRec), 256) + 256;
}

hipError_t launch_reduce(const acrl_reduce_desc& p, hipStream_t s) {
  uint8_t* ws = static_cast<uint8_t*>(p.workspace);
  SeqRec* rec = reinterpret_cast<SeqRec*>(ws);
  size_t off = align_up((size_t)p.B * sizeof(SeqRec), 256);
  double* gy = reinterpret_cast<double*>(ws + off);
  off += align_up((size_t)p.n_groups * sizeof(double), 256);
  double* gc = reinterpret_cast<double*>(ws + off);
  off += align_up((size_t)p.n_groups * sizeof(double), 256);
  GroupRec* grec = reinterpret_cast<GroupRec*>(ws + off);
  off += align_up((size_t)p.n_groups * sizeof(GroupRec), 256);
  uint32_t* unsorted = reinterpret_cast<uint32_t*>(ws + off);
  hipLaunchKernelGGL(clear_flag_kernel, dim3(1), dim3(1), 0, s, unsorted);
  if (p.B > 0) {
    // 16-byte slot loads when every row of slots starts 16-byte aligned
    auto al = [](const void* q, uintptr_t a) { return ((uintptr_t)q & (a - 1)) == 0; };
    const bool vec = p.L % 4 == 0 && al(p.logp_pi, 16) && al(p.logp_mu, 16) && al(p.mask, 4) &&
                     al(p.entropy_pi, 16) && al(p.entropy_mu, 16) && al(p.d_tok, 16);
    if (vec)
      hipLaunchKernelGGL(reduce_seq_kernel<4>, dim3((unsigned)p.B), dim3(kRedThreads), 0, s, p, rec, unsorted);
    else
      hipLaunchKernelGGL(reduce_seq_kernel<1>, dim3((unsigned)p.B), dim3(kRedThreads), 0, s, p, rec, unsorted);
  }
  if (p.n_groups > 0)
    hipLaunchKernelGGL(reduce_group_kernel, dim3((unsigned)p.n_groups), dim3(kRedThreads), 0, s, p,
                       (const SeqRec*)rec, (const uint32_t*)unsorted, gy, gc, grec);
  hipLaunchKernelGGL(reduce_batch_kernel, dim3(1), dim3(kBatchThreads), 0, s, p, (const GroupRec*)grec,
                     (const double*)gy, (const double*)gc);
  return hipGetLastError();
}

// ------------------------------------------------------------------ fixed scratch
// Device memory for acrl_discrepancy_reduce_noalloc: the reduce's per-response
// and per-group records live here instead of in a caller workspace.  Each
// device holds its own copy for the life of the process; host code reaches
// it only through the address hipGetSymbolAddress returns for that device
// (the array's name is a host-side stand-in, not a device address).
static __device__ __align__(256) uint8_t scratch[kReduceScratchBytes];

namespace {
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxScratchDevices];  // device address of `scratch` per device, once looked up
}  // namespace

hipError_t reduce_scratch(void** ptr) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxScratchDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* a = nullptr;
    e = hipGetSymbolAddress(&a, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!a) return hipErrorInvalidSymbol;
    g_scratch_ptr[dev] = a;
  }
  *ptr = g_scratch_ptr[dev];
  return hipSuccess;
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
