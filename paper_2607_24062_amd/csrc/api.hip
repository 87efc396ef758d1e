// api.hip -- the extern "C" entry points of libacrl: argument validation on
// the host, device capability check, workspace sizing, kernel dispatch.
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <mutex>

#include "acrl_internal.h"

namespace acrl {

static thread_local char g_last_error[512] = "";

void set_error(const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_last_error, sizeof g_last_error, fmt, ap);
  va_end(ap);
}

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_dev_mu;
int g_dev_state[kMaxDevices];  // 0 unknown, 1 gfx950, 2 other

acrl_status check_device() {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) {
    set_error("hipGetDevice failed: %s", hipGetErrorString(e));
    return ACRL_ERR_HIP;
  }
  if (dev < 0 || dev >= kMaxDevices) {
    set_error("device index %d out of range", dev);
    return ACRL_ERR_UNSUPPORTED;
  }
  std::lock_guard<std::mutex> lk(g_dev_mu);
  if (g_dev_state[dev] == 0) {
    hipDeviceProp_t prop;
    e = hipGetDeviceProperties(&prop, dev);
    if (e != hipSuccess) {
      set_error("hipGetDeviceProperties failed: %s", hipGetErrorString(e));
      return ACRL_ERR_HIP;
    }
    g_dev_state[dev] = strncmp(prop.gcnArchName, "gfx950", 6) == 0 ? 1 : 2;
    if (g_dev_state[dev] == 2) set_error("device %d is %s; libacrl supports gfx950 only", dev, prop.gcnArchName);
  }
  if (g_dev_state[dev] != 1) {
    set_error("device %d is not gfx950; libacrl supports gfx950 only", dev);
    return ACRL_ERR_UNSUPPORTED;
  }
  return ACRL_OK;
}

acrl_status hip_status(hipError_t e, const char* what) {
  if (e == hipSuccess) return ACRL_OK;
  set_error("%s: %s", what, hipGetErrorString(e));
  return ACRL_ERR_HIP;
}

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

#define ACRL_REQUIRE(cond, ...)       \
  do {                                \
    if (!(cond)) {                    \
      acrl::set_error(__VA_ARGS__);   \
      return ACRL_ERR_INVALID_ARG;    \
    }                                 \
  } while (0)

size_t quantize_ws(int scaling) { return scaling == ACRL_SCALE_PER_TENSOR ? 256 : 0; }

// The packed operand images are addressed in 16-byte units with 32-bit
// indices: (rows rounded up to 256) * 2d / 16 must stay below 2^32.
bool score_size_ok(int64_t rows, int64_t d) {
  const int64_t padded = (rows + 255) / 256 * 256;
  return padded * (d / 8) < ((int64_t)1 << 32);
}

acrl_status validate_score(const acrl_score_desc* d) {
  ACRL_REQUIRE(d, "desc is NULL");
  ACRL_REQUIRE(d->n_rows >= 0 && d->n_rows < (int64_t)INT32_MAX - 512, "n_rows %lld out of range",
               (long long)d->n_rows);
  ACRL_REQUIRE(d->d > 0 && d->d % 128 == 0, "d = %lld must be a positive multiple of 128",
               (long long)d->d);
  ACRL_REQUIRE(d->V > 0 && d->V < (int64_t)INT32_MAX - 512, "V = %lld out of range", (long long)d->V);
  ACRL_REQUIRE(score_size_ok(d->V, d->d) && score_size_ok(d->n_rows, d->d),
               "rows x d too large (rows rounded up to 256, times d/8, must be below 2^32)");
  ACRL_REQUIRE(d->mu_scaling == ACRL_SCALE_PER_TENSOR || d->mu_scaling == ACRL_SCALE_PER_ROW ||
                   d->mu_scaling == ACRL_SCALE_MX32,
               "mu_scaling %d unknown", d->mu_scaling);
  ACRL_REQUIRE(d->inv_temperature > 0.0f && d->inv_temperature < 1e30f,
               "inv_temperature must be positive and finite");
  ACRL_REQUIRE(d->policies == ACRL_POLICY_BOTH || d->policies == ACRL_POLICY_PI || d->policies == ACRL_POLICY_MU,
               "policies %d unknown", d->policies);
  const bool pi = d->policies != ACRL_POLICY_MU, mu = d->policies != ACRL_POLICY_PI;
  const bool div = d->kl_pi_mu || d->kl_mu_pi || d->l2;
  ACRL_REQUIRE(!div || (pi && mu), "the full-vocabulary measures need both policies");
  if (d->packed_weights) {
    const size_t need = packed_weights_layout(d->V, d->d, d->mu_scaling).bytes;
    ACRL_REQUIRE(d->packed_weights_bytes >= need, "packed_weights has %zu bytes, needs %zu",
                 d->packed_weights_bytes, need);
    ACRL_REQUIRE(aligned16(d->packed_weights), "packed_weights must be 16-byte aligned");
  }
  if (pi && !d->packed_weights) {
    ACRL_REQUIRE(d->w, "w is required");
    ACRL_REQUIRE(aligned16(d->w), "w must be 16-byte aligned");
  }
  if (mu) {
    ACRL_REQUIRE(d->wq_scales && (d->wq || d->packed_weights), "wq and wq_scales are required");
    ACRL_REQUIRE(aligned16(d->wq) && aligned16(d->wq_scales), "wq, wq_scales must be 16-byte aligned");
  }
  if (d->n_rows > 0) {
    ACRL_REQUIRE(d->token_ids, "token_ids is required");
    if (pi) {
      ACRL_REQUIRE(d->h && d->logp_pi, "h and logp_pi are required");
      ACRL_REQUIRE(aligned16(d->h), "h must be 16-byte aligned");
    }
    if (mu) {
      ACRL_REQUIRE(d->hq && d->hq_scales && d->logp_mu, "hq, hq_scales and logp_mu are required");
      ACRL_REQUIRE(aligned16(d->hq) && aligned16(d->hq_scales), "hq, hq_scales must be 16-byte aligned");
    }
  }
  return ACRL_OK;
}

// rows per pass of the full-vocabulary measures (0: not asked for)
int64_t div_rows_of(const acrl_score_desc* d) {
  const bool div = d->kl_pi_mu || d->kl_mu_pi || d->l2;
  return div ? (d->div_chunk > 0 ? d->div_chunk : kDivergenceChunk) : 0;
}

acrl_status validate_reduce(const acrl_reduce_desc* d) {
  ACRL_REQUIRE(d, "desc is NULL");
  ACRL_REQUIRE(d->B >= 0 && d->L >= 0 && d->n_groups >= 0, "B, L, n_groups must be >= 0");
  ACRL_REQUIRE(d->B < (int64_t)INT32_MAX && d->n_groups < (int64_t)INT32_MAX, "B or n_groups too large");
  ACRL_REQUIRE(d->stats, "stats is required");
  if (d->B > 0) {
    ACRL_REQUIRE(d->seq_mean_d && d->group_of_seq, "seq_mean_d and group_of_seq are required");
    ACRL_REQUIRE(d->n_groups > 0, "n_groups must be > 0 when B > 0");
    if (d->L > 0)
      ACRL_REQUIRE(d->logp_pi && d->logp_mu && d->mask, "logp_pi, logp_mu and mask are required");
  }
  if (d->n_groups > 0) ACRL_REQUIRE(d->group_y, "group_y is required");
  return ACRL_OK;
}

}  // namespace
}  // namespace acrl

using acrl::set_error;

extern "C" {

const char* acrl_status_string(acrl_status status) {
  switch (status) {
    case ACRL_OK: return "ok";
    case ACRL_ERR_INVALID_ARG: return "invalid argument";
    case ACRL_ERR_UNSUPPORTED: return "unsupported";
    case ACRL_ERR_WORKSPACE: return "workspace too small";
    case ACRL_ERR_HIP: return "HIP runtime error";
    default: return "unknown status";
  }
}

const char* acrl_last_error(void) { return acrl::g_last_error; }

int acrl_abi_version(void) { return ACRL_ABI_VERSION; }

void acrl_abi_struct_sizes(size_t* score_desc, size_t* reduce_desc, size_t* controller_desc,
                           size_t* sample_desc, size_t* surrogate_desc, size_t* backward_desc) {
  if (score_desc) *score_desc = sizeof(acrl_score_desc);
  if (reduce_desc) *reduce_desc = sizeof(acrl_reduce_desc);
  if (controller_desc) *controller_desc = sizeof(acrl_controller_desc);
  if (sample_desc) *sample_desc = sizeof(acrl_sample_desc);
  if (surrogate_desc) *surrogate_desc = sizeof(acrl_surrogate_desc);
  if (backward_desc) *backward_desc = sizeof(acrl_backward_desc);
}

acrl_status acrl_quantize_workspace_size(int64_t rows, int64_t cols, int scaling, size_t* bytes) {
  ACRL_REQUIRE(bytes, "bytes is NULL");
  ACRL_REQUIRE(rows >= 0 && cols > 0, "rows must be >= 0 and cols > 0");
  ACRL_REQUIRE(scaling >= ACRL_SCALE_PER_TENSOR && scaling <= ACRL_SCALE_MX32, "scaling %d unknown", scaling);
  *bytes = acrl::quantize_ws(scaling);
  return ACRL_OK;
}

acrl_status acrl_quantize_fp8(const void* x, int64_t rows, int64_t cols, int64_t ld, int scaling,
                              int rounding, void* q, void* scales, void* workspace,
                              size_t workspace_bytes, void* stream) {
  ACRL_REQUIRE(rows >= 0, "rows = %lld must be >= 0", (long long)rows);
  ACRL_REQUIRE(cols > 0 && cols % 32 == 0, "cols = %lld must be a positive multiple of 32", (long long)cols);
  ACRL_REQUIRE(ld >= cols && ld % 8 == 0, "ld = %lld must be >= cols and a multiple of 8", (long long)ld);
  ACRL_REQUIRE(scaling >= ACRL_SCALE_PER_TENSOR && scaling <= ACRL_SCALE_MX32, "scaling %d unknown", scaling);
  ACRL_REQUIRE(rounding == ACRL_ROUND_NEAREST_EVEN || rounding == ACRL_ROUND_TOWARD_ZERO,
               "rounding %d unknown", rounding);
  ACRL_REQUIRE(scales, "scales is NULL");
  if (rows > 0) {
    ACRL_REQUIRE(x && q, "x and q are required");
    ACRL_REQUIRE(acrl::aligned16(x) && acrl::aligned16(q), "x and q must be 16-byte aligned");
  }
  ACRL_REQUIRE(rows * (cols / 32) < ((int64_t)1 << 40), "tensor too large");
  const size_t need = acrl::quantize_ws(scaling);
  if (need > 0 && (!workspace || workspace_bytes < need)) {
    set_error("per-tensor quantization needs %zu workspace bytes, got %zu", need, workspace_bytes);
    return ACRL_ERR_WORKSPACE;
  }
  acrl_status st = acrl::check_device();
  if (st != ACRL_OK) return st;
  return acrl::hip_status(acrl::launch_quantize(static_cast<const uint16_t*>(x), rows, cols, ld,
                                                scaling, rounding, static_cast<uint8_t*>(q),
                                                scales, workspace, (hipStream_t)stream),
                          "acrl_quantize_fp8 launch");
}

acrl_status acrl_fp8_encode(const float* x, int64_t n, int rounding, void* q, void* stream) {
  ACRL_REQUIRE(n >= 0, "n must be >= 0");
  ACRL_REQUIRE(rounding == ACRL_ROUND_NEAREST_EVEN || rounding == ACRL_ROUND_TOWARD_ZERO,
               "rounding %d unknown", rounding);
  if (n > 0) {
    ACRL_REQUIRE(x && q, "x and q are required");
    ACRL_REQUIRE(acrl::aligned16(x) && acrl::aligned16(q), "x and q must be 16-byte aligned");
  }
  acrl_status st = acrl::check_device();
  if (st != ACRL_OK) return st;
  return acrl::hip_status(
      acrl::launch_fp8_encode(x, n, rounding, static_cast<uint8_t*>(q), (hipStream_t)stream),
      "acrl_fp8_encode launch");
}

acrl_status acrl_score_workspace_size(int64_t n_rows, int64_t d, int64_t V, int mu_scaling, size_t* bytes) {
  ACRL_REQUIRE(bytes, "bytes is NULL");
  ACRL_REQUIRE(n_rows >= 0 && n_rows < (int64_t)INT32_MAX - 512, "n_rows out of range");
  ACRL_REQUIRE(d > 0 && d % 128 == 0, "d must be a positive multiple of 128");
  ACRL_REQUIRE(V > 0 && V < (int64_t)INT32_MAX - 512, "V out of range");
  ACRL_REQUIRE(mu_scaling >= ACRL_SCALE_PER_TENSOR && mu_scaling <= ACRL_SCALE_MX32, "mu_scaling unknown");
  ACRL_REQUIRE(acrl::score_size_ok(V, d) && acrl::score_size_ok(n_rows, d), "rows x d too large");
  *bytes = acrl::plan_score(n_rows, d, V).ws_bytes;
  return ACRL_OK;
}

acrl_status acrl_score_div_workspace_size(int64_t n_rows, int64_t d, int64_t V, int mu_scaling, int64_t div_chunk,
                                          size_t* bytes) {
  acrl_status st = acrl_score_workspace_size(n_rows, d, V, mu_scaling, bytes);
  if (st != ACRL_OK) return st;
  ACRL_REQUIRE(div_chunk >= 0 && div_chunk <= ((int64_t)1 << 24), "div_chunk must lie in [0, 2^24]");
  *bytes = acrl::plan_score(n_rows, d, V, div_chunk > 0 ? div_chunk : acrl::kDivergenceChunk).ws_bytes;
  return ACRL_OK;
}

acrl_status acrl_score_workspace_query(const acrl_score_desc* desc, size_t* bytes) {
  ACRL_REQUIRE(desc && bytes, "desc and bytes are required");
  acrl_status st = acrl_score_workspace_size(desc->n_rows, desc->d, desc->V, desc->mu_scaling, bytes);
  if (st != ACRL_OK) return st;
  ACRL_REQUIRE(desc->div_chunk >= 0 && desc->div_chunk <= ((int64_t)1 << 24), "div_chunk must lie in [0, 2^24]");
  *bytes = acrl::plan_score(desc->n_rows, desc->d, desc->V, acrl::div_rows_of(desc), desc->packed_weights != nullptr)
               .ws_bytes;
  return ACRL_OK;
}

acrl_status acrl_packed_weights_size(int64_t V, int64_t d, int mu_scaling, size_t* bytes) {
  ACRL_REQUIRE(bytes, "bytes is NULL");
  ACRL_REQUIRE(d > 0 && d % 128 == 0, "d must be a positive multiple of 128");
  ACRL_REQUIRE(V > 0 && V < (int64_t)INT32_MAX - 512, "V out of range");
  ACRL_REQUIRE(mu_scaling >= ACRL_SCALE_PER_TENSOR && mu_scaling <= ACRL_SCALE_MX32, "mu_scaling unknown");
  ACRL_REQUIRE(acrl::score_size_ok(V, d), "V x d too large");
  *bytes = acrl::packed_weights_layout(V, d, mu_scaling).bytes;
  return ACRL_OK;
}

acrl_status acrl_pack_weights(const void* w, const void* wq, const void* wq_scales, int64_t V, int64_t d,
                              int mu_scaling, void* packed, size_t packed_bytes, void* stream) {
  size_t need = 0;
  acrl_status st = acrl_packed_weights_size(V, d, mu_scaling, &need);
  if (st != ACRL_OK) return st;
  ACRL_REQUIRE(w && wq && wq_scales && packed, "w, wq, wq_scales and packed are required");
  ACRL_REQUIRE(acrl::aligned16(w) && acrl::aligned16(wq) && acrl::aligned16(wq_scales) && acrl::aligned16(packed),
               "w, wq, wq_scales and packed must be 16-byte aligned");
  if (packed_bytes < need) {
    set_error("acrl_pack_weights needs %zu bytes, got %zu", need, packed_bytes);
    return ACRL_ERR_WORKSPACE;
  }
  st = acrl::check_device();
  if (st != ACRL_OK) return st;
  return acrl::hip_status(acrl::launch_pack_weights(w, wq, wq_scales, V, d, mu_scaling, packed, (hipStream_t)stream),
                          "acrl_pack_weights launch");
}

acrl_status acrl_score_pi_mu(const acrl_score_desc* desc, void* stream) {
  acrl_status st = acrl::validate_score(desc);
  if (st != ACRL_OK) return st;
  ACRL_REQUIRE(desc->div_chunk >= 0 && desc->div_chunk <= ((int64_t)1 << 24), "div_chunk must lie in [0, 2^24]");
  const acrl::ScorePlan plan = acrl::plan_score(desc->n_rows, desc->d, desc->V, acrl::div_rows_of(desc),
                                                desc->packed_weights != nullptr);
  if (desc->n_rows > 0 && (!desc->workspace || desc->workspace_bytes < plan.ws_bytes)) {
    set_error("acrl_score_pi_mu needs %zu workspace bytes, got %zu", plan.ws_bytes, desc->workspace_bytes);
    return ACRL_ERR_WORKSPACE;
  }
  if (desc->n_rows > 0 && !acrl::aligned16(desc->workspace)) {
    set_error("workspace must be 16-byte aligned");
    return ACRL_ERR_INVALID_ARG;
  }
  st = acrl::check_device();
  if (st != ACRL_OK) return st;
  return acrl::hip_status(acrl::launch_score(*desc, plan, (hipStream_t)stream), "acrl_score_pi_mu launch");
}

acrl_status acrl_sample_mu(const acrl_sample_desc* d, void* stream) {
  ACRL_REQUIRE(d, "desc is NULL");
  ACRL_REQUIRE(d->n_rows >= 0 && d->n_rows < (int64_t)INT32_MAX - 512, "n_rows %lld out of range",
               (long long)d->n_rows);
  ACRL_REQUIRE(d->d > 0 && d->d % 128 == 0, "d = %lld must be a positive multiple of 128", (long long)d->d);
  ACRL_REQUIRE(d->V > 0 && d->V < (int64_t)INT32_MAX - 512, "V = %lld out of range", (long long)d->V);
  ACRL_REQUIRE(acrl::score_size_ok(d->V, d->d) && acrl::score_size_ok(d->n_rows, d->d), "rows x d too large");
  ACRL_REQUIRE(d->mu_scaling == ACRL_SCALE_PER_TENSOR || d->mu_scaling == ACRL_SCALE_PER_ROW ||
                   d->mu_scaling == ACRL_SCALE_MX32,
               "mu_scaling %d unknown", d->mu_scaling);
  ACRL_REQUIRE(d->inv_temperature > 0.0f && d->inv_temperature < 1e30f,
               "inv_temperature must be positive and finite");
  ACRL_REQUIRE(d->row_offset >= 0 && d->row_offset + d->n_rows <= ((int64_t)1 << 32),
               "row_offset + n_rows must lie in [0, 2^32] (the generator's token counter)");
  ACRL_REQUIRE(d->wq_scales && (d->wq || d->packed_weights), "wq and wq_scales are required");
  ACRL_REQUIRE(acrl::aligned16(d->wq) && acrl::aligned16(d->wq_scales), "wq and wq_scales must be 16-byte aligned");
  if (d->packed_weights) {
    const size_t need = acrl::packed_weights_layout(d->V, d->d, d->mu_scaling).bytes;
    ACRL_REQUIRE(d->packed_weights_bytes >= need, "packed_weights has %zu bytes, needs %zu",
                 d->packed_weights_bytes, need);
    ACRL_REQUIRE(acrl::aligned16(d->packed_weights), "packed_weights must be 16-byte aligned");
  }
  if (d->n_rows > 0) {
    ACRL_REQUIRE(d->hq && d->hq_scales && d->ids, "hq, hq_scales and ids are required");
    ACRL_REQUIRE(acrl::aligned16(d->hq) && acrl::aligned16(d->hq_scales), "hq and hq_scales must be 16-byte aligned");
  }
  const acrl::ScorePlan plan = acrl::plan_score(d->n_rows, d->d, d->V, 0, d->packed_weights != nullptr);
  if (d->n_rows > 0 && (!d->workspace || d->workspace_bytes < plan.ws_bytes)) {
    set_error("acrl_sample_mu needs %zu workspace bytes, got %zu", plan.ws_bytes, d->workspace_bytes);
    return ACRL_ERR_WORKSPACE;
  }
  if (d->n_rows > 0 && !acrl::aligned16(d->workspace)) {
    set_error("workspace must be 16-byte aligned");
    return ACRL_ERR_INVALID_ARG;
  }
  acrl_status st = acrl::check_device();
  if (st != ACRL_OK) return st;
  return acrl::hip_status(acrl::launch_sample(*d, plan, (hipStream_t)stream), "acrl_sample_mu launch");
}

acrl_status acrl_reduce_workspace_size(int64_t B, int64_t L, int64_t n_groups, size_t* bytes) {
  ACRL_REQUIRE(bytes, "bytes is NULL");
  ACRL_REQUIRE(B >= 0 && L >= 0 && n_groups >= 0, "B, L, n_groups must be >= 0");
  *bytes = acrl::reduce_workspace_bytes(B, L, n_groups);
  return ACRL_OK;
}

acrl_status acrl_discrepancy_reduce(const acrl_reduce_desc* desc, void* stream) {
  acrl_status st = acrl::validate_reduce(desc);
  if (st != ACRL_OK) return st;
  const size_t need = acrl::reduce_workspace_bytes(desc->B, desc->L, desc->n_groups);
  if (!desc->workspace || desc->workspace_bytes < need) {
    set_error("acrl_discrepancy_reduce needs %zu workspace bytes, got %zu", need, desc->workspace_bytes);
    return ACRL_ERR_WORKSPACE;
  }
  st = acrl::check_device();
  if (st != ACRL_OK) return st;
  return acrl::hip_status(acrl::launch_reduce(*desc, (hipStream_t)stream), "acrl_discrepancy_reduce launch");
}

acrl_status acrl_discrepancy_reduce_noalloc(const acrl_reduce_desc* desc, void* stream) {
  acrl_status st = acrl::validate_reduce(desc);
  if (st != ACRL_OK) return st;
  const size_t need = acrl::reduce_workspace_bytes(desc->B, desc->L, desc->n_groups);
  if (need > acrl::kReduceScratchBytes) {
    set_error("acrl_discrepancy_reduce_noalloc: B = %lld, n_groups = %lld need %zu scratch bytes, above the "
              "fixed %zu (use acrl_discrepancy_reduce with a workspace)",
              (long long)desc->B, (long long)desc->n_groups, need, acrl::kReduceScratchBytes);
    return ACRL_ERR_WORKSPACE;
  }
  st = acrl::check_device();
  if (st != ACRL_OK) return st;
  void* scratch = nullptr;
  st = acrl::hip_status(acrl::reduce_scratch(&scratch), "acrl_discrepancy_reduce_noalloc scratch lookup");
  if (st != ACRL_OK) return st;
  acrl_reduce_desc d = *desc;
  d.workspace = scratch;
  d.workspace_bytes = acrl::kReduceScratchBytes;
  return acrl::hip_status(acrl::launch_reduce(d, (hipStream_t)stream), "acrl_discrepancy_reduce_noalloc launch");
}

acrl_status acrl_controller_step(const acrl_controller_desc* d, void* stream) {
  ACRL_REQUIRE(d, "desc is NULL");
  ACRL_REQUIRE(d->B >= 0 && d->L >= 0 && d->n_groups >= 0, "B, L and n_groups must be >= 0");
  ACRL_REQUIRE(d->X > 0.0f && d->X < 1e30f, "X must be > 0 (got %g)", (double)d->X);
  ACRL_REQUIRE(d->gamma > 0.0f && d->gamma < 1e30f, "gamma must be > 0 (got %g)", (double)d->gamma);
  ACRL_REQUIRE(d->C > 1.0f && d->C < 1e30f, "C must be > 1 (got %g)", (double)d->C);
  ACRL_REQUIRE(d->y_level == ACRL_Y_GROUP || d->y_level == ACRL_Y_SEQUENCE || d->y_level == ACRL_Y_BATCH,
               "y_level %d unknown", d->y_level);
  ACRL_REQUIRE(d->mode >= ACRL_CTRL_ACRL && d->mode <= ACRL_CTRL_FALLBACK, "mode %d unknown", d->mode);
  if (d->mode == ACRL_CTRL_CONTINUOUS)
    ACRL_REQUIRE(d->k > 0.0f && d->k < 1e30f, "k must be > 0 (got %g)", (double)d->k);
  if (d->B > 0 && d->L > 0) {
    ACRL_REQUIRE(d->mask && d->logp_pi && d->logp_mu && d->adv && d->weight,
                 "mask, logp_pi, logp_mu, adv and weight are required");
    const bool reads_y = d->mode == ACRL_CTRL_ACRL || d->mode == ACRL_CTRL_FALLBACK;
    if (reads_y && d->y_level == ACRL_Y_GROUP)
      ACRL_REQUIRE(d->group_y && d->group_of_seq, "group_y and group_of_seq are required");
    if (reads_y && d->y_level == ACRL_Y_SEQUENCE) ACRL_REQUIRE(d->seq_mean_d, "seq_mean_d is required");
    if (reads_y && d->y_level == ACRL_Y_BATCH) ACRL_REQUIRE(d->stats, "stats is required");
    if (d->mode == ACRL_CTRL_MIS) ACRL_REQUIRE(d->seq_sum_logratio, "seq_sum_logratio is required for MIS");
  }
  acrl_status st = acrl::check_device();
  if (st != ACRL_OK) return st;
  return acrl::hip_status(acrl::launch_controller(*d, (hipStream_t)stream), "acrl_controller_step launch");
}

acrl_status acrl_surrogate_workspace_size(int64_t B, int64_t n_groups, size_t* bytes) {
  ACRL_REQUIRE(bytes, "bytes is NULL");
  ACRL_REQUIRE(B >= 0 && n_groups >= 0, "B and n_groups must be >= 0");
  *bytes = acrl::surrogate_workspace_bytes(B, n_groups);
  return ACRL_OK;
}

acrl_status acrl_surrogate(const acrl_surrogate_desc* d, void* stream) {
  ACRL_REQUIRE(d, "desc is NULL");
  ACRL_REQUIRE(d->B >= 0 && d->L >= 0 && d->n_groups >= 0, "B, L and n_groups must be >= 0");
  ACRL_REQUIRE(d->B < (int64_t)INT32_MAX && d->n_groups < (int64_t)INT32_MAX, "B or n_groups too large");
  ACRL_REQUIRE(d->B == 0 || d->n_groups > 0, "n_groups must be > 0 when B > 0");
  ACRL_REQUIRE(d->eps_low >= 0.0f && d->eps_low < 1.0f, "eps_low must lie in [0, 1) (got %g)", (double)d->eps_low);
  ACRL_REQUIRE(d->eps_high >= 0.0f && d->eps_high < 1e30f, "eps_high must be >= 0 (got %g)", (double)d->eps_high);
  ACRL_REQUIRE(d->loss, "loss is required");
  if (d->B > 0) ACRL_REQUIRE(d->group_of_seq, "group_of_seq is required");
  if (d->B > 0 && d->L > 0)
    ACRL_REQUIRE(d->mask && d->logp_new && d->logp_old && d->adv && d->coef,
                 "mask, logp_new, logp_old, adv and coef are required");
  const size_t need = acrl::surrogate_workspace_bytes(d->B, d->n_groups);
  if (!d->workspace || d->workspace_bytes < need) {
    set_error("acrl_surrogate needs %zu workspace bytes, got %zu", need, d->workspace_bytes);
    return ACRL_ERR_WORKSPACE;
  }
  acrl_status st = acrl::check_device();
  if (st != ACRL_OK) return st;
  return acrl::hip_status(acrl::launch_surrogate(*d, (hipStream_t)stream), "acrl_surrogate launch");
}

static acrl_status validate_backward_sizes(int64_t n_rows, int64_t d, int64_t V, int64_t chunk) {
  ACRL_REQUIRE(n_rows >= 0 && n_rows < (int64_t)INT32_MAX - 512, "n_rows %lld out of range", (long long)n_rows);
  ACRL_REQUIRE(d > 0 && d % 128 == 0, "d = %lld must be a positive multiple of 128", (long long)d);
  ACRL_REQUIRE(V > 0 && V < ((int64_t)1 << 23), "V = %lld must lie in (0, 2^23)", (long long)V);
  ACRL_REQUIRE(acrl::score_size_ok(V, d), "V x d too large (V rounded up to 256, times d/8, must be below 2^32)");
  ACRL_REQUIRE(chunk >= 0 && chunk <= ((int64_t)1 << 23), "token_chunk must lie in [0, 2^23]");
  const int64_t c = acrl::plan_backward(n_rows, d, V, chunk).chunk;
  ACRL_REQUIRE(acrl::score_size_ok(c, d), "token_chunk x d too large");
  return ACRL_OK;
}

acrl_status acrl_backward_workspace_size(int64_t n_rows, int64_t d, int64_t V, int64_t token_chunk, size_t* bytes) {
  ACRL_REQUIRE(bytes, "bytes is NULL");
  acrl_status st = validate_backward_sizes(n_rows, d, V, token_chunk);
  if (st != ACRL_OK) return st;
  *bytes = acrl::plan_backward(n_rows, d, V, token_chunk).ws_bytes;
  return ACRL_OK;
}

acrl_status acrl_lm_head_backward(const acrl_backward_desc* d, void* stream) {
  ACRL_REQUIRE(d, "desc is NULL");
  acrl_status st = validate_backward_sizes(d->n_rows, d->d, d->V, d->token_chunk);
  if (st != ACRL_OK) return st;
  ACRL_REQUIRE(d->inv_temperature > 0.0f && d->inv_temperature < 1e30f,
               "inv_temperature must be positive and finite");
  ACRL_REQUIRE(d->dh || d->dw, "at least one of dh and dw is required");
  if (d->dw || d->n_rows > 0) {
    ACRL_REQUIRE(d->w, "w is required");
    ACRL_REQUIRE(acrl::aligned16(d->w), "w must be 16-byte aligned");
  }
  if (d->n_rows > 0) {
    ACRL_REQUIRE(d->h && d->token_ids && d->coef && d->lse, "h, token_ids, coef and lse are required");
    ACRL_REQUIRE(acrl::aligned16(d->h), "h must be 16-byte aligned");
  }
  const acrl::BackwardPlan plan = acrl::plan_backward(d->n_rows, d->d, d->V, d->token_chunk);
  if (d->n_rows > 0 && (!d->workspace || d->workspace_bytes < plan.ws_bytes)) {
    set_error("acrl_lm_head_backward needs %zu workspace bytes, got %zu", plan.ws_bytes, d->workspace_bytes);
    return ACRL_ERR_WORKSPACE;
  }
  if (d->n_rows > 0 && !acrl::aligned16(d->workspace)) {
    set_error("workspace must be 16-byte aligned");
    return ACRL_ERR_INVALID_ARG;
  }
  st = acrl::check_device();
  if (st != ACRL_OK) return st;
  return acrl::hip_status(acrl::launch_backward(*d, plan, (hipStream_t)stream), "acrl_lm_head_backward launch");
}

acrl_status acrl_reference_from_groups(const float* group_y, const int32_t* group_nseq, int64_t n_groups,
                                       float* X_out) {
  ACRL_REQUIRE(group_y && group_nseq && X_out && n_groups >= 0, "null argument or negative n_groups");
  double s = 0.0;
  int64_t n = 0;
  for (int64_t g = 0; g < n_groups; ++g)
    if (group_nseq[g] > 0) {
      s += group_y[g];
      ++n;
    }
  ACRL_REQUIRE(n > 0, "no non-empty group");
  *X_out = (float)(s / (double)n);
  return ACRL_OK;
}

}  // extern "C"
