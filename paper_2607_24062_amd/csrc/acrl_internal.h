// acrl_internal.h -- shared internals of libacrl (HIP, gfx950 only).
//
// Device helpers used by several kernels (number formats, wavefront
// reductions) and the launcher interface between the host API and the
// kernels.  Not installed; not part of the ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/acrl.h"

namespace acrl {

// ------------------------------------------------------------------ host
// Thread-local message of the last failure; set by the API layer.
void set_error(const char* fmt, ...);

// Launchers: return hipSuccess or the first HIP error.
hipError_t launch_fp8_encode(const float* x, int64_t n, int rounding, uint8_t* q, hipStream_t s);
hipError_t launch_quantize(const uint16_t* x, int64_t rows, int64_t cols, int64_t ld, int scaling,
                           int rounding, uint8_t* q, void* scales, void* workspace, hipStream_t s);

struct ScorePlan {
  int n_ttiles;         // token tiles of 256 rows
  int n_vtiles;         // vocabulary tiles of 256 rows
  int tiles_per_strip;  // vocabulary tiles per workgroup
  int n_strips;         // vocabulary strips (partial softmax states per row)
  int n_tblocks;        // token-tile blocks of kBlockT tiles (grid rasterization)
  int n_sblocks;        // strip blocks of kBlockS strips
  int n_blocks_pad;     // n_tblocks * n_sblocks rounded up to a multiple of 8
  int grid;             // workgroups launched (n_blocks_pad * kBlockT * kBlockS)
  size_t ws_part_offset[2];  // byte offsets of the (M, S, U) partials of pi / mu
  size_t ws_logit_offset[2]; // byte offsets of the sampled-token logits of pi / mu
  size_t ws_pack_offset[4];  // byte offsets of the packed W, H (bf16) and Wq, Hq (e4m3)
  size_t ws_mx_offset[2];    // MX: packed E8M0 scale images of Wq and Hq
  size_t ws_best_offset;     // sampling: the strips' best key, logit and row
  int div_tiles;             // full-vocabulary measures: token tiles per pass (0 = not planned)
  size_t ws_zbuf_offset;     //   mu's logits of one pass
  size_t ws_aq_offset;       //   mu's lse of the pass rows
  size_t ws_dpart_offset;    //   pi's strip sums of the measures
  size_t ws_queue_offset;    // the persistent grid's per-XCD claim counters
  size_t ws_bytes;
};
// div_rows > 0 plans the full-vocabulary measures in passes of div_rows rows;
// prepacked: W's and Wq's images come from the caller (no workspace for them).
ScorePlan plan_score(int64_t n_rows, int64_t d, int64_t V, int64_t div_rows = 0, bool prepacked = false);
constexpr int64_t kDivergenceChunk = 16384;  // default rows per pass of the full-vocabulary measures
// Caller-owned packed LM head (acrl_pack_weights): byte offsets of the W,
// Wq and Wq-MX-scale images.
struct PackedWeightsLayout {
  size_t w_offset, wq_offset, mx_offset, bytes;
};
PackedWeightsLayout packed_weights_layout(int64_t V, int64_t d, int mu_scaling);
hipError_t launch_pack_weights(const void* w, const void* wq, const void* wq_scales, int64_t V, int64_t d,
                               int mu_scaling, void* packed, hipStream_t s);
hipError_t launch_score(const acrl_score_desc& desc, const ScorePlan& plan, hipStream_t s);
hipError_t launch_sample(const acrl_sample_desc& desc, const ScorePlan& plan, hipStream_t s);

// LM-head backward of the surrogate: rows are processed in passes of `chunk`
// tokens; the workspace holds the packed operand images of one pass.
constexpr int64_t kBackwardChunk = 16384;
struct BackwardPlan {
  int64_t chunk;        // rows per pass (a multiple of 256)
  int n_vtiles;         // vocabulary tiles of 256 rows
  int n_dtiles;         // hidden-dimension tiles of 256 rows
  int kch_v;            // 64-byte K chunks of a row whose K runs over the (padded) vocabulary
  size_t off_w, off_wt, off_h, off_ht, off_zt, off_zv;  // image offsets in the workspace
  size_t off_queue;     // the products' per-XCD claim counters (persistent grid)
  size_t ws_bytes;
};
BackwardPlan plan_backward(int64_t n_rows, int64_t d, int64_t V, int64_t chunk);
hipError_t launch_backward(const acrl_backward_desc& desc, const BackwardPlan& plan, hipStream_t s);

size_t surrogate_workspace_bytes(int64_t B, int64_t n_groups);
hipError_t launch_surrogate(const acrl_surrogate_desc& desc, hipStream_t s);

size_t reduce_workspace_bytes(int64_t B, int64_t L, int64_t n_groups);
hipError_t launch_reduce(const acrl_reduce_desc& desc, hipStream_t s);
// Fixed device scratch of the allocation-free reduce (one copy per device):
// its device address on the current device, looked up once per device.
constexpr size_t kReduceScratchBytes = (size_t)ACRL_REDUCE_SCRATCH_BYTES;
constexpr int kMaxScratchDevices = 64;
hipError_t reduce_scratch(void** ptr);
hipError_t launch_controller(const acrl_controller_desc& desc, hipStream_t s);

// ------------------------------------------------------------------ device
#ifdef __HIPCC__

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

__device__ __forceinline__ float bf16_lo(uint32_t packed) { return __uint_as_float(packed << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t packed) { return __uint_as_float(packed & 0xFFFF0000u); }

// Encode fp32 -> OCP E4M3 with nearest-even rounding, saturating at +-448,
// NaN -> 0x7F | sign.  The gfx950 converter rounds to nearest-even; the
// clamp supplies the saturation and the NaN test keeps the sign of a NaN.
__device__ __forceinline__ uint32_t e4m3_pack4_rne(float a, float b, float c, float d) {
  const float lo = -448.0f, hi = 448.0f;
  uint32_t r = __builtin_amdgcn_cvt_pk_fp8_f32(fminf(fmaxf(a, lo), hi), fminf(fmaxf(b, lo), hi), 0, false);
  r = __builtin_amdgcn_cvt_pk_fp8_f32(fminf(fmaxf(c, lo), hi), fminf(fmaxf(d, lo), hi), r, true);
  // NaN inputs: the clamp turned them into +-448; restore the NaN code.
  const float v[4] = {a, b, c, d};
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    if (v[k] != v[k]) {
      const uint32_t code = ((__float_as_uint(v[k]) >> 24) & 0x80u) | 0x7Fu;
      r = (r & ~(0xFFu << (8 * k))) | (code << (8 * k));
    }
  }
  return r;
}

// Encode fp32 -> OCP E4M3 truncating the magnitude (toward zero); +-448
// saturation and NaN handling as above.  Pure integer work on the fp32 bits.
__device__ __forceinline__ uint32_t e4m3_rtz(float x) {
  const uint32_t u = __float_as_uint(x);
  const uint32_t s = (u >> 24) & 0x80u;
  const uint32_t a = u & 0x7FFFFFFFu;
  if (a > 0x7F800000u) return s | 0x7Fu;              // NaN
  if (a >= 0x43E00000u) return s | 0x7Eu;             // |x| >= 448 (and inf)
  if (a < 0x3C800000u) {                              // |x| < 2^-6: subnormal codes
    const float m = truncf(__uint_as_float(a) * 512.0f);  // exact scaling by 2^9
    return s | (uint32_t)m;
  }
  return s | ((((a >> 23) - 120u) << 3) | ((a >> 20) & 7u));
}

__device__ __forceinline__ uint32_t e4m3_pack4_rtz(float a, float b, float c, float d) {
  return e4m3_rtz(a) | (e4m3_rtz(b) << 8) | (e4m3_rtz(c) << 16) | (e4m3_rtz(d) << 24);
}

template <int ROUND>
__device__ __forceinline__ uint32_t e4m3_pack4(float a, float b, float c, float d) {
  if constexpr (ROUND == ACRL_ROUND_TOWARD_ZERO) return e4m3_pack4_rtz(a, b, c, d);
  else return e4m3_pack4_rne(a, b, c, d);
}

// --- wavefront reductions (64 lanes): DPP inside each 16-lane row, then
// cross-row lane exchanges.
template <int CTRL>
__device__ __forceinline__ float dpp_f32(float v) {
  return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), CTRL, 0xF, 0xF, true));
}

__device__ __forceinline__ float wave_max(float v) {
  v = fmaxf(v, dpp_f32<0xB1>(v));   // quad_perm [1,0,3,2]: lane ^ 1
  v = fmaxf(v, dpp_f32<0x4E>(v));   // quad_perm [2,3,0,1]: lane ^ 2
  v = fmaxf(v, dpp_f32<0x124>(v));  // row_ror:4
  v = fmaxf(v, dpp_f32<0x128>(v));  // row_ror:8
  v = fmaxf(v, __shfl_xor(v, 16));
  v = fmaxf(v, __shfl_xor(v, 32));
  return v;
}

__device__ __forceinline__ double wave_sum(double v) {
#pragma unroll
  for (int m = 1; m < 64; m <<= 1) v += __shfl_xor(v, m);
  return v;
}

#endif  // __HIPCC__

}  // namespace acrl
