// quantize.hip -- FP8 (OCP E4M3) quantization of bf16 matrices for the
// inference policy mu: per-tensor, per-row (per-token activations /
// per-channel weights, Sec. 5.1 of the ACRL paper) and MX32 (one E8M0 scale
// per 32 consecutive elements, the MXFP8 of Sec. 5.2).
//
// All three are HBM-bound streams: 2 bytes in and 1 byte out per element
// (per-tensor reads the tensor twice: amax pass, then encode).  Loads are
// 16-byte vectors, one wavefront per row for the row kernels, so each
// wave-instruction touches 1 KiB of contiguous memory.
#include "acrl_internal.h"

namespace acrl {
namespace {

// Group scale s = amax / 448 (fp32, correctly rounded); 1 for an all-zero group.
__device__ __forceinline__ float group_scale(float amax) {
  return amax == 0.0f ? 1.0f : amax / 448.0f;
}

__device__ __forceinline__ float absmax8(uint4 v) {
  float m = fmaxf(fabsf(bf16_lo(v.x)), fabsf(bf16_hi(v.x)));
  m = fmaxf(m, fmaxf(fabsf(bf16_lo(v.y)), fabsf(bf16_hi(v.y))));
  m = fmaxf(m, fmaxf(fabsf(bf16_lo(v.z)), fabsf(bf16_hi(v.z))));
  m = fmaxf(m, fmaxf(fabsf(bf16_lo(v.w)), fabsf(bf16_hi(v.w))));
  return m;
}

// 8 bf16 -> 8 e4m3 bytes of x / s.
template <int ROUND>
__device__ __forceinline__ uint2 encode8_div(uint4 v, float s) {
  uint2 r;
  r.x = e4m3_pack4<ROUND>(bf16_lo(v.x) / s, bf16_hi(v.x) / s, bf16_lo(v.y) / s, bf16_hi(v.y) / s);
  r.y = e4m3_pack4<ROUND>(bf16_lo(v.z) / s, bf16_hi(v.z) / s, bf16_lo(v.w) / s, bf16_hi(v.w) / s);
  return r;
}

// 8 bf16 -> 8 e4m3 bytes of x * 2^k (exact power-of-two scaling).
template <int ROUND>
__device__ __forceinline__ uint2 encode8_ldexp(uint4 v, int k) {
  uint2 r;
  r.x = e4m3_pack4<ROUND>(ldexpf(bf16_lo(v.x), k), ldexpf(bf16_hi(v.x), k),
                          ldexpf(bf16_lo(v.y), k), ldexpf(bf16_hi(v.y), k));
  r.y = e4m3_pack4<ROUND>(ldexpf(bf16_lo(v.z), k), ldexpf(bf16_hi(v.z), k),
                          ldexpf(bf16_lo(v.w), k), ldexpf(bf16_hi(v.w), k));
  return r;
}

constexpr int kRowThreads = 256;       // 4 rows (one per wavefront) per workgroup
constexpr int kRowRegVecs = 16;        // rows up to 64*16*8 = 8192 elements stay in VGPRs

// One wavefront per row.  tensor_amax == nullptr: per-row scale from the
// row's own amax (written to scales[row]); otherwise the per-tensor amax (as
// fp32 bits) gives the scale, and block 0 writes it to scales[0].
template <int ROUND>
__global__ __launch_bounds__(kRowThreads) void quantize_rows_kernel(
    const uint16_t* __restrict__ x, int64_t rows, int64_t cols, int64_t ld,
    uint8_t* __restrict__ q, float* __restrict__ scales, const uint32_t* __restrict__ tensor_amax) {
  const int lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * (kRowThreads / 64) + (threadIdx.x >> 6);
  if (row >= rows) return;
  const uint4* src = reinterpret_cast<const uint4*>(x + row * ld);
  uint2* dst = reinterpret_cast<uint2*>(q + row * cols);
  const int64_t nvec = cols >> 3;
  const bool in_regs = nvec <= 64 * kRowRegVecs;

  uint4 buf[kRowRegVecs];
  float s;
  if (tensor_amax) {
    s = group_scale(__uint_as_float(*tensor_amax));
    if (row == 0 && lane == 0) scales[0] = s;
    if (in_regs) {
#pragma unroll
      for (int it = 0; it < kRowRegVecs; ++it) {
        const int64_t v = lane + 64 * it;
        if (v < nvec) buf[it] = src[v];
      }
    }
  } else {
    float amax = 0.0f;
    if (in_regs) {
#pragma unroll
      for (int it = 0; it < kRowRegVecs; ++it) {
        const int64_t v = lane + 64 * it;
        if (v < nvec) {
          buf[it] = src[v];
          amax = fmaxf(amax, absmax8(buf[it]));
        }
      }
    } else {
      for (int64_t v = lane; v < nvec; v += 64) amax = fmaxf(amax, absmax8(src[v]));
    }
    amax = wave_max(amax);
    s = group_scale(amax);
    if (lane == 0) scales[row] = s;
  }
  if (in_regs) {
#pragma unroll
    for (int it = 0; it < kRowRegVecs; ++it) {
      const int64_t v = lane + 64 * it;
      if (v < nvec) dst[v] = encode8_div<ROUND>(buf[it], s);
    }
  } else {
    for (int64_t v = lane; v < nvec; v += 64) dst[v] = encode8_div<ROUND>(src[v], s);
  }
}

__global__ void zero_u32_kernel(uint32_t* p) { *p = 0u; }

// Per-tensor amax: grid-stride over 16-byte vectors; the magnitudes are
// non-negative floats, whose bit patterns order like unsigned integers, so
// the grid-wide max is an atomicMax on the bits.
__global__ __launch_bounds__(256) void amax_kernel(const uint16_t* __restrict__ x, int64_t rows,
                                                   int64_t cols, int64_t ld, uint32_t* amax_bits) {
  const int64_t nvec_row = cols >> 3;
  const int64_t total = rows * nvec_row;
  float m = 0.0f;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total;
       i += (int64_t)gridDim.x * blockDim.x) {
    const int64_t r = i / nvec_row, v = i - r * nvec_row;
    m = fmaxf(m, absmax8(reinterpret_cast<const uint4*>(x + r * ld)[v]));
  }
  m = wave_max(m);
  if ((threadIdx.x & 63) == 0) atomicMax(amax_bits, __float_as_uint(m));
}

// MX32: one thread per 32-element block (64 bytes in, 32 bytes + 1 scale out).
template <int ROUND>
__global__ __launch_bounds__(256) void quantize_mx_kernel(const uint16_t* __restrict__ x, int64_t rows,
                                                          int64_t cols, int64_t ld,
                                                          uint8_t* __restrict__ q,
                                                          uint8_t* __restrict__ scales) {
  const int64_t nb_row = cols >> 5;
  const int64_t total = rows * nb_row;
  for (int64_t blk = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; blk < total;
       blk += (int64_t)gridDim.x * blockDim.x) {
    const int64_t r = blk / nb_row, b = blk - r * nb_row;
    const uint4* src = reinterpret_cast<const uint4*>(x + r * ld + 32 * b);
    uint4 v[4];
    float amax = 0.0f;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      v[k] = src[k];
      amax = fmaxf(amax, absmax8(v[k]));
    }
    // E8M0 code = clamp(floor(log2 amax) - 8 + 127, 0, 254); 0 for a zero block.
    int code = 0;
    if (amax > 0.0f) {
      int e2;
      (void)frexpf(amax, &e2);  // amax = f * 2^e2 with f in [0.5, 1)
      code = min(max(e2 - 1 - 8 + 127, 0), 254);
    }
    scales[blk] = (uint8_t)code;
    const int k2 = 127 - code;
    uint2 o[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) o[k] = encode8_ldexp<ROUND>(v[k], k2);
    uint4* dst = reinterpret_cast<uint4*>(q + r * cols + 32 * b);
    dst[0] = make_uint4(o[0].x, o[0].y, o[1].x, o[1].y);
    dst[1] = make_uint4(o[2].x, o[2].y, o[3].x, o[3].y);
  }
}

template <int ROUND>
__global__ __launch_bounds__(256) void encode_kernel(const float* __restrict__ x, int64_t n,
                                                     uint8_t* __restrict__ q) {
  const int64_t n4 = n >> 2;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n4;
       i += (int64_t)gridDim.x * blockDim.x) {
    const float4 v = reinterpret_cast<const float4*>(x)[i];
    reinterpret_cast<uint32_t*>(q)[i] = e4m3_pack4<ROUND>(v.x, v.y, v.z, v.w);
  }
  // tail (n % 4 elements), handled by the first threads of block 0
  if (blockIdx.x == 0 && threadIdx.x < (n & 3)) {
    const int64_t i = (n4 << 2) + threadIdx.x;
    q[i] = (uint8_t)(e4m3_pack4<ROUND>(x[i], 0.f, 0.f, 0.f) & 0xFFu);
  }
}

inline unsigned grid_for(int64_t work, int per_block, unsigned cap) {
  int64_t g = (work + per_block - 1) / per_block;
  if (g < 1) g = 1;
  if (g > cap) g = cap;
  return (unsigned)g;
}

template <int ROUND>
hipError_t launch_quantize_t(const uint16_t* x, int64_t rows, int64_t cols, int64_t ld,
                             int scaling, uint8_t* q, void* scales, void* workspace,
                             hipStream_t s) {
  if (rows == 0) {
    if (scaling == ACRL_SCALE_PER_TENSOR) {
      // the scale of an empty tensor is 1 (amax = 0)
      hipLaunchKernelGGL(zero_u32_kernel, dim3(1), dim3(1), 0, s, (uint32_t*)workspace);
      hipLaunchKernelGGL((quantize_rows_kernel<ROUND>), dim3(1), dim3(kRowThreads), 0, s, x,
                         (int64_t)1, (int64_t)0, ld, q, (float*)scales,
                         (const uint32_t*)workspace);
    }
    return hipGetLastError();
  }
  if (scaling == ACRL_SCALE_MX32) {
    const int64_t blocks = rows * (cols >> 5);
    hipLaunchKernelGGL((quantize_mx_kernel<ROUND>), dim3(grid_for(blocks, 256, 1u << 20)),
                       dim3(256), 0, s, x, rows, cols, ld, q, (uint8_t*)scales);
    return hipGetLastError();
  }
  const uint32_t* amax = nullptr;
  if (scaling == ACRL_SCALE_PER_TENSOR) {
    uint32_t* bits = (uint32_t*)workspace;
    hipLaunchKernelGGL(zero_u32_kernel, dim3(1), dim3(1), 0, s, bits);
    hipLaunchKernelGGL(amax_kernel, dim3(grid_for(rows * (cols >> 3), 256 * 8, 4096)), dim3(256),
                       0, s, x, rows, cols, ld, bits);
    amax = bits;
  }
  const int rows_per_block = kRowThreads / 64;
  hipLaunchKernelGGL((quantize_rows_kernel<ROUND>),
                     dim3((unsigned)((rows + rows_per_block - 1) / rows_per_block)),
                     dim3(kRowThreads), 0, s, x, rows, cols, ld, q, (float*)scales, amax);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_quantize(const uint16_t* x, int64_t rows, int64_t cols, int64_t ld, int scaling,
                           int rounding, uint8_t* q, void* scales, void* workspace, hipStream_t s) {
  if (rounding == ACRL_ROUND_TOWARD_ZERO)
    return launch_quantize_t<ACRL_ROUND_TOWARD_ZERO>(x, rows, cols, ld, scaling, q, scales,
                                                     workspace, s);
  return launch_quantize_t<ACRL_ROUND_NEAREST_EVEN>(x, rows, cols, ld, scaling, q, scales,
                                                    workspace, s);
}

hipError_t launch_fp8_encode(const float* x, int64_t n, int rounding, uint8_t* q, hipStream_t s) {
  if (n == 0) return hipSuccess;
  const unsigned g = grid_for((n + 3) / 4, 256, 1u << 16);
  if (rounding == ACRL_ROUND_TOWARD_ZERO)
    hipLaunchKernelGGL(encode_kernel<ACRL_ROUND_TOWARD_ZERO>, dim3(g), dim3(256), 0, s, x, n, q);
  else
    hipLaunchKernelGGL(encode_kernel<ACRL_ROUND_NEAREST_EVEN>, dim3(g), dim3(256), 0, s, x, n, q);
  return hipGetLastError();
}

}  // namespace acrl
