// quantize.hip -- FP8 (OCP E4M3) quantization of bf16 matrices for the
// inference policy mu: per-tensor, per-row (per-token activations /
// per-channel weights, Sec. 5.1 of the ACRL paper) and MX32 (one E8M0 scale
// per 32 consecutive elements, the MXFP8 of Sec. 5.2).
//
// All three are HBM-bound streams: 2 bytes in and 1 byte out per element
// (per-tensor reads the tensor twice: amax pass, then encode).  Loads and
// stores are 16-byte vectors, one wavefront per row for the row kernels.
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

// x / s correctly rounded, from r = 1/s (correctly rounded, once per group)
// and one correction step: y = x r, the residual x - y s (exact in one FMA)
// times r moves y onto the correctly rounded quotient (Markstein).  The sign
// comes from y, so -0 stays -0.  For bf16 x with |x| <= amax and s = amax /
// 448 the result equals the divide, bit for bit, wherever the quotient can
// reach a nonzero E4M3 code (|x / s| >= 2^-12), and has its sign elsewhere,
// for every finite bf16 amax >= 2^-64 (checked over all such amax and x);
// groups with a smaller or non-finite amax take the divide.
constexpr float kRcpMinAmax = 0x1p-64f;
__device__ __forceinline__ bool rcp_ok(float amax) { return amax >= kRcpMinAmax && amax < INFINITY; }
__device__ __forceinline__ float div_rcp(float x, float s, float r) {
  const float y = __fmul_rn(x, r);
  return __builtin_copysignf(fmaf(fmaf(-y, s, x), r, y), y);
}

// 8 bf16 -> 8 e4m3 bytes of x / s by div_rcp.
template <int ROUND>
__device__ __forceinline__ uint2 encode8_rcp(uint4 v, float s, float r) {
  uint2 o;
  o.x = e4m3_pack4<ROUND>(div_rcp(bf16_lo(v.x), s, r), div_rcp(bf16_hi(v.x), s, r),
                          div_rcp(bf16_lo(v.y), s, r), div_rcp(bf16_hi(v.y), s, r));
  o.y = e4m3_pack4<ROUND>(div_rcp(bf16_lo(v.z), s, r), div_rcp(bf16_hi(v.z), s, r),
                          div_rcp(bf16_lo(v.w), s, r), div_rcp(bf16_hi(v.w), s, r));
  return o;
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
constexpr int kRowRegPairs = 8;        // rows up to 64*8*16 = 8192 elements stay in VGPRs

// 16 bf16 (two 16-byte vectors) -> 16 e4m3 bytes of x / s (RCP: by div_rcp).
template <int ROUND, bool RCP>
__device__ __forceinline__ uint4 encode16(uint4 a, uint4 b, float s, float r) {
  uint2 lo, hi;
  if constexpr (RCP) {
    lo = encode8_rcp<ROUND>(a, s, r);
    hi = encode8_rcp<ROUND>(b, s, r);
  } else {
    lo = encode8_div<ROUND>(a, s);
    hi = encode8_div<ROUND>(b, s);
  }
  return make_uint4(lo.x, lo.y, hi.x, hi.y);
}

// One wavefront per row; lane l owns the 32-byte pieces l, l + 64, ... of the
// row (two 16-byte loads, one 16-byte store each).  tensor_amax == nullptr:
// per-row scale from the row's own amax (written to scales[row]); otherwise
// the per-tensor amax (as fp32 bits) gives the scale, and block 0 writes it
// to scales[0].
template <int ROUND>
__global__ __launch_bounds__(kRowThreads) void quantize_rows_kernel(
    const uint16_t* __restrict__ x, int64_t rows, int64_t cols, int64_t ld,
    uint8_t* __restrict__ q, float* __restrict__ scales, const uint32_t* __restrict__ tensor_amax) {
  const int lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * (kRowThreads / 64) + (threadIdx.x >> 6);
  if (row >= rows) return;
  const uint4* src = reinterpret_cast<const uint4*>(x + row * ld);
  uint4* dst = reinterpret_cast<uint4*>(q + row * cols);
  const int64_t npair = cols >> 4;  // cols is a multiple of 32
  const bool in_regs = npair <= 64 * kRowRegPairs;

  uint4 buf[2 * kRowRegPairs];
  float s, amax;
  if (tensor_amax) {
    amax = __uint_as_float(*tensor_amax);
    s = group_scale(amax);
    if (row == 0 && lane == 0) scales[0] = s;
    if (in_regs) {
#pragma unroll
      for (int it = 0; it < kRowRegPairs; ++it) {
        const int64_t v = lane + 64 * it;
        if (v < npair) {
          buf[2 * it] = src[2 * v];
          buf[2 * it + 1] = src[2 * v + 1];
        }
      }
    }
  } else {
    amax = 0.0f;
    if (in_regs) {
#pragma unroll
      for (int it = 0; it < kRowRegPairs; ++it) {
        const int64_t v = lane + 64 * it;
        if (v < npair) {
          buf[2 * it] = src[2 * v];
          buf[2 * it + 1] = src[2 * v + 1];
          amax = fmaxf(amax, fmaxf(absmax8(buf[2 * it]), absmax8(buf[2 * it + 1])));
        }
      }
    } else {
      for (int64_t v = lane; v < npair; v += 64)
        amax = fmaxf(amax, fmaxf(absmax8(src[2 * v]), absmax8(src[2 * v + 1])));
    }
    amax = wave_max(amax);
    s = group_scale(amax);
    if (lane == 0) scales[row] = s;
  }
  auto store = [&](auto rcp_tag) {
    constexpr bool RCP = decltype(rcp_tag)::value;
    const float r = RCP ? 1.0f / s : 0.0f;
    if (in_regs) {
#pragma unroll
      for (int it = 0; it < kRowRegPairs; ++it) {
        const int64_t v = lane + 64 * it;
        if (v < npair) dst[v] = encode16<ROUND, RCP>(buf[2 * it], buf[2 * it + 1], s, r);
      }
    } else {
      for (int64_t v = lane; v < npair; v += 64) dst[v] = encode16<ROUND, RCP>(src[2 * v], src[2 * v + 1], s, r);
    }
  };
  if (rcp_ok(amax)) store(std::true_type{});  // uniform over the wavefront
  else store(std::false_type{});
}

__global__ void zero_u32_kernel(uint32_t* p) { *p = 0u; }

// Per-tensor amax: one wavefront per row (rows strided over the grid), eight
// 16-byte loads in flight per lane.  The magnitudes are non-negative floats,
// whose bit patterns order like unsigned integers, so the grid-wide max is an
// atomicMax on the bits (one per wavefront).
constexpr int kAmaxUnroll = 8;
// Contiguous tensors (ld == cols): the tensor as one array of 16-byte
// vectors, each workgroup sweeping its own contiguous range with kAmaxUnroll
// loads in flight per thread; one atomic per workgroup.
__global__ __launch_bounds__(256) void amax_flat_kernel(const uint4* __restrict__ x, int64_t nvec,
                                                        int64_t per_block, uint32_t* amax_bits) {
  __shared__ float sh[4];
  const int64_t begin = (int64_t)blockIdx.x * per_block;
  const int64_t end = min(begin + per_block, nvec);
  int64_t i = begin + threadIdx.x;
  float m = 0.0f;
  for (; i + 256 * (kAmaxUnroll - 1) < end; i += 256 * kAmaxUnroll) {
    uint4 t[kAmaxUnroll];
#pragma unroll
    for (int k = 0; k < kAmaxUnroll; ++k) t[k] = x[i + 256 * k];
#pragma unroll
    for (int k = 0; k < kAmaxUnroll; ++k) m = fmaxf(m, absmax8(t[k]));
  }
  for (; i < end; i += 256) m = fmaxf(m, absmax8(x[i]));
  m = wave_max(m);
  if ((threadIdx.x & 63) == 0) sh[threadIdx.x >> 6] = m;
  __syncthreads();
  if (threadIdx.x == 0) atomicMax(amax_bits, __float_as_uint(fmaxf(fmaxf(sh[0], sh[1]), fmaxf(sh[2], sh[3]))));
}

__global__ __launch_bounds__(256) void amax_kernel(const uint16_t* __restrict__ x, int64_t rows,
                                                   int64_t cols, int64_t ld, uint32_t* amax_bits) {
  const int lane = threadIdx.x & 63;
  const int64_t nvec = cols >> 3;
  const int64_t nwaves = (int64_t)gridDim.x * 4;
  float m = 0.0f;
  for (int64_t r = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6); r < rows; r += nwaves) {
    const uint4* src = reinterpret_cast<const uint4*>(x + r * ld);
    int64_t v = lane;
    for (; v + 64 * (kAmaxUnroll - 1) < nvec; v += 64 * kAmaxUnroll) {
      uint4 t[kAmaxUnroll];
#pragma unroll
      for (int k = 0; k < kAmaxUnroll; ++k) t[k] = src[v + 64 * k];
#pragma unroll
      for (int k = 0; k < kAmaxUnroll; ++k) m = fmaxf(m, absmax8(t[k]));
    }
    for (; v < nvec; v += 64) m = fmaxf(m, absmax8(src[v]));
  }
  m = wave_max(m);
  if (lane == 0) atomicMax(amax_bits, __float_as_uint(m));
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
    if (ld == cols) {
      const int64_t nvec = rows * (cols >> 3);
      const unsigned g = grid_for(nvec, 256 * kAmaxUnroll, 2048);
      const int64_t unit = 256 * kAmaxUnroll;
      const int64_t per_block = ((nvec + g - 1) / g + unit - 1) / unit * unit;
      hipLaunchKernelGGL(amax_flat_kernel, dim3(g), dim3(256), 0, s, reinterpret_cast<const uint4*>(x), nvec,
                         per_block, bits);
    } else {
      hipLaunchKernelGGL(amax_kernel, dim3(grid_for(rows, 4, 8192)), dim3(256), 0, s, x, rows, cols, ld,
                         bits);
    }
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
