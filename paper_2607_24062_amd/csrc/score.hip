// score.hip -- sampled-token log-probabilities and entropies of every token
// under the BF16 training policy pi and the FP8 / MXFP8 inference policy mu
// (the quantities pi(a_t|theta_old), mu(a_t|theta_old) of Eq. distance_metric
// and of rho in Sec. 4.1 of the ACRL paper).
//
// Design (gfx950):
//  * The LM-head product is computed transposed, logits^T = W H^T, so that the
//    MFMA accumulator layout puts ONE TOKEN PER LANE COLUMN: lane l of a 32x32
//    block holds token column l%32 and 16 vocabulary rows.  The softmax
//    statistics of a token are then reduced inside each lane across all the
//    vocabulary rows it sees; lanes and waves are merged once per workgroup.
//  * Workgroup tile: 256 vocabulary rows x 256 tokens, 4 waves (2 x 2), each
//    wave 128 x 128 = 4 x 4 MFMA 32x32 blocks (256 fp32 accumulators / lane).
//    BF16: v_mfma_f32_32x32x16_bf16.  FP8: v_mfma_f32_32x32x64_f8f6f4.
//    MXFP8: v_mfma_scale_f32_32x32x64_f8f6f4 with per-lane E8M0 block scales.
//  * K is streamed in 128-byte chunks per row (64 bf16 or 128 fp8 values),
//    double-buffered in LDS (2 x 64 KiB) with an XOR swizzle of the 16-byte
//    columns so that fragment reads are bank-conflict free.
//  * Each workgroup sweeps a strip of vocabulary tiles for one token tile and
//    keeps a running (max, sum, entropy-sum) state per token in registers:
//    the [rows, V] logits never reach memory.  Online update, in log2 units
//    y = z*log2(e):  M = max y,  S = sum 2^(y-M),  U = sum 2^(y-M) (y-M);
//    lse = ln2 (M + log2 S), entropy = ln2 (log2 S - U/S).
//  * The strip's state per token goes to a workspace (split-V partials); a
//    merge kernel combines the strips and writes logp = z[a_t] - lse.
#include "acrl_internal.h"

namespace acrl {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef int i32x8 __attribute__((ext_vector_type(8)));

enum ScoreMode { kBF16 = 0, kFP8Tensor = 1, kFP8Row = 2, kMX = 3 };

constexpr int kTileV = 256;            // vocabulary rows per workgroup tile
constexpr int kTileT = 256;            // tokens per workgroup tile
constexpr int kChunk = 128;            // bytes of K per row per pipeline stage
constexpr int kThreads = 256;
constexpr int kStageBytes = (kTileV + kTileT) * kChunk;  // 64 KiB
constexpr float kInitMax = -1.0e30f;   // running max before any logit was seen

struct ScoreParams {
  const uint8_t* a;        // W (bf16) or Wq (e4m3): [V, row_bytes]
  const uint8_t* b;        // H or Hq: [n_rows, row_bytes]
  int64_t row_bytes;
  int n_chunks;            // row_bytes / kChunk
  int V;
  int n_rows;
  int n_vtiles;
  int tiles_per_strip;
  int n_strips;
  const float* a_scale;    // FP8 per-row: [V]; per-tensor: [1]
  const float* b_scale;    // FP8 per-row: [n_rows]; per-tensor: [1]
  const uint8_t* a_mx;     // MX: E8M0 [V, d/32]
  const uint8_t* b_mx;     // MX: E8M0 [n_rows, d/32]
  int mx_row_bytes;        // d / 32
  float inv_temp;
  const int32_t* ids;
  float* part;             // [3][n_strips][n_rows]: M, S, U of each strip
  float* logit;            // [n_rows]: z[a_t] (natural units)
};

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// Combine two partial softmax states (log2 units).
__device__ __forceinline__ void merge_state(float& M, float& S, float& U, float M2, float S2,
                                            float U2) {
  if (S2 == 0.0f) return;  // empty state (its M is only a reference point)
  if (S == 0.0f) {
    M = M2; S = S2; U = U2;
    return;
  }
  const float Mn = fmaxf(M, M2);
  const float d1 = M - Mn, d2 = M2 - Mn;
  const float a1 = fast_exp2(d1), a2 = fast_exp2(d2);
  U = a1 * fmaf(d1, S, U) + a2 * fmaf(d2, S2, U2);
  S = a1 * S + a2 * S2;
  M = Mn;
}

// 16 bytes per lane from global memory straight into LDS: lane l of the wave
// writes lds_wave_base + 16*l (gfx950 global_load_lds_dwordx4).
__device__ __forceinline__ void load16_to_lds(const void* gsrc, uint8_t* lds_wave_base) {
  __builtin_amdgcn_global_load_lds(
      (const void __attribute__((address_space(1)))*)gsrc,
      (void __attribute__((address_space(3)))*)lds_wave_base, 16, 0, 0);
}

__device__ __forceinline__ void wait_vm_all() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }

// acc[b][j][i] with 16b + i == idx, as an exact one-hot weighted sum: the
// weights max(1 - |idx - k|, 0) are exactly 0 or 1, so no lane masks or
// dynamically indexed registers are needed.
__device__ __forceinline__ float pick64(const f32x16 (&a)[4][4], int j, int idx) {
  float fi = (float)idx;
  // keep the weight arithmetic inside the (rarely taken) branch of the caller
  asm volatile("v_mov_b32 %0, %0" : "+v"(fi));
  float z = 0.0f;
#pragma unroll
  for (int b = 0; b < 4; ++b)
#pragma unroll
    for (int i = 0; i < 16; ++i)
      z = fmaf(fmaxf(1.0f - fabsf(fi - (float)(16 * b + i)), 0.0f), a[b][j][i], z);
  return z;
}

template <int MODE>
__global__ __attribute__((amdgpu_flat_work_group_size(kThreads, kThreads), amdgpu_waves_per_eu(1, 1)))
void score_kernel(ScoreParams p) {
  __shared__ __attribute__((aligned(1024))) uint8_t lds[2 * kStageBytes];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wv = wave & 1;   // which 128-row half of the vocabulary tile
  const int wt = wave >> 1;  // which 128-token half of the token tile
  const int r32 = lane & 31, g = lane >> 5, sw = lane & 7;

  const int st = blockIdx.x % p.n_strips;
  const int t0 = (blockIdx.x / p.n_strips) * kTileT;
  const int vt_begin = st * p.tiles_per_strip;
  const int vt_end = min(vt_begin + p.tiles_per_strip, p.n_vtiles);
  const int n_iter = (vt_end - vt_begin) * p.n_chunks;

  // ---- per-lane tokens: column r32 of each of the wave's 4 token blocks
  int tok[4], id[4];
  float c2[4], cz[4];
  float M[4], S[4], U[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    tok[j] = t0 + wt * 128 + j * 32 + r32;
    const int tc = min(tok[j], p.n_rows - 1);
    id[j] = p.ids[tc];
    float ct = p.inv_temp;
    if constexpr (MODE == kFP8Row) ct *= p.b_scale[tc];
    if constexpr (MODE == kFP8Tensor) ct *= p.b_scale[0] * p.a_scale[0];
    cz[j] = ct;            // logit = acc * (row scale) * cz
    c2[j] = ct * kLog2e;   // y     = acc * (row scale) * c2
    M[j] = kInitMax;
    S[j] = 0.0f;
    U[j] = 0.0f;
  }

  f32x16 acc[4][4];
#pragma unroll
  for (int b = 0; b < 4; ++b)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[b][j] = f32x16{};

  // ---- global -> LDS: wave w moves rows [64w, 64w+64) of both operand
  // tiles, 8 rows (1 KiB) per instruction.  Lane l fills LDS slot l of the
  // 1 KiB block: row 8k + l/8, swizzled column l%8, i.e. logical column
  // (l%8) ^ (row%8) of that row.
  const int lrow = lane >> 3;                     // row within the 8-row block
  const int lcol = ((lane & 7) ^ lrow) << 4;      // byte offset of the logical column
  uint32_t mxa_next[4], mxb_next[4], mxa[4], mxb[4];

  // Row offsets are 32-bit and relative to a wave-uniform base row, so the
  // loads take the scalar-base + vector-offset form.  Rows past the end of W
  // (or of H) are clamped to its last row; the base row is clamped too, so
  // every offset is in [0, 64).
  const int b_first = t0 + wave * 64;
  const int b_base = min(b_first, p.n_rows - 1);
  auto issue_loads = [&](int it, int stage) {
    const int q = it / p.n_chunks;
    const int kc = it - q * p.n_chunks;
    const int v0 = (vt_begin + q) * kTileV;
    const int a_first = v0 + wave * 64;
    const int a_base = min(a_first, p.V - 1);
    const uint8_t* ga = p.a + (int64_t)a_base * p.row_bytes + (int64_t)kc * kChunk;
    const uint8_t* gb = p.b + (int64_t)b_base * p.row_bytes + (int64_t)kc * kChunk;
    const uint32_t rb = (uint32_t)p.row_bytes;
    uint8_t* la = lds + stage * kStageBytes + (wave * 64) * kChunk;
    uint8_t* lb = la + kTileV * kChunk;
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      const int row = min(a_first + 8 * k + lrow, p.V - 1) - a_base;
      load16_to_lds(ga + ((uint32_t)row * rb + (uint32_t)lcol), la + k * 8 * kChunk);
    }
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      const int row = min(b_first + 8 * k + lrow, p.n_rows - 1) - b_base;
      load16_to_lds(gb + ((uint32_t)row * rb + (uint32_t)lcol), lb + k * 8 * kChunk);
    }
    if constexpr (MODE == kMX) {
      // the four E8M0 scales of the chunk's MX blocks for this lane's row
      const uint32_t mrb = (uint32_t)p.mx_row_bytes;
      const int sa_first = v0 + wv * 128, sb_first = t0 + wt * 128;
      const int sa_base = min(sa_first, p.V - 1), sb_base = min(sb_first, p.n_rows - 1);
      const uint8_t* sa = p.a_mx + (int64_t)sa_base * p.mx_row_bytes + kc * 4;
      const uint8_t* sb = p.b_mx + (int64_t)sb_base * p.mx_row_bytes + kc * 4;
#pragma unroll
      for (int b = 0; b < 4; ++b) {
        const int row = min(sa_first + b * 32 + r32, p.V - 1) - sa_base;
        mxa_next[b] = *reinterpret_cast<const uint32_t*>(sa + (uint32_t)row * mrb);
      }
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int row = min(sb_first + j * 32 + r32, p.n_rows - 1) - sb_base;
        mxb_next[j] = *reinterpret_cast<const uint32_t*>(sb + (uint32_t)row * mrb);
      }
    }
  };

  // K permutation inside a 128-byte chunk.  BF16 (4 MFMA steps of K=16):
  // lane group g supplies bytes [64g, 64g+64) of its row, step s the s-th
  // 16-byte piece.  FP8 (2 steps of K=64): an f8f6f4 operand is two 16-byte
  // halves per lane, and the MFMA treats register half h of BOTH lane groups
  // as its K block h (whose E8M0 scale lanes 32h..32h+31 supply).  Step s
  // therefore feeds half h with MX block 2s+h of the chunk: lane group g
  // takes its 16-byte piece g, i.e. 16-byte column 2(2s+h)+g of the row.
  // A (W rows) and B (H rows) use the same permutation, so dot products are
  // unchanged, and each MX block keeps its own scale.
  auto compute = [&](int stage) {
    const uint8_t* As = lds + stage * kStageBytes + (wv * 128 + r32) * kChunk;
    const uint8_t* Bs = lds + stage * kStageBytes + (kTileV + wt * 128 + r32) * kChunk;
    if constexpr (MODE == kBF16) {
#pragma unroll
      for (int s = 0; s < 4; ++s) {
        const int off = ((4 * g + s) ^ sw) << 4;
        bf16x8 bv[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) bv[j] = *reinterpret_cast<const bf16x8*>(Bs + j * 32 * kChunk + off);
#pragma unroll
        for (int b = 0; b < 4; ++b) {
          const bf16x8 af = *reinterpret_cast<const bf16x8*>(As + b * 32 * kChunk + off);
#pragma unroll
          for (int j = 0; j < 4; ++j)
            acc[b][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af, bv[j], acc[b][j], 0, 0, 0);
        }
      }
    } else {
#pragma unroll
      for (int s = 0; s < 2; ++s) {
        const int off0 = ((4 * s + g) ^ sw) << 4;      // register half 0: block 2s
        const int off1 = ((4 * s + 2 + g) ^ sw) << 4;  // register half 1: block 2s+1
        i32x8 bv[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const uint4 x0 = *reinterpret_cast<const uint4*>(Bs + j * 32 * kChunk + off0);
          const uint4 x1 = *reinterpret_cast<const uint4*>(Bs + j * 32 * kChunk + off1);
          bv[j] = i32x8{(int)x0.x, (int)x0.y, (int)x0.z, (int)x0.w, (int)x1.x, (int)x1.y, (int)x1.z, (int)x1.w};
        }
#pragma unroll
        for (int b = 0; b < 4; ++b) {
          const uint4 x0 = *reinterpret_cast<const uint4*>(As + b * 32 * kChunk + off0);
          const uint4 x1 = *reinterpret_cast<const uint4*>(As + b * 32 * kChunk + off1);
          const i32x8 af = i32x8{(int)x0.x, (int)x0.y, (int)x0.z, (int)x0.w, (int)x1.x, (int)x1.y, (int)x1.z, (int)x1.w};
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            if constexpr (MODE == kMX) {
              // lane group g supplies the scale of K block g of this step
              const int sa = (mxa[b] >> (8 * (2 * s + g))) & 0xFF;
              const int sb = (mxb[j] >> (8 * (2 * s + g))) & 0xFF;
              acc[b][j] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(af, bv[j], acc[b][j],
                                                                         0, 0, 0, sa, 0, sb);
            } else {
              acc[b][j] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(af, bv[j], acc[b][j],
                                                                         0, 0, 0, 0, 0, 0);
            }
          }
        }
      }
    }
  };

  // Fold one finished vocabulary tile into the running per-token states.
  // acc[b][j][i] is the logit (before scaling) of vocabulary row
  // v0 + 32b + 8(i/4) + 4g + (i%4) and token tok[j].
  // Fold one finished vocabulary tile into the running per-token states.
  // acc[b][j][i] is the logit (before scaling) of vocabulary row
  // v0 + 32b + 8(i/4) + 4g + (i%4) and token tok[j]; the 64 rows a lane holds
  // increase with 16b + i.  Rows past V were loaded as copies of row V-1, so
  // they hold a genuine logit: they may enter the max, and only their
  // contributions to S and U are removed, by the weight min(max(nv - idx, 0), 1)
  // where nv is the number of valid rows of the lane (a prefix of its rows).
  auto epilogue = [&](int tile) {
    const int v0 = tile * kTileV + wv * 128;
    const bool partial = v0 + 128 > p.V;
    float nv = 64.0f;
    if (partial) {
      const int lim = p.V - v0 - 4 * g;  // row offset o is valid iff o < lim
      int n = 0;
#pragma unroll
      for (int k = 0; k < 16; ++k) n += min(max(lim - 8 * k, 0), 4);
      nv = (float)n;
    }
    if constexpr (MODE == kFP8Row) {
      // multiply in the per-row weight scales, four consecutive rows at a time
#pragma unroll
      for (int b = 0; b < 4; ++b)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int r0 = v0 + b * 32 + 8 * q + 4 * g;
          float f[4];
          if (!partial) {
            const float4 v = *reinterpret_cast<const float4*>(p.a_scale + r0);
            f[0] = v.x; f[1] = v.y; f[2] = v.z; f[3] = v.w;
          } else {
#pragma unroll
            for (int k = 0; k < 4; ++k) f[k] = p.a_scale[min(r0 + k, p.V - 1)];
          }
#pragma unroll
          for (int j = 0; j < 4; ++j)
#pragma unroll
            for (int k = 0; k < 4; ++k) acc[b][j][4 * q + k] *= f[k];
          __builtin_amdgcn_sched_barrier(0);
        }
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      float mraw = -INFINITY;
#pragma unroll
      for (int b = 0; b < 4; ++b) {
#pragma unroll
        for (int i = 0; i < 16; ++i) mraw = fmaxf(mraw, acc[b][j][i]);
        __builtin_amdgcn_sched_barrier(0);
      }
      const float Mn = fmaxf(M[j], mraw * c2[j]);
      const float dM = M[j] - Mn;
      const float al = fast_exp2(dM);
      U[j] = al * fmaf(dM, S[j], U[j]);
      S[j] *= al;
      M[j] = Mn;
      const float nM = -Mn;
      float s0 = 0.f, u0 = 0.f;
#pragma unroll
      for (int b = 0; b < 4; ++b) {
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const float t = fmaf(acc[b][j][i], c2[j], nM);
          float e = fast_exp2(t);
          if (partial) e *= fminf(fmaxf(nv - (float)(16 * b + i), 0.0f), 1.0f);
          s0 += e;
          u0 = fmaf(e, t, u0);
        }
        __builtin_amdgcn_sched_barrier(0);
      }
      S[j] += s0;
      U[j] += u0;
      // the sampled token a_t: rare branch, taken by the one lane holding it
      const int rel = id[j] - v0;
      if ((unsigned)rel < 128u && ((rel >> 2) & 1) == g) {
        const int idx = (rel >> 5) * 16 + ((rel & 31) >> 3) * 4 + (rel & 3);
        const float z = pick64(acc, j, idx) * cz[j];
        if (tok[j] < p.n_rows && id[j] < p.V) p.logit[tok[j]] = z;
      }
      __builtin_amdgcn_sched_barrier(0);
    }
  };

  issue_loads(0, 0);
  if constexpr (MODE == kMX) {
#pragma unroll
    for (int k = 0; k < 4; ++k) { mxa[k] = mxa_next[k]; mxb[k] = mxb_next[k]; }
  }
  wait_vm_all();
  __syncthreads();
  int it = 0;
  for (int q = 0; q < vt_end - vt_begin; ++q) {
#pragma unroll
    for (int b = 0; b < 4; ++b)
#pragma unroll
      for (int j = 0; j < 4; ++j) acc[b][j] = f32x16{};
    for (int kc = 0; kc < p.n_chunks; ++kc, ++it) {
      const int stage = it & 1;
      if (it + 1 < n_iter) issue_loads(it + 1, stage ^ 1);  // lands in the other stage
      compute(stage);
      if constexpr (MODE == kMX) {
#pragma unroll
        for (int k = 0; k < 4; ++k) { mxa[k] = mxa_next[k]; mxb[k] = mxb_next[k]; }
      }
      wait_vm_all();
      __syncthreads();
    }
    epilogue(vt_begin + q);
  }

  // ---- merge the lane pair (l, l^32), then the two vocabulary halves
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const float M2 = __shfl_xor(M[j], 32), S2 = __shfl_xor(S[j], 32), U2 = __shfl_xor(U[j], 32);
    merge_state(M[j], S[j], U[j], M2, S2, U2);
  }
  float* xch = reinterpret_cast<float*>(lds);  // LDS is free after the last barrier
  if (wv == 1 && g == 0) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int k = wt * 128 + j * 32 + r32;
      xch[3 * k + 0] = M[j];
      xch[3 * k + 1] = S[j];
      xch[3 * k + 2] = U[j];
    }
  }
  __syncthreads();
  if (wv == 0 && g == 0) {
    const int64_t plane = (int64_t)p.n_strips * p.n_rows;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int k = wt * 128 + j * 32 + r32;
      merge_state(M[j], S[j], U[j], xch[3 * k + 0], xch[3 * k + 1], xch[3 * k + 2]);
      if (tok[j] < p.n_rows) {
        const int64_t o = (int64_t)st * p.n_rows + tok[j];
        p.part[o] = M[j];
        p.part[plane + o] = S[j];
        p.part[2 * plane + o] = U[j];
      }
    }
  }
}

struct MergeParams {
  int n_rows;
  int n_strips;
  int V;
  const float* part[2];
  const float* logit[2];
  const int32_t* ids;
  const uint8_t* mask;
  const int32_t* out_slot;
  float* logp[2];
  float* entropy[2];
  float* lse[2];
  float* zout[2];
  int32_t* error_flag;
};

// One thread per row: combine the strips' states of pi and mu.
__global__ __launch_bounds__(256) void merge_kernel(MergeParams p) {
  const int r = blockIdx.x * blockDim.x + threadIdx.x;
  if (r >= p.n_rows) return;
  const int slot = p.out_slot ? p.out_slot[r] : r;
  const bool active = p.mask ? p.mask[r] != 0 : true;
  const int id = p.ids[r];
  const bool id_ok = id >= 0 && id < p.V;
  if (active && !id_ok && p.error_flag) atomicOr(p.error_flag, 1);
  const int64_t plane = (int64_t)p.n_strips * p.n_rows;
#pragma unroll
  for (int q = 0; q < 2; ++q) {
    float lse = 0.f, ent = 0.f, lp = 0.f, z = 0.f;
    if (active) {
      float M = kInitMax, S = 0.f, U = 0.f;
      for (int s = 0; s < p.n_strips; ++s) {
        const int64_t o = (int64_t)s * p.n_rows + r;
        merge_state(M, S, U, p.part[q][o], p.part[q][plane + o], p.part[q][2 * plane + o]);
      }
      const float l2s = log2f(S);
      lse = (M + l2s) * kLn2;
      ent = (l2s - U / S) * kLn2;
      z = id_ok ? p.logit[q][r] : __builtin_nanf("");
      lp = z - lse;
    }
    p.logp[q][slot] = lp;
    if (p.entropy[q]) p.entropy[q][slot] = ent;
    if (p.lse[q]) p.lse[q][slot] = lse;
    if (p.zout[q]) p.zout[q][slot] = z;
  }
}

inline size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

thread_local hipEvent_t g_trace[4];
thread_local bool g_trace_on = false;

inline void trace(int k, hipStream_t s) {
  if (g_trace_on) (void)hipEventRecord(g_trace[k], s);
}

}  // namespace

void set_score_trace(void* const* events, int n) {
  g_trace_on = n == 4;
  for (int k = 0; k < 4; ++k) g_trace[k] = g_trace_on ? (hipEvent_t)events[k] : nullptr;
}

ScorePlan plan_score(int64_t n_rows, int64_t d, int64_t V) {
  (void)d;
  ScorePlan pl{};
  pl.n_ttiles = (int)((n_rows + kTileT - 1) / kTileT);
  pl.n_vtiles = (int)((V + kTileV - 1) / kTileV);
  // Choose the number of vocabulary strips: one workgroup per CU (256 CUs),
  // minimise the makespan ceil(WGs/256) * tiles-per-WG; ties -> fewer strips.
  const int64_t cus = 256;
  int best_s = 1;
  int64_t best_cost = -1;
  for (int s = 1; s <= pl.n_vtiles; ++s) {
    const int64_t tps = (pl.n_vtiles + s - 1) / s;
    const int64_t strips = (pl.n_vtiles + tps - 1) / tps;
    if (strips != s) continue;  // same as a smaller s
    const int64_t wgs = (int64_t)pl.n_ttiles * s;
    const int64_t cost = ((wgs + cus - 1) / cus) * tps;
    if (best_cost < 0 || cost < best_cost) {
      best_cost = cost;
      best_s = s;
    }
  }
  pl.tiles_per_strip = (pl.n_vtiles + best_s - 1) / best_s;
  pl.n_strips = (pl.n_vtiles + pl.tiles_per_strip - 1) / pl.tiles_per_strip;
  const size_t part_bytes = align_up((size_t)3 * pl.n_strips * (size_t)n_rows * sizeof(float), 256);
  const size_t logit_bytes = align_up((size_t)n_rows * sizeof(float), 256);
  size_t off = 0;
  for (int q = 0; q < 2; ++q) {
    pl.ws_part_offset[q] = off;
    off += part_bytes;
  }
  for (int q = 0; q < 2; ++q) {
    pl.ws_logit_offset[q] = off;
    off += logit_bytes;
  }
  pl.ws_bytes = off;
  return pl;
}

hipError_t launch_score(const acrl_score_desc& dsc, const ScorePlan& pl, hipStream_t s) {
  if (dsc.n_rows == 0) return hipSuccess;
  uint8_t* ws = static_cast<uint8_t*>(dsc.workspace);
  const unsigned grid = (unsigned)((int64_t)pl.n_ttiles * pl.n_strips);

  ScoreParams pp{};
  pp.V = (int)dsc.V;
  pp.n_rows = (int)dsc.n_rows;
  pp.n_vtiles = pl.n_vtiles;
  pp.tiles_per_strip = pl.tiles_per_strip;
  pp.n_strips = pl.n_strips;
  pp.inv_temp = dsc.inv_temperature;
  pp.ids = dsc.token_ids;
  pp.mx_row_bytes = (int)(dsc.d / 32);

  // pi: bf16 operands
  pp.a = static_cast<const uint8_t*>(dsc.w);
  pp.b = static_cast<const uint8_t*>(dsc.h);
  pp.row_bytes = dsc.d * 2;
  pp.n_chunks = (int)(pp.row_bytes / kChunk);
  pp.part = reinterpret_cast<float*>(ws + pl.ws_part_offset[0]);
  pp.logit = reinterpret_cast<float*>(ws + pl.ws_logit_offset[0]);
  trace(0, s);
  hipLaunchKernelGGL(score_kernel<kBF16>, dim3(grid), dim3(kThreads), 0, s, pp);
  trace(1, s);

  // mu: e4m3 operands
  ScoreParams pm = pp;
  pm.a = static_cast<const uint8_t*>(dsc.wq);
  pm.b = static_cast<const uint8_t*>(dsc.hq);
  pm.row_bytes = dsc.d;
  pm.n_chunks = (int)(pm.row_bytes / kChunk);
  pm.part = reinterpret_cast<float*>(ws + pl.ws_part_offset[1]);
  pm.logit = reinterpret_cast<float*>(ws + pl.ws_logit_offset[1]);
  if (dsc.mu_scaling == ACRL_SCALE_MX32) {
    pm.a_mx = static_cast<const uint8_t*>(dsc.wq_scales);
    pm.b_mx = static_cast<const uint8_t*>(dsc.hq_scales);
    hipLaunchKernelGGL(score_kernel<kMX>, dim3(grid), dim3(kThreads), 0, s, pm);
  } else {
    pm.a_scale = static_cast<const float*>(dsc.wq_scales);
    pm.b_scale = static_cast<const float*>(dsc.hq_scales);
    if (dsc.mu_scaling == ACRL_SCALE_PER_ROW)
      hipLaunchKernelGGL(score_kernel<kFP8Row>, dim3(grid), dim3(kThreads), 0, s, pm);
    else
      hipLaunchKernelGGL(score_kernel<kFP8Tensor>, dim3(grid), dim3(kThreads), 0, s, pm);
  }

  trace(2, s);
  MergeParams mp{};
  mp.n_rows = (int)dsc.n_rows;
  mp.n_strips = pl.n_strips;
  mp.V = (int)dsc.V;
  for (int q = 0; q < 2; ++q) {
    mp.part[q] = reinterpret_cast<const float*>(ws + pl.ws_part_offset[q]);
    mp.logit[q] = reinterpret_cast<const float*>(ws + pl.ws_logit_offset[q]);
  }
  mp.ids = dsc.token_ids;
  mp.mask = dsc.mask;
  mp.out_slot = dsc.out_slot;
  mp.logp[0] = dsc.logp_pi;       mp.logp[1] = dsc.logp_mu;
  mp.entropy[0] = dsc.entropy_pi; mp.entropy[1] = dsc.entropy_mu;
  mp.lse[0] = dsc.lse_pi;         mp.lse[1] = dsc.lse_mu;
  mp.zout[0] = dsc.logit_pi;      mp.zout[1] = dsc.logit_mu;
  mp.error_flag = dsc.error_flag;
  hipLaunchKernelGGL(merge_kernel, dim3((unsigned)((dsc.n_rows + 255) / 256)), dim3(256), 0, s, mp);
  trace(3, s);
  return hipGetLastError();
}

}  // namespace acrl
