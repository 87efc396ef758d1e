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
//  * Workgroup tile: 256 vocabulary rows x 256 tokens, one workgroup per CU,
//    4 waves of 128 x 128 (256 accumulators per lane) or 8 waves of 128 x 64
//    (128 accumulators, two waves per SIMD), chosen per instantiation.
//    BF16: v_mfma_f32_32x32x16_bf16.  FP8: v_mfma_f32_32x32x64_f8f6f4.
//    MXFP8: v_mfma_scale_f32_32x32x64_f8f6f4 with per-lane E8M0 block scales.
//  * K is streamed in 64-byte chunks per row (32 bf16 or 64 fp8 values) from
//    packed tile images straight into LDS (buffer_load ... lds), in a ring of
//    5 stages (4 for the per-row and MX scorers) with one barrier per chunk
//    and an XOR swizzle of the 16-byte columns so that fragment reads are
//    bank-conflict free.
//  * Each workgroup sweeps a strip of vocabulary tiles for one token tile and
//    keeps a running (max, sum, entropy-sum) state per token in registers:
//    the [rows, V] logits never reach memory.  Online update, in log2 units
//    y = z*log2(e):  M = max y,  S = sum 2^(y-M),  U = sum 2^(y-M) (y-M);
//    lse = ln2 (M + log2 S), entropy = ln2 (log2 S - U/S).
//  * The strip's state per token goes to a workspace (split-V partials); a
//    merge kernel combines the strips and writes logp = z[a_t] - lse.
//  * The scoring launches are persistent: one workgroup per CU takes
//    (token tile, strip) units from per-XCD queues in the workspace, its own
//    XCD's first, so that faster XCDs take more of them.
//  * The full-vocabulary KL / Euclidean measures fold into the pi kernel's
//    epilogue, against mu's logits stored by mu's pass of the same rows.
#include <algorithm>
#include <type_traits>

#include "acrl_internal.h"

namespace acrl {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef int i32x8 __attribute__((ext_vector_type(8)));
typedef int i32x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

enum ScoreMode { kBF16 = 0, kFP8Tensor = 1, kFP8Row = 2, kMX = 3 };

// What a workgroup does with each finished accumulator tile.
enum Epilogue {
  kEpiSoftmax = 0,  // online log-softmax statistics + sampled-token logit (scoring)
  kEpiSample = 1,   // the same plus a Gumbel-max draw (sampling from mu)
  kEpiGrad = 2,     // dZ = coef (onehot - softmax) / tau as bf16 operand images (backward)
  kEpiStore = 3,    // the product tile itself, fp32, stored (optionally on top of C)
  kEpiSoftmaxZ = 4, // kEpiSoftmax + the tile's logits stored (mu's pass of the full-vocabulary measures)
  kEpiSoftmaxDiv = 5, // kEpiSoftmax + the measures' sums against mu's stored logits (pi's pass)
};

constexpr int kTileV = 256;            // vocabulary rows per workgroup tile
constexpr int kTileT = 256;            // tokens per workgroup tile
constexpr int kChunk = 64;             // bytes of K per row per pipeline stage
constexpr int kThreads = 256;          // 4 waves; score_kernel<..., 8> runs 8 (two per SIMD)
constexpr int kStageBytes = (kTileV + kTileT) * kChunk;  // 32 KiB
constexpr int kPackBlock = kTileV * kChunk;               // packed image of one (tile, chunk): 16 KiB
constexpr float kInitMax = -1.0e30f;   // running max before any logit was seen
// Grid rasterization: the 32 workgroups an XCD runs at the same time (one per
// CU) form a block of kBlockT token tiles x kBlockS vocabulary strips, so
// each H chunk is shared by 4 and each W chunk by 8 workgroups in that
// XCD's L2 (8 x 4 measured a few percent faster than 4 x 8 at 4096 x
// 151936).  Workgroups are dispatched to the 8 XCDs round-robin.
constexpr int kXcds = 8;
constexpr int kBlockT = 8;
constexpr int kBlockS = 4;

struct ScoreParams {
  const uint8_t* a;        // packed W (bf16) or Wq (e4m3): [n_vtiles][n_chunks][16 KiB]
  const uint8_t* b;        // packed H or Hq: [n_ttiles][n_chunks][16 KiB]
  int n_chunks;            // bytes per row / kChunk
  int V;
  int n_rows;
  int n_vtiles;
  int tiles_per_strip;
  int n_strips;
  int n_ttiles;
  int n_tblocks;
  const float* a_scale;    // FP8 per-row: [V]; per-tensor: [1]
  const float* b_scale;    // FP8 per-row: [n_rows]; per-tensor: [1]
  const uint8_t* a_mx;     // MX: packed E8M0 image of W's scales (pack_mx_kernel)
  const uint8_t* b_mx;     // MX: packed E8M0 image of H's scales
  int mx_row_bytes;        // d / 32
  float inv_temp;
  const int32_t* ids;
  float* part;             // [3][n_strips][n_rows]: M, S, U of each strip
  float* logit;            // [n_rows]: z[a_t] (natural units)
  // sampling (Gumbel-max) only
  uint32_t seed_lo, seed_hi;
  int64_t row_offset;      // global token index of row 0 (the generator's counter)
  float* best_key;         // [n_strips][n_rows]: the strip's largest Gumbel key (log2 units)
  float* best_logit;       // [n_strips][n_rows]: its logit (natural units)
  int32_t* best_id;        // [n_strips][n_rows]: its vocabulary row
  // gradient of the surrogate (kEpiGrad) only
  const float* g_coef;     // [slots] d loss / d logp of each token
  const float* g_lse;      // [slots] log-sum-exp of pi's logits (natural units)
  const int32_t* g_slot;   // [n_rows] slot of each row (NULL: slot = row + g_slot_offset)
  int64_t g_slot_offset;
  uint8_t* gz_t;           // dZ image, rows = tokens, K = vocabulary: [n_ttiles][kch_v][256][64 B]
  uint8_t* gz_v;           // dZ image, rows = vocabulary, K = tokens: [n_vtiles][kch_t][256][64 B]
  int kch_v;               // 64-byte K chunks of a gz_t row (= n_vtiles * 8)
  int kch_t;               // 64-byte K chunks of a gz_v row (= n_ttiles * 8)
  // plain product (kEpiStore) only: C[m, n] (m = A row, n = B row), row-major
  float* c;
  int64_t ldc;
  int c_rows;              // valid A rows (M)
  int c_accumulate;        // 1: C += product (C is read once before the K loop)
  // row chunks and the full-vocabulary measures (kEpiSoftmaxZ, kEpiSoftmaxDiv)
  int tt_offset;           // token tile of this launch's tile 0 (n_ttiles counts the launch's tiles)
  float* zbuf;             // mu's logits of the launch's rows (natural units), accumulator layout (zbuf_index)
  const float* aq2;        // [256 n_ttiles] mu's log-sum-exp of the launch's rows, log2 units
  float* dpart;            // [5][2 n_vtiles][dp_rows] sums of the measures per 128 vocabulary rows (kEpiSoftmaxDiv)
  int64_t dp_rows;         // row stride of dpart's planes
  // persistent grid: one claim counter per XCD (kQueueStride ints apart,
  // zero at launch) and the units in each XCD's queue
  int* queue;
  int units_per_xcd;
};
constexpr int kQueueStride = 16;  // 64 bytes between the XCDs' counters

// Offset (in floats) of the first of the logits lane `lane` holds for 32 x 32
// block (bv, bt) -- vocabulary rows 32 bv + 8 (i/4) + 4 (lane/32) + i%4,
// token 32 bt + lane%32 of the tile -- of token tile tt and vocabulary tile
// vt in the stored logits of a pass.  Each (tt, vt) tile is 256 KiB, each
// 32 x 32 block 4 KiB; values i = 4m .. 4m + 3 of lane l sit at floats
// 256 m + 4 l .. 256 m + 4 l + 3 of the block, so one 16-byte access per
// lane and m moves 1 KiB of contiguous memory per wavefront.  The layout is
// that of the 32x32 MFMA accumulators, whatever the wave count of the mu
// kernel that stores and the pi kernel that reads.
constexpr int kZRun = 256;  // floats between the runs m and m + 1 of a block
__device__ __forceinline__ int64_t zbuf_index(int tt, int n_vtiles, int vt, int bv, int bt, int lane) {
  return (((int64_t)tt * n_vtiles + vt) * 64 + bv * 8 + bt) * 1024 + lane * 4;
}

// Philox4x32-10 (Salmon et al., SC 2011): 10 rounds on a 128-bit counter
// under a 64-bit key; each round multiplies words 0 and 2 by the round
// constants and mixes the high halves with the other words and the key, the
// key advancing by the Weyl constants.
__device__ __forceinline__ void philox4x32_10(uint32_t c0, uint32_t c1, uint32_t c2, uint32_t c3, uint32_t k0,
                                              uint32_t k1, uint32_t (&out)[4]) {
#pragma unroll
  for (int round = 0; round < 10; ++round) {
    const uint32_t hi0 = __umulhi(0xD2511F53u, c0), lo0 = 0xD2511F53u * c0;
    const uint32_t hi1 = __umulhi(0xCD9E8D57u, c2), lo1 = 0xCD9E8D57u * c2;
    const uint32_t n0 = hi1 ^ c1 ^ k0, n2 = hi0 ^ c3 ^ k1;
    c0 = n0;
    c1 = lo1;
    c2 = n2;
    c3 = lo0;
    k0 += 0x9E3779B9u;
    k1 += 0xBB67AE85u;
  }
  out[0] = c0;
  out[1] = c1;
  out[2] = c2;
  out[3] = c3;
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// Combine two partial softmax states (log2 units).
__device__ __forceinline__ void merge_state(float& M, float& S, float& U, float M2, float S2,
                                            float U2) {
#pragma clang fp contract(off)
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

// Buffer resource of `bytes` bytes at `base` (raw, unswizzled; gfx9 dword 3).
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes, 0x00020000);
}

// SIZE (4 or 16) bytes per lane from a buffer straight into LDS: lane l of
// the wave writes lds_wave_base + SIZE*l (buffer_load ... lds).  voffset is
// the lane's byte offset, soffset a wave-uniform byte offset.
template <int SIZE>
__device__ __forceinline__ void buffer_to_lds(__amdgpu_buffer_rsrc_t r, uint32_t voffset, uint32_t soffset,
                                              uint8_t* lds_wave_base) {
  auto* l = (__attribute__((address_space(3))) void*)lds_wave_base;
  if constexpr (SIZE == 16) __builtin_amdgcn_raw_ptr_buffer_load_lds(r, l, 16, (int)voffset, (int)soffset, 0, 0);
  else if constexpr (SIZE == 4) __builtin_amdgcn_raw_ptr_buffer_load_lds(r, l, 4, (int)voffset, (int)soffset, 0, 0);
  else static_assert(SIZE == 16, "size must be 4 or 16");
}

// One accumulator value, read out of its AGPR exactly here (an opaque read:
// the compiler may neither hoist it nor keep a VGPR copy of the whole tile).
__device__ __forceinline__ float acc_read(float a) {
  float r;
  asm volatile("v_accvgpr_read_b32 %0, %1" : "=v"(r) : "a"(a));
  return r;
}


// Workgroup barrier once at most N vector-memory loads of this wave are
// outstanding and all its LDS reads have completed.  Written as one asm
// statement (a compiler memory barrier, not a fence): a release fence would
// also wait for every buffer -> LDS load still in flight, draining the
// pipeline; ordering against those loads comes from the vmcnt count.
template <int N>
__device__ __forceinline__ void wait_loads_and_barrier() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)\n\ts_barrier" ::"n"(N) : "memory");
}

// Scheduling group of n LDS reads (the builtin takes literal sizes only;
// n is a constant once the caller's loop is unrolled).
__device__ __forceinline__ void sched_ds_reads(int n) {
  switch (n) {
    case 1: __builtin_amdgcn_sched_group_barrier(0x100, 1, 0); break;
    case 2: __builtin_amdgcn_sched_group_barrier(0x100, 2, 0); break;
    case 3: __builtin_amdgcn_sched_group_barrier(0x100, 3, 0); break;
    case 5: __builtin_amdgcn_sched_group_barrier(0x100, 5, 0); break;
    case 10: __builtin_amdgcn_sched_group_barrier(0x100, 10, 0); break;
    case 12: __builtin_amdgcn_sched_group_barrier(0x100, 12, 0); break;
    case 15: __builtin_amdgcn_sched_group_barrier(0x100, 15, 0); break;
    default: break;
  }
}

// MXFP8 product whose E8M0 scales are byte oa of sa (A rows) and byte ob of
// sb (B rows).  The byte selects are immediates of the instruction; oa and ob
// are constants once the caller's loops are unrolled.
template <int OA>
__device__ __forceinline__ f32x16 mfma_mx_b(const i32x8& a, const i32x8& b, const f32x16& c, int sa, int sb,
                                            int ob) {
  switch (ob) {
    case 0: return __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a, b, c, 0, 0, OA, sa, 0, sb);
    case 1: return __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a, b, c, 0, 0, OA, sa, 1, sb);
    case 2: return __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a, b, c, 0, 0, OA, sa, 2, sb);
    default: return __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a, b, c, 0, 0, OA, sa, 3, sb);
  }
}
__device__ __forceinline__ f32x16 mfma_mx(const i32x8& a, const i32x8& b, const f32x16& c, int sa, int oa, int sb,
                                          int ob) {
  switch (oa) {
    case 0: return mfma_mx_b<0>(a, b, c, sa, sb, ob);
    case 1: return mfma_mx_b<1>(a, b, c, sa, sb, ob);
    case 2: return mfma_mx_b<2>(a, b, c, sa, sb, ob);
    default: return mfma_mx_b<3>(a, b, c, sa, sb, ob);
  }
}

// Wait until at most N vector-memory loads of this wave are outstanding
// (gfx9 s_waitcnt encoding: vmcnt in bits 3:0 and 15:14, expcnt and lgkmcnt
// left at their maxima).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (15 << 8) | ((N >> 4) << 14));
}

// Operand stages in LDS (one 64-byte K chunk of every row of both tiles per
// stage).  MX also streams the E8M0 scales of the chunk's two MX blocks with
// each stage (2 bytes per row of both tiles, 1 KiB, from the packed scale
// images), and the per-row FP8 mode keeps the weight-row scales of the last
// NS + 1 vocabulary tiles (a tile's scales arrive with its first chunk, up to
// NS chunks before the previous tile's epilogue reads its own), so both keep
// one operand stage less.
template <int MODE>
struct Pipe {
  static constexpr int kStages = (MODE == kMX || MODE == kFP8Row) ? 4 : 5;
  static constexpr int kScaleBytes = (MODE == kMX) ? (kTileV + kTileT) * 2 : 0;  // per stage
  static constexpr int kRowScaleSlots = kStages + 1;
  static constexpr int kRowScaleBytes = (MODE == kFP8Row) ? kRowScaleSlots * kTileV * 4 : 0;
  // buffer -> LDS loads per chunk per wave: the two 16 KiB tile images spread
  // over NW waves (1 KiB per load), plus one quarter of the MX scales (4
  // bytes per lane)
  template <int NW>
  static constexpr int loads_per_chunk() { return 2 * (16 / NW) + (MODE == kMX ? 1 : 0); }
};

// NW = 4: one wave per SIMD, each wave 128 vocabulary rows x 128 tokens
// (4 x 4 blocks of 32 x 32, 256 accumulators per lane).  NW = 8: two waves
// per SIMD, each 128 x 64 (4 x 2 blocks, 128 accumulators): while one wave
// waits at the chunk barrier or runs its softmax epilogue the other keeps
// the SIMD's matrix core busy.
// PERSIST: one workgroup per CU claims units from per-XCD queues (below);
// otherwise one workgroup per unit.
template <int MODE, int EPI, int NW, bool PERSIST>
__global__ __attribute__((amdgpu_flat_work_group_size(NW * 64, NW * 64), amdgpu_waves_per_eu(NW / 4, NW / 4)))
void score_kernel(ScoreParams p) {
  static_assert(NW == 4 || NW == 8, "4 or 8 waves");
  constexpr int JT = 16 / NW;   // token blocks of 32 per wave
  constexpr int TW = 32 * JT;   // tokens per wave
  constexpr bool SAMPLE = EPI == kEpiSample;
  constexpr bool DIV = EPI == kEpiSoftmaxDiv;
  constexpr bool SOFTMAX = EPI == kEpiSoftmax || EPI == kEpiSample || EPI == kEpiSoftmaxZ || DIV;
  static_assert(MODE == kBF16 || SOFTMAX, "the backward epilogues take bf16 operands");
  static_assert(!DIV || MODE == kBF16, "the measures are accumulated in pi's pass");
  constexpr int NS = Pipe<MODE>::kStages;
  // FP8 per-tensor / MX scorers start each tile's accumulators with an
  // inline-zero MFMA instead of clearing them after the epilogue (measured:
  // faster there; the BF16 and per-row FP8 kernels keep the clearing)
  constexpr bool kZeroStart = SOFTMAX && (MODE == kFP8Tensor || MODE == kMX);
  constexpr int SB = Pipe<MODE>::kScaleBytes;
  constexpr int LPC = Pipe<MODE>::template loads_per_chunk<NW>();
  constexpr int RSB = Pipe<MODE>::kRowScaleBytes;
  static_assert(MODE != kMX || NW == 4, "the MX scale stream is spread over 4 waves");
  __shared__ __attribute__((aligned(1024))) uint8_t lds[NS * (kStageBytes + SB) + RSB];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wv = wave & 1;   // which 128-row half of the vocabulary tile
  const int wt = wave >> 1;  // which 128-token half of the token tile
  const int r32 = lane & 31, g = lane >> 5;
  const int sw = (lane >> 2) & 3;  // swizzle of this lane's fragment row (see below)

  // ---- one unit of work: token tile tt (of the launch) against vocabulary
  // strip st (the dispatch below picks the units)
  auto unit = [&](int tt, int st) {
  if (tt >= p.n_ttiles || st >= p.n_strips) return;  // padding of the grid
  const int ttg = tt + p.tt_offset;  // token tile in the whole call
  const int t0 = ttg * kTileT;
  const int vt_begin = st * p.tiles_per_strip;
  const int vt_end = min(vt_begin + p.tiles_per_strip, p.n_vtiles);
  const int n_iter = (vt_end - vt_begin) * p.n_chunks;

  // ---- per-lane tokens: column r32 of each of the wave's 4 token blocks
  int tok[4], id[4];
  float c2[4], cz[4];
  float gl2[4], gc[4];  // backward: lse (log2 units) and coef / tau of the lane's tokens
  float M[4], S[4], U[4];
  float bk[4], bz[4];  // sampling: best Gumbel key of the lane and its logit
  int bi[4];           //           and vocabulary row
#pragma unroll
  for (int j = 0; j < JT; ++j) {
    tok[j] = t0 + wt * TW + j * 32 + r32;
    const int tc = min(tok[j], p.n_rows - 1);
    id[j] = (EPI == kEpiSample || EPI == kEpiStore) ? -1 : p.ids[tc];
    gl2[j] = 0.0f;
    gc[j] = 0.0f;
    if constexpr (EPI == kEpiGrad) {
      // rows past the end and rows with coef 0 (masked) get dZ = 0
      const int64_t slot = p.g_slot ? (int64_t)p.g_slot[tc] : p.g_slot_offset + tc;
      const float cf = tok[j] < p.n_rows ? p.g_coef[slot] : 0.0f;
      gc[j] = cf * p.inv_temp;
      gl2[j] = cf != 0.0f ? p.g_lse[slot] * kLog2e : 0.0f;
    }
    bk[j] = -INFINITY;
    bz[j] = 0.0f;
    bi[j] = 0;
    float ct = p.inv_temp;
    if constexpr (MODE == kFP8Row) ct *= p.b_scale[tc];
    if constexpr (MODE == kFP8Tensor) ct *= p.b_scale[0] * p.a_scale[0];
    cz[j] = ct;            // logit = acc * (row scale) * cz
    c2[j] = ct * kLog2e;   // y     = acc * (row scale) * c2
    M[j] = kInitMax;
    S[j] = 0.0f;
    U[j] = 0.0f;
  }

  f32x16 acc[4][JT];
#pragma unroll
  for (int b = 0; b < 4; ++b)
#pragma unroll
    for (int j = 0; j < JT; ++j) acc[b][j] = f32x16{};
  if constexpr (EPI == kEpiStore) {
    // one output tile per workgroup: start from C when accumulating
    if (p.c_accumulate) {
      const int m0 = vt_begin * kTileV + wv * 128 + 4 * g;
#pragma unroll
      for (int b = 0; b < 4; ++b)
#pragma unroll
        for (int j = 0; j < JT; ++j)
#pragma unroll
          for (int i = 0; i < 16; ++i) {
            const int m = m0 + 32 * b + 8 * (i >> 2) + (i & 3);
            if (m < p.c_rows && tok[j] < p.n_rows) acc[b][j][i] = p.c[(int64_t)m * p.ldc + tok[j]];
          }
    }
  }

  // ---- global -> LDS.  A stage holds one 64-byte K chunk of all 256 + 256
  // rows (W tile rows first).  Operands come packed (pack_kernel): the
  // 16 KiB image of each (256-row tile, chunk) pair is stored contiguously
  // exactly as the stage holds it, so a wave moves 4 KiB of contiguous
  // memory per tile with 4 buffer -> LDS loads of 1 KiB (lane l: bytes
  // [16l, 16l+16) of the KiB).  In the image a row's 16-byte column c sits at
  // position c ^ ((row/4) % 4): the 16 lanes one LDS cycle serves read 16
  // consecutive rows and hit 16 distinct bank groups.  Rows past the end of
  // W / H hold copies of its last row.
  const int wave_u = __builtin_amdgcn_readfirstlane(wave);
  const uint32_t lane_off = (uint32_t)lane * 16;
  const uint32_t tile_bytes = (uint32_t)p.n_chunks * kPackBlock;  // packed bytes of one tile
  const int b_rows = min(kTileT, p.n_rows - t0);  // valid rows of the token tile
  const __amdgpu_buffer_rsrc_t rsrc_b = make_rsrc(p.b + (int64_t)ttg * tile_bytes, tile_bytes);
  auto stage_at = [&](int stg) { return lds + stg * kStageBytes; };
  auto scales_at = [&](int stg) { return lds + NS * kStageBytes + stg * SB; };
  auto rowscales_at = [&](int q) {  // FP8 per-row: weight-row scales of tile q
    return reinterpret_cast<float*>(lds + NS * (kStageBytes + SB) + (q % Pipe<MODE>::kRowScaleSlots) * kTileV * 4);
  };

  auto issue_chunk = [&](int q, int kc, int stg) {  // chunk kc of the strip's tile q into stage stg
    const int v0 = (vt_begin + q) * kTileV;
    const int a_rows = min(kTileV, p.V - v0);  // valid rows of the vocabulary tile
    const __amdgpu_buffer_rsrc_t rsrc_a = make_rsrc(p.a + (int64_t)(vt_begin + q) * tile_bytes, tile_bytes);
    const uint32_t soff = (uint32_t)kc * kPackBlock + (uint32_t)wave_u * (kPackBlock / NW);
    uint8_t* la = stage_at(stg) + wave_u * (kPackBlock / NW);
    uint8_t* lb = la + kTileV * kChunk;
#pragma unroll
    for (int k = 0; k < 16 / NW; ++k) buffer_to_lds<16>(rsrc_a, lane_off, soff + k * 1024, la + k * 1024);
#pragma unroll
    for (int k = 0; k < 16 / NW; ++k) buffer_to_lds<16>(rsrc_b, lane_off, soff + k * 1024, lb + k * 1024);
    if constexpr (MODE == kFP8Row) {
      // with a tile's first chunk: its 256 weight-row scales (lane l of wave
      // w moves row 64w + l); they land long before the tile's epilogue
      if (kc == 0 && (NW == 4 || wave_u < 4)) {  // 64 rows per wave
        const __amdgpu_buffer_rsrc_t rs = make_rsrc(p.a_scale + v0, (uint32_t)a_rows * 4);
        buffer_to_lds<4>(rs, (uint32_t)min(wave_u * 64 + lane, a_rows - 1) * 4, 0,
                         reinterpret_cast<uint8_t*>(rowscales_at(q)) + wave_u * 64 * 4);
      }
    }
    if constexpr (MODE == kMX) {
      // the chunk's E8M0 scales (MX blocks 2kc, 2kc+1: 2 bytes per row) of
      // the 256 W rows (waves 0, 1) and the 256 H rows (waves 2, 3), 256
      // contiguous bytes per wave in the packed scale images
      const uint32_t tmx = (uint32_t)kTileV * (uint32_t)p.mx_row_bytes;  // bytes of one tile's image
      const __amdgpu_buffer_rsrc_t rs = wave_u < 2 ? make_rsrc(p.a_mx + (int64_t)(vt_begin + q) * tmx, tmx)
                                                   : make_rsrc(p.b_mx + (int64_t)ttg * tmx, tmx);
      buffer_to_lds<4>(rs, (uint32_t)lane * 4u, (uint32_t)kc * 512u + (uint32_t)(wave_u & 1) * 256u,
                       scales_at(stg) + wave_u * 256);
    }
  };

  // ---- MFMA fragments.  K permutation inside a chunk (the same for W and
  // H rows, so dot products are unchanged).  BF16 (2 MFMA steps of K=16):
  // lane group g of step s supplies 16-byte column 2s+g of its row.  FP8
  // (1 step of K=64): an f8f6f4 operand is two 16-byte halves per lane, and
  // the MFMA treats register half h of BOTH lane groups as its K block h,
  // whose E8M0 scale the lanes of group h supply; half h therefore holds MX
  // block h of the chunk, lane group g its 16-byte piece g (column 2h+g).
  // A group = one (step, vocabulary block b): 4 MFMAs sharing the A fragment.
  constexpr int G = (MODE == kBF16) ? 8 : 4;  // groups per chunk
  using FragT = typename std::conditional<MODE == kBF16, bf16x8, i32x8>::type;
  auto frag_off = [&](int grp) {  // byte offset of the fragment's first 16-byte piece in its row
    if constexpr (MODE == kBF16) return ((2 * (grp >> 2) + g) ^ sw) << 4;
    else return (g ^ sw) << 4;
  };
  // LDS reads use typed vector loads: the compiler then trusts them not to
  // alias the LDS written by the buffer -> LDS loads and adds no vmcnt wait of
  // its own before them (such a wait would drain the whole pipeline).  The
  // order of DMA and reads comes from the explicit vmcnt waits and barriers.
  auto read16x2 = [&](const uint8_t* row) -> FragT {
    if constexpr (MODE == kBF16) {
      return *reinterpret_cast<const bf16x8*>(row);
    } else {
      const int off0 = (g ^ sw) << 4, off1 = ((2 + g) ^ sw) << 4;
      const i32x4 x0 = *reinterpret_cast<const i32x4*>(row + off0);
      const i32x4 x1 = *reinterpret_cast<const i32x4*>(row + off1);
      return __builtin_shufflevector(x0, x1, 0, 1, 2, 3, 4, 5, 6, 7);
    }
  };
  // A fragment of group grp (vocabulary block grp%4), B fragments of its step
  auto read_a = [&](int stg, int grp) -> FragT {
    const uint8_t* row = stage_at(stg) + (wv * 128 + (grp & 3) * 32 + r32) * kChunk;
    if constexpr (MODE == kBF16) return read16x2(row + frag_off(grp));
    else return read16x2(row);
  };
  auto read_b = [&](int stg, int grp, FragT (&bf)[JT]) {
#pragma unroll
    for (int j = 0; j < JT; ++j) {
      const uint8_t* row = stage_at(stg) + (kTileV + wt * TW + j * 32 + r32) * kChunk;
      if constexpr (MODE == kBF16) bf[j] = read16x2(row + frag_off(grp));
      else bf[j] = read16x2(row);
    }
  };
  // MX scales of the chunk in stage stg (512 bytes of W rows, then 512 of H
  // rows, in the order pack_mx_kernel writes): one dword per lane and
  // operand holds the block-2kc+g scales of the lane's row in each of the
  // wave's four 32-row blocks, byte b for block b.
  auto read_sa = [&](int stg) -> int {
    return *reinterpret_cast<const int*>(scales_at(stg) + ((wv * 2 + g) * 32 + r32) * 4);
  };
  auto read_sb = [&](int stg) -> int {
    return *reinterpret_cast<const int*>(scales_at(stg) + 2 * kTileV + ((wt * 2 + g) * 32 + r32) * 4);
  };
  // zc: the accumulators start from zero (the first K step of a tile), so
  // the MFMA takes an inline zero instead of them and no clearing is needed
  auto mfma_group = [&](auto zc_tag, int grp, const FragT& fa, const FragT (&fb)[JT], int sa, int sb) {
    constexpr bool kZero = decltype(zc_tag)::value;
    const int bb = grp & 3;
#pragma unroll
    for (int j = 0; j < JT; ++j) {
      const f32x16 c = kZero ? f32x16{} : acc[bb][j];
      if constexpr (MODE == kBF16) {
        acc[bb][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa, fb[j], c, 0, 0, 0);
      } else if constexpr (MODE == kMX) {
        acc[bb][j] = mfma_mx(fa, fb[j], c, sa, bb, sb, j);
      } else {
        (void)sa;
        (void)sb;
        acc[bb][j] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(fa, fb[j], c, 0, 0, 0, 0, 0, 0);
      }
    }
  };

  // Fold one finished vocabulary tile into the running per-token states.
  // acc[b][j][i] is the logit (before scaling) of vocabulary row
  // v0 + 32b + 8(i/4) + 4g + (i%4) and token tok[j]; the 64 rows a lane holds
  // increase with 16b + i.  Online softmax at the granularity of these
  // 16-value blocks: each block is read once, its maximum re-bases the
  // running state, then its exponentials, sums and (rarely) the sampled
  // logit come from the same 16 registers.  Rows past V were loaded as
  // copies of row V-1, so they hold a genuine logit: they may enter the
  // maximum, and only their contributions to S and U are removed, by the
  // weight min(max(nv - idx, 0), 1) with nv the lane's count of valid rows
  // (a prefix of its rows).
  auto epilogue = [&](int tile, int q) {
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
    // keep the tail weights derived from nv inside the epilogue (else they
    // are computed before the K loop and held across it)
    asm volatile("v_mov_b32 %0, %0" : "+v"(nv));
    // full-vocabulary measures: mu's lse (log2 units) of the lane's tokens
    // and the tile's five sums per token (live only in the epilogue)
    float a2[4], dv[5][4];
    // the lane's token row in the tile and its 128-row slot of the sums,
    // formed here through an opaque move (else the addresses below are
    // hoisted out of the tile loop and held across it)
    int dv_row = wt * TW + r32, dv_slot = wv;
    asm volatile("v_mov_b32 %0, %0\n\tv_mov_b32 %1, %1" : "+v"(dv_row), "+v"(dv_slot));
    if constexpr (DIV) {
#pragma unroll
      for (int j = 0; j < JT; ++j) {
        a2[j] = p.aq2[tt * kTileT + dv_row + j * 32];
#pragma unroll
        for (int c = 0; c < 5; ++c) dv[c][j] = 0.0f;
      }
    }
    // The pass, written for instruction-level parallelism (one wave per
    // SIMD: nothing else hides latencies): all 16 exponents of a block are
    // formed before any is used, maxima and sums are trees.  The tail tile
    // (rows past V present) takes its own copy of the code.
    auto run = [&](auto tail_tag) {
      // every fused multiply-add below is written out (fmaf): no contraction
      // of the rest, so every variant rounds the statistics alike
#pragma clang fp contract(off)
      constexpr bool kTail = decltype(tail_tag)::value;
      uint32_t pw[JT][2];  // sampling: the Philox words the odd block of a pair uses
      (void)pw;
#pragma unroll
      for (int b = 0; b < 4; ++b) {
#pragma unroll
        for (int j = 0; j < JT; ++j) {
          float rs[16];
          if constexpr (MODE == kFP8Row) {
            // the block's 16 weight-row scales, read per token block (fewer
            // live registers than keeping them across the token blocks)
            const float* rsl = rowscales_at(q) + wv * 128 + b * 32 + 4 * g;
#pragma unroll
            for (int qq = 0; qq < 4; ++qq) {
              const f32x4 f = *reinterpret_cast<const f32x4*>(rsl + 8 * qq);
              rs[4 * qq + 0] = f[0]; rs[4 * qq + 1] = f[1]; rs[4 * qq + 2] = f[2]; rs[4 * qq + 3] = f[3];
            }
          }
          float v[16];
#pragma unroll
          for (int i = 0; i < 16; ++i) {
            // (the 8-wave per-row FP8 kernels and the 8-wave passes of the
            // full-vocabulary measures keep their accumulators in VGPRs, the
            // MFMA's VGPR form: 12 instead of 112 bytes spilled per lane in
            // the persistent per-row scorer, mu 1.5-7 % faster, and 12
            // instead of 104 in pi's measures pass, the measures 6 ms
            // cheaper at d = 4096; the plain BF16 and per-tensor FP8 scorers
            // ran slower that way)
            v[i] = ((MODE == kFP8Row || EPI == kEpiSoftmaxZ || DIV) && NW == 8) ? acc[b][j][i]
                                                                                : acc_read(acc[b][j][i]);
            if constexpr (MODE == kFP8Row) v[i] *= rs[i];
          }
          if constexpr (EPI == kEpiSoftmaxZ) {
            // the logits z = acc * scale (natural units) of the block, as the
            // lane holds them (64 contiguous bytes)
            // (the lane's offset passes through an opaque move, else the
            // offsets of all blocks are formed once and held across the loop)
            int zo = (int)zbuf_index(0, 0, 0, wv * 4 + b, wt * JT + j, lane);
            asm volatile("v_mov_b32 %0, %0" : "+v"(zo));
            float* zr = p.zbuf + zbuf_index(tt, p.n_vtiles, tile, 0, 0, 0) + zo;
#pragma unroll
            for (int qq = 0; qq < 4; ++qq)
              __builtin_nontemporal_store(  // streamed: read back once, by the pi pass
                  f32x4{v[4 * qq] * cz[j], v[4 * qq + 1] * cz[j], v[4 * qq + 2] * cz[j], v[4 * qq + 3] * cz[j]},
                  reinterpret_cast<f32x4*>(zr + kZRun * qq));
          }
          float mx[8];
#pragma unroll
          for (int i = 0; i < 8; ++i) mx[i] = fmaxf(v[2 * i], v[2 * i + 1]);
#pragma unroll
          for (int w = 4; w >= 1; w >>= 1)
#pragma unroll
            for (int i = 0; i < w; ++i) mx[i] = fmaxf(mx[i], mx[i + w]);
          const float Mn = fmaxf(M[j], mx[0] * c2[j]);
          const float dM = M[j] - Mn;
          const float al = fast_exp2(dM);
          U[j] = al * fmaf(dM, S[j], U[j]);
          S[j] *= al;
          M[j] = Mn;
          const float nM = -Mn;
          // exponentials and sums in two halves of H = 8 values (fewer live
          // registers than all 16 at once).  Every variant sums in this same
          // order, so pi and mu give bitwise equal statistics on equal logits.
          constexpr int H = 8;
          float sh[16 / H], uh[16 / H];
#pragma unroll
          for (int h0 = 0; h0 < 16; h0 += H) {
            float t[H], e[H];
#pragma unroll
            for (int i = 0; i < H; ++i) t[i] = fmaf(v[h0 + i], c2[j], nM);
#pragma unroll
            for (int i = 0; i < H; ++i) e[i] = fast_exp2(t[i]);
            if constexpr (kTail) {
#pragma unroll
              for (int i = 0; i < H; ++i) e[i] *= fminf(fmaxf(nv - (float)(16 * b + h0 + i), 0.0f), 1.0f);
            }
            float s8[H / 2], u8[H / 2];
#pragma unroll
            for (int i = 0; i < H / 2; ++i) {
              s8[i] = e[2 * i] + e[2 * i + 1];
              u8[i] = fmaf(e[2 * i + 1], t[2 * i + 1], e[2 * i] * t[2 * i]);
            }
#pragma unroll
            for (int w = H / 4; w >= 1; w >>= 1)
#pragma unroll
              for (int i = 0; i < w; ++i) {
                s8[i] += s8[i + w];
                u8[i] += u8[i + w];
              }
            sh[h0 / H] = s8[0];
            uh[h0 / H] = u8[0];
          }
          if constexpr (H == 8) {
            sh[0] += sh[1];
            uh[0] += uh[1];
          }
          S[j] += sh[0];
          U[j] += uh[0];
          // finish the update here, ahead of the branch below: otherwise the
          // pass is sunk past it and the values of all 16 blocks stay live
          asm volatile("" : "+v"(M[j]), "+v"(S[j]), "+v"(U[j]));
          if constexpr (SAMPLE) {
            // Blockwise Gumbel-max.  The lane's 16 rows v0 + 32b + 8q + 4g + jj
            // (in increasing order) are one block k = 2 (v0 + 32b) / 32 + g
            // of the draw: its key is the block's log-sum-exp plus one
            // Gumbel, lse2 - log2(-log2 u) in log2 units (a monotone map of
            // lse - ln(-ln u)), lse2 = M + log2 of the block's share of S
            // (sh[0], relative to the running maximum M just set).  Only a
            // block that beats the lane's best so far draws its row: inverse
            // CDF of the block's softmax with the second uniform.  Uniforms:
            // Philox on counter ((v0 + 32b) / 64, token, g, 0), words 2e and
            // 2e + 1 for e = b mod 2, so one call serves the blocks of b and
            // b + 1 (the second pair is kept in pw).
            const uint32_t tokg = (uint32_t)(p.row_offset + tok[j]);
            uint32_t wk, wp;
            if (b % 2 == 0) {
              uint32_t w4[4];
              philox4x32_10((uint32_t)(v0 + 32 * b) >> 6, tokg, (uint32_t)g, 0u, p.seed_lo, p.seed_hi, w4);
              wk = w4[0];
              wp = w4[1];
              pw[j][0] = w4[2];
              pw[j][1] = w4[3];
            } else {
              wk = pw[j][0];
              wp = pw[j][1];
            }
            const float u = ((float)(wk >> 9) + 0.5f) * 0x1p-23f;
            const float key = M[j] + __builtin_amdgcn_logf(sh[0]) - __builtin_amdgcn_logf(-__builtin_amdgcn_logf(u));
            if (key > bk[j]) {
              // the block's row: the first whose cumulative weight exceeds
              // u' times the block's total (in row order), else its last row
              // of nonzero weight; weights 2^(y - M) as in the sums above
              const float up = ((float)(wp >> 9) + 0.5f) * 0x1p-23f;
              // two passes over the weights (recomputed: fewer live registers)
              auto weight = [&](int i) {
                float e = fast_exp2(fmaf(v[i], c2[j], -M[j]));
                if constexpr (kTail) e *= fminf(fmaxf(nv - (float)(16 * b + i), 0.0f), 1.0f);
                return e;
              };
              float tot = 0.0f;
#pragma unroll
              for (int i = 0; i < 16; ++i) tot += weight(i);
              const float target = up * tot;
              float c = 0.0f, zsel = 0.0f, zlast = 0.0f;
              int isel = -1, ilast = 0;
#pragma unroll
              for (int i = 0; i < 16; ++i) {
                const float ei = weight(i);
                c += ei;
                const bool hit = isel < 0 && c > target;
                isel = hit ? i : isel;
                zsel = hit ? v[i] : zsel;
                const bool pos = ei > 0.0f;
                ilast = pos ? i : ilast;
                zlast = pos ? v[i] : zlast;
              }
              if (isel < 0) {
                isel = ilast;
                zsel = zlast;
              }
              bk[j] = key;
              bz[j] = zsel * cz[j];
              bi[j] = v0 + 32 * b + 8 * (isel >> 2) + 4 * g + (isel & 3);
            }
          }
          // the sampled token a_t: rare branch, taken by the one lane holding it
          const int rel = id[j] - v0;
          if ((unsigned)rel < 128u && (rel >> 5) == b && ((rel >> 2) & 1) == g) {
            float fi = (float)(((rel & 31) >> 3) * 4 + (rel & 3));
            asm volatile("v_mov_b32 %0, %0" : "+v"(fi));  // keep the weights inside the branch
            float z = 0.0f;
#pragma unroll
            for (int i = 0; i < 16; ++i) z = fmaf(fmaxf(1.0f - fabsf(fi - (float)i), 0.0f), v[i], z);
            if (tok[j] < p.n_rows && id[j] < p.V) p.logit[tok[j]] = z * cz[j];
          }
          if constexpr (DIV) {
            // no contraction in this block: z = acc * c must be rounded as
            // mu's pass rounds the logits it stores (an fma of z - zq would
            // leave the product's rounding error where equal logits need 0)
#pragma clang fp contract(off)
            // Full-vocabulary measures against mu's logits zq and mu's final
            // lse A_q: with pt = exp(z - A_q) and q = exp(zq - A_q) (so that
            // p = pt exp(A_q - A_p)), the sums of pt (z - zq), q (zq - z),
            // (pt - q)^2, (pt - q) pt and pt^2 over the vocabulary give both
            // KL divergences and |p - q|_2 exactly once A_p is known
            // (div_finalize_kernel).  No running maximum enters, so the sums
            // need no rescaling; pt and q come from one formula, so equal
            // logits give pt == q bit for bit.  The logits are read out of
            // the accumulators again, four at a time (fewer live registers
            // than keeping the 16 of the softmax pass).  mu's logits of the
            // same 16 entries were stored by mu's pass.
            // (the lane offset passes through an opaque move here, so that the
            // loads are issued at this point and not hoisted ahead of the
            // softmax pass, where their registers would be spilled)
            int zo = (int)zbuf_index(0, 0, 0, wv * 4 + b, wt * JT + j, lane);
            asm volatile("v_mov_b32 %0, %0" : "+v"(zo));
            const float* zr = p.zbuf + zbuf_index(tt, p.n_vtiles, tile, 0, 0, 0) + zo;
            float zq[16];
#pragma unroll
            for (int qq = 0; qq < 4; ++qq) {
              const f32x4 f = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(zr + kZRun * qq));
              zq[4 * qq] = f[0]; zq[4 * qq + 1] = f[1]; zq[4 * qq + 2] = f[2]; zq[4 * qq + 3] = f[3];
            }
            float k1 = 0.0f, k2 = 0.0f, la = 0.0f, lb = 0.0f, lc = 0.0f;
#pragma unroll
            for (int qq = 0; qq < 4; ++qq) {
#pragma unroll
              for (int ii = 0; ii < 4; ++ii) {
                const int i = 4 * qq + ii;
                const float zp = acc[b][j][i] * cz[j];  // (VGPR form, see above)
                float ep = fast_exp2(fmaf(zp, kLog2e, -a2[j]));
                float eq = fast_exp2(fmaf(zq[i], kLog2e, -a2[j]));
                if constexpr (kTail) {
                  const float wt1 = fminf(fmaxf(nv - (float)(16 * b + i), 0.0f), 1.0f);
                  ep *= wt1;
                  eq *= wt1;
                }
                const float dz = zp - zq[i], dd = ep - eq;
                k1 = fmaf(ep, dz, k1);
                k2 = fmaf(-eq, dz, k2);
                la = fmaf(dd, dd, la);
                lb = fmaf(dd, ep, lb);
                lc = fmaf(ep, ep, lc);
              }
              __builtin_amdgcn_sched_barrier(0);
            }
            dv[0][j] += k1;
            dv[1][j] += k2;
            dv[2][j] += la;
            dv[3][j] += lb;
            dv[4][j] += lc;
            // complete the sums here (else they are sunk to their use at the
            // end of the tile and the loaded values of every block stay live)
            asm volatile("" : "+v"(dv[0][j]), "+v"(dv[1][j]), "+v"(dv[2][j]), "+v"(dv[3][j]), "+v"(dv[4][j]));
          }
          __builtin_amdgcn_sched_barrier(0);
        }
      }
    };
    if (partial) run(std::true_type{});
    else run(std::false_type{});
    if constexpr (DIV) {
      // the tile's sums per token: lanes l and l ^ 32 (the two 4-row halves
      // of every 8 rows) add up, then one lane stores the wave's 128-row
      // share, slot 2 tile + wv of the pass row
      const int64_t plane = (int64_t)p.n_vtiles * 2 * p.dp_rows;
#pragma unroll
      for (int j = 0; j < JT; ++j) {
#pragma unroll
        for (int c = 0; c < 5; ++c) dv[c][j] += __shfl_xor(dv[c][j], 32);
        if (g == 0) {
          const int64_t o = (int64_t)(2 * tile + dv_slot) * p.dp_rows + tt * kTileT + dv_row + j * 32;
#pragma unroll
          for (int c = 0; c < 5; ++c) p.dpart[c * plane + o] = dv[c][j];
        }
      }
    }
    // stores must not count in the pipeline's waits
    if constexpr (EPI == kEpiSoftmaxZ || DIV) wait_vmcnt<0>();
  };

  // Backward (kEpiGrad): dZ[t, v] = coef_t (delta(v, a_t) - p_tv) / tau of the
  // finished tile, p = 2^(y - lse2) from the accumulators, rounded to bf16 and
  // stored into the two operand images of the gradient products: rows =
  // tokens (K = vocabulary) for dH = dZ W and rows = vocabulary (K = tokens)
  // for dW = dZ^T H, in the packed layout pack_kernel writes (16-byte column
  // c of row r at position c ^ ((r/4) % 4) of its 64-byte chunk row).  Rows
  // past V and tokens past n_rows or with coef 0 store 0 (the select also
  // drops a non-finite p of such a row).
  auto grad_epilogue = [&](int tile) {
    const int vw = tile * kTileV + wv * 128;  // first vocabulary row of this wave
    const bool odd = (lane & 1) != 0;
    auto pack2 = [](float lo, float hi) -> uint32_t {
      return (uint32_t)__builtin_bit_cast(uint16_t, (__bf16)lo) |
             ((uint32_t)__builtin_bit_cast(uint16_t, (__bf16)hi) << 16);
    };
#pragma unroll
    for (int b = 0; b < 4; ++b) {
#pragma unroll
      for (int j = 0; j < JT; ++j) {
        float dz[16];
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const int v = vw + 32 * b + 8 * (i >> 2) + 4 * g + (i & 3);
          const float pr = fast_exp2(fmaf(acc_read(acc[b][j][i]), c2[j], -gl2[j]));
          const float oh = v == id[j] ? 1.0f : 0.0f;
          dz[i] = (v < p.V && gc[j] != 0.0f) ? gc[j] * (oh - pr) : 0.0f;
        }
        // rows = tokens: the lane's token row, 4 consecutive vocabulary
        // values (8 bytes) per 16-byte column q
        {
          const int rr = wt * TW + 32 * j + r32;
          const int kc = tile * 8 + wv * 4 + b;
          uint8_t* row = p.gz_t + (((int64_t)tt * p.kch_v + kc) * kTileT + rr) * kChunk + 8 * g;
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const uint2 w2 = make_uint2(pack2(dz[4 * q], dz[4 * q + 1]), pack2(dz[4 * q + 2], dz[4 * q + 3]));
            *reinterpret_cast<uint2*>(row + ((q ^ ((rr >> 2) & 3)) << 4)) = w2;
          }
        }
        // rows = vocabulary: lanes 2m, 2m+1 hold tokens 2m, 2m+1 of one row;
        // after one exchange the even lane stores the pair of row i, the odd
        // lane the pair of row i+1 (4 bytes each)
        {
          const int kc = tt * 8 + wt * JT + j;
          uint8_t* img = p.gz_v + ((int64_t)tile * p.kch_t + kc) * kTileV * kChunk;
#pragma unroll
          for (int i = 0; i < 16; i += 2) {
            const float send = odd ? dz[i] : dz[i + 1];
            const float recv = __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(send), 0xB1, 0xF, 0xF, true));
            const uint32_t w1 = odd ? pack2(recv, dz[i + 1]) : pack2(dz[i], recv);
            const int row = wv * 128 + 32 * b + 8 * (i >> 2) + 4 * g + (i & 3) + (odd ? 1 : 0);
            *reinterpret_cast<uint32_t*>(img + row * kChunk + ((((r32 >> 3) ^ ((row >> 2) & 3))) << 4) +
                                         2 * (r32 & 6)) = w1;
          }
        }
      }
    }
    // The pipeline's waits count outstanding vector-memory operations; these
    // stores would count with the operand loads, so they drain here.
    wait_vmcnt<0>();
  };

  // Plain product (kEpiStore): C[m, n] = the tile (after the initial C when
  // accumulating); m = A row, n = B row; 32 lanes store 32 consecutive n.
  auto store_epilogue = [&](int tile) {
    const int m0 = tile * kTileV + wv * 128 + 4 * g;
#pragma unroll
    for (int b = 0; b < 4; ++b)
#pragma unroll
      for (int j = 0; j < JT; ++j)
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const int m = m0 + 32 * b + 8 * (i >> 2) + (i & 3);
          const float x = acc[b][j][i];  // (VGPR form: the 8-wave products)
          if (m < p.c_rows && tok[j] < p.n_rows) p.c[(int64_t)m * p.ldc + tok[j]] = x;
        }
  };

  // ---- the pipeline.  Chunks 0..NS-1 are requested up front, one per
  // stage.  Fragments are read L MFMA groups ahead of their use, so every LDS
  // read is covered by 4L MFMAs.  In chunk c the first read of chunk c+1
  // comes L groups before the end; just before it every wave waits for its
  // part of chunk c+1, the workgroup meets at the one barrier of the chunk
  // (after which no wave reads chunk c's stage any more) and chunk c+NS is
  // requested into that stage.  The steady-state chunk body is straight-line
  // code; the last NS chunks of a workgroup take a second copy that waits
  // for all loads and requests nothing.
  constexpr int L = (MODE == kBF16) ? 2 : 1;
  int qi = 0, kci = 0;  // tile and chunk of the next chunk to request
  auto advance_issue = [&]() {
    if (++kci == p.n_chunks) {
      kci = 0;
      ++qi;
    }
  };
#pragma unroll
  for (int c = 0; c < NS; ++c) {
    if (c < n_iter) {
      issue_chunk(qi, kci, c);
      advance_issue();
    }
  }
  if (n_iter < NS) wait_vmcnt<0>();
  else wait_vmcnt<(NS - 1) * LPC>();
  __syncthreads();

  // Fragments a chunk starts with (its first L groups' A, its first B step,
  // MX scales).  Two sets alternate between even and odd chunks (every tile
  // has an even number of chunks), so the next chunk's fragments are read
  // straight into the registers it will use.
  struct Frags {
    FragT a[L], b[JT];
    int sa, sb;  // MX: the chunk's scale dwords of the W and H rows
  };
  Frags f0, f1;
#pragma unroll
  for (int l = 0; l < L; ++l) f0.a[l] = read_a(0, l);
  read_b(0, 0, f0.b);
  f0.sa = f0.sb = f1.sa = f1.sb = 0;
  if constexpr (MODE == kMX) {
    f0.sa = read_sa(0);
    f0.sb = read_sb(0);
  }

  // LDS read instructions issued in group k (for group k + L)
  auto reads_at = [](int k) constexpr {
    const int t = k + L, tt = t % G;
    constexpr int per_frag = (MODE == kBF16) ? 1 : 2;
    int n = per_frag;                                                      // A
    if (tt % 4 == 0) n += JT * per_frag + (MODE == kMX && tt == 0 ? 2 : 0);  // B of a new step (+ MX scales)
    return n;
  };
  int stg = 0;  // stage of the current chunk
  // first_tag: the tile's first chunk, whose first K step starts the
  // accumulators from zero
  auto chunk = [&](auto steady_tag, auto first_tag, int it, Frags& cur, Frags& nxt) {
    constexpr bool kSteady = decltype(steady_tag)::value;
    constexpr bool kFirst = decltype(first_tag)::value;
    const bool has_next = kSteady || it + 1 < n_iter;
    const int nst = stg + 1 == NS ? 0 : stg + 1;
    FragT af[G];       // A of this chunk's groups
    FragT bf[2][JT];    // B of this chunk's K steps (BF16: 2, FP8: 1)
#pragma unroll
    for (int l = 0; l < L; ++l) af[l] = cur.a[l];
#pragma unroll
    for (int j = 0; j < JT; ++j) bf[0][j] = cur.b[j];
#pragma unroll
    for (int k = 0; k < G; ++k) {
      const int t = k + L;  // group whose fragments are read now
      if (t == G && has_next) {
        // chunk it+1 must have landed (chunks it+2 .. it+NS-1 may be in flight)
        if constexpr (kSteady) wait_loads_and_barrier<(NS - 2) * LPC>();
        else wait_loads_and_barrier<0>();
        if (kSteady || it + NS < n_iter) {
          issue_chunk(qi, kci, stg);
          advance_issue();
        }
      }
      if (t < G) {
        af[t] = read_a(stg, t);
        if (t % 4 == 0) read_b(stg, t, bf[t / 4]);  // BF16: second K step
      } else if (has_next) {
        nxt.a[t - G] = read_a(nst, t - G);
        if (t == G) {
          read_b(nst, 0, nxt.b);
          if constexpr (MODE == kMX) {
            nxt.sa = read_sa(nst);
            nxt.sb = read_sb(nst);
          }
        }
      }
      if (kFirst && k < 4) mfma_group(std::true_type{}, k, af[k], bf[k / 4], cur.sa, cur.sb);
      else mfma_group(std::false_type{}, k, af[k], bf[k / 4], cur.sa, cur.sb);
      if constexpr (kSteady) {
        // keep this group's LDS reads ahead of its MFMAs (the scheduler
        // would otherwise sink each read to just before its use)
        sched_ds_reads(reads_at(k));
        __builtin_amdgcn_sched_group_barrier(0x008, JT, 0);  // JT MFMAs
      }
    }
    stg = nst;
  };

  int it = 0;
  for (int q = 0; q < vt_end - vt_begin; ++q) {
    // steady chunks: [0, kc_steady); the rest request nothing new or only
    // while requests remain, and wait for every load
    const int kc_steady = min(p.n_chunks, max(0, n_iter - NS - it));
    int kc = 0;
    if constexpr (kZeroStart) {
    // the first pair (every tile has an even number >= 2 of chunks): its
    // first chunk starts the accumulators from an inline zero
    if (kc_steady >= 2) {
      chunk(std::true_type{}, std::true_type{}, it, f0, f1);
      chunk(std::true_type{}, std::false_type{}, it + 1, f1, f0);
    } else {
      chunk(std::false_type{}, std::true_type{}, it, f0, f1);
      chunk(std::false_type{}, std::false_type{}, it + 1, f1, f0);
    }
    kc = 2;
    it += 2;
    }
    for (; kc + 1 < kc_steady; kc += 2, it += 2) {
      chunk(std::true_type{}, std::false_type{}, it, f0, f1);
      chunk(std::true_type{}, std::false_type{}, it + 1, f1, f0);
    }
    for (; kc < p.n_chunks; kc += 2, it += 2) {
      chunk(std::false_type{}, std::false_type{}, it, f0, f1);
      chunk(std::false_type{}, std::false_type{}, it + 1, f1, f0);
    }
    if constexpr (SOFTMAX) epilogue(vt_begin + q, q);
    else if constexpr (EPI == kEpiGrad) grad_epilogue(vt_begin + q);
    else store_epilogue(vt_begin + q);
    if constexpr (!kZeroStart) {
#pragma unroll
      for (int b = 0; b < 4; ++b)
#pragma unroll
        for (int j = 0; j < JT; ++j) acc[b][j] = f32x16{};
    }
  }
  if constexpr (!SOFTMAX) return;
  __syncthreads();  // every wave is done with the stages before LDS is reused

  // ---- merge the lane pair (l, l^32), then the two vocabulary halves
  // (sampling: the larger key wins, the smaller row on a tie)
  auto take_best = [](float& k, float& z, int& i, float k2, float z2, int i2) {
    if (k2 > k || (k2 == k && i2 < i)) {
      k = k2;
      z = z2;
      i = i2;
    }
  };
#pragma unroll
  for (int j = 0; j < JT; ++j) {
    const float M2 = __shfl_xor(M[j], 32), S2 = __shfl_xor(S[j], 32), U2 = __shfl_xor(U[j], 32);
    merge_state(M[j], S[j], U[j], M2, S2, U2);
    if constexpr (SAMPLE) {
      const float k2 = __shfl_xor(bk[j], 32), z2 = __shfl_xor(bz[j], 32);
      const int i2 = __shfl_xor(bi[j], 32);
      take_best(bk[j], bz[j], bi[j], k2, z2, i2);
    }
  }
  constexpr int XS = SAMPLE ? 6 : 3;  // floats exchanged per token
  float* xch = reinterpret_cast<float*>(lds);  // LDS is free after the last barrier
  if (wv == 1 && g == 0) {
#pragma unroll
    for (int j = 0; j < JT; ++j) {
      const int k = wt * TW + j * 32 + r32;
      xch[XS * k + 0] = M[j];
      xch[XS * k + 1] = S[j];
      xch[XS * k + 2] = U[j];
      if constexpr (SAMPLE) {
        xch[XS * k + 3] = bk[j];
        xch[XS * k + 4] = bz[j];
        xch[XS * k + 5] = __int_as_float(bi[j]);
      }
    }
  }
  __syncthreads();
  if (wv == 0 && g == 0) {
    const int64_t plane = (int64_t)p.n_strips * p.n_rows;
#pragma unroll
    for (int j = 0; j < JT; ++j) {
      const int k = wt * TW + j * 32 + r32;
      merge_state(M[j], S[j], U[j], xch[XS * k + 0], xch[XS * k + 1], xch[XS * k + 2]);
      if constexpr (SAMPLE)
        take_best(bk[j], bz[j], bi[j], xch[XS * k + 3], xch[XS * k + 4], __float_as_int(xch[XS * k + 5]));
      if (tok[j] < p.n_rows) {
        const int64_t o = (int64_t)st * p.n_rows + tok[j];
        p.part[o] = M[j];
        p.part[plane + o] = S[j];
        p.part[2 * plane + o] = U[j];
        if constexpr (SAMPLE) {
          p.best_key[o] = bk[j];
          p.best_logit[o] = bz[j];
          p.best_id[o] = bi[j];
        }
      }
    }
  }
  };  // unit

  // ---- which units this workgroup runs.  Unit i of XCD x is the i-th
  // workgroup that XCD would get from a grid of one workgroup per unit
  // (workgroups go to the XCDs round robin): blocks of kBlockT token tiles x
  // kBlockS strips, so that an XCD's concurrent units share W and H chunks
  // in its L2.  Persistent: one workgroup per CU takes the next unit of its
  // own XCD's queue, and once that is empty the next of the other XCDs'
  // queues, so that XCDs that run faster take more units (a fixed share per
  // XCD leaves the faster ones idle at the end).  Every claim is one atomic
  // on the queue's counter; a workgroup exits once every queue is empty.
  constexpr int per = kBlockT * kBlockS;
  auto run_unit = [&](int x, int i) {
    const int blk = (i / per) * kXcds + x, k = i % per;
    unit((blk % p.n_tblocks) * kBlockT + k / kBlockS, (blk / p.n_tblocks) * kBlockS + k % kBlockS);
  };
  if constexpr (!PERSIST) {
    run_unit((int)(blockIdx.x % kXcds), (int)(blockIdx.x / kXcds));
  } else {
    // the XCD this workgroup runs on (XCC_ID hardware register, bits 3:0)
    const int xcc = (int)(__builtin_amdgcn_s_getreg((3 << 11) | 20) & (kXcds - 1));
    int* slot = reinterpret_cast<int*>(lds);  // the stages are free between units
    for (;;) {
      if (tid == 0) {
        int claim = -1;
        for (int a = 0; a < kXcds && claim < 0; ++a) {
          const int x = (xcc + a) & (kXcds - 1);
          const int t = atomicAdd(p.queue + kQueueStride * x, 1);
          if (t < p.units_per_xcd) claim = x * p.units_per_xcd + t;
        }
        *slot = claim;
      }
      __syncthreads();
      const int c = *slot;
      __syncthreads();  // every wave has its claim before the stages are written
      if (c < 0) break;
      const int x = c / p.units_per_xcd;
      run_unit(x, c - x * p.units_per_xcd);
      __syncthreads();  // the unit's last LDS reads are done
    }
  }
}

__global__ void clear_queue_kernel(int* q) { q[kQueueStride * threadIdx.x] = 0; }

// Waves per workgroup of each instantiation (measured on the MI355X): two
// per SIMD where the variant runs faster that way (the per-row FP8 scorer,
// the measures' passes and the backward's plain products hold their
// accumulators in VGPRs there); one per SIMD otherwise.  The blockwise
// sampling variants fit their registers at 4 waves (no spills) and run as
// fast or faster there than at 8 (q8b 85.2 vs 85.4 ms, q17b 27.0 vs
// 30.6 ms), where they spill around the epilogue; the dZ pass spills at 8.
template <int MODE, int EPI>
constexpr int waves_for() {
  return ((EPI == kEpiSoftmax && (MODE == kBF16 || MODE == kFP8Tensor || MODE == kFP8Row)) ||
          (EPI == kEpiSoftmaxZ && (MODE == kFP8Tensor || MODE == kFP8Row)) ||
          (EPI == kEpiSoftmaxDiv && MODE == kBF16) || EPI == kEpiStore)
             ? 8
             : 4;
}

// Scoring launches: `grid` units (a multiple of kXcds).  The softmax
// epilogues run persistent, one workgroup per CU (measured on the MI355X,
// against one workgroup per unit, results bitwise equal: pi 5 % faster at
// d = 4096 and 5120, 3 % at d = 2048; per-tensor FP8 mu 2.5 %, MX 1 %,
// per-row FP8 mu 6 % at d = 2048 and 1.5 % at d = 4096), except the per-row
// FP8 pass that stores its logits (the unit loop spills it to 104 bytes per
// lane, and the measures call ran no faster).  p.queue must point at
// kXcds * kQueueStride ints of workspace, cleared here.  The backward's
// plain products run persistent too (8 waves, VGPR accumulators: the q8b
// backward 502 -> 490 ms, of which ~1 ms from the persistent grid); its dZ
// pass takes one workgroup per unit (no faster persistent).
inline int device_cus() {
  int dev = 0, n = 0;
  if (hipGetDevice(&dev) != hipSuccess || hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
      n <= 0)
    n = 256;
  return n;
}

template <int MODE, int EPI>
void launch_score_kernel(unsigned grid, const ScoreParams& p, hipStream_t s) {
  constexpr int NW = waves_for<MODE, EPI>();
  constexpr bool kPersist = (EPI == kEpiSoftmax || EPI == kEpiSample || EPI == kEpiSoftmaxZ || EPI == kEpiSoftmaxDiv ||
                             EPI == kEpiStore) &&
                            !(MODE == kFP8Row && EPI == kEpiSoftmaxZ);
  if constexpr (kPersist) {
    ScoreParams q = p;
    q.units_per_xcd = (int)(grid / kXcds);
    hipLaunchKernelGGL(clear_queue_kernel, dim3(1), dim3(kXcds), 0, s, q.queue);
    const unsigned wgs = std::min<unsigned>(grid, (unsigned)device_cus());
    hipLaunchKernelGGL((score_kernel<MODE, EPI, NW, true>), dim3(wgs), dim3(NW * 64), 0, s, q);
  } else {
    hipLaunchKernelGGL((score_kernel<MODE, EPI, NW, false>), dim3(grid), dim3(NW * 64), 0, s, p);
  }
}

// Packed operand image read by score_kernel: for each 256-row tile and each
// 64-byte chunk of the rows, one 16 KiB block holding the tile's 256 row
// pieces in row order, the four 16-byte columns of row r permuted to
// positions c ^ ((r/4) % 4).  Rows past `rows` repeat the last row.  One
// thread per 16 bytes; eight consecutive threads move one 128-byte line of a
// source row (chunks 2p, 2p+1), so a wavefront reads 8 whole lines of 8
// consecutive rows and writes two contiguous 512-byte runs (row_bytes is a
// multiple of 128).  `units` = n_tiles * 256 * (row_bytes / 16) < 2^32.
__global__ __launch_bounds__(256) void pack_kernel(const uint8_t* __restrict__ src, uint32_t rows,
                                                   uint32_t row_bytes, uint32_t units, uint8_t* __restrict__ dst) {
  const uint32_t n_chunks = row_bytes / kChunk;
  const uint32_t n_pairs = n_chunks / 2;
  for (uint32_t u = blockIdx.x * blockDim.x + threadIdx.x; u < units; u += gridDim.x * blockDim.x) {
    const uint32_t c16 = u & 7, rest = u >> 3;
    const uint32_t rr = rest % kTileV, tp = rest / kTileV;  // tp = tile * n_pairs + pair
    const uint32_t tile = tp / n_pairs, pr = tp - tile * n_pairs;
    const uint32_t piece = pr * 8 + c16;  // 16-byte piece of the source row
    const uint32_t kc = piece >> 2, c = piece & 3;
    const uint32_t row = tile * kTileV + rr;
    const uint32_t pos = c ^ ((rr >> 2) & 3);
    const uint32_t sr = row < rows ? row : rows - 1;
    const uint4 v = *reinterpret_cast<const uint4*>(src + (size_t)sr * row_bytes + piece * 16);
    *reinterpret_cast<uint4*>(dst + ((size_t)(tile * n_chunks + kc) * kTileV + rr) * kChunk + pos * 16) = v;
  }
}

// Packed MX scale image read by score_kernel: for each 256-row tile and each
// 64-byte chunk kc, 128 dwords holding the E8M0 scales of MX blocks 2kc,
// 2kc+1 of the tile's 256 rows (512 bytes).  Dword (h, g, r) = (2h + g) * 32
// + r carries block 2kc + g of rows 128h + 32b + r in its bytes b = 0..3: the
// dword one lane of a 128-row wave half needs for its four 32-row blocks.
// Rows past `rows` repeat the last row.  One thread per dword; `units` =
// n_tiles * n_chunks * 128 < 2^32.
__global__ __launch_bounds__(256) void pack_mx_kernel(const uint8_t* __restrict__ src, uint32_t rows,
                                                      uint32_t n_chunks, uint32_t units, uint32_t* __restrict__ dst) {
  const uint32_t row_bytes = 2 * n_chunks;  // d / 32 scale bytes per row
  for (uint32_t u = blockIdx.x * blockDim.x + threadIdx.x; u < units; u += gridDim.x * blockDim.x) {
    const uint32_t r = u & 31, g = (u >> 5) & 1, h = (u >> 6) & 1, tc = u >> 7;  // tc = tile * n_chunks + kc
    const uint32_t tile = tc / n_chunks, kc = tc - tile * n_chunks;
    uint32_t word = 0;
#pragma unroll
    for (uint32_t b = 0; b < 4; ++b) {
      const uint32_t row = tile * kTileV + h * 128 + b * 32 + r;
      const uint32_t sr = row < rows ? row : rows - 1;
      word |= (uint32_t)src[(size_t)sr * row_bytes + 2 * kc + g] << (8 * b);
    }
    dst[u] = word;
  }
}

inline void launch_pack_mx(const void* scales, int64_t rows, int64_t d, int64_t n_tiles, uint8_t* dst,
                           hipStream_t s) {
  const int64_t n_chunks = d / kChunk;  // a row holds d / 32 scale bytes = 2 per chunk
  const int64_t units = n_tiles * n_chunks * 128;  // one dword per 4 rows and MX block
  const unsigned blocks = (unsigned)std::min<int64_t>((units + 255) / 256, 8192);
  hipLaunchKernelGGL(pack_mx_kernel, dim3(blocks), dim3(256), 0, s, static_cast<const uint8_t*>(scales),
                     (uint32_t)rows, (uint32_t)n_chunks, (uint32_t)units, reinterpret_cast<uint32_t*>(dst));
}

// Transposed packed image: the rows of the image are the COLUMNS k of
// x [rows, cols] (bf16) and its K dimension runs along x's rows, in the
// layout pack_kernel writes (one 16 KiB block per (256-column tile, 32-row
// chunk); 16-byte column c of image row k at position c ^ ((k/4) % 4)).
// Rows of x past `rows` and columns past `cols` read as 0.  One workgroup
// per block: thread t builds image row k = 256 tile + t from 32 loads that
// the workgroup issues as coalesced 512-byte row segments.
__global__ __launch_bounds__(256) void pack_t_kernel(const uint16_t* __restrict__ x, int64_t rows, int64_t cols,
                                                     int n_rchunks, uint8_t* __restrict__ dst) {
  const int64_t blk = blockIdx.x;
  const int64_t ktile = blk / n_rchunks, rc = blk % n_rchunks;
  const int t = threadIdx.x;
  const int64_t k = ktile * kTileV + t;
  uint32_t w[16];
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    uint32_t lohi[2];
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int64_t r = rc * 32 + 2 * i + h;
      lohi[h] = (r < rows && k < cols) ? (uint32_t)x[r * cols + k] : 0u;
    }
    w[i] = lohi[0] | (lohi[1] << 16);
  }
  uint8_t* row = dst + (blk * kTileV + t) * kChunk;
#pragma unroll
  for (int c = 0; c < 4; ++c)
    *reinterpret_cast<uint4*>(row + ((c ^ ((t >> 2) & 3)) << 4)) =
        make_uint4(w[4 * c], w[4 * c + 1], w[4 * c + 2], w[4 * c + 3]);
}

__global__ __launch_bounds__(256) void fill_zero_kernel(float* __restrict__ p, int64_t n) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
    p[i] = 0.0f;
}

// lse of row r in log2 units (M + log2 S) from the strips' (M, S, U) states.
__device__ __forceinline__ float merged_lse2(const float* part, int64_t plane, int n_strips, int n_rows, int r) {
  float M = kInitMax, S = 0.f, U = 0.f;
  for (int s = 0; s < n_strips; ++s) {
    const int64_t o = (int64_t)s * n_rows + r;
    merge_state(M, S, U, part[o], part[plane + o], part[2 * plane + o]);
  }
  return M + log2f(S);
}

// mu's log-sum-exp (log2 units) of rows r0 .. r0 + rows - 1 for the pi pass
// of the full-vocabulary measures; entries rows .. cap - 1 (token-tile
// padding) get 0.
__global__ __launch_bounds__(256) void lse2_kernel(const float* __restrict__ part, int n_strips, int n_rows, int r0,
                                                   int rows, int cap, float* __restrict__ out) {
  const int k = blockIdx.x * blockDim.x + threadIdx.x;
  if (k >= cap) return;
  out[k] = k < rows ? merged_lse2(part, (int64_t)n_strips * n_rows, n_strips, n_rows, r0 + k) : 0.0f;
}

struct DivParams {
  int n_rows;              // rows of the whole call
  int n_strips;
  int r0;                  // first row of this pass
  int rows;                // rows of this pass
  int n_parts;             // partial sums per row: 2 per vocabulary tile
  int64_t dp_rows;         // row stride of dpart's planes
  const float* part_pi;    // pi's (M, S, U) strip states
  const float* aq2;        // mu's lse of the pass rows (log2 units)
  const float* dpart;      // [5][n_parts][dp_rows] sums per 128 vocabulary rows
  const uint8_t* mask;
  const int32_t* out_slot;
  float* kl_pm;            // [slots] KL(pi || mu), nullable
  float* kl_mp;            // [slots] KL(mu || pi), nullable
  float* l2;               // [slots] Euclidean distance, nullable
};

// The measures of the pass rows from the pi kernel's sums (one per 128
// vocabulary rows), taken against mu's lse A_q.  A workgroup takes 32 rows;
// its 8 thread groups add the parts s = g, g + 8, ... of each row, and one
// thread per row adds the 8 group sums in order.  With D = A_p - A_q (nats)
// and r = exp(-D), so that p = r pt:
//   KL(pi||mu) = sum p ((z - zq) - D) = r sum pt (z - zq) - D,
//   KL(mu||pi) = sum q ((zq - z) + D) = sum q (zq - z) + D,
//   |p - q|^2  = sum ((pt - q) + (r - 1) pt)^2
//              = sum (pt - q)^2 + 2 (r - 1) sum (pt - q) pt + (r - 1)^2 sum pt^2,
// using sum p = sum q = 1.  Every term is small for nearby policies, so no
// large quantities cancel.  pt = exp(z - A_q) <= exp(D) and pt^2 are formed
// in fp32: rows with |D| > 32 nats (where they could overflow) get NaN.  The
// three terms of |p - q|^2 can cancel: for peaked distributions whose top
// logits differ (D != 0 while p ~ q), and by ~exp(2D) when pi's lse is far
// above mu's (r << 1).  The terms are rounded to fp32 per entry and their
// parts added in fp64 here, so the error of the result is about 3e-7 times
// the sum of their magnitudes: the distance is NaN where that exceeds 1 % of
// |p - q|^2 plus 1e-8 (an error above ~1e-4 on the distance).
constexpr int kFinRows = 32, kFinGroups = 8;
__global__ __launch_bounds__(kFinRows * kFinGroups) void div_finalize_kernel(DivParams p) {
  __shared__ double part_sums[5][kFinGroups][kFinRows];
  const int rl = threadIdx.x % kFinRows, grp = threadIdx.x / kFinRows;
  const int k = blockIdx.x * kFinRows + rl;
  const bool in = k < p.rows;
  const int r = p.r0 + (in ? k : 0);
  const bool active = in && (p.mask ? p.mask[r] != 0 : true);
  double sum[5] = {0.0, 0.0, 0.0, 0.0, 0.0};  // the parts add up in fp64
  if (active) {
    const int64_t plane = (int64_t)p.n_parts * p.dp_rows;
    for (int s = grp; s < p.n_parts; s += kFinGroups)
#pragma unroll
      for (int c = 0; c < 5; ++c) sum[c] += (double)p.dpart[c * plane + (int64_t)s * p.dp_rows + k];
  }
#pragma unroll
  for (int c = 0; c < 5; ++c) part_sums[c][grp][rl] = sum[c];
  __syncthreads();
  if (grp != 0 || !in) return;
  float kpm = 0.f, kmp = 0.f, l2 = 0.f;
  if (active) {
#pragma unroll
    for (int c = 0; c < 5; ++c) {
      sum[c] = part_sums[c][0][rl];
      for (int g2 = 1; g2 < kFinGroups; ++g2) sum[c] += part_sums[c][g2][rl];
    }
    const float ap = merged_lse2(p.part_pi, (int64_t)p.n_strips * p.n_rows, p.n_strips, p.n_rows, r);
    const double D = ((double)ap - (double)p.aq2[k]) * (double)kLn2;
    // (infinite logits leave non-finite sums)
    bool finite = true;
#pragma unroll
    for (int c = 0; c < 5; ++c) finite = finite && isfinite(sum[c]);
    if (fabs(D) <= 32.0 && finite) {
      const double rm1 = expm1(-D);
      kpm = (float)(fma(rm1, sum[0], sum[0]) - D);
      kmp = (float)(sum[1] + D);
      const double l2sq = sum[2] + rm1 * (2.0 * sum[3] + rm1 * sum[4]);
      const double mag = sum[2] + fabs(2.0 * rm1 * sum[3]) + rm1 * rm1 * sum[4];
      l2 = 3e-7 * mag <= 1e-2 * l2sq + 1e-8 ? (float)sqrt(fmax(l2sq, 0.0)) : __builtin_nanf("");
    } else {
      kpm = kmp = l2 = __builtin_nanf("");
    }
  }
  const int slot = p.out_slot ? p.out_slot[r] : r;
  if (p.kl_pm) p.kl_pm[slot] = kpm;
  if (p.kl_mp) p.kl_mp[slot] = kmp;
  if (p.l2) p.l2[slot] = l2;
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
  int q_begin, q_end;      // policies merged: [q_begin, q_end) of {pi, mu}
};

// One thread per row: combine the strips' states of pi and / or mu.
__global__ __launch_bounds__(256) void merge_kernel(MergeParams p) {
  const int r = blockIdx.x * blockDim.x + threadIdx.x;
  if (r >= p.n_rows) return;
  const int slot = p.out_slot ? p.out_slot[r] : r;
  const bool active = p.mask ? p.mask[r] != 0 : true;
  const int id = p.ids[r];
  const bool id_ok = id >= 0 && id < p.V;
  if (active && !id_ok && p.error_flag) atomicOr(p.error_flag, 1);
  const int64_t plane = (int64_t)p.n_strips * p.n_rows;
  for (int q = p.q_begin; q < p.q_end; ++q) {
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

struct SampleMergeParams {
  int n_rows;
  int n_strips;
  const float* part;
  const float* best_key;
  const float* best_logit;
  const int32_t* best_id;
  int32_t* ids;
  float* logp;
};

// One thread per row: the sampled row is the strips' best Gumbel key (the
// smaller row on a tie); its log-probability is its logit minus the merged
// log-sum-exp.
__global__ __launch_bounds__(256) void sample_merge_kernel(SampleMergeParams p) {
  const int r = blockIdx.x * blockDim.x + threadIdx.x;
  if (r >= p.n_rows) return;
  const int64_t plane = (int64_t)p.n_strips * p.n_rows;
  float M = kInitMax, S = 0.f, U = 0.f;
  float bk = -INFINITY, bz = 0.f;
  int bi = 0;
  for (int s = 0; s < p.n_strips; ++s) {
    const int64_t o = (int64_t)s * p.n_rows + r;
    merge_state(M, S, U, p.part[o], p.part[plane + o], p.part[2 * plane + o]);
    const float k = p.best_key[o];
    const int i = p.best_id[o];
    if (k > bk || (k == bk && i < bi)) {
      bk = k;
      bz = p.best_logit[o];
      bi = i;
    }
  }
  p.ids[r] = bi;
  if (p.logp) p.logp[r] = bz - (M + log2f(S)) * kLn2;
}

inline size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

}  // namespace

PackedWeightsLayout packed_weights_layout(int64_t V, int64_t d, int mu_scaling) {
  PackedWeightsLayout l{};
  const size_t vrows = (size_t)((V + kTileV - 1) / kTileV) * kTileV;
  l.w_offset = 0;
  l.wq_offset = align_up(vrows * 2 * (size_t)d, 256);
  l.mx_offset = l.wq_offset + align_up(vrows * (size_t)d, 256);
  l.bytes = l.mx_offset + (mu_scaling == ACRL_SCALE_MX32 ? align_up(vrows * (size_t)(d / 32), 256) : 0);
  return l;
}

hipError_t launch_pack_weights(const void* w, const void* wq, const void* wq_scales, int64_t V, int64_t d,
                               int mu_scaling, void* packed, hipStream_t s) {
  const PackedWeightsLayout l = packed_weights_layout(V, d, mu_scaling);
  uint8_t* dst = static_cast<uint8_t*>(packed);
  const int64_t n_vtiles = (V + kTileV - 1) / kTileV;
  const void* srcs[2] = {w, wq};
  const size_t offs[2] = {l.w_offset, l.wq_offset};
  for (int q = 0; q < 2; ++q) {
    const int64_t row_bytes = q == 0 ? 2 * d : d;
    const int64_t units = n_vtiles * kTileV * (row_bytes / 16);
    const unsigned blocks = (unsigned)std::min<int64_t>((units + 255) / 256, 8192);
    hipLaunchKernelGGL(pack_kernel, dim3(blocks), dim3(256), 0, s, static_cast<const uint8_t*>(srcs[q]),
                       (uint32_t)V, (uint32_t)row_bytes, (uint32_t)units, dst + offs[q]);
  }
  if (mu_scaling == ACRL_SCALE_MX32) launch_pack_mx(wq_scales, V, d, n_vtiles, dst + l.mx_offset, s);
  return hipGetLastError();
}

ScorePlan plan_score(int64_t n_rows, int64_t d, int64_t V, int64_t div_rows, bool prepacked) {
  ScorePlan pl{};
  pl.n_ttiles = (int)((n_rows + kTileT - 1) / kTileT);
  pl.n_vtiles = (int)((V + kTileV - 1) / kTileV);
  pl.n_tblocks = (pl.n_ttiles + kBlockT - 1) / kBlockT;
  // Strips: a multiple of kBlockS (or every tile its own strip when there
  // are fewer tiles), at most kMaxTilesPerStrip tiles each.  One workgroup
  // per CU (256 CUs): minimise the makespan ceil(grid / 256) *
  // (tiles-per-strip + 1/2), the half tile standing for a workgroup's fixed
  // cost (prologue, state merge, partial writes); ties -> fewer strips.  The
  // cap bounds a workgroup's duration: workgroup times differ by up to ~7 %
  // between XCDs and CUs, and the last workgroups of a CU end spread over
  // about one workgroup time (measured on the MI355X: 75-tile strips at
  // d = 4096 take ~8 ms and left ~4 % of the CU time idle; 15-19-tile
  // strips ran the pi and mu kernels 2-3 % faster).
  constexpr int kMaxTilesPerStrip = 20;
  const int64_t cus = 256;
  int best_s = 0;
  int64_t best_cost = -1;
  auto consider = [&](int s) {
    const int tps = (pl.n_vtiles + s - 1) / s;
    if (tps > kMaxTilesPerStrip) return;  // always reachable: s = n_vtiles gives 1 or 2
    const int strips = (pl.n_vtiles + tps - 1) / tps;
    const int sblocks = (strips + kBlockS - 1) / kBlockS;
    int blocks = pl.n_tblocks * sblocks;
    blocks = (blocks + kXcds - 1) / kXcds * kXcds;
    const int64_t grid = (int64_t)blocks * kBlockT * kBlockS;
    const int64_t cost = ((grid + cus - 1) / cus) * (2 * tps + 1);
    if (best_cost < 0 || cost < best_cost) {
      best_cost = cost;
      best_s = strips;
    }
  };
  if (pl.n_vtiles <= kBlockS) consider(pl.n_vtiles);
  for (int s = kBlockS; s <= pl.n_vtiles; s += kBlockS) consider(s);
  pl.tiles_per_strip = (pl.n_vtiles + best_s - 1) / best_s;
  pl.n_strips = (pl.n_vtiles + pl.tiles_per_strip - 1) / pl.tiles_per_strip;
  pl.n_sblocks = (pl.n_strips + kBlockS - 1) / kBlockS;
  pl.n_blocks_pad = (pl.n_tblocks * pl.n_sblocks + kXcds - 1) / kXcds * kXcds;
  pl.grid = pl.n_blocks_pad * kBlockT * kBlockS;
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
  // sampling: the strips' best Gumbel key, its logit and row
  pl.ws_best_offset = off;
  off += 3 * align_up((size_t)pl.n_strips * (size_t)n_rows * sizeof(float), 256);
  // packed operands: W, H (2d bytes per row), Wq, Hq (d bytes per row);
  // the weight images (W, Wq and Wq's MX scales) only when they do not come
  // prepacked by the caller
  const size_t vrows = (size_t)pl.n_vtiles * kTileV, trows = (size_t)pl.n_ttiles * kTileT;
  const size_t pack_bytes[4] = {vrows * 2 * (size_t)d, trows * 2 * (size_t)d, vrows * (size_t)d, trows * (size_t)d};
  for (int q = 0; q < 4; ++q) {
    pl.ws_pack_offset[q] = off;
    if (!(prepacked && (q == 0 || q == 2))) off += align_up(pack_bytes[q], 256);
  }
  // MX: packed E8M0 scale images of Wq and Hq (d/32 bytes per row)
  const size_t mx_bytes[2] = {vrows * (size_t)(d / 32), trows * (size_t)(d / 32)};
  for (int q = 0; q < 2; ++q) {
    pl.ws_mx_offset[q] = off;
    if (!(prepacked && q == 0)) off += align_up(mx_bytes[q], 256);
  }
  // full-vocabulary measures, per pass of div_tiles token tiles: mu's
  // logits (256 KiB per pair of token and vocabulary tiles), mu's lse of the
  // pass rows and pi's five sums per row and 128 vocabulary rows.  The
  // passes needed at div_rows rows each share the token tiles evenly, so
  // that no short last pass runs a grid of a few units per CU.
  pl.div_tiles = 0;
  if (div_rows > 0) {
    const int64_t req = std::max<int64_t>((div_rows + kTileT - 1) / kTileT, 1);
    const int64_t tiles = std::max<int64_t>(pl.n_ttiles, 1);
    const int64_t passes = (tiles + req - 1) / req;
    pl.div_tiles = (int)((tiles + passes - 1) / passes);
    const size_t prow = (size_t)pl.div_tiles * kTileT;
    pl.ws_zbuf_offset = off;
    off += prow * pl.n_vtiles * kTileV * sizeof(float);
    pl.ws_aq_offset = off;
    off += align_up(prow * sizeof(float), 256);
    pl.ws_dpart_offset = off;
    off += align_up((size_t)5 * 2 * pl.n_vtiles * prow * sizeof(float), 256);
  }
  // the persistent grid's per-XCD claim counters (cleared before each launch)
  pl.ws_queue_offset = off;
  off += align_up((size_t)kXcds * kQueueStride * sizeof(int), 256);
  pl.ws_bytes = off;
  return pl;
}

hipError_t launch_score(const acrl_score_desc& dsc, const ScorePlan& pl, hipStream_t s) {
  if (dsc.n_rows == 0) return hipSuccess;
  uint8_t* ws = static_cast<uint8_t*>(dsc.workspace);
  const unsigned grid = (unsigned)pl.grid;

  ScoreParams pp{};
  pp.V = (int)dsc.V;
  pp.n_rows = (int)dsc.n_rows;
  pp.n_vtiles = pl.n_vtiles;
  pp.tiles_per_strip = pl.tiles_per_strip;
  pp.n_strips = pl.n_strips;
  pp.n_ttiles = pl.n_ttiles;
  pp.n_tblocks = pl.n_tblocks;
  pp.inv_temp = dsc.inv_temperature;
  pp.ids = dsc.token_ids;
  pp.mx_row_bytes = (int)(dsc.d / 32);
  pp.queue = reinterpret_cast<int*>(ws + pl.ws_queue_offset);

  const bool do_pi = dsc.policies != ACRL_POLICY_MU;
  const bool do_mu = dsc.policies != ACRL_POLICY_PI;
  const uint8_t* pw = static_cast<const uint8_t*>(dsc.packed_weights);
  const PackedWeightsLayout pwl = packed_weights_layout(dsc.V, dsc.d, dsc.mu_scaling);

  // operands -> packed images in the workspace (the weight images only when
  // the caller did not pass them prepacked)
  const void* srcs[4] = {dsc.w, dsc.h, dsc.wq, dsc.hq};
  const int64_t src_rows[4] = {dsc.V, dsc.n_rows, dsc.V, dsc.n_rows};
  const int64_t src_tiles[4] = {pl.n_vtiles, pl.n_ttiles, pl.n_vtiles, pl.n_ttiles};
  for (int q = 0; q < 4; ++q) {
    if (!(q < 2 ? do_pi : do_mu)) continue;
    if (pw && (q == 0 || q == 2)) continue;
    const int64_t row_bytes = q < 2 ? 2 * dsc.d : dsc.d;
    const int64_t units = src_tiles[q] * kTileV * (row_bytes / 16);
    const unsigned blocks = (unsigned)std::min<int64_t>((units + 255) / 256, 8192);
    hipLaunchKernelGGL(pack_kernel, dim3(blocks), dim3(256), 0, s, static_cast<const uint8_t*>(srcs[q]),
                       (uint32_t)src_rows[q], (uint32_t)row_bytes, (uint32_t)units, ws + pl.ws_pack_offset[q]);
  }

  // pi: bf16 operands
  pp.a = pw ? pw + pwl.w_offset : ws + pl.ws_pack_offset[0];
  pp.b = ws + pl.ws_pack_offset[1];
  pp.n_chunks = (int)(2 * dsc.d / kChunk);
  pp.part = reinterpret_cast<float*>(ws + pl.ws_part_offset[0]);
  pp.logit = reinterpret_cast<float*>(ws + pl.ws_logit_offset[0]);

  // mu: e4m3 operands
  ScoreParams pm = pp;
  pm.a = pw ? pw + pwl.wq_offset : ws + pl.ws_pack_offset[2];
  pm.b = ws + pl.ws_pack_offset[3];
  pm.n_chunks = (int)(dsc.d / kChunk);
  pm.part = reinterpret_cast<float*>(ws + pl.ws_part_offset[1]);
  pm.logit = reinterpret_cast<float*>(ws + pl.ws_logit_offset[1]);
  if (dsc.mu_scaling == ACRL_SCALE_MX32) {
    if (do_mu && !pw) launch_pack_mx(dsc.wq_scales, dsc.V, dsc.d, pl.n_vtiles, ws + pl.ws_mx_offset[0], s);
    if (do_mu) launch_pack_mx(dsc.hq_scales, dsc.n_rows, dsc.d, pl.n_ttiles, ws + pl.ws_mx_offset[1], s);
    pm.a_mx = pw ? pw + pwl.mx_offset : ws + pl.ws_mx_offset[0];
    pm.b_mx = ws + pl.ws_mx_offset[1];
  } else {
    pm.a_scale = static_cast<const float*>(dsc.wq_scales);
    pm.b_scale = static_cast<const float*>(dsc.hq_scales);
  }
  auto launch_mu = [&](const ScoreParams& q, unsigned g, auto epi_tag) {
    constexpr int E = decltype(epi_tag)::value;
    if (dsc.mu_scaling == ACRL_SCALE_MX32)
      launch_score_kernel<kMX, E>(g, q, s);
    else if (dsc.mu_scaling == ACRL_SCALE_PER_ROW)
      launch_score_kernel<kFP8Row, E>(g, q, s);
    else
      launch_score_kernel<kFP8Tensor, E>(g, q, s);
  };
  const bool div = dsc.kl_pi_mu || dsc.kl_mu_pi || dsc.l2;  // both policies (checked by the caller)
  if (!div) {
    if (do_pi) launch_score_kernel<kBF16, kEpiSoftmax>(grid, pp, s);
    if (do_mu) launch_mu(pm, grid, std::integral_constant<int, kEpiSoftmax>{});
  } else {
    // passes of div_tiles token tiles: mu (softmax + its logits stored),
    // mu's lse of the pass rows, pi (softmax + the measures' sums against
    // mu's logits), then the measures of the pass rows
    float* zq = reinterpret_cast<float*>(ws + pl.ws_zbuf_offset);
    float* aq2 = reinterpret_cast<float*>(ws + pl.ws_aq_offset);
    float* dpart = reinterpret_cast<float*>(ws + pl.ws_dpart_offset);
    const int cap = pl.div_tiles * kTileT;
    for (int tt0 = 0; tt0 < pl.n_ttiles; tt0 += pl.div_tiles) {
      const int nt = std::min(pl.div_tiles, pl.n_ttiles - tt0);
      const int ntb = (nt + kBlockT - 1) / kBlockT;
      const unsigned g = (unsigned)((ntb * pl.n_sblocks + kXcds - 1) / kXcds * kXcds * kBlockT * kBlockS);
      const int r0 = tt0 * kTileT;
      const int rows = (int)std::min<int64_t>(dsc.n_rows - r0, (int64_t)nt * kTileT);
      ScoreParams pq = pm;
      pq.tt_offset = tt0;
      pq.n_ttiles = nt;
      pq.n_tblocks = ntb;
      pq.zbuf = zq;
      launch_mu(pq, g, std::integral_constant<int, kEpiSoftmaxZ>{});
      hipLaunchKernelGGL(lse2_kernel, dim3((unsigned)((cap + 255) / 256)), dim3(256), 0, s, pm.part, pl.n_strips,
                         (int)dsc.n_rows, r0, rows, cap, aq2);
      ScoreParams pz = pp;
      pz.tt_offset = tt0;
      pz.n_ttiles = nt;
      pz.n_tblocks = ntb;
      pz.zbuf = zq;
      pz.aq2 = aq2;
      pz.dpart = dpart;
      pz.dp_rows = cap;
      launch_score_kernel<kBF16, kEpiSoftmaxDiv>(g, pz, s);
      DivParams dp{};
      dp.n_rows = (int)dsc.n_rows;
      dp.n_strips = pl.n_strips;
      dp.r0 = r0;
      dp.rows = rows;
      dp.n_parts = 2 * pl.n_vtiles;
      dp.dp_rows = cap;
      dp.part_pi = pp.part;
      dp.aq2 = aq2;
      dp.dpart = dpart;
      dp.mask = dsc.mask;
      dp.out_slot = dsc.out_slot;
      dp.kl_pm = dsc.kl_pi_mu;
      dp.kl_mp = dsc.kl_mu_pi;
      dp.l2 = dsc.l2;
      hipLaunchKernelGGL(div_finalize_kernel, dim3((unsigned)((rows + kFinRows - 1) / kFinRows)),
                         dim3(kFinRows * kFinGroups), 0, s, dp);
    }
  }

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
  mp.q_begin = do_pi ? 0 : 1;
  mp.q_end = do_mu ? 2 : 1;
  hipLaunchKernelGGL(merge_kernel, dim3((unsigned)((dsc.n_rows + 255) / 256)), dim3(256), 0, s, mp);
  return hipGetLastError();
}

// ------------------------------------------------------------------ backward
// Grid of a plain product (kEpiStore): one unit per output tile, in the
// scoring kernel's XCD-aware raster (A tiles play the vocabulary strips, B
// tiles the token tiles).
static void gemm_grid(int n_atiles, int n_btiles, ScoreParams& pp, unsigned& grid) {
  pp.n_vtiles = n_atiles;
  pp.tiles_per_strip = 1;
  pp.n_strips = n_atiles;
  pp.n_ttiles = n_btiles;
  pp.n_tblocks = (n_btiles + kBlockT - 1) / kBlockT;
  const int n_sblocks = (n_atiles + kBlockS - 1) / kBlockS;
  const int blocks = (pp.n_tblocks * n_sblocks + kXcds - 1) / kXcds * kXcds;
  grid = (unsigned)(blocks * kBlockT * kBlockS);
}

BackwardPlan plan_backward(int64_t n_rows, int64_t d, int64_t V, int64_t chunk) {
  BackwardPlan pl{};
  pl.chunk = chunk <= 0 ? kBackwardChunk : (chunk + kTileT - 1) / kTileT * kTileT;
  if (n_rows < pl.chunk) pl.chunk = (n_rows + kTileT - 1) / kTileT * kTileT;
  if (pl.chunk == 0) pl.chunk = kTileT;
  pl.n_vtiles = (int)((V + kTileV - 1) / kTileV);
  pl.n_dtiles = (int)((d + kTileV - 1) / kTileV);
  pl.kch_v = pl.n_vtiles * 8;
  const int n_ttiles = (int)(pl.chunk / kTileT);
  const size_t vrows = (size_t)pl.n_vtiles * kTileV, drows = (size_t)pl.n_dtiles * kTileV;
  const size_t crows = (size_t)pl.chunk;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off += align_up(bytes, 256);
    return o;
  };
  pl.off_w = take(vrows * 2 * (size_t)d);                  // W, rows = vocabulary, K = d
  pl.off_wt = take(drows * vrows * 2);                     // W^T, rows = d, K = vocabulary
  pl.off_h = take(crows * 2 * (size_t)d);                  // H chunk, rows = tokens, K = d
  pl.off_ht = take(drows * crows * 2);                     // H^T chunk, rows = d, K = tokens
  pl.off_zt = take((size_t)n_ttiles * kTileT * vrows * 2); // dZ, rows = tokens, K = vocabulary
  pl.off_zv = take(vrows * crows * 2);                     // dZ^T, rows = vocabulary, K = tokens
  pl.off_queue = take((size_t)kXcds * kQueueStride * sizeof(int));  // the products' claim counters
  pl.ws_bytes = off;
  return pl;
}

hipError_t launch_backward(const acrl_backward_desc& dsc, const BackwardPlan& pl, hipStream_t s) {
  uint8_t* ws = static_cast<uint8_t*>(dsc.workspace);
  const int64_t d = dsc.d, V = dsc.V;
  float* dh = dsc.dh;
  float* dw = dsc.dw;
  if (dsc.n_rows == 0) {
    if (dw && !dsc.accumulate_dw)
      hipLaunchKernelGGL(fill_zero_kernel, dim3(4096), dim3(256), 0, s, dw, V * d);
    return hipGetLastError();
  }
  uint8_t* img_w = ws + pl.off_w;
  uint8_t* img_wt = ws + pl.off_wt;
  uint8_t* img_h = ws + pl.off_h;
  uint8_t* img_ht = ws + pl.off_ht;
  uint8_t* img_zt = ws + pl.off_zt;
  uint8_t* img_zv = ws + pl.off_zv;
  const uint16_t* w = static_cast<const uint16_t*>(dsc.w);
  const uint16_t* h = static_cast<const uint16_t*>(dsc.h);
  // W (rows = vocabulary, for the recomputed logits) and W^T (rows = d, for dH), once per call
  {
    const int64_t units = (int64_t)pl.n_vtiles * kTileV * (2 * d / 16);
    hipLaunchKernelGGL(pack_kernel, dim3((unsigned)std::min<int64_t>((units + 255) / 256, 8192)), dim3(256), 0, s,
                       reinterpret_cast<const uint8_t*>(w), (uint32_t)V, (uint32_t)(2 * d), (uint32_t)units, img_w);
    if (dh)
      hipLaunchKernelGGL(pack_t_kernel, dim3((unsigned)((int64_t)pl.n_dtiles * pl.kch_v)), dim3(256), 0, s, w, V, d,
                         pl.kch_v, img_wt);
  }
  for (int64_t r0 = 0; r0 < dsc.n_rows; r0 += pl.chunk) {
    const int64_t rows = std::min<int64_t>(pl.chunk, dsc.n_rows - r0);
    const int n_ttiles = (int)((rows + kTileT - 1) / kTileT);
    const int kch_t = n_ttiles * 8;
    const int64_t units = (int64_t)n_ttiles * kTileT * (2 * d / 16);
    hipLaunchKernelGGL(pack_kernel, dim3((unsigned)std::min<int64_t>((units + 255) / 256, 8192)), dim3(256), 0, s,
                       reinterpret_cast<const uint8_t*>(h + r0 * d), (uint32_t)rows, (uint32_t)(2 * d),
                       (uint32_t)units, img_h);
    if (dw)
      hipLaunchKernelGGL(pack_t_kernel, dim3((unsigned)((int64_t)pl.n_dtiles * kch_t)), dim3(256), 0, s, h + r0 * d,
                         rows, d, kch_t, img_ht);
    // dZ of the chunk from the recomputed logits (vocabulary strips as in scoring)
    {
      const ScorePlan sp = plan_score(rows, d, V);
      ScoreParams pg{};
      pg.a = img_w;
      pg.b = img_h;
      pg.n_chunks = (int)(2 * d / kChunk);
      pg.V = (int)V;
      pg.n_rows = (int)rows;
      pg.n_vtiles = sp.n_vtiles;
      pg.tiles_per_strip = sp.tiles_per_strip;
      pg.n_strips = sp.n_strips;
      pg.n_ttiles = sp.n_ttiles;
      pg.n_tblocks = sp.n_tblocks;
      pg.inv_temp = dsc.inv_temperature;
      pg.ids = dsc.token_ids + r0;
      pg.g_coef = dsc.coef;
      pg.g_lse = dsc.lse;
      pg.g_slot = dsc.row_slot ? dsc.row_slot + r0 : nullptr;
      pg.g_slot_offset = r0;
      pg.gz_t = img_zt;
      pg.gz_v = img_zv;
      pg.kch_v = pl.kch_v;
      pg.kch_t = kch_t;
      launch_score_kernel<kBF16, kEpiGrad>((unsigned)sp.grid, pg, s);
    }
    // dH[chunk] = dZ W: A = dZ (rows = tokens), B = W^T (rows = d), K = vocabulary
    if (dh) {
      ScoreParams pc{};
      unsigned grid = 0;
      gemm_grid(n_ttiles, pl.n_dtiles, pc, grid);
      pc.a = img_zt;
      pc.b = img_wt;
      pc.n_chunks = pl.kch_v;
      pc.n_rows = (int)d;
      pc.V = (int)rows;
      pc.c = dh + r0 * d;
      pc.ldc = d;
      pc.c_rows = (int)rows;
      pc.c_accumulate = 0;
      pc.queue = reinterpret_cast<int*>(ws + pl.off_queue);
      launch_score_kernel<kBF16, kEpiStore>(grid, pc, s);
    }
    // dW (+)= dZ^T H: A = dZ^T (rows = vocabulary), B = H^T (rows = d), K = tokens
    if (dw) {
      ScoreParams pc{};
      unsigned grid = 0;
      gemm_grid(pl.n_vtiles, pl.n_dtiles, pc, grid);
      pc.a = img_zv;
      pc.b = img_ht;
      pc.n_chunks = kch_t;
      pc.n_rows = (int)d;
      pc.V = (int)V;
      pc.c = dw;
      pc.ldc = d;
      pc.c_rows = (int)V;
      pc.c_accumulate = (r0 > 0 || dsc.accumulate_dw) ? 1 : 0;
      pc.queue = reinterpret_cast<int*>(ws + pl.off_queue);
      launch_score_kernel<kBF16, kEpiStore>(grid, pc, s);
    }
  }
  return hipGetLastError();
}

hipError_t launch_sample(const acrl_sample_desc& dsc, const ScorePlan& pl, hipStream_t s) {
  if (dsc.n_rows == 0) return hipSuccess;
  uint8_t* ws = static_cast<uint8_t*>(dsc.workspace);
  const uint8_t* pw = static_cast<const uint8_t*>(dsc.packed_weights);
  const PackedWeightsLayout pwl = packed_weights_layout(dsc.V, dsc.d, dsc.mu_scaling);
  const void* srcs[2] = {dsc.wq, dsc.hq};
  const int64_t src_rows[2] = {dsc.V, dsc.n_rows};
  const int64_t src_tiles[2] = {pl.n_vtiles, pl.n_ttiles};
  for (int q = 0; q < 2; ++q) {
    if (q == 0 && pw) continue;  // Wq comes prepacked
    const int64_t units = src_tiles[q] * kTileV * (dsc.d / 16);
    const unsigned blocks = (unsigned)std::min<int64_t>((units + 255) / 256, 8192);
    hipLaunchKernelGGL(pack_kernel, dim3(blocks), dim3(256), 0, s, static_cast<const uint8_t*>(srcs[q]),
                       (uint32_t)src_rows[q], (uint32_t)dsc.d, (uint32_t)units, ws + pl.ws_pack_offset[2 + q]);
  }
  ScoreParams pm{};
  pm.V = (int)dsc.V;
  pm.n_rows = (int)dsc.n_rows;
  pm.n_vtiles = pl.n_vtiles;
  pm.tiles_per_strip = pl.tiles_per_strip;
  pm.n_strips = pl.n_strips;
  pm.n_ttiles = pl.n_ttiles;
  pm.n_tblocks = pl.n_tblocks;
  pm.inv_temp = dsc.inv_temperature;
  pm.mx_row_bytes = (int)(dsc.d / 32);
  pm.queue = reinterpret_cast<int*>(ws + pl.ws_queue_offset);
  pm.a = pw ? pw + pwl.wq_offset : ws + pl.ws_pack_offset[2];
  pm.b = ws + pl.ws_pack_offset[3];
  pm.n_chunks = (int)(dsc.d / kChunk);
  pm.part = reinterpret_cast<float*>(ws + pl.ws_part_offset[1]);
  pm.seed_lo = (uint32_t)dsc.seed;
  pm.seed_hi = (uint32_t)(dsc.seed >> 32);
  pm.row_offset = dsc.row_offset;
  const size_t best_plane = align_up((size_t)pl.n_strips * (size_t)dsc.n_rows * sizeof(float), 256);
  pm.best_key = reinterpret_cast<float*>(ws + pl.ws_best_offset);
  pm.best_logit = reinterpret_cast<float*>(ws + pl.ws_best_offset + best_plane);
  pm.best_id = reinterpret_cast<int32_t*>(ws + pl.ws_best_offset + 2 * best_plane);
  const unsigned grid = (unsigned)pl.grid;
  if (dsc.mu_scaling == ACRL_SCALE_MX32) {
    if (!pw) launch_pack_mx(dsc.wq_scales, dsc.V, dsc.d, pl.n_vtiles, ws + pl.ws_mx_offset[0], s);
    launch_pack_mx(dsc.hq_scales, dsc.n_rows, dsc.d, pl.n_ttiles, ws + pl.ws_mx_offset[1], s);
    pm.a_mx = pw ? pw + pwl.mx_offset : ws + pl.ws_mx_offset[0];
    pm.b_mx = ws + pl.ws_mx_offset[1];
    launch_score_kernel<kMX, kEpiSample>(grid, pm, s);
  } else {
    pm.a_scale = static_cast<const float*>(dsc.wq_scales);
    pm.b_scale = static_cast<const float*>(dsc.hq_scales);
    if (dsc.mu_scaling == ACRL_SCALE_PER_ROW)
      launch_score_kernel<kFP8Row, kEpiSample>(grid, pm, s);
    else
      launch_score_kernel<kFP8Tensor, kEpiSample>(grid, pm, s);
  }
  SampleMergeParams mp{};
  mp.n_rows = (int)dsc.n_rows;
  mp.n_strips = pl.n_strips;
  mp.part = pm.part;
  mp.best_key = pm.best_key;
  mp.best_logit = pm.best_logit;
  mp.best_id = pm.best_id;
  mp.ids = dsc.ids;
  mp.logp = dsc.logp_mu;
  hipLaunchKernelGGL(sample_merge_kernel, dim3((unsigned)((dsc.n_rows + 255) / 256)), dim3(256), 0, s, mp);
  return hipGetLastError();
}

}  // namespace acrl
