// Projected-KV cache builder on bf16 MFMA (gfx950).
//
// Sec. 3.2, linear projection of the KV of L_s sampled target layers (App. A:
// L_s = 3) back to one layer, k' = W_K [k^(1); ...; k^(L_s)] and likewise for
// V, with the "Proj + RoPE fix" variant rotating k' at the token's position.
// For every token listed, the projected K/V are written into the drafter's
// paged cache.
//
// GEMM formulation: per tensor (K or V), out^T = W x^T with the weights as the
// MFMA A operand (rows = output channels) and the tokens' stacked source
// vectors as the B operand (columns = tokens), so each accumulator lane holds
// one token and four consecutive channels per register quad.  A workgroup owns
// 256 channels (two KV heads) x 256 tokens; its four waves own one head x 128
// tokens each, so the RoPE partners (channel m and m + 64 of a head) sit in
// the same lane.  The reduction runs over L_s d_kv inputs in chunks of KC
// (a chunk never straddles a head of a source layer, so a token's chunk is
// 2 KC contiguous bytes in its page slot; the page walk is done once per
// workgroup).
//
// Operand movement: both tiles go straight from global memory into LDS with
// global_load_lds_dwordx4 (no register staging, no LDS store instructions),
// NS stages deep: NS - 1 chunks are in flight while one is computed, one
// barrier per chunk.  Each load is a wave-wide 1 KB block of LDS, so the rows
// are unpadded and an XOR swizzle on the load side keeps the fragment reads
// free of bank conflicts.  A chunk's loads are issued one per four MFMAs of
// the chunk before it.
//
// Epilogue: RoPE on keys in registers (angles reduced in float64, sine and
// cosine from the hardware units), bf16 rounding, and 8-byte stores into the
// destination page slots.  With few tokens the reduction is split over
// workgroups; each writes float32 partial sums and kvproj_combine_kernel adds
// them, rotates and scatters.
//
// Work order: channel tile fastest, then split, token tile, tensor.  The
// hardware hands workgroup i to XCD i % 8; xcd_remap gives each XCD a
// contiguous range, so the channel tiles that read one token tile share that
// XCD's L2.
//
// Calls with few tokens (where this tiling would split the reduction) take
// kvproj_direct_kernel instead: 64-channel x up-to-64-token tiles that keep
// the whole reduction, so no float32 partials go to memory and no combine
// kernel runs.
#include <type_traits>

#include "kvproj_common.h"

namespace kvshot {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

#ifndef KVSHOT_KVPROJ_KC
#define KVSHOT_KVPROJ_KC 32
#endif
#ifndef KVSHOT_KVPROJ_NS
#define KVSHOT_KVPROJ_NS 4
#endif
typedef __attribute__((address_space(3))) void lds_void;

__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 v) { return __builtin_bit_cast(bf16x8, v); }

__device__ __forceinline__ int clampi(int v, int lo, int hi) { return v < lo ? lo : (v > hi ? hi : v); }

// vmcnt(n) with no wait on the other counters (gfx9 encoding: vmcnt bits [3:0] and [15:14])
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

// Barrier without the memory fence of __syncthreads (which would also wait for
// the operand prefetches still in flight).  The wave's own LDS reads complete
// first, so that no read of a ring stage is still in flight when the barrier
// lets its refill start; the clobber keeps the compiler from moving LDS
// accesses across it.
__device__ __forceinline__ void lds_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

// One wave-wide 16-byte load from global memory straight into LDS: lane L's 16 bytes land at
// `lds` + 16 L (global_load_lds_dwordx4; M0 holds the wave-uniform LDS address, set one wait
// state ahead).  Issued as inline asm: the compiler's own form makes every later LDS read wait
// for all such loads in flight (it cannot tell the stages apart), which would serialise the
// prefetch.  Nothing else in these kernels uses M0.
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
__device__ __forceinline__ void load_to_lds16(const void* src, const void* lds) {
  const uint32_t la = (uint32_t)(uintptr_t)(lds_void*)lds;
  asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off" ::"v"(src), "s"(la) : "memory", "m0");
}
#pragma clang diagnostic pop

// Row swizzle of the LDS operand tiles (rows of KC bf16 = KC / 8 pieces of 16 bytes): piece q
// of row r is stored in slot q ^ swizzle(r).  Chosen so that 8 or 16 consecutive rows read at
// one logical piece cover distinct 4-byte bank groups with 32 or 64 banks, and so that it
// depends on bits 0..4 of r only (a fragment row is 32 i + lane % 32 above a multiple of 32).
template <int KC>
__device__ __forceinline__ int swizzle(int r) {
  if constexpr (KC == 64) return (r ^ ((r >> 3) & 3)) & 7;
  else if constexpr (KC == 32) return ((r >> 1) ^ (r >> 2)) & 3;
  else return ((r >> 2) ^ (r >> 3)) & 1;
}

// KC: reduction indices per chunk; NS: LDS stages (chunks in flight: NS - 1).
template <bool SPLIT, int KC, int NS>
__global__ __launch_bounds__(256, 1) void kvproj_kernel(KvProjParams p) {
  constexpr int kPieces = KC / 8;                   // 16-byte pieces per operand row and chunk
  constexpr int kRowsPerLoad = 64 / kPieces;        // operand rows one wave-wide 16-byte load covers
  constexpr int kLoads = kProjTile / kRowsPerLoad / 4;   // loads per wave, operand and chunk
  constexpr int kStageElems = kProjTile * KC;       // one operand tile (bf16)
  constexpr int kSteps = KC / 16;                   // MFMA k-steps per chunk
  static_assert(KC == 16 || KC == 32 || KC == 64, "chunk");
  static_assert(NS >= 2 && NS * 2 * kStageElems * 2 <= 136 * 1024, "stages fit in LDS");
  // Operand rows are KC * 2 bytes with no padding.  Piece q of row r sits at physical slot
  // q ^ swz(r) (see swizzle()): the lanes one LDS cycle serves -- 8 or 16 consecutive rows at
  // one logical piece -- then hit distinct bank groups.
  __shared__ __attribute__((aligned(16))) uint16_t smem[NS * 2 * kStageElems];
  __shared__ int64_t t_src[kProjTile];   // source element offset of each token's slot (page, slot)
  __shared__ int64_t t_dst[kProjTile];   // destination element offset
  __shared__ int32_t t_pos[kProjTile];   // position, clamped to the RoPE table
  __shared__ const uint16_t* t_layer[2][kProjMaxLayers];   // source pools [K, V][layer]
  __shared__ double t_rev[kHalfDim];     // RoPE revolutions per position of channel pair m

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int hh = lane >> 5;
  const int wc = w & 1;      // head of the channel tile
  const int wt = w >> 1;     // half of the token tile

  int wi = xcd_remap(blockIdx.x, gridDim.x);
  if (wi >= p.work_items) return;
  const int mt = wi % p.m_tiles;
  wi /= p.m_tiles;
  const int split = wi % p.splits;
  wi /= p.splits;
  const int nt = wi % p.n_tiles;
  const int g = wi / p.n_tiles;                   // 0: keys, 1: values
  const int n0 = nt * kProjTile;
  const int d_kv = p.hkv * kHeadDim;
  const int K = p.layers * d_kv;
  const int nchunks = K / 64;                     // split boundaries are in 64-wide chunks
  const int cbeg = (int)((int64_t)split * nchunks / p.splits);
  const int cend = (int)((int64_t)(split + 1) * nchunks / p.splits);

  // ---- the tile's tokens: page walk once, kept in LDS ----
  {
    const int tk = n0 + tid < p.n_tokens ? n0 + tid : p.n_tokens - 1;
    const int b = clampi(p.token_seq[tk], 0, p.batch - 1);
    const int t = clampi(p.token_pos[tk], 0, (p.max_pages_per_seq << p.page_shift) - 1);
    const int lp = t >> p.page_shift;
    const int slot = t & ((1 << p.page_shift) - 1);
    const int sp = physical_page(p.page_table, b, p.max_pages_per_seq, lp, p.num_pages);
    const int dp = physical_page(p.dst_page_table, b, p.max_pages_per_seq, lp, p.dst_num_pages);
    t_src[tid] = (int64_t)sp * p.page_stride + (int64_t)slot * p.slot_stride;
    t_dst[tid] = (int64_t)dp * p.dst_page_stride + (int64_t)slot * p.dst_slot_stride;
    t_pos[tid] = t < p.max_position ? t : p.max_position - 1;
    if (tid < kHalfDim) t_rev[tid] = p.rope_rev[tid];
    if (tid == 0) {   // constant indices: the kernel arguments stay in scalar registers
#pragma unroll
      for (int l = 0; l < kProjMaxLayers; ++l) {
        t_layer[0][l] = p.k_src[l];
        t_layer[1][l] = p.v_src[l];
      }
    }
  }
  __syncthreads();

  // ---- operand loads straight into LDS (global_load_lds_dwordx4: lane L of a load lands at
  // base + 16 L).  Load j of wave w fills rows kRowsPerLoad (4 w + j) + L / kPieces, physical
  // slot L % kPieces, so lane L fetches the logical piece that belongs there. ----
  int64_t soff[kLoads];
  int32_t woff[kLoads];
#pragma unroll
  for (int j = 0; j < kLoads; ++j) {
    const int r = kRowsPerLoad * (kLoads * w + j) + lane / kPieces;
    const int q = (lane % kPieces) ^ swizzle<KC>(r);
    soff[j] = t_src[r] + 8 * q;
    const int wrow = mt * kProjTile + r;
    woff[j] = (wrow < d_kv ? wrow : d_kv - 1) * K + 8 * q;
  }
  const uint16_t* wsrc = g ? p.w_v : p.w_k;
  const int nch = (cend - cbeg) * (64 / KC);      // chunks of this split (the split plan counts 64-wide ones)
  const int k_first = cbeg * 64;
  // the 2 kLoads loads of chunk c into `stage`: the first kLoads are weight rows, the rest token rows
  struct Target {
    const uint16_t* w;    // weight columns of the chunk
    const uint16_t* x;    // the chunk's head-half of the source layer
    uint16_t* lds;        // the stage
  };
  // Cursor on the chunk whose loads are issued next: chunk cur_c starts at reduction index
  // k_first + cur_c KC, offset cur_rem into source layer cur_l.  It moves one chunk at a time and
  // stops at the last chunk; the layer's pool pointer is read from LDS again only when a chunk
  // starts a new layer (a chunk never straddles one), so no chunk waits on that read or divides.
  int cur_c = 0, cur_l = k_first / d_kv;
  int cur_rem = k_first - cur_l * d_kv;
  const uint16_t* cur_pool = t_layer[g][cur_l];
  auto advance = [&]() {
    if (cur_c + 1 < nch) {
      ++cur_c;
      cur_rem += KC;
      if (cur_rem == d_kv) {
        cur_rem = 0;
        ++cur_l;
        cur_pool = t_layer[g][cur_l];
      }
    }
  };
  auto target = [&](int stage) {
    Target t;
    t.w = wsrc + k_first + cur_c * KC;
    t.x = cur_pool + (int64_t)(cur_rem >> 7) * p.head_stride + (cur_rem & 127);
    t.lds = smem + stage * 2 * kStageElems + (kLoads * w) * 512;
    return t;
  };
  auto issue_one = [&](const Target& t, int idx) {
    if (idx < kLoads) load_to_lds16(t.w + woff[idx], t.lds + idx * 512);
    else load_to_lds16(t.x + soff[idx - kLoads], t.lds + kStageElems + (idx - kLoads) * 512);
  };

  f32x16 acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.0f;

  // fragment reads: row R = (wave base) + 32 i + lane % 32 has swizzle(R) == swizzle(lane % 32); lane half hh
  // covers logical pieces hh kSteps .. hh kSteps + kSteps - 1, k-step s takes piece hh kSteps + s
  const int swz = swizzle<KC>(lane & 31);
  int frag_off[kSteps];
#pragma unroll
  for (int st = 0; st < kSteps; ++st) frag_off[st] = 8 * ((hh * kSteps + st) ^ swz);
  static_assert(2 * kLoads == 4 * kSteps, "one load per four MFMAs");
  static_assert(NS >= 3, "the next chunk is read while a later one is still in flight");
  // Fragments of one k-step, double-buffered across k-steps and across chunks.
  bf16x8 a[2][4], b[2][4];
  auto read = [&](int stage, int st, bf16x8 (&fa)[4], bf16x8 (&fb)[4]) {
    const uint16_t* A = smem + stage * 2 * kStageElems + (128 * wc + (lane & 31)) * KC;
    const uint16_t* B = smem + stage * 2 * kStageElems + kStageElems + (128 * wt + (lane & 31)) * KC;
#pragma unroll
    for (int i = 0; i < 4; ++i) fa[i] = as_bf16x8(*(const u32x4*)(A + 32 * i * KC + frag_off[st]));
#pragma unroll
    for (int j = 0; j < 4; ++j) fb[j] = as_bf16x8(*(const u32x4*)(B + 32 * j * KC + frag_off[st]));
  };
  // Chunk c from `stage` (its first k-step's fragments already read), with the loads of a later
  // chunk (`nt`) issued one per four MFMAs (so no wave stalls on a burst of load issues before its
  // first MFMA) and the next k-step's fragments read during the current one -- in the last k-step,
  // those of chunk c + 1's first k-step from `next_stage`.  The chunk's one barrier sits before
  // its last k-step: by then every wave has its share of chunk c + 1 in LDS (the wait before the
  // barrier) and has finished reading chunk c - 1, whose stage the loads refill; so the first
  // reads of the next chunk no longer wait behind a barrier with nothing to compute.  The order is
  // pinned with scheduling barriers.
  auto compute = [&](int stage, int next_stage, const Target& nt) {
#pragma unroll
    for (int st = 0; st < kSteps; ++st) {
      if (st + 1 == kSteps) {
        // in flight may stay: the NS - 3 chunks after c + 1 and this chunk's loads so far
        wait_vmcnt<(NS - 3) * 2 * kLoads + 4 * (kSteps - 1)>();
        lds_barrier();
        __builtin_amdgcn_sched_barrier(0);
      }
      if (st + 1 < kSteps) read(stage, st + 1, a[(st + 1) & 1], b[(st + 1) & 1]);
      else read(next_stage, 0, a[(st + 1) & 1], b[(st + 1) & 1]);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
#pragma unroll
        for (int j = 0; j < 4; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[st & 1][i], b[st & 1][j], acc[i][j], 0, 0, 0);
        __builtin_amdgcn_sched_barrier(0);
        issue_one(nt, 4 * st + i);
        __builtin_amdgcn_sched_barrier(0);
      }
    }
  };
  static_assert(kSteps % 2 == 0, "a chunk's first k-step uses fragment buffer 0");

  // ---- main loop.  Chunks 0 .. NS - 2 are issued up front, chunk 0 is waited for and its first
  // k-step read; iteration c computes c from stage c % NS while issuing chunk c + NS - 1 into the
  // stage of chunk c - 1 (free: every wave finished reading it before chunk c - 1's barrier).
  // Loads past the last chunk re-read it into a stage nobody reads again, and the last chunk's
  // reads of "the next chunk" read a stage whose values are never used. ----
#pragma unroll
  for (int c = 0; c < NS - 1; ++c) {
    const Target t = target(c);
#pragma unroll
    for (int idx = 0; idx < 2 * kLoads; ++idx) issue_one(t, idx);
    advance();
  }
  wait_vmcnt<(NS - 2) * 2 * kLoads>();
  lds_barrier();
  read(0, 0, a[0], b[0]);
  int stage = 0;
  for (int c = 0; c < nch; ++c) {
    const int next_stage = stage == NS - 1 ? 0 : stage + 1;
    compute(stage, next_stage, target(stage == 0 ? NS - 1 : stage - 1));   // the cursor is at chunk c + NS - 1 (clamped)
    advance();
    stage = next_stage;
  }
  wait_vmcnt<0>();     // the trailing re-reads land before the workgroup ends

  const int head = mt * 2 + wc;       // this wave's KV head
  if constexpr (SPLIT) {
    // float32 partial sums, [split][token][K channels | V channels]
    if (head >= p.hkv) return;
    float* part = p.part + (int64_t)split * p.n_tokens * (2 * d_kv) + g * d_kv + head * kHeadDim + 4 * hh;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int token = n0 + 128 * wt + 32 * j + (lane & 31);
      if (token >= p.n_tokens) continue;
      float* dst = part + (int64_t)token * (2 * d_kv);
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int q = 0; q < 4; ++q)
          *(float4*)(dst + 32 * i + 8 * q) =
              make_float4(acc[i][j][4 * q], acc[i][j][4 * q + 1], acc[i][j][4 * q + 2], acc[i][j][4 * q + 3]);
    }
    return;
  } else {
    // RoPE (keys) and bf16 rounding in registers, then 8-byte stores straight into the page
    // slots (L2 merges a row's sixteen 16-byte pieces): the lane of token column t and half hh
    // holds channels 32 i + 8 q + 4 hh .. + 3 of its head in register quad q of block i, and
    // channel m (i < 2) pairs with m + 64, held in block i + 2 of the same lane.
    const int head = mt * 2 + wc;
    if (head < p.hkv) {
      uint16_t* dst = (g ? p.v_dst : p.k_dst) + (int64_t)head * p.dst_head_stride + 4 * hh;
      // keys: the angle of channel pair m at position t is t theta^(-2m/128); in revolutions,
      // t * rev[m] is formed in float64 and reduced to [0, 1) exactly enough that the
      // hardware's sine and cosine of one revolution (v_sin_f32 / v_cos_f32) stay within
      // 3e-7 of the float64 values -- far below a bf16 step of the output
      auto emit = [&](int j, auto rot_t) {
        constexpr bool kRot = decltype(rot_t)::value;
        const int tl = 128 * wt + 32 * j + (lane & 31);
        if (n0 + tl >= p.n_tokens) return;
        uint16_t* row = dst + t_dst[tl];
        const double pos = (double)t_pos[tl];
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            float x1[4], x2[4];
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              x1[e] = acc[i][j][4 * q + e];
              x2[e] = acc[i + 2][j][4 * q + e];
            }
            if constexpr (kRot) {
#pragma unroll
              for (int e = 0; e < 4; ++e) {
                double r = pos * t_rev[32 * i + 8 * q + 4 * hh + e];
                r -= floor(r);
                const float u = (float)r;
                const float c = __builtin_amdgcn_cosf(u), sn = __builtin_amdgcn_sinf(u);
                const float y1 = x1[e] * c - x2[e] * sn;
                const float y2 = x2[e] * c + x1[e] * sn;
                x1[e] = y1;
                x2[e] = y2;
              }
            }
            u32x2 v1, v2;
            v1[0] = pack_bf16x2(x1[0], x1[1]);
            v1[1] = pack_bf16x2(x1[2], x1[3]);
            v2[0] = pack_bf16x2(x2[0], x2[1]);
            v2[1] = pack_bf16x2(x2[2], x2[3]);
            *(u32x2*)(row + 32 * i + 8 * q) = v1;
            *(u32x2*)(row + 64 + 32 * i + 8 * q) = v2;
          }
      };
      if (g == 0 && p.rope_keys) {
#pragma unroll
        for (int j = 0; j < 4; ++j) emit(j, std::true_type{});
      } else {
#pragma unroll
        for (int j = 0; j < 4; ++j) emit(j, std::false_type{});
      }
    }
  }
}

// ---- direct kernel: calls with few tokens ----
// A workgroup owns one RoPE pair of 32-channel slices of a head (channels
// 32 s .. 32 s + 31 and their partners + 64: tile rows 0..31 and 32..63) x
// 16 TB tokens, and the whole reduction, so no partial sums leave the chip.
// The reduction runs in chunks of 128 inputs (one head of one source layer:
// 256 contiguous bytes of every weight row and of every token's page slot).
// Each chunk goes into an NBUF-stage LDS ring with global_load_lds_dwordx4,
// four rows of 256 bytes per wave-wide load, so that neighbouring lanes read
// neighbouring bytes: loading the MFMA fragments straight from global memory
// (each lane a different row) moves a third as many bytes per CU per second
// from L2.  The four waves take one 32-wide k-step of every chunk each
// (v_mfma_f32_16x16x32_bf16 over the whole 64 x 16 TB tile) and add their
// sums through LDS at the end in wave order; keys are then rotated (angles
// reduced in float64, hardware sine and cosine), rounded and stored.  The work
// order puts a channel slice's token tiles next to each other, so they run on
// one XCD and its weight rows come from HBM once.
template <int TB, int NBUF>
__global__ __launch_bounds__(256, 1) void kvproj_direct_kernel(KvProjParams p) {
  constexpr int NW = 4;
  constexpr int kTok = 16 * TB;
  constexpr int kRowB = 256;                       // bytes of a row of a chunk
  constexpr int kStage = (64 + kTok) * kRowB;      // weight rows, then token rows
  constexpr int kLA = 64 / 4 / NW;                 // weight loads per wave and chunk (4 rows each)
  constexpr int kLB = kTok / 4 / NW;               // token loads per wave and chunk
  constexpr int kLoads = kLA + kLB;
  constexpr int kRow = 68;                         // floats per token row of the merge buffer (64 + 4 of padding)
  static_assert(NBUF >= 2 && NBUF * kStage <= 150 * 1024, "ring fits in LDS");
  static_assert(NW * kTok * kRow * 4 <= NBUF * kStage, "merge buffer fits in the ring");
  typedef float f32x4 __attribute__((ext_vector_type(4)));
  __shared__ __attribute__((aligned(16))) unsigned char ring[NBUF * kStage];
  __shared__ int64_t t_src[kTok];
  __shared__ int64_t t_dst[kTok];
  __shared__ int32_t t_pos[kTok];
  __shared__ double t_rev[kHalfDim];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wi = xcd_remap(blockIdx.x, gridDim.x);
  if (wi >= p.work_items) return;
  const int tt = wi % p.n_tiles;                  // token tile
  const int ct = wi / p.n_tiles;                  // channel slice: tensor, head, half
  const int pairs = 2 * p.hkv;
  const int g = ct / pairs;                       // 0: keys, 1: values
  const int head = (ct % pairs) >> 1;
  const int half = ct & 1;
  const int n0 = tt * kTok;
  const int d_kv = p.hkv * kHeadDim;
  const int K = p.layers * d_kv;
  const int nch = K / kHeadDim;                   // chunks: (layer, head) of the sources

  if (tid < kTok) {
    const int tk = n0 + tid < p.n_tokens ? n0 + tid : p.n_tokens - 1;
    const int b = clampi(p.token_seq[tk], 0, p.batch - 1);
    const int t = clampi(p.token_pos[tk], 0, (p.max_pages_per_seq << p.page_shift) - 1);
    const int lp = t >> p.page_shift;
    const int slot = t & ((1 << p.page_shift) - 1);
    const int sp = physical_page(p.page_table, b, p.max_pages_per_seq, lp, p.num_pages);
    const int dp = physical_page(p.dst_page_table, b, p.max_pages_per_seq, lp, p.dst_num_pages);
    t_src[tid] = (int64_t)sp * p.page_stride + (int64_t)slot * p.slot_stride;
    t_dst[tid] = (int64_t)dp * p.dst_page_stride + (int64_t)slot * p.dst_slot_stride;
    t_pos[tid] = t < p.max_position ? t : p.max_position - 1;
  } else if (tid >= 128 && tid < 128 + kHalfDim) {
    t_rev[tid - 128] = p.rope_rev[tid - 128];
  }
  __syncthreads();

  // ---- loads: lane L of a wave-wide load fills row (4 rows per load) L / 16, physical 16-byte piece
  // L % 16, holding logical piece (L % 16) ^ (row % 16) (so the fragment reads below are free of bank
  // conflicts).  Wave w loads weight rows 16 w .. 16 w + 15 and token rows 4 TB w .. 4 TB w + 4 TB - 1. ----
  const int lrow = lane >> 4;
  const uint16_t* wsrc = g ? p.w_v : p.w_k;
  int32_t aoff[kLA];     // element offsets in the weight matrix (chunk 0)
  int64_t boff[kLB];     // element offsets in a source pool (chunk 0 of the token's slot)
#pragma unroll
  for (int i = 0; i < kLA; ++i) {
    const int R = 16 * w + 4 * i + lrow;
    const int ch = head * kHeadDim + 32 * half + (R & 31) + 64 * (R >> 5);
    aoff[i] = ch * K + 8 * ((lane & 15) ^ (R & 15));
  }
#pragma unroll
  for (int j = 0; j < kLB; ++j) {
    const int R = 4 * kLB * w + 4 * j + lrow;
    boff[j] = t_src[R] + 8 * ((lane & 15) ^ (R & 15));
  }
  const uint16_t* src_l0 = g ? p.v_src[0] : p.k_src[0];
  const uint16_t* src_l1 = g ? p.v_src[1] : p.k_src[1];
  const uint16_t* src_l2 = g ? p.v_src[2] : p.k_src[2];
  const uint16_t* src_l3 = g ? p.v_src[3] : p.k_src[3];
  // the kLoads loads of chunk c into `stage`: weight rows first, then token rows
  struct Target {
    const uint16_t* wc;    // the chunk's columns of the weight rows
    const uint16_t* x;     // the chunk's (layer, head) in the source pool
    unsigned char* st;     // the stage
  };
  auto target = [&](int c, int stage) {
    const int l = c / p.hkv;
    const int hd = c - l * p.hkv;
    const uint16_t* x = l == 0 ? src_l0 : (l == 1 ? src_l1 : (l == 2 ? src_l2 : src_l3));
    Target t;
    t.x = x + (int64_t)hd * p.head_stride;
    t.wc = wsrc + c * kHeadDim;
    t.st = ring + stage * kStage;
    return t;
  };
  auto issue_one = [&](const Target& t, int idx) {
    if (idx < kLA) load_to_lds16(t.wc + aoff[idx], t.st + (16 * w + 4 * idx) * kRowB);
    else load_to_lds16(t.x + boff[idx - kLA], t.st + (64 + 4 * kLB * w + 4 * (idx - kLA)) * kRowB);
  };

  // ---- fragments: wave w takes k-step w of every chunk (inputs 32 w .. 32 w + 31 of the head): lane
  // (r = l % 16, q = l / 16) reads logical piece 4 w + q of rows 16 i + r (weights) and 64 + 16 j + r (tokens) ----
  const int r = lane & 15, q = lane >> 4;
  const int frag = r * kRowB + 16 * ((4 * w + q) ^ r);
  f32x4 acc[4][TB];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < TB; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
  // One chunk from `stage`, with the loads of a later chunk (`nt`, if `more`) spread between its MFMAs:
  // a wave that waits to hand a load to the address unit then has matrix work in flight, instead of
  // issuing a burst of loads and then computing.  The order is pinned with scheduling barriers.
  auto compute = [&](int stage, const Target& nt, bool more) {
    const unsigned char* st = ring + stage * kStage + frag;
    bf16x8 a[4], bv[TB];
#pragma unroll
    for (int i = 0; i < 4; ++i) a[i] = as_bf16x8(*(const u32x4*)(st + 16 * i * kRowB));
#pragma unroll
    for (int j = 0; j < TB; ++j) bv[j] = as_bf16x8(*(const u32x4*)(st + (64 + 16 * j) * kRowB));
#pragma unroll
    for (int m = 0; m < 4 * TB; ++m) {
      const int i = m / TB, j = m % TB;
      acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[i], bv[j], acc[i][j], 0, 0, 0);
      // load k goes after MFMA (k * 4 TB) / kLoads, so the kLoads loads spread evenly over the 4 TB MFMAs
#pragma unroll
      for (int k = 0; k < kLoads; ++k)
        if ((k * 4 * TB) / kLoads == m) {
          __builtin_amdgcn_sched_barrier(0);
          if (more) issue_one(nt, k);
          __builtin_amdgcn_sched_barrier(0);
        }
    }
  };

  // ---- ring: chunks 0 .. NBUF - 2 up front; iteration c waits for its own loads of chunk c (the younger
  // chunks in flight may stay so), passes a barrier (all of chunk c has landed and every wave is done
  // with chunk c - 1), issues chunk c + NBUF - 1 into the stage chunk c - 1 used, and computes c. ----
#pragma unroll
  for (int c = 0; c < NBUF - 1; ++c)
    if (c < nch) {
      const Target t = target(c, c);
#pragma unroll
      for (int k = 0; k < kLoads; ++k) issue_one(t, k);
    }
  int stage = 0;
  for (int c = 0; c < nch; ++c) {
    const int younger = nch - 1 - c;              // chunks issued after c (at most NBUF - 2)
    if (younger >= NBUF - 2) wait_vmcnt<(NBUF - 2) * kLoads>();
    else if (NBUF > 3 && younger == NBUF - 3) wait_vmcnt<(NBUF > 3 ? NBUF - 3 : 0) * kLoads>();
    else if (NBUF > 4 && younger == NBUF - 4) wait_vmcnt<(NBUF > 4 ? NBUF - 4 : 0) * kLoads>();
    else wait_vmcnt<0>();
    lds_barrier();
    const int nxt = c + NBUF - 1;
    compute(stage, target(nxt < nch ? nxt : nch - 1, stage == 0 ? NBUF - 1 : stage - 1), nxt < nch);
    stage = stage == NBUF - 1 ? 0 : stage + 1;
  }

  // ---- merge: wave w's sums at red[w][token][row] (the ring, free once every wave is past the last chunk);
  // lane l of block (i, j) holds rows 16 i + 4 (l / 16) .. + 3 of token 16 j + l % 16 ----
  lds_barrier();
  float* red = (float*)ring;
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < TB; ++j)
      *(f32x4*)(red + (w * kTok + 16 * j + r) * kRow + 16 * i + 4 * q) = acc[i][j];
  __syncthreads();

  // item (token n, quad e4): channels 32 half + 4 e4 .. + 3 (tile rows 4 e4 ..) and their partners + 64
  uint16_t* dst_base = (g ? p.v_dst : p.k_dst) + (int64_t)head * p.dst_head_stride + 32 * half;
  const bool rot = g == 0 && p.rope_keys;
  for (int item = tid; item < kTok * 8; item += NW * 64) {
    const int n = item >> 3, e4 = item & 7;
    if (n0 + n >= p.n_tokens) continue;
    float x1[4] = {0.f, 0.f, 0.f, 0.f}, x2[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ww = 0; ww < NW; ++ww) {
      const float* row = red + (ww * kTok + n) * kRow;
      const f32x4 u = *(const f32x4*)(row + 4 * e4);
      const f32x4 v = *(const f32x4*)(row + 32 + 4 * e4);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        x1[e] += u[e];
        x2[e] += v[e];
      }
    }
    if (rot) {
      // angle of channel pair m at position t: t theta^(-2m/128) = t rev[m] revolutions, reduced to
      // [0, 1) in float64 before the hardware sine and cosine (input in revolutions)
      const double pos = (double)t_pos[n];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        double rv = pos * t_rev[32 * half + 4 * e4 + e];
        rv -= floor(rv);
        const float u = (float)rv;
        const float cs = __builtin_amdgcn_cosf(u), sn = __builtin_amdgcn_sinf(u);
        const float y1 = x1[e] * cs - x2[e] * sn;
        const float y2 = x2[e] * cs + x1[e] * sn;
        x1[e] = y1;
        x2[e] = y2;
      }
    }
    uint16_t* dst = dst_base + t_dst[n] + 4 * e4;
    u32x2 lo, hi;
    lo[0] = pack_bf16x2(x1[0], x1[1]);
    lo[1] = pack_bf16x2(x1[2], x1[3]);
    hi[0] = pack_bf16x2(x2[0], x2[1]);
    hi[1] = pack_bf16x2(x2[2], x2[3]);
    *(u32x2*)dst = lo;
    *(u32x2*)(dst + 64) = hi;
  }
}

// Sum of the split partials, RoPE on keys, bf16 rounding, scatter.  Thread =
// (token, tensor, head, quad q): channels 4q .. 4q + 3 and 64 + 4q .. + 3.
__global__ __launch_bounds__(256) void kvproj_combine_kernel(KvProjParams p) {
  const int d_kv = p.hkv * kHeadDim;
  int64_t r = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int q = (int)(r & 15);
  r >>= 4;
  const int head = (int)(r % p.hkv);
  r /= p.hkv;
  const int g = (int)(r & 1);
  const int64_t token = r >> 1;
  if (token >= p.n_tokens) return;
  const int64_t plane = (int64_t)p.n_tokens * 2 * d_kv;
  const float* src = p.part + token * 2 * d_kv + g * d_kv + head * kHeadDim + 4 * q;
  float4 x1 = make_float4(0.f, 0.f, 0.f, 0.f), x2 = x1;
  for (int s = 0; s < p.splits; ++s) {
    const float4 a = *(const float4*)(src + s * plane);
    const float4 b = *(const float4*)(src + s * plane + 64);
    x1.x += a.x; x1.y += a.y; x1.z += a.z; x1.w += a.w;
    x2.x += b.x; x2.y += b.y; x2.z += b.z; x2.w += b.w;
  }
  const int bseq = clampi(p.token_seq[token], 0, p.batch - 1);
  const int t = clampi(p.token_pos[token], 0, (p.max_pages_per_seq << p.page_shift) - 1);
  if (g == 0 && p.rope_keys) {
    const float2* cs = p.rope + (int64_t)(t < p.max_position ? t : p.max_position - 1) * kHalfDim + 4 * q;
    float a1[4] = {x1.x, x1.y, x1.z, x1.w}, a2[4] = {x2.x, x2.y, x2.z, x2.w};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const float2 c = cs[e];
      const float y1 = a1[e] * c.x - a2[e] * c.y;
      const float y2 = a2[e] * c.x + a1[e] * c.y;
      a1[e] = y1;
      a2[e] = y2;
    }
    x1 = make_float4(a1[0], a1[1], a1[2], a1[3]);
    x2 = make_float4(a2[0], a2[1], a2[2], a2[3]);
  }
  const int dp = physical_page(p.dst_page_table, bseq, p.max_pages_per_seq, t >> p.page_shift, p.dst_num_pages);
  uint16_t* dst = (g ? p.v_dst : p.k_dst) + (int64_t)dp * p.dst_page_stride +
                  (int64_t)(t & ((1 << p.page_shift) - 1)) * p.dst_slot_stride + (int64_t)head * p.dst_head_stride +
                  4 * q;
  u32x2 lo, hi;
  lo[0] = pack_bf16x2(x1.x, x1.y);
  lo[1] = pack_bf16x2(x1.z, x1.w);
  hi[0] = pack_bf16x2(x2.x, x2.y);
  hi[1] = pack_bf16x2(x2.z, x2.w);
  *(u32x2*)dst = lo;
  *(u32x2*)(dst + 64) = hi;
}

// Contract check, one thread per token: flag = min over bad tokens of 8 * token + code.
__global__ __launch_bounds__(256) void kvproj_validate_kernel(KvProjParams p, int32_t* flag) {
  const int tk = blockIdx.x * 256 + threadIdx.x;
  if (tk >= p.n_tokens) return;
  int code = 0;
  const int b = p.token_seq[tk];
  const int t = p.token_pos[tk];
  const int cap = p.max_pages_per_seq << p.page_shift;
  if (b < 0 || b >= p.batch) {
    code = 1;
  } else if (t < 0 || t >= cap || t >= p.max_position) {
    code = 2;
  } else {
    const int64_t e = (int64_t)b * p.max_pages_per_seq + (t >> p.page_shift);
    const int sp = p.page_table[e];
    const int dp = p.dst_page_table[e];
    if (sp < 0 || sp >= p.num_pages) code = 3;
    else if (dp < 0 || dp >= p.dst_num_pages) code = 4;
  }
  if (code) atomicMin(flag, tk * 8 + code);
}

__global__ void fill_kernel(int32_t* flag, int32_t v) { *flag = v; }

}  // namespace

hipError_t launch_kvproj(const KvProjParams& p, hipStream_t s) {
  const int grid = (p.work_items + 7) / 8 * 8;
  constexpr int KC = KVSHOT_KVPROJ_KC, NS = KVSHOT_KVPROJ_NS;
  if (p.splits > 1)
    hipLaunchKernelGGL((kvproj_kernel<true, KC, NS>), dim3(grid), dim3(256), 0, s, p);
  else
    hipLaunchKernelGGL((kvproj_kernel<false, KC, NS>), dim3(grid), dim3(256), 0, s, p);
  return hipGetLastError();
}

#ifndef KVSHOT_KVPROJ_DIRECT_NBUF
#define KVSHOT_KVPROJ_DIRECT_NBUF 4
#endif

hipError_t launch_kvproj_direct(const KvProjParams& p, hipStream_t s) {
  // ring stages: KVSHOT_KVPROJ_DIRECT_NBUF, fewer where (64 + 16 tile16) rows of 256 bytes per stage do not fit
  constexpr int NB = KVSHOT_KVPROJ_DIRECT_NBUF;
  constexpr int NB4 = NB * 32 * 1024 <= 150 * 1024 ? NB : 4;
  const dim3 grid((p.work_items + 7) / 8 * 8), block(256);
  switch (p.tile16) {
    case 1: hipLaunchKernelGGL((kvproj_direct_kernel<1, NB>), grid, block, 0, s, p); break;
    case 2: hipLaunchKernelGGL((kvproj_direct_kernel<2, NB>), grid, block, 0, s, p); break;
    case 3: hipLaunchKernelGGL((kvproj_direct_kernel<3, NB>), grid, block, 0, s, p); break;
    case 4: hipLaunchKernelGGL((kvproj_direct_kernel<4, NB4>), grid, block, 0, s, p); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_kvproj_combine(const KvProjParams& p, hipStream_t s) {
  const int64_t threads = (int64_t)p.n_tokens * 2 * p.hkv * 16;
  hipLaunchKernelGGL(kvproj_combine_kernel, dim3((unsigned)((threads + 255) / 256)), dim3(256), 0, s, p);
  return hipGetLastError();
}

hipError_t launch_kvproj_validate(const KvProjParams& p, int32_t* flag, hipStream_t s) {
  hipLaunchKernelGGL(fill_kernel, dim3(1), dim3(1), 0, s, flag, (int32_t)0x7fffffff);
  hipLaunchKernelGGL(kvproj_validate_kernel, dim3((p.n_tokens + 255) / 256), dim3(256), 0, s, p, flag);
  return hipGetLastError();
}

}  // namespace kvshot
