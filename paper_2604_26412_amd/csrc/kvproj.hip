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
// the operand prefetches still in flight); the clobber keeps the compiler from
// moving LDS accesses across it.
__device__ __forceinline__ void lds_barrier() { asm volatile("s_barrier" ::: "memory"); }

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
  auto target = [&](int c, int stage) {
    const int k0 = k_first + c * KC;
    const int l = k0 / d_kv;
    const int rem = k0 - l * d_kv;
    Target t;
    t.w = wsrc + k0;
    t.x = t_layer[g][l] + (int64_t)(rem >> 7) * p.head_stride + (rem & 127);
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
  // One chunk from `stage`, with the loads of a later chunk (`nt`) issued one per four MFMAs (so
  // no wave stalls on a burst of load issues before its first MFMA) and the next k-step's
  // fragments read during the current one.  The order is pinned with scheduling barriers.
  auto compute = [&](int stage, const Target& nt) {
    const uint16_t* A = smem + stage * 2 * kStageElems + (128 * wc + (lane & 31)) * KC;
    const uint16_t* B = smem + stage * 2 * kStageElems + kStageElems + (128 * wt + (lane & 31)) * KC;
    bf16x8 a[2][4], b[2][4];
    auto read = [&](int st, bf16x8 (&fa)[4], bf16x8 (&fb)[4]) {
#pragma unroll
      for (int i = 0; i < 4; ++i) fa[i] = as_bf16x8(*(const u32x4*)(A + 32 * i * KC + frag_off[st]));
#pragma unroll
      for (int j = 0; j < 4; ++j) fb[j] = as_bf16x8(*(const u32x4*)(B + 32 * j * KC + frag_off[st]));
    };
    read(0, a[0], b[0]);
#pragma unroll
    for (int st = 0; st < kSteps; ++st) {
      if (st + 1 < kSteps) read(st + 1, a[(st + 1) & 1], b[(st + 1) & 1]);
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

  // ---- main loop.  Chunks 0 .. NS - 2 are issued up front; iteration c waits for chunk c (the
  // NS - 2 younger chunks may stay in flight), passes a barrier (every wave is then done with
  // chunk c - 1, so its stage is free) and computes c while issuing chunk c + NS - 1 into that
  // stage.  Loads past the last chunk re-read it into a stage nobody reads again. ----
#pragma unroll
  for (int c = 0; c < NS - 1; ++c) {
    const Target t = target(c < nch ? c : nch - 1, c);
#pragma unroll
    for (int idx = 0; idx < 2 * kLoads; ++idx) issue_one(t, idx);
  }
  int stage = 0;
  for (int c = 0; c < nch; ++c) {
    wait_vmcnt<(NS - 2) * 2 * kLoads>();
    lds_barrier();
    const int nxt = c + NS - 1;
    compute(stage, target(nxt < nch ? nxt : nch - 1, stage == 0 ? NS - 1 : stage - 1));
    stage = stage == NS - 1 ? 0 : stage + 1;
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
