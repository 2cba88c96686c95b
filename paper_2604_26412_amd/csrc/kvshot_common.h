// Internal definitions shared by the draft-attention kernels and the host API.
//
// Device-side index code lives here once: logical token -> (page, slot) ->
// element offset, draft position, and the tree ancestry of a wave's nodes.
// The attention kernels and the debug exports both call these functions.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace kvshot {

constexpr int kHeadDim = 128;
constexpr int kHalfDim = 64;          // RoPE pairs (m, m + 64)
constexpr int kBlockKeys = 32;        // keys per inner-loop block (one 32x32 MFMA tile)
constexpr int kMaxDraft = 64;         // tree masks are 64-bit
constexpr int kMaxSplits = 64;
constexpr int kMaxRows = 256;         // G * queries per (sequence, KV head)

// Everything one attention launch needs; passed by value.
struct AttnParams {
  const void* q;                // [B][nq][Hq][D]
  const void* k_pages;
  const void* v_pages;
  const int32_t* page_table;    // [B][max_pages_per_seq]
  const int32_t* ctx_lens;      // [B]
  const void* draft_k;          // [B][max_draft][Hkv][D]
  const void* draft_v;
  const int32_t* step_offsets;  // [B] (step mode) or null
  const int32_t* parents;       // [B][n_nodes] (tree mode) or null
  const int32_t* query_nodes;   // [B][nq] tree node of each query row, or null (row j is node j)
  const int32_t* pos_base;      // [B] position of draft step 0 / tree depth 0, or null (the prefix length)
  const float2* rope;           // [max_position][64] (cos, sin)
  void* out;                    // [B][nq][Hq][D]
  float* lse;                   // [B][nq][Hq] or null
  float* part_o;                // [B][Hkv][rows_pad][splits][D]
  float2* part_ml;              // [B][Hkv][rows_pad][splits] (max in log2 units, sum)
  int64_t page_stride, head_stride, slot_stride;  // elements
  int32_t batch, nq, hq, hkv, group;
  int32_t page_shift, max_pages_per_seq, num_pages, max_draft;
  int32_t rows, rows_pad;       // rows = group * nq
  int32_t splits, blocks_per_split, max_ctx;
  int32_t row_groups;           // workgroups sharing one (sequence, KV head, split), each with its own rows
  int32_t max_position;
  int32_t tree;                 // 0 step, 1 tree
  int32_t n_nodes;              // tree mode: draft-tree nodes (draft keys) per sequence
  int32_t out_fp32;
  float qscale;                 // softmax scale * log2(e): scores come out in log2 units
  // Length-balanced schedule (batch <= 64, 32-row tiles, one-wave workgroups): `items` work items
  // per KV head are shared out over the sequences in proportion to their lengths
  // (balanced_schedule).  Item i of KV head h writes its partial at rows ((h * items + i) *
  // rows_pad + r); a sequence's items are consecutive.
  int32_t balanced;
  int32_t items;
  int32_t min_chunk;            // blocks per item at least
  int32_t* seq_splits;          // [2][64]: each sequence's split count, then its first item, for the combine
};

struct CombineParams {
  const float* part_o;
  const float2* part_ml;
  void* out;
  float* lse;
  int32_t batch, nq, hq, hkv, group, rows, rows_pad, splits, out_fp32;
  // balanced schedule: each sequence's split count and first item ([2][64]), written by the attention
  // kernel, and the items per KV head (null / 0: every sequence has `splits` splits)
  const int32_t* seq_splits;
  int32_t items;
};

// ---------------------------------------------------------------------------
// bf16 helpers (bit patterns in uint16)
// ---------------------------------------------------------------------------
__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// Round-to-nearest-even float -> bf16 bits (compiles to v_cvt_pk_bf16_f32 on gfx950).
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
  bf16x2_t v;
  v[0] = (__bf16)lo;
  v[1] = (__bf16)hi;
  return __builtin_bit_cast(uint32_t, v);
}

// ---------------------------------------------------------------------------
// index code
// ---------------------------------------------------------------------------

// Prefix length actually served: clamped to what the page table row can hold.
__device__ __forceinline__ int clamp_ctx(int t, int max_pages_per_seq, int page_shift) {
  const int cap = max_pages_per_seq << page_shift;
  return t < 0 ? 0 : (t > cap ? cap : t);
}

// Physical page holding logical page `lpage` of sequence b (clamped into the pool).
__device__ __forceinline__ int physical_page(const int32_t* page_table, int b, int max_pages_per_seq,
                                             int lpage, int num_pages) {
  int pid = page_table[(int64_t)b * max_pages_per_seq + lpage];
  pid = pid < 0 ? 0 : pid;
  return pid >= num_pages ? num_pages - 1 : pid;
}

// Element offset of (page, kv_head, slot, d = 0).
__device__ __forceinline__ int64_t kv_offset(int pid, int head, int slot, int64_t page_stride,
                                             int64_t head_stride, int64_t slot_stride) {
  return (int64_t)pid * page_stride + (int64_t)head * head_stride + (int64_t)slot * slot_stride;
}

// The hardware hands workgroup `id` of a 1-D grid to XCD id % 8.  Renumber so
// that each XCD works through a contiguous range of work items (neighbouring
// items, which share K/V or page-table rows, then share that XCD's L2).
__device__ __forceinline__ int xcd_remap(int id, int n) {
#ifdef KVSHOT_NO_XCD_REMAP
  return id;
#endif
  if ((n & 7) != 0) return id;
  return (id & 7) * (n >> 3) + (id >> 3);
}

// Position of draft step 0 (tree depth 0) of sequence b: the caller's
// pos_base[b] when given (clamped to [0, max_position]; positions are clamped
// to the RoPE table again where used), else the prefix length T.
__device__ __forceinline__ int position_base(const AttnParams& p, int b, int T) {
  if (!p.pos_base) return T;
  const int v = p.pos_base[b];
  return v < 0 ? 0 : (v > p.max_position ? p.max_position : v);
}

// Tree node whose query sits in query row j of sequence b (clamped to the tree).
__device__ __forceinline__ int query_node(const AttnParams& p, int b, int j) {
  if (!p.query_nodes) return j;
  const int v = p.query_nodes[(int64_t)b * p.nq + j];
  return v < 0 ? 0 : (v >= p.n_nodes ? p.n_nodes - 1 : v);
}

// Length-balanced split schedule, evaluated by one wave (batch <= 64, lane b = sequence b).
// Sequence b has nb_b = ceil(T_b / 32) prefix blocks (T_b clamped as the kernels clamp it).  The
// chunk is the smallest multiple of min_chunk whose split counts splits_b = max(1, ceil(nb_b /
// chunk)) sum to at most `items` (or the longest prefix, when even one split each does not fit).
// Sequence b owns work items [first_b, first_b + splits_b); its prefix is cut evenly, split s
// covering blocks [s per_b, (s + 1) per_b) with per_b = ceil(nb_b / splits_b) <= chunk, so the
// last split is never empty.  A pure function of the lengths.
struct BalancedSlot {
  int ctx;      // this lane's sequence: prefix length (clamped)
  int splits;   // its split count
  int per;      // its blocks per split
  int first;    // exclusive prefix of split counts
};
// Wave-wide sum and prefix of small non-negative per-lane values (< 2^bits) from
// bit-plane ballots: no cross-lane data movement through LDS, so no LDS latency
// on the chain.
__device__ __forceinline__ int wave_sum_small(int v, int bits) {
  int total = 0;
  for (int bit = 0; bit < bits; ++bit) total += __popcll(__ballot((v >> bit) & 1)) << bit;
  return total;
}
__device__ __forceinline__ int wave_exclusive_prefix_small(int v, int bits, int lane) {
  const uint64_t below = lane == 0 ? 0ull : (~0ull >> (64 - lane));   // lanes < lane
  int pre = 0;
  for (int bit = 0; bit < bits; ++bit) pre += __popcll(__ballot((v >> bit) & 1) & below) << bit;
  return pre;
}

// ceil(a / c) for 0 <= a <= 2^25 and uniform c >= 1: a float reciprocal estimate (within one of the
// quotient at these sizes), corrected by one
__device__ __forceinline__ int ceil_div_small(int a, int c, float rc) {
  const int num = a + c - 1;
  int q = (int)((float)num * rc);
  if (q * c > num) --q;
  else if ((q + 1) * c <= num) ++q;
  return q;
}

__device__ __forceinline__ BalancedSlot balanced_schedule(const int32_t* ctx_lens, int batch, int max_ctx,
                                                          int max_pages_per_seq, int page_shift, int items,
                                                          int min_chunk, int lane) {
  int nb = 0, t = 0;
  if (lane < batch) {
    t = clamp_ctx(ctx_lens[lane], max_pages_per_seq, page_shift);
    t = t > max_ctx ? max_ctx : t;
    nb = (t + kBlockKeys - 1) / kBlockKeys;
  }
  // the longest prefix, by a bit-serial wave max (block counts <= 2^25: prefixes <= 2^30 keys)
  int maxnb = 0;
  for (int bit = 25; bit >= 0; --bit) {
    const int cand = maxnb | (1 << bit);
    if (__ballot(nb >= cand)) maxnb = cand;
  }
  // a sequence takes at most kMaxSplits items (what the combine merges)
  auto splits_of = [&](int chunk, float rc) {
    return lane < batch ? min(kMaxSplits, max(1, ceil_div_small(nb, chunk, rc))) : 0;
  };
  auto total_splits = [&](int chunk) {
    return wave_sum_small(splits_of(chunk, 1.0f / (float)chunk), 7);
  };
  // chunk = min_chunk * k: the smallest k in [1, kmax] that fits (kmax covers the longest prefix)
  const int kmax = max(1, (maxnb + min_chunk - 1) / min_chunk);
  int lo = 1, hi = kmax;
  while (lo < hi) {
    const int mid = (lo + hi) >> 1;
    if (total_splits(mid * min_chunk) <= items) hi = mid;
    else lo = mid + 1;
  }
  const int chunk = lo * min_chunk;
  BalancedSlot r;
  r.ctx = t;
  r.splits = splits_of(chunk, 1.0f / (float)chunk);
  r.per = lane < batch ? (nb + r.splits - 1) / r.splits : 0;
  r.first = wave_exclusive_prefix_small(r.splits, 7, lane);
  return r;
}

// Element offset of draft row s of sequence b, KV head h.
__device__ __forceinline__ int64_t draft_offset(int b, int s, int h, int max_draft, int hkv) {
  return (((int64_t)b * max_draft + s) * hkv + h) * kHeadDim;
}

// Tree ancestry of the (up to 64) nodes of one sequence, one node per lane.
// Returns the ancestor-or-self bitmask of node `lane` and sets its depth.
// Pointer jumping: after k rounds each lane holds the ancestors within
// distance < 2^k and a pointer to the one at distance 2^k; six rounds cover
// any chain of 64 nodes.  A parent outside {-1} U [0, i) is treated as a root.
__device__ __forceinline__ uint64_t tree_ancestry_wave(const int32_t* parents_row, int n, int lane, int* depth) {
  int p = -1;
  if (lane < n) {
    p = parents_row[lane];
    if (p < -1 || p >= lane) p = -1;
  }
  uint64_t anc = lane < n ? (1ull << lane) : 0ull;
  int jump = p;
#pragma unroll
  for (int it = 0; it < 6; ++it) {
    const int src = jump >= 0 ? jump : lane;
    const uint32_t lo = __shfl((uint32_t)anc, src);
    const uint32_t hi = __shfl((uint32_t)(anc >> 32), src);
    const int jj = __shfl(jump, src);
    if (jump >= 0) {
      anc |= ((uint64_t)hi << 32) | lo;
      jump = jj;
    }
  }
  *depth = lane < n ? __popcll(anc) - 1 : 0;
  return anc;
}

}  // namespace kvshot

// Launchers (defined in the .hip files).
namespace kvshot {
hipError_t launch_attn_mfma(const AttnParams& p, int kernel_row_tiles, hipStream_t s);
hipError_t launch_attn_tall(const AttnParams& p, hipStream_t s);
int tall_waves_per_wg();
int tall_max_blocks();
hipError_t launch_attn_generic(const AttnParams& p, int bf16_in, hipStream_t s);
hipError_t launch_combine(const CombineParams& p, hipStream_t s);
hipError_t launch_gather_kv(const AttnParams& p, int max_ctx, void* k_dense, void* v_dense, int bf16, hipStream_t s);
hipError_t launch_tree_mask(const int32_t* parents, int batch, int n, uint64_t* anc, int32_t* depth, hipStream_t s);
hipError_t launch_validate(const AttnParams& p, int max_ctx_hint, int32_t* flag, hipStream_t s);
hipError_t launch_stream_read(const void* src, int64_t bytes, void* sink, int blocks, hipStream_t s);
int mfma_waves_per_wg(int row_tiles);
int mfma_wgs_per_cu(int kernel_row_tiles);
int mfma_key_streams(int kernel_row_tiles);
int mfma_kernel_row_tiles(int row_tiles);
}  // namespace kvshot
