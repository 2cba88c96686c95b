// Level-wise draft-tree growth (Sec. 3.5, tree (8, 10, 60)): top-k with
// log-softmax over the vocabulary, best-first frontier expansion and the final
// selection of the tree's nodes.
//
// kvshot_topk_logprobs.  A level's frontier holds few rows (10 per sequence),
// each a whole vocabulary, so one workgroup per row would leave most of the
// chip idle: every row is cut into chunks of 16384 logits, one workgroup of
// 256 threads per chunk, 64 logits per thread held in registers (all eight
// 16-byte loads of a thread issued together; element loads where rows are not
// 16-byte aligned).  Per chunk:
//   * each thread's max and its sum of exp(z - max): the chunk's log-sum-exp
//     parts (m, s), combined across lanes and waves with the usual rescale;
//   * a threshold T: the k-th largest of the maxima of the 16 lane rows (16
//     lanes x 64 logits each).  Those k maxima are k distinct logits >= T, so
//     every logit of the chunk's top k is >= T;
//   * the logits >= T (threads whose max is below T skip the scan) are
//     appended to an LDS list, usually a few dozen, and ranked by counting
//     the entries that beat each one.  Should more than 1024 pass (a flat
//     distribution with many equal logits), k rounds of workgroup arg-max
//     over the registers give the same k pairs.
// Reductions across lanes use DPP moves within 16-lane rows and lane reads
// across rows; no LDS round trip.  A pair (logit, token) travels as one
// 64-bit key -- the logit's bits mapped to an unsigned order, then the
// complemented token id -- so "beats" is one unsigned comparison.
// A row of one chunk finishes in place; otherwise each chunk writes (k best
// pairs, m, s) to the workspace and a merge kernel, one workgroup per row,
// combines the log-sum-exp parts and ranks the chunks' k best keys the same way.
// Order of the pairs: logit descending, then token id ascending, so every
// row's result is unique.
//
// kvshot_tree_expand / kvshot_tree_select: one workgroup of 256 threads per
// sequence, one candidate per thread (at most 256).  Candidate c is ordered by
// (score descending, c ascending); c enumerates (frontier node, proposal rank)
// or (depth, rank in level), so that order is exactly the tie rule of the
// reading.  Each candidate's rank is the number of keys that beat it; the
// expansion writes ranks below k, the selection keeps ranks below n and
// numbers the kept ones in (depth, rank) order with a ballot prefix count.
#include "kvshot_tree.h"

#include <hip/hip_runtime.h>

#include <cstdint>
#include <climits>

namespace {

constexpr int kTopK = 16;                       // largest k
constexpr int kMaxCand = 256;                   // candidates of one expansion or selection
constexpr int kThreads = 256;
constexpr int kPerThread = 64;                  // logits per thread, in registers
constexpr int kChunk = kThreads * kPerThread;   // logits per workgroup
constexpr int kMaxChunks = 64;                  // vocabulary <= 64 chunks
constexpr int kCandCap = 1024;                  // threshold-passing logits kept in LDS
constexpr int kRecord = kTopK + 1;              // workspace words (64-bit) per chunk: keys, then (m, s)
constexpr float kLog2e = 1.4426950408889634f;

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// ---- keys: larger key = larger value, then smaller index

__device__ __forceinline__ uint32_t ordered(float v) {
  const uint32_t b = __float_as_uint(v);
  return b ^ ((uint32_t)((int32_t)b >> 31) | 0x80000000u);
}

__device__ __forceinline__ uint64_t pair_key(float v, int i) {
  return ((uint64_t)ordered(v) << 32) | (uint32_t)~(uint32_t)i;
}

__device__ __forceinline__ float key_value(uint64_t key) {
  const uint32_t o = (uint32_t)(key >> 32);
  return __uint_as_float((o & 0x80000000u) ? (o ^ 0x80000000u) : ~o);
}

__device__ __forceinline__ int key_index(uint64_t key) { return (int)~(uint32_t)key; }

// ---- lane reductions: DPP within a row of 16 lanes, lane reads across rows

constexpr int kQuadSwap1 = 0xB1;    // quad_perm [1, 0, 3, 2]
constexpr int kQuadSwap2 = 0x4E;    // quad_perm [2, 3, 0, 1]
constexpr int kHalfMirror = 0x141;  // row_half_mirror: lane i <- 7 - i within 8
constexpr int kMirror = 0x140;      // row_mirror: lane i <- 15 - i within 16

template <int C>
__device__ __forceinline__ float dpp(float v) {
  return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), C, 0xF, 0xF, false));
}

template <int C>
__device__ __forceinline__ uint64_t dpp(uint64_t v) {
  const uint32_t lo = (uint32_t)__builtin_amdgcn_mov_dpp((int)(uint32_t)v, C, 0xF, 0xF, false);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_mov_dpp((int)(uint32_t)(v >> 32), C, 0xF, 0xF, false);
  return ((uint64_t)hi << 32) | lo;
}

// every lane of a 16-lane row gets the row's max / sum
__device__ __forceinline__ float row_max(float v) {
  v = fmaxf(v, dpp<kQuadSwap1>(v));
  v = fmaxf(v, dpp<kQuadSwap2>(v));
  v = fmaxf(v, dpp<kHalfMirror>(v));
  return fmaxf(v, dpp<kMirror>(v));
}

__device__ __forceinline__ float row_sum(float v) {
  v += dpp<kQuadSwap1>(v);
  v += dpp<kQuadSwap2>(v);
  v += dpp<kHalfMirror>(v);
  return v + dpp<kMirror>(v);
}

__device__ __forceinline__ uint64_t umax(uint64_t a, uint64_t b) { return a > b ? a : b; }

__device__ __forceinline__ uint64_t row_max(uint64_t v) {
  v = umax(v, dpp<kQuadSwap1>(v));
  v = umax(v, dpp<kQuadSwap2>(v));
  v = umax(v, dpp<kHalfMirror>(v));
  return umax(v, dpp<kMirror>(v));
}

__device__ __forceinline__ float lane_read(float v, int l) {
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), l));
}

__device__ __forceinline__ uint64_t lane_read(uint64_t v, int l) {
  const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)v, l);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(v >> 32), l);
  return ((uint64_t)hi << 32) | lo;
}

// whole-wave results, the same in every lane
__device__ __forceinline__ float wave_max(float v) {
  v = row_max(v);
  return fmaxf(fmaxf(lane_read(v, 0), lane_read(v, 16)), fmaxf(lane_read(v, 32), lane_read(v, 48)));
}

__device__ __forceinline__ float wave_sum(float v) {
  v = row_sum(v);
  return (lane_read(v, 0) + lane_read(v, 16)) + (lane_read(v, 32) + lane_read(v, 48));
}

__device__ __forceinline__ uint64_t wave_max(uint64_t v) {
  v = row_max(v);
  return umax(umax(lane_read(v, 0), lane_read(v, 16)), umax(lane_read(v, 32), lane_read(v, 48)));
}

// s * e^(m - M), zero for an empty part
__device__ __forceinline__ float rescale(float s, float m, float M) {
  return m == -INFINITY ? 0.0f : s * __builtin_amdgcn_exp2f((m - M) * kLog2e);
}

// number of the n keys in LDS that beat `key`
__device__ __forceinline__ int rank_of(const uint64_t* keys, int n, uint64_t key) {
  int rank = 0;
#pragma unroll 8
  for (int j = 0; j < n; ++j) rank += keys[j] > key ? 1 : 0;
  return rank;
}

__device__ __forceinline__ uint64_t pack_ms(float m, float s) {
  return ((uint64_t)__float_as_uint(s) << 32) | __float_as_uint(m);
}

// One chunk of one row.  Writes the final tokens / log-probabilities when the
// row is a single chunk, else the chunk's record in `ws`.
template <bool BF16>
__global__ __launch_bounds__(kThreads) void topk_chunk_kernel(const void* logits, int vocab, int64_t row_stride, int k,
                                                              int chunks, bool vec, int32_t* tokens,
                                                              float* logprobs, uint64_t* ws) {
  __shared__ float row_m[16], row_s[16];
  __shared__ float sh_T, sh_M, sh_S;
  __shared__ uint64_t win[4];
  __shared__ uint64_t cand[kCandCap];
  __shared__ int cand_n;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int row = blockIdx.x / chunks;
  const int chunk = blockIdx.x - row * chunks;
  const int base = chunk * kChunk;

  // logit z[8g + e] is token base + 8 (256 g + tid) + e; 16-byte loads where the rows are aligned
  float z[kPerThread];
#pragma unroll
  for (int g = 0; g < kPerThread / 8; ++g) {
    const int t0 = base + 8 * (kThreads * g + tid);
    if (vec && t0 + 8 <= vocab) {
      if constexpr (BF16) {
        const u32x4 q = *(const u32x4*)((const uint16_t*)logits + row * row_stride + t0);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          z[8 * g + 2 * e] = __uint_as_float(q[e] << 16);
          z[8 * g + 2 * e + 1] = __uint_as_float(q[e] & 0xffff0000u);
        }
      } else {
        const float* r = (const float*)logits + row * row_stride + t0;
        const float4 a = *(const float4*)r, c = *(const float4*)(r + 4);
        z[8 * g + 0] = a.x; z[8 * g + 1] = a.y; z[8 * g + 2] = a.z; z[8 * g + 3] = a.w;
        z[8 * g + 4] = c.x; z[8 * g + 5] = c.y; z[8 * g + 6] = c.z; z[8 * g + 7] = c.w;
      }
    } else {
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int t = t0 + e;
        float v = -INFINITY;
        if (t < vocab) {
          if constexpr (BF16)
            v = __uint_as_float((uint32_t)((const uint16_t*)logits)[row * row_stride + t] << 16);
          else
            v = ((const float*)logits)[row * row_stride + t];
        }
        z[8 * g + e] = v;
      }
    }
  }
  // token of z[i] = tbase + off(i), off(i) a constant of the unrolled loops; comparisons of tokens are
  // made on offsets so that no per-element token is ever held in a register
  const int tbase = base + 8 * tid;
  const int vrel = vocab - tbase;                 // z[i] is a logit iff off(i) < vrel
  auto off = [](int i) { return 8 * kThreads * (i >> 3) + (i & 7); };

  // the thread's log-sum-exp part, then its row's
  float mt = -INFINITY;
#pragma unroll
  for (int i = 0; i < kPerThread; ++i) mt = fmaxf(mt, z[i]);
  float st = 0.0f;
  if (mt != -INFINITY) {
    const float off = mt * kLog2e;
#pragma unroll
    for (int i = 0; i < kPerThread; ++i) st += __builtin_amdgcn_exp2f(fmaf(z[i], kLog2e, -off));
  }
  const float mr = row_max(mt);
  const float sr = row_sum(rescale(st, mt, mr));
  if ((lane & 15) == 0) {
    row_m[tid >> 4] = mr;
    row_s[tid >> 4] = sr;
  }
  if (tid == 0) cand_n = 0;
  __syncthreads();
  if (tid < 16) {
    // T = the k-th largest row maximum (k <= 16)
    const float v = row_m[tid];
    int greater = 0, equal = 0;
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      greater += row_m[j] > v ? 1 : 0;
      equal += row_m[j] == v ? 1 : 0;
    }
    if (greater < k && greater + equal >= k) sh_T = v;
    if (tid == 0) {
      float M = -INFINITY;
#pragma unroll
      for (int j = 0; j < 16; ++j) M = fmaxf(M, row_m[j]);
      float S = 0.0f;
#pragma unroll
      for (int j = 0; j < 16; ++j) S += rescale(row_s[j], row_m[j], M);
      sh_M = M;
      sh_S = S;
    }
  }
  __syncthreads();
  const float T = sh_T;

  // logits >= T into the LDS list
  if (mt >= T) {
#pragma unroll
    for (int i = 0; i < kPerThread; ++i) {
      if ((z[i] >= T) & (off(i) < vrel)) {
        const int p = atomicAdd(&cand_n, 1);
        if (p < kCandCap) cand[p] = pair_key(z[i], tbase + off(i));
      }
    }
  }
  __syncthreads();
  const int n = cand_n;

  const bool final_row = chunks == 1;
  const float lse = sh_M + logf(sh_S);
  uint64_t* rec = final_row ? nullptr : ws + (int64_t)blockIdx.x * kRecord;
  auto emit = [&](int r, uint64_t key) {
    if (final_row) {
      tokens[(int64_t)row * k + r] = key_index(key);
      logprobs[(int64_t)row * k + r] = key_value(key) - lse;
    } else {
      rec[r] = key;
    }
  };
  if (!final_row && tid == 0) rec[kTopK] = pack_ms(sh_M, sh_S);

  if (n <= kCandCap) {
    for (int c = tid; c < n; c += kThreads) {
      const uint64_t key = cand[c];
      const int rank = rank_of(cand, n, key);
      if (rank < k) emit(rank, key);
    }
    if (tid >= n && tid < k) emit(tid, 0ull);   // a chunk with fewer than k logits: keys below every pair
    return;
  }

  // many logits tie at the threshold: k rounds of workgroup arg-max, each
  // taking the best pair ordered after the previous winner (lv, li); token
  // ids relative to tbase
  float lv = INFINITY;
  int li = -1;
  for (int r = 0; r < k; ++r) {
    const int lrel = li - tbase;
    float bv = -INFINITY;
    int bi = -1;                                  // element index: tokens rise with it, so the first of equal
#pragma unroll                                    // values is the best and a later equal one never replaces it
    for (int i = 0; i < kPerThread; ++i) {
      const float v = z[i];
      const bool after = (v < lv) | ((v == lv) & (off(i) > lrel));
      if ((off(i) < vrel) & after & (v > bv)) {
        bv = v;
        bi = i;
      }
    }
    const uint64_t best = wave_max(bi < 0 ? (uint64_t)0 : pair_key(bv, tbase + off(bi)));
    if (lane == 0) win[w] = best;
    __syncthreads();
    const uint64_t top = umax(umax(win[0], win[1]), umax(win[2], win[3]));
    lv = key_value(top);
    li = key_index(top);
    if (tid == 0) emit(r, top);
    __syncthreads();
  }
}

// One row of several chunks: combine the chunks' log-sum-exp parts and rank
// their k best keys.
__global__ __launch_bounds__(kThreads) void topk_merge_kernel(int k, int chunks, const uint64_t* ws, int32_t* tokens,
                                                              float* logprobs) {
  __shared__ uint64_t keys[kMaxChunks * kTopK];
  __shared__ float sh_lse;
  const int tid = threadIdx.x, lane = tid & 63;
  const int row = blockIdx.x;
  const uint64_t* rec = ws + (int64_t)row * chunks * kRecord;
  const int n = chunks * k;
  for (int c = tid; c < n; c += kThreads) {
    const int j = c / k;
    keys[c] = rec[j * kRecord + (c - j * k)];
  }
  if (tid < 64) {
    const uint64_t ms = lane < chunks ? rec[lane * kRecord + kTopK] : pack_ms(-INFINITY, 0.0f);
    const float m = __uint_as_float((uint32_t)ms), s = __uint_as_float((uint32_t)(ms >> 32));
    const float M = wave_max(m);
    const float S = wave_sum(rescale(s, m, M));
    if (lane == 0) sh_lse = M + logf(S);
  }
  __syncthreads();
  const float lse = sh_lse;
  for (int c = tid; c < n; c += kThreads) {
    const uint64_t key = keys[c];
    const int rank = rank_of(keys, n, key);
    if (rank < k) {
      tokens[(int64_t)row * k + rank] = key_index(key);
      logprobs[(int64_t)row * k + rank] = key_value(key) - lse;
    }
  }
}

int chunks_for(int vocab) { return (vocab + kChunk - 1) / kChunk; }

__global__ __launch_bounds__(kThreads) void tree_expand_kernel(int frontier, int proposals, int k, const float* scores,
                                                               const int32_t* tokens, const float* logprobs,
                                                               int32_t* next_parent, int32_t* next_tokens,
                                                               float* next_scores) {
  __shared__ uint64_t keys[kMaxCand];
  const int b = blockIdx.x, c = threadIdx.x;
  const int C = frontier * proposals;
  float sc = 0.0f;
  uint64_t key = 0ull;
  if (c < C) {
    sc = scores[(int64_t)b * frontier + c / proposals] + logprobs[(int64_t)b * C + c];
    key = pair_key(sc, c);
    keys[c] = key;
  }
  __syncthreads();
  if (c < C) {
    const int rank = rank_of(keys, C, key);
    if (rank < k) {
      const int64_t o = (int64_t)b * k + rank;
      next_parent[o] = c / proposals;
      next_tokens[o] = tokens[(int64_t)b * C + c];
      next_scores[o] = sc;
    }
  }
}

__global__ __launch_bounds__(kThreads) void tree_select_kernel(int depth, int k, int n, const int32_t* level_parent,
                                                               const int32_t* level_tokens, const float* level_scores,
                                                               int32_t* parents, int32_t* tokens, int32_t* depths,
                                                               float* scores) {
  __shared__ uint64_t keys[kMaxCand];
  __shared__ int pos[kMaxCand];
  __shared__ int wave_kept[4];
  const int b = blockIdx.x, c = threadIdx.x, lane = c & 63, w = c >> 6;
  const int C = depth * k;
  // candidate c = (depth d, rank i) of sequence b sits at level block d: [depth][batch][k]
  const int64_t at = ((int64_t)(c / k) * gridDim.x + b) * k + c % k;
  float sc = 0.0f;
  uint64_t key = 0ull;
  if (c < C) {
    sc = level_scores[at];
    key = pair_key(sc, c);
    keys[c] = key;
  }
  __syncthreads();
  const bool kept = c < C && rank_of(keys, C, key) < n;
  // output position: kept candidates before c, in (depth, rank) order
  const uint64_t mask = __ballot(kept);
  if (lane == 0) wave_kept[w] = __popcll(mask);
  __syncthreads();
  int p = __popcll(mask & ((1ull << lane) - 1ull));
  for (int j = 0; j < w; ++j) p += wave_kept[j];
  if (c < kMaxCand) pos[c] = kept ? p : -1;
  __syncthreads();
  if (kept) {
    const int d = c / k;
    int par = level_parent[at];
    par = par < 0 ? 0 : (par >= k ? k - 1 : par);
    const int64_t o = (int64_t)b * n + p;
    parents[o] = d == 0 ? -1 : pos[(d - 1) * k + par];
    tokens[o] = level_tokens[at];
    depths[o] = d;
    scores[o] = sc;
  }
}

bool aligned(const void* p, unsigned a) { return ((uintptr_t)p % a) == 0; }

}  // namespace

extern "C" int64_t kvshot_topk_workspace_bytes(int32_t rows, int32_t vocab) {
  if (rows < 1 || vocab < 1 || chunks_for(vocab) > kMaxChunks) return -1;
  const int chunks = chunks_for(vocab);
  return chunks == 1 ? 0 : (int64_t)rows * chunks * kRecord * (int64_t)sizeof(uint64_t);
}

extern "C" kvshot_status kvshot_topk_logprobs(const void* logits, int32_t dtype, int32_t rows, int32_t vocab,
                                              int64_t row_stride, int32_t k, int32_t* tokens, float* logprobs,
                                              void* workspace, int64_t workspace_bytes, void* stream) {
  if (!logits || !tokens || !logprobs || rows < 1 || vocab < 1 || k < 1 || k > kTopK || k > vocab)
    return KVSHOT_ERR_INVALID_ARG;
  if (dtype != KVSHOT_BF16 && dtype != KVSHOT_FP32) return KVSHOT_ERR_INVALID_ARG;
  const unsigned elem = dtype == KVSHOT_BF16 ? 2u : 4u;
  if (row_stride < vocab || !aligned(logits, elem) || !aligned(tokens, 4) || !aligned(logprobs, 4))
    return KVSHOT_ERR_INVALID_ARG;
  const bool vec = aligned(logits, 16) && (row_stride * elem) % 16 == 0;
  const int chunks = chunks_for(vocab);
  if (chunks > kMaxChunks || (int64_t)rows * chunks > INT_MAX) return KVSHOT_ERR_INVALID_ARG;
  const int64_t need = kvshot_topk_workspace_bytes(rows, vocab);
  if (need > 0 && (!workspace || workspace_bytes < need || !aligned(workspace, 8))) return KVSHOT_ERR_INVALID_ARG;
  hipStream_t s = (hipStream_t)stream;
  uint64_t* ws = (uint64_t*)workspace;
  const dim3 grid((unsigned)(rows * chunks));
  if (dtype == KVSHOT_BF16)
    hipLaunchKernelGGL(topk_chunk_kernel<true>, grid, dim3(kThreads), 0, s, logits, (int)vocab, row_stride, (int)k,
                       chunks, vec, tokens, logprobs, ws);
  else
    hipLaunchKernelGGL(topk_chunk_kernel<false>, grid, dim3(kThreads), 0, s, logits, (int)vocab, row_stride, (int)k,
                       chunks, vec, tokens, logprobs, ws);
  if (chunks > 1)
    hipLaunchKernelGGL(topk_merge_kernel, dim3(rows), dim3(kThreads), 0, s, (int)k, chunks, ws, tokens, logprobs);
  return hipGetLastError() == hipSuccess ? KVSHOT_OK : KVSHOT_ERR_DEVICE;
}

extern "C" kvshot_status kvshot_tree_expand(int32_t batch, int32_t frontier, int32_t proposals, int32_t k,
                                            const float* scores, const int32_t* tokens, const float* logprobs,
                                            int32_t* next_parent, int32_t* next_tokens, float* next_scores,
                                            void* stream) {
  if (batch < 1 || frontier < 1 || frontier > 16 || proposals < 1 || proposals > 16 || k < 1 || k > kTopK ||
      k > frontier * proposals)
    return KVSHOT_ERR_INVALID_ARG;
  if (!scores || !tokens || !logprobs || !next_parent || !next_tokens || !next_scores) return KVSHOT_ERR_INVALID_ARG;
  hipLaunchKernelGGL(tree_expand_kernel, dim3(batch), dim3(kThreads), 0, (hipStream_t)stream, (int)frontier,
                     (int)proposals, (int)k, scores, tokens, logprobs, next_parent, next_tokens, next_scores);
  return hipGetLastError() == hipSuccess ? KVSHOT_OK : KVSHOT_ERR_DEVICE;
}

extern "C" kvshot_status kvshot_tree_select(int32_t batch, int32_t depth, int32_t k, int32_t n,
                                            const int32_t* level_parent, const int32_t* level_tokens,
                                            const float* level_scores, int32_t* parents, int32_t* tokens,
                                            int32_t* depths, float* scores, void* stream) {
  if (batch < 1 || depth < 1 || k < 1 || k > kTopK || depth * k > kMaxCand || n < 1 || n > depth * k)
    return KVSHOT_ERR_INVALID_ARG;
  if (!level_parent || !level_tokens || !level_scores || !parents || !tokens || !depths || !scores)
    return KVSHOT_ERR_INVALID_ARG;
  hipLaunchKernelGGL(tree_select_kernel, dim3(batch), dim3(kThreads), 0, (hipStream_t)stream, (int)depth, (int)k, (int)n,
                     level_parent, level_tokens, level_scores, parents, tokens, depths, scores);
  return hipGetLastError() == hipSuccess ? KVSHOT_OK : KVSHOT_ERR_DEVICE;
}
