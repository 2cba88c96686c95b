// Level-wise draft-tree growth (Sec. 3.5, tree (8, 10, 60)): top-k with
// log-softmax over the vocabulary, best-first frontier expansion and the final
// selection of the tree's nodes.
//
// kvshot_topk_logprobs.  A level's frontier holds few rows (10 per sequence),
// each a whole vocabulary, so one workgroup per row would leave most of the
// chip idle: every row is cut into chunks of 16384 logits, one workgroup of
// 256 threads per chunk, 64 logits per thread held in registers (all eight
// 16-byte loads of a thread issued together).  Per chunk:
//   * each thread's max and its sum of exp(z - max): the chunk's log-sum-exp
//     parts (m, s), combined across lanes and waves with the usual rescale;
//   * a threshold T: the k-th largest of the maxima of the 16 lane rows (16
//     lanes x 64 logits each).  Those k maxima are k distinct logits >= T, so
//     every logit of the chunk's top k is >= T;
//   * the logits >= T are appended to an LDS list, usually a few dozen, and
//     ranked by counting the entries that beat each one.  Threads first
//     append their groups of 8 logits whose max is >= T, and one thread per
//     group then appends that group's logits >= T.  Should more than 256
//     groups or 1024 logits pass (a flat distribution with many equal
//     logits), k rounds of workgroup arg-max over the registers give the same
//     k pairs.
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
// kvshot_tree_level runs the same chunk workgroups in level mode: the last
// chunk of each frontier row to finish merges that row, and the last merged
// row of each sequence expands the frontier, so a whole level is one launch.
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
#include <cfloat>
#include <climits>

namespace {

constexpr int kTopK = 16;                       // largest k
constexpr int kMaxCand = 256;                   // candidates of one expansion or selection
constexpr int kThreads = 256;
constexpr int kPerThread = 64;                  // logits per thread, in registers
constexpr int kChunk = kThreads * kPerThread;   // logits per workgroup
constexpr int kMaxChunks = 64;                  // vocabulary <= 64 chunks
constexpr int kCandCap = 1024;                  // threshold-passing logits kept in LDS
constexpr int kSlots = kThreads;                // threshold-passing groups of 8 logits kept in LDS
constexpr int kRecord = kTopK + 1;              // workspace words (64-bit) per chunk: keys, then (m, s)
constexpr int kCounterStride = 64;              // 32-bit words between two arrival counters: a 256-byte line
                                                // each, since device atomics on one line serialize
constexpr float kLog2e = 1.4426950408889634f;

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// ---- keys: larger key = larger value, then smaller index

// -0 + 0 = +0, so both zeros get one key: equal values tie, as in every float comparison
__device__ __forceinline__ uint32_t ordered(float v) {
  const uint32_t b = __float_as_uint(v + 0.0f);
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

__device__ __forceinline__ uint64_t lane_read(uint64_t v, int l) {
  const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)v, l);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(v >> 32), l);
  return ((uint64_t)hi << 32) | lo;
}

// whole-wave maximum, the same in every lane
__device__ __forceinline__ uint64_t wave_max(uint64_t v) {
  v = row_max(v);
  return umax(umax(lane_read(v, 0), lane_read(v, 16)), umax(lane_read(v, 32), lane_read(v, 48)));
}

// s * e^(m - M), zero for an empty part
__device__ __forceinline__ float rescale(float s, float m, float M) {
  return m == -INFINITY ? 0.0f : s * __builtin_amdgcn_exp2f((m - M) * kLog2e);
}

// Room for `cnt` (0..8) entries of this lane in an LDS list whose length is
// `*counter`: the lane's offset among the wave's requests from eight ballots
// (lane L asks for more than b entries), then one atomic for the whole wave.
// Called by every lane of the wave (uniform control flow).
__device__ __forceinline__ int wave_alloc(int cnt, int* counter) {
  const int lane = threadIdx.x & 63;
  const uint64_t below = (1ull << lane) - 1ull;
  int prefix = 0, total = 0;
#pragma unroll
  for (int b = 0; b < 8; ++b) {
    const uint64_t m = __ballot(cnt > b);
    prefix += __popcll(m & below);
    total += __popcll(m);
  }
  int base = 0;
  if (total > 0) {
    if (lane == 0) base = atomicAdd(counter, total);
    base = __builtin_amdgcn_readfirstlane(base);
  }
  return base + prefix;
}

// number of the n keys in LDS that beat `key`
__device__ __forceinline__ int rank_of(const uint64_t* keys, int n, uint64_t key) {
  int rank = 0;
#pragma unroll 8
  for (int j = 0; j < n; ++j) rank += keys[j] > key ? 1 : 0;
  return rank;
}

// Chunk records are written and read with agent-scope relaxed atomic stores
// and loads: the compiler gives them the device-coherence bit, so they are
// performed at the device's point of coherence and no L2 write-back or
// invalidation (a release or acquire fence) is needed for another XCD to see
// them.
__device__ __forceinline__ void store_rec(uint64_t* p, uint64_t v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ uint64_t load_rec(const uint64_t* p) {
  return __hip_atomic_load(const_cast<uint64_t*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ uint64_t pack_ms(float m, float s) {
  return ((uint64_t)__float_as_uint(s) << 32) | __float_as_uint(m);
}

// log-sum-exp of a row from its chunks' (m, s) parts (staged in LDS),
// combined in chunk order -- the same order everywhere, so every path gets the
// same float32 value
__device__ __forceinline__ float chunk_lse(const uint64_t* ms, int chunks) {
  float M = -INFINITY;
  for (int j = 0; j < chunks; ++j) M = fmaxf(M, __uint_as_float((uint32_t)ms[j]));
  float S = 0.0f;
  for (int j = 0; j < chunks; ++j) S += rescale(__uint_as_float((uint32_t)(ms[j] >> 32)), __uint_as_float((uint32_t)ms[j]), M);
  return M + logf(S);
}

// Where a tree level goes: the frontier's scores and the next frontier, plus
// the arrival counters (zero between calls) and the row records.
struct LevelArgs {
  int batch, frontier;
  const float* scores;
  int32_t* next_parent;
  int32_t* next_tokens;
  float* next_scores;
  unsigned int* counters;   // per sequence 17 lines: 16 frontier-row counters, then its own
  uint64_t* rows;           // one record per frontier row: its k best keys, then its log-sum-exp
};

// One chunk of one row.  Top-k mode (LEVEL false): writes the final tokens /
// log-probabilities when the row is a single chunk, else the chunk's record in
// `ws`.  Level mode: always writes the record; the last chunk of a row to
// arrive (device-scope counters, no waiting) merges the row, and the last row
// of a sequence expands the frontier.
template <bool BF16, bool LEVEL>
__global__ __launch_bounds__(kThreads) void topk_chunk_kernel(const void* logits, int vocab, int64_t row_stride, int k,
                                                              int chunks, bool vec, int32_t* tokens,
                                                              float* logprobs, uint64_t* ws, LevelArgs L) {
  __shared__ float row_m[16], row_s[16];
  __shared__ float sh_T, sh_M, sh_S;
  __shared__ uint64_t win[4];
  __shared__ uint64_t cand[kCandCap + 1];         // + a spare slot for writes that are thrown away
  __shared__ float4 slot_v[kSlots][2];
  __shared__ int slot_t[kSlots];
  __shared__ int cand_n, slot_n;
  __shared__ int sh_last;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int row = blockIdx.x / chunks;
  const int chunk = blockIdx.x - row * chunks;
  // Chunk c covers tokens [c * 16384, (c + 1) * 16384).  Where rows are 16-byte aligned and the
  // vocabulary is a multiple of 8 and at least one chunk long, a row's last chunk is read as the
  // 16384 tokens ending at the vocabulary's end, those of the previous chunk masked to -inf: every
  // 16-byte load of every thread is then unconditional and in flight before the first use.
  // Otherwise (short or unaligned rows) tokens are read one by one, eight at a time, -inf past
  // the end.  Logits are finite, so -inf marks exactly the elements that are not this chunk's.
  const bool shifted = vec && (vocab & 7) == 0 && vocab >= kChunk;
  const int lo = chunk * kChunk;                                   // first token of the chunk
  const int base = shifted ? min(lo, vocab - kChunk) : lo;         // first token read
  float z[kPerThread];                                             // z[8g + e]: token base + 8 (256 g + tid) + e
  const int64_t row0 = row * row_stride;
  if (shifted) {
    if constexpr (BF16) {
      const uint16_t* r = (const uint16_t*)logits + row0 + base + 8 * tid;
      u32x4 q[kPerThread / 8];
#pragma unroll
      for (int g = 0; g < kPerThread / 8; ++g) q[g] = *(const u32x4*)(r + 8 * kThreads * g);
#pragma unroll
      for (int g = 0; g < kPerThread / 8; ++g)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          z[8 * g + 2 * e] = __uint_as_float(q[g][e] << 16);
          z[8 * g + 2 * e + 1] = __uint_as_float(q[g][e] & 0xffff0000u);
        }
    } else {
      const float* r = (const float*)logits + row0 + base + 8 * tid;
      float4 q[kPerThread / 4];
#pragma unroll
      for (int g = 0; g < kPerThread / 8; ++g) {
        q[2 * g] = *(const float4*)(r + 8 * kThreads * g);
        q[2 * g + 1] = *(const float4*)(r + 8 * kThreads * g + 4);
      }
#pragma unroll
      for (int j = 0; j < kPerThread / 4; ++j) {
        z[4 * j + 0] = q[j].x;
        z[4 * j + 1] = q[j].y;
        z[4 * j + 2] = q[j].z;
        z[4 * j + 3] = q[j].w;
      }
    }
    if (base < lo) {                              // the last chunk: drop the previous chunk's tokens
      const int keep = lo - base - 8 * tid;       // z[i] is kept iff 8 * 256 (i / 8) + i % 8 >= keep
#pragma unroll
      for (int i = 0; i < kPerThread; ++i)
        if (8 * kThreads * (i >> 3) + (i & 7) < keep) z[i] = -INFINITY;
    }
  } else {
#pragma unroll
    for (int g = 0; g < kPerThread / 8; ++g) {
      uint32_t raw[8];                            // loaded first, converted after: eight loads in flight
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int t = base + 8 * (kThreads * g + tid) + e;
        raw[e] = BF16 ? 0xff80u : 0xff800000u;    // -inf
        if (t < vocab) {
          if constexpr (BF16)
            raw[e] = ((const uint16_t*)logits)[row0 + t];
          else
            raw[e] = ((const uint32_t*)logits)[row0 + t];
        }
      }
#pragma unroll
      for (int e = 0; e < 8; ++e) z[8 * g + e] = __uint_as_float(BF16 ? raw[e] << 16 : raw[e]);
    }
  }
  // token of z[i] = tbase + off(i), off(i) a constant of the unrolled loops; comparisons of tokens are
  // made on offsets so that no per-element token is ever held in a register
  const int tbase = base + 8 * tid;
  auto off = [](int i) { return 8 * kThreads * (i >> 3) + (i & 7); };

  // the thread's log-sum-exp part, then its row's
  float gm[kPerThread / 8];                       // max of each group of 8: the scan below skips groups
  float mt = -INFINITY;
#pragma unroll
  for (int g = 0; g < kPerThread / 8; ++g) {
    gm[g] = z[8 * g];
#pragma unroll
    for (int e = 1; e < 8; ++e) gm[g] = fmaxf(gm[g], z[8 * g + e]);
    mt = fmaxf(mt, gm[g]);
  }
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
  if (tid == 0) {
    cand_n = 0;
    slot_n = 0;
  }
  __syncthreads();
  if (tid < 16) {
    // lanes 0..15 of wave 0 -- one DPP row -- hold the 16 lane rows' parts: the chunk's (M, S), and
    // T = the k-th largest row maximum (k <= 16)
    const float v = row_m[tid];
    const float M = row_max(v);
    const float S = row_sum(rescale(row_s[tid], v, M));
    int greater = 0, equal = 0;
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      greater += row_m[j] > v ? 1 : 0;
      equal += row_m[j] == v ? 1 : 0;
    }
    if (greater < k && greater + equal >= k) sh_T = v;
    if (tid == 0) {
      sh_M = M;
      sh_S = S;
    }
  }
  __syncthreads();
  const float T = fmaxf(sh_T, -FLT_MAX);           // never below the smallest logit: -inf never passes

  // logits >= T into the LDS list, in two steps that spread the work over the threads: every
  // thread appends its groups of 8 whose max is >= T (the 8 logits and the first token) to a slot
  // list; then thread t turns slot t into the keys of its logits >= T.
  int gcnt = 0;
  if (mt >= T) {
#pragma unroll
    for (int g = 0; g < kPerThread / 8; ++g) gcnt += gm[g] >= T ? 1 : 0;
  }
  int p_slot = wave_alloc(gcnt, &slot_n);
  if (gcnt > 0) {
    int p = p_slot;
#pragma unroll
    for (int g = 0; g < kPerThread / 8; ++g)
      if (gm[g] >= T) {
        if (p < kSlots) {
          slot_v[p][0] = float4{z[8 * g], z[8 * g + 1], z[8 * g + 2], z[8 * g + 3]};
          slot_v[p][1] = float4{z[8 * g + 4], z[8 * g + 5], z[8 * g + 6], z[8 * g + 7]};
          slot_t[p] = tbase + off(8 * g);
        }
        ++p;
      }
  }
  __syncthreads();
  const int ns = slot_n;
  if (ns <= kSlots && (tid & ~63) < ns) {         // waves that hold a slot (wave-uniform)
    const bool mine = tid < ns;
    const float4 a = mine ? slot_v[tid][0] : float4{-INFINITY, -INFINITY, -INFINITY, -INFINITY};
    const float4 c = mine ? slot_v[tid][1] : float4{-INFINITY, -INFINITY, -INFINITY, -INFINITY};
    const float v[8] = {a.x, a.y, a.z, a.w, c.x, c.y, c.z, c.w};
    int cnt = 0;
#pragma unroll
    for (int e = 0; e < 8; ++e) cnt += v[e] >= T ? 1 : 0;
    int p = wave_alloc(cnt, &cand_n);
    if (mine) {
      const int t0 = slot_t[tid];
#pragma unroll
      for (int e = 0; e < 8; ++e) {               // branch-free: a logit below T goes to the spare slot
        const bool pass = v[e] >= T;
        cand[pass && p < kCandCap ? p : kCandCap] = pair_key(v[e], t0 + e);
        p += pass ? 1 : 0;
      }
    }
  }
  __syncthreads();
  const int n = ns <= kSlots ? cand_n : kCandCap + 1;   // too many groups: the arg-max rounds below

  const bool final_row = !LEVEL && chunks == 1;
  const float lse = sh_M + logf(sh_S);
  uint64_t* rec = final_row ? nullptr : ws + (int64_t)blockIdx.x * kRecord;
  auto emit = [&](int r, uint64_t key) {
    if (final_row) {
      tokens[(int64_t)row * k + r] = key_index(key);
      logprobs[(int64_t)row * k + r] = key_value(key) - lse;
    } else {
      store_rec(rec + r, key);
    }
  };
  if (!final_row && tid == 0) store_rec(rec + kTopK, pack_ms(sh_M, sh_S));

  if (n <= kCandCap) {
    for (int c = tid; c < n; c += kThreads) {
      const uint64_t key = cand[c];
      const int rank = rank_of(cand, n, key);
      if (rank < k) emit(rank, key);
    }
    if (tid >= n && tid < k) emit(tid, 0ull);   // a chunk with fewer than k logits: keys below every pair
  } else {
    // many logits tie at the threshold: k rounds of workgroup arg-max, each
    // taking the best pair ordered after the previous winner (lv, li); token
    // ids relative to tbase
    float lv = INFINITY;
    int li = -1;
    for (int r = 0; r < k; ++r) {
      const int lrel = li - tbase;
      float bv = -INFINITY;
      int bi = -1;                                // element index: tokens rise with it, so the first of equal
#pragma unroll                                    // values is the best and a later equal one never replaces it
      for (int i = 0; i < kPerThread; ++i) {
        const float v = z[i];
        const bool after = (v < lv) | ((v == lv) & (off(i) > lrel));
        if (after & (v > bv)) {                   // v > bv >= -inf: only logits
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
  if constexpr (!LEVEL) return;

  // ---- level mode.  Arrival is counted twice: the last chunk of a frontier row to finish merges
  // that row's chunks (its k best keys and its log-sum-exp, a row record), and the last row of a
  // sequence to be merged expands the sequence's frontier.  Before counting in, every thread waits
  // for its record stores to complete at the point of coherence (the asm also keeps the compiler
  // from moving them past this point), so they precede the count; records are read back with
  // device-coherent loads.  Each counter has a 256-byte line of its own.
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  __syncthreads();
  const int F = L.frontier;
  const int b = row / F;
  // counter lines of sequence b: b * 17 + f for its frontier rows, b * 17 + 16 for itself
  unsigned int* row_counter = &L.counters[((int64_t)b * (kTopK + 1) + (row - b * F)) * kCounterStride];
  unsigned int* seq_counter = &L.counters[((int64_t)b * (kTopK + 1) + kTopK) * kCounterStride];
  if (tid == 0) sh_last = atomicAdd(row_counter, 1u) == (unsigned)(chunks - 1);
  __syncthreads();
  if (!sh_last) return;

  __shared__ uint64_t parts[kMaxChunks];          // (m, s) of the row's chunk j
  __shared__ uint64_t ekeys[kMaxCand];
  // Each chunk's keys are sorted, best first, so the largest of the chunks' k-th keys is below or
  // at the row's k-th key: only keys at or above it can be among the row's k best.
  const uint64_t* rrec = ws + (int64_t)row * chunks * kRecord;
  const int per_row = chunks * k;                 // <= 1024 keys
  for (int c = tid; c < per_row; c += kThreads) {
    const int j = c / k;
    cand[c] = load_rec(rrec + j * kRecord + (c - j * k));
  }
  if (tid < chunks) parts[tid] = load_rec(rrec + tid * kRecord + kTopK);
  if (tid == 0) cand_n = 0;
  __syncthreads();
  if (tid < 64) {                                 // chunks <= 64: one lane per chunk
    const uint64_t kth = wave_max(tid < chunks ? cand[tid * k + k - 1] : (uint64_t)0);
    if (tid == 0) win[0] = kth;
  }
  __syncthreads();
  const uint64_t floor_key = win[0];
  uint64_t* top = cand + per_row;                 // the keys that pass, after the row's keys
  const int room = kCandCap - per_row;
  for (int c = tid; c < per_row; c += kThreads) {
    const uint64_t key = cand[c];
    if (key >= floor_key) {
      const int p = atomicAdd(&cand_n, 1);
      if (p < room) top[p] = key;
    }
  }
  __syncthreads();
  const int m = cand_n;
  const uint64_t* pool = m <= room ? top : cand;  // no room left after the row's keys: rank them all
  const int pn = m <= room ? m : per_row;
  uint64_t* rowrec = L.rows + (int64_t)row * kRecord;
  for (int c = tid; c < pn; c += kThreads) {
    const uint64_t key = pool[c];
    const int rank = rank_of(pool, pn, key);
    if (rank < k) store_rec(rowrec + rank, key);
  }
  if (tid == 0) {
    store_rec(rowrec + kTopK, __float_as_uint(chunk_lse(parts, chunks)));
    atomicExch(row_counter, 0u);                  // ready for the next call
  }
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  __syncthreads();
  if (tid == 0) sh_last = atomicAdd(seq_counter, 1u) == (unsigned)(F - 1);
  __syncthreads();
  if (!sh_last) return;

  // expansion: candidate c = (frontier node c / k, proposal rank c % k)
  const int C = F * k;
  float sc = 0.0f;
  uint64_t key = 0ull, ekey = 0ull;
  if (tid < C) {
    const uint64_t* fr = L.rows + ((int64_t)b * F + tid / k) * kRecord;
    key = load_rec(fr + tid % k);
    const float lp = key_value(key) - __uint_as_float((uint32_t)load_rec(fr + kTopK));
    sc = L.scores[(int64_t)b * F + tid / k] + lp;
    ekey = pair_key(sc, tid);
    ekeys[tid] = ekey;
  }
  __syncthreads();
  if (tid < C) {
    const int rank = rank_of(ekeys, C, ekey);
    if (rank < k) {
      const int64_t o = (int64_t)b * k + rank;
      L.next_parent[o] = tid / k;
      L.next_tokens[o] = key_index(key);
      L.next_scores[o] = sc;
    }
  }
  if (tid == 0) atomicExch(seq_counter, 0u);      // ready for the next call
}

// One row of several chunks: combine the chunks' log-sum-exp parts and rank
// their k best keys.
__global__ __launch_bounds__(kThreads) void topk_merge_kernel(int k, int chunks, const uint64_t* ws, int32_t* tokens,
                                                              float* logprobs) {
  __shared__ uint64_t keys[kMaxChunks * kTopK];
  __shared__ uint64_t parts[kMaxChunks];
  __shared__ float sh_lse;
  const int tid = threadIdx.x;
  const int row = blockIdx.x;
  const uint64_t* rec = ws + (int64_t)row * chunks * kRecord;
  const int n = chunks * k;
  for (int c = tid; c < n; c += kThreads) {
    const int j = c / k;
    keys[c] = load_rec(rec + j * kRecord + (c - j * k));
  }
  if (tid < chunks) parts[tid] = load_rec(rec + tid * kRecord + kTopK);
  __syncthreads();
  if (tid == 0) sh_lse = chunk_lse(parts, chunks);
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
  const LevelArgs none{};
  if (dtype == KVSHOT_BF16)
    hipLaunchKernelGGL((topk_chunk_kernel<true, false>), grid, dim3(kThreads), 0, s, logits, (int)vocab, row_stride,
                       (int)k, chunks, vec, tokens, logprobs, ws, none);
  else
    hipLaunchKernelGGL((topk_chunk_kernel<false, false>), grid, dim3(kThreads), 0, s, logits, (int)vocab, row_stride,
                       (int)k, chunks, vec, tokens, logprobs, ws, none);
  if (chunks > 1)
    hipLaunchKernelGGL(topk_merge_kernel, dim3(rows), dim3(kThreads), 0, s, (int)k, chunks, ws, tokens, logprobs);
  return hipGetLastError() == hipSuccess ? KVSHOT_OK : KVSHOT_ERR_DEVICE;
}

namespace {
// workspace: counters (17 lines of 256 bytes per sequence, whatever the frontier, so that calls with
// different frontier sizes can share a workspace), chunk records, row records
int64_t level_counter_bytes(int32_t batch) { return (int64_t)batch * (kTopK + 1) * kCounterStride * 4; }
}  // namespace

extern "C" int64_t kvshot_tree_level_workspace_bytes(int32_t batch, int32_t frontier, int32_t vocab) {
  if (batch < 1 || frontier < 1 || frontier > kTopK || vocab < 1 || chunks_for(vocab) > kMaxChunks) return -1;
  return level_counter_bytes(batch) +
         (int64_t)batch * frontier * (chunks_for(vocab) + 1) * kRecord * (int64_t)sizeof(uint64_t);
}

extern "C" kvshot_status kvshot_tree_level(const void* logits, int32_t dtype, int32_t batch, int32_t frontier,
                                           int32_t vocab, int64_t row_stride, int32_t k, const float* scores,
                                           int32_t* next_parent, int32_t* next_tokens, float* next_scores,
                                           void* workspace, int64_t workspace_bytes, void* stream) {
  if (!logits || !scores || !next_parent || !next_tokens || !next_scores || !workspace) return KVSHOT_ERR_INVALID_ARG;
  if (batch < 1 || frontier < 1 || frontier > kTopK || k < 1 || k > kTopK || vocab < k) return KVSHOT_ERR_INVALID_ARG;
  if (dtype != KVSHOT_BF16 && dtype != KVSHOT_FP32) return KVSHOT_ERR_INVALID_ARG;
  const unsigned elem = dtype == KVSHOT_BF16 ? 2u : 4u;
  if (row_stride < vocab || !aligned(logits, elem) || !aligned(workspace, 256)) return KVSHOT_ERR_INVALID_ARG;
  const int64_t need = kvshot_tree_level_workspace_bytes(batch, frontier, vocab);
  const int chunks = chunks_for(vocab);
  const int64_t rows = (int64_t)batch * frontier;
  if (need < 0 || workspace_bytes < need || rows * chunks > INT_MAX) return KVSHOT_ERR_INVALID_ARG;
  const bool vec = aligned(logits, 16) && (row_stride * elem) % 16 == 0;
  LevelArgs L;
  L.batch = batch;
  L.frontier = frontier;
  L.scores = scores;
  L.next_parent = next_parent;
  L.next_tokens = next_tokens;
  L.next_scores = next_scores;
  L.counters = (unsigned int*)workspace;
  uint64_t* ws = (uint64_t*)((char*)workspace + level_counter_bytes(batch));
  L.rows = ws + rows * chunks * kRecord;
  hipStream_t s = (hipStream_t)stream;
  const dim3 grid((unsigned)(rows * chunks));
  if (dtype == KVSHOT_BF16)
    hipLaunchKernelGGL((topk_chunk_kernel<true, true>), grid, dim3(kThreads), 0, s, logits, (int)vocab, row_stride,
                       (int)k, chunks, vec, nullptr, nullptr, ws, L);
  else
    hipLaunchKernelGGL((topk_chunk_kernel<false, true>), grid, dim3(kThreads), 0, s, logits, (int)vocab, row_stride,
                       (int)k, chunks, vec, nullptr, nullptr, ws, L);
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
