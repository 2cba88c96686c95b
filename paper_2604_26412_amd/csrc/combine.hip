// Cross-split merge of split-K partial softmax states: one wave per query
// row, the merge itself is combine_row.  (Merging inside the attention kernel,
// in the last workgroup to finish, measured slower: the device-scope fences it
// needs write back and invalidate a whole XCD L2 per workgroup.  The merge has
// little data to move, so its time is the launch and two dependent loads.)
#include "kvshot_common.h"

namespace kvshot {
namespace {

// Merge the split partials of one query row into its output (one wave; every
// lane takes two channels).  Split s left (m_s, l_s, O_s): its running max
// (log2 units), its sum of 2^(score - m_s) and its unnormalised output.  The
// row's result is sum_s O_s 2^(m_s - M) / sum_s l_s 2^(m_s - M), M = max_s m_s,
// the softmax-weighted sum over the union of the splits' keys; splits that saw
// no key (l_s = 0) carry no weight.
__device__ __forceinline__ void combine_row(const float* part_o, const float2* part_ml, int64_t base, int64_t stride,
                                            int splits, void* out, int64_t orow, bool out_fp32, float* lse_out,
                                            int lane) {
  // Eight splits' rows are loaded at once, with no branch between them, so
  // their latencies overlap (the first eight also with the (m, l) load); a
  // split of weight zero is skipped by a select, so whatever its row holds
  // never reaches the sum.
  float2 v[8];
  auto load_rows = [&](int s0) {
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int s = s0 + u < splits ? s0 + u : splits - 1;
      v[u] = *(const float2*)(part_o + (base + s * stride) * kHeadDim + lane * 2);
    }
  };
  load_rows(0);
  float ms = -INFINITY, ls = 0.0f;
  if (lane < splits) {
    const float2 t = part_ml[base + lane * stride];
    ms = t.y > 0.0f ? t.x : -INFINITY;
    ls = t.y;
  }
  float M = ms;
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) M = fmaxf(M, __shfl_xor(M, o));
  const float Mu = M == -INFINITY ? 0.0f : M;
  const float wgt = ls > 0.0f ? __builtin_amdgcn_exp2f(ms - Mu) : 0.0f;
  float L = wgt * ls;
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) L += __shfl_xor(L, o);
  float2 acc = make_float2(0.0f, 0.0f);
  for (int s0 = 0; s0 < splits; s0 += 8) {
    if (s0 > 0) load_rows(s0);
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const float ws = __shfl(wgt, s0 + u);    // s0 + u < kMaxSplits = 64; lanes past `splits` hold 0
      acc.x = ws != 0.0f ? acc.x + ws * v[u].x : acc.x;
      acc.y = ws != 0.0f ? acc.y + ws * v[u].y : acc.y;
    }
  }
  const float inv = 1.0f / L;
  if (out_fp32)
    *(float2*)((float*)out + orow + lane * 2) = make_float2(acc.x * inv, acc.y * inv);
  else
    *(uint32_t*)((uint16_t*)out + orow + lane * 2) = pack_bf16x2(acc.x * inv, acc.y * inv);
  if (lse_out && lane == 0) *lse_out = (M + __log2f(L)) * 0.693147180559945309f;
}

__global__ __launch_bounds__(256) void combine_kernel(CombineParams p) {
  const int lane = threadIdx.x & 63;
  const int64_t wid = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int64_t total = (int64_t)p.batch * p.hkv * p.rows;
  if (wid >= total) return;
  const int r = (int)(wid % p.rows);
  const int64_t bh = wid / p.rows;
  const int h = (int)(bh % p.hkv);
  const int b = (int)(bh / p.hkv);
  const int j = r / p.group;
  const int hq = h * p.group + (r - j * p.group);
  const int64_t q_index = ((int64_t)b * p.nq + j) * p.hq + hq;
  int splits = p.splits;
  int64_t base = (bh * p.rows_pad + r) * p.splits, stride = 1;
  if (p.seq_splits) {
    // this sequence's split count and first item under the attention kernel's balanced schedule (its
    // items' partials sit rows_pad rows apart); with one split the attention kernel wrote the output
    splits = p.seq_splits[b];
    if (splits <= 1) return;
    splits = splits > kMaxSplits ? kMaxSplits : splits;
    int first = p.seq_splits[64 + b];
    first = first < 0 ? 0 : (first > p.items - splits ? p.items - splits : first);
    base = ((int64_t)h * p.items + first) * p.rows_pad + r;
    stride = p.rows_pad;
  }
  combine_row(p.part_o, p.part_ml, base, stride, splits, p.out, q_index * kHeadDim, p.out_fp32 != 0,
              p.lse ? p.lse + q_index : nullptr, lane);
}

// Plans with at most four splits and one split count for every row (trees, small batches): one wave
// merges two neighbouring rows of one (sequence, KV head), lanes 0-31 holding the first row's split
// weights and lanes 32-63 the second's, so its eight row loads are all distinct rows of partials.
// (With one row per wave, four of the eight loads re-read the last split, and twice as many waves
// each move half the data: the tree's merge ran at about 2.5 TB/s.)  Same arithmetic, same
// summation order as combine_row.
__global__ __launch_bounds__(256) void combine_pair_kernel(CombineParams p) {
  const int lane = threadIdx.x & 63;
  const int half = lane >> 5;
  const int64_t wid = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int pairs = (p.rows + 1) / 2;
  const int64_t total = (int64_t)p.batch * p.hkv * pairs;
  if (wid >= total) return;
  const int r0 = (int)(wid % pairs) * 2;
  const int64_t bh = wid / pairs;
  const bool second = r0 + 1 < p.rows;
  const int splits = p.splits;
  int64_t base[2];
  base[0] = (bh * p.rows_pad + r0) * splits;
  base[1] = (bh * p.rows_pad + (second ? r0 + 1 : r0)) * splits;
  float2 v[2][4];
#pragma unroll
  for (int q = 0; q < 2; ++q)
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int s = u < splits ? u : splits - 1;
      v[q][u] = *(const float2*)(p.part_o + (base[q] + s) * kHeadDim + lane * 2);
    }
  // lane 32 q + s holds split s of row q
  const int ls_idx = lane & 31;
  float ms = -INFINITY, ls = 0.0f;
  if (ls_idx < splits) {
    const float2 t = p.part_ml[base[half] + ls_idx];
    ms = t.y > 0.0f ? t.x : -INFINITY;
    ls = t.y;
  }
  float M = ms;
#pragma unroll
  for (int o = 16; o >= 1; o >>= 1) M = fmaxf(M, __shfl_xor(M, o));
  const float Mu = M == -INFINITY ? 0.0f : M;
  const float wgt = ls > 0.0f ? __builtin_amdgcn_exp2f(ms - Mu) : 0.0f;
  float L = wgt * ls;
#pragma unroll
  for (int o = 16; o >= 1; o >>= 1) L += __shfl_xor(L, o);
  const int b = (int)(bh / p.hkv), h = (int)(bh % p.hkv);
#pragma unroll
  for (int q = 0; q < 2; ++q) {
    float2 acc = make_float2(0.0f, 0.0f);
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const float ws = __shfl(wgt, 32 * q + u);   // lanes past `splits` in each half hold 0
      acc.x = ws != 0.0f ? acc.x + ws * v[q][u].x : acc.x;
      acc.y = ws != 0.0f ? acc.y + ws * v[q][u].y : acc.y;
    }
    const float Lq = __shfl(L, 32 * q);
    const float Mq = __shfl(M, 32 * q);
    if (q == 1 && !second) break;
    const int r = r0 + q;
    const int j = r / p.group;
    const int hq = h * p.group + (r - j * p.group);
    const int64_t q_index = ((int64_t)b * p.nq + j) * p.hq + hq;
    const int64_t orow = q_index * kHeadDim;
    const float inv = 1.0f / Lq;
    if (p.out_fp32)
      *(float2*)((float*)p.out + orow + lane * 2) = make_float2(acc.x * inv, acc.y * inv);
    else
      *(uint32_t*)((uint16_t*)p.out + orow + lane * 2) = pack_bf16x2(acc.x * inv, acc.y * inv);
    if (p.lse && lane == 0) p.lse[q_index] = (Mq + __log2f(Lq)) * 0.693147180559945309f;
  }
}

}  // namespace

hipError_t launch_combine(const CombineParams& p, hipStream_t s) {
  if (!p.seq_splits && p.splits <= 4) {
    const int64_t waves = (int64_t)p.batch * p.hkv * ((p.rows + 1) / 2);
    hipLaunchKernelGGL(combine_pair_kernel, dim3((unsigned)((waves + 3) / 4)), dim3(256), 0, s, p);
    return hipGetLastError();
  }
  const int64_t waves = (int64_t)p.batch * p.hkv * p.rows;
  const int64_t blocks = (waves + 3) / 4;
  hipLaunchKernelGGL(combine_kernel, dim3((unsigned)blocks), dim3(256), 0, s, p);
  return hipGetLastError();
}

}  // namespace kvshot
