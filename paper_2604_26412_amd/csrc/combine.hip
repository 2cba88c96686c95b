// Cross-split merge of split-K partial softmax states.
//
// Split s of a query row left (m_s, l_s, O_s): its running max (log2 units),
// its sum of exp2(score - m_s) and its unnormalised output.  The row's result
// is sum_s O_s 2^(m_s - M) / sum_s l_s 2^(m_s - M) with M = max_s m_s, which is
// the same softmax-weighted sum over the union of the splits' keys.  Splits
// that saw no key (l_s = 0) carry no weight.
#include "kvshot_common.h"

namespace kvshot {
namespace {

constexpr float kLn2 = 0.693147180559945309f;

__global__ __launch_bounds__(256) void combine_kernel(CombineParams p) {
  const int lane = threadIdx.x & 63;
  const int64_t wid = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int64_t total = (int64_t)p.batch * p.hkv * p.rows;
  if (wid >= total) return;
  const int r = (int)(wid % p.rows);
  const int64_t bh = wid / p.rows;
  const int h = (int)(bh % p.hkv);
  const int b = (int)(bh / p.hkv);
  const int64_t base = (bh * p.rows_pad + r) * p.splits;

  float ms = -INFINITY, ls = 0.0f;
  if (lane < p.splits) {
    const float2 t = p.part_ml[base + lane];
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
  for (int s = 0; s < p.splits; ++s) {
    const float ws = __shfl(wgt, s);
    if (ws != 0.0f) {
      const float2 v = *(const float2*)(p.part_o + (base + s) * kHeadDim + lane * 2);
      acc.x += ws * v.x;
      acc.y += ws * v.y;
    }
  }
  const float inv = 1.0f / L;
  const int j = r / p.group;
  const int hq = h * p.group + (r - j * p.group);
  const int64_t orow = (((int64_t)b * p.nq + j) * p.hq + hq) * kHeadDim + lane * 2;
  if (p.out_fp32)
    *(float2*)((float*)p.out + orow) = make_float2(acc.x * inv, acc.y * inv);
  else
    *(uint32_t*)((uint16_t*)p.out + orow) = pack_bf16x2(acc.x * inv, acc.y * inv);
  if (p.lse && lane == 0) p.lse[((int64_t)b * p.nq + j) * p.hq + hq] = (M + __log2f(L)) * kLn2;
}

}  // namespace

hipError_t launch_combine(const CombineParams& p, hipStream_t s) {
  const int64_t waves = (int64_t)p.batch * p.hkv * p.rows;
  const int64_t blocks = (waves + 3) / 4;
  hipLaunchKernelGGL(combine_kernel, dim3((unsigned)blocks), dim3(256), 0, s, p);
  return hipGetLastError();
}

}  // namespace kvshot
