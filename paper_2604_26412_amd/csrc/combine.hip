// Cross-split merge of split-K partial softmax states: one wave per query
// row, the merge itself is combine_row.  (Merging inside the attention kernel,
// in the last workgroup to finish, measured slower: the device-scope fences it
// needs write back and invalidate a whole XCD L2 per workgroup.)
#include "kvshot_common.h"

namespace kvshot {
namespace {

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
  combine_row(p.part_o, p.part_ml, (bh * p.rows_pad + r) * p.splits, p.splits, p.out, q_index * kHeadDim,
              p.out_fp32 != 0, p.lse ? p.lse + q_index : nullptr, lane);
}

}  // namespace

hipError_t launch_combine(const CombineParams& p, hipStream_t s) {
  const int64_t waves = (int64_t)p.batch * p.hkv * p.rows;
  const int64_t blocks = (waves + 3) / 4;
  hipLaunchKernelGGL(combine_kernel, dim3((unsigned)blocks), dim3(256), 0, s, p);
  return hipGetLastError();
}

}  // namespace kvshot
