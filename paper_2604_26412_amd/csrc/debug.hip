// Debug and validation kernels.  They run the same index code as the
// attention kernels (kvshot_common.h) so tests can check that code bit for bit.
#include "kvshot_common.h"

namespace kvshot {
namespace {

// One thread per (token, 16-byte chunk) of the dense logical view.
__global__ __launch_bounds__(256) void gather_kv_kernel(AttnParams p, int max_ctx, void* k_dense, void* v_dense,
                                                        int elem_bytes) {
  const int chunks = kHeadDim * elem_bytes / 16;
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int h = blockIdx.y, b = blockIdx.z;
  const int tok = (int)(idx / chunks), ch = (int)(idx % chunks);
  if (tok >= max_ctx) return;
  const int T = clamp_ctx(p.ctx_lens[b], p.max_pages_per_seq, p.page_shift);
  const int64_t dst = ((((int64_t)b * max_ctx + tok) * p.hkv + h) * kHeadDim) * elem_bytes + ch * 16;
  uint4 kv = make_uint4(0, 0, 0, 0), vv = make_uint4(0, 0, 0, 0);
  if (tok < T) {
    const int pid = physical_page(p.page_table, b, p.max_pages_per_seq, tok >> p.page_shift, p.num_pages);
    const int64_t off = kv_offset(pid, h, tok & ((1 << p.page_shift) - 1), p.page_stride, p.head_stride,
                                  p.slot_stride) * elem_bytes + ch * 16;
    kv = *(const uint4*)((const unsigned char*)p.k_pages + off);
    vv = *(const uint4*)((const unsigned char*)p.v_pages + off);
  }
  *(uint4*)((unsigned char*)k_dense + dst) = kv;
  *(uint4*)((unsigned char*)v_dense + dst) = vv;
}

// One wave per sequence.
__global__ __launch_bounds__(64) void tree_mask_kernel(const int32_t* parents, int n, uint64_t* anc, int32_t* depth) {
  const int b = blockIdx.x, lane = threadIdx.x;
  int d = 0;
  const uint64_t a = tree_ancestry_wave(parents + (int64_t)b * n, n, lane, &d);
  if (lane < n) {
    anc[(int64_t)b * n + lane] = a;
    depth[(int64_t)b * n + lane] = d;
  }
}

__global__ void flag_init_kernel(int32_t* flag) { *flag = 0x7fffffff; }

// One workgroup per sequence: checks its length, its used page ids, its step
// offset and its parents; records the smallest violation code seen.
__global__ __launch_bounds__(256) void validate_kernel(AttnParams p, int max_ctx_hint, int32_t* flag) {
  const int b = blockIdx.x;
  const int t = threadIdx.x;
  const int T = p.ctx_lens[b];
  if (t == 0 && (T < 0 || T > max_ctx_hint)) atomicMin(flag, 1);
  const int Tc = T < 0 ? 0 : (T > max_ctx_hint ? max_ctx_hint : T);
  const int used = (Tc + (1 << p.page_shift) - 1) >> p.page_shift;
  for (int lp = t; lp < used; lp += 256) {
    const int pid = p.page_table[(int64_t)b * p.max_pages_per_seq + lp];
    if (pid < 0 || pid >= p.num_pages) atomicMin(flag, 2);
  }
  if (p.step_offsets && t == 0) {
    const int s0 = p.step_offsets[b];
    if (s0 < 0 || s0 + p.nq > p.max_draft) atomicMin(flag, 3);
  }
  if (p.parents && t < p.n_nodes) {
    const int par = p.parents[(int64_t)b * p.n_nodes + t];
    if (par < -1 || par >= t) atomicMin(flag, 4);
  }
  if (p.query_nodes && t < p.nq) {
    const int node = p.query_nodes[(int64_t)b * p.nq + t];
    if (node < 0 || node >= p.n_nodes) atomicMin(flag, 5);
  }
  if (p.pos_base && t < 64) {
    // the highest position this sequence's draft queries and keys use must have a RoPE table entry
    const int base = p.pos_base[b];
    int top = 0;
    if (p.tree) {
      int depth = 0;
      (void)tree_ancestry_wave(p.parents + (int64_t)b * p.n_nodes, p.n_nodes, t, &depth);
      top = depth;
#pragma unroll
      for (int o = 32; o > 0; o >>= 1) top = max(top, __shfl_xor(top, o));
    } else {
      int s0 = p.step_offsets ? p.step_offsets[b] : 0;
      s0 = s0 < 0 ? 0 : s0;
      top = s0 + p.nq - 1;
    }
    if (t == 0 && (base < 0 || (int64_t)base + top >= p.max_position)) atomicMin(flag, 6);
  }
}

// Streaming read of `n16` 16-byte words with non-temporal loads: each lane
// folds what it reads with xor so the loads cannot be dropped, and every
// workgroup stores one word.  Used only to measure the device's practical
// read bandwidth.
typedef uint32_t sr_u32x4 __attribute__((ext_vector_type(4)));
__global__ __launch_bounds__(256) void stream_read_kernel(const sr_u32x4* __restrict__ src, int64_t n16,
                                                          sr_u32x4* sink) {
  const int64_t stride = (int64_t)gridDim.x * 256 * 8;
  sr_u32x4 acc = {0, 0, 0, 0};
  for (int64_t i = (int64_t)blockIdx.x * 256 * 8 + threadIdx.x; i < n16; i += stride) {
    sr_u32x4 v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u)
      v[u] = (i + u * 256 < n16) ? __builtin_nontemporal_load(src + i + u * 256) : sr_u32x4{0, 0, 0, 0};
#pragma unroll
    for (int u = 0; u < 8; ++u) acc ^= v[u];
  }
  __shared__ sr_u32x4 red[256];
  red[threadIdx.x] = acc;
  __syncthreads();
  if (threadIdx.x == 0) {
    sr_u32x4 r = {0, 0, 0, 0};
    for (int k = 0; k < 256; ++k) r ^= red[k];
    sink[blockIdx.x] = r;
  }
}

// Dense bf16 matrix work with no memory traffic: every wave issues iters x 16
// 32x32x16 products into four accumulators in turn, and each workgroup stores
// one word so the products cannot be dropped.  One workgroup of four waves per
// CU (one wave per SIMD).  Used only to measure the rate the matrix cores
// sustain when every SIMD runs them.
typedef __bf16 mr_bf16x8 __attribute__((ext_vector_type(8)));
typedef float mr_f32x16 __attribute__((ext_vector_type(16)));
__global__ __launch_bounds__(256, 1) void mfma_rate_kernel(int iters, sr_u32x4* sink) {
  const int lane = threadIdx.x & 63;
  mr_bf16x8 a, b;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    a[i] = (__bf16)(0.001f * (float)(lane + i));
    b[i] = (__bf16)(0.002f * (float)(lane - i));
  }
  mr_f32x16 acc[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) acc[j] = mr_f32x16{};
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int r = 0; r < 4; ++r)
#pragma unroll
      for (int j = 0; j < 4; ++j) acc[j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc[j], 0, 0, 0);
  }
  float s = 0.0f;
#pragma unroll
  for (int j = 0; j < 4; ++j)
#pragma unroll
    for (int e = 0; e < 16; ++e) s += acc[j][e];
  __shared__ uint32_t red[256];
  red[threadIdx.x] = __float_as_uint(s);
  __syncthreads();
  if (threadIdx.x == 0) {
    uint32_t r = 0;
    for (int k = 0; k < 256; ++k) r ^= red[k];
    sink[blockIdx.x] = sr_u32x4{r, 0u, 0u, 0u};
  }
}

}  // namespace

hipError_t launch_mfma_rate(int blocks, int iters, void* sink, hipStream_t s) {
  hipLaunchKernelGGL(mfma_rate_kernel, dim3(blocks), dim3(256), 0, s, iters, (sr_u32x4*)sink);
  return hipGetLastError();
}

hipError_t launch_stream_read(const void* src, int64_t bytes, void* sink, int blocks, hipStream_t s) {
  hipLaunchKernelGGL(stream_read_kernel, dim3(blocks), dim3(256), 0, s, (const sr_u32x4*)src, bytes / 16,
                     (sr_u32x4*)sink);
  return hipGetLastError();
}

hipError_t launch_gather_kv(const AttnParams& p, int max_ctx, void* k_dense, void* v_dense, int bf16,
                            hipStream_t s) {
  const int eb = bf16 ? 2 : 4;
  const int64_t threads = (int64_t)max_ctx * (kHeadDim * eb / 16);
  const dim3 grid((unsigned)((threads + 255) / 256), p.hkv, p.batch);
  hipLaunchKernelGGL(gather_kv_kernel, grid, dim3(256), 0, s, p, max_ctx, k_dense, v_dense, eb);
  return hipGetLastError();
}

hipError_t launch_tree_mask(const int32_t* parents, int batch, int n, uint64_t* anc, int32_t* depth, hipStream_t s) {
  hipLaunchKernelGGL(tree_mask_kernel, dim3(batch), dim3(64), 0, s, parents, n, anc, depth);
  return hipGetLastError();
}

hipError_t launch_validate(const AttnParams& p, int max_ctx_hint, int32_t* flag, hipStream_t s) {
  hipLaunchKernelGGL(flag_init_kernel, dim3(1), dim3(1), 0, s, flag);
  hipLaunchKernelGGL(validate_kernel, dim3(p.batch), dim3(256), 0, s, p, max_ctx_hint, flag);
  return hipGetLastError();
}

}  // namespace kvshot
