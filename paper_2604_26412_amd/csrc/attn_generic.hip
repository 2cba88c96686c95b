// Generic draft attention on the vector ALU, for float32 inputs (and as a
// second bf16 path behind an option).  Same split-K plan, partial layout and
// index code as the MFMA kernel; arithmetic entirely in float32.
//
// A 256-thread workgroup serves one (split, KV head, sequence).  Thread t owns
// query row (t / 16) of a 16-row tile and the 8 channels 8 * (t % 16) .. +7.
// Scores are reduced across the 16 threads of a row with xor shuffles (every
// lane of the row ends with the same bits), then each key updates the online
// softmax state (Sec. 2.2, Eq. 2, accumulated one key at a time).
#include "kvshot_common.h"

namespace kvshot {
namespace {

constexpr float kLn2 = 0.693147180559945309f;

template <bool BF16>
__device__ __forceinline__ void load8(const void* base, int64_t off, float (&x)[8]) {
  if constexpr (BF16) {
    const uint4 v = *(const uint4*)((const uint16_t*)base + off);
    const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      x[2 * i] = bf16_lo(w[i]);
      x[2 * i + 1] = bf16_hi(w[i]);
    }
  } else {
    const float4 a = *(const float4*)((const float*)base + off);
    const float4 c = *(const float4*)((const float*)base + off + 4);
    x[0] = a.x; x[1] = a.y; x[2] = a.z; x[3] = a.w;
    x[4] = c.x; x[5] = c.y; x[6] = c.z; x[7] = c.w;
  }
}

// Rotate the 8 channels of chunk c (channels 8c..8c+7) given the row's data at
// chunk c and at its RoPE partner chunk c ^ 8.
__device__ __forceinline__ void rope8(const float (&x)[8], const float (&xp)[8], int c, const float2* cs,
                                      float (&y)[8]) {
  const bool low = c < 8;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const int m = (c & 7) * 8 + e;
    const float2 t = cs[m];
    y[e] = low ? x[e] * t.x - xp[e] * t.y : x[e] * t.x + xp[e] * t.y;
  }
}

__device__ __forceinline__ float row16_sum(float v) {
  v += __shfl_xor(v, 1);
  v += __shfl_xor(v, 2);
  v += __shfl_xor(v, 4);
  v += __shfl_xor(v, 8);
  return v;
}

template <bool BF16>
__global__ __launch_bounds__(256) void attn_generic_kernel(AttnParams p) {
  const int t = threadIdx.x;
  const int lane = t & 63;
  const int rr = t >> 4;      // row within the 16-row tile
  const int c = t & 15;       // channel chunk
  const int split = blockIdx.x, h = blockIdx.y, b = blockIdx.z;

  int T = clamp_ctx(p.ctx_lens[b], p.max_pages_per_seq, p.page_shift);
  T = T > p.max_ctx ? p.max_ctx : T;
  const int key_beg = split * p.blocks_per_split * kBlockKeys;
  const int key_end = min(key_beg + p.blocks_per_split * kBlockKeys, T);
  const bool last = split == p.splits - 1;

  int s0 = 0, S = p.tree ? p.n_nodes : p.nq;
  if (!p.tree) {
    s0 = p.step_offsets[b];
    s0 = s0 < 0 ? 0 : (s0 > p.max_draft - p.nq ? p.max_draft - p.nq : s0);
    S = s0 + p.nq;
  }
  uint64_t anc_mine = 0;
  int depth_mine = 0;
  if (p.tree) anc_mine = tree_ancestry_wave(p.parents + (int64_t)b * p.n_nodes, p.n_nodes, lane, &depth_mine);
  const int P = position_base(p, b, T);            // position of draft step 0 / tree depth 0

  const int pmask = (1 << p.page_shift) - 1;
  const int64_t row = (int64_t)b * p.max_pages_per_seq;

  for (int r0 = 0; r0 < p.rows; r0 += 16) {
    const int r = r0 + rr;
    const bool row_ok = r < p.rows;
    const int rc = row_ok ? r : p.rows - 1;
    const int j = rc / p.group;
    const int g = rc - j * p.group;
    const int hq = h * p.group + g;
    uint64_t row_anc = 0;
    int qpos;
    if (p.tree) {
      const int node = query_node(p, b, j);
      const uint32_t lo = __shfl((uint32_t)anc_mine, node), hi = __shfl((uint32_t)(anc_mine >> 32), node);
      row_anc = ((uint64_t)hi << 32) | lo;
      qpos = P + __shfl(depth_mine, node);
    } else {
      qpos = P + s0 + j;
    }
    qpos = qpos >= p.max_position ? p.max_position - 1 : qpos;

    float qv[8];
    {
      const int64_t qoff = (((int64_t)b * p.nq + j) * p.hq + hq) * kHeadDim;
      float x[8], xp[8];
      load8<BF16>(p.q, qoff + c * 8, x);
      load8<BF16>(p.q, qoff + (c ^ 8) * 8, xp);
      rope8(x, xp, c, p.rope + (int64_t)qpos * kHalfDim, qv);
#pragma unroll
      for (int e = 0; e < 8; ++e) qv[e] *= row_ok ? p.qscale : 0.0f;
    }

    float m = -INFINITY, l = 0.0f, o[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    auto update = [&](float sc, const float (&v)[8]) {
      const float mn = fmaxf(m, sc);
      const float mu = mn == -INFINITY ? 0.0f : mn;
      const float alpha = exp2f(m - mu);
      const float pk = exp2f(sc - mu);
      l = l * alpha + pk;
#pragma unroll
      for (int e = 0; e < 8; ++e) o[e] = o[e] * alpha + (pk != 0.0f ? pk * v[e] : 0.0f);
      m = mn;
    };

    for (int key = key_beg; key < key_end; ++key) {
      const int pid = physical_page(p.page_table, b, p.max_pages_per_seq, key >> p.page_shift, p.num_pages);
      const int64_t off = kv_offset(pid, h, key & pmask, p.page_stride, p.head_stride, p.slot_stride) + c * 8;
      float kx[8], vx[8];
      load8<BF16>(p.k_pages, off, kx);
      load8<BF16>(p.v_pages, off, vx);
      float part = 0.0f;
#pragma unroll
      for (int e = 0; e < 8; ++e) part += qv[e] * kx[e];
      update(row16_sum(part), vx);
    }
    if (last) {
      for (int s = 0; s < S; ++s) {
        const int64_t off = draft_offset(b, s, h, p.max_draft, p.hkv);
        float kx[8], kp[8], kr[8], vx[8];
        load8<BF16>(p.draft_k, off + c * 8, kx);
        load8<BF16>(p.draft_k, off + (c ^ 8) * 8, kp);
        load8<BF16>(p.draft_v, off + c * 8, vx);
        int kpos = p.tree ? P + __shfl(depth_mine, s) : P + s;
        kpos = kpos >= p.max_position ? p.max_position - 1 : kpos;
        rope8(kx, kp, c, p.rope + (int64_t)kpos * kHalfDim, kr);
        float part = 0.0f;
#pragma unroll
        for (int e = 0; e < 8; ++e) part += qv[e] * kr[e];
        const float sc = row16_sum(part);
        const bool ok = p.tree ? ((row_anc >> s) & 1ull) != 0 : s <= s0 + j;
        update(ok ? sc : -INFINITY, vx);
      }
    }

    if (!row_ok) continue;
    if (p.splits == 1) {
      const float inv = 1.0f / l;
      const int64_t orow = (((int64_t)b * p.nq + j) * p.hq + hq) * kHeadDim + c * 8;
      if (p.out_fp32) {
        float* op = (float*)p.out + orow;
        *(float4*)op = make_float4(o[0] * inv, o[1] * inv, o[2] * inv, o[3] * inv);
        *(float4*)(op + 4) = make_float4(o[4] * inv, o[5] * inv, o[6] * inv, o[7] * inv);
      } else {
        uint4 v;
        v.x = pack_bf16x2(o[0] * inv, o[1] * inv);
        v.y = pack_bf16x2(o[2] * inv, o[3] * inv);
        v.z = pack_bf16x2(o[4] * inv, o[5] * inv);
        v.w = pack_bf16x2(o[6] * inv, o[7] * inv);
        *(uint4*)((uint16_t*)p.out + orow) = v;
      }
      if (p.lse && c == 0) p.lse[((int64_t)b * p.nq + j) * p.hq + hq] = (m + log2f(l)) * kLn2;
    } else {
      const int64_t prow = (((int64_t)b * p.hkv + h) * p.rows_pad + r) * p.splits + split;
      float* po = p.part_o + prow * kHeadDim + c * 8;
      *(float4*)po = make_float4(o[0], o[1], o[2], o[3]);
      *(float4*)(po + 4) = make_float4(o[4], o[5], o[6], o[7]);
      if (c == 0) p.part_ml[prow] = make_float2(m, l);
    }
  }
}

}  // namespace

hipError_t launch_attn_generic(const AttnParams& p, int bf16_in, hipStream_t s) {
  const dim3 grid(p.splits, p.hkv, p.batch);
  if (bf16_in)
    hipLaunchKernelGGL(attn_generic_kernel<true>, grid, dim3(256), 0, s, p);
  else
    hipLaunchKernelGGL(attn_generic_kernel<false>, grid, dim3(256), 0, s, p);
  return hipGetLastError();
}

}  // namespace kvshot
