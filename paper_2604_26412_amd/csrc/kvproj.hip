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
// the same lane.  The reduction runs over L_s d_kv inputs in chunks of 64:
// chunk k0 is half of one head of one source layer, so a token's chunk is 128
// contiguous bytes in the paged pool (gathered through the page table once per
// workgroup) and a weight row's chunk is 128 contiguous bytes.  Both operands
// are staged through LDS, double buffered, one barrier per chunk.  Within a
// chunk, a lane of half h covers reduction indices 32 h .. 32 h + 31 and MFMA
// k-step s takes 32 h + 8 s .. + 7 from both operands (any pairing of operand
// slots with reduction indices gives the same sum when A and B agree).
//
// Epilogue: RoPE in registers (float32, table rows at each token's position),
// bf16 rounding, a transpose through LDS into [token][channel] rows, and
// 16-byte stores of each (token, head) row into its destination page slot.
// With few tokens the reduction is split over workgroups; each writes float32
// partial sums and kvproj_combine_kernel adds them, rotates and scatters.
//
// Work order: channel tile fastest, then split, token tile, tensor.  The
// hardware hands workgroup i to XCD i % 8; xcd_remap gives each XCD a
// contiguous range, so the channel tiles that read one token tile share that
// XCD's L2.
#include "kvproj_common.h"

namespace kvshot {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr int kKC = 64;                           // reduction indices per chunk
constexpr int kPitch = kKC + 8;                   // operand row pitch (bf16): 144 B, rows shift by 4 banks
constexpr int kOpElems = kProjTile * kPitch;      // one operand tile
constexpr int kOutPitch = kProjTile + 8;          // output tile row pitch (bf16)
constexpr int kRows = kProjTile / 32;             // operand rows each thread stages: 32 i + tid / 8
static_assert(kProjTile * kOutPitch <= 4 * kOpElems, "the output tile reuses the operand buffers");

__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 v) { return __builtin_bit_cast(bf16x8, v); }

__device__ __forceinline__ int clampi(int v, int lo, int hi) { return v < lo ? lo : (v > hi ? hi : v); }

template <bool SPLIT>
__global__ __launch_bounds__(256, 1) void kvproj_kernel(KvProjParams p) {
  __shared__ __attribute__((aligned(16))) uint16_t lds[2][2][kOpElems];   // [buffer][weights, tokens]
  __shared__ int64_t t_src[kProjTile];   // source element offset of each token's slot (page, slot)
  __shared__ int64_t t_dst[kProjTile];   // destination element offset
  __shared__ int32_t t_pos[kProjTile];   // position, clamped to the RoPE table
  __shared__ const uint16_t* t_layer[2][kProjMaxLayers];   // source pools [K, V][layer]

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
  const int nchunks = K / kKC;
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
    if (tid == 0) {   // constant indices: the kernel arguments stay in scalar registers
#pragma unroll
      for (int l = 0; l < kProjMaxLayers; ++l) {
        t_layer[0][l] = p.k_src[l];
        t_layer[1][l] = p.v_src[l];
      }
    }
  }
  __syncthreads();

  const int row = tid >> 3;          // staging row within each group of 32
  const int piece = (tid & 7) * 8;   // staging element offset within the chunk
  int64_t soff[kRows];
  int32_t woff[kRows];
#pragma unroll
  for (int i = 0; i < kRows; ++i) {
    soff[i] = t_src[32 * i + row] + piece;
    const int wrow = mt * kProjTile + 32 * i + row;
    woff[i] = (wrow < d_kv ? wrow : d_kv - 1) * K + piece;
  }
  const uint16_t* wsrc = g ? p.w_v : p.w_k;

  u32x4 xr[kRows], wr[kRows];
  auto gload = [&](int c) {
    const int k0 = c * kKC;
    const int l = k0 / d_kv;
    const int rem = k0 - l * d_kv;
    const uint16_t* src = t_layer[g][l] + (int64_t)(rem >> 7) * p.head_stride + (rem & 127);
#pragma unroll
    for (int i = 0; i < kRows; ++i) xr[i] = *(const u32x4*)(src + soff[i]);
#pragma unroll
    for (int i = 0; i < kRows; ++i) wr[i] = *(const u32x4*)(wsrc + woff[i] + k0);
  };
  auto lstore = [&](int buf) {
#pragma unroll
    for (int i = 0; i < kRows; ++i) *(u32x4*)&lds[buf][0][(32 * i + row) * kPitch + piece] = wr[i];
#pragma unroll
    for (int i = 0; i < kRows; ++i) *(u32x4*)&lds[buf][1][(32 * i + row) * kPitch + piece] = xr[i];
  };

  f32x16 acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.0f;

  auto compute = [&](int buf) {
    const uint16_t* A = &lds[buf][0][(128 * wc + (lane & 31)) * kPitch + 32 * hh];
    const uint16_t* B = &lds[buf][1][(128 * wt + (lane & 31)) * kPitch + 32 * hh];
#pragma unroll
    for (int s = 0; s < kKC / 16; ++s) {
      bf16x8 a[4], b[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) a[i] = as_bf16x8(*(const u32x4*)(A + 32 * i * kPitch + 8 * s));
#pragma unroll
      for (int j = 0; j < 4; ++j) b[j] = as_bf16x8(*(const u32x4*)(B + 32 * j * kPitch + 8 * s));
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
    }
  };

  // ---- main loop: chunk c computes from buffer c & 1 while chunk c + 1 is loaded ----
  gload(cbeg);
  lstore(0);
  __syncthreads();
  for (int c = cbeg; c < cend; ++c) {
    const int buf = (c - cbeg) & 1;
    gload(c + 1 < cend ? c + 1 : c);    // the last refill re-reads its own chunk into the idle buffer
    compute(buf);
    lstore(buf ^ 1);
    __syncthreads();
  }

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
    // RoPE (keys), bf16 rounding and a transpose into an LDS tile [token][channel] (the loop's
    // last barrier freed the operand buffers).  Channel m = 32 i + 8 q + 4 hh + e of the head
    // (i < 2) pairs with m + 64, held in block i + 2 of the same lane.
    const bool rot = g == 0 && p.rope_keys;
    uint16_t* O = &lds[0][0][0];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int tl = 128 * wt + 32 * j + (lane & 31);
      const float2* cs = p.rope + (int64_t)t_pos[tl] * kHalfDim;
      uint16_t* orow = O + tl * kOutPitch + 128 * wc + 4 * hh;
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int m = 32 * i + 8 * q + 4 * hh;
          float x1[4], x2[4];
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            x1[e] = acc[i][j][4 * q + e];
            x2[e] = acc[i + 2][j][4 * q + e];
          }
          // branch-free: values take cos = 1, sin = 0, which leaves them exactly as they are
          const float4 c01 = *(const float4*)(cs + m);
          const float4 c23 = *(const float4*)(cs + m + 2);
          const float cv[4] = {rot ? c01.x : 1.0f, rot ? c01.z : 1.0f, rot ? c23.x : 1.0f, rot ? c23.z : 1.0f};
          const float sv[4] = {rot ? c01.y : 0.0f, rot ? c01.w : 0.0f, rot ? c23.y : 0.0f, rot ? c23.w : 0.0f};
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const float y1 = x1[e] * cv[e] - x2[e] * sv[e];
            const float y2 = x2[e] * cv[e] + x1[e] * sv[e];
            x1[e] = y1;
            x2[e] = y2;
          }
          u32x2 v1, v2;
          v1[0] = pack_bf16x2(x1[0], x1[1]);
          v1[1] = pack_bf16x2(x1[2], x1[3]);
          v2[0] = pack_bf16x2(x2[0], x2[1]);
          v2[1] = pack_bf16x2(x2[2], x2[3]);
          *(u32x2*)(orow + 32 * i + 8 * q) = v1;
          *(u32x2*)(orow + 64 + 32 * i + 8 * q) = v2;
        }
    }
    __syncthreads();
    // one (token, head) row is 16 pieces of 16 bytes; thread t stores pieces t, t + 256, ...
    uint16_t* dst = g ? p.v_dst : p.k_dst;
#pragma unroll 4
    for (int it = 0; it < kProjTile * 2 * 16 / 256; ++it) {
      const int id = it * 256 + tid;
      const int tl = id >> 5, hd = (id >> 4) & 1, pc = (id & 15) * 8;
      const int hx = mt * 2 + hd;
      if (n0 + tl < p.n_tokens && hx < p.hkv)
        *(u32x4*)(dst + t_dst[tl] + (int64_t)hx * p.dst_head_stride + pc) =
            *(const u32x4*)(O + tl * kOutPitch + hd * kHeadDim + pc);
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
  if (p.splits > 1)
    hipLaunchKernelGGL(kvproj_kernel<true>, dim3(grid), dim3(256), 0, s, p);
  else
    hipLaunchKernelGGL(kvproj_kernel<false>, dim3(grid), dim3(256), 0, s, p);
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
