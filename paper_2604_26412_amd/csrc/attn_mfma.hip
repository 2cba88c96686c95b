// Split-K flash-decode draft attention on bf16 MFMA (gfx950).
//
// One workgroup serves one (split, KV head, sequence).  Its query tile is every
// query head of the KV head's group times every draft query of the sequence
// (rows = G * n), so each target K/V block is read from HBM once for all of
// them (grouped-query folding).  The memory attended is the target prefix of
// the sequence followed by its draft keys (Sec. 3.4.1, Eq. 7; App. B).
//
// Per 32-key block a wave computes S^T = K * Q^T with v_mfma_f32_32x32x16_bf16,
// so each lane ends up owning one query row (lane % 32) and 16 of the block's
// keys: the online-softmax row max needs one cross-half exchange and the
// rescale of the output accumulator is lane-local.  O^T = V^T * P^T runs on the
// same MFMA; V is transposed through LDS.  K goes straight from HBM into the
// MFMA operand registers.
//
// Row tiles: rows are padded to 32 * RT.  A workgroup has NW waves; wave w
// owns row tile w % RT and key stream w / RT; the KS = NW / RT key streams
// interleave 32-key blocks and are merged through LDS at the end.
#include "kvshot_common.h"

namespace kvshot {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr int kVtPitch = 40;                               // bf16 per V^T row: 32 keys + 8 pad (80 B)
constexpr int kVtBytes = kHeadDim * kVtPitch * 2;          // 10 KB per wave
constexpr float kLn2 = 0.693147180559945309f;

__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 v) { return __builtin_bit_cast(bf16x8, v); }

__device__ __forceinline__ int32_t load_scalar_i32(const int32_t* base, int64_t idx) {
  // uniform address -> scalar load (constant address space)
  const __attribute__((address_space(4))) int32_t* cp =
      (const __attribute__((address_space(4))) int32_t*)(base);
  return cp[idx];
}

// Rotate one lane's (d, d + 64) pairs by the table angles and scale; q chunk kc
// holds d = kc * 16 + hh * 8 + e, so chunks kc and kc + 4 pair up in-lane.
__device__ __forceinline__ void rope_rotate_to_bf16(const u32x4 (&raw)[8], const float2* cs, float scale,
                                                    bf16x8 (&dst)[8]) {
#pragma unroll
  for (int kc = 0; kc < 4; ++kc) {
    u32x4 lo, hi;
#pragma unroll
    for (int e2 = 0; e2 < 4; ++e2) {
      const uint32_t a = raw[kc][e2], bq = raw[kc + 4][e2];
      const float x1a = bf16_lo(a), x1b = bf16_hi(a);
      const float x2a = bf16_lo(bq), x2b = bf16_hi(bq);
      const float2 ca = cs[kc * 16 + 2 * e2], cb = cs[kc * 16 + 2 * e2 + 1];
      const float y1a = (x1a * ca.x - x2a * ca.y) * scale, y1b = (x1b * cb.x - x2b * cb.y) * scale;
      const float y2a = (x2a * ca.x + x1a * ca.y) * scale, y2b = (x2b * cb.x + x1b * cb.y) * scale;
      lo[e2] = pack_bf16x2(y1a, y1b);
      hi[e2] = pack_bf16x2(y2a, y2b);
    }
    dst[kc] = as_bf16x8(lo);
    dst[kc + 4] = as_bf16x8(hi);
  }
}

// Write one lane's V chunk (key `key`, d = t * 16 + hh * 8 + e) transposed into V^T.
__device__ __forceinline__ void store_vt(uint16_t* vt, const u32x4 (&v)[8], int key, int hh) {
#pragma unroll
  for (int t = 0; t < 8; ++t) {
#pragma unroll
    for (int e2 = 0; e2 < 4; ++e2) {
      const int d = t * 16 + hh * 8 + 2 * e2;
      vt[d * kVtPitch + key] = (uint16_t)(v[t][e2] & 0xffffu);
      vt[(d + 1) * kVtPitch + key] = (uint16_t)(v[t][e2] >> 16);
    }
  }
}

struct SoftmaxState {
  float m;   // running max (log2 units), identical in both lane halves
  float l;   // this lane's partial sum over its keys
};

// One 32-key block: S^T from K operands, masked online softmax, O^T += V^T P^T.
// `valid` bit v: key of accumulator register v is visible to this lane's row.
__device__ __forceinline__ void attend_block(const bf16x8 (&kop)[8], const bf16x8 (&qop)[8], const uint16_t* vt,
                                             int l32, int hh, uint32_t valid, f32x16 (&oacc)[4],
                                             SoftmaxState& st) {
  f32x16 s = {};
#pragma unroll
  for (int kc = 0; kc < 8; ++kc) s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kop[kc], qop[kc], s, 0, 0, 0);

  float bm = -INFINITY;
#pragma unroll
  for (int v = 0; v < 16; ++v) {
    s[v] = ((valid >> v) & 1u) ? s[v] : -INFINITY;
    bm = fmaxf(bm, s[v]);
  }
  bm = fmaxf(bm, __shfl_xor(bm, 32));
  const float mn = fmaxf(st.m, bm);
  const float mu = mn == -INFINITY ? 0.0f : mn;
  const float alpha = __builtin_amdgcn_exp2f(st.m - mu);
  float ps = 0.0f;
  u32x4 pw[2];
#pragma unroll
  for (int v = 0; v < 16; v += 2) {
    const float p0 = __builtin_amdgcn_exp2f(s[v] - mu);
    const float p1 = __builtin_amdgcn_exp2f(s[v + 1] - mu);
    ps += p0 + p1;
    pw[v >> 3][(v & 7) >> 1] = pack_bf16x2(p0, p1);
  }
  st.l = st.l * alpha + ps;
  st.m = mn;
  if (__any(alpha != 1.0f)) {
#pragma unroll
    for (int dt = 0; dt < 4; ++dt)
#pragma unroll
      for (int v = 0; v < 16; ++v) oacc[dt][v] *= alpha;
  }
#pragma unroll
  for (int dt = 0; dt < 4; ++dt) {
#pragma unroll
    for (int sidx = 0; sidx < 2; ++sidx) {
      const u32x4 a = *(const u32x4*)(vt + (dt * 32 + l32) * kVtPitch + 16 * sidx + 8 * hh);
      oacc[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(a), as_bf16x8(pw[sidx]), oacc[dt], 0, 0, 0);
    }
  }
}

__device__ __forceinline__ void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

template <int RT, int NW>
__global__ __launch_bounds__(NW * 64) void attn_mfma_kernel(AttnParams p) {
  constexpr int KS = NW / RT;
  constexpr int kMergeBytes = (KS - 1) * RT * 64 * (64 * 4 + 8);
  constexpr int kLdsBytes = (NW * kVtBytes > kMergeBytes) ? NW * kVtBytes : kMergeBytes;
  __shared__ __attribute__((aligned(16))) unsigned char lds[kLdsBytes];

  const int lane = threadIdx.x & 63;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);   // wave index, kept in an SGPR
  const int rt = w % RT;
  const int ks = w / RT;
  const int l32 = lane & 31;
  const int hh = lane >> 5;
  const int split = blockIdx.x, h = blockIdx.y, b = blockIdx.z;

  int T = clamp_ctx(p.ctx_lens[b], p.max_pages_per_seq, p.page_shift);
  T = T > p.max_ctx ? p.max_ctx : T;
  const int nbt = (T + kBlockKeys - 1) / kBlockKeys;
  const int blk0 = split * p.blocks_per_split;
  const int blk1 = min(blk0 + p.blocks_per_split, nbt);
  const bool last = split == p.splits - 1;

  int s0 = 0, S = p.nq;
  if (!p.tree) {
    s0 = p.step_offsets[b];
    s0 = s0 < 0 ? 0 : (s0 > p.max_draft - p.nq ? p.max_draft - p.nq : s0);
    S = s0 + p.nq;
  }

  // query row of this lane
  const int r = rt * 32 + l32;
  const bool row_ok = r < p.rows;
  const int rr = row_ok ? r : p.rows - 1;
  const int j = rr / p.group;
  const int g = rr - j * p.group;
  const int hq = h * p.group + g;

  uint64_t anc_mine = 0, row_anc = 0;
  int depth_mine = 0, qpos;
  if (p.tree) {
    anc_mine = tree_ancestry_wave(p.parents + (int64_t)b * p.nq, p.nq, lane, &depth_mine);
    const uint32_t lo = __shfl((uint32_t)anc_mine, j), hi = __shfl((uint32_t)(anc_mine >> 32), j);
    row_anc = ((uint64_t)hi << 32) | lo;
    qpos = T + __shfl(depth_mine, j);
  } else {
    qpos = T + s0 + j;
  }
  qpos = qpos >= p.max_position ? p.max_position - 1 : qpos;

  // ---- query operand: rotated, scaled into log2 units, bf16 ----
  bf16x8 qop[8];
  {
    const uint16_t* qp = (const uint16_t*)p.q + (((int64_t)b * p.nq + j) * p.hq + hq) * kHeadDim + hh * 8;
    u32x4 raw[8];
#pragma unroll
    for (int kc = 0; kc < 8; ++kc) raw[kc] = *(const u32x4*)(qp + kc * 16);
    rope_rotate_to_bf16(raw, p.rope + (int64_t)qpos * kHalfDim + hh * 8, row_ok ? p.qscale : 0.0f, qop);
  }

  uint16_t* vt = (uint16_t*)(lds + w * kVtBytes);

  // K-operand row rho = l32 holds key kperm(rho), chosen so that accumulator
  // register v of lane (row, hh) holds key 16 * (v / 8) + 8 * hh + v % 8.
  const int kperm = ((l32 >> 4) << 4) + (((l32 >> 2) & 1) << 3) + (((l32 >> 3) & 1) << 2) + (l32 & 3);

  f32x16 oacc[4];
#pragma unroll
  for (int dt = 0; dt < 4; ++dt) oacc[dt] = f32x16{};
  SoftmaxState st{-INFINITY, 0.0f};

  const int64_t ps = p.page_stride, hs = p.head_stride, ss = p.slot_stride;
  const uint16_t* kbase = (const uint16_t*)p.k_pages;
  const uint16_t* vbase = (const uint16_t*)p.v_pages;
  const int pmask = (1 << p.page_shift) - 1;
  const int lp_last = T > 0 ? (T - 1) >> p.page_shift : 0;

  // ---- target blocks: blk = blk0 + ks + KS * i ----
  int blk = blk0 + ks;
  u32x4 kcur[8], vcur[8];
  int pidA = 0, pidB = 0;
  auto block_pids = [&](int bk, int& a, int& bb) {
    const int key0 = bk * kBlockKeys;
    int la = key0 >> p.page_shift, lb = (key0 + 16) >> p.page_shift;
    la = la > lp_last ? lp_last : la;
    lb = lb > lp_last ? lp_last : lb;
    const int64_t row = (int64_t)b * p.max_pages_per_seq;
    a = load_scalar_i32(p.page_table, row + la);
    bb = load_scalar_i32(p.page_table, row + lb);
    a = a < 0 ? 0 : (a >= p.num_pages ? p.num_pages - 1 : a);
    bb = bb < 0 ? 0 : (bb >= p.num_pages ? p.num_pages - 1 : bb);
  };
  auto issue_loads = [&](int bk, int a, int bb, u32x4 (&kd)[8], u32x4 (&vd)[8]) {
    const int key0 = bk * kBlockKeys;
    // for page sizes >= 32 both halves of the block share one page (a == bb)
    const int kk = key0 + kperm;
    const int kpid = (kperm >= 16) ? bb : a;
    const uint16_t* kp = kbase + kv_offset(kpid, h, kk & pmask, ps, hs, ss) + hh * 8;
    const int vk = key0 + l32;
    const int vpid = (l32 >= 16) ? bb : a;
    const uint16_t* vp = vbase + kv_offset(vpid, h, vk & pmask, ps, hs, ss) + hh * 8;
#pragma unroll
    for (int kc = 0; kc < 8; ++kc) kd[kc] = *(const u32x4*)(kp + kc * 16);
#pragma unroll
    for (int t = 0; t < 8; ++t) vd[t] = *(const u32x4*)(vp + t * 16);
  };

  if (blk < blk1) {
    block_pids(blk, pidA, pidB);
    issue_loads(blk, pidA, pidB, kcur, vcur);
  }
  for (; blk < blk1; blk += KS) {
    const int key0 = blk * kBlockKeys;
    const int nblk = blk + KS;
    int nA = 0, nB = 0;
    if (nblk < blk1) block_pids(nblk, nA, nB);
    const bool tail = key0 + kBlockKeys > T;
    if (tail) {
      // zero V rows past the prefix so masked weights never meet NaN
      if (key0 + l32 >= T) {
#pragma unroll
        for (int t = 0; t < 8; ++t) vcur[t] = u32x4{0u, 0u, 0u, 0u};
      }
    }
    store_vt(vt, vcur, l32, hh);
    wave_lds_sync();
    bf16x8 kop[8];
#pragma unroll
    for (int kc = 0; kc < 8; ++kc) kop[kc] = as_bf16x8(kcur[kc]);
    if (nblk < blk1) issue_loads(nblk, nA, nB, kcur, vcur);
    uint32_t valid = 0xffffu;
    if (tail) {
      valid = 0;
#pragma unroll
      for (int v = 0; v < 16; ++v) valid |= (uint32_t)(key0 + 16 * (v >> 3) + 8 * hh + (v & 7) < T) << v;
    }
    attend_block(kop, qop, vt, l32, hh, valid, oacc, st);
    wave_lds_sync();
  }

  // ---- draft blocks (last split only): keys 0..S-1 ----
  if (last) {
    const int nbd = (S + kBlockKeys - 1) / kBlockKeys;
    int depth_k = 0;
    for (int db = ks; db < nbd; db += KS) {
      const int key0 = db * kBlockKeys;
      const int ks_k = key0 + kperm;          // draft key behind this lane's K row
      const int ks_v = key0 + l32;            // draft key behind this lane's V row
      const int sk = ks_k < S ? ks_k : S - 1;
      const int sv = ks_v < S ? ks_v : S - 1;
      const uint16_t* kp = (const uint16_t*)p.draft_k + draft_offset(b, sk, h, p.max_draft, p.hkv) + hh * 8;
      const uint16_t* vp = (const uint16_t*)p.draft_v + draft_offset(b, sv, h, p.max_draft, p.hkv) + hh * 8;
      u32x4 kraw[8], vraw[8];
#pragma unroll
      for (int kc = 0; kc < 8; ++kc) kraw[kc] = *(const u32x4*)(kp + kc * 16);
#pragma unroll
      for (int t = 0; t < 8; ++t) vraw[t] = *(const u32x4*)(vp + t * 16);
      if (ks_v >= S) {
#pragma unroll
        for (int t = 0; t < 8; ++t) vraw[t] = u32x4{0u, 0u, 0u, 0u};
      }
      int kpos;
      if (p.tree) {
        depth_k = __shfl(depth_mine, sk & 63);
        kpos = T + depth_k;
      } else {
        kpos = T + sk;
      }
      kpos = kpos >= p.max_position ? p.max_position - 1 : kpos;
      bf16x8 kop[8];
      rope_rotate_to_bf16(kraw, p.rope + (int64_t)kpos * kHalfDim + hh * 8, 1.0f, kop);
      store_vt(vt, vraw, l32, hh);
      wave_lds_sync();
      uint32_t valid = 0;
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int s = key0 + 16 * (v >> 3) + 8 * hh + (v & 7);
        bool ok = s < S;
        if (p.tree) ok = ok && ((row_anc >> (s & 63)) & 1ull);
        else ok = ok && (s <= s0 + j);
        valid |= (uint32_t)ok << v;
      }
      attend_block(kop, qop, vt, l32, hh, valid, oacc, st);
      wave_lds_sync();
    }
  }

  // ---- merge the key streams of each row tile ----
  float l_row = st.l + __shfl_xor(st.l, 32);
  float M = st.m;
  if constexpr (KS > 1) {
    __syncthreads();
    float* mo = (float*)lds;
    float2* mml = (float2*)(lds + (KS - 1) * RT * 64 * 64 * 4);
    if (ks > 0) {
      const int slot = (ks - 1) * RT + rt;
#pragma unroll
      for (int dt = 0; dt < 4; ++dt)
#pragma unroll
        for (int v = 0; v < 16; ++v) mo[(slot * 64 + dt * 16 + v) * 64 + lane] = oacc[dt][v];
      mml[slot * 64 + lane] = make_float2(st.m, l_row);
    }
    __syncthreads();
    if (ks == 0) {
      float mk[KS - 1], lk[KS - 1];
#pragma unroll
      for (int k = 0; k < KS - 1; ++k) {
        const float2 t = mml[(k * RT + rt) * 64 + lane];
        mk[k] = t.x;
        lk[k] = t.y;
        M = fmaxf(M, t.x);
      }
      const float Mu = M == -INFINITY ? 0.0f : M;
      const float f0 = __builtin_amdgcn_exp2f(st.m - Mu);
      l_row *= f0;
#pragma unroll
      for (int dt = 0; dt < 4; ++dt)
#pragma unroll
        for (int v = 0; v < 16; ++v) oacc[dt][v] *= f0;
#pragma unroll
      for (int k = 0; k < KS - 1; ++k) {
        const float fk = __builtin_amdgcn_exp2f(mk[k] - Mu);
        l_row += lk[k] * fk;
        const int slot = k * RT + rt;
#pragma unroll
        for (int dt = 0; dt < 4; ++dt)
#pragma unroll
          for (int v = 0; v < 16; ++v) oacc[dt][v] += mo[(slot * 64 + dt * 16 + v) * 64 + lane] * fk;
      }
    }
  }
  if (ks != 0 || !row_ok) return;

  // ---- write: final output (one split) or split partial ----
  if (p.splits == 1) {
    const float inv = 1.0f / l_row;
    const int64_t orow = (((int64_t)b * p.nq + j) * p.hq + hq) * kHeadDim;
#pragma unroll
    for (int dt = 0; dt < 4; ++dt) {
#pragma unroll
      for (int q4 = 0; q4 < 4; ++q4) {
        const int d = dt * 32 + q4 * 8 + hh * 4;
        const float o0 = oacc[dt][q4 * 4 + 0] * inv, o1 = oacc[dt][q4 * 4 + 1] * inv;
        const float o2 = oacc[dt][q4 * 4 + 2] * inv, o3 = oacc[dt][q4 * 4 + 3] * inv;
        if (p.out_fp32) {
          *(f32x4*)((float*)p.out + orow + d) = f32x4{o0, o1, o2, o3};
        } else {
          *(u32x2*)((uint16_t*)p.out + orow + d) = u32x2{pack_bf16x2(o0, o1), pack_bf16x2(o2, o3)};
        }
      }
    }
    if (p.lse && hh == 0) p.lse[((int64_t)b * p.nq + j) * p.hq + hq] = (M + __log2f(l_row)) * kLn2;
  } else {
    const int64_t prow = (((int64_t)b * p.hkv + h) * p.rows_pad + r) * p.splits + split;
    float* po = p.part_o + prow * kHeadDim;
#pragma unroll
    for (int dt = 0; dt < 4; ++dt)
#pragma unroll
      for (int q4 = 0; q4 < 4; ++q4) {
        const int d = dt * 32 + q4 * 8 + hh * 4;
        *(f32x4*)(po + d) = f32x4{oacc[dt][q4 * 4 + 0], oacc[dt][q4 * 4 + 1], oacc[dt][q4 * 4 + 2],
                                  oacc[dt][q4 * 4 + 3]};
      }
    if (hh == 0) p.part_ml[prow] = make_float2(M, l_row);
  }
}

}  // namespace

int mfma_waves_per_wg(int row_tiles) { return row_tiles >= 8 ? 8 : 4; }

hipError_t launch_attn_mfma(const AttnParams& p, int row_tiles, hipStream_t s) {
  const dim3 grid(p.splits, p.hkv, p.batch);
  switch (row_tiles) {
    case 1: hipLaunchKernelGGL((attn_mfma_kernel<1, 4>), grid, dim3(256), 0, s, p); break;
    case 2: hipLaunchKernelGGL((attn_mfma_kernel<2, 4>), grid, dim3(256), 0, s, p); break;
    case 4: hipLaunchKernelGGL((attn_mfma_kernel<4, 4>), grid, dim3(256), 0, s, p); break;
    case 8: hipLaunchKernelGGL((attn_mfma_kernel<8, 8>), grid, dim3(512), 0, s, p); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace kvshot
