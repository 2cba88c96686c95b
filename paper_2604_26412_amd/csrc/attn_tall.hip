// Split-K draft attention for tall query tiles on bf16 MFMA (gfx950): 256
// query rows per (sequence, KV head) and workgroup -- the rows of a draft
// tree (Sec. 3.5: 60 nodes x 4 query heads of a KV group) or of a step call
// with 33..64 draft queries per sequence.  It computes what attn_mfma.hip
// computes (masked softmax attention of each query row over the target prefix
// followed by the visible draft keys, Sec. 3.4.1 Eq. 7 and App. B); only the
// data movement and the query's precision handling differ.
//
// Work: one workgroup of NW waves per (row group, split, KV head, sequence);
// wave w owns query rows 32 (NW rg + w) .. + 31 and all NW waves share every
// 32-key K/V block through LDS, so each block is read from HBM once for all
// 256 rows.
//
// Data movement: K and V blocks go from global memory straight into an LDS
// ring of NBUF blocks (global_load_lds_dwordx4: no register staging, no LDS
// store instructions), NBUF - 1 blocks in flight.  Block it is waited for
// (vmcnt), a barrier makes it visible and frees the buffer of block it - 1,
// which then receives block it + NBUF - 1.  The draft blocks (last split)
// continue the same ring after the target blocks.  Page ids of the split are
// staged in LDS once, so the loop issues no memory reads but its own loads;
// a block's rows 0..15 and 16..31 each lie in one page, whose base address is
// formed in SGPRs, and a lane adds a fixed 32-bit offset.
//
// LDS tiles are unpadded (256-byte rows), with the 16-byte chunks of each row
// permuted (chunk c of row r sits in slot c ^ swz(r)) so that the MFMA operand
// reads hit distinct banks: 16 rows read at one chunk (K) and 4 rows x 64
// bytes read by the transposed V load.
//
// Precision: the rotated, scaled query is carried as a bf16 pair hi + lo (two
// QK products), so the query's rounding leaves the scores; this matters on
// keys with outlier channels, where a single bf16 query moves the output by
// about as much as the whole error budget allows.
#include "attn_mfma_common.h"

namespace kvshot {
namespace {

using namespace mfma;

constexpr int kTallTile = kBlockKeys * kHeadDim * 2;     // 8192 bytes: one 32-key K or V tile
constexpr int kTallMaxBlocks = 512;                      // target blocks per workgroup (page ids staged in LDS)

// Slot of chunk c in K tile row r is c ^ kswz(r): the 16 rows kperm(0..15) read
// at one chunk fall in 16 distinct 16-byte bank groups.
__device__ __forceinline__ int kswz(int r) { return ((r & 3) << 2) | ((r >> 2) & 3); }
// Slot of chunk c in V tile row r is c ^ vswz(r): four consecutive rows read
// at chunks 4 dt .. 4 dt + 3 fall in 16 distinct 16-byte bank groups.
__device__ __forceinline__ int vswz(int r) { return (r & 3) << 2; }

// vmcnt(n) with no wait on the other counters (gfx9 encoding: vmcnt bits [3:0] and [15:14])
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

// Barrier without the memory fence of __syncthreads (which would also wait for
// the ring loads still in flight); the clobber keeps LDS accesses on their side.
__device__ __forceinline__ void lds_barrier() { asm volatile("s_barrier" ::: "memory"); }

typedef __attribute__((address_space(3))) void lds_void;

#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
// One wave-wide 16-byte load from global memory straight into LDS: lane L's
// bytes land at `lds` + 16 L.  M0 holds the wave-uniform LDS address, set one
// wait state ahead.  Inline asm: the compiler's own form would make every
// later LDS read wait for all of these loads in flight.
__device__ __forceinline__ void lds_load_sbase(const void* sbase, uint32_t voff, const void* lds) {
  const uint32_t la = (uint32_t)(uintptr_t)(lds_void*)lds;
  asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, %1" ::"v"(voff), "s"(sbase), "s"(la)
               : "memory", "m0");
}
// Same, with a full 64-bit address per lane.
__device__ __forceinline__ void lds_load_vaddr(const void* src, const void* lds) {
  const uint32_t la = (uint32_t)(uintptr_t)(lds_void*)lds;
  asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off" ::"v"(src), "s"(la)
               : "memory", "m0");
}
#pragma clang diagnostic pop

template <int NW, int NBUF>
__global__ __launch_bounds__(NW * 64, 8 / NW) void attn_tall_kernel(AttnParams p) {
  static_assert(NW == 4 || NW == 8, "4 or 8 waves");
  static_assert(NBUF >= 3, "ring depth");
  constexpr int kLPW = 8 / NW;                   // load instructions per wave, tile and block
  constexpr int kRingBytes = NBUF * 2 * kTallTile;
  __shared__ __attribute__((aligned(16))) unsigned char lds[kRingBytes + kTallMaxBlocks * 8];
  int2* ids = (int2*)(lds + kRingBytes);

  const int lane = threadIdx.x & 63;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int l32 = lane & 31;
  const int hh = lane >> 5;
  int wi = xcd_remap(blockIdx.x, gridDim.x);    // work item: (row group, split, KV head, sequence)
  const int rg = wi % p.row_groups;
  wi /= p.row_groups;
  const int split = wi % p.splits;
  wi /= p.splits;
  const int h = wi % p.hkv;
  const int b = wi / p.hkv;

  int T = clamp_ctx(p.ctx_lens[b], p.max_pages_per_seq, p.page_shift);
  T = T > p.max_ctx ? p.max_ctx : T;
  const int nbt = (T + kBlockKeys - 1) / kBlockKeys;
  const int blk0 = split * p.blocks_per_split;
  const int blk1 = min(blk0 + p.blocks_per_split, nbt);
  int nt = blk1 > blk0 ? blk1 - blk0 : 0;
  nt = nt > kTallMaxBlocks ? kTallMaxBlocks : nt;   // the plan never asks for more
  const bool last = split == p.splits - 1;

  int s0 = 0, S = p.tree ? p.n_nodes : p.nq;
  if (!p.tree) {
    s0 = p.step_offsets[b];
    s0 = s0 < 0 ? 0 : (s0 > p.max_draft - p.nq ? p.max_draft - p.nq : s0);
    S = s0 + p.nq;
  }
  const int nd = last ? (S + kBlockKeys - 1) / kBlockKeys : 0;
  const int ntot = nt + nd;                      // ring blocks: target blocks, then draft blocks
  const int P = position_base(p, b, T);

  // ---- page ids of the split's target blocks (rows 0..15, rows 16..31), clamped into the pool ----
  const int ps = p.page_shift;
  const int pmask = (1 << ps) - 1;
  const int lp_last = T > 0 ? (T - 1) >> ps : 0;
  const int64_t pt_row = (int64_t)b * p.max_pages_per_seq;
  for (int i = threadIdx.x; i < nt; i += NW * 64) {
    const int key0 = (blk0 + i) * kBlockKeys;
    const int la = min(key0 >> ps, lp_last), lb = min((key0 + 16) >> ps, lp_last);
    int pa = p.page_table[pt_row + la], pb = p.page_table[pt_row + lb];
    pa = pa < 0 ? 0 : (pa >= p.num_pages ? p.num_pages - 1 : pa);
    pb = pb < 0 ? 0 : (pb >= p.num_pages ? p.num_pages - 1 : pb);
    ids[i] = make_int2(pa, pb);
  }

  // ---- query rows of this wave: rows (NW rg + w) * 32 + lane % 32, rotated, scaled, split hi + lo ----
  uint64_t anc_mine = 0;
  int depth_mine = 0;
  if (p.tree) anc_mine = tree_ancestry_wave(p.parents + (int64_t)b * p.n_nodes, p.n_nodes, lane, &depth_mine);
  const int r = (rg * NW + w) * 32 + l32;
  const bool row_ok = r < p.rows;
  const int rr = row_ok ? r : p.rows - 1;
  const int jrow = rr / p.group;
  const int hqr = h * p.group + (rr - jrow * p.group);
  uint64_t row_anc = 0;
  int qpos;
  if (p.tree) {
    const int node = query_node(p, b, jrow);
    const uint32_t lo = __shfl((uint32_t)anc_mine, node), hi = __shfl((uint32_t)(anc_mine >> 32), node);
    row_anc = ((uint64_t)hi << 32) | lo;
    qpos = P + __shfl(depth_mine, node);
  } else {
    qpos = P + s0 + jrow;
  }
  qpos = qpos >= p.max_position ? p.max_position - 1 : qpos;
  bf16x8 qhi[8], qlo[8];
  {
    const uint16_t* qp = (const uint16_t*)p.q + (((int64_t)b * p.nq + jrow) * p.hq + hqr) * kHeadDim + hh * 8;
    u32x4 raw[8];
#pragma unroll
    for (int kc = 0; kc < 8; ++kc) raw[kc] = *(const u32x4*)(qp + kc * 16);
    rope_rotate_split(raw, p.rope + (int64_t)qpos * kHalfDim + hh * 8, row_ok ? p.qscale : 0.0f, qhi, qlo);
  }
  __syncthreads();                               // page ids visible; every load above has returned

  // ---- ring loads.  Load instruction t (0..7) of a tile fills rows 4t .. 4t+3: lane L takes row
  // 4t + L / 16 and the chunk that belongs in slot L % 16.  Wave w issues instructions w kLPW .. ----
  const int64_t pstr_b = p.page_stride * 2, hoff_b = (int64_t)h * p.head_stride * 2;
  const uint32_t sstr_b = (uint32_t)(p.slot_stride * 2);
  const char* kbase = (const char*)p.k_pages;
  const char* vbase = (const char*)p.v_pages;
  uint32_t kvo[kLPW], vvo[kLPW];                // lane offsets from the half-page base
  int lrow[kLPW], kchunk[kLPW], vchunk[kLPW];
#pragma unroll
  for (int i = 0; i < kLPW; ++i) {
    const int t = w * kLPW + i;
    lrow[i] = 4 * t + (lane >> 4);
    kchunk[i] = (lane & 15) ^ kswz(lrow[i]);
    vchunk[i] = (lane & 15) ^ vswz(lrow[i]);
    kvo[i] = (uint32_t)(lrow[i] & 15) * sstr_b + (uint32_t)kchunk[i] * 16u;
    vvo[i] = (uint32_t)(lrow[i] & 15) * sstr_b + (uint32_t)vchunk[i] * 16u;
  }
  // all of this wave's instructions of a block lie in one half of it (rows 0..15 or 16..31)
  const bool upper = (w * kLPW) >= 4;
  const uint16_t* dkbase = (const uint16_t*)p.draft_k;
  const uint16_t* dvbase = (const uint16_t*)p.draft_v;
  auto issue = [&](int it, int buf) {
    it = it < ntot ? it : ntot - 1;              // past the end: repeat the last block (keeps vmcnt uniform)
    unsigned char* kt = lds + buf * 2 * kTallTile;
    unsigned char* vt = kt + kTallTile;
    if (it < nt) {
      const int key0 = (blk0 + it) * kBlockKeys;
      const int2 pid = ids[it];
      if (key0 + kBlockKeys <= T) {
        const int page = __builtin_amdgcn_readfirstlane(upper ? pid.y : pid.x);
        const int hk = key0 + (upper ? 16 : 0);
        const int64_t off = (int64_t)page * pstr_b + hoff_b + (int64_t)(hk & pmask) * sstr_b;
#pragma unroll
        for (int i = 0; i < kLPW; ++i) {
          const int t = w * kLPW + i;
          lds_load_sbase(kbase + off, kvo[i], kt + t * 1024);
          lds_load_sbase(vbase + off, vvo[i], vt + t * 1024);
        }
      } else {
        // the block holding position T - 1: rows past it load row T - 1 (finite, masked out)
#pragma unroll
        for (int i = 0; i < kLPW; ++i) {
          const int t = w * kLPW + i;
          const int key = min(key0 + lrow[i], T - 1);
          const int page = (key >> ps) == (key0 >> ps) ? pid.x : pid.y;
          const int64_t e = (int64_t)page * pstr_b + hoff_b + (int64_t)(key & pmask) * sstr_b;
          lds_load_vaddr(kbase + e + kchunk[i] * 16, kt + t * 1024);
          lds_load_vaddr(vbase + e + vchunk[i] * 16, vt + t * 1024);
        }
      }
    } else {
      // draft keys (raw, rotated after the operand read); rows past S load row S - 1
      const int dkey0 = (it - nt) * kBlockKeys;
#pragma unroll
      for (int i = 0; i < kLPW; ++i) {
        const int t = w * kLPW + i;
        const int s = min(dkey0 + lrow[i], S - 1);
        const int64_t e = draft_offset(b, s, h, p.max_draft, p.hkv);
        lds_load_vaddr(dkbase + e + kchunk[i] * 8, kt + t * 1024);
        lds_load_vaddr(dvbase + e + vchunk[i] * 8, vt + t * 1024);
      }
    }
  };

  // ---- operand read addresses (bytes within a tile) ----
  // K operand row rho = l32 reads tile row kperm(rho), so that accumulator register v of lane
  // (row, hh) holds key 16 (v / 8) + 8 hh + v % 8; chunk 2 kc + hh of that row.
  const int kperm = ((l32 >> 4) << 4) + (((l32 >> 2) & 1) << 3) + (((l32 >> 3) & 1) << 2) + (l32 & 3);
  const int kr_base = kperm * 256;
  const int ks = kswz(kperm);
  // transposed V read: 16-lane group gr reads keys 8 (gr / 2) + (lane % 16) / 4 (+ 4 for the second
  // read, + 16 for the second key half) of channels 32 dt + 16 (gr % 2) + 4 (lane % 4) .. + 3
  const int gr = lane >> 4, sg = lane & 15;
  const int vrow = (gr >> 1) * 8 + (sg >> 2);           // +4 and +16 keep vswz (it uses r % 4 only)
  const int vcc = 2 * (gr & 1) + ((sg & 3) >> 1);       // chunk within the 64-byte group of dt
  const int v_rd = vrow * 256 + 8 * (sg & 1);
  const int vs = vswz(vrow);

  auto read_k = [&](const unsigned char* kt, u32x4 (&kop)[8]) {
#pragma unroll
    for (int kc = 0; kc < 8; ++kc) kop[kc] = *(const u32x4*)(kt + kr_base + 16 * ((2 * kc + hh) ^ ks));
  };
  auto read_v = [&](const unsigned char* vt, bf16x8 (&vop)[4][2]) {
    typedef __attribute__((address_space(3))) s16x4 lds_s16x4;
    const __attribute__((address_space(3))) unsigned char* vb =
        (const __attribute__((address_space(3))) unsigned char*)(vt) + v_rd;
#pragma unroll
    for (int dt = 0; dt < 4; ++dt) {
      const int co = 16 * ((4 * dt + vcc) ^ vs);
#pragma unroll
      for (int sidx = 0; sidx < 2; ++sidx) {
        const s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(vb + co + (16 * sidx) * 256));
        const s16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(vb + co + (16 * sidx + 4) * 256));
        const u32x2 lo2 = __builtin_bit_cast(u32x2, lo), hi2 = __builtin_bit_cast(u32x2, hi);
        vop[dt][sidx] = as_bf16x8(u32x4{lo2[0], lo2[1], hi2[0], hi2[1]});
      }
    }
  };

  // Rotate the raw draft keys of this wave's rows of a K tile in place: row lrow[i] holds draft key
  // key0 + lrow[i] at position P + s (step) or P + depth(s) (tree); lane L holds chunk kchunk[i] (channels
  // 8 c .. 8 c + 7), whose RoPE partners (m, m + 64) are chunk c ^ 8 of the same row.
  auto rotate_draft_rows = [&](unsigned char* kt, int key0) {
#pragma unroll
    for (int i = 0; i < kLPW; ++i) {
      const int row = lrow[i];
      const int c = kchunk[i];
      const int s = min(key0 + row, S - 1);
      int kpos = p.tree ? P + __shfl(depth_mine, s & 63) : P + s;
      kpos = kpos >= p.max_position ? p.max_position - 1 : kpos;
      unsigned char* rowp = kt + row * 256;
      const u32x4 mine = *(const u32x4*)(rowp + 16 * (c ^ kswz(row)));
      const u32x4 part = *(const u32x4*)(rowp + 16 * ((c ^ 8) ^ kswz(row)));
      const float2* cs = p.rope + (int64_t)kpos * kHalfDim + 8 * (c & 7);
      const float sign = c < 8 ? -1.0f : 1.0f;   // first half: x cos - y sin; second half: x cos + y sin
      u32x4 outv;
#pragma unroll
      for (int e2 = 0; e2 < 4; ++e2) {
        const float2 ca = cs[2 * e2], cb = cs[2 * e2 + 1];
        const float xa = bf16_lo(mine[e2]), xb = bf16_hi(mine[e2]);
        const float ya = bf16_lo(part[e2]), yb = bf16_hi(part[e2]);
        outv[e2] = pack_bf16x2(xa * ca.x + sign * ya * ca.y, xb * cb.x + sign * yb * cb.y);
      }
      *(u32x4*)(rowp + 16 * (c ^ kswz(row))) = outv;
    }
  };

  f32x16 oacc[4];
#pragma unroll
  for (int dt = 0; dt < 4; ++dt) oacc[dt] = f32x16{};
  SoftmaxState st{-INFINITY, 0.0f};

  // one block: S^T = K (Qhi + Qlo)^T, mask, online softmax, O^T += V^T P^T
  auto compute = [&](const bf16x8 (&kop)[8], const unsigned char* vt, bool masked, uint32_t valid) {
    f32x16 sacc = f32x16{};
#pragma unroll
    for (int kc = 0; kc < 8; ++kc) {
      sacc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kop[kc], qhi[kc], sacc, 0, 0, 0);
      sacc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kop[kc], qlo[kc], sacc, 0, 0, 0);
    }
    bf16x8 vop[4][2];
    read_v(vt, vop);
    if (masked) apply_mask(sacc, valid);
    u32x4 pw[2];
    float alpha;
    bool rescale;
    softmax_front(sacc, st, pw, alpha, rescale);
    if (rescale) {
#pragma unroll
      for (int dt = 0; dt < 4; ++dt)
#pragma unroll
        for (int v = 0; v < 16; ++v) oacc[dt][v] *= alpha;
    }
#pragma unroll
    for (int dt = 0; dt < 4; ++dt)
#pragma unroll
      for (int sidx = 0; sidx < 2; ++sidx)
        oacc[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vop[dt][sidx], as_bf16x8(pw[sidx]), oacc[dt], 0, 0, 0);
  };

  if (ntot > 0) {
#pragma unroll
    for (int u = 0; u < NBUF - 1; ++u) issue(u, u);
    int ibuf = NBUF - 1;                         // buffer the next issue fills
    int cbuf = 0;                                // buffer of block it
    for (int it = 0; it < ntot; ++it) {
      // this wave's loads of block it are done once at most the NBUF - 2 younger blocks remain
      wait_vmcnt<(NBUF - 2) * 2 * kLPW>();
      lds_barrier();                             // everyone's block it has landed; block it - 1 is done
      issue(it + NBUF - 1, ibuf);
      ibuf = ibuf == NBUF - 1 ? 0 : ibuf + 1;
      unsigned char* kt = lds + cbuf * 2 * kTallTile;
      const unsigned char* vt = kt + kTallTile;
      cbuf = cbuf == NBUF - 1 ? 0 : cbuf + 1;
      uint32_t valid = 0xffffu;
      bool masked;
      if (it < nt) {
        const int key0 = (blk0 + it) * kBlockKeys;
        masked = key0 + kBlockKeys > T;
        if (masked) {
          valid = 0;
#pragma unroll
          for (int v = 0; v < 16; ++v) valid |= (uint32_t)(key0 + 16 * (v >> 3) + 8 * hh + (v & 7) < T) << v;
        }
      } else {
        // draft block: this wave rotates its own rows of the raw keys in place (chunk c pairs with
        // chunk c ^ 8, in the same row), then the barrier publishes the rotated tile
        const int key0 = (it - nt) * kBlockKeys;
        rotate_draft_rows(kt, key0);
        __builtin_amdgcn_s_waitcnt(0xc07f);      // lgkmcnt(0): this wave's rotated rows are written
        lds_barrier();
        masked = true;
        valid = 0;
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const int s = key0 + 16 * (v >> 3) + 8 * hh + (v & 7);
          bool ok = s < S;
          if (p.tree) ok = ok && ((row_anc >> (s & 63)) & 1ull);
          else ok = ok && (s <= s0 + jrow);
          valid |= (uint32_t)ok << v;
        }
      }
      u32x4 kraw[8];
      read_k(kt, kraw);
      bf16x8 kop[8];
#pragma unroll
      for (int kc = 0; kc < 8; ++kc) kop[kc] = as_bf16x8(kraw[kc]);
      compute(kop, vt, masked, valid);
    }
    wait_vmcnt<0>();                             // the repeat loads past the end drain before exit
  }

  // ---- write: final output (one split) or split partial ----
  if (!row_ok) return;
  const float l_row = st.l + __shfl_xor(st.l, 32);
  const float M = st.m;
  if (p.splits == 1) {
    const float inv = 1.0f / l_row;
    const int64_t orow = (((int64_t)b * p.nq + jrow) * p.hq + hqr) * kHeadDim;
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
    if (p.lse && hh == 0) p.lse[((int64_t)b * p.nq + jrow) * p.hq + hqr] = (M + __log2f(l_row)) * kLn2;
  } else {
    const int64_t prow = (((int64_t)b * p.hkv + h) * p.rows_pad + r) * p.splits + split;
    float* po = p.part_o + prow * kHeadDim;
#pragma unroll
    for (int dt = 0; dt < 4; ++dt)
#pragma unroll
      for (int q4 = 0; q4 < 4; ++q4) {
        const int d = dt * 32 + q4 * 8 + hh * 4;
        *(f32x4*)(po + d) =
            f32x4{oacc[dt][q4 * 4 + 0], oacc[dt][q4 * 4 + 1], oacc[dt][q4 * 4 + 2], oacc[dt][q4 * 4 + 3]};
      }
    if (hh == 0) p.part_ml[prow] = make_float2(M, l_row);
  }
}

}  // namespace

#ifndef KVSHOT_TALL_WAVES
#define KVSHOT_TALL_WAVES 8
#endif
#ifndef KVSHOT_TALL_NBUF
#define KVSHOT_TALL_NBUF 4
#endif

int tall_waves_per_wg() { return KVSHOT_TALL_WAVES; }
int tall_max_blocks() { return kTallMaxBlocks; }

hipError_t launch_attn_tall(const AttnParams& p, hipStream_t s) {
  const dim3 grid((unsigned)((int64_t)p.splits * p.row_groups * p.hkv * p.batch));
  hipLaunchKernelGGL((attn_tall_kernel<KVSHOT_TALL_WAVES, KVSHOT_TALL_NBUF>), grid, dim3(KVSHOT_TALL_WAVES * 64), 0,
                     s, p);
  return hipGetLastError();
}

}  // namespace kvshot
