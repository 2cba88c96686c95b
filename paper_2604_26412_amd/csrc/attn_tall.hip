// Split-K draft attention for tall query tiles on bf16 MFMA (gfx950): 256
// query rows per (sequence, KV head) and workgroup -- the rows of a draft
// tree (Sec. 3.5: 60 nodes x 4 query heads of a KV group) or of a step call
// with 33..64 draft queries per sequence.  It computes what attn_mfma.hip
// computes (masked softmax attention of each query row over the target prefix
// followed by the visible draft keys, Sec. 3.4.1 Eq. 7 and App. B); only the
// data movement and the query's precision handling differ.
//
// Work: one workgroup of 8 waves per (row group, split, KV head, sequence);
// wave w owns query rows 32 (8 rg + w) .. + 31 and all 8 waves share every
// 32-key K/V block through LDS, so each block is read from HBM once for all
// 256 rows.  Waves w and w + 4 share a SIMD: waves 0..3 run each block as
// QK, softmax, PV, while waves 4..7 run the previous block's softmax and PV
// around this block's QK products, so the two waves of a SIMD tend to be in
// different phases (matrix core vs vector ALU) instead of contending for one.
//
// Data movement: K and V blocks go from global memory straight into an LDS
// ring of NBUF blocks (global_load_lds_dwordx4: no register staging, no LDS
// store instructions), NBUF - 2 blocks in flight.  Barrier j follows each
// wave's wait for its own loads of block j; it publishes block j and frees the
// buffer of block j - 2, which then receives block j + NBUF - 2.  The byte
// offsets of each block's two page halves are staged in LDS once, so the loop
// issues no memory reads but its own loads; a half's base address is formed
// in SGPRs and a lane adds a fixed 32-bit offset.  The draft blocks (last
// split) are loaded and rotated into their own LDS blocks before the loop.
//
// LDS tiles are unpadded (256-byte rows), with the 16-byte chunks of each row
// permuted (chunk c of row r sits in slot c ^ swz(r)) so that the MFMA operand
// reads hit distinct banks: 16 rows read at one chunk (K) and 4 rows x 64
// bytes read by the transposed V load.
//
// Precision: the rotated, scaled query is carried as a bf16 pair hi + lo (two
// QK products), so the query's rounding leaves the scores; this matters on
// keys with outlier channels, where a single bf16 query moves the output by
// about as much as the whole error budget allows.  The row sums are taken from
// the same bf16 weights the PV product uses.
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
// the ring loads still in flight).  The wave's own LDS reads complete first, so
// that no read of a ring buffer is still in flight when the barrier lets its
// refill start; the clobber keeps LDS accesses on their side.
__device__ __forceinline__ void lds_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

typedef __attribute__((address_space(3))) void lds_void;
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

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

// NW waves per workgroup, each owning TPW 32-row query tiles (NW * TPW = 8: 256 rows); NBUF ring blocks.
// PHASE (8 waves): waves w and w + 4 share a SIMD; waves 0..3 run block j as QK, softmax, PV, while
// waves 4..7 run block j - 1's softmax and PV around block j's QK products, so that one wave of each
// SIMD is in its matrix phase while the other is in its vector phase.
template <int NW, int TPW, int NBUF, bool PHASE>
__global__ __launch_bounds__(NW * 64, 1) void attn_tall_kernel(AttnParams p) {
  static_assert((NW == 4 || NW == 8) && NW * TPW == 8, "4 or 8 waves, 256 rows");
  static_assert(NBUF >= 4, "ring depth");
  constexpr int kLPW = 8 / NW;                   // load instructions per wave, tile and block
  constexpr int kBlk = 2 * kTallTile;            // one block in LDS: K tile, then V tile
  constexpr int kRingBytes = NBUF * kBlk;
  constexpr int kDraftBytes = 2 * kBlk;          // draft keys 0..63
  __shared__ __attribute__((aligned(16))) unsigned char lds[kRingBytes + kDraftBytes + kTallMaxBlocks * 16];
  unsigned char* dlds = lds + kRingBytes;
  // byte offset (from the pool base) of row 0 / row 16 of each target block of the split
  int64_t* boff = (int64_t*)(lds + kRingBytes + kDraftBytes);

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
  const int ntot = nt + nd;                      // blocks: target blocks, then draft blocks
  const int P = position_base(p, b, T);

  // ---- base offsets of the split's target blocks (page clamped into the pool) ----
  const int ps = p.page_shift;
  const int pmask = (1 << ps) - 1;
  const int lp_last = T > 0 ? (T - 1) >> ps : 0;
  const int64_t pt_row = (int64_t)b * p.max_pages_per_seq;
  const int64_t pstr_b = p.page_stride * 2, hoff_b = (int64_t)h * p.head_stride * 2;
  const int64_t sstr_b = p.slot_stride * 2;
  for (int i = threadIdx.x; i < nt; i += NW * 64) {
    const int key0 = (blk0 + i) * kBlockKeys;
    const int la = min(key0 >> ps, lp_last), lb = min((key0 + 16) >> ps, lp_last);
    int pa = p.page_table[pt_row + la], pb = p.page_table[pt_row + lb];
    pa = pa < 0 ? 0 : (pa >= p.num_pages ? p.num_pages - 1 : pa);
    pb = pb < 0 ? 0 : (pb >= p.num_pages ? p.num_pages - 1 : pb);
    boff[2 * i] = (int64_t)pa * pstr_b + hoff_b + (int64_t)(key0 & pmask) * sstr_b;
    boff[2 * i + 1] = (int64_t)pb * pstr_b + hoff_b + (int64_t)((key0 + 16) & pmask) * sstr_b;
  }

  // ---- load slots: load instruction t (0..7) of a tile fills rows 4t .. 4t+3; lane L takes row
  // 4t + L / 16 and the chunk that belongs in slot L % 16.  Wave w issues instructions w kLPW .. ----
  uint32_t kvo[kLPW], vvo[kLPW];                // lane offsets from the half's base
  int lrow[kLPW], kchunk[kLPW], vchunk[kLPW];
#pragma unroll
  for (int i = 0; i < kLPW; ++i) {
    const int t = w * kLPW + i;
    lrow[i] = 4 * t + (lane >> 4);
    kchunk[i] = (lane & 15) ^ kswz(lrow[i]);
    vchunk[i] = (lane & 15) ^ vswz(lrow[i]);
    kvo[i] = (uint32_t)((lrow[i] & 15) * sstr_b) + (uint32_t)kchunk[i] * 16u;
    vvo[i] = (uint32_t)((lrow[i] & 15) * sstr_b) + (uint32_t)vchunk[i] * 16u;
  }
  const int upper = (w * kLPW) >= 4 ? 1 : 0;     // this wave's instructions lie in rows 16..31

  // ---- draft keys and values (last split) into their own LDS blocks; rows past S load row S - 1 ----
  const uint16_t* dkbase = (const uint16_t*)p.draft_k;
  const uint16_t* dvbase = (const uint16_t*)p.draft_v;
  for (int db = 0; db < nd; ++db) {
#pragma unroll
    for (int i = 0; i < kLPW; ++i) {
      const int t = w * kLPW + i;
      const int s = min(db * kBlockKeys + lrow[i], S - 1);
      const int64_t e = draft_offset(b, s, h, p.max_draft, p.hkv);
      lds_load_vaddr(dkbase + e + kchunk[i] * 8, dlds + db * kBlk + t * 1024);
      lds_load_vaddr(dvbase + e + vchunk[i] * 8, dlds + db * kBlk + kTallTile + t * 1024);
    }
  }

  // ---- query rows of this wave: tile i holds rows (8 rg + TPW w + i) * 32 + lane % 32, rotated,
  // scaled, split hi + lo ----
  uint64_t anc_mine = 0;
  int depth_mine = 0;
  if (p.tree) anc_mine = tree_ancestry_wave(p.parents + (int64_t)b * p.n_nodes, p.n_nodes, lane, &depth_mine);
  int r[TPW], jrow[TPW], hqr[TPW], draft_lim[TPW];
  bool row_ok[TPW];
  uint64_t row_anc[TPW];
  bf16x8 qhi[TPW][8], qlo[TPW][8];
#pragma unroll
  for (int i = 0; i < TPW; ++i) {
    r[i] = (rg * 8 + w * TPW + i) * 32 + l32;
    row_ok[i] = r[i] < p.rows;
    const int rr = row_ok[i] ? r[i] : p.rows - 1;
    jrow[i] = rr / p.group;
    hqr[i] = h * p.group + (rr - jrow[i] * p.group);
    row_anc[i] = 0;
    int qpos;
    if (p.tree) {
      const int node = query_node(p, b, jrow[i]);
      const uint32_t lo = __shfl((uint32_t)anc_mine, node), hi = __shfl((uint32_t)(anc_mine >> 32), node);
      row_anc[i] = ((uint64_t)hi << 32) | lo;
      qpos = P + __shfl(depth_mine, node);
    } else {
      qpos = P + s0 + jrow[i];
    }
    qpos = qpos >= p.max_position ? p.max_position - 1 : qpos;
    draft_lim[i] = p.tree ? S - 1 : min(s0 + jrow[i], S - 1);
    const uint16_t* qp = (const uint16_t*)p.q + (((int64_t)b * p.nq + jrow[i]) * p.hq + hqr[i]) * kHeadDim + hh * 8;
    u32x4 raw[8];
#pragma unroll
    for (int kc = 0; kc < 8; ++kc) raw[kc] = *(const u32x4*)(qp + kc * 16);
    rope_rotate_split(raw, p.rope + (int64_t)qpos * kHalfDim + hh * 8, row_ok[i] ? p.qscale : 0.0f, qhi[i], qlo[i]);
  }
  __syncthreads();                               // base offsets and draft rows landed; all loads above returned

  // ---- rotate the raw draft keys in place: this wave's rows (chunk c pairs with chunk c ^ 8) ----
  for (int db = 0; db < nd; ++db) {
#pragma unroll
    for (int i = 0; i < kLPW; ++i) {
      const int row = lrow[i];
      const int c = kchunk[i];
      const int s = min(db * kBlockKeys + row, S - 1);
      int kpos = p.tree ? P + __shfl(depth_mine, s & 63) : P + s;
      kpos = kpos >= p.max_position ? p.max_position - 1 : kpos;
      unsigned char* rowp = dlds + db * kBlk + row * 256;
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
  }
  if (nd > 0) {
    __builtin_amdgcn_s_waitcnt(0xc07f);          // lgkmcnt(0): this wave's rotated rows are written
    lds_barrier();
  }

  // ---- target ring loads ----
  const char* kbase = (const char*)p.k_pages;
  const char* vbase = (const char*)p.v_pages;
  // block it (clamped to the last target block; repeats keep vmcnt uniform) into ring buffer buf
  auto issue = [&](int it, int buf) {
    it = it < nt ? it : nt - 1;
    unsigned char* kt = lds + buf * kBlk;
    unsigned char* vt = kt + kTallTile;
    const int key0 = (blk0 + it) * kBlockKeys;
    if (key0 + kBlockKeys <= T) {
      const int64_t off = __builtin_amdgcn_readfirstlane((int)(boff[2 * it + upper] & 0xffffffff)) |
                          ((int64_t)__builtin_amdgcn_readfirstlane((int)(boff[2 * it + upper] >> 32)) << 32);
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
        const int half = (key - key0) >> 4;
        const int64_t e = boff[2 * it + half] + (int64_t)(key - key0 - 16 * half) * sstr_b;
        lds_load_vaddr(kbase + e + kchunk[i] * 16, kt + t * 1024);
        lds_load_vaddr(vbase + e + vchunk[i] * 16, vt + t * 1024);
      }
    }
  };
  // LDS block of block it, whose ring buffer (for a target block) is buf
  auto tile = [&](int it, int buf) -> const unsigned char* {
    return it < nt ? lds + buf * kBlk : dlds + (it - nt) * kBlk;
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

  auto read_k = [&](const unsigned char* kt, bf16x8 (&kop)[8]) {
#pragma unroll
    for (int kc = 0; kc < 8; ++kc)
      kop[kc] = as_bf16x8(*(const u32x4*)(kt + kr_base + 16 * ((2 * kc + hh) ^ ks)));
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
  // S^T = K (Qhi + Qlo)^T for every tile of the wave; each K operand feeds 2 TPW products
  auto qk = [&](const bf16x8 (&kop)[8], f32x16 (&sacc)[TPW]) {
#pragma unroll
    for (int i = 0; i < TPW; ++i) sacc[i] = f32x16{};
#pragma unroll
    for (int kc = 0; kc < 8; ++kc) {
#pragma unroll
      for (int i = 0; i < TPW; ++i) {
        sacc[i] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kop[kc], qhi[i][kc], sacc[i], 0, 0, 0);
        sacc[i] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kop[kc], qlo[i][kc], sacc[i], 0, 0, 0);
      }
    }
  };
  // Visibility bits of block it's keys for this lane's row: bit v covers the key of accumulator
  // register v, key0 + 16 (v / 8) + 8 hh + v % 8, so each byte covers 8 consecutive keys.
  // Keys at or below `lim` are visible (prefix tail, causal steps); a tree takes its row's
  // ancestor bits.  Arithmetic only, so that nothing here costs a per-key loop.
  auto run8 = [](int base, int lim) -> uint32_t {
    const int n = min(max(lim - base + 1, 0), 8);
    return (1u << n) - 1u;
  };
  auto block_valid = [&](int it, int i) -> uint32_t {
    if (it < nt) {
      const int b0 = (blk0 + it) * kBlockKeys + 8 * hh;
      return run8(b0, T - 1) | (run8(b0 + 16, T - 1) << 8);
    }
    const int b0 = (it - nt) * kBlockKeys + 8 * hh;
    if (p.tree) {
      return (uint32_t)((row_anc[i] >> b0) & 0xffu) | ((uint32_t)((row_anc[i] >> (b0 + 16)) & 0xffu) << 8);
    }
    return run8(b0, draft_lim[i]) | (run8(b0 + 16, draft_lim[i]) << 8);
  };
  // only the block holding position T - 1 and the draft blocks need a mask (uniform)
  auto block_masked = [&](int it) -> bool { return it >= nt || (blk0 + it + 1) * kBlockKeys > T; };

  f32x16 oacc[TPW][4];
  float m_run[TPW], l_run[TPW];
#pragma unroll
  for (int i = 0; i < TPW; ++i) {
#pragma unroll
    for (int dt = 0; dt < 4; ++dt) oacc[i][dt] = f32x16{};
    m_run[i] = -INFINITY;
    l_run[i] = 0.0f;
  }
  const uint32_t ones = 0x3f803f80u;             // (1, 1) in bf16

  // Softmax of block it's scores s (consumed), then O^T += V^T P^T.  The QK products of the next
  // block, when there is one (`kn`: its K operands), are issued between the softmax's VALU work.
  auto block_step = [&](f32x16 (&s)[TPW], int it, int buf, const bf16x8* kn, f32x16 (*s_next)[TPW]) {
    if (block_masked(it)) {
#pragma unroll
      for (int i = 0; i < TPW; ++i) apply_mask(s[i], block_valid(it, i));
    }
    float mu[TPW], alpha[TPW];
    bool jump_any = false;
#pragma unroll
    for (int i = 0; i < TPW; ++i) {
      float bm = -INFINITY;
#pragma unroll
      for (int v = 0; v < 16; ++v) bm = fmaxf(bm, s[i][v]);
      bm = fmaxf(bm, other_half(bm));
      const bool jump = bm > m_run[i] + kRescaleSlack;   // false while both are -inf
      const float mn = jump ? bm : m_run[i];
      mu[i] = mn == -INFINITY ? 0.0f : mn;
      alpha[i] = __builtin_amdgcn_exp2f(m_run[i] - mu[i]);
      m_run[i] = mn;
      jump_any = jump_any || jump;
    }
    if (kn) qk(*(const bf16x8(*)[8])kn, *s_next);
    uint32_t pk[TPW][8];                         // weights of registers 2e, 2e + 1 as a bf16 pair
#pragma unroll
    for (int i = 0; i < TPW; ++i) {
#pragma unroll
      for (int v = 0; v < 16; v += 2) {
        const float p0 = __builtin_amdgcn_exp2f(s[i][v] - mu[i]);
        const float p1 = __builtin_amdgcn_exp2f(s[i][v + 1] - mu[i]);
        pk[i][v >> 1] = pack_bf16x2(p0, p1);
      }
    }
    if (kn) {
      // one product, then three VALU operations of the softmax, 16 TPW times
#pragma unroll
      for (int g = 0; g < 16 * TPW; ++g) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x002, 3, 0);
      }
    }
#pragma unroll
    for (int i = 0; i < TPW; ++i) {
      // row sum from the bf16 weights the product uses (the same rounding as the numerator)
      float ps0 = 0.0f, ps1 = 0.0f;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        ps0 = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, pk[i][e]), __builtin_bit_cast(bf16x2, ones),
                                              ps0, false);
        ps1 = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, pk[i][e + 4]),
                                              __builtin_bit_cast(bf16x2, ones), ps1, false);
      }
      l_run[i] = l_run[i] * alpha[i] + (ps0 + ps1);
    }
    u32x4 pw[TPW][2];
#pragma unroll
    for (int i = 0; i < TPW; ++i) {
      pw[i][0] = u32x4{pk[i][0], pk[i][1], pk[i][2], pk[i][3]};
      pw[i][1] = u32x4{pk[i][4], pk[i][5], pk[i][6], pk[i][7]};
      // the weights are formed here, between the products above, not sunk past the rescale branch
      asm volatile("" ::"v"(pw[i][0]), "v"(pw[i][1]), "v"(l_run[i]));
    }
    if (__any(jump_any)) {
#pragma unroll
      for (int i = 0; i < TPW; ++i)
#pragma unroll
        for (int dt = 0; dt < 4; ++dt)
#pragma unroll
          for (int v = 0; v < 16; ++v) oacc[i][dt][v] *= alpha[i];
    }
    bf16x8 vop[4][2];
    read_v(tile(it, buf) + kTallTile, vop);
#pragma unroll
    for (int dt = 0; dt < 4; ++dt)
#pragma unroll
      for (int sidx = 0; sidx < 2; ++sidx)
#pragma unroll
        for (int i = 0; i < TPW; ++i)
          oacc[i][dt] =
              __builtin_amdgcn_mfma_f32_32x32x16_bf16(vop[dt][sidx], as_bf16x8(pw[i][sidx]), oacc[i][dt], 0, 0, 0);
    // every V^T read issued before the first product, so one LDS latency is exposed instead of four
    __builtin_amdgcn_sched_group_barrier(0x100, 16, 0);
    __builtin_amdgcn_sched_group_barrier(0x008, 8 * TPW, 0);
  };

  if (ntot > 0) {
    // Ring protocol (every wave issues its share of every block): barrier j (j >= 1) follows this
    // wave's wait for block j; then every wave is done with block j - 2 (the late waves read block
    // j - 1's V after barrier j), whose buffer receives block j + NBUF - 2.  NBUF - 2 blocks in flight.
    if (nt > 0) {
#pragma unroll
      for (int u = 0; u < NBUF - 1; ++u) issue(u, u);
    }
    wait_vmcnt<(NBUF - 2) * 2 * kLPW>();         // block 0 (if it is a target block) has landed
    lds_barrier();
    const bool late = PHASE && w >= NW / 2;      // one block behind in the softmax and PV
    f32x16 sa[TPW], sb[TPW];                     // late waves: scores of blocks j - 1 and j, in turn
    int ibuf = NBUF - 1;                         // ring buffer of the next issue
    int cbuf = 0;                            // ring buffer of block j
    auto next_buf = [](int x) { return x == NBUF - 1 ? 0 : x + 1; };
    auto barrier_j = [&](int j) {
      wait_vmcnt<(NBUF - 3) * 2 * kLPW>();
      lds_barrier();
      if (nt > 0) issue(j + NBUF - 2, ibuf);
      ibuf = next_buf(ibuf);
    };
    if (late) {
      {
        bf16x8 kop[8];
        read_k(tile(0, 0), kop);
        qk(kop, sa);
      }
      // step j: block j - 1's softmax and PV, block j's QK in between
      auto step = [&](int j, f32x16 (&s_prev)[TPW], f32x16 (&s_cur)[TPW]) {
        barrier_j(j);
        const int pbuf = cbuf;
        cbuf = next_buf(cbuf);
        bf16x8 kn[8];
        read_k(tile(j, cbuf), kn);
        block_step(s_prev, j - 1, pbuf, &kn[0], &s_cur);
      };
      int j = 1;
      for (; j + 1 < ntot; j += 2) {
        step(j, sa, sb);
        step(j + 1, sb, sa);
      }
      if (j < ntot) {
        step(j, sa, sb);
        block_step(sb, ntot - 1, cbuf, nullptr, nullptr);
      } else {
        block_step(sa, ntot - 1, cbuf, nullptr, nullptr);
      }
    } else {
      for (int j = 0; j < ntot; ++j) {
        if (j > 0) barrier_j(j);
        bf16x8 kop[8];
        read_k(tile(j, cbuf), kop);
        qk(kop, sa);
        block_step(sa, j, cbuf, nullptr, nullptr);
        cbuf = next_buf(cbuf);
      }
    }
    wait_vmcnt<0>();                             // the repeat loads past the end drain before exit
  }

  // ---- write: final output (one split) or split partial ----
#pragma unroll
  for (int i = 0; i < TPW; ++i) {
    if (!row_ok[i]) continue;
    const float l_row = l_run[i] + __shfl_xor(l_run[i], 32);
    const float M = m_run[i];
    if (p.splits == 1) {
      const float inv = 1.0f / l_row;
      const int64_t orow = (((int64_t)b * p.nq + jrow[i]) * p.hq + hqr[i]) * kHeadDim;
#pragma unroll
      for (int dt = 0; dt < 4; ++dt) {
#pragma unroll
        for (int q4 = 0; q4 < 4; ++q4) {
          const int d = dt * 32 + q4 * 8 + hh * 4;
          const float o0 = oacc[i][dt][q4 * 4 + 0] * inv, o1 = oacc[i][dt][q4 * 4 + 1] * inv;
          const float o2 = oacc[i][dt][q4 * 4 + 2] * inv, o3 = oacc[i][dt][q4 * 4 + 3] * inv;
          if (p.out_fp32) {
            *(f32x4*)((float*)p.out + orow + d) = f32x4{o0, o1, o2, o3};
          } else {
            *(u32x2*)((uint16_t*)p.out + orow + d) = u32x2{pack_bf16x2(o0, o1), pack_bf16x2(o2, o3)};
          }
        }
      }
      if (p.lse && hh == 0) p.lse[((int64_t)b * p.nq + jrow[i]) * p.hq + hqr[i]] = (M + __log2f(l_row)) * kLn2;
    } else {
      const int64_t prow = (((int64_t)b * p.hkv + h) * p.rows_pad + r[i]) * p.splits + split;
      float* po = p.part_o + prow * kHeadDim;
#pragma unroll
      for (int dt = 0; dt < 4; ++dt)
#pragma unroll
        for (int q4 = 0; q4 < 4; ++q4) {
          const int d = dt * 32 + q4 * 8 + hh * 4;
          *(f32x4*)(po + d) = f32x4{oacc[i][dt][q4 * 4 + 0], oacc[i][dt][q4 * 4 + 1], oacc[i][dt][q4 * 4 + 2],
                                    oacc[i][dt][q4 * 4 + 3]};
        }
      if (hh == 0) p.part_ml[prow] = make_float2(M, l_row);
    }
  }
}

}  // namespace

#ifndef KVSHOT_TALL_WAVES
#define KVSHOT_TALL_WAVES 8
#endif
constexpr int kTallTilesPerWave = 8 / KVSHOT_TALL_WAVES;
#ifndef KVSHOT_TALL_PHASE
#define KVSHOT_TALL_PHASE 1
#endif
#ifndef KVSHOT_TALL_NBUF
#define KVSHOT_TALL_NBUF 6
#endif

// 32-row tiles of one workgroup (256 rows)
int tall_waves_per_wg() { return KVSHOT_TALL_WAVES; }
int tall_max_blocks() { return kTallMaxBlocks; }

hipError_t launch_attn_tall(const AttnParams& p, hipStream_t s) {
  const dim3 grid((unsigned)((int64_t)p.splits * p.row_groups * p.hkv * p.batch));
  hipLaunchKernelGGL((attn_tall_kernel<KVSHOT_TALL_WAVES, kTallTilesPerWave, KVSHOT_TALL_NBUF, KVSHOT_TALL_PHASE != 0>), grid,
                     dim3(KVSHOT_TALL_WAVES * 64), 0, s, p);
  return hipGetLastError();
}

}  // namespace kvshot
