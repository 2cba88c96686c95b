// Split-K flash-decode draft attention on bf16 MFMA (gfx950).
//
// One workgroup serves one (split, KV head, sequence).  Its query tile is every
// query head of the KV head's group times every draft query of the sequence
// (rows = G * n), so each target K/V block is read from HBM once for all of
// them (grouped-query folding).  The memory attended is the target prefix of
// the sequence followed by its draft keys (Sec. 3.4.1, Eq. 7; App. B).
//
// Data movement per 32-key block: K and V rows are read from HBM with fully
// coalesced 16-byte non-temporal loads (each load instruction covers four
// whole 256-byte rows) into registers, then written row-major into LDS.
// MFMA operands come back out of LDS: K rows with ds_read_b128, and V
// transposed with ds_read_b64_tr_b16 (each 16-lane group turns a 4-key x
// 16-channel tile into 4 keys per channel lane).
//
// Math per block and wave: S^T = K * Q^T (v_mfma_f32_32x32x16_bf16), so each
// lane owns one query row (lane % 32) and 16 of the block's keys; the online
// softmax row max needs one cross-half exchange and the output rescale is
// lane-local.  O^T += V^T * P^T on the same MFMA, with P taken straight from
// the S^T accumulator (the K rows are permuted so that the accumulator layout
// is the B-operand layout of the second product).
//
// Row tiles: rows are padded to 32 * RT.  A workgroup has NW waves, each
// owning TPW row tiles; RW = RT / TPW waves cover the rows of one key stream.
// Wave w owns tiles (w % RW) * TPW .. + TPW - 1 of key stream w / RW.  The RW
// waves of a key stream share its LDS tiles (each loads 8 / RW of the block's
// load instructions); the KS = NW / RW key streams interleave blocks and
// merge through LDS at the end.  With TPW > 1 every K and V^T operand read
// from LDS feeds TPW MFMAs.
#include "attn_mfma_common.h"

// 1: a block's V^T operand reads are issued before its softmax
#ifndef KVSHOT_VREAD_EARLY
#define KVSHOT_VREAD_EARLY 1
#endif
// 1: the eight K operand reads of a block are all issued before its first MFMA
#ifndef KVSHOT_KREAD_FIRST
#define KVSHOT_KREAD_FIRST 1
#endif

namespace kvshot {
namespace {

using namespace mfma;


// LDS row pitches (bf16 elements).  K rows are read 16 rows x 16 bytes at a
// time (pitch = 68 dwords spreads them over distinct banks); V rows are read by
// the transpose load 4 rows x 32 bytes per 16 lanes (pitch = 80 dwords).
constexpr int kKPitch = 136;
constexpr int kVPitch = 160;
constexpr int kKTileBytes = kBlockKeys * kKPitch * 2;    // 8704
constexpr int kVTileBytes = kBlockKeys * kVPitch * 2;    // 10240
constexpr int kStreamBytes = kKTileBytes + kVTileBytes;
template <int RW>
__device__ __forceinline__ void tile_sync() {
  if constexpr (RW > 1) {
    __syncthreads();
  } else {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  }
}

// RT: 32-row query tiles per workgroup; TPW: of which each wave owns (one K/V
// operand read from LDS then feeds TPW MFMAs, and the tiles give a wave
// independent MFMA and softmax chains); NW: waves per workgroup; PF: blocks
// of K/V in flight per wave (register staging ring); QSPLIT: query kept as a
// bf16 hi/lo pair (two QK^T products); WPS: waves per SIMD the register
// budget allows.
template <int RT, int TPW, int NW, int PF, bool QSPLIT, int WPS>
__global__ __launch_bounds__(NW * 64, WPS) void attn_mfma_kernel(AttnParams p) {
  constexpr int RW = RT / TPW;             // waves sharing one key stream's tiles
  constexpr int KS = NW / RW;              // key streams per workgroup
  constexpr int kLoadsPerWave = 8 / RW;    // 16-byte load instructions per K (and per V) tile and wave
  static_assert(RW * TPW == RT && KS * RW == NW && kLoadsPerWave * RW == 8, "tile/wave configuration");
  constexpr int kMergeBytes = (KS - 1) * RT * 64 * (64 * 4 + 8);
  constexpr int kBufs = RW > 1 ? 2 : 1;    // waves that share tiles double-buffer them
  constexpr int kTileBytes = KS * kBufs * kStreamBytes;
  constexpr int kLdsBytes = kTileBytes > kMergeBytes ? kTileBytes : kMergeBytes;
  __shared__ __attribute__((aligned(16))) unsigned char lds[kLdsBytes];

  const int lane = threadIdx.x & 63;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);   // wave index, kept in an SGPR
  const int rt = w % RW;
  const int ks = w / RW;
  const int l32 = lane & 31;
  const int hh = lane >> 5;
  int wi = xcd_remap(blockIdx.x, gridDim.x);
  const int rg = wi % p.row_groups;
  wi /= p.row_groups;
  int h, item = 0;
  if (!p.balanced) {
    wi /= p.splits;                                // (split, KV head, sequence); the split is decoded below
    h = wi % p.hkv;
  } else {
    item = wi % p.items;                           // (item, KV head)
    h = (wi / p.items) % p.hkv;
  }

  // One split: query rows of sequence b (prefix length T) against its target blocks [blk0, blk1),
  // plus its draft keys when `last`; written as part `part` of `nparts`, or as the output when
  // nparts == 1.
  auto segment = [&](const int b, const int T, const int part, const int nparts, const int blk0, const int blk1,
                     const bool last) {
  const int nt = blk1 > blk0 ? blk1 - blk0 : 0;

  int s0 = 0, S = p.tree ? p.n_nodes : p.nq;
  if (!p.tree) {
    s0 = p.step_offsets[b];
    s0 = s0 < 0 ? 0 : (s0 > p.max_draft - p.nq ? p.max_draft - p.nq : s0);
    S = s0 + p.nq;
  }
  const int nd = last ? (S + kBlockKeys - 1) / kBlockKeys : 0;
  const int P = position_base(p, b, T);            // position of draft step 0 / tree depth 0

  uint16_t* ktile = (uint16_t*)(lds + ks * kBufs * kStreamBytes);
  uint16_t* vtile = (uint16_t*)(lds + ks * kBufs * kStreamBytes + kKTileBytes);

  // K-operand row rho = l32 reads tile row kperm(rho), chosen so that
  // accumulator register v of lane (row, hh) holds key 16 * (v / 8) + 8 * hh + v % 8.
  const int kperm = ((l32 >> 4) << 4) + (((l32 >> 2) & 1) << 3) + (((l32 >> 3) & 1) << 2) + (l32 & 3);
  const int k_rd = kperm * kKPitch + hh * 8;
  // transpose-read base: 16-lane group gr reads keys 8*(gr/2) + (lane%16)/4 of
  // channels 16*(gr%2) + 4*(lane%4) .. +3; lane i of the group receives channel
  // 16*(gr%2) + i of four consecutive keys
  const int gr = lane >> 4, sg = lane & 15;
  const int vt_off = ((gr >> 1) * 8 + (sg >> 2)) * kVPitch + (gr & 1) * 16 + 4 * (sg & 3);
  // coalesced load / LDS write slot of this lane in load instruction t: row 4t + lane/16, 16-byte chunk lane%16
  const int ld_row = lane >> 4, ld_chunk = lane & 15;

  const int64_t pstr = p.page_stride, hstr = p.head_stride, sstr = p.slot_stride;
  const uint16_t* kbase = (const uint16_t*)p.k_pages;
  const uint16_t* vbase = (const uint16_t*)p.v_pages;
  const uint16_t* dkbase = (const uint16_t*)p.draft_k;
  const uint16_t* dvbase = (const uint16_t*)p.draft_v;
  const int pmask = (1 << p.page_shift) - 1;
  const int lp_last = T > 0 ? (T - 1) >> p.page_shift : 0;
  const int64_t pt_row = (int64_t)b * p.max_pages_per_seq;

  // Page ids of target block tb, read with a vector load (lane 0: the page of
  // rows 0..15, lane 1: the page of rows 16..31).  Loading them a ring cycle
  // ahead on the vector memory queue keeps the page-table latency off the
  // block loop: a scalar load would share its wait counter with LDS reads.
  auto load_ids = [&](int tb) -> int {
    const int key0 = (blk0 + tb) * kBlockKeys;
    int la = key0 >> p.page_shift, lb = (key0 + 16) >> p.page_shift;
    la = la > lp_last ? lp_last : la;
    lb = lb > lp_last ? lp_last : lb;
    return p.page_table[pt_row + ((lane & 1) ? lb : la)];
  };
  // Issue this wave's share of the loads of target block tb into kd / vd.
  // Rows 0..15 and 16..31 of a block each lie in one page (P >= 16); their
  // base addresses are wave-uniform, and a lane adds a small 32-bit offset.
  const uint32_t sstr_b = (uint32_t)(sstr * 2);
  const int64_t hoff = (int64_t)h * hstr;
  auto issue_target = [&](int tb, int ids, u32x4 (&kd)[kLoadsPerWave], u32x4 (&vd)[kLoadsPerWave]) {
    const int key0 = (blk0 + tb) * kBlockKeys;
    int pa = __builtin_amdgcn_readlane(ids, 0);
    int pb = __builtin_amdgcn_readlane(ids, 1);
    pa = pa < 0 ? 0 : (pa >= p.num_pages ? p.num_pages - 1 : pa);
    pb = pb < 0 ? 0 : (pb >= p.num_pages ? p.num_pages - 1 : pb);
    const int64_t ea = (int64_t)pa * pstr + hoff + (int64_t)(key0 & pmask) * sstr;
    const int64_t eb = (int64_t)pb * pstr + hoff + (int64_t)((key0 + 16) & pmask) * sstr;
    const char* ka = (const char*)(kbase + ea);
    const char* kb = (const char*)(kbase + eb);
    const char* va = (const char*)(vbase + ea);
    const char* vb2 = (const char*)(vbase + eb);
#pragma unroll
    for (int i = 0; i < kLoadsPerWave; ++i) {
      const int t = rt + RW * i;                  // load instruction index: rows 4t .. 4t+3
      const uint32_t off = (uint32_t)(4 * (t & 3) + ld_row) * sstr_b + (uint32_t)ld_chunk * 16u;
      // the prefix K/V is read exactly once: whole lines, non-temporal
      kd[i] = __builtin_nontemporal_load((const u32x4*)((t >= 4 ? kb : ka) + off));
      vd[i] = __builtin_nontemporal_load((const u32x4*)((t >= 4 ? vb2 : va) + off));
    }
  };
  // Start the K/V stream before the query setup so the two dependent load
  // chains of the prologue overlap.
  // Every refill of a ring slot is issued, past the last block as a repeat
  // read of block nt - 1, so that the number of loads behind each slot is the
  // same on every path: the compiler then waits for just that slot's loads
  // instead of draining all of them.
  const int last_blk = nt - 1;
  u32x4 kst[PF][kLoadsPerWave], vst[PF][kLoadsPerWave];
  int idr[PF];                                     // page ids of the block each slot loads next
  if (nt > 0) {
#pragma unroll
    for (int u = 0; u < PF; ++u) idr[u] = load_ids(min(ks + KS * u, last_blk));
#pragma unroll
    for (int u = 0; u < PF; ++u) {
      issue_target(min(ks + KS * u, last_blk), idr[u], kst[u], vst[u]);
      idr[u] = load_ids(min(ks + KS * (u + PF), last_blk));
    }
  }
  // load block tb (clamped by the caller) into a slot, then the page ids of the
  // block that slot loads next
  auto refill = [&](int tb, u32x4 (&kd)[kLoadsPerWave], u32x4 (&vd)[kLoadsPerWave], int& ids) {
    issue_target(tb, ids, kd, vd);
    ids = load_ids(min(tb + KS * PF, last_blk));
  };

  // ---- query rows of this lane: tile rt * TPW + i holds rows (rg * RT + rt * TPW + i) * 32 + lane % 32 ----
  uint64_t anc_mine = 0;
  int depth_mine = 0;
  if (p.tree) anc_mine = tree_ancestry_wave(p.parents + (int64_t)b * p.n_nodes, p.n_nodes, lane, &depth_mine);
  int r[TPW], jrow[TPW], hqr[TPW];
  bool row_ok[TPW];
  uint64_t row_anc[TPW];
  bf16x8 qop[TPW][8];
  bf16x8 qlo[QSPLIT ? TPW : 1][QSPLIT ? 8 : 1];
#pragma unroll
  for (int i = 0; i < TPW; ++i) {
    r[i] = (rg * RT + rt * TPW + i) * 32 + l32;
    row_ok[i] = r[i] < p.rows;
    const int rr = row_ok[i] ? r[i] : p.rows - 1;
    jrow[i] = rr / p.group;
    hqr[i] = h * p.group + (rr - jrow[i] * p.group);
    int qpos;
    row_anc[i] = 0;
    if (p.tree) {
      const int node = query_node(p, b, jrow[i]);
      const uint32_t lo = __shfl((uint32_t)anc_mine, node), hi = __shfl((uint32_t)(anc_mine >> 32), node);
      row_anc[i] = ((uint64_t)hi << 32) | lo;
      qpos = P + __shfl(depth_mine, node);
    } else {
      qpos = P + s0 + jrow[i];
    }
    qpos = qpos >= p.max_position ? p.max_position - 1 : qpos;
    // query operand: rotated, scaled into log2 units, bf16 (hi/lo pair when split)
    const uint16_t* qp = (const uint16_t*)p.q + (((int64_t)b * p.nq + jrow[i]) * p.hq + hqr[i]) * kHeadDim + hh * 8;
    u32x4 raw[8];
#pragma unroll
    for (int kc = 0; kc < 8; ++kc) raw[kc] = *(const u32x4*)(qp + kc * 16);
    const float2* cs = p.rope + (int64_t)qpos * kHalfDim + hh * 8;
    if constexpr (QSPLIT) rope_rotate_split(raw, cs, row_ok[i] ? p.qscale : 0.0f, qop[i], qlo[i]);
    else rope_rotate_to_bf16(raw, cs, row_ok[i] ? p.qscale : 0.0f, qop[i]);
  }
  // S^T = K Q^T for every tile of the wave; each K operand chunk is read once
  auto qk = [&](const bf16x8 (&kop)[8], f32x16 (&acc)[TPW]) {
#pragma unroll
    for (int i = 0; i < TPW; ++i) acc[i] = f32x16{};
#pragma unroll
    for (int kc = 0; kc < 8; ++kc) {
#pragma unroll
      for (int i = 0; i < TPW; ++i) {
        acc[i] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kop[kc], qop[i][kc], acc[i], 0, 0, 0);
        if constexpr (QSPLIT) acc[i] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kop[kc], qlo[i][kc], acc[i], 0, 0, 0);
      }
    }
  };

  f32x16 oacc[TPW][4];
  SoftmaxState st[TPW];
#pragma unroll
  for (int i = 0; i < TPW; ++i) {
#pragma unroll
    for (int dt = 0; dt < 4; ++dt) oacc[i][dt] = f32x16{};
    st[i] = SoftmaxState{-INFINITY, 0.0f};
  }

  // Softmax update of every tile: weights P as bf16 B operands in pw, output
  // accumulators rescaled when a row's reference max moved.  Bit v of
  // valid[i]: key of accumulator register v is visible to tile i's row (only
  // when `masked`).
  auto softmax_tiles = [&](f32x16 (&sacc)[TPW], bool masked, const uint32_t (&valid)[TPW], u32x4 (&pw)[TPW][2]) {
    float alpha[TPW];
    bool rescale[TPW];
#pragma unroll
    for (int i = 0; i < TPW; ++i) {
      if (masked) apply_mask(sacc[i], valid[i]);
      softmax_front(sacc[i], st[i], pw[i], alpha[i], rescale[i]);
    }
#pragma unroll
    for (int i = 0; i < TPW; ++i) {
      if (rescale[i]) {
#pragma unroll
        for (int dt = 0; dt < 4; ++dt)
#pragma unroll
          for (int v = 0; v < 16; ++v) oacc[i][dt][v] *= alpha[i];
      }
    }
  };
  // O^T += V^T P^T with each V^T operand read once for all tiles
  auto pv_tiles = [&](const u32x4 (&pw)[TPW][2], const uint16_t* vt) {
    typedef __attribute__((address_space(3))) s16x4 lds_s16x4;
    const __attribute__((address_space(3))) uint16_t* vb =
        (const __attribute__((address_space(3))) uint16_t*)(vt) + vt_off;
#pragma unroll
    for (int dt = 0; dt < 4; ++dt) {
#pragma unroll
      for (int sidx = 0; sidx < 2; ++sidx) {
        // keys 16*sidx + 8*hh + 0..3 and + 4..7 of channel dt*32 + lane%32
        const s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
            (lds_s16x4*)(vb + (16 * sidx) * kVPitch + dt * 32));
        const s16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
            (lds_s16x4*)(vb + (16 * sidx + 4) * kVPitch + dt * 32));
        const u32x2 lo2 = __builtin_bit_cast(u32x2, lo), hi2 = __builtin_bit_cast(u32x2, hi);
        const bf16x8 a = as_bf16x8(u32x4{lo2[0], lo2[1], hi2[0], hi2[1]});
#pragma unroll
        for (int i = 0; i < TPW; ++i)
          oacc[i][dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, as_bf16x8(pw[i][sidx]), oacc[i][dt], 0, 0, 0);
      }
    }
  };
  // V^T operands of a block: 4 channel tiles x 2 key halves, each two transposed reads
  auto read_v = [&](const uint16_t* vt, bf16x8 (&vop)[4][2]) {
    typedef __attribute__((address_space(3))) s16x4 lds_s16x4;
    const __attribute__((address_space(3))) uint16_t* vb =
        (const __attribute__((address_space(3))) uint16_t*)(vt) + vt_off;
#pragma unroll
    for (int dt = 0; dt < 4; ++dt) {
#pragma unroll
      for (int sidx = 0; sidx < 2; ++sidx) {
        const s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
            (lds_s16x4*)(vb + (16 * sidx) * kVPitch + dt * 32));
        const s16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
            (lds_s16x4*)(vb + (16 * sidx + 4) * kVPitch + dt * 32));
        const u32x2 lo2 = __builtin_bit_cast(u32x2, lo), hi2 = __builtin_bit_cast(u32x2, hi);
        vop[dt][sidx] = as_bf16x8(u32x4{lo2[0], lo2[1], hi2[0], hi2[1]});
      }
    }
  };
  auto pv_regs = [&](const u32x4 (&pw)[TPW][2], const bf16x8 (&vop)[4][2]) {
#pragma unroll
    for (int dt = 0; dt < 4; ++dt)
#pragma unroll
      for (int sidx = 0; sidx < 2; ++sidx)
#pragma unroll
        for (int i = 0; i < TPW; ++i)
          oacc[i][dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vop[dt][sidx], as_bf16x8(pw[i][sidx]), oacc[i][dt], 0,
                                                                0, 0);
  };
  auto softmax_pv_tiles = [&](f32x16 (&sacc)[TPW], const uint16_t* vt, bool masked, const uint32_t (&valid)[TPW]) {
    u32x4 pw[TPW][2];
#if KVSHOT_VREAD_EARLY
    // the block's V^T operands are read before the softmax (in the same basic block as the
    // products before it), so their LDS latency overlaps the softmax instead of following it
    bf16x8 vop[4][2];
    read_v(vt, vop);
    softmax_tiles(sacc, masked, valid, pw);
    pv_regs(pw, vop);
#else
    softmax_tiles(sacc, masked, valid, pw);
    pv_tiles(pw, vt);
#endif
  };

  // Stage this wave's share of a block into the LDS tiles; rows at or past
  // `kend` get zero V so masked weights never meet NaN.
  auto stage = [&](int key0, int kend, u32x4 (&kd)[kLoadsPerWave], u32x4 (&vd)[kLoadsPerWave], int buf) {
    if (key0 + kBlockKeys > kend) {
#pragma unroll
      for (int i = 0; i < kLoadsPerWave; ++i)
        if (key0 + 4 * (rt + RW * i) + ld_row >= kend) vd[i] = u32x4{0u, 0u, 0u, 0u};
    }
    uint16_t* kt = ktile + buf * (kStreamBytes / 2);
    uint16_t* vt = vtile + buf * (kStreamBytes / 2);
#pragma unroll
    for (int i = 0; i < kLoadsPerWave; ++i) {
      const int kr = 4 * (rt + RW * i) + ld_row;
      *(u32x4*)(kt + kr * kKPitch + ld_chunk * 8) = kd[i];
      *(u32x4*)(vt + kr * kVPitch + ld_chunk * 8) = vd[i];
    }
  };
  // S^T of a staged target block
  auto qk_target = [&](int buf, f32x16 (&sacc)[TPW]) {
    const uint16_t* kt = ktile + buf * (kStreamBytes / 2);
    bf16x8 kop[8];
#pragma unroll
    for (int kc = 0; kc < 8; ++kc) kop[kc] = as_bf16x8(*(const u32x4*)(kt + k_rd + kc * 16));
    qk(kop, sacc);
#if KVSHOT_KREAD_FIRST
    // all eight operand reads in flight before the first product
    __builtin_amdgcn_sched_group_barrier(0x100, 8, 0);
    __builtin_amdgcn_sched_group_barrier(0x008, 8 * TPW * (QSPLIT ? 2 : 1), 0);
#endif
  };
  // Visibility of a target block's keys: only the block holding position T - 1 is masked
  auto target_valid = [&](int key0, uint32_t (&valid)[TPW]) {
    const bool masked = key0 + kBlockKeys > T;
    uint32_t vbits = 0xffffu;
    if (masked) {
      vbits = 0;
#pragma unroll
      for (int v = 0; v < 16; ++v) vbits |= (uint32_t)(key0 + 16 * (v >> 3) + 8 * hh + (v & 7) < T) << v;
    }
#pragma unroll
    for (int i = 0; i < TPW; ++i) valid[i] = vbits;    // the prefix is visible to every row alike
    return masked;
  };
  // QK^T, masking and the softmax / PV update of a staged target block
  auto compute_target = [&](int key0, int buf) {
    f32x16 sacc[TPW];
    qk_target(buf, sacc);
    uint32_t valid[TPW];
    const bool masked = target_valid(key0, valid);
    softmax_pv_tiles(sacc, vtile + buf * (kStreamBytes / 2), masked, valid);
  };

  // ---- target blocks: tb = ks + KS * it, software-pipelined PF blocks ahead ----
  // (the first PF blocks were issued before the query setup; a wave's share of
  // a block is 8 / RW load instructions, so waves that share their tiles with
  // others keep more blocks in flight)
  {
    const int iters = (nt + KS - 1) / KS;          // same for every wave of the workgroup
    if constexpr (RW == 1) {
      // private tiles: stage block it from ring slot it % PF, refill the slot
      // with block it + PF, compute (wave-local ordering only)
      for (int it0 = 0; it0 < iters; it0 += PF) {
#pragma unroll
        for (int u = 0; u < PF; ++u) {
          const int tb = ks + KS * (it0 + u);
          const bool active = tb < nt;
          const int key0 = (blk0 + tb) * kBlockKeys;
          if (active) stage(key0, T, kst[u], vst[u], 0);
          tile_sync<RW>();
          refill(min(tb + KS * PF, last_blk), kst[u], vst[u], idr[u]);
          if (active) compute_target(key0, 0);
          tile_sync<RW>();
        }
      }
    } else {
      // shared, double-buffered tiles: one barrier per block.  Block it is
      // computed from buffer it % 2 while block it + 1 is staged into the
      // other one (last read before the previous barrier).
      if (iters > 0) {
        if (ks < nt) stage((blk0 + ks) * kBlockKeys, T, kst[0], vst[0], 0);
        refill(min(ks + KS * PF, last_blk), kst[0], vst[0], idr[0]);
        __syncthreads();
      }
      for (int it0 = 0; it0 < iters; it0 += PF) {
#pragma unroll
        for (int u = 0; u < PF; ++u) {
          const int it = it0 + u;                  // iterations past the last block only keep the pattern
          const int tb = ks + KS * it;
          if (tb < nt) compute_target((blk0 + tb) * kBlockKeys, it & 1);
          const int nb = tb + KS;                  // next block: its loads sit in ring slot (u + 1) % PF
          if (nb < nt) stage((blk0 + nb) * kBlockKeys, T, kst[(u + 1) % PF], vst[(u + 1) % PF], (it + 1) & 1);
          refill(min(nb + KS * PF, last_blk), kst[(u + 1) % PF], vst[(u + 1) % PF], idr[(u + 1) % PF]);
          __syncthreads();
        }
      }
    }
  }

  // ---- draft blocks (last split only): keys 0..S-1, rotated at their own positions ----
  {
    const int iters = (nd + KS - 1) / KS;
    for (int it = 0; it < iters; ++it) {
      const int db = ks + KS * it;
      const bool active = db < nd;
      const int key0 = db * kBlockKeys;
      if (active) {
        u32x4 kd[kLoadsPerWave], vd[kLoadsPerWave];
#pragma unroll
        for (int i = 0; i < kLoadsPerWave; ++i) {
          int s = key0 + 4 * (rt + RW * i) + ld_row;
          s = s < S ? s : S - 1;
          const int64_t off = draft_offset(b, s, h, p.max_draft, p.hkv) + ld_chunk * 8;
          kd[i] = *(const u32x4*)(dkbase + off);
          vd[i] = *(const u32x4*)(dvbase + off);
        }
        stage(key0, S, kd, vd, 0);
      }
      tile_sync<RW>();
      if (active) {
        u32x4 kraw[8];
#pragma unroll
        for (int kc = 0; kc < 8; ++kc) kraw[kc] = *(const u32x4*)(ktile + k_rd + kc * 16);
        const int sk = min(key0 + kperm, S - 1);
        int kpos = p.tree ? P + __shfl(depth_mine, sk & 63) : P + sk;
        kpos = kpos >= p.max_position ? p.max_position - 1 : kpos;
        bf16x8 kop[8];
        rope_rotate_to_bf16(kraw, p.rope + (int64_t)kpos * kHalfDim + hh * 8, 1.0f, kop);
        uint32_t valid[TPW];
#pragma unroll
        for (int i = 0; i < TPW; ++i) {
          valid[i] = 0;
#pragma unroll
          for (int v = 0; v < 16; ++v) {
            const int s = key0 + 16 * (v >> 3) + 8 * hh + (v & 7);
            bool ok = s < S;
            if (p.tree) ok = ok && ((row_anc[i] >> (s & 63)) & 1ull);
            else ok = ok && (s <= s0 + jrow[i]);
            valid[i] |= (uint32_t)ok << v;
          }
        }
        f32x16 sacc[TPW];
        qk(kop, sacc);
        softmax_pv_tiles(sacc, vtile, true, valid);
      }
      tile_sync<RW>();
    }
  }

  // ---- merge the key streams of each row tile ----
  float l_row[TPW], M[TPW];
#pragma unroll
  for (int i = 0; i < TPW; ++i) {
    l_row[i] = st[i].l + __shfl_xor(st[i].l, 32);
    M[i] = st[i].m;
  }
  if constexpr (KS > 1) {
    static_assert(TPW == 1, "key streams are merged for one tile per wave");
    __syncthreads();
    float* mo = (float*)lds;
    float2* mml = (float2*)(lds + (KS - 1) * RT * 64 * 64 * 4);
    if (ks > 0) {
      const int slot = (ks - 1) * RT + rt;
#pragma unroll
      for (int dt = 0; dt < 4; ++dt)
#pragma unroll
        for (int v = 0; v < 16; ++v) mo[(slot * 64 + dt * 16 + v) * 64 + lane] = oacc[0][dt][v];
      mml[slot * 64 + lane] = make_float2(st[0].m, l_row[0]);
    }
    __syncthreads();
    if (ks == 0) {
      float mk[KS - 1], lk[KS - 1];
#pragma unroll
      for (int k = 0; k < KS - 1; ++k) {
        const float2 t = mml[(k * RT + rt) * 64 + lane];
        mk[k] = t.x;
        lk[k] = t.y;
        M[0] = fmaxf(M[0], t.x);
      }
      const float Mu = M[0] == -INFINITY ? 0.0f : M[0];
      const float f0 = __builtin_amdgcn_exp2f(st[0].m - Mu);
      l_row[0] *= f0;
#pragma unroll
      for (int dt = 0; dt < 4; ++dt)
#pragma unroll
        for (int v = 0; v < 16; ++v) oacc[0][dt][v] *= f0;
#pragma unroll
      for (int k = 0; k < KS - 1; ++k) {
        const float fk = __builtin_amdgcn_exp2f(mk[k] - Mu);
        l_row[0] += lk[k] * fk;
        const int slot = k * RT + rt;
#pragma unroll
        for (int dt = 0; dt < 4; ++dt)
#pragma unroll
          for (int v = 0; v < 16; ++v) oacc[0][dt][v] += mo[(slot * 64 + dt * 16 + v) * 64 + lane] * fk;
      }
    }
  }
  if (ks != 0) return;

  // ---- write: final output (one part) or partial ----
#pragma unroll
  for (int i = 0; i < TPW; ++i) {
    if (!row_ok[i]) continue;
    if (nparts == 1) {
      const float inv = 1.0f / l_row[i];
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
      if (p.lse && hh == 0)
        p.lse[((int64_t)b * p.nq + jrow[i]) * p.hq + hqr[i]] = (M[i] + __log2f(l_row[i])) * kLn2;
    } else {
      const int64_t prow = p.balanced ? ((int64_t)h * p.items + item) * p.rows_pad + r[i]
                                      : (((int64_t)b * p.hkv + h) * p.rows_pad + r[i]) * p.splits + part;
      float* po = p.part_o + prow * kHeadDim;
#pragma unroll
      for (int dt = 0; dt < 4; ++dt)
#pragma unroll
        for (int q4 = 0; q4 < 4; ++q4) {
          const int d = dt * 32 + q4 * 8 + hh * 4;
          *(f32x4*)(po + d) = f32x4{oacc[i][dt][q4 * 4 + 0], oacc[i][dt][q4 * 4 + 1], oacc[i][dt][q4 * 4 + 2],
                                    oacc[i][dt][q4 * 4 + 3]};
        }
      if (hh == 0) p.part_ml[prow] = make_float2(M[i], l_row[i]);
    }
  }
  };  // segment

  if (!p.balanced) {
    // every sequence split alike: work item (row group, split, KV head, sequence)
    int wj = xcd_remap(blockIdx.x, gridDim.x) / p.row_groups;
    const int split = wj % p.splits;
    const int b = wj / p.splits / p.hkv;
    int T = clamp_ctx(p.ctx_lens[b], p.max_pages_per_seq, p.page_shift);
    T = T > p.max_ctx ? p.max_ctx : T;
    const int nbt = (T + kBlockKeys - 1) / kBlockKeys;
    const int blk0 = split * p.blocks_per_split;
    segment(b, T, split, p.splits, blk0, min(blk0 + p.blocks_per_split, nbt), split == p.splits - 1);
    return;
  }
  // length-balanced: this item's sequence and split, from the lengths
  const BalancedSlot sl = balanced_schedule(p.ctx_lens, p.batch, p.max_ctx, p.max_pages_per_seq, p.page_shift,
                                            p.items, p.min_chunk, lane);
  const uint64_t own = __ballot(lane < p.batch && item >= sl.first && item < sl.first + sl.splits);
  if (own == 0) return;                            // past the last split of the batch (whole workgroup)
  const int b = __builtin_amdgcn_readfirstlane(__builtin_ctzll(own));
  const int nsplit = __builtin_amdgcn_readfirstlane(__shfl(sl.splits, b));
  const int first = __builtin_amdgcn_readfirstlane(__shfl(sl.first, b));
  const int split = item - first;
  const int per = __builtin_amdgcn_readfirstlane(__shfl(sl.per, b));
  const int T = __builtin_amdgcn_readfirstlane(__shfl(sl.ctx, b));
  // the combine reads each sequence's split count and first item (one writer per sequence)
  if (split == 0 && h == 0 && rg == 0 && threadIdx.x == 0) {
    p.seq_splits[b] = nsplit;
    p.seq_splits[64 + b] = first;
  }
  const int nbt = (T + kBlockKeys - 1) / kBlockKeys;
  segment(b, T, split, nsplit, split * per, min(split * per + per, nbt), split == nsplit - 1);
}

}  // namespace

// Per row-tile configuration (waves per SIMD, blocks in flight, query split).
#ifndef KVSHOT_RT1_WPS
#define KVSHOT_RT1_WPS 1
#endif
#ifndef KVSHOT_RT1_PF
#define KVSHOT_RT1_PF 1
#endif
// one-wave workgroups of the balanced schedule: blocks in flight per wave
#ifndef KVSHOT_BAL_PF
#define KVSHOT_BAL_PF 1
#endif
#ifndef KVSHOT_QSPLIT_MAX_RT
#define KVSHOT_QSPLIT_MAX_RT 8
#endif
// 64- and 128-row tiles: one wave per SIMD (the hi/lo query needs more than 256 registers)
#ifndef KVSHOT_RT24_WPS
#define KVSHOT_RT24_WPS 1
#endif
#ifndef KVSHOT_RT2_PF
#define KVSHOT_RT2_PF 2
#endif
#ifndef KVSHOT_RT4_PF
#define KVSHOT_RT4_PF 4
#endif
// 256-row tiles: 8 waves with one tile each (0) or 4 waves with two tiles each (1)
#ifndef KVSHOT_RT8_PF
#define KVSHOT_RT8_PF 2
#endif
#ifndef KVSHOT_RT8_TWO_TILES
#define KVSHOT_RT8_TWO_TILES 0
#endif

int mfma_waves_per_wg(int kernel_row_tiles) {
  return kernel_row_tiles >= 8 && !KVSHOT_RT8_TWO_TILES ? 8 : 4;
}

// Key streams (waves that see the same query rows but different blocks) of
// the kernel for `kernel_row_tiles`; block counts per split are rounded to it.
int mfma_key_streams(int kernel_row_tiles) {
  const int tiles_per_wave = kernel_row_tiles >= 8 && KVSHOT_RT8_TWO_TILES ? 2 : 1;
  return mfma_waves_per_wg(kernel_row_tiles) * tiles_per_wave / kernel_row_tiles;
}

// Workgroups of the kernel for `kernel_row_tiles` that one CU (4 SIMDs) holds at once.
int mfma_wgs_per_cu(int kernel_row_tiles) {
  int wps = 2;
  if (kernel_row_tiles == 1) wps = KVSHOT_RT1_WPS;
  if (kernel_row_tiles == 2 || kernel_row_tiles == 4) wps = KVSHOT_RT24_WPS;
  if (kernel_row_tiles >= 8 && KVSHOT_RT8_TWO_TILES) wps = 1;
  const int wgs = 4 * wps / mfma_waves_per_wg(kernel_row_tiles);
  return wgs < 1 ? 1 : wgs;
}

// Largest query tile one workgroup holds (in 32-row tiles); taller tiles run
// as several workgroups per (sequence, KV head, split), each with its own rows
// and its own copy of the K/V stream (kept on one L2 by the XCD renumbering).
// One workgroup for 256 rows measures faster than two for 128 rows each.
#ifndef KVSHOT_MAX_KERNEL_ROW_TILES
#define KVSHOT_MAX_KERNEL_ROW_TILES 8
#endif
int mfma_kernel_row_tiles(int row_tiles) {
  return row_tiles > KVSHOT_MAX_KERNEL_ROW_TILES ? KVSHOT_MAX_KERNEL_ROW_TILES : row_tiles;
}

hipError_t launch_attn_mfma(const AttnParams& p, int kernel_row_tiles, hipStream_t s) {
  const dim3 grid((unsigned)(p.balanced ? (int64_t)p.items * p.row_groups * p.hkv
                                         : (int64_t)p.splits * p.row_groups * p.hkv * p.batch));
  constexpr bool q1 = KVSHOT_QSPLIT_MAX_RT >= 1, q2 = KVSHOT_QSPLIT_MAX_RT >= 2, q4 = KVSHOT_QSPLIT_MAX_RT >= 4,
                 q8 = KVSHOT_QSPLIT_MAX_RT >= 8;
  switch (kernel_row_tiles) {
    case 1:
      // balanced schedule: one-wave workgroups, each wave its own item (four items per CU)
      if (p.balanced)
        hipLaunchKernelGGL((attn_mfma_kernel<1, 1, 1, KVSHOT_BAL_PF, q1, KVSHOT_RT1_WPS>), grid, dim3(64), 0, s, p);
      else
        hipLaunchKernelGGL((attn_mfma_kernel<1, 1, 4, KVSHOT_RT1_PF, q1, KVSHOT_RT1_WPS>), grid, dim3(256), 0, s, p);
      break;
    case 2:
      hipLaunchKernelGGL((attn_mfma_kernel<2, 1, 4, KVSHOT_RT2_PF, q2, KVSHOT_RT24_WPS>), grid, dim3(256), 0, s, p);
      break;
    case 4:
      hipLaunchKernelGGL((attn_mfma_kernel<4, 1, 4, KVSHOT_RT4_PF, q4, KVSHOT_RT24_WPS>), grid, dim3(256), 0, s, p);
      break;
    case 8:
      if constexpr (KVSHOT_RT8_TWO_TILES)
        hipLaunchKernelGGL((attn_mfma_kernel<8, 2, 4, 2, q8, 1>), grid, dim3(256), 0, s, p);
      else
        hipLaunchKernelGGL((attn_mfma_kernel<8, 1, 8, KVSHOT_RT8_PF, q8, 2>), grid, dim3(512), 0, s, p);
      break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace kvshot
