// Gated delta fusion of the hybrid drafter on bf16 MFMA (gfx950).
//
// Sec. 3.4.1, Eqs. (delta) and (fusion), shapes from App. B ("Shared gate"):
// for each draft token, Delta = o - n, g = sigmoid(W_g [n; o; Delta] + b_g)
// and h = n + g * (W_Delta Delta).  The gate and the delta projection land on
// the same output element, so one workgroup computes both for a tile of TT
// tokens (64, or 128 for large token counts, where the bigger tile halves how
// often each weight chunk is read from L2) x 128 channels and applies the
// epilogue in registers.
//
// Reduction space: four segments of length d -- (n, W_g[:, 0:d]),
// (o, W_g[:, d:2d]) and (Delta, W_g[:, 2d:3d]) into the gate accumulator,
// (Delta, W_Delta) into the delta accumulator.  With few tokens (one draft
// step of a batch) the segments, and then halves of them, are split over
// workgroups so the grid still fills the chip; with 128-token tiles the
// reduction index range of all four segments is split instead (each split
// reads only its part of n and o).  A second kernel sums the split partials
// and applies the epilogue.
//
// Operands: activations are the A operand (rows = tokens).  They are staged
// through LDS, where Delta is formed once per element (o - n in float32,
// rounded to bf16).  Weights are the B operand (columns = channels), loaded
// straight into registers.  Within a chunk of kKC reduction indices, a lane of
// half h covers indices h kKC/2 .. (h + 1) kKC/2 - 1, and MFMA k-step s takes
// indices h kKC/2 + 8s .. + 7 from both operands (any pairing of operand
// slots with reduction indices gives the same sum, as long as A and B agree).
//
// Weight layouts: the row-major matrices as given (a lane's 16-byte loads
// are kKC contiguous bytes of one weight row, so one load instruction touches
// 32 rows), or a packed copy made once by fusion_pack_kernel in which the
// 16-byte pieces sit in exactly the order the waves load them:
//   [channel tile][segment][chunk][wave][k-step s][lane][8 values],
// so every load instruction reads 1 KB contiguous and one workgroup's chunk of
// a segment is contiguous.
#include "fusion_common.h"

namespace kvshot {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

#ifndef KVSHOT_FUSION_STAGE_FIRST
#define KVSHOT_FUSION_STAGE_FIRST 1
#endif
#ifndef KVSHOT_FUSION_KC
#define KVSHOT_FUSION_KC 64
#endif
constexpr int kKC = KVSHOT_FUSION_KC;                  // reduction chunk per loop iteration (d % (2 kKC) == 0)
constexpr int kSteps = kKC / 16;                       // MFMA k-steps per chunk
constexpr int kHalfSpan = kKC / 2;                     // reduction indices per lane half and chunk
constexpr int kPitch = kKC + 8;                        // LDS row pitch (bf16): rows shift by 4 banks, so 16-byte row reads are conflict-free
constexpr int kRowPieces = kKC / 8;                    // 16-byte pieces per activation row and chunk
static_assert(kKC == 64 || kKC == 128, "chunk size");

__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 v) { return __builtin_bit_cast(bf16x8, v); }

// o - n per bf16 element (exact in float32), rounded to bf16
__device__ __forceinline__ u32x4 bf16x8_sub(u32x4 o, u32x4 n) {
  u32x4 r;
#pragma unroll
  for (int e = 0; e < 4; ++e) r[e] = pack_bf16x2(bf16_lo(o[e]) - bf16_lo(n[e]), bf16_hi(o[e]) - bf16_hi(n[e]));
  return r;
}

__device__ __forceinline__ float sigmoidf_fast(float z) {
  // 1 / (1 + 2^(-z log2 e)); saturates to exactly 0 and 1 for large |z|
  return __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(-z * 1.4426950408889634f));
}

// NSEG: segments of the reduction space this workgroup covers (4: all of
// them; 2 or 1 when split).  Segment i of a split is seg0 + i; a split covers
// the index range kbeg .. kbeg + d / kparts - 1 of its segments.  PF: chunks in
// flight (activation and weight registers of each).  TT: tokens per tile.
// WPS: workgroups per CU the register budget allows (a split kernel with one
// segment is small enough for two, which hides each one's per-chunk latency).
template <int NSEG, int PF, bool PACKED, int WPS, int TT>
__global__ __launch_bounds__(256, WPS) void fusion_kernel(FusionParams p) {
  static_assert(PF >= 2, "activations are staged one chunk ahead of the slot being computed");
  static_assert(TT == 64 || TT == 128, "token tile");
  constexpr int kAPieces = TT * kRowPieces / 256;       // pieces per thread and tensor
  constexpr int kTileElems = TT * kPitch;              // one activation tile
  constexpr int kTB = TT / 32;                         // 32-token MFMA blocks per tile
  __shared__ __attribute__((aligned(16))) uint16_t lds[2][3][kTileElems];   // [buffer][n, o, Delta]

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int hh = lane >> 5;
  // work item: token tile fastest, then channel tile, then split.  Consecutive
  // items share one XCD's L2: the token tiles of a channel tile read the same
  // weights, and the items of one split read only that split's part of the
  // activations, so an XCD fetches a split's activations rather than all of
  // them (with the split outermost, 480 tokens fetch 1.2x the weight bytes
  // instead of 1.5x)
  int wi = xcd_remap(blockIdx.x, gridDim.x);
  const int mt = wi % p.m_tiles;
  wi /= p.m_tiles;
  const int ntile = wi % p.n_tiles;
  const int split = wi / p.n_tiles;
  const int m0 = mt * TT;
  const int d = p.d;
  const int kparts = p.kparts;                          // reduction-index parts per segment
  const int seg0 = NSEG == 4 ? 0 : (split / kparts) * NSEG;
  const int klen = d / kparts;
  const int kbeg = (split % kparts) * klen;
  const int nchunks = klen / kKC;

  const bool cross_only = p.cross_only != 0;
  const bool has_n = seg0 == 0 && !cross_only;          // segment 0 reads n (zero when cross-only)
  const bool has_o = seg0 <= 1 && seg0 + NSEG > 1;      // segment 1 reads o
  const bool has_delta = seg0 + NSEG > 2;               // segments 2 and 3 read Delta
  const bool load_n = !cross_only && (has_n || has_delta);
  const bool load_o = has_o || has_delta;
  // loads are issued unconditionally (from o when n is absent) and masked by select, so the loop has no branches
  const uint16_t* nsrc = cross_only ? p.o : p.n;

  // ---- activations: thread t stages 16-byte pieces t and t + 256 of each tile ----
  auto load_a = [&](int chunk, u32x4 (&an)[kAPieces], u32x4 (&ao)[kAPieces]) {
    const int k0 = kbeg + chunk * kKC;
#pragma unroll
    for (int i = 0; i < kAPieces; ++i) {
      const int pc = tid + 256 * i;
      int m = m0 + pc / kRowPieces;
      m = m < p.tokens ? m : p.tokens - 1;
      const int64_t off = (int64_t)m * d + k0 + 8 * (pc % kRowPieces);
      const u32x4 vn = *(const u32x4*)(nsrc + (load_n ? off : 0));    // an unneeded tile reads one line
      const u32x4 vo = *(const u32x4*)(p.o + (load_o ? off : 0));
      an[i] = load_n ? vn : u32x4{0u, 0u, 0u, 0u};
      ao[i] = load_o ? vo : u32x4{0u, 0u, 0u, 0u};
    }
  };
  // one piece of the all-segment path, as loaded: n is zeroed for cross-only calls where it is
  // staged (a select here would make the wave wait for the load)
  auto load_a_piece = [&](int chunk, int i, u32x4 (&an)[kAPieces], u32x4 (&ao)[kAPieces]) {
    const int pc = tid + 256 * i;
    int m = m0 + pc / kRowPieces;
    m = m < p.tokens ? m : p.tokens - 1;
    const int64_t off = (int64_t)m * d + kbeg + chunk * kKC + 8 * (pc % kRowPieces);
    an[i] = *(const u32x4*)(nsrc + off);
    ao[i] = *(const u32x4*)(p.o + off);
  };
  auto stage_a = [&](int buf, const u32x4 (&an)[kAPieces], const u32x4 (&ao)[kAPieces]) {
#pragma unroll
    for (int i = 0; i < kAPieces; ++i) {
      const int pc = tid + 256 * i;
      const int row = pc / kRowPieces;
      const bool valid = m0 + row < p.tokens;           // rows past the last token stay zero
      const u32x4 vn = valid ? an[i] : u32x4{0u, 0u, 0u, 0u};
      const u32x4 vo = valid ? ao[i] : u32x4{0u, 0u, 0u, 0u};
      uint16_t* dst = &lds[buf][0][row * kPitch + 8 * (pc % kRowPieces)];
      *(u32x4*)dst = vn;
      *(u32x4*)(dst + kTileElems) = vo;
      *(u32x4*)(dst + 2 * kTileElems) = bf16x8_sub(vo, vn);
    }
  };

  // ---- weights: this lane's output channel and the weight row of each segment ----
  const int wc = ntile * kFusionChannels + w * 32 + (lane & 31);
  const uint16_t* wrow[NSEG];
#pragma unroll
  for (int i = 0; i < NSEG; ++i) {
    const int seg = seg0 + i;
    wrow[i] = seg < 3 ? p.w_g + (int64_t)wc * 3 * d + (int64_t)seg * d : p.w_delta + (int64_t)wc * d;
  }
  // packed layout: piece (channel tile, segment, chunk, wave, s, lane) at
  // ((((ntile * 4 + seg) * chunks_per_segment + chunk) * 4 + w) * kSteps + s) * 512 + lane * 8
  const int chunks_per_segment = d / kKC;
  const uint16_t* wpk[NSEG];
#pragma unroll
  for (int i = 0; i < NSEG; ++i)
    wpk[i] = p.w_packed + ((((int64_t)ntile * 4 + seg0 + i) * chunks_per_segment + kbeg / kKC) * 4 + w) * kSteps * 512 +
             lane * 8;
  auto load_w_one = [&](int chunk, int i, int s, u32x4 (&dst)[NSEG][kSteps]) {
    if constexpr (PACKED) dst[i][s] = *(const u32x4*)(wpk[i] + (int64_t)chunk * (4 * kSteps * 512) + s * 512);
    else dst[i][s] = *(const u32x4*)(wrow[i] + kbeg + chunk * kKC + kHalfSpan * hh + 8 * s);
  };
  auto load_w = [&](int chunk, u32x4 (&dst)[NSEG][kSteps]) {
    if constexpr (PACKED) {
#pragma unroll
      for (int i = 0; i < NSEG; ++i)
#pragma unroll
        for (int s = 0; s < kSteps; ++s)
          dst[i][s] = *(const u32x4*)(wpk[i] + (int64_t)chunk * (4 * kSteps * 512) + s * 512);
    } else {
      const int k = kbeg + chunk * kKC + kHalfSpan * hh;
#pragma unroll
      for (int i = 0; i < NSEG; ++i)
#pragma unroll
        for (int s = 0; s < kSteps; ++s) dst[i][s] = *(const u32x4*)(wrow[i] + k + 8 * s);
    }
  };

  // Accumulators: with all four segments, [0] gate and [1] delta projection;
  // with a split, one per segment of the split.  Segment seg reads activation
  // tile min(seg, 2) (n, o, Delta) -- an address, not a branch.
  constexpr int NACC = NSEG == 4 ? 2 : NSEG;
  f32x16 acc[NACC][kTB];
#pragma unroll
  for (int a = 0; a < NACC; ++a)
#pragma unroll
    for (int t = 0; t < kTB; ++t) acc[a][t] = f32x16{};
  int tile_of[NSEG];
#pragma unroll
  for (int i = 0; i < NSEG; ++i) tile_of[i] = min(seg0 + i, 2) * kTileElems;

  // Fragments of one k-step: [32-token block][tensor read] (all four segments: n, o and Delta, the
  // last one feeding both accumulators; a split: one read per segment).
  constexpr int NF = NSEG == 4 ? 3 : NSEG;
  auto read_frags = [&](const uint16_t* base, int s, bf16x8 (&f)[kTB][NF]) {
#pragma unroll
    for (int t = 0; t < kTB; ++t) {
      const int off = (32 * t + (lane & 31)) * kPitch + kHalfSpan * hh + 8 * s;
      if constexpr (NSEG == 4) {
#pragma unroll
        for (int j = 0; j < 3; ++j) f[t][j] = as_bf16x8(*(const u32x4*)(base + j * kTileElems + off));
      } else {
#pragma unroll
        for (int i = 0; i < NSEG; ++i) f[t][i] = as_bf16x8(*(const u32x4*)(base + tile_of[i] + off));
      }
    }
  };
  auto mfmas = [&](int s, const bf16x8 (&f)[kTB][NF], const u32x4 (&wr)[NSEG][kSteps]) {
#pragma unroll
    for (int t = 0; t < kTB; ++t) {
      if constexpr (NSEG == 4) {
        acc[0][t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(f[t][0], as_bf16x8(wr[0][s]), acc[0][t], 0, 0, 0);
        acc[0][t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(f[t][1], as_bf16x8(wr[1][s]), acc[0][t], 0, 0, 0);
        acc[0][t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(f[t][2], as_bf16x8(wr[2][s]), acc[0][t], 0, 0, 0);
        acc[1][t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(f[t][2], as_bf16x8(wr[3][s]), acc[1][t], 0, 0, 0);
      } else {
#pragma unroll
        for (int i = 0; i < NSEG; ++i)
          acc[i][t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(f[t][i], as_bf16x8(wr[i][s]), acc[i][t], 0, 0, 0);
      }
    }
  };
  // One chunk from LDS buffer buf.  The operand reads of k-step s + 1 are issued before the
  // products of k-step s (scheduling barriers keep them there), so their LDS latency hides behind
  // the matrix core instead of stalling each product on a read issued just before it.
  auto compute = [&](int buf, const u32x4 (&wr)[NSEG][kSteps]) {
    const uint16_t* base = &lds[buf][0][0];
    bf16x8 f[2][kTB][NF];
    read_frags(base, 0, f[0]);
#pragma unroll
    for (int s = 0; s < kSteps; ++s) {
      if (s + 1 < kSteps) read_frags(base, s + 1, f[(s + 1) & 1]);
      __builtin_amdgcn_sched_barrier(0);
      mfmas(s, f[s & 1], wr);
      __builtin_amdgcn_sched_barrier(0);
    }
  };

  u32x4 ran[PF][kAPieces], rao[PF][kAPieces];
  u32x4 wreg[PF][NSEG][kSteps];
  const int last = nchunks - 1;
  if constexpr (NSEG == 4) {
    // ---- main loop, software-pipelined (all four segments) ----
    // Chunk c is computed in kSteps regions, one per MFMA k-step, from LDS
    // buffer c & 1 and ring slot c % PF.  After each product the wave issues
    // one small item, held in place by scheduling barriers, so that it goes
    // out while the matrix core works through the product before it:
    //  - the LDS read of the fragment that product has just freed, for the
    //    next k-step (in the last region: chunk c + 1's first k-step, from the
    //    other buffer, after the chunk's one barrier);
    //  - one part of an activation piece of chunk c + 1 (its n and o written
    //    to the other buffer, one word of its Delta formed, or its Delta
    //    written), in the regions before the barrier;
    //  - the global loads that refill the ring with chunk c + PF: in region
    //    r the weights of k-step r - 1 (region 0: the previous slot's last
    //    k-step), and piece i of the activations in the region after the
    //    one that stages piece i of chunk c + 1 (whose registers that frees).
    // Every item list is fixed at compile time, so the code of a chunk is one
    // straight sequence.  Rows past the last token hold copies of the last
    // token's row: their outputs are never stored, and no other row reads them.
    constexpr int kNMF = 4 * kTB;                                   // products per region
    constexpr int kStageRegions = kSteps - 1;                       // regions that stage (the last one has the barrier)
    constexpr int kQ = 6;                                           // items per staged piece
    bf16x8 f[kTB][3];
    u32x4 dl[kAPieces];                                             // Delta of each piece, formed one word at a time
#pragma unroll
    for (int u = 0; u < PF; ++u) {
      load_a(min(u, last), ran[u], rao[u]);
      load_w(min(u, last), wreg[u]);
    }
    stage_a(0, ran[0], rao[0]);
    __syncthreads();
#pragma unroll
    for (int t = 0; t < kTB; ++t) {
      const int off = (32 * t + (lane & 31)) * kPitch + kHalfSpan * hh;
#pragma unroll
      for (int j = 0; j < 3; ++j) f[t][j] = as_bf16x8(*(const u32x4*)(&lds[0][j][0] + off));
    }
    // Nothing in flight on entry: otherwise the prologue's load order, merged with the loop's own at
    // the loop head, makes the compiler wait for every load at the top of each iteration.
    __builtin_amdgcn_s_waitcnt(0);
    // chunk c from ring slot u = c % PF (u is a constant at every call)
    auto chunk = [&](const int c, const int u) __attribute__((always_inline)) {
      const int refill = min(c + PF, last);
      const int refill_prev = min(c - 1 + PF, last);              // chunk c = 0: the data the slot already holds
      u32x4 (&an1)[kAPieces] = ran[(u + 1) % PF];
      u32x4 (&ao1)[kAPieces] = rao[(u + 1) % PF];
      uint16_t* nbuf = &lds[(c + 1) & 1][0][0];
      const uint16_t* cbuf = &lds[c & 1][0][0];
#pragma unroll
      for (int r = 0; r < kSteps; ++r) {
        if (r == kSteps - 1) {
          __builtin_amdgcn_sched_barrier(0);
          __syncthreads();                                        // chunk c + 1 staged; buffer c & 1 free after this region's reads
          __builtin_amdgcn_sched_barrier(0);
        }
        const uint16_t* rbase = r + 1 < kSteps ? cbuf : nbuf;
        const int rs = r + 1 < kSteps ? r + 1 : 0;
        // Items of region r, in order: the kQ parts of each piece staged in r (piece i is staged
        // in region i kStageRegions / kAPieces: n and o written, Delta formed one word at a time,
        // Delta written), the NSEG weight loads, and the loads of the slot's pieces whose
        // counterparts were staged in the region before.  Item it follows product it kNMF / n_all.
        int npc = 0, first_pc = 0, nld = 0, first_ld = 0;
#pragma unroll
        for (int i = 0; i < kAPieces; ++i) {
          const int sr = (i * kStageRegions) / kAPieces;
          if (sr == r) { first_pc = npc == 0 ? i : first_pc; ++npc; }
          if (sr + 1 == r) { first_ld = nld == 0 ? i : first_ld; ++nld; }
        }
        const int n_all = kQ * npc + 4 + nld;
#pragma unroll
        for (int slot = 0; slot < kNMF; ++slot) {
          const int t = slot >> 2, g = slot & 3;
          // product g of block t: gate n, o, Delta; then the delta projection from Delta
          if (g == 0) acc[0][t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(f[t][0], as_bf16x8(wreg[u][0][r]), acc[0][t], 0, 0, 0);
          if (g == 1) acc[0][t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(f[t][1], as_bf16x8(wreg[u][1][r]), acc[0][t], 0, 0, 0);
          if (g == 2) acc[0][t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(f[t][2], as_bf16x8(wreg[u][2][r]), acc[0][t], 0, 0, 0);
          if (g == 3) acc[1][t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(f[t][2], as_bf16x8(wreg[u][3][r]), acc[1][t], 0, 0, 0);
          __builtin_amdgcn_sched_barrier(0);
          // the fragment this product freed (Delta after its second use)
          {
            const int off = (32 * t + (lane & 31)) * kPitch + kHalfSpan * hh + 8 * rs;
            if (g == 0) f[t][0] = as_bf16x8(*(const u32x4*)(rbase + off));
            if (g == 1) f[t][1] = as_bf16x8(*(const u32x4*)(rbase + kTileElems + off));
            if (g == 3) f[t][2] = as_bf16x8(*(const u32x4*)(rbase + 2 * kTileElems + off));
          }
          // this slot's share of the region's items
          const int it_lo = (slot * n_all + kNMF - 1) / kNMF, it_hi = ((slot + 1) * n_all + kNMF - 1) / kNMF;
#pragma unroll
          for (int k = 0; k < 2; ++k) {
            const int it = it_lo + k;
            if (it >= it_hi) break;
            if (it < kQ * npc) {
              const int i = first_pc + it / kQ, q = it % kQ;
              const int pc = tid + 256 * i;
              uint16_t* dst = nbuf + (pc / kRowPieces) * kPitch + 8 * (pc % kRowPieces);
              if (q == 0) {
                an1[i] = load_n ? an1[i] : u32x4{0u, 0u, 0u, 0u};
                *(u32x4*)dst = an1[i];
                *(u32x4*)(dst + kTileElems) = ao1[i];
              } else if (q < kQ - 1) {
                const int e = q - 1;                                // o - n per bf16 element (exact in float32), rounded to bf16
                dl[i][e] = pack_bf16x2(bf16_lo(ao1[i][e]) - bf16_lo(an1[i][e]), bf16_hi(ao1[i][e]) - bf16_hi(an1[i][e]));
              } else {
                *(u32x4*)(dst + 2 * kTileElems) = dl[i];
              }
            } else if (it < kQ * npc + 4) {
              const int sg = it - kQ * npc;
              if (r > 0) load_w_one(refill, sg, r - 1, wreg[u]);
              else load_w_one(refill_prev, sg, kSteps - 1, wreg[(u + PF - 1) % PF]);
            } else {
              load_a_piece(refill, first_ld + (it - kQ * npc - 4), ran[u], rao[u]);
            }
          }
          __builtin_amdgcn_sched_barrier(0);
        }
      }
      // the last region's weights are refilled in the next chunk's first region
    };
    // Whole ring groups in the loop and the rest after it: a chunk skipped inside the loop would
    // leave different loads in flight on one path into the loop head, and the compiler would then
    // wait for every load there.
    int c0 = 0;
    for (; c0 + PF <= nchunks; c0 += PF) {
#pragma unroll
      for (int u = 0; u < PF; ++u) chunk(c0 + u, u);
    }
#pragma unroll
    for (int u = 0; u + 1 < PF; ++u)
      if (c0 + u < nchunks) chunk(c0 + u, u);
  } else {
  // ---- main loop of the split kernels ----
  // Ring slot c % PF holds the activation and weight registers of chunk c.
  // Chunk c is computed from LDS buffer c & 1 and its weight slot; then the
  // activations of chunk c + 1 go to the other buffer, and the slot is
  // refilled with chunk c + PF.  Every refill is issued (clamped to the last
  // chunk; iterations past the last chunk only keep the pattern), so the
  // loads behind each slot are the same on every path and the waits cover
  // just the slot in use.
#pragma unroll
  for (int u = 0; u < PF; ++u) {
    load_a(min(u, last), ran[u], rao[u]);
    load_w(min(u, last), wreg[u]);
  }
  stage_a(0, ran[0], rao[0]);
  __syncthreads();
  for (int c0 = 0; c0 < nchunks; c0 += PF) {
#pragma unroll
    for (int u = 0; u < PF; ++u) {
      const int c = c0 + u;
#if KVSHOT_FUSION_STAGE_FIRST
      // the other buffer's activations first: their LDS writes overlap this chunk's products
      if (c + 1 < nchunks) stage_a((c + 1) & 1, ran[(u + 1) % PF], rao[(u + 1) % PF]);
      if (c < nchunks) compute(c & 1, wreg[u]);
#else
      if (c < nchunks) compute(c & 1, wreg[u]);
      if (c + 1 < nchunks) stage_a((c + 1) & 1, ran[(u + 1) % PF], rao[(u + 1) % PF]);
#endif
      load_a(min(c + PF, last), ran[u], rao[u]);
      load_w(min(c + PF, last), wreg[u]);
      __syncthreads();
    }
  }
  }

  // ---- epilogue: accumulator register v of lane (channel, hh) is token 8(v/4) + 4hh + v%4 of its 32-row tile ----
  const bool fused = p.splits == 1;
  const float bias = fused ? p.b_g[wc] : 0.0f;
#pragma unroll
  for (int t = 0; t < kTB; ++t) {
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      const int m = m0 + 32 * t + 8 * (v >> 2) + 4 * hh + (v & 3);
      if (m >= p.tokens) continue;
      const int64_t idx = (int64_t)m * d + wc;
      // this workgroup's share of the gate pre-activation and of the delta projection
      float zg = 0.0f, zd = 0.0f;
      if constexpr (NSEG == 4) {
        zg = acc[0][t][v];
        zd = acc[1][t][v];
      } else {
#pragma unroll
        for (int i = 0; i < NSEG; ++i) {
          if (seg0 + i < 3) zg += acc[i][t][v];
          else zd += acc[i][t][v];
        }
      }
      if (fused) {
        const float g = sigmoidf_fast(zg + bias);
        const float nv = cross_only ? 0.0f : __uint_as_float((uint32_t)p.n[idx] << 16);
        const float hv = nv + g * zd;
        if (p.out_fp32) ((float*)p.h)[idx] = hv;
        else ((uint16_t*)p.h)[idx] = (uint16_t)(pack_bf16x2(hv, 0.0f) & 0xffffu);
        if (p.g_out) p.g_out[idx] = g;
      } else {
        const int64_t plane = (int64_t)p.tokens * d;
        if (seg0 < 3) p.part[(2 * split) * plane + idx] = zg;
        if (seg0 + NSEG > 3) p.part[(2 * split + 1) * plane + idx] = zd;
      }
    }
  }
}

// Split partials -> epilogue: sums, in split order (deterministic), the gate
// planes and the delta-projection planes that the splits wrote, then
// h = n + sigmoid(gate + b_g) * delta projection.  One thread per four channels.
__global__ __launch_bounds__(256) void fusion_combine_kernel(FusionParams p) {
  const int64_t quads = (int64_t)p.tokens * p.d / 4;
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= quads) return;
  const int64_t idx = 4 * i;                            // element (m, c), c % 4 == 0
  const int c = (int)(idx % p.d);
  const int64_t plane = (int64_t)p.tokens * p.d;
  f32x4 g = {0.f, 0.f, 0.f, 0.f}, e = {0.f, 0.f, 0.f, 0.f};
  for (int s = 0; s < p.splits; ++s) {
    if ((p.part_g_mask >> s) & 1u) g += *(const f32x4*)(p.part + (2 * s) * plane + idx);
    if ((p.part_d_mask >> s) & 1u) e += *(const f32x4*)(p.part + (2 * s + 1) * plane + idx);
  }
  const f32x4 b = *(const f32x4*)(p.b_g + c);
  f32x4 nv = {0.f, 0.f, 0.f, 0.f};
  if (!p.cross_only) {
    const uint2 nn = *(const uint2*)(p.n + idx);
    nv = f32x4{bf16_lo(nn.x), bf16_hi(nn.x), bf16_lo(nn.y), bf16_hi(nn.y)};
  }
  f32x4 ga, hv;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    ga[j] = sigmoidf_fast(g[j] + b[j]);
    hv[j] = nv[j] + ga[j] * e[j];
  }
  if (p.out_fp32) *(f32x4*)((float*)p.h + idx) = hv;
  else *(uint2*)((uint16_t*)p.h + idx) = make_uint2(pack_bf16x2(hv[0], hv[1]), pack_bf16x2(hv[2], hv[3]));
  if (p.g_out) *(f32x4*)(p.g_out + idx) = ga;
}

#ifndef KVSHOT_FUSION_PF4
#define KVSHOT_FUSION_PF4 2
#endif
#ifndef KVSHOT_FUSION_PF2
#define KVSHOT_FUSION_PF2 3
#endif
#ifndef KVSHOT_FUSION_PF1
#define KVSHOT_FUSION_PF1 4
#endif

#ifndef KVSHOT_FUSION_PF4_TT128
#define KVSHOT_FUSION_PF4_TT128 2
#endif

template <bool PACKED>
void launch_fusion_t(const FusionParams& p, hipStream_t s) {
  const dim3 grid((unsigned)((int64_t)p.m_tiles * p.n_tiles * p.splits));
  if (p.tile_tokens == 128) {   // every split covers all four segments (kparts == splits)
    hipLaunchKernelGGL((fusion_kernel<4, KVSHOT_FUSION_PF4_TT128, PACKED, 1, 128>), grid, dim3(256), 0, s, p);
    return;
  }
  if (p.splits <= 1) hipLaunchKernelGGL((fusion_kernel<4, KVSHOT_FUSION_PF4, PACKED, 1, 64>), grid, dim3(256), 0, s, p);
  else if (p.splits == 2)
    hipLaunchKernelGGL((fusion_kernel<2, KVSHOT_FUSION_PF2, PACKED, 1, 64>), grid, dim3(256), 0, s, p);
  else hipLaunchKernelGGL((fusion_kernel<1, KVSHOT_FUSION_PF1, PACKED, 2, 64>), grid, dim3(256), 0, s, p);
}

// One thread per 16-byte piece of the packed copy: it reads the 8 weights of
// that piece from the row-major matrices (see the layout above).
__global__ __launch_bounds__(256) void fusion_pack_kernel(const uint16_t* w_g, const uint16_t* w_delta,
                                                           uint16_t* packed, int d) {
  const int64_t pieces = (int64_t)d * d / 2;             // 4 d^2 values / 8 per piece
  const int64_t q = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (q >= pieces) return;
  const int cps = d / kKC;
  const int lane = (int)(q & 63);
  const int s = (int)((q >> 6) % kSteps);
  const int w = (int)((q / (64 * kSteps)) & 3);
  int64_t r = q / (256 * kSteps);
  const int chunk = (int)(r % cps);
  r /= cps;
  const int seg = (int)(r & 3);
  const int ntile = (int)(r >> 2);
  const int c = ntile * kFusionChannels + w * 32 + (lane & 31);
  const int k = chunk * kKC + kHalfSpan * (lane >> 5) + 8 * s;
  const uint16_t* src = seg < 3 ? w_g + (int64_t)c * 3 * d + (int64_t)seg * d + k : w_delta + (int64_t)c * d + k;
  *(u32x4*)(packed + q * 8) = *(const u32x4*)src;
}

}  // namespace

hipError_t launch_fusion(const FusionParams& p, hipStream_t s) {
  if (p.w_packed) launch_fusion_t<true>(p, s);
  else launch_fusion_t<false>(p, s);
  return hipGetLastError();
}

hipError_t launch_fusion_pack(const uint16_t* w_g, const uint16_t* w_delta, uint16_t* packed, int d, hipStream_t s) {
  const int64_t pieces = (int64_t)d * d / 2;
  hipLaunchKernelGGL(fusion_pack_kernel, dim3((unsigned)((pieces + 255) / 256)), dim3(256), 0, s, w_g, w_delta,
                     packed, d);
  return hipGetLastError();
}

hipError_t launch_fusion_combine(const FusionParams& p, hipStream_t s) {
  const int64_t quads = (int64_t)p.tokens * p.d / 4;
  hipLaunchKernelGGL(fusion_combine_kernel, dim3((unsigned)((quads + 255) / 256)), dim3(256), 0, s, p);
  return hipGetLastError();
}

}  // namespace kvshot
