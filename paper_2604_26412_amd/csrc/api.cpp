// Host side of the C ABI declared in include/kvshot_draft_attn.h: argument
// validation, the handle (workspace, RoPE table, profiling events), the split-K
// plan and kernel launches.  No call here synchronises the host except
// destroy, validate and profile_read.
#include "kvshot_draft_attn.h"

#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>
#include <cstdlib>
#include <cstring>
#include <mutex>
#include <new>
#include <vector>

#include "device_guard.h"
#include "kvshot_common.h"

namespace kvshot {
// the matrix-rate probe (csrc/debug.hip); declared here, beside its one caller
hipError_t launch_mfma_rate(int blocks, int iters, void* sink, hipStream_t s);
}  // namespace kvshot

using namespace kvshot;

namespace {

constexpr int kProfileRing = 1024;

struct ProfileSlot {
  hipEvent_t ev[3];
  int has_combine;
};

}  // namespace

struct kvshot_ctx {
  kvshot_config cfg;
  int device;
  int group;
  int page_shift;
  int rows_pad_max;
  int max_splits;
  int num_cus;
  float2* rope = nullptr;
  float* part_o = nullptr;
  float2* part_ml = nullptr;
  int32_t* flag = nullptr;
  int32_t* seq_splits = nullptr;   // [2][64]: per-sequence split counts and first items of a balanced call
  size_t ws_rows = 0;       // capacity of the partial workspace in (row, split) entries
  int opt_splits = 0, opt_path = 0, opt_profile = 0;
  std::vector<ProfileSlot> prof;
  int64_t prof_head = 0, prof_tail = 0;
  double attn_ms = 0.0, combine_ms = 0.0;
  int64_t calls = 0;
};

namespace {

bool is_pow2(int v) { return v > 0 && (v & (v - 1)) == 0; }
bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

struct Plan {
  int path;        // 1 mfma, 2 generic
  int row_tiles;   // 32-row query tiles per (sequence, KV head)
  int kernel_row_tiles;  // of which one workgroup holds (row_groups = row_tiles / kernel_row_tiles)
  int row_groups;
  int key_streams;
  int splits;
  int blocks_per_split;
  int rows, rows_pad;
  int waves_per_wg;
  int balanced;    // length-balanced schedule: `items` work items per (KV head, row group)
  int items;
  int min_chunk;
};

// 32-row tiles from which the tall-tile kernel serves a call
constexpr int kTallRowTiles = 8;

bool use_tall_kernel() {
#ifdef KVSHOT_NO_TALL
  return false;
#else
  return true;
#endif
}

int round_tiles(int rows) {
  const int t = (rows + 31) / 32;
  return t <= 1 ? 1 : (t <= 2 ? 2 : (t <= 4 ? 4 : 8));
}

Plan make_plan(const kvshot_ctx* c, int batch, int nq, int max_ctx, bool allow_tall = true) {
  Plan pl{};
  pl.rows = c->group * nq;
  const bool generic = c->cfg.dtype == KVSHOT_FP32 || c->opt_path == 2;
  pl.path = generic ? 2 : 1;
  pl.row_tiles = round_tiles(pl.rows);
  pl.rows_pad = pl.row_tiles * 32;
  if (generic) {
    pl.kernel_row_tiles = pl.row_tiles;
    pl.row_groups = 1;
    pl.waves_per_wg = 4;
    pl.key_streams = 1;
  } else if (pl.row_tiles >= kTallRowTiles && allow_tall && c->opt_path != 3 && use_tall_kernel()) {
    // 256-row tiles (draft trees, 33..64 queries at G = 4): the tall-tile kernel
    pl.path = 3;
    pl.kernel_row_tiles = kTallRowTiles;
    pl.row_groups = pl.row_tiles / pl.kernel_row_tiles;
    pl.waves_per_wg = tall_waves_per_wg();
    pl.key_streams = 1;
  } else {
    pl.kernel_row_tiles = mfma_kernel_row_tiles(pl.row_tiles);
    pl.row_groups = pl.row_tiles / pl.kernel_row_tiles;
    pl.waves_per_wg = mfma_waves_per_wg(pl.kernel_row_tiles);
    pl.key_streams = mfma_key_streams(pl.kernel_row_tiles);
  }
  const int nb = (max_ctx + kBlockKeys - 1) / kBlockKeys;
  const int pairs = batch * c->cfg.num_kv_heads * pl.row_groups;   // workgroups per split
  int splits;
  if (c->opt_splits > 0) {
    splits = c->opt_splits;
  } else {
    // One round of resident workgroups over the chip: split the context only
    // when the (sequence, KV head) pairs alone leave CUs idle, and keep >= 4
    // blocks per wave.  (Each workgroup starts with a dependent chain of
    // loads -- length, page ids, K/V, RoPE table -- that only other resident
    // workgroups can hide, so more, shorter workgroups lose.)
    const int per_cu = generic ? 2 : (pl.path == 3 ? 1 : mfma_wgs_per_cu(pl.kernel_row_tiles));
    const int target_wgs = c->num_cus * per_cu;
    splits = (target_wgs + pairs - 1) / pairs;
    const int cap = nb / (pl.key_streams * 4);
    splits = splits > cap ? cap : splits;
  }
  if (splits < 1) splits = 1;
  // the tall-tile kernel stages a split's page ids in LDS: at most tall_max_blocks() blocks per split
  if (pl.path == 3 && nb > (int64_t)splits * tall_max_blocks()) splits = (nb + tall_max_blocks() - 1) / tall_max_blocks();
  if (splits > c->max_splits) splits = c->max_splits;
  // the workspace must hold this call's partials
  while (splits > 1 && (size_t)batch * c->cfg.num_kv_heads * pl.rows_pad * splits > c->ws_rows) --splits;
  int bps = nb > 0 ? (nb + splits - 1) / splits : 0;
  bps = ((bps + pl.key_streams - 1) / pl.key_streams) * pl.key_streams;
  if (bps > 0) splits = (nb + bps - 1) / bps;
  if (splits < 1) splits = 1;
  // more blocks per split than the tall-tile kernel stages (contexts beyond what the split cap
  // covers, or a forced split count): the general kernel serves the call
  if (pl.path == 3 && bps > tall_max_blocks()) return make_plan(c, batch, nq, max_ctx, false);
  pl.splits = splits;
  pl.blocks_per_split = bps;
  // Ragged batches of 32-row tiles on the general MFMA kernel: one-wave workgroups, one round of
  // them over the chip (four per CU), shared out as work items per KV head over the sequences in
  // proportion to their lengths (computed on the device from ctx_lens), instead of giving every
  // sequence the same split count.  With four times the items of four-wave workgroups, a sequence's
  // whole-number share of them is four times finer.  Only for batches of at most a quarter as many
  // sequences as items: larger batches fill the chip with one workgroup per (sequence, KV head) and
  // their unsplit plan needs no partials and no combine (64 x 32K: the balanced plan's combine adds
  // 16 us to a 1.26 ms step).
  if (pl.path == 1 && pl.kernel_row_tiles == 1 && c->opt_splits == 0 && batch >= 2 && batch <= 64) {
    const int per_cu = mfma_wgs_per_cu(1) * mfma_waves_per_wg(1);   // one-wave workgroups per CU
    int items = c->num_cus * per_cu / c->cfg.num_kv_heads;
    while (items > 1 && (size_t)c->cfg.num_kv_heads * pl.rows_pad * items > c->ws_rows) --items;
    if (4 * batch <= items) {
      pl.balanced = 1;
      pl.items = items;
      pl.min_chunk = 1;
      pl.waves_per_wg = 1;
      pl.key_streams = 1;
      pl.splits = items;              // the grid's items per KV head; a sequence takes at most kMaxSplits
      pl.blocks_per_split = 0;
    }
  }
  return pl;
}

void fill_params(const kvshot_ctx* c, const Plan& pl, int batch, int nq, int max_ctx, AttnParams& p) {
  const kvshot_config& g = c->cfg;
  std::memset(&p, 0, sizeof(p));
  p.rope = c->rope;
  p.part_o = c->part_o;
  p.part_ml = c->part_ml;
  p.page_stride = g.page_stride;
  p.head_stride = g.head_stride;
  p.slot_stride = g.slot_stride;
  p.batch = batch;
  p.nq = nq;
  p.hq = g.num_q_heads;
  p.hkv = g.num_kv_heads;
  p.group = c->group;
  p.page_shift = c->page_shift;
  p.max_pages_per_seq = g.max_pages_per_seq;
  p.num_pages = g.num_pages;
  p.max_draft = g.max_draft;
  p.rows = pl.rows;
  p.rows_pad = pl.rows_pad;
  p.row_groups = pl.row_groups;
  p.splits = pl.splits;
  p.blocks_per_split = pl.blocks_per_split;
  p.balanced = pl.balanced;
  p.items = pl.items;
  p.min_chunk = pl.min_chunk;
  p.max_ctx = max_ctx;
  p.max_position = (int32_t)g.max_position;
  p.out_fp32 = g.out_dtype == KVSHOT_FP32;
  const float scale = g.softmax_scale != 0.0f ? g.softmax_scale : (float)(1.0 / std::sqrt((double)g.head_dim));
  p.qscale = (float)((double)scale * 1.4426950408889634);
}

kvshot_status drain_profile(kvshot_ctx* c, bool all) {
  // fold finished (or, if `all`, every) recorded call into the sums
  while (c->prof_tail < c->prof_head) {
    ProfileSlot& s = c->prof[c->prof_tail % kProfileRing];
    if (!all && hipEventQuery(s.ev[2]) != hipSuccess) break;
    if (hipEventSynchronize(s.ev[2]) != hipSuccess) return KVSHOT_ERR_DEVICE;
    float a = 0.f, b = 0.f;
    if (hipEventElapsedTime(&a, s.ev[0], s.ev[1]) != hipSuccess) return KVSHOT_ERR_DEVICE;
    if (s.has_combine && hipEventElapsedTime(&b, s.ev[1], s.ev[2]) != hipSuccess) return KVSHOT_ERR_DEVICE;
    c->attn_ms += a;
    c->combine_ms += b;
    c->calls += 1;
    ++c->prof_tail;
  }
  return KVSHOT_OK;
}

// Workspace of one call: where the split partials go, and whether profiling events may be recorded.
struct Workspace {
  float* part_o;
  float2* part_ml;
  int32_t* seq_splits;
  bool profile;
};

kvshot_status run_call(kvshot_ctx* c, const kvshot_call& a, void* stream, const Workspace* ws = nullptr);

kvshot_status run_call(kvshot_ctx* c, const kvshot_call& a, void* stream, const Workspace* ws) {
  if (!c) return KVSHOT_ERR_INVALID_ARG;
  const kvshot_config& g = c->cfg;
  const bool tree = a.mode == KVSHOT_MODE_TREE;
  const int batch = a.batch, nq = a.n_queries, max_ctx = a.max_ctx_len_hint;
  if (a.mode != KVSHOT_MODE_STEP && a.mode != KVSHOT_MODE_TREE) return KVSHOT_ERR_INVALID_ARG;
  if (a.reserved != 0) return KVSHOT_ERR_INVALID_ARG;
  if (batch < 1 || batch > g.max_batch || nq < 1 || nq > g.max_draft) return KVSHOT_ERR_INVALID_ARG;
  if (tree && (a.n_nodes < 1 || a.n_nodes > g.max_draft)) return KVSHOT_ERR_INVALID_ARG;
  if (tree && !a.query_nodes && a.n_nodes != nq) return KVSHOT_ERR_INVALID_ARG;
  if (!tree && a.query_nodes) return KVSHOT_ERR_INVALID_ARG;
  if (c->group * nq > kMaxRows) return KVSHOT_ERR_UNSUPPORTED;
  if (max_ctx < 0 || (int64_t)max_ctx > (int64_t)g.max_pages_per_seq * g.page_size) return KVSHOT_ERR_INVALID_ARG;
  if ((int64_t)max_ctx + g.max_draft > g.max_position) return KVSHOT_ERR_INVALID_ARG;
  if (!a.q || !a.k_pages || !a.v_pages || !a.page_table || !a.ctx_lens || !a.draft_k || !a.draft_v || !a.out)
    return KVSHOT_ERR_INVALID_ARG;
  if (tree ? !a.parents : !a.step_offsets) return KVSHOT_ERR_INVALID_ARG;
  if (!aligned16(a.q) || !aligned16(a.k_pages) || !aligned16(a.v_pages) || !aligned16(a.draft_k) ||
      !aligned16(a.draft_v) || !aligned16(a.out))
    return KVSHOT_ERR_INVALID_ARG;
  if ((c->opt_path == 1 || c->opt_path == 3) && g.dtype != KVSHOT_BF16) return KVSHOT_ERR_UNSUPPORTED;
  const DeviceGuard dg(c->device);
  if (!dg.ok()) return KVSHOT_ERR_DEVICE;
  kvshot_status st = KVSHOT_OK;

  const Plan pl = make_plan(c, batch, nq, max_ctx);
  AttnParams p;
  fill_params(c, pl, batch, nq, max_ctx, p);
  p.seq_splits = c->seq_splits;
  if (ws) {
    p.part_o = ws->part_o;
    p.part_ml = ws->part_ml;
    p.seq_splits = ws->seq_splits;
  }
  p.q = a.q;
  p.k_pages = a.k_pages;
  p.v_pages = a.v_pages;
  p.page_table = a.page_table;
  p.ctx_lens = a.ctx_lens;
  p.draft_k = a.draft_k;
  p.draft_v = a.draft_v;
  p.tree = tree ? 1 : 0;
  p.n_nodes = tree ? a.n_nodes : nq;
  p.step_offsets = tree ? nullptr : a.step_offsets;
  p.parents = tree ? a.parents : nullptr;
  p.query_nodes = tree ? a.query_nodes : nullptr;
  p.pos_base = a.pos_base;
  p.out = a.out;
  p.lse = a.lse;
  void* out = a.out;
  float* lse = a.lse;
  hipStream_t s = (hipStream_t)stream;

  ProfileSlot* slot = nullptr;
  if (c->opt_profile && (!ws || ws->profile)) {
    if (c->prof_head - c->prof_tail >= kProfileRing) {
      st = drain_profile(c, false);
      if (st != KVSHOT_OK) return st;
      if (c->prof_head - c->prof_tail >= kProfileRing) {
        // ring full of unfinished calls: wait for the oldest
        ProfileSlot& o = c->prof[c->prof_tail % kProfileRing];
        if (hipEventSynchronize(o.ev[2]) != hipSuccess) return KVSHOT_ERR_DEVICE;
        st = drain_profile(c, false);
        if (st != KVSHOT_OK) return st;
      }
    }
    slot = &c->prof[c->prof_head % kProfileRing];
    if (hipEventRecord(slot->ev[0], s) != hipSuccess) return KVSHOT_ERR_DEVICE;
  }
  hipError_t e = pl.path == 1   ? launch_attn_mfma(p, pl.kernel_row_tiles, s)
                 : pl.path == 3 ? launch_attn_tall(p, s)
                                : launch_attn_generic(p, g.dtype == KVSHOT_BF16, s);
  if (e != hipSuccess) return KVSHOT_ERR_DEVICE;
  if (slot && hipEventRecord(slot->ev[1], s) != hipSuccess) return KVSHOT_ERR_DEVICE;
  if (pl.splits > 1) {
    CombineParams cp{};
    cp.part_o = p.part_o;
    cp.part_ml = p.part_ml;
    cp.out = out;
    cp.lse = lse;
    cp.batch = batch;
    cp.nq = nq;
    cp.hq = g.num_q_heads;
    cp.hkv = g.num_kv_heads;
    cp.group = c->group;
    cp.rows = pl.rows;
    cp.rows_pad = pl.rows_pad;
    cp.splits = pl.splits;
    cp.out_fp32 = g.out_dtype == KVSHOT_FP32;
    cp.seq_splits = pl.balanced ? p.seq_splits : nullptr;
    cp.items = pl.balanced ? pl.items : 0;
    if (launch_combine(cp, s) != hipSuccess) return KVSHOT_ERR_DEVICE;
  }
  if (slot) {
    if (hipEventRecord(slot->ev[2], s) != hipSuccess) return KVSHOT_ERR_DEVICE;
    slot->has_combine = pl.splits > 1;
    ++c->prof_head;
  }
  return KVSHOT_OK;
}

kvshot_status validate_impl(kvshot_ctx* c, const kvshot_call& a, int32_t* first_bad, void* stream) {
  if (first_bad) *first_bad = 0;
  if (!c || !a.page_table || !a.ctx_lens) return KVSHOT_ERR_INVALID_ARG;
  const kvshot_config& g = c->cfg;
  const bool tree = a.mode == KVSHOT_MODE_TREE;
  if (a.mode != KVSHOT_MODE_STEP && a.mode != KVSHOT_MODE_TREE) return KVSHOT_ERR_INVALID_ARG;
  if (a.batch < 1 || a.batch > g.max_batch || a.n_queries < 1 || a.n_queries > g.max_draft)
    return KVSHOT_ERR_INVALID_ARG;
  if (tree && (a.n_nodes < 1 || a.n_nodes > g.max_draft)) return KVSHOT_ERR_INVALID_ARG;
  if (a.max_ctx_len_hint < 0 || (int64_t)a.max_ctx_len_hint > (int64_t)g.max_pages_per_seq * g.page_size)
    return KVSHOT_ERR_INVALID_ARG;
  const DeviceGuard dg(c->device);
  if (!dg.ok()) return KVSHOT_ERR_DEVICE;
  kvshot_status st = KVSHOT_OK;
  const Plan pl = make_plan(c, a.batch, a.n_queries, a.max_ctx_len_hint);
  AttnParams p;
  fill_params(c, pl, a.batch, a.n_queries, a.max_ctx_len_hint, p);
  p.page_table = a.page_table;
  p.ctx_lens = a.ctx_lens;
  p.step_offsets = a.step_offsets;
  p.parents = a.parents;
  p.tree = tree ? 1 : 0;
  p.n_nodes = tree ? a.n_nodes : a.n_queries;
  p.query_nodes = tree ? a.query_nodes : nullptr;
  p.pos_base = a.pos_base;
  hipStream_t s = (hipStream_t)stream;
  if (launch_validate(p, a.max_ctx_len_hint, c->flag, s) != hipSuccess) return KVSHOT_ERR_DEVICE;
  int32_t flag = 0;
  if (hipMemcpyAsync(&flag, c->flag, sizeof(flag), hipMemcpyDeviceToHost, s) != hipSuccess) return KVSHOT_ERR_DEVICE;
  if (hipStreamSynchronize(s) != hipSuccess) return KVSHOT_ERR_DEVICE;
  if (flag == 0x7fffffff) return KVSHOT_OK;
  if (first_bad) *first_bad = flag;
  return KVSHOT_ERR_DATA;
}

// ---------------------------------------------------------------------------
// Static scratch for kvshot_draft_attn_call_noalloc: the split partials of a
// call that may not allocate.  One copy per GPU, held until the process ends.
// Its device address is resolved once per device (with that device current)
// and kept; host code uses that address, never the array's name.
// ---------------------------------------------------------------------------
constexpr size_t kScratchBytes = (size_t)32 << 20;
constexpr int kMaxDevices = 64;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// Resolve this device's scratch address (the device is current).  Idempotent.
kvshot_status resolve_scratch(int device) {
  if (device < 0 || device >= kMaxDevices) return KVSHOT_ERR_UNSUPPORTED;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch_ptr[device]) return KVSHOT_OK;
  void* ptr = nullptr;
  if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || !ptr) {
    (void)hipGetLastError();
    return KVSHOT_ERR_DEVICE;
  }
  g_scratch_ptr[device] = ptr;
  return KVSHOT_OK;
}

void* scratch_ptr(int device) {
  if (device < 0 || device >= kMaxDevices) return nullptr;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  return g_scratch_ptr[device];
}

// Scratch bytes a plan uses: split partials O float32 ([batch][Hkv][rows_pad][splits], or
// [Hkv][items][rows_pad] under the balanced schedule) x D, then (m, l) float2 per partial row, then
// the per-sequence split counts and first items of a balanced plan ([2][64] int32), each at the
// next 256-byte boundary.
size_t partial_rows(const kvshot_ctx* c, const Plan& pl, int batch) {
  if (pl.splits <= 1) return 0;
  if (pl.balanced) return (size_t)c->cfg.num_kv_heads * pl.items * pl.rows_pad;
  return (size_t)batch * c->cfg.num_kv_heads * pl.rows_pad * pl.splits;
}

size_t partial_bytes(const kvshot_ctx* c, const Plan& pl, int batch, size_t* ml_offset, size_t* seq_offset) {
  *ml_offset = 0;
  *seq_offset = 0;
  if (pl.splits <= 1) return 0;
  const size_t rows = partial_rows(c, pl, batch);
  *ml_offset = (rows * kHeadDim * sizeof(float) + 255) & ~(size_t)255;
  *seq_offset = (*ml_offset + rows * sizeof(float2) + 255) & ~(size_t)255;
  return *seq_offset + (pl.balanced ? 2 * 64 * sizeof(int32_t) : 0);
}

void free_ctx(kvshot_ctx* c) {
  if (!c) return;
  const DeviceGuard dg(c->device);
  (void)hipDeviceSynchronize();
  if (c->rope) (void)hipFree(c->rope);
  if (c->part_o) (void)hipFree(c->part_o);
  if (c->part_ml) (void)hipFree(c->part_ml);
  if (c->flag) (void)hipFree(c->flag);
  if (c->seq_splits) (void)hipFree(c->seq_splits);
  for (auto& s : c->prof)
    for (auto& e : s.ev)
      if (e) (void)hipEventDestroy(e);
  delete c;
}

}  // namespace

extern "C" {

const char* kvshot_status_string(int32_t s) {
  switch (s) {
    case KVSHOT_OK: return "ok";
    case KVSHOT_ERR_INVALID_ARG: return "invalid argument";
    case KVSHOT_ERR_UNSUPPORTED: return "unsupported configuration";
    case KVSHOT_ERR_OUT_OF_MEMORY: return "device out of memory";
    case KVSHOT_ERR_DEVICE: return "HIP device error";
    case KVSHOT_ERR_DATA: return "contract violation in device data";
    case KVSHOT_ERR_SCRATCH: return "the call's split partials exceed the no-allocation scratch buffer";
    default: return "unknown status";
  }
}

kvshot_status kvshot_draft_attn_init(const kvshot_config* cfg, kvshot_handle* out) {
  if (!cfg || !out) return KVSHOT_ERR_INVALID_ARG;
  *out = nullptr;
  kvshot_config g = *cfg;
  if (g.num_q_heads < 1 || g.num_kv_heads < 1 || g.num_q_heads % g.num_kv_heads != 0) return KVSHOT_ERR_INVALID_ARG;
  if (g.num_q_heads / g.num_kv_heads > 8) return KVSHOT_ERR_UNSUPPORTED;
  if (g.head_dim != kHeadDim) return KVSHOT_ERR_UNSUPPORTED;
  if (!is_pow2(g.page_size) || g.page_size < 16 || g.page_size > 256) return KVSHOT_ERR_INVALID_ARG;
  if ((g.dtype != KVSHOT_BF16 && g.dtype != KVSHOT_FP32) || (g.out_dtype != KVSHOT_BF16 && g.out_dtype != KVSHOT_FP32))
    return KVSHOT_ERR_INVALID_ARG;
  if (g.max_batch < 1 || g.max_batch > 65535) return KVSHOT_ERR_INVALID_ARG;
  if (g.max_draft < 1 || g.max_draft > kMaxDraft) return KVSHOT_ERR_INVALID_ARG;
  if (g.max_pages_per_seq < 1 || g.num_pages < 1) return KVSHOT_ERR_INVALID_ARG;
  if ((int64_t)g.max_pages_per_seq * g.page_size > (1ll << 30)) return KVSHOT_ERR_INVALID_ARG;
  if (g.max_position < 1 || g.max_position > (1ll << 24)) return KVSHOT_ERR_INVALID_ARG;
  if (!(g.rope_theta > 0.0) || !std::isfinite(g.rope_theta)) return KVSHOT_ERR_INVALID_ARG;
  if (!std::isfinite(g.softmax_scale) || g.softmax_scale < 0.0f) return KVSHOT_ERR_INVALID_ARG;
  if (g.reserved != 0) return KVSHOT_ERR_INVALID_ARG;
  if (g.page_stride == 0) g.page_stride = (int64_t)g.num_kv_heads * g.page_size * g.head_dim;
  if (g.head_stride == 0) g.head_stride = (int64_t)g.page_size * g.head_dim;
  if (g.slot_stride == 0) g.slot_stride = g.head_dim;
  if (g.page_stride < 0 || g.head_stride < 0 || g.slot_stride < g.head_dim) return KVSHOT_ERR_INVALID_ARG;
  if (g.page_stride % 8 || g.head_stride % 8 || g.slot_stride % 8) return KVSHOT_ERR_INVALID_ARG;

  kvshot_ctx* c = new (std::nothrow) kvshot_ctx();
  if (!c) return KVSHOT_ERR_OUT_OF_MEMORY;
  c->cfg = g;
  c->group = g.num_q_heads / g.num_kv_heads;
  c->page_shift = 0;
  while ((1 << c->page_shift) < g.page_size) ++c->page_shift;
  if (hipGetDevice(&c->device) != hipSuccess) {
    delete c;
    return KVSHOT_ERR_DEVICE;
  }
  hipDeviceProp_t prop;
  if (hipGetDeviceProperties(&prop, c->device) != hipSuccess) {
    delete c;
    return KVSHOT_ERR_DEVICE;
  }
  c->num_cus = prop.multiProcessorCount > 0 ? prop.multiProcessorCount : 256;
  const int rows_max = c->group * g.max_draft;
  c->rows_pad_max = round_tiles(rows_max) * 32;
  const int64_t max_ctx = (int64_t)g.max_pages_per_seq * g.page_size;
  const int64_t nb_max = (max_ctx + kBlockKeys - 1) / kBlockKeys;
  c->max_splits = (int)(nb_max < kMaxSplits ? (nb_max < 1 ? 1 : nb_max) : kMaxSplits);
  c->ws_rows = (size_t)g.max_batch * g.num_kv_heads * c->rows_pad_max * c->max_splits;

  // RoPE table: angle p * theta^(-2m/D) in float64, cos/sin rounded to float32
  const size_t nrope = (size_t)g.max_position * kHalfDim;
  std::vector<float2> tab(nrope);
  for (int64_t pos = 0; pos < g.max_position; ++pos)
    for (int m = 0; m < kHalfDim; ++m) {
      const double inv = std::pow(g.rope_theta, -2.0 * m / (double)g.head_dim);
      const double a = (double)pos * inv;
      tab[(size_t)pos * kHalfDim + m] = make_float2((float)std::cos(a), (float)std::sin(a));
    }
  if (hipMalloc((void**)&c->rope, nrope * sizeof(float2)) != hipSuccess ||
      hipMalloc((void**)&c->part_o, c->ws_rows * kHeadDim * sizeof(float)) != hipSuccess ||
      hipMalloc((void**)&c->part_ml, c->ws_rows * sizeof(float2)) != hipSuccess ||
      hipMalloc((void**)&c->flag, sizeof(int32_t)) != hipSuccess ||
      hipMalloc((void**)&c->seq_splits, 2 * 64 * sizeof(int32_t)) != hipSuccess) {
    (void)hipGetLastError();
    free_ctx(c);
    return KVSHOT_ERR_OUT_OF_MEMORY;
  }
  if (hipMemcpy(c->rope, tab.data(), nrope * sizeof(float2), hipMemcpyHostToDevice) != hipSuccess) {
    free_ctx(c);
    return KVSHOT_ERR_DEVICE;
  }
  // the no-allocation call's scratch address on this device (resolved once per device)
  const kvshot_status sst = resolve_scratch(c->device);
  if (sst != KVSHOT_OK) {
    free_ctx(c);
    return sst;
  }
  *out = c;
  return KVSHOT_OK;
}

kvshot_status kvshot_draft_attn_destroy(kvshot_handle h) {
  free_ctx(h);
  return KVSHOT_OK;
}

kvshot_status kvshot_draft_attn_step(kvshot_handle h, int32_t batch, int32_t n_new, int32_t max_ctx_len_hint,
                                     const void* q, const void* k_pages, const void* v_pages,
                                     const int32_t* page_table, const int32_t* ctx_lens, const void* draft_k,
                                     const void* draft_v, const int32_t* step_offsets, void* out, float* lse,
                                     void* stream) {
  kvshot_call a{};
  a.mode = KVSHOT_MODE_STEP;
  a.batch = batch;
  a.n_queries = n_new;
  a.max_ctx_len_hint = max_ctx_len_hint;
  a.q = q;
  a.k_pages = k_pages;
  a.v_pages = v_pages;
  a.page_table = page_table;
  a.ctx_lens = ctx_lens;
  a.draft_k = draft_k;
  a.draft_v = draft_v;
  a.step_offsets = step_offsets;
  a.out = out;
  a.lse = lse;
  return run_call(h, a, stream);
}

kvshot_status kvshot_draft_attn_tree(kvshot_handle h, int32_t batch, int32_t n_nodes, int32_t max_ctx_len_hint,
                                     const void* q, const void* k_pages, const void* v_pages,
                                     const int32_t* page_table, const int32_t* ctx_lens, const void* draft_k,
                                     const void* draft_v, const int32_t* parents, void* out, float* lse,
                                     void* stream) {
  kvshot_call a{};
  a.mode = KVSHOT_MODE_TREE;
  a.batch = batch;
  a.n_queries = n_nodes;
  a.n_nodes = n_nodes;
  a.max_ctx_len_hint = max_ctx_len_hint;
  a.q = q;
  a.k_pages = k_pages;
  a.v_pages = v_pages;
  a.page_table = page_table;
  a.ctx_lens = ctx_lens;
  a.draft_k = draft_k;
  a.draft_v = draft_v;
  a.parents = parents;
  a.out = out;
  a.lse = lse;
  return run_call(h, a, stream);
}

kvshot_status kvshot_draft_attn_call_noalloc(kvshot_handle h, const kvshot_call* call, void* stream) {
  if (!h || !call) return KVSHOT_ERR_INVALID_ARG;
  const kvshot_call& a = *call;
  if (a.batch < 1 || a.batch > h->cfg.max_batch || a.n_queries < 1 || a.n_queries > h->cfg.max_draft ||
      a.max_ctx_len_hint < 0)
    return KVSHOT_ERR_INVALID_ARG;
  void* base = scratch_ptr(h->device);
  if (!base) return KVSHOT_ERR_DEVICE;
  // the same plan as kvshot_draft_attn_call, so both return the same bits
  const Plan pl = make_plan(h, a.batch, a.n_queries, a.max_ctx_len_hint);
  size_t ml_off = 0, seq_off = 0;
  if (partial_bytes(h, pl, a.batch, &ml_off, &seq_off) > kScratchBytes) return KVSHOT_ERR_SCRATCH;
  Workspace ws;
  ws.part_o = (float*)base;
  ws.part_ml = (float2*)((unsigned char*)base + ml_off);
  ws.seq_splits = (int32_t*)((unsigned char*)base + seq_off);
  ws.profile = false;
  return run_call(h, a, stream, &ws);
}


kvshot_status kvshot_draft_attn_call(kvshot_handle h, const kvshot_call* call, void* stream) {
  if (!call) return KVSHOT_ERR_INVALID_ARG;
  return run_call(h, *call, stream);
}

kvshot_status kvshot_draft_attn_validate(kvshot_handle h, int32_t batch, int32_t n_queries, int32_t max_ctx_len_hint,
                                         const int32_t* page_table, const int32_t* ctx_lens,
                                         const int32_t* step_offsets, const int32_t* parents, int32_t* first_bad,
                                         void* stream) {
  kvshot_call a{};
  a.mode = parents ? KVSHOT_MODE_TREE : KVSHOT_MODE_STEP;
  a.batch = batch;
  a.n_queries = n_queries;
  a.n_nodes = n_queries;
  a.max_ctx_len_hint = max_ctx_len_hint;
  a.page_table = page_table;
  a.ctx_lens = ctx_lens;
  a.step_offsets = step_offsets;
  a.parents = parents;
  return validate_impl(h, a, first_bad, stream);
}

kvshot_status kvshot_draft_attn_validate_call(kvshot_handle h, const kvshot_call* call, int32_t* first_bad,
                                              void* stream) {
  if (first_bad) *first_bad = 0;
  if (!call) return KVSHOT_ERR_INVALID_ARG;
  return validate_impl(h, *call, first_bad, stream);
}

kvshot_status kvshot_draft_attn_set_option(kvshot_handle h, int32_t option, int64_t value) {
  if (!h) return KVSHOT_ERR_INVALID_ARG;
  switch (option) {
    case KVSHOT_OPT_SPLITS:
      if (value < 0 || value > kMaxSplits) return KVSHOT_ERR_INVALID_ARG;
      h->opt_splits = (int)value;
      return KVSHOT_OK;
    case KVSHOT_OPT_PATH:
      if (value < 0 || value > 3) return KVSHOT_ERR_INVALID_ARG;
      if ((value == 1 || value == 3) && h->cfg.dtype != KVSHOT_BF16) return KVSHOT_ERR_UNSUPPORTED;
      h->opt_path = (int)value;
      return KVSHOT_OK;
    case KVSHOT_OPT_PROFILE:
      if (value != 0 && value != 1) return KVSHOT_ERR_INVALID_ARG;
      if (value && h->prof.empty()) {
        const DeviceGuard dg(h->device);
        if (!dg.ok()) return KVSHOT_ERR_DEVICE;
        h->prof.resize(kProfileRing);
        for (auto& s : h->prof) {
          for (auto& e : s.ev) {
            e = nullptr;
            if (hipEventCreate(&e) != hipSuccess) return KVSHOT_ERR_DEVICE;
          }
          s.has_combine = 0;
        }
      }
      h->opt_profile = (int)value;
      return KVSHOT_OK;
    default:
      return KVSHOT_ERR_INVALID_ARG;
  }
}

kvshot_status kvshot_draft_attn_plan(kvshot_handle h, int32_t batch, int32_t n_queries, int32_t max_ctx_len_hint,
                                     int32_t* splits, int32_t* path, int32_t* row_tiles, int32_t* workgroups) {
  if (!h || batch < 1 || batch > h->cfg.max_batch || n_queries < 1 || n_queries > h->cfg.max_draft ||
      max_ctx_len_hint < 0)
    return KVSHOT_ERR_INVALID_ARG;
  const Plan pl = make_plan(h, batch, n_queries, max_ctx_len_hint);
  if (splits) *splits = pl.splits;
  if (path) *path = pl.path;
  if (row_tiles) *row_tiles = pl.row_tiles;
  if (workgroups)
    *workgroups = pl.balanced ? pl.items * pl.row_groups * h->cfg.num_kv_heads
                              : pl.splits * pl.row_groups * h->cfg.num_kv_heads * batch;
  return KVSHOT_OK;
}

kvshot_status kvshot_draft_attn_profile_read(kvshot_handle h, double* attn_ms, double* combine_ms, int64_t* calls) {
  if (!h) return KVSHOT_ERR_INVALID_ARG;
  const DeviceGuard dg(h->device);
  if (!dg.ok()) return KVSHOT_ERR_DEVICE;
  kvshot_status st = drain_profile(h, true);
  if (st != KVSHOT_OK) return st;
  if (attn_ms) *attn_ms = h->attn_ms;
  if (combine_ms) *combine_ms = h->combine_ms;
  if (calls) *calls = h->calls;
  h->attn_ms = h->combine_ms = 0.0;
  h->calls = 0;
  return KVSHOT_OK;
}

kvshot_status kvshot_debug_gather_kv(kvshot_handle h, int32_t batch, int32_t max_ctx, const void* k_pages,
                                     const void* v_pages, const int32_t* page_table, const int32_t* ctx_lens,
                                     void* k_dense, void* v_dense, void* stream) {
  if (!h || !k_pages || !v_pages || !page_table || !ctx_lens || !k_dense || !v_dense) return KVSHOT_ERR_INVALID_ARG;
  if (batch < 1 || batch > h->cfg.max_batch || max_ctx < 1) return KVSHOT_ERR_INVALID_ARG;
  if (!aligned16(k_pages) || !aligned16(v_pages) || !aligned16(k_dense) || !aligned16(v_dense))
    return KVSHOT_ERR_INVALID_ARG;
  const DeviceGuard dg(h->device);
  if (!dg.ok()) return KVSHOT_ERR_DEVICE;
  kvshot_status st = KVSHOT_OK;
  const Plan pl = make_plan(h, batch, 1, 0);
  AttnParams p;
  fill_params(h, pl, batch, 1, max_ctx, p);
  p.k_pages = k_pages;
  p.v_pages = v_pages;
  p.page_table = page_table;
  p.ctx_lens = ctx_lens;
  if (launch_gather_kv(p, max_ctx, k_dense, v_dense, h->cfg.dtype == KVSHOT_BF16, (hipStream_t)stream) != hipSuccess)
    return KVSHOT_ERR_DEVICE;
  return KVSHOT_OK;
}

kvshot_status kvshot_debug_tree_mask(kvshot_handle h, int32_t batch, int32_t n_nodes, const int32_t* parents,
                                     uint64_t* anc_out, int32_t* depth_out, void* stream) {
  if (!h || !parents || !anc_out || !depth_out) return KVSHOT_ERR_INVALID_ARG;
  if (batch < 1 || batch > h->cfg.max_batch || n_nodes < 1 || n_nodes > kMaxDraft) return KVSHOT_ERR_INVALID_ARG;
  const DeviceGuard dg(h->device);
  if (!dg.ok()) return KVSHOT_ERR_DEVICE;
  kvshot_status st = KVSHOT_OK;
  if (launch_tree_mask(parents, batch, n_nodes, anc_out, depth_out, (hipStream_t)stream) != hipSuccess)
    return KVSHOT_ERR_DEVICE;
  return KVSHOT_OK;
}

kvshot_status kvshot_debug_stream_read(const void* src, int64_t bytes, void* sink, int32_t sink_words,
                                       void* stream) {
  if (!src || !sink || bytes < 16 || sink_words < 1 || !aligned16(src) || !aligned16(sink))
    return KVSHOT_ERR_INVALID_ARG;
  if (launch_stream_read(src, bytes, sink, sink_words, (hipStream_t)stream) != hipSuccess) return KVSHOT_ERR_DEVICE;
  return KVSHOT_OK;
}

kvshot_status kvshot_debug_mfma_rate(int32_t workgroups, int32_t iters, void* sink, void* stream) {
  if (workgroups < 1 || iters < 1 || !sink || !aligned16(sink)) return KVSHOT_ERR_INVALID_ARG;
  if (launch_mfma_rate(workgroups, iters, sink, (hipStream_t)stream) != hipSuccess) return KVSHOT_ERR_DEVICE;
  return KVSHOT_OK;
}

}  // extern "C"
