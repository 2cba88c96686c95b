// Host side of the projected-KV cache builder ABI (include/kvshot_kvproj.h):
// argument validation, the RoPE table, the split plan, the partial workspace
// and kernel launches.  No call here synchronises the host except destroy,
// validate and profile_read.
#include "kvshot_kvproj.h"

#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>
#include <new>
#include <vector>

#include "device_guard.h"
#include "kvproj_common.h"

using namespace kvshot;

namespace {
constexpr int kProjProfileRing = 1024;
struct ProjProfileSlot {
  hipEvent_t ev[3];
  int has_combine;
};
}  // namespace

struct kvshot_kvproj_ctx {
  kvshot_kvproj_config cfg;
  int device = 0, num_cus = 256, page_shift = 0;
  float2* rope = nullptr;
  double* rope_rev = nullptr;
  float* part = nullptr;
  size_t ws_rows = 0;           // capacity of the partial workspace in (split, token) rows of 2 d_kv floats
  int32_t* flag = nullptr;
  int opt_splits = 0, opt_profile = 0, opt_path = 0;
  std::vector<ProjProfileSlot> prof;
  int64_t prof_head = 0, prof_tail = 0;
  double main_ms = 0.0, combine_ms = 0.0;
  int64_t calls = 0;
};

namespace {

bool is_pow2(int v) { return v > 0 && (v & (v - 1)) == 0; }
bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

int m_tiles_of(const kvshot_kvproj_ctx* c) { return (c->cfg.num_kv_heads + 1) / 2; }
int n_tiles_of(int n_tokens) { return (n_tokens + kProjTile - 1) / kProjTile; }
int chunks_of(const kvshot_kvproj_ctx* c) { return c->cfg.num_layers * c->cfg.num_kv_heads * kHeadDim / 64; }

// Reduction splits: enough workgroups to give every CU one (one workgroup
// fills a CU's LDS), at most 16 and at most one chunk per split, capped by
// the workspace.  Large calls (a grid of >= one workgroup per CU) do not split.
int plan_splits(const kvshot_kvproj_ctx* c, int n_tokens) {
  const int64_t tiles = 2ll * m_tiles_of(c) * n_tiles_of(n_tokens);
  int s = 1;
  if (c->opt_splits > 0) {
    s = c->opt_splits;
  } else if (tiles < c->num_cus) {
    s = (int)(c->num_cus / tiles);
    if (s > kProjMaxSplits) s = kProjMaxSplits;
  }
  if (s > chunks_of(c)) s = chunks_of(c);
  while (s > 1 && (size_t)s * n_tokens > c->ws_rows) --s;
  return s < 1 ? 1 : s;
}

// Plan of a call.  Path 1 is the tiled kernel (256 channels x 256 tokens per
// workgroup, split reductions when that grid is below one workgroup per CU);
// path 2 the direct kernel (64 channels x 16 tile16 tokens per workgroup, the
// whole reduction in one workgroup, no partial sums).  The direct tile height
// minimises the operand bytes of the busiest CU: ceil(workgroups / CUs) x
// (64 + 16 tile16) rows of the reduction.  The automatic choice compares two
// estimates fitted to MI355X timings (Hkv 4 to 16, 64 to 16384 tokens): a
// direct round costs about 4 us plus its operand rows at 60 GB/s per CU (one
// workgroup per CU), a tiled round 6 us plus 512 rows at 32 GB/s per CU, and
// split partials are written and read back at about 5 TB/s plus 2 us.
struct ProjPlan {
  int path = 1, splits = 1, tile16 = 0, tiles = 0, workgroups = 0;
};

ProjPlan direct_plan(const kvshot_kvproj_ctx* c, int n_tokens, double* est_us) {
  ProjPlan pl;
  pl.path = 2;
  const int64_t slices = 4ll * c->cfg.num_kv_heads;   // (tensor, head, half)
  const double row_bytes = 2.0 * c->cfg.num_layers * c->cfg.num_kv_heads * kHeadDim;
  double best = -1.0;
  for (int tb = 1; tb <= kProjDirectMaxTile16; ++tb) {
    const int64_t tiles = (n_tokens + 16 * tb - 1) / (16 * tb);
    const int64_t wgs = slices * tiles;
    const int64_t rounds = (wgs + c->num_cus - 1) / c->num_cus;
    const double us = (double)rounds * (4.0 + (64 + 16 * tb) * row_bytes / 60e3);
    if (best < 0 || us < best) {
      best = us;
      pl.tile16 = tb;
      pl.tiles = (int)tiles;
      pl.workgroups = (int)wgs;
    }
  }
  *est_us = best;
  return pl;
}

ProjPlan tiled_plan(const kvshot_kvproj_ctx* c, int n_tokens, double* est_us) {
  ProjPlan pl;
  pl.path = 1;
  pl.splits = plan_splits(c, n_tokens);
  pl.tiles = n_tiles_of(n_tokens);
  pl.workgroups = 2 * m_tiles_of(c) * pl.tiles * pl.splits;
  const double row_bytes = 2.0 * c->cfg.num_layers * c->cfg.num_kv_heads * kHeadDim / pl.splits;
  const int64_t rounds = (pl.workgroups + c->num_cus - 1) / c->num_cus;
  double us = (double)rounds * (6.0 + 512 * row_bytes / 32e3);
  if (pl.splits > 1)
    us += 2.0 + 2.0 * pl.splits * (double)n_tokens * 2 * c->cfg.num_kv_heads * kHeadDim * 4 / 5e6;
  *est_us = us;
  return pl;
}

ProjPlan make_plan(const kvshot_kvproj_ctx* c, int n_tokens) {
  double td = 0.0, tt = 0.0;
  const ProjPlan d = direct_plan(c, n_tokens, &td);
  const ProjPlan t = tiled_plan(c, n_tokens, &tt);
  if (c->opt_path == 2) return d;
  if (c->opt_path == 1 || c->opt_splits > 0) return t;
  return td < tt ? d : t;
}

void free_proj(kvshot_kvproj_ctx* c) {
  if (!c) return;
  {
    const DeviceGuard dg(c->device);
    (void)hipDeviceSynchronize();
    for (auto& s : c->prof)
      for (auto& e : s.ev)
        if (e) (void)hipEventDestroy(e);
    if (c->rope) (void)hipFree(c->rope);
    if (c->rope_rev) (void)hipFree(c->rope_rev);
    if (c->part) (void)hipFree(c->part);
    if (c->flag) (void)hipFree(c->flag);
  }
  delete c;
}

kvshot_status drain_profile(kvshot_kvproj_ctx* c, bool all) {
  while (c->prof_tail < c->prof_head) {
    ProjProfileSlot& s = c->prof[c->prof_tail % kProjProfileRing];
    if (!all && hipEventQuery(s.ev[2]) != hipSuccess) break;
    if (hipEventSynchronize(s.ev[2]) != hipSuccess) return KVSHOT_ERR_DEVICE;
    float a = 0.f, b = 0.f;
    if (hipEventElapsedTime(&a, s.ev[0], s.ev[1]) != hipSuccess) return KVSHOT_ERR_DEVICE;
    if (s.has_combine && hipEventElapsedTime(&b, s.ev[1], s.ev[2]) != hipSuccess) return KVSHOT_ERR_DEVICE;
    c->main_ms += a;
    c->combine_ms += b;
    c->calls += 1;
    ++c->prof_tail;
  }
  return KVSHOT_OK;
}

// Fills the parameters shared by the call and validate; checks sizes and the table pointers.
kvshot_status base_params(const kvshot_kvproj_ctx* c, int32_t n_tokens, int32_t batch, const int32_t* page_table,
                          const int32_t* token_seq, const int32_t* token_pos, const int32_t* dst_page_table,
                          KvProjParams* out) {
  if (n_tokens < 1 || n_tokens > c->cfg.max_tokens || batch < 1) return KVSHOT_ERR_INVALID_ARG;
  if (!page_table || !token_seq || !token_pos) return KVSHOT_ERR_INVALID_ARG;
  KvProjParams& p = *out;
  p = KvProjParams{};
  const kvshot_kvproj_config& g = c->cfg;
  p.page_table = page_table;
  p.dst_page_table = dst_page_table ? dst_page_table : page_table;
  p.token_seq = token_seq;
  p.token_pos = token_pos;
  p.rope = c->rope;
  p.rope_rev = c->rope_rev;
  p.part = c->part;
  p.page_stride = g.page_stride;
  p.head_stride = g.head_stride;
  p.slot_stride = g.slot_stride;
  p.dst_page_stride = g.dst_page_stride;
  p.dst_head_stride = g.dst_head_stride;
  p.dst_slot_stride = g.dst_slot_stride;
  p.n_tokens = n_tokens;
  p.batch = batch;
  p.hkv = g.num_kv_heads;
  p.layers = g.num_layers;
  p.page_shift = c->page_shift;
  p.max_pages_per_seq = g.max_pages_per_seq;
  p.num_pages = g.num_pages;
  p.dst_num_pages = g.dst_num_pages;
  p.max_position = (int32_t)g.max_position;
  p.m_tiles = m_tiles_of(c);
  p.n_tiles = n_tiles_of(n_tokens);
  return KVSHOT_OK;
}

}  // namespace

extern "C" {

kvshot_status kvshot_kvproj_init(const kvshot_kvproj_config* cfg, kvshot_kvproj_handle* out) {
  if (!cfg || !out) return KVSHOT_ERR_INVALID_ARG;
  *out = nullptr;
  kvshot_kvproj_config g = *cfg;
  if (g.head_dim != kHeadDim) return KVSHOT_ERR_UNSUPPORTED;
  if (g.num_kv_heads < 1 || g.num_kv_heads > 16) return KVSHOT_ERR_INVALID_ARG;
  if (g.num_layers < 1 || g.num_layers > kProjMaxLayers) return KVSHOT_ERR_INVALID_ARG;
  if (!is_pow2(g.page_size) || g.page_size < 16 || g.page_size > 256) return KVSHOT_ERR_INVALID_ARG;
  if (g.max_pages_per_seq < 1 || g.num_pages < 1 || g.dst_num_pages < 1) return KVSHOT_ERR_INVALID_ARG;
  if ((int64_t)g.max_pages_per_seq * g.page_size > (1ll << 30)) return KVSHOT_ERR_INVALID_ARG;
  if (g.max_tokens < 1 || g.max_tokens > (1 << 26)) return KVSHOT_ERR_INVALID_ARG;
  if (g.max_position < 1 || g.max_position > (1ll << 24)) return KVSHOT_ERR_INVALID_ARG;
  if (!(g.rope_theta > 0.0) || !std::isfinite(g.rope_theta)) return KVSHOT_ERR_INVALID_ARG;
  const int64_t dense_page = (int64_t)g.num_kv_heads * g.page_size * kHeadDim;
  if (g.page_stride == 0) g.page_stride = dense_page;
  if (g.head_stride == 0) g.head_stride = (int64_t)g.page_size * kHeadDim;
  if (g.slot_stride == 0) g.slot_stride = kHeadDim;
  if (g.dst_page_stride == 0) g.dst_page_stride = dense_page;
  if (g.dst_head_stride == 0) g.dst_head_stride = (int64_t)g.page_size * kHeadDim;
  if (g.dst_slot_stride == 0) g.dst_slot_stride = kHeadDim;
  const int64_t strides[6] = {g.page_stride, g.head_stride, g.slot_stride,
                              g.dst_page_stride, g.dst_head_stride, g.dst_slot_stride};
  for (int64_t s : strides)
    if (s < 0 || s % 8) return KVSHOT_ERR_INVALID_ARG;
  if (g.slot_stride < kHeadDim || g.dst_slot_stride < kHeadDim) return KVSHOT_ERR_INVALID_ARG;

  kvshot_kvproj_ctx* c = new (std::nothrow) kvshot_kvproj_ctx();
  if (!c) return KVSHOT_ERR_OUT_OF_MEMORY;
  c->cfg = g;
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
  const int64_t rows = (int64_t)kProjMaxSplits * g.max_tokens;
  c->ws_rows = (size_t)(rows < kProjWorkspaceRows ? rows : kProjWorkspaceRows);
  const size_t d_kv = (size_t)g.num_kv_heads * kHeadDim;

  // RoPE table: angle p * theta^(-2m/D) in float64, cos/sin rounded to float32
  const size_t nrope = (size_t)g.max_position * kHalfDim;
  std::vector<float2> tab(nrope);
  for (int64_t pos = 0; pos < g.max_position; ++pos)
    for (int m = 0; m < kHalfDim; ++m) {
      const double a = (double)pos * std::pow(g.rope_theta, -2.0 * m / (double)kHeadDim);
      tab[(size_t)pos * kHalfDim + m] = make_float2((float)std::cos(a), (float)std::sin(a));
    }
  // the same angles in revolutions per position, for the fused kernel's own range reduction
  double rev[kHalfDim];
  for (int m = 0; m < kHalfDim; ++m)
    rev[m] = std::pow(g.rope_theta, -2.0 * m / (double)kHeadDim) / (2.0 * 3.14159265358979323846);
  if (hipMalloc((void**)&c->rope, nrope * sizeof(float2)) != hipSuccess ||
      hipMalloc((void**)&c->rope_rev, sizeof(rev)) != hipSuccess ||
      hipMalloc((void**)&c->part, c->ws_rows * 2 * d_kv * sizeof(float)) != hipSuccess ||
      hipMalloc((void**)&c->flag, sizeof(int32_t)) != hipSuccess) {
    (void)hipGetLastError();
    free_proj(c);
    return KVSHOT_ERR_OUT_OF_MEMORY;
  }
  if (hipMemcpy(c->rope, tab.data(), nrope * sizeof(float2), hipMemcpyHostToDevice) != hipSuccess ||
      hipMemcpy(c->rope_rev, rev, sizeof(rev), hipMemcpyHostToDevice) != hipSuccess) {
    free_proj(c);
    return KVSHOT_ERR_DEVICE;
  }
  *out = c;
  return KVSHOT_OK;
}

kvshot_status kvshot_kvproj_destroy(kvshot_kvproj_handle h) {
  free_proj(h);
  return KVSHOT_OK;
}

kvshot_status kvshot_kv_project(kvshot_kvproj_handle h, int32_t n_tokens, int32_t batch, const void* const* k_src,
                                const void* const* v_src, const int32_t* page_table, const int32_t* token_seq,
                                const int32_t* token_pos, const void* w_k, const void* w_v, void* k_dst,
                                void* v_dst, const int32_t* dst_page_table, int32_t flags, void* stream) {
  if (!h) return KVSHOT_ERR_INVALID_ARG;
  if (flags & ~KVSHOT_KVPROJ_ROPE) return KVSHOT_ERR_INVALID_ARG;
  KvProjParams p;
  const kvshot_status st = base_params(h, n_tokens, batch, page_table, token_seq, token_pos, dst_page_table, &p);
  if (st != KVSHOT_OK) return st;
  if (!k_src || !v_src || !w_k || !w_v || !k_dst || !v_dst) return KVSHOT_ERR_INVALID_ARG;
  for (int l = 0; l < h->cfg.num_layers; ++l) {
    if (!k_src[l] || !v_src[l] || !aligned16(k_src[l]) || !aligned16(v_src[l])) return KVSHOT_ERR_INVALID_ARG;
    p.k_src[l] = (const uint16_t*)k_src[l];
    p.v_src[l] = (const uint16_t*)v_src[l];
  }
  for (int l = h->cfg.num_layers; l < kProjMaxLayers; ++l) {
    p.k_src[l] = p.k_src[0];
    p.v_src[l] = p.v_src[0];
  }
  if (!aligned16(w_k) || !aligned16(w_v) || !aligned16(k_dst) || !aligned16(v_dst)) return KVSHOT_ERR_INVALID_ARG;
  const DeviceGuard dg(h->device);
  if (!dg.ok()) return KVSHOT_ERR_DEVICE;
  p.w_k = (const uint16_t*)w_k;
  p.w_v = (const uint16_t*)w_v;
  p.k_dst = (uint16_t*)k_dst;
  p.v_dst = (uint16_t*)v_dst;
  p.rope_keys = (flags & KVSHOT_KVPROJ_ROPE) ? 1 : 0;
  const ProjPlan pl = make_plan(h, n_tokens);
  p.splits = pl.splits;
  p.n_tiles = pl.tiles;
  p.tile16 = pl.tile16;
  p.work_items = pl.workgroups;
  hipStream_t s = (hipStream_t)stream;

  ProjProfileSlot* slot = nullptr;
  if (h->opt_profile) {
    if (drain_profile(h, false) != KVSHOT_OK) return KVSHOT_ERR_DEVICE;
    if (h->prof_head - h->prof_tail >= kProjProfileRing && drain_profile(h, true) != KVSHOT_OK)
      return KVSHOT_ERR_DEVICE;
    slot = &h->prof[h->prof_head % kProjProfileRing];
    slot->has_combine = p.splits > 1;
    if (hipEventRecord(slot->ev[0], s) != hipSuccess) return KVSHOT_ERR_DEVICE;
  }
  if ((pl.path == 2 ? launch_kvproj_direct(p, s) : launch_kvproj(p, s)) != hipSuccess) return KVSHOT_ERR_DEVICE;
  if (slot && hipEventRecord(slot->ev[1], s) != hipSuccess) return KVSHOT_ERR_DEVICE;
  if (p.splits > 1 && launch_kvproj_combine(p, s) != hipSuccess) return KVSHOT_ERR_DEVICE;
  if (slot) {
    if (hipEventRecord(slot->ev[2], s) != hipSuccess) return KVSHOT_ERR_DEVICE;
    ++h->prof_head;
  }
  return KVSHOT_OK;
}

kvshot_status kvshot_kv_project_validate(kvshot_kvproj_handle h, int32_t n_tokens, int32_t batch,
                                         const int32_t* page_table, const int32_t* token_seq,
                                         const int32_t* token_pos, const int32_t* dst_page_table,
                                         int32_t* bad_token, int32_t* bad_code, void* stream) {
  if (!h) return KVSHOT_ERR_INVALID_ARG;
  KvProjParams p;
  const kvshot_status st = base_params(h, n_tokens, batch, page_table, token_seq, token_pos, dst_page_table, &p);
  if (st != KVSHOT_OK) return st;
  const DeviceGuard dg(h->device);
  if (!dg.ok()) return KVSHOT_ERR_DEVICE;
  hipStream_t s = (hipStream_t)stream;
  if (launch_kvproj_validate(p, h->flag, s) != hipSuccess) return KVSHOT_ERR_DEVICE;
  int32_t v = 0;
  if (hipMemcpyAsync(&v, h->flag, sizeof(v), hipMemcpyDeviceToHost, s) != hipSuccess ||
      hipStreamSynchronize(s) != hipSuccess)
    return KVSHOT_ERR_DEVICE;
  if (v == 0x7fffffff) {
    if (bad_token) *bad_token = -1;
    if (bad_code) *bad_code = 0;
    return KVSHOT_OK;
  }
  if (bad_token) *bad_token = v / 8;
  if (bad_code) *bad_code = v % 8;
  return KVSHOT_ERR_DATA;
}

kvshot_status kvshot_kvproj_set_option(kvshot_kvproj_handle h, int32_t option, int64_t value) {
  if (!h) return KVSHOT_ERR_INVALID_ARG;
  switch (option) {
    case KVSHOT_OPT_SPLITS:
      if (value < 0 || value > kProjMaxSplits) return KVSHOT_ERR_INVALID_ARG;
      h->opt_splits = (int)value;
      return KVSHOT_OK;
    case KVSHOT_OPT_PATH:
      if (value < 0 || value > 2) return KVSHOT_ERR_INVALID_ARG;
      h->opt_path = (int)value;
      return KVSHOT_OK;
    case KVSHOT_OPT_PROFILE:
      if (value != 0 && value != 1) return KVSHOT_ERR_INVALID_ARG;
      if (value && h->prof.empty()) {
        const DeviceGuard dg(h->device);
        if (!dg.ok()) return KVSHOT_ERR_DEVICE;
        h->prof.resize(kProjProfileRing);
        for (auto& sl : h->prof) {
          for (auto& e : sl.ev) {
            e = nullptr;
            if (hipEventCreate(&e) != hipSuccess) return KVSHOT_ERR_DEVICE;
          }
          sl.has_combine = 0;
        }
      }
      h->opt_profile = (int)value;
      return KVSHOT_OK;
    default:
      return KVSHOT_ERR_INVALID_ARG;
  }
}

kvshot_status kvshot_kvproj_plan(kvshot_kvproj_handle h, int32_t n_tokens, int32_t* splits, int32_t* path,
                                 int32_t* tile_tokens, int32_t* workgroups) {
  if (!h || n_tokens < 1 || n_tokens > h->cfg.max_tokens) return KVSHOT_ERR_INVALID_ARG;
  const ProjPlan pl = make_plan(h, n_tokens);
  if (splits) *splits = pl.splits;
  if (path) *path = pl.path;
  if (tile_tokens) *tile_tokens = pl.path == 2 ? 16 * pl.tile16 : kProjTile;
  if (workgroups) *workgroups = pl.workgroups;
  return KVSHOT_OK;
}

kvshot_status kvshot_kvproj_profile_read(kvshot_kvproj_handle h, double* main_ms, double* combine_ms,
                                         int64_t* calls) {
  if (!h) return KVSHOT_ERR_INVALID_ARG;
  const DeviceGuard dg(h->device);
  if (!dg.ok()) return KVSHOT_ERR_DEVICE;
  const kvshot_status st = drain_profile(h, true);
  if (st != KVSHOT_OK) return st;
  if (main_ms) *main_ms = h->main_ms;
  if (combine_ms) *combine_ms = h->combine_ms;
  if (calls) *calls = h->calls;
  h->main_ms = h->combine_ms = 0.0;
  h->calls = 0;
  return KVSHOT_OK;
}

}  // extern "C"
