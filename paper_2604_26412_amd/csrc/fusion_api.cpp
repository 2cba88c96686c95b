// Host side of the gated delta fusion ABI (include/kvshot_fusion.h): argument
// validation, the split plan, the partial workspace and kernel launches.  No
// call here synchronises the host except destroy and profile_read.
#include "kvshot_fusion.h"

#include <hip/hip_runtime.h>

#include <cstdint>
#include <new>
#include <vector>

#include "device_guard.h"
#include "fusion_common.h"

using namespace kvshot;

namespace {
constexpr int kFusionProfileRing = 1024;
struct FusionProfileSlot {
  hipEvent_t ev[3];
  int has_combine;
};
}  // namespace

struct kvshot_fusion_ctx {
  int d = 0, max_tokens = 0, device = 0, num_cus = 256;
  float* part = nullptr;
  size_t ws_pairs = 0;          // capacity of the partial workspace in (gate, delta) pairs of floats
  int opt_splits = 0, opt_profile = 0, opt_tile = 0;
  std::vector<FusionProfileSlot> prof;
  int64_t prof_head = 0, prof_tail = 0;
  double main_ms = 0.0, combine_ms = 0.0;
  int64_t calls = 0;
};

namespace {

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

int m_tiles_of(int tokens, int tile = kFusionTokens) { return (tokens + tile - 1) / tile; }

// Automatic plans consider 128-token tiles from this many tokens.
constexpr int kFusionBigTileMin = 128;

// The plan of a call: token tile, reduction splits and how a split divides the
// reduction space.
//  - 64-token tiles: the largest power of two (<= 8) that keeps the grid within
//    two workgroups per CU (two resident workgroups hide each other's
//    per-chunk latency: d = 4096, graph replay, 128 tokens 62 -> 50 us with 8
//    splits instead of 4, 480 tokens 121 -> 107 us with 2 instead of 1, other
//    sizes unchanged); splits take segments first (2: segments {0, 1} and
//    {2, 3}; 4: one each), then halves of a segment (8).  16 splits measured
//    slower: the larger partial sum costs more in the combine than the main
//    kernel gains.
//  - 128-token tiles: each weight chunk is read from L2 half as often.  The
//    largest power of two (<= 4) that keeps the grid within one workgroup per
//    CU (a 128-token workgroup holds a CU's registers); a split takes a part of
//    the reduction index range of all four segments, so it reads only that
//    part of n and o.  Automatic plans take them from kFusionBigTileMin tokens
//    on.  Measured at d = 4096 (main kernel + combine, graph replay, 64 ->
//    128-token tiles): 128 tokens 53 -> 46 us, 192 tokens 71 -> 52 us, 256
//    tokens 75 -> 53 us, 384 tokens 98 -> 71 us, 480 tokens 109 -> 83 us, 640
//    tokens 150 -> 120 us, 1024 tokens 172 -> 154 us.
// Both capped by the workspace.
struct FusionPlan {
  int tile = kFusionTokens, splits = 1, kparts = 1, m_tiles = 0;
};

FusionPlan plan_tile(const kvshot_fusion_ctx* c, int tokens, int tile) {
  FusionPlan pl;
  const int64_t ntl = c->d / kFusionChannels;
  pl.tile = tile;
  pl.m_tiles = m_tiles_of(tokens, tile);
  const int64_t tiles = (int64_t)pl.m_tiles * ntl;
  int s = 1;
  if (c->opt_splits > 0) s = c->opt_splits;
  else if (tile == 128)
    while (s < 4 && tiles * s * 2 <= (int64_t)c->num_cus) s *= 2;
  else
    while (s < 8 && tiles * s * 2 <= 2 * (int64_t)c->num_cus) s *= 2;
  while (s > 1 && (size_t)s * tokens * c->d > c->ws_pairs) s /= 2;
  pl.splits = s;
  pl.kparts = tile == 128 ? s : (s > 4 ? s / 4 : 1);
  return pl;
}

FusionPlan make_plan(const kvshot_fusion_ctx* c, int tokens) {
  const FusionPlan small = plan_tile(c, tokens, kFusionTokens);
  if (c->opt_tile == 1 || c->opt_splits > 4) return small;
  const FusionPlan big = plan_tile(c, tokens, 128);
  if (c->opt_tile == 2) return big;
  return c->opt_splits > 0 || tokens < kFusionBigTileMin ? small : big;
}

void free_fusion(kvshot_fusion_ctx* c) {
  if (!c) return;
  {
    const DeviceGuard dg(c->device);
    (void)hipDeviceSynchronize();
    for (auto& s : c->prof)
      for (auto& e : s.ev)
        if (e) (void)hipEventDestroy(e);
    if (c->part) (void)hipFree(c->part);
  }
  delete c;
}

kvshot_status drain_profile(kvshot_fusion_ctx* c, bool all) {
  while (c->prof_tail < c->prof_head) {
    FusionProfileSlot& s = c->prof[c->prof_tail % kFusionProfileRing];
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

kvshot_status run_fusion(kvshot_fusion_handle h, int32_t tokens, const void* n, const void* o, const void* w_g,
                         const void* w_delta, const void* packed, const float* b_g, void* h_out, float* g_out,
                         int32_t flags, void* stream) {
  if (!h) return KVSHOT_ERR_INVALID_ARG;
  if (flags & ~(KVSHOT_FUSION_CROSS_ONLY | KVSHOT_FUSION_OUT_FP32)) return KVSHOT_ERR_INVALID_ARG;
  const bool cross_only = (flags & KVSHOT_FUSION_CROSS_ONLY) != 0;
  if (tokens < 1 || tokens > h->max_tokens) return KVSHOT_ERR_INVALID_ARG;
  if ((!n && !cross_only) || !o || !b_g || !h_out || (!packed && (!w_g || !w_delta))) return KVSHOT_ERR_INVALID_ARG;
  if ((n && !aligned16(n)) || !aligned16(o) || !aligned16(b_g) || !aligned16(h_out) || (g_out && !aligned16(g_out)) ||
      (packed && !aligned16(packed)) || (w_g && !aligned16(w_g)) || (w_delta && !aligned16(w_delta)))
    return KVSHOT_ERR_INVALID_ARG;
  const DeviceGuard dg(h->device);
  if (!dg.ok()) return KVSHOT_ERR_DEVICE;

  FusionParams p{};
  p.n = (const uint16_t*)n;
  p.o = (const uint16_t*)o;
  p.w_g = packed ? nullptr : (const uint16_t*)w_g;
  p.b_g = b_g;
  p.w_delta = packed ? nullptr : (const uint16_t*)w_delta;
  p.w_packed = (const uint16_t*)packed;
  p.h = h_out;
  p.g_out = g_out;
  p.part = h->part;
  p.tokens = tokens;
  p.d = h->d;
  const FusionPlan pl = make_plan(h, tokens);
  p.m_tiles = pl.m_tiles;
  p.n_tiles = h->d / kFusionChannels;
  p.splits = pl.splits;
  p.kparts = pl.kparts;
  p.tile_tokens = pl.tile;
  // which partial planes each split writes: split s covers segments [seg0, seg0 + nseg)
  // (segments 0-2 feed the gate, segment 3 the delta projection)
  {
    const int nseg = 4 * pl.kparts / pl.splits;
    for (int sp = 0; sp < p.splits; ++sp) {
      const int seg0 = (sp / pl.kparts) * nseg;
      if (seg0 < 3) p.part_g_mask |= 1u << sp;
      if (seg0 + nseg > 3) p.part_d_mask |= 1u << sp;
    }
  }
  p.cross_only = cross_only ? 1 : 0;
  p.out_fp32 = (flags & KVSHOT_FUSION_OUT_FP32) ? 1 : 0;
  hipStream_t s = (hipStream_t)stream;

  FusionProfileSlot* slot = nullptr;
  if (h->opt_profile) {
    if (drain_profile(h, false) != KVSHOT_OK) return KVSHOT_ERR_DEVICE;
    if (h->prof_head - h->prof_tail >= kFusionProfileRing && drain_profile(h, true) != KVSHOT_OK)
      return KVSHOT_ERR_DEVICE;
    slot = &h->prof[h->prof_head % kFusionProfileRing];
    slot->has_combine = p.splits > 1;
    if (hipEventRecord(slot->ev[0], s) != hipSuccess) return KVSHOT_ERR_DEVICE;
  }
  if (launch_fusion(p, s) != hipSuccess) return KVSHOT_ERR_DEVICE;
  if (slot && hipEventRecord(slot->ev[1], s) != hipSuccess) return KVSHOT_ERR_DEVICE;
  if (p.splits > 1 && launch_fusion_combine(p, s) != hipSuccess) return KVSHOT_ERR_DEVICE;
  if (slot) {
    if (hipEventRecord(slot->ev[2], s) != hipSuccess) return KVSHOT_ERR_DEVICE;
    ++h->prof_head;
  }
  return KVSHOT_OK;
}

}  // namespace

extern "C" {

kvshot_status kvshot_fusion_init(int32_t d, int32_t max_tokens, kvshot_fusion_handle* out) {
  if (!out) return KVSHOT_ERR_INVALID_ARG;
  *out = nullptr;
  if (d < 256 || d % 256 != 0 || d > (1 << 16)) return KVSHOT_ERR_INVALID_ARG;
  if (max_tokens < 1 || (int64_t)max_tokens * d > (1ll << 31)) return KVSHOT_ERR_INVALID_ARG;
  kvshot_fusion_ctx* c = new (std::nothrow) kvshot_fusion_ctx();
  if (!c) return KVSHOT_ERR_OUT_OF_MEMORY;
  c->d = d;
  c->max_tokens = max_tokens;
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
  // workspace: the largest automatic plan, and at least 16 splits of one token tile
  size_t need = (size_t)kFusionMaxSplits * (max_tokens < kFusionTokens ? max_tokens : kFusionTokens) * d;
  c->ws_pairs = (size_t)-1;
  for (int m = 1; m <= m_tiles_of(max_tokens); ++m) {
    const int tokens = m * kFusionTokens < max_tokens ? m * kFusionTokens : max_tokens;
    const size_t s = (size_t)make_plan(c, tokens).splits;
    if (s > 1 && s * tokens * d > need) need = s * tokens * d;
  }
  c->ws_pairs = need;
  if (hipMalloc((void**)&c->part, need * 2 * sizeof(float)) != hipSuccess) {
    (void)hipGetLastError();
    delete c;
    return KVSHOT_ERR_OUT_OF_MEMORY;
  }
  *out = c;
  return KVSHOT_OK;
}

kvshot_status kvshot_fusion_destroy(kvshot_fusion_handle h) {
  free_fusion(h);
  return KVSHOT_OK;
}

kvshot_status kvshot_gated_delta_fusion(kvshot_fusion_handle h, int32_t tokens, const void* n, const void* o,
                                        const void* w_g, const float* b_g, const void* w_delta, void* h_out,
                                        float* g_out, int32_t flags, void* stream) {
  return run_fusion(h, tokens, n, o, w_g, w_delta, nullptr, b_g, h_out, g_out, flags, stream);
}

kvshot_status kvshot_fusion_pack_weights(kvshot_fusion_handle h, const void* w_g, const void* w_delta, void* packed,
                                         void* stream) {
  if (!h || !w_g || !w_delta || !packed) return KVSHOT_ERR_INVALID_ARG;
  if (!aligned16(w_g) || !aligned16(w_delta) || !aligned16(packed)) return KVSHOT_ERR_INVALID_ARG;
  const DeviceGuard dg(h->device);
  if (!dg.ok()) return KVSHOT_ERR_DEVICE;
  if (launch_fusion_pack((const uint16_t*)w_g, (const uint16_t*)w_delta, (uint16_t*)packed, h->d,
                         (hipStream_t)stream) != hipSuccess)
    return KVSHOT_ERR_DEVICE;
  return KVSHOT_OK;
}

kvshot_status kvshot_gated_delta_fusion_packed(kvshot_fusion_handle h, int32_t tokens, const void* n, const void* o,
                                               const void* packed, const float* b_g, void* h_out, float* g_out,
                                               int32_t flags, void* stream) {
  if (!packed) return KVSHOT_ERR_INVALID_ARG;
  return run_fusion(h, tokens, n, o, nullptr, nullptr, packed, b_g, h_out, g_out, flags, stream);
}

kvshot_status kvshot_fusion_set_option(kvshot_fusion_handle h, int32_t option, int64_t value) {
  if (!h) return KVSHOT_ERR_INVALID_ARG;
  switch (option) {
    case KVSHOT_OPT_SPLITS:
      if (value != 0 && value != 1 && value != 2 && value != 4 && value != 8 && value != 16)
        return KVSHOT_ERR_INVALID_ARG;
      h->opt_splits = (int)value;
      return KVSHOT_OK;
    case KVSHOT_OPT_PATH:
      if (value < 0 || value > 2) return KVSHOT_ERR_INVALID_ARG;
      h->opt_tile = (int)value;
      return KVSHOT_OK;
    case KVSHOT_OPT_PROFILE:
      if (value != 0 && value != 1) return KVSHOT_ERR_INVALID_ARG;
      if (value && h->prof.empty()) {
        const DeviceGuard dg(h->device);
        if (!dg.ok()) return KVSHOT_ERR_DEVICE;
        h->prof.resize(kFusionProfileRing);
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

kvshot_status kvshot_fusion_plan(kvshot_fusion_handle h, int32_t tokens, int32_t* splits, int32_t* workgroups) {
  if (!h || tokens < 1 || tokens > h->max_tokens) return KVSHOT_ERR_INVALID_ARG;
  const FusionPlan pl = make_plan(h, tokens);
  if (splits) *splits = pl.splits;
  if (workgroups) *workgroups = pl.m_tiles * (h->d / kFusionChannels) * pl.splits;
  return KVSHOT_OK;
}

kvshot_status kvshot_fusion_profile_read(kvshot_fusion_handle h, double* main_ms, double* combine_ms,
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
