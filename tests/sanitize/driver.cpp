// Drives the library's host API (attention, gated-delta fusion, projected-KV
// builder) through valid and invalid calls on the host-memory HIP stand-in in
// hip_stub.cpp, so that AddressSanitizer and UBSan see every host-side path:
// argument checks, plans, workspace and scratch sizing, option and profile
// bookkeeping, validation, init failures and destruction.  Exits non-zero on a
// wrong status or a bad launch parameter; the sanitizers abort on their own
// findings.
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <vector>

#include "kvshot_draft_attn.h"
#include "kvshot_fusion.h"
#include "kvshot_kvproj.h"

extern int g_launches;
extern int g_bad_params;

static int g_fail = 0;
#define EXPECT(cond)                                                   \
  do {                                                                 \
    if (!(cond)) {                                                     \
      std::fprintf(stderr, "FAIL %s:%d: %s\n", __FILE__, __LINE__, #cond); \
      ++g_fail;                                                        \
    }                                                                  \
  } while (0)

// stands for every device buffer: the host side never reads through these pointers
alignas(256) static unsigned char g_buf[1 << 20];
static void* dev(size_t off = 0) { return g_buf + off; }

static kvshot_config attn_cfg() {
  kvshot_config g;
  std::memset(&g, 0, sizeof(g));
  g.num_q_heads = 32;
  g.num_kv_heads = 8;
  g.head_dim = 128;
  g.page_size = 16;
  g.dtype = KVSHOT_BF16;
  g.out_dtype = KVSHOT_BF16;
  g.max_batch = 64;
  g.max_draft = 64;
  g.max_pages_per_seq = 2048;
  g.num_pages = 131072;
  g.max_position = 32768 + 128;
  g.rope_theta = 1e6;
  return g;
}

static kvshot_call step_call(int batch, int n, int hint) {
  kvshot_call a;
  std::memset(&a, 0, sizeof(a));
  a.mode = KVSHOT_MODE_STEP;
  a.batch = batch;
  a.n_queries = n;
  a.n_nodes = n;
  a.max_ctx_len_hint = hint;
  a.q = dev();
  a.k_pages = dev();
  a.v_pages = dev();
  a.page_table = (const int32_t*)dev();
  a.ctx_lens = (const int32_t*)dev();
  a.draft_k = dev();
  a.draft_v = dev();
  a.step_offsets = (const int32_t*)dev();
  a.out = dev();
  return a;
}

static void attention() {
  kvshot_config g = attn_cfg();
  kvshot_handle h = nullptr;
  EXPECT(kvshot_draft_attn_init(nullptr, &h) == KVSHOT_ERR_INVALID_ARG);
  EXPECT(kvshot_draft_attn_init(&g, nullptr) == KVSHOT_ERR_INVALID_ARG);
  {
    kvshot_config b = g;
    b.head_dim = 64;
    EXPECT(kvshot_draft_attn_init(&b, &h) != KVSHOT_OK);
    b = g;
    b.num_q_heads = 30;
    EXPECT(kvshot_draft_attn_init(&b, &h) == KVSHOT_ERR_INVALID_ARG);
    b = g;
    b.page_size = 24;
    EXPECT(kvshot_draft_attn_init(&b, &h) == KVSHOT_ERR_INVALID_ARG);
    b = g;
    b.max_draft = 65;
    EXPECT(kvshot_draft_attn_init(&b, &h) == KVSHOT_ERR_INVALID_ARG);
    b = g;
    b.reserved = 1;
    EXPECT(kvshot_draft_attn_init(&b, &h) == KVSHOT_ERR_INVALID_ARG);
  }
  EXPECT(kvshot_draft_attn_init(&g, &h) == KVSHOT_OK);
  if (!h) return;
  // plans over the shapes the tests and the bench use
  const int shapes[][3] = {{64, 8, 32768}, {16, 6, 8192}, {8, 60, 16384}, {1, 8, 4096}, {3, 1, 0},
                           {64, 64, 32768}, {2, 33, 100}, {64, 1, 16}, {1, 64, 32768}};
  for (auto& sh : shapes) {
    int32_t splits = 0, path = 0, rt = 0, wgs = 0;
    EXPECT(kvshot_draft_attn_plan(h, sh[0], sh[1], sh[2], &splits, &path, &rt, &wgs) == KVSHOT_OK);
    EXPECT(splits >= 1 && wgs >= 1);
  }
  // calls: step, tree, general with pos_base and query nodes, every path option, forced splits
  for (int path = 0; path <= 3; ++path) {
    EXPECT(kvshot_draft_attn_set_option(h, KVSHOT_OPT_PATH, path) == KVSHOT_OK);
    for (int splits : {0, 1, 3, 64}) {
      EXPECT(kvshot_draft_attn_set_option(h, KVSHOT_OPT_SPLITS, splits) == KVSHOT_OK);
      for (auto& sh : shapes) {
        kvshot_call a = step_call(sh[0], sh[1], sh[2]);
        EXPECT(kvshot_draft_attn_call(h, &a, nullptr) == KVSHOT_OK);
        a.mode = KVSHOT_MODE_TREE;
        a.parents = (const int32_t*)dev();
        a.step_offsets = nullptr;
        EXPECT(kvshot_draft_attn_call(h, &a, nullptr) == KVSHOT_OK);
        a.query_nodes = (const int32_t*)dev();
        a.pos_base = (const int32_t*)dev();
        a.lse = (float*)dev();
        EXPECT(kvshot_draft_attn_call(h, &a, nullptr) == KVSHOT_OK);
        const kvshot_status st = kvshot_draft_attn_call_noalloc(h, &a, nullptr);
        EXPECT(st == KVSHOT_OK || st == KVSHOT_ERR_SCRATCH);
      }
    }
  }
  EXPECT(kvshot_draft_attn_set_option(h, KVSHOT_OPT_PATH, 0) == KVSHOT_OK);
  EXPECT(kvshot_draft_attn_set_option(h, KVSHOT_OPT_SPLITS, 0) == KVSHOT_OK);
  EXPECT(kvshot_draft_attn_set_option(h, KVSHOT_OPT_PATH, 4) == KVSHOT_ERR_INVALID_ARG);
  EXPECT(kvshot_draft_attn_set_option(h, 99, 0) == KVSHOT_ERR_INVALID_ARG);
  // wrappers and argument errors
  EXPECT(kvshot_draft_attn_step(h, 4, 8, 4096, dev(), dev(), dev(), (const int32_t*)dev(), (const int32_t*)dev(),
                                dev(), dev(), (const int32_t*)dev(), dev(), nullptr, nullptr) == KVSHOT_OK);
  EXPECT(kvshot_draft_attn_tree(h, 8, 60, 16384, dev(), dev(), dev(), (const int32_t*)dev(), (const int32_t*)dev(),
                                dev(), dev(), (const int32_t*)dev(), dev(), (float*)dev(), nullptr) == KVSHOT_OK);
  {
    kvshot_call a = step_call(65, 8, 4096);
    EXPECT(kvshot_draft_attn_call(h, &a, nullptr) == KVSHOT_ERR_INVALID_ARG);
    a = step_call(4, 0, 4096);
    EXPECT(kvshot_draft_attn_call(h, &a, nullptr) == KVSHOT_ERR_INVALID_ARG);
    a = step_call(4, 8, 1 << 30);
    EXPECT(kvshot_draft_attn_call(h, &a, nullptr) == KVSHOT_ERR_INVALID_ARG);
    a = step_call(4, 8, 4096);
    a.q = nullptr;
    EXPECT(kvshot_draft_attn_call(h, &a, nullptr) == KVSHOT_ERR_INVALID_ARG);
    a = step_call(4, 8, 4096);
    a.reserved = 7;
    EXPECT(kvshot_draft_attn_call(h, &a, nullptr) == KVSHOT_ERR_INVALID_ARG);
    EXPECT(kvshot_draft_attn_call(h, nullptr, nullptr) == KVSHOT_ERR_INVALID_ARG);
    EXPECT(kvshot_draft_attn_call(nullptr, &a, nullptr) == KVSHOT_ERR_INVALID_ARG);
  }
  // validation (the stand-in reports no violation)
  int32_t bad = -2;
  EXPECT(kvshot_draft_attn_validate(h, 4, 8, 4096, (const int32_t*)dev(), (const int32_t*)dev(), (const int32_t*)dev(),
                                    nullptr, &bad, nullptr) == KVSHOT_OK);
  {
    kvshot_call a = step_call(8, 60, 16384);
    a.mode = KVSHOT_MODE_TREE;
    a.parents = (const int32_t*)dev();
    EXPECT(kvshot_draft_attn_validate_call(h, &a, &bad, nullptr) == KVSHOT_OK);
  }
  // profiling: more calls than the event ring holds, then a read
  EXPECT(kvshot_draft_attn_set_option(h, KVSHOT_OPT_PROFILE, 1) == KVSHOT_OK);
  for (int i = 0; i < 1500; ++i) {
    kvshot_call a = step_call(16, 6, 8192);
    EXPECT(kvshot_draft_attn_call(h, &a, nullptr) == KVSHOT_OK);
  }
  double am = 0, cm = 0;
  int64_t calls = 0;
  EXPECT(kvshot_draft_attn_profile_read(h, &am, &cm, &calls) == KVSHOT_OK);
  EXPECT(calls == 1500);
  EXPECT(kvshot_draft_attn_set_option(h, KVSHOT_OPT_PROFILE, 0) == KVSHOT_OK);
  // debug entry points
  EXPECT(kvshot_debug_gather_kv(h, 2, 256, dev(), dev(), (const int32_t*)dev(), (const int32_t*)dev(), dev(), dev(),
                                nullptr) == KVSHOT_OK);
  EXPECT(kvshot_debug_stream_read(dev(), 1 << 20, dev(), 256, nullptr) == KVSHOT_OK);
  EXPECT(kvshot_debug_mfma_rate(256, 16, dev(), nullptr) == KVSHOT_OK);
  EXPECT(kvshot_debug_mfma_rate(0, 16, dev(), nullptr) == KVSHOT_ERR_INVALID_ARG);
  EXPECT(kvshot_debug_mfma_rate(256, 0, dev(), nullptr) == KVSHOT_ERR_INVALID_ARG);
  EXPECT(kvshot_debug_mfma_rate(256, 16, nullptr, nullptr) == KVSHOT_ERR_INVALID_ARG);
  for (int s = 0; s <= 7; ++s) EXPECT(kvshot_status_string(s) != nullptr);
  EXPECT(kvshot_draft_attn_destroy(h) == KVSHOT_OK);
  EXPECT(kvshot_draft_attn_destroy(nullptr) == KVSHOT_OK);
  // a float32 handle (generic path) with strided pages
  g.dtype = KVSHOT_FP32;
  g.out_dtype = KVSHOT_FP32;
  g.page_stride = 8 * 16 * 128 + 64;
  g.slot_stride = 136;
  g.head_stride = 16 * 136;
  h = nullptr;
  EXPECT(kvshot_draft_attn_init(&g, &h) == KVSHOT_OK);
  if (h) {
    kvshot_call a = step_call(4, 4, 256);
    EXPECT(kvshot_draft_attn_call(h, &a, nullptr) == KVSHOT_OK);
    EXPECT(kvshot_draft_attn_destroy(h) == KVSHOT_OK);
  }
}

static void fusion() {
  kvshot_fusion_handle h = nullptr;
  EXPECT(kvshot_fusion_init(100, 8, &h) == KVSHOT_ERR_INVALID_ARG);
  EXPECT(kvshot_fusion_init(4096, 0, &h) == KVSHOT_ERR_INVALID_ARG);
  EXPECT(kvshot_fusion_init(4096, 1024, &h) == KVSHOT_OK);
  if (!h) return;
  for (int tile = 0; tile <= 2; ++tile)
  for (int tokens : {1, 37, 64, 100, 256, 384, 480, 1024}) {
    for (int splits : {0, 1, 2, 4, 8, 16}) {
      EXPECT(kvshot_fusion_set_option(h, KVSHOT_OPT_PATH, tile) == KVSHOT_OK);
      EXPECT(kvshot_fusion_set_option(h, KVSHOT_OPT_SPLITS, splits) == KVSHOT_OK);
      int32_t s = 0, w = 0;
      EXPECT(kvshot_fusion_plan(h, tokens, &s, &w) == KVSHOT_OK);
      EXPECT(kvshot_gated_delta_fusion(h, tokens, dev(), dev(), dev(), (const float*)dev(), dev(), dev(), nullptr, 0,
                                       nullptr) == KVSHOT_OK);
      EXPECT(kvshot_gated_delta_fusion_packed(h, tokens, dev(), dev(), dev(), (const float*)dev(), dev(),
                                              (float*)dev(), 0, nullptr) == KVSHOT_OK);
    }
  }
  EXPECT(kvshot_fusion_set_option(h, KVSHOT_OPT_PATH, 0) == KVSHOT_OK);
  EXPECT(kvshot_fusion_set_option(h, KVSHOT_OPT_SPLITS, 0) == KVSHOT_OK);
  EXPECT(kvshot_fusion_set_option(h, KVSHOT_OPT_PATH, 3) == KVSHOT_ERR_INVALID_ARG);
  EXPECT(kvshot_fusion_pack_weights(h, dev(), dev(), dev(), nullptr) == KVSHOT_OK);
  EXPECT(kvshot_gated_delta_fusion(h, 1025, dev(), dev(), dev(), (const float*)dev(), dev(), dev(), nullptr, 0,
                                   nullptr) == KVSHOT_ERR_INVALID_ARG);
  EXPECT(kvshot_gated_delta_fusion(h, 8, nullptr, dev(), dev(), (const float*)dev(), dev(), dev(), nullptr, 0,
                                   nullptr) == KVSHOT_ERR_INVALID_ARG);
  EXPECT(kvshot_fusion_set_option(h, KVSHOT_OPT_PROFILE, 1) == KVSHOT_OK);
  for (int i = 0; i < 1100; ++i)
    EXPECT(kvshot_gated_delta_fusion(h, 480, dev(), dev(), dev(), (const float*)dev(), dev(), dev(), nullptr, 0,
                                     nullptr) == KVSHOT_OK);
  double a = 0, c = 0;
  int64_t calls = 0;
  EXPECT(kvshot_fusion_profile_read(h, &a, &c, &calls) == KVSHOT_OK);
  EXPECT(calls == 1100);
  EXPECT(kvshot_fusion_destroy(h) == KVSHOT_OK);
  EXPECT(kvshot_fusion_destroy(nullptr) == KVSHOT_OK);
}

static void kvproj() {
  kvshot_kvproj_config g;
  std::memset(&g, 0, sizeof(g));
  g.num_kv_heads = 8;
  g.head_dim = 128;
  g.num_layers = 3;
  g.page_size = 16;
  g.max_pages_per_seq = 2048;
  g.num_pages = 4096;
  g.dst_num_pages = 4096;
  g.max_tokens = 40000;
  g.max_position = 32768;
  g.rope_theta = 1e6;
  kvshot_kvproj_handle h = nullptr;
  {
    kvshot_kvproj_config b = g;
    b.num_layers = 5;
    EXPECT(kvshot_kvproj_init(&b, &h) == KVSHOT_ERR_INVALID_ARG);
    b = g;
    b.rope_theta = -1.0;
    EXPECT(kvshot_kvproj_init(&b, &h) == KVSHOT_ERR_INVALID_ARG);
    b = g;
    b.slot_stride = 100;
    EXPECT(kvshot_kvproj_init(&b, &h) == KVSHOT_ERR_INVALID_ARG);
  }
  EXPECT(kvshot_kvproj_init(&g, &h) == KVSHOT_OK);
  if (!h) return;
  const void* ks[3] = {dev(), dev(4096), dev(8192)};
  const void* vs[3] = {dev(16), dev(4112), dev(8208)};
  for (int path = 0; path <= 2; ++path) {
    EXPECT(kvshot_kvproj_set_option(h, KVSHOT_OPT_PATH, path) == KVSHOT_OK);
    for (int splits : {0, 1, 5, 16}) {
      EXPECT(kvshot_kvproj_set_option(h, KVSHOT_OPT_SPLITS, splits) == KVSHOT_OK);
      for (int n : {1, 7, 64, 287, 480, 1536, 4096, 33000, 40000}) {
        int32_t s = 0, p = 0, t = 0, w = 0;
        EXPECT(kvshot_kvproj_plan(h, n, &s, &p, &t, &w) == KVSHOT_OK);
        EXPECT(s >= 1 && (p == 1 || p == 2) && t >= 16 && w >= 1);
        EXPECT(kvshot_kv_project(h, n, 64, ks, vs, (const int32_t*)dev(), (const int32_t*)dev(),
                                 (const int32_t*)dev(), dev(), dev(), dev(), dev(), nullptr, KVSHOT_KVPROJ_ROPE,
                                 nullptr) == KVSHOT_OK);
      }
    }
  }
  EXPECT(kvshot_kvproj_set_option(h, KVSHOT_OPT_PATH, 3) == KVSHOT_ERR_INVALID_ARG);
  EXPECT(kvshot_kvproj_set_option(h, KVSHOT_OPT_SPLITS, 17) == KVSHOT_ERR_INVALID_ARG);
  EXPECT(kvshot_kv_project(h, 40001, 64, ks, vs, (const int32_t*)dev(), (const int32_t*)dev(), (const int32_t*)dev(),
                           dev(), dev(), dev(), dev(), nullptr, 0, nullptr) == KVSHOT_ERR_INVALID_ARG);
  EXPECT(kvshot_kv_project(h, 10, 64, ks, vs, (const int32_t*)dev(), (const int32_t*)dev(), (const int32_t*)dev(),
                           dev(2), dev(), dev(), dev(), nullptr, 0, nullptr) == KVSHOT_ERR_INVALID_ARG);
  int32_t bt = -2, bc = -2;
  EXPECT(kvshot_kv_project_validate(h, 287, 64, (const int32_t*)dev(), (const int32_t*)dev(), (const int32_t*)dev(),
                                    nullptr, &bt, &bc, nullptr) == KVSHOT_OK);
  EXPECT(bt == -1 && bc == 0);
  EXPECT(kvshot_kvproj_set_option(h, KVSHOT_OPT_PROFILE, 1) == KVSHOT_OK);
  for (int i = 0; i < 1100; ++i)
    EXPECT(kvshot_kv_project(h, 287, 64, ks, vs, (const int32_t*)dev(), (const int32_t*)dev(), (const int32_t*)dev(),
                             dev(), dev(), dev(), dev(), nullptr, KVSHOT_KVPROJ_ROPE, nullptr) == KVSHOT_OK);
  double a = 0, c = 0;
  int64_t calls = 0;
  EXPECT(kvshot_kvproj_profile_read(h, &a, &c, &calls) == KVSHOT_OK);
  EXPECT(calls == 1100);
  EXPECT(kvshot_kvproj_destroy(h) == KVSHOT_OK);
  EXPECT(kvshot_kvproj_destroy(nullptr) == KVSHOT_OK);
}

int main() {
  attention();
  fusion();
  kvproj();
  std::printf("launches %d, bad launch parameters %d, failed expectations %d\n", g_launches, g_bad_params, g_fail);
  return (g_fail == 0 && g_bad_params == 0 && g_launches > 0) ? 0 : 1;
}
