/*
 * kvshot_kvproj.h -- C ABI of the projected-KV cache builder on MI355X (gfx950).
 *
 * Operation (KVShot, arXiv 2604.26412, Sec. 3.2, KV-only reuse: the "linear
 * projection" injection and its "Proj + RoPE fix" variant; App. A, "Target KV
 * layers": L_s = 3 uniformly spaced target layers).  A KV-only drafter attends
 * one layer's worth of KV built from L_s sampled target layers.  For every
 * listed token (sequence b, position t) with K vectors k^(1) .. k^(L_s) and V
 * vectors v^(1) .. v^(L_s) in the L_s source caches (d_kv = Hkv * 128 values
 * each, head-major: index h * 128 + d),
 *
 *     k' = W_K [k^(1); ...; k^(L_s)]      v' = W_V [v^(1); ...; v^(L_s)]
 *     W_K, W_V in R^{d_kv x L_s d_kv}, row c = output channel c (input index
 *     l d_kv + h 128 + d = channel d of head h of the l-th given layer)
 *
 * and with KVSHOT_KVPROJ_ROPE the projected key is rotated at the token's
 * position t (rotate-half: channel m pairs with m + 64, angle
 * t theta^(-2m/128)); values are never rotated.  k' and v' are rounded to
 * bf16 and written into slot t % P of page dst_page_table[b][t / P] of the
 * destination pools -- the cache kvshot_draft_attn_* then reads as the target
 * prefix.  The source keys are used as stored (rotated or not, as the target
 * engine keeps them).
 *
 * Arithmetic: bf16 products on MFMA with float32 accumulation over the
 * L_s d_kv inputs (in a fixed order per plan: split reductions on the tiled
 * path, per-wave partial sums added in wave order on the direct path); RoPE
 * in float32 (a table built in float64, or on the tiled path without splits
 * angles reduced in float64); one rounding to bf16.
 *
 * Conventions (as in kvshot_draft_attn.h): array pointers are DEVICE pointers
 * unless marked (host); bf16 is passed as raw 16-bit patterns; the caller owns
 * every array until the work queued on `stream` (a hipStream_t, NULL = default
 * stream) has finished; functions never throw or abort, and argument errors are
 * returned before anything is queued.  Data-dependent violations (a sequence,
 * position or page id out of range) never make a kernel access memory out of
 * bounds: indices are clamped and the result is then unspecified;
 * kvshot_kv_project_validate detects them.  A handle may be used by one stream
 * at a time.
 */
#ifndef KVSHOT_KVPROJ_H
#define KVSHOT_KVPROJ_H

#include <stdint.h>

#include "kvshot_draft_attn.h"

#ifdef __cplusplus
extern "C" {
#endif

typedef struct kvshot_kvproj_ctx* kvshot_kvproj_handle;

enum {
  KVSHOT_KVPROJ_ROPE = 1 /* rotate projected keys at their positions */
};

typedef struct kvshot_kvproj_config {
  int32_t num_kv_heads;       /* Hkv of every source layer and of the projected cache; 1..16 */
  int32_t head_dim;           /* must be 128 */
  int32_t num_layers;         /* L_s; 1..4 */
  int32_t page_size;          /* P, power of two in [16, 256], sources and destination */
  int32_t max_pages_per_seq;  /* row stride (entries) of both page tables */
  int32_t num_pages;          /* pages in each source pool (ids are clamped to it) */
  int32_t dst_num_pages;      /* pages in each destination pool */
  int32_t max_tokens;         /* most tokens one call lists; sizes the split workspace */
  int64_t max_position;       /* positions 0 .. max_position - 1 get a RoPE table entry */
  double rope_theta;          /* RoPE base, > 0 (1e6 for Qwen3) */
  int64_t page_stride;        /* source layout in elements, as in kvshot_config; 0 -> Hkv * P * 128 */
  int64_t head_stride;        /* 0 -> P * 128 */
  int64_t slot_stride;        /* 0 -> 128 */
  int64_t dst_page_stride;    /* destination layout, same meaning and defaults */
  int64_t dst_head_stride;
  int64_t dst_slot_stride;
} kvshot_kvproj_config;

/* Validates `cfg`, selects the current HIP device, builds the RoPE table and
 * allocates the split workspace (at most 8192 x 2 d_kv floats: 64 MB when
 * d_kv = 1024).  *out receives the handle.  Host pointers. */
kvshot_status kvshot_kvproj_init(const kvshot_kvproj_config* cfg, kvshot_kvproj_handle* out);

/* Releases the handle's device memory (synchronises the device).  NULL is a no-op. */
kvshot_status kvshot_kvproj_destroy(kvshot_kvproj_handle h);

/* Projects and scatters n_tokens tokens.
 *   k_src, v_src    (host) arrays of num_layers device pointers: the source
 *                   layers' K and V pools, in stacking order
 *   page_table      int32 [batch][max_pages_per_seq]: the sources' pages
 *   token_seq       int32 [n_tokens]: sequence of each token, in [0, batch)
 *   token_pos       int32 [n_tokens]: its position t, with t < max_position and
 *                   t < max_pages_per_seq * P
 *   w_k, w_v        bf16 [d_kv][num_layers d_kv], row-major
 *   k_dst, v_dst    the destination pools (bf16), written only at the listed
 *                   tokens' slots; they must not overlap a source pool
 *   dst_page_table  nullable int32 [batch][max_pages_per_seq]; NULL -> page_table
 *   flags           0 or KVSHOT_KVPROJ_ROPE
 * 1 <= n_tokens <= max_tokens, 1 <= batch.  Every device pointer must be
 * 16-byte aligned.  Two tokens that map to the same destination slot leave one
 * of the two results there, unspecified which. */
kvshot_status kvshot_kv_project(kvshot_kvproj_handle h, int32_t n_tokens, int32_t batch,
                                const void* const* k_src, const void* const* v_src,
                                const int32_t* page_table, const int32_t* token_seq, const int32_t* token_pos,
                                const void* w_k, const void* w_v, void* k_dst, void* v_dst,
                                const int32_t* dst_page_table, int32_t flags, void* stream);

/* Checks the listed tokens against the contract (synchronises `stream`).
 * Returns KVSHOT_OK, or KVSHOT_ERR_DATA with *bad_token = the first offending
 * token and *bad_code = 1 (sequence), 2 (position), 3 (source page id),
 * 4 (destination page id).  Host outputs, each nullable. */
kvshot_status kvshot_kv_project_validate(kvshot_kvproj_handle h, int32_t n_tokens, int32_t batch,
                                         const int32_t* page_table, const int32_t* token_seq,
                                         const int32_t* token_pos, const int32_t* dst_page_table,
                                         int32_t* bad_token, int32_t* bad_code, void* stream);

/* Options: KVSHOT_OPT_SPLITS (0 automatic, else 1 .. 16 workgroups along the
 * reduction of the tiled path, capped by the workspace), KVSHOT_OPT_PATH
 * (0 automatic: the direct path where the tiled one would split its
 * reduction, unless KVSHOT_OPT_SPLITS is set; 1 the tiled path, 256 channels x
 * 256 tokens per workgroup; 2 the direct path, 64 channels x up to 64 tokens
 * per workgroup with the whole reduction, no partial sums) and
 * KVSHOT_OPT_PROFILE (1: HIP events around each kernel of every call), as for
 * the attention handle. */
kvshot_status kvshot_kvproj_set_option(kvshot_kvproj_handle h, int32_t option, int64_t value);

/* Plan of a call with n_tokens tokens: reduction splits (1 on the direct
 * path), path (1 tiled, 2 direct), tokens per workgroup tile and workgroups of
 * the main kernel.  Host outputs, each nullable. */
kvshot_status kvshot_kvproj_plan(kvshot_kvproj_handle h, int32_t n_tokens, int32_t* splits, int32_t* path,
                                 int32_t* tile_tokens, int32_t* workgroups);

/* With KVSHOT_OPT_PROFILE on: synchronises, then returns the summed event time
 * (ms) of the main kernel and of the split combine kernel since the last read,
 * and the call count; resets the sums.  Host outputs. */
kvshot_status kvshot_kvproj_profile_read(kvshot_kvproj_handle h, double* main_ms, double* combine_ms,
                                         int64_t* calls);

#ifdef __cplusplus
}
#endif

#endif /* KVSHOT_KVPROJ_H */
