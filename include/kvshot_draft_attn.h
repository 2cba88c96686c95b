/*
 * kvshot_draft_attn.h -- C ABI of the draft-step attention library for MI355X (gfx950).
 *
 * Operation (KVShot, arXiv 2604.26412):
 *   A drafter query re-attends the target model's un-aggregated per-token K/V
 *   with its own query (Sec. 2.2, Eq. 2).  The memory a draft step attends is
 *   the target KV of the verified prefix followed by the drafter's own KV for
 *   later draft positions, as in an ordinary autoregressive KV cache
 *   (Sec. 3.4.1, Eq. 7; App. B, "Cross-attention memory").  Draft tokens are a
 *   linear chain of steps or a tree (Sec. 3.5, tree (8, 10, 60)).
 *
 *   For sequence b with T_b prefix tokens, query head hq (KV head hq / G,
 *   G = num_q_heads / num_kv_heads) and query row j:
 *     out = sum_{allowed keys} softmax(scale * <rope(q, pos_j), key>) * value
 *   where the keys are the T_b target keys (stored already rotated, used as
 *   is) followed by the draft keys, each rotated at its own position, and
 *     step mode: query j sits at draft step s0 + j (s0 = step_offsets[b]),
 *                position T_b + s0 + j; draft key s sits at position T_b + s
 *                and is visible to query j iff s <= s0 + j;
 *     tree mode: node i sits at position T_b + depth(i); draft key s is node s's
 *                key at T_b + depth(s), visible to node i iff s is i or one of
 *                its ancestors (parents[i] == -1 marks a root).
 *   RoPE is rotate-half: channel m pairs with m + D/2, angle pos * theta^(-2m/D).
 *   scale defaults to 1/sqrt(head_dim).
 *
 * Conventions for every call:
 *   - Every array pointer is a DEVICE pointer unless marked (host).
 *   - bf16 data is passed as raw 16-bit patterns; fp32 as IEEE float.
 *   - The caller owns every array and keeps it alive until the work queued on
 *     `stream` (a hipStream_t, NULL = default stream) has finished.
 *   - Functions never throw or abort.  Argument errors found on the host are
 *     returned before anything is queued and leave `out` untouched.  Queued
 *     work performs no host synchronisation (except validate, which does).
 *   - Data-dependent contract violations (a page id outside the pool, a length
 *     above the hint, a bad parent) never make a kernel read out of bounds:
 *     indices are clamped.  The result is then unspecified; call
 *     kvshot_draft_attn_validate to detect them.
 *   - A handle may be used by one stream at a time.
 */
#ifndef KVSHOT_DRAFT_ATTN_H
#define KVSHOT_DRAFT_ATTN_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  KVSHOT_OK = 0,
  KVSHOT_ERR_INVALID_ARG = 1,   /* null pointer, size out of range, inconsistent config */
  KVSHOT_ERR_UNSUPPORTED = 2,   /* valid but not implemented (head_dim != 128, ...) */
  KVSHOT_ERR_OUT_OF_MEMORY = 3, /* device allocation in init failed */
  KVSHOT_ERR_DEVICE = 4,        /* a HIP call or kernel launch failed */
  KVSHOT_ERR_DATA = 5,          /* validate found a contract violation in device data */
  KVSHOT_ERR_SCRATCH = 6        /* kvshot_draft_attn_call_noalloc: the call needs more scratch than it has */
} kvshot_status;

typedef enum { KVSHOT_BF16 = 0, KVSHOT_FP32 = 1 } kvshot_dtype;

typedef struct kvshot_config {
  int32_t num_q_heads;        /* Hq; Hq % Hkv == 0 and G = Hq / Hkv <= 8 */
  int32_t num_kv_heads;       /* Hkv >= 1 */
  int32_t head_dim;           /* D; must be 128 */
  int32_t page_size;          /* P; power of two in [16, 256] */
  int32_t dtype;              /* kvshot_dtype of q, K/V pages and draft K/V */
  int32_t out_dtype;          /* kvshot_dtype of out */
  int32_t max_batch;          /* largest batch any call will pass */
  int32_t max_draft;          /* rows of the draft K/V arrays per sequence; 1..64 */
  int32_t max_pages_per_seq;  /* row stride (entries) of page_table */
  int32_t num_pages;          /* pages in the K (and V) pool; page ids are clamped to it */
  int64_t max_position;       /* positions 0..max_position-1 get a RoPE table entry */
  double rope_theta;          /* RoPE base, > 0 (1e6 for Qwen3) */
  float softmax_scale;        /* 0 -> 1/sqrt(head_dim) */
  int32_t reserved;           /* must be 0 */
  int64_t page_stride;        /* elements between pages; 0 -> Hkv * P * D */
  int64_t head_stride;        /* elements between KV heads in a page; 0 -> P * D */
  int64_t slot_stride;        /* elements between slots in a page; 0 -> D.  head_dim is contiguous. */
} kvshot_config;

typedef struct kvshot_ctx* kvshot_handle;

/* Validates `cfg`, selects the current HIP device, allocates the split-K
 * workspace and builds the RoPE cos/sin table (float64 on the host, rounded to
 * float32).  On success *out receives a handle.  Host pointers. */
kvshot_status kvshot_draft_attn_init(const kvshot_config* cfg, kvshot_handle* out);

/* Releases the handle's device memory (synchronises the device).  NULL is a no-op. */
kvshot_status kvshot_draft_attn_destroy(kvshot_handle h);

/* Step mode: n_new causal draft steps per sequence folded into one call.
 *   q            [batch][n_new][Hq][D]  pre-RoPE draft queries
 *   k_pages      target keys (already rotated), v_pages target values: element
 *                (page, kv_head, slot, d) at page*page_stride + kv_head*head_stride
 *                + slot*slot_stride + d
 *   page_table   int32 [batch][max_pages_per_seq]; token t of sequence b is in
 *                slot t % P of page page_table[b][t / P]; entries at or past
 *                ceil(ctx_lens[b] / P) are never read
 *   ctx_lens     int32 [batch]; 0 <= T_b <= max_ctx_len_hint
 *   draft_k/v    [batch][max_draft][Hkv][D]; draft_k pre-RoPE; rows
 *                [0, step_offsets[b] + n_new) are read
 *   step_offsets int32 [batch]; 0 <= s0 and s0 + n_new <= max_draft
 *   out          [batch][n_new][Hq][D] in out_dtype
 *   lse          nullable float32 [batch][n_new][Hq], natural-log sum of exp of scores
 *   max_ctx_len_hint (host) bounds T_b and sizes the split-K grid.
 * Requirements: 1 <= batch <= max_batch, 1 <= n_new <= max_draft,
 * G * n_new <= 256, max_ctx_len_hint <= max_pages_per_seq * P and
 * max_ctx_len_hint + max_draft <= max_position. */
kvshot_status kvshot_draft_attn_step(kvshot_handle h, int32_t batch, int32_t n_new, int32_t max_ctx_len_hint,
                                     const void* q, const void* k_pages, const void* v_pages,
                                     const int32_t* page_table, const int32_t* ctx_lens,
                                     const void* draft_k, const void* draft_v, const int32_t* step_offsets,
                                     void* out, float* lse, void* stream);

/* Tree mode: n_nodes draft-tree nodes per sequence.
 *   q            [batch][n_nodes][Hq][D]  pre-RoPE, node order
 *   draft_k/v    [batch][max_draft][Hkv][D]; row i is node i's key/value
 *   parents      int32 [batch][n_nodes]; parents[b][i] in {-1} U [0, i)
 * Other arguments as in kvshot_draft_attn_step; 1 <= n_nodes <= max_draft. */
kvshot_status kvshot_draft_attn_tree(kvshot_handle h, int32_t batch, int32_t n_nodes, int32_t max_ctx_len_hint,
                                     const void* q, const void* k_pages, const void* v_pages,
                                     const int32_t* page_table, const int32_t* ctx_lens,
                                     const void* draft_k, const void* draft_v, const int32_t* parents,
                                     void* out, float* lse, void* stream);

/* General form of a call (step or tree), with two additions:
 *
 *   pos_base     nullable int32 [batch]: position of draft step 0 (step mode)
 *                or of depth 0 (tree mode) for sequence b.  NULL means
 *                ctx_lens[b], as in kvshot_draft_attn_step / _tree.  A separate
 *                base lets the prefix hold keys that are not one position per
 *                slot: the KV of L_s sampled target layers concatenated along
 *                the sequence (the head-concatenation injection of Sec. 3.2,
 *                read as one softmax over the L_s x T keys), while the draft
 *                tokens keep positions T + step.  Values are clamped to
 *                [0, max_position], positions to the RoPE table.
 *   query_nodes  tree mode, nullable int32 [batch][n_queries]: the tree node
 *                whose query fills query row j.  The draft keys are always all
 *                n_nodes nodes, so only the newest level's nodes need queries
 *                when a tree grows level by level (Sec. 3.5, tree (8, 10, 60)).
 *                NULL means row j is node j (then n_queries == n_nodes).  Values
 *                are clamped to [0, n_nodes).
 *
 * Step mode: n_nodes is ignored; query j sits at pos_base + s0 + j and sees
 * draft keys s <= s0 + j, each at pos_base + s.  Tree mode: query row j (node
 * i = query_nodes[b][j]) sits at pos_base + depth(i) and sees the draft keys
 * of i and its ancestors, key s at pos_base + depth(s).
 * Requirements as for kvshot_draft_attn_step / _tree, with G * n_queries <= 256,
 * 1 <= n_queries <= max_draft and, in tree mode, 1 <= n_nodes <= max_draft. */
enum { KVSHOT_MODE_STEP = 0, KVSHOT_MODE_TREE = 1 };
typedef struct kvshot_call {
  int32_t mode;                 /* KVSHOT_MODE_STEP or KVSHOT_MODE_TREE */
  int32_t batch;
  int32_t n_queries;            /* query rows per sequence */
  int32_t n_nodes;              /* tree mode: nodes (draft keys) per sequence */
  int32_t max_ctx_len_hint;     /* bounds ctx_lens, sizes the split-K grid */
  int32_t reserved;             /* must be 0 */
  const void* q;                /* [batch][n_queries][Hq][D] */
  const void* k_pages;
  const void* v_pages;
  const int32_t* page_table;
  const int32_t* ctx_lens;
  const void* draft_k;          /* [batch][max_draft][Hkv][D] */
  const void* draft_v;
  const int32_t* step_offsets;  /* step mode: [batch] */
  const int32_t* parents;       /* tree mode: [batch][n_nodes] */
  const int32_t* query_nodes;   /* tree mode, nullable: [batch][n_queries] */
  const int32_t* pos_base;      /* nullable: [batch] */
  void* out;                    /* [batch][n_queries][Hq][D] */
  float* lse;                   /* nullable: [batch][n_queries][Hq] */
} kvshot_call;

/* Runs the call described by *call (host struct; device pointers inside). */
kvshot_status kvshot_draft_attn_call(kvshot_handle h, const kvshot_call* call, void* stream);

/* kvshot_draft_attn_call for callers that cannot allocate device memory
 * (code under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc).  Same arguments, plan, kernels and result bits as
 * kvshot_draft_attn_call; the difference is where the split-K partials go:
 * a 32 MiB array in the library's static device memory (one copy per GPU,
 * held until the process ends; its address is resolved once per device by
 * kvshot_draft_attn_init), instead of the handle's workspace.  The call
 * allocates nothing and records no profiling events.
 *   - A call whose partials exceed 32 MiB (batch x num_kv_heads x padded rows
 *     x splits x (128 x 4 + 8) bytes, the partial (m, l) rows aligned to 256
 *     bytes, plus 256 bytes of per-sequence split counts for a ragged batch;
 *     a one-split plan needs none) returns KVSHOT_ERR_SCRATCH and queues
 *     nothing.
 *   - Every call on one GPU shares that GPU's scratch: calls that overlap in
 *     time on one GPU (from any handle, stream or thread) race and give
 *     undefined results.  Calls ordered on one stream are safe.
 *   - The scratch keeps the last call's contents; nothing in it needs to start
 *     at zero (every partial a call reads is written earlier in the call). */
kvshot_status kvshot_draft_attn_call_noalloc(kvshot_handle h, const kvshot_call* call, void* stream);

/* kvshot_draft_attn_validate for a kvshot_call: also checks query_nodes
 * (code 5: a node outside [0, n_nodes)) and pos_base (code 6: negative, or a
 * draft position beyond the RoPE table).  Synchronises `stream`. */
kvshot_status kvshot_draft_attn_validate_call(kvshot_handle h, const kvshot_call* call, int32_t* first_bad,
                                              void* stream);

/* Checks device-side contract data for a call with these sizes: every page id a
 * call would read lies in [0, num_pages), 0 <= ctx_lens[b] <= max_ctx_len_hint,
 * step offsets in range (if step_offsets != NULL), parents in {-1} U [0, i)
 * (if parents != NULL).  Synchronises `stream`.  Returns KVSHOT_OK or
 * KVSHOT_ERR_DATA; *first_bad (host, nullable) receives a code naming the
 * first kind of violation found (0 none, 1 ctx_len, 2 page id, 3 step offset,
 * 4 parent). */
kvshot_status kvshot_draft_attn_validate(kvshot_handle h, int32_t batch, int32_t n_queries, int32_t max_ctx_len_hint,
                                         const int32_t* page_table, const int32_t* ctx_lens,
                                         const int32_t* step_offsets, const int32_t* parents,
                                         int32_t* first_bad, void* stream);

/* Tuning and introspection. */
typedef enum {
  KVSHOT_OPT_SPLITS = 0,   /* value 0: automatic split-K count; n > 0: use n (clamped to the workspace) */
  KVSHOT_OPT_PATH = 1,     /* 0 automatic, 1 MFMA kernels (bf16 only; 256-row query tiles take the
                              tall-tile kernel), 2 generic VALU kernel, 3 the general MFMA kernel for
                              every tile height (bf16 only) */
  KVSHOT_OPT_PROFILE = 2   /* 1: record HIP events around the attention and combine kernels of every call */
} kvshot_option;
kvshot_status kvshot_draft_attn_set_option(kvshot_handle h, int32_t option, int64_t value);

/* Plan a call would use: split count, path (1 MFMA, 2 generic), 32-row query tiles,
 * and grid size in workgroups of the attention kernel.  Host outputs, each nullable. */
kvshot_status kvshot_draft_attn_plan(kvshot_handle h, int32_t batch, int32_t n_queries, int32_t max_ctx_len_hint,
                                     int32_t* splits, int32_t* path, int32_t* row_tiles, int32_t* workgroups);

/* With KVSHOT_OPT_PROFILE on: synchronises, then returns the summed event time
 * (ms) of the attention kernel and of the combine kernel over the calls since
 * the last read, and the call count; resets the sums.  Host outputs. */
kvshot_status kvshot_draft_attn_profile_read(kvshot_handle h, double* attn_ms, double* combine_ms, int64_t* calls);

/* Debug: the dense logical view [batch][max_ctx][Hkv][D] (dtype of the pools)
 * of the paged target K/V, produced by the same page-addressing code the
 * attention kernels use.  Positions >= ctx_lens[b] are written as zero. */
kvshot_status kvshot_debug_gather_kv(kvshot_handle h, int32_t batch, int32_t max_ctx, const void* k_pages,
                                     const void* v_pages, const int32_t* page_table, const int32_t* ctx_lens,
                                     void* k_dense, void* v_dense, void* stream);

/* Debug: ancestor-or-self bitmasks (bit s of anc_out[b][i] set iff node s is i or
 * an ancestor of i) and depths of the draft trees, produced by the same code the
 * tree kernels use.  anc_out uint64 [batch][n_nodes], depth_out int32 [batch][n_nodes]. */
kvshot_status kvshot_debug_tree_mask(kvshot_handle h, int32_t batch, int32_t n_nodes, const int32_t* parents,
                                     uint64_t* anc_out, int32_t* depth_out, void* stream);

/* Measurement helper: reads `bytes` (rounded down to a multiple of 16) of
 * device memory `src` once with 16-byte loads, using `sink_words` workgroups;
 * each workgroup writes one 16-byte word of `sink` (device, >= 16*sink_words
 * bytes).  Times the device's practical streaming-read bandwidth. */
kvshot_status kvshot_debug_stream_read(const void* src, int64_t bytes, void* sink, int32_t sink_words, void* stream);

/* Measurement helper: `workgroups` workgroups of four waves (one per SIMD of a
 * CU) each issue `iters` x 16 dense bf16 32x32x16 matrix products per wave,
 * with no memory traffic; each workgroup writes one 16-byte word of `sink`
 * (device, >= 16*workgroups bytes).  A launch performs workgroups x 4 x iters
 * x 16 x 32768 flops.  Times the rate the matrix cores sustain when every SIMD
 * runs them (the clock the chip holds under that load included), the
 * counterpart of the streaming-read probe for matrix-bound kernels.
 * Returns KVSHOT_ERR_INVALID_ARG for workgroups or iters below 1 or a null or
 * unaligned sink. */
kvshot_status kvshot_debug_mfma_rate(int32_t workgroups, int32_t iters, void* sink, void* stream);

/* Static text for a status code. */
const char* kvshot_status_string(int32_t status);

#ifdef __cplusplus
}
#endif

#endif /* KVSHOT_DRAFT_ATTN_H */
