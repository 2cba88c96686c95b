/*
 * kvshot_fusion.h -- C ABI of the hybrid drafter's gated delta fusion on MI355X (gfx950).
 *
 * Operation (KVShot, arXiv 2604.26412, Sec. 3.4.1, Eqs. (delta) and (fusion);
 * shapes from App. B, "Shared gate"): for every draft token i with
 * self-attention output n_i and cross-attention output o_i, both in R^d,
 *     Delta_i = o_i - n_i
 *     g_i     = sigmoid(W_g [n_i; o_i; Delta_i] + b_g)       W_g in R^{d x 3d}, b_g in R^d
 *     h_i     = n_i + g_i (elementwise) (W_Delta Delta_i)     W_Delta in R^{d x d}
 * The cross-only variant (Sec. 3.4.2) removes the self-attention output from
 * the forward pass: with KVSHOT_FUSION_CROSS_ONLY, n is read as zero (n may then
 * be NULL), so Delta = o and h = g * (W_Delta o).
 *
 * Conventions (as in kvshot_draft_attn.h): array pointers are DEVICE pointers
 * unless marked (host); bf16 is passed as raw 16-bit patterns; the caller owns
 * every array until the work queued on `stream` (a hipStream_t, NULL = default
 * stream) has finished; functions never throw or abort, and argument errors
 * are returned before anything is queued.  A handle may be used by one stream
 * at a time.
 */
#ifndef KVSHOT_FUSION_H
#define KVSHOT_FUSION_H

#include <stdint.h>

#include "kvshot_draft_attn.h"

#ifdef __cplusplus
extern "C" {
#endif

typedef struct kvshot_fusion_ctx* kvshot_fusion_handle;

enum {
  KVSHOT_FUSION_CROSS_ONLY = 1, /* read n as zero */
  KVSHOT_FUSION_OUT_FP32 = 2    /* h is float32 instead of bf16 */
};

/* Validates the sizes and allocates the split-K partial workspace (at most
 * 16 x min(max_tokens, 64) x d pairs of floats, 32 MB when d = 4096, or the
 * largest automatic plan if bigger).  d must be a positive multiple of 256.  Selects nothing else on
 * the device.  *out receives the handle.  Host pointers. */
kvshot_status kvshot_fusion_init(int32_t d, int32_t max_tokens, kvshot_fusion_handle* out);

/* Releases the handle's device memory (synchronises the device).  NULL is a no-op. */
kvshot_status kvshot_fusion_destroy(kvshot_fusion_handle h);

/* One fusion call over `tokens` rows.
 *   n, o      bf16 [tokens][d], row-major (n ignored, and may be NULL, with CROSS_ONLY)
 *   w_g       bf16 [d][3d]: row c holds output channel c's weights over [n | o | Delta]
 *   b_g       float32 [d]
 *   w_delta   bf16 [d][d]: row c holds output channel c's weights over Delta
 *   h         [tokens][d], bf16 (float32 with KVSHOT_FUSION_OUT_FP32)
 *   g_out     nullable float32 [tokens][d]: the gate g
 * Every device pointer must be 16-byte aligned.  1 <= tokens <= max_tokens.
 * The products run on bf16 MFMA with float32 accumulation; Delta is formed in
 * float32 from the bf16 inputs and rounded to bf16 for the product. */
kvshot_status kvshot_gated_delta_fusion(kvshot_fusion_handle h, int32_t tokens, const void* n, const void* o,
                                        const void* w_g, const float* b_g, const void* w_delta, void* h_out,
                                        float* g_out, int32_t flags, void* stream);

/* Packs both weight matrices, once, into the order the fusion kernel's waves
 * load them (16-byte pieces [channel tile][segment][64-wide chunk][wave][k-step]
 * [lane]), so every weight load of a call reads 1 KB contiguous instead of
 * 32 B from each of 32 rows.  w_g, w_delta as for kvshot_gated_delta_fusion;
 * packed: bf16 [4 d^2], caller-owned, 16-byte aligned.  Queued on `stream`;
 * the packed copy is only valid for handles with the same d. */
kvshot_status kvshot_fusion_pack_weights(kvshot_fusion_handle h, const void* w_g, const void* w_delta, void* packed,
                                         void* stream);

/* kvshot_gated_delta_fusion with the weights given as the packed copy made by
 * kvshot_fusion_pack_weights (same results bit for bit; faster). */
kvshot_status kvshot_gated_delta_fusion_packed(kvshot_fusion_handle h, int32_t tokens, const void* n, const void* o,
                                               const void* packed, const float* b_g, void* h_out, float* g_out,
                                               int32_t flags, void* stream);

/* Options: KVSHOT_OPT_SPLITS (0 automatic, else 1, 2, 4, 8 or 16 workgroups
 * along the reduction; capped by the workspace), KVSHOT_OPT_PATH (the token
 * tile: 0 automatic -- 128 tokens per workgroup for calls of 128 tokens or
 * more, else 64; 1 always 64; 2 always 128, except with 8 or 16 forced
 * splits, which take 64) and KVSHOT_OPT_PROFILE (1: HIP events around each
 * kernel of every call), as for the attention handle.  Every plan computes the
 * same function; the split plan only changes the float32 summation order. */
kvshot_status kvshot_fusion_set_option(kvshot_fusion_handle h, int32_t option, int64_t value);

/* Plan of a call with `tokens` rows: reduction splits and workgroups of the
 * main kernel.  Host outputs, each nullable. */
kvshot_status kvshot_fusion_plan(kvshot_fusion_handle h, int32_t tokens, int32_t* splits, int32_t* workgroups);

/* With KVSHOT_OPT_PROFILE on: synchronises, then returns the summed event time
 * (ms) of the main kernel and of the split combine kernel since the last read,
 * and the call count; resets the sums.  Host outputs. */
kvshot_status kvshot_fusion_profile_read(kvshot_fusion_handle h, double* main_ms, double* combine_ms,
                                         int64_t* calls);

#ifdef __cplusplus
}
#endif

#endif /* KVSHOT_FUSION_H */
