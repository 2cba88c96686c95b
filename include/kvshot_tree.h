/*
 * kvshot_tree.h -- C ABI of level-wise draft-tree growth on MI355X (gfx950).
 *
 * KVShot (arXiv 2604.26412) drafts trees of shape (8, 10, 60) -- depth 8,
 * top-k 10 at each level, at most 60 candidate tokens (Sec. 3.5) -- and
 * verifies them in one target pass; the tree's parent array is what
 * kvshot_draft_attn_tree takes.  The paper gives only the shape; these calls
 * implement level-wise best-first growth:
 *   1. kvshot_topk_logprobs: for every frontier node's drafter logits z over
 *      the vocabulary, the top-k tokens by logit (ties: smaller token id) and
 *      their log-probabilities z - logsumexp(z);
 *   2. kvshot_tree_expand: per sequence, the k best children of the frontier,
 *      a child (f, v) scoring score(f) + logprob (ties: smaller frontier index,
 *      then better proposal rank);
 *   (kvshot_tree_level does 1 and 2 for one level in a single launch.)
 *   3. kvshot_tree_select: per sequence, the n best frontier nodes of all levels
 *      (ties: shallower, then earlier in its level) as a tree ordered by depth,
 *      then rank, with parents indexing that order (-1: a child of the root).
 * Log-probabilities are never positive, so a child never outscores its parent:
 * the selected set contains every selected node's parent.
 *
 * Arithmetic: logits bf16 or float32, log-sum-exp and scores in float32.
 * Conventions as in kvshot_draft_attn.h: device pointers unless marked (host);
 * the caller owns every array until the work queued on `stream` has finished;
 * argument errors are returned before anything is queued; no call allocates.
 * Logits must be finite.
 */
#ifndef KVSHOT_TREE_H
#define KVSHOT_TREE_H

#include <stdint.h>

#include "kvshot_draft_attn.h"

#ifdef __cplusplus
extern "C" {
#endif

/* Bytes of workspace kvshot_topk_logprobs needs for `rows` rows of `vocab`
 * logits: 0 when a row fits one chunk of 16384 logits, else 136 bytes per
 * row and chunk.  -1 for rows < 1, vocab < 1 or vocab > 64 * 16384. */
int64_t kvshot_topk_workspace_bytes(int32_t rows, int32_t vocab);

/* logits    [rows] rows of `vocab` values, row r at logits + r * row_stride
 *           (elements); dtype KVSHOT_BF16 or KVSHOT_FP32
 * tokens    int32 [rows][k], logprobs float32 [rows][k], best first
 * workspace device scratch of workspace_bytes >= kvshot_topk_workspace_bytes
 *           (may be null when that is 0), 8-byte aligned; its contents on entry
 *           do not matter and are left undefined
 * 1 <= k <= 16, k <= vocab <= 64 * 16384, rows >= 1, row_stride >= vocab, logits
 * aligned to its element size.  Rows that start on 16-byte boundaries (logits
 * 16-byte aligned, row_stride a multiple of 8 bf16 / 4 float32 values) are read
 * with 16-byte loads, others element by element.
 * One or two launches on `stream`. */
kvshot_status kvshot_topk_logprobs(const void* logits, int32_t dtype, int32_t rows, int32_t vocab,
                                   int64_t row_stride, int32_t k, int32_t* tokens, float* logprobs,
                                   void* workspace, int64_t workspace_bytes, void* stream);

/* scores    float32 [batch][frontier]: the frontier's scores (zeros for the root)
 * tokens    int32 [batch][frontier][proposals], logprobs float32 [batch][frontier][proposals]
 *           (the frontier nodes' kvshot_topk_logprobs rows)
 * next_parent int32 [batch][k] (index in the frontier), next_tokens int32 [batch][k],
 * next_scores float32 [batch][k]: the next frontier, best first
 * 1 <= frontier <= 16, 1 <= proposals <= 16, 1 <= k <= frontier * proposals, k <= 16. */
kvshot_status kvshot_tree_expand(int32_t batch, int32_t frontier, int32_t proposals, int32_t k, const float* scores,
                                 const int32_t* tokens, const float* logprobs, int32_t* next_parent,
                                 int32_t* next_tokens, float* next_scores, void* stream);

/* Bytes of workspace kvshot_tree_level needs: 17 * 256 bytes of counters per
 * sequence, then 136 bytes per frontier row and per (frontier row, chunk of
 * 16384 logits).  -1 for batch < 1, frontier outside 1..16, vocab < 1 or
 * vocab > 64 * 16384. */
int64_t kvshot_tree_level_workspace_bytes(int32_t batch, int32_t frontier, int32_t vocab);

/* One level of growth in one launch: the same result as kvshot_topk_logprobs
 * over the batch * frontier rows followed by kvshot_tree_expand with
 * proposals = k (bit for bit: the same float32 operations in the same order).
 * logits    row b * frontier + f (frontier node f of sequence b) at
 *           logits + (b * frontier + f) * row_stride, `vocab` values each;
 *           dtype, alignment and row_stride as for kvshot_topk_logprobs
 * scores    float32 [batch][frontier]: the frontier's scores (zeros for the root)
 * next_parent, next_tokens int32 [batch][k], next_scores float32 [batch][k]
 * workspace device scratch of workspace_bytes >= kvshot_tree_level_workspace_bytes,
 *           256-byte aligned.  Its counters must be zero before the first call
 *           (fill the workspace with zeros once); every call leaves them zero.
 *           Calls with any frontier size may share a workspace sized for the
 *           largest; a call with another batch size needs a workspace of its
 *           own (or one filled with zeros again).  Calls that share a
 *           workspace must not run concurrently.
 * 1 <= frontier <= 16, 1 <= k <= 16, k <= vocab <= 64 * 16384. */
kvshot_status kvshot_tree_level(const void* logits, int32_t dtype, int32_t batch, int32_t frontier, int32_t vocab,
                                int64_t row_stride, int32_t k, const float* scores, int32_t* next_parent,
                                int32_t* next_tokens, float* next_scores, void* workspace, int64_t workspace_bytes,
                                void* stream);

/* level_parent, level_tokens int32 [depth][batch][k], level_scores float32 [depth][batch][k]:
 *           kvshot_tree_expand's outputs of levels 1 .. depth, each level one contiguous
 *           [batch][k] block (level 1's parents are ignored)
 * parents, tokens, depths int32 [batch][n], scores float32 [batch][n]: the tree
 * 1 <= depth, 1 <= k <= 16, depth * k <= 256, 1 <= n <= depth * k. */
kvshot_status kvshot_tree_select(int32_t batch, int32_t depth, int32_t k, int32_t n, const int32_t* level_parent,
                                 const int32_t* level_tokens, const float* level_scores, int32_t* parents,
                                 int32_t* tokens, int32_t* depths, float* scores, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* KVSHOT_TREE_H */
