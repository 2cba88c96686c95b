"""CPU oracle for draft-step attention over reused target KV -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and ``bench.py``'s ``cpu_baseline``
leg may import or call anything in this package.  The product path (the HIP
library and its Python binding) never imports it and shares no code with it.

What it computes (KVShot, arXiv 2604.26412):
  * a drafter query re-attends the target's un-aggregated K/V with its own
    query (Sec. 2.2, Eq. 2);
  * the cross-attention memory of a draft step is the target KV of the verified
    prefix plus the drafter's own KV for later draft positions, laid out like
    an ordinary autoregressive KV cache (Sec. 3.4.1, Eq. 7; App. B,
    "Cross-attention memory");
  * draft tokens may be organised as a tree (Sec. 3.5, tree shape (8, 10, 60)).

The method reaches plain masked softmax attention exactly, so the oracle is
that definition written out in float64 NumPy, with explicit masks and its own
page gather.  Conventions the paper leaves open (softmax scale, RoPE variant,
draft positions, diagonal inclusivity, tree semantics, GQA mapping) are fixed
by the readings listed in each function's docstring.

Parity status per function:
  * ``masked_attention``        -- pinned (closed forms, brute force, SDPA reduction)
  * ``gather_prefix``           -- pinned (scatter/gather round trip, bit-exact)
  * ``rope``                    -- pinned for internal consistency (identity at 0,
                                   norm, relative position, complex form); the
                                   choice of the rotate-half variant itself is a
                                   convention: parity unpinned against the paper
  * ``tree_ancestry``           -- pinned (chain == causal, star == self, brute walk)
  * ``draft_attention_step`` / ``draft_attention_tree`` -- pinned through the
    above plus step-by-step == folded and page-permutation invariance; the
    softmax scale (1/sqrt(D)) and GQA head mapping are conventions:
    parity unpinned against the paper.
  * ``fusion.gated_delta_fusion`` -- the hybrid drafter's gated delta rule
    (Sec. 3.4.1, Eqs. (delta) and (fusion)); pinned (gate shut gives n, gate
    open with W_Delta = I gives o, block identity of [n; o; Delta], unit
    Delta selects a column); the cross-only variant (n read as zero) is a
    reading: parity unpinned.
  * ``kvproj.project_kv`` -- the projected-KV cache builder of KV-only
    drafters (Sec. 3.2, linear projection of the L_s sampled layers' KV and
    its RoPE-fix variant; App. A, L_s = 3); pinned (selection matrix returns
    a layer's KV bit for bit, scalar brute force, closed-form rotation of a
    unit key, linearity, page-permutation invariance).  The stacking order
    and the rotation of the projected key at the token's position are
    readings: parity unpinned against the paper.
  * ``metrics`` -- step-wise acceptance rates, retention and MAT (Sec. 3.1,
    Metrics); pinned by the paper's complete acceptance-rate table (App. C),
    the printed retention ratios and a telescoping identity.  Reading
    conditional rates from accepted lengths is unpinned beyond that identity.
  * ``tree_grow`` -- level-wise growth of the (8, 10, 60) draft tree (Sec.
    3.5): row-wise top-k with log-softmax, best-first frontier selection,
    final selection of the n best nodes.  The selection rule is a reading
    (the paper gives the shape only): parity unpinned against the paper;
    pinned by a plain scan, a closed-form two-token example, the greedy
    chain at k = 1, one level against a brute force over the whole
    vocabulary, and closure / order / optimality invariants.
"""
from .attention import (  # noqa: F401
    decode,
    gather_prefix,
    rope,
    rope_inv_freq,
    masked_attention,
    tree_ancestry,
    draft_attention_step,
    draft_attention_tree,
    draft_attention,
    gather_dense,
)
from .fusion import gated_delta_fusion, sigmoid  # noqa: F401,E402
from .kvproj import project_kv, scatter_tokens, stacked_layers  # noqa: F401,E402
from .metrics import acceptance_counts, acceptance_rates, mat_from_alphas, retention  # noqa: F401,E402
from .tree_grow import finalize as tree_finalize, grow_level, grow_tree, log_softmax_topk  # noqa: F401,E402
