"""Seeded synthetic inputs for draft-step attention over reused target KV.

This module only *makes inputs*: random tensors, their bf16 encoding, page
tables, ragged lengths, step offsets and draft-tree parent arrays.  It holds
none of the attention arithmetic.  Both the CPU oracle (via the tests) and the
HIP path are fed the very same bit patterns produced here.

Recipe (all values N(0, 1) unless stated):
  * generator: ``numpy.random.Generator(PCG64(SeedSequence([seed, tensor_id])))``;
    float32 samples are rounded to bf16 with round-to-nearest-even on the bits;
  * target K/V are generated per sequence in logical token order and then
    scattered into physical pages, so the logical data does not depend on the
    page table;
  * pages are HND: ``pages[page][kv_head][slot][head_dim]``;
  * the page pool has ~1% spare pages; spare pages and unused tail slots are
    filled with NaN, and page-table padding is -1 (poisoning: a kernel that
    reads them, or multiplies a masked weight by them, produces NaN);
  * outlier channels (optional): for each KV head, ``n_outlier`` distinct
    channels of the target *keys* are multiplied by ``outlier_scale`` before
    rounding;
  * draft trees: node 0 is the only root, and node i > 0 picks its parent
    uniformly among earlier nodes with depth <= max_depth - 2 and fewer than
    ``max_branch`` children (so depth index <= max_depth - 1).

The shapes follow the Qwen3-8B attention geometry the paper's target model
uses (32 query heads, 8 KV heads, head_dim 128).  They are synthetic stand-ins:
no dataset, no trained weights.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import List, Optional, Sequence

import numpy as np

BF16_NAN = np.uint16(0x7FC0)

# tensor ids inside one seed's stream family
_TID_Q = 1
_TID_DK = 2
_TID_DV = 3
_TID_PERM = 4
_TID_LENS = 5
_TID_OFFS = 6
_TID_OUTLIER = 7
_TID_LOGITS = 8
_TID_PEAKS = 9
_TID_K = 1000   # + b
_TID_V = 2000   # + b
_TID_TREE = 3000  # + b


def rng_for(seed: int, tensor_id: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([int(seed), int(tensor_id)])))


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 values to bf16 (round-to-nearest-even) and return the raw uint16 bits."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32).astype(np.uint64)
    bias = np.uint64(0x7FFF) + ((u >> np.uint64(16)) & np.uint64(1))
    bits = ((u + bias) >> np.uint64(16)).astype(np.uint16)
    nan = np.isnan(x)
    if nan.any():
        bits[nan] = BF16_NAN
    return bits


def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    """Exact widening of bf16 bits to float32 (test convenience; not used by the oracle)."""
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def _normal(seed: int, tid: int, shape, chunk: int = 1 << 24) -> np.ndarray:
    g = rng_for(seed, tid)
    n = int(np.prod(shape))
    out = np.empty(n, dtype=np.float32)
    for s in range(0, n, chunk):
        e = min(n, s + chunk)
        out[s:e] = g.standard_normal(e - s, dtype=np.float32)
    return out.reshape(shape)


def _encode(x: np.ndarray, dtype: str) -> np.ndarray:
    if dtype == "bf16":
        return f32_to_bf16_bits(x)
    if dtype == "fp32":
        return np.ascontiguousarray(x, dtype=np.float32)
    raise ValueError(dtype)


def _nan_fill(dtype: str):
    return BF16_NAN if dtype == "bf16" else np.float32(np.nan)


def random_tree(seed: int, b: int, n_nodes: int, max_depth: int = 8, max_branch: int = 4) -> np.ndarray:
    """Parent array of one seeded random draft tree (node 0 is the root, parents[i] < i)."""
    g = rng_for(seed, _TID_TREE + b)
    parents = np.full(n_nodes, -1, dtype=np.int32)
    depth = np.zeros(n_nodes, dtype=np.int32)
    children = np.zeros(n_nodes, dtype=np.int32)
    for i in range(1, n_nodes):
        cand = [j for j in range(i) if depth[j] <= max_depth - 2 and children[j] < max_branch]
        if not cand:
            raise ValueError("tree capacity exhausted")
        p = cand[int(g.integers(len(cand)))]
        parents[i] = p
        depth[i] = depth[p] + 1
        children[p] += 1
    return parents


@dataclass
class DraftCase:
    """One draft-attention call's inputs (host arrays) plus its static geometry."""
    mode: str                      # "step" or "tree"
    dtype: str                     # "bf16" (uint16 bit patterns) or "fp32"
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    page_size: int
    max_draft: int
    n_new: int                     # queries per sequence (draft steps, or tree nodes)
    q: np.ndarray                  # [B][n_new][Hq][D]
    k_pages: np.ndarray            # [num_pages][Hkv][P][D]
    v_pages: np.ndarray
    page_table: np.ndarray         # int32 [B][max_pages_per_seq], padding -1
    ctx_lens: np.ndarray           # int32 [B]
    draft_k: np.ndarray            # [B][max_draft][Hkv][D]  (pre-RoPE)
    draft_v: np.ndarray
    step_offsets: Optional[np.ndarray] = None   # int32 [B] (step mode)
    parents: Optional[np.ndarray] = None        # int32 [B][n_nodes] (tree mode; n_nodes == n_new without query_nodes)
    query_nodes: Optional[np.ndarray] = None    # int32 [B][n_new]: tree node of each query row (tree mode)
    pos_base: Optional[np.ndarray] = None       # int32 [B]: position of draft step 0 / depth 0 (default ctx_lens)
    rope_theta: float = 1e6
    softmax_scale: float = 0.0                  # 0 -> 1/sqrt(head_dim)
    seed: int = 0
    name: str = ""
    meta: dict = field(default_factory=dict)

    @property
    def batch(self) -> int:
        return int(self.q.shape[0])

    @property
    def num_pages(self) -> int:
        return int(self.k_pages.shape[0])

    @property
    def max_pages_per_seq(self) -> int:
        return int(self.page_table.shape[1])

    @property
    def scale(self) -> float:
        return self.softmax_scale if self.softmax_scale != 0.0 else 1.0 / float(np.sqrt(self.head_dim))

    def draft_len(self, b: int) -> int:
        """Number of draft keys sequence b's queries can see in total."""
        if self.mode == "step":
            return int(self.step_offsets[b]) + self.n_new
        return int(self.parents.shape[1])


def build_pages(seed: int, ctx_lens: Sequence[int], num_kv_heads: int, head_dim: int, page_size: int,
                dtype: str, *, shuffle: bool = True, spare_frac: float = 0.01, poison: bool = True,
                n_outlier: int = 0, outlier_scale: float = 8.0, min_pages_per_seq: int = 1,
                max_pages_per_seq: Optional[int] = None):
    """Target K/V pools, page table and per-sequence logical K/V (float32, pre-rounding ignored).

    Returns (k_pages, v_pages, page_table).
    """
    B = len(ctx_lens)
    npages = [max(min_pages_per_seq, -(-int(t) // page_size)) if t > 0 else 0 for t in ctx_lens]
    used = int(sum(npages))
    spare = max(1, int(np.ceil(used * spare_frac)))
    pool = used + spare
    mpps = max_pages_per_seq if max_pages_per_seq is not None else max(1, max(npages) if npages else 1)
    if mpps < max(npages):
        raise ValueError("max_pages_per_seq too small")
    perm = rng_for(seed, _TID_PERM).permutation(pool).astype(np.int32) if shuffle \
        else np.arange(pool, dtype=np.int32)
    edt = np.uint16 if dtype == "bf16" else np.float32
    fill = _nan_fill(dtype) if poison else edt(0)
    k_pages = np.full((pool, num_kv_heads, page_size, head_dim), fill, dtype=edt)
    v_pages = np.full((pool, num_kv_heads, page_size, head_dim), fill, dtype=edt)
    page_table = np.full((B, mpps), -1, dtype=np.int32)
    outl = None
    if n_outlier > 0:
        g = rng_for(seed, _TID_OUTLIER)
        outl = np.stack([g.choice(head_dim, size=n_outlier, replace=False) for _ in range(num_kv_heads)])
    cursor = 0
    for b, T in enumerate(ctx_lens):
        T = int(T)
        if npages[b] == 0:
            continue
        ids = perm[cursor:cursor + npages[b]]
        cursor += npages[b]
        page_table[b, :npages[b]] = ids
        if T == 0:
            continue
        K = _normal(seed, _TID_K + b, (T, num_kv_heads, head_dim))
        V = _normal(seed, _TID_V + b, (T, num_kv_heads, head_dim))
        if outl is not None:
            for h in range(num_kv_heads):
                K[:, h, outl[h]] *= np.float32(outlier_scale)
        Ke = _encode(K, dtype)
        Ve = _encode(V, dtype)
        t = np.arange(T)
        k_pages[ids[t // page_size], :, t % page_size, :] = Ke
        v_pages[ids[t // page_size], :, t % page_size, :] = Ve
    return k_pages, v_pages, page_table


def make_case(*, mode: str = "step", batch: int = 1, ctx_lens=None, n_new: int = 4,
              num_q_heads: int = 32, num_kv_heads: int = 8, head_dim: int = 128, page_size: int = 16,
              dtype: str = "bf16", seed: int = 0, max_draft: Optional[int] = None, step_offsets=None,
              parents=None, shuffle: bool = True, poison: bool = True, n_outlier: int = 0,
              outlier_scale: float = 8.0, rope_theta: float = 1e6, softmax_scale: float = 0.0, name: str = "",
              max_pages_per_seq: Optional[int] = None) -> DraftCase:
    if ctx_lens is None:
        ctx_lens = [256] * batch
    ctx_lens = np.asarray(ctx_lens, dtype=np.int32)
    B = len(ctx_lens)
    if mode == "step":
        if step_offsets is None:
            step_offsets = np.zeros(B, dtype=np.int32)
        step_offsets = np.asarray(step_offsets, dtype=np.int32)
        need = int((step_offsets + n_new).max())
    else:
        if parents is None:
            parents = np.stack([random_tree(seed, b, n_new) for b in range(B)])
        parents = np.asarray(parents, dtype=np.int32)
        need = n_new
    if max_draft is None:
        max_draft = need
    if max_draft < need:
        raise ValueError("max_draft too small")
    k_pages, v_pages, page_table = build_pages(seed, ctx_lens, num_kv_heads, head_dim, page_size, dtype,
                                               shuffle=shuffle, poison=poison, n_outlier=n_outlier,
                                               outlier_scale=outlier_scale, max_pages_per_seq=max_pages_per_seq)
    q = _encode(_normal(seed, _TID_Q, (B, n_new, num_q_heads, head_dim)), dtype)
    dk = _encode(_normal(seed, _TID_DK, (B, max_draft, num_kv_heads, head_dim)), dtype)
    dv = _encode(_normal(seed, _TID_DV, (B, max_draft, num_kv_heads, head_dim)), dtype)
    if poison:
        # draft slots no query can see are poison too
        for b in range(B):
            s_len = int(step_offsets[b]) + n_new if mode == "step" else n_new
            dk[b, s_len:] = _nan_fill(dtype)
            dv[b, s_len:] = _nan_fill(dtype)
    return DraftCase(mode=mode, dtype=dtype, num_q_heads=num_q_heads, num_kv_heads=num_kv_heads,
                     head_dim=head_dim, page_size=page_size, max_draft=max_draft, n_new=n_new, q=q,
                     k_pages=k_pages, v_pages=v_pages, page_table=page_table, ctx_lens=ctx_lens,
                     draft_k=dk, draft_v=dv, step_offsets=step_offsets if mode == "step" else None,
                     parents=parents if mode == "tree" else None, rope_theta=rope_theta,
                     softmax_scale=softmax_scale, seed=seed, name=name)


# ---------------------------------------------------------------------------
# The five workload shapes (Qwen3-8B-shaped synthetic stand-ins).
# ---------------------------------------------------------------------------

def ragged_lengths(seed: int, batch: int, lo: int, hi: int) -> np.ndarray:
    return rng_for(seed, _TID_LENS).integers(lo, hi + 1, size=batch).astype(np.int32)


def ragged_offsets(seed: int, batch: int, hi: int) -> np.ndarray:
    return rng_for(seed, _TID_OFFS).integers(0, hi + 1, size=batch).astype(np.int32)


WORKLOADS = {
    # tiny fp32 case: batch 1, ctx 256, k=4 causal draft steps, one contiguous 256-token page
    "tiny_fp32_ctx256": dict(mode="step", ctx_lens=[256], n_new=4, dtype="fp32", page_size=256,
                             shuffle=False, seed=1001),
    # one Qwen3-8B-shaped sequence, ctx 4096, k=8, outlier key channels, shuffled 16-token pages
    "single_ctx4096_k8": dict(mode="step", ctx_lens=[4096], n_new=8, dtype="bf16", page_size=16,
                              n_outlier=4, seed=1002),
    # ragged batch of 16, ctx ~ U[512, 8192], k=6, per-sequence step offsets U{0..8}
    "ragged_b16_k6": dict(mode="step", n_new=6, dtype="bf16", page_size=16, seed=1003, max_draft=16),
    # long range: batch 64 x ctx 32768, k=8 (too large for host generation in tests)
    "long_b64_ctx32k_k8": dict(mode="step", ctx_lens=[32768] * 64, n_new=8, dtype="bf16", page_size=16,
                               seed=1004),
    # draft tree: batch 8 x ctx 16384, 60-node tree (depth <= 8, branching <= 4)
    "tree_b8_ctx16k_n60": dict(mode="tree", ctx_lens=[16384] * 8, n_new=60, dtype="bf16", page_size=16,
                               seed=1005),
}


def workload(name: str, **overrides) -> DraftCase:
    spec = dict(WORKLOADS[name])
    spec.update(overrides)
    if name.startswith("ragged") and "ctx_lens" not in overrides:
        spec["ctx_lens"] = ragged_lengths(spec["seed"], 16, 512, 8192)
        spec["step_offsets"] = ragged_offsets(spec["seed"], 16, 8)
    return make_case(name=name, **spec)


def algorithmic_bytes(case_or_dims, *, elem_bytes: int = 2) -> int:
    """Unique bytes one call must move: target K+V once, q, draft K/V seen, page-table entries, output."""
    c = case_or_dims
    D, Hkv, Hq, P = c.head_dim, c.num_kv_heads, c.num_q_heads, c.page_size
    tot = 0
    for b in range(c.batch):
        T = int(c.ctx_lens[b])
        tot += 2 * T * Hkv * D * elem_bytes
        tot += -(-T // P) * 4
        tot += 2 * c.draft_len(b) * Hkv * D * elem_bytes
    tot += 2 * c.batch * c.n_new * Hq * D * elem_bytes  # q in, out
    return tot


# ---------------------------------------------------------------------------
# gated delta fusion inputs (the hybrid drafter's fusion step, Sec. 3.4.1):
# self- and cross-attention outputs of one drafter layer and the fusion's
# weights, in the linear-layer storage of App. B's shapes.
# ---------------------------------------------------------------------------

_TID_FN, _TID_FO, _TID_FWG, _TID_FB, _TID_FWD = 4001, 4002, 4003, 4004, 4005


@dataclass
class FusionCase:
    """Inputs of one fusion call: bf16 bits for activations and weights, float32 bias."""
    tokens: int
    d: int
    n: np.ndarray         # uint16 [tokens][d]
    o: np.ndarray         # uint16 [tokens][d]
    w_g: np.ndarray       # uint16 [d][3d]
    b_g: np.ndarray       # float32 [d]
    w_delta: np.ndarray   # uint16 [d][d]


def fusion_case(tokens: int, d: int, seed: int = 2001, gate_bias_mean: float = -2.0) -> FusionCase:
    """Seeded fusion inputs: n, o ~ N(0, 1); W_g ~ N(0, 1/(3d)); W_Delta ~ N(0, 1/d);
    b_g ~ N(gate_bias_mean, 1) (a mostly shut gate, as trained gates settle low)."""
    n = f32_to_bf16_bits(_normal(seed, _TID_FN, (tokens, d)))
    o = f32_to_bf16_bits(_normal(seed, _TID_FO, (tokens, d)))
    w_g = f32_to_bf16_bits(_normal(seed, _TID_FWG, (d, 3 * d)) / np.float32(np.sqrt(3.0 * d)))
    b_g = (_normal(seed, _TID_FB, (d,)) + np.float32(gate_bias_mean)).astype(np.float32)
    w_delta = f32_to_bf16_bits(_normal(seed, _TID_FWD, (d, d)) / np.float32(np.sqrt(float(d))))
    return FusionCase(tokens=tokens, d=d, n=n, o=o, w_g=w_g, b_g=b_g, w_delta=w_delta)


# Fusion workloads: d = 4096 is the Qwen3-8B hidden size the drafter shares.
FUSION_WORKLOADS = {
    # one draft step of a 64-sequence batch: 64 tokens
    "fusion_t64_d4096": dict(tokens=64, d=4096, seed=2001),
    # every node of eight 60-node draft trees in one call: 480 tokens
    "fusion_t480_d4096": dict(tokens=480, d=4096, seed=2002),
}


def fusion_algorithmic(tokens: int, d: int) -> dict:
    """Unique bytes (bf16 activations and weights, float32 bias, bf16 output) and flops of one call."""
    weights = (3 * d * d + d * d) * 2 + d * 4
    acts = 2 * tokens * d * 2 + tokens * d * 2
    flops = 2 * tokens * d * (3 * d) + 2 * tokens * d * d
    return dict(bytes=weights + acts, flops=flops)


# ---------------------------------------------------------------------------
# projected-KV cache builder (KV-only drafters): L_s source layer caches and the
# tokens whose projected K/V enter the drafter's cache
# ---------------------------------------------------------------------------

_TID_PPERM, _TID_PNEW, _TID_PWK, _TID_PWV = 5001, 5002, 5003, 5004
_TID_PSRC = 6_000_000   # + (2 layer + kv) * 100_000 + b


@dataclass
class KvProjCase:
    """Inputs of one projection call (bf16 bits; pools [page][Hkv][P][D])."""
    k_src: List[np.ndarray]
    v_src: List[np.ndarray]
    page_table: np.ndarray     # int32 [B][max_pages_per_seq], -1 padding
    ctx_lens: np.ndarray       # int32 [B]
    token_seq: np.ndarray      # int32 [N]
    token_pos: np.ndarray      # int32 [N]
    w_k: np.ndarray            # uint16 [d_kv][L d_kv]
    w_v: np.ndarray
    page_size: int
    rope_theta: float = 1e6

    @property
    def layers(self) -> int:
        return len(self.k_src)

    @property
    def num_pages(self) -> int:
        return int(self.k_src[0].shape[0])

    @property
    def num_kv_heads(self) -> int:
        return int(self.k_src[0].shape[1])

    @property
    def max_pages_per_seq(self) -> int:
        return int(self.page_table.shape[1])

    @property
    def n_tokens(self) -> int:
        return int(self.token_seq.shape[0])


def kvproj_case(*, batch: int, ctx_lens, new_tokens, layers: int = 3, num_kv_heads: int = 8, head_dim: int = 128,
                page_size: int = 16, seed: int = 3001, shuffle: bool = True, poison: bool = True,
                rope_theta: float = 1e6) -> KvProjCase:
    """Source caches of ``layers`` sampled target layers and the tokens to project.

    Sequence b holds ctx_lens[b] tokens in every source layer (N(0, 1) K and V,
    generated per layer in logical order and scattered through one shared,
    permuted page table; ~1% spare pages and unused slots hold NaN).  The tokens
    to project are the last new_tokens[b] positions of each sequence (all of them
    at prefill), sequence-major.  W_K, W_V ~ N(0, 1 / (layers d_kv)) so the
    projected vectors have unit scale.
    """
    ctx = [int(t) for t in ctx_lens]
    new = [int(t) for t in new_tokens]
    assert len(ctx) == batch and len(new) == batch and all(0 <= n <= t for n, t in zip(new, ctx))
    npages = [-(-t // page_size) for t in ctx]
    pool = int(sum(npages)) + max(1, int(np.ceil(sum(npages) * 0.01)))
    perm = rng_for(seed, _TID_PPERM).permutation(pool).astype(np.int32) if shuffle \
        else np.arange(pool, dtype=np.int32)
    mpps = max(1, max(npages))
    table = np.full((batch, mpps), -1, dtype=np.int32)
    fill = BF16_NAN if poison else np.uint16(0)
    k_src = [np.full((pool, num_kv_heads, page_size, head_dim), fill, np.uint16) for _ in range(layers)]
    v_src = [np.full((pool, num_kv_heads, page_size, head_dim), fill, np.uint16) for _ in range(layers)]
    cursor = 0
    for b, T in enumerate(ctx):
        ids = perm[cursor:cursor + npages[b]]
        cursor += npages[b]
        table[b, :npages[b]] = ids
        t = np.arange(T)
        for layer in range(layers):
            for kv, pools in ((0, k_src), (1, v_src)):
                x = f32_to_bf16_bits(_normal(seed, _TID_PSRC + (2 * layer + kv) * 100_000 + b,
                                             (T, num_kv_heads, head_dim)))
                pools[layer][ids[t // page_size], :, t % page_size, :] = x
    seq = np.concatenate([np.full(n, b, np.int32) for b, n in enumerate(new)]) if sum(new) else np.zeros(0, np.int32)
    pos = np.concatenate([np.arange(t - n, t, dtype=np.int32) for t, n in zip(ctx, new)]) if sum(new) \
        else np.zeros(0, np.int32)
    d_kv = num_kv_heads * head_dim
    sd = np.float32(1.0 / np.sqrt(layers * d_kv))
    w_k = f32_to_bf16_bits(_normal(seed, _TID_PWK, (d_kv, layers * d_kv)) * sd)
    w_v = f32_to_bf16_bits(_normal(seed, _TID_PWV, (d_kv, layers * d_kv)) * sd)
    return KvProjCase(k_src=k_src, v_src=v_src, page_table=table, ctx_lens=np.asarray(ctx, np.int32),
                      token_seq=seq.astype(np.int32), token_pos=pos.astype(np.int32), w_k=w_k, w_v=w_v,
                      page_size=page_size, rope_theta=rope_theta)


def verify_counts(seed: int, batch: int, hi: int = 8) -> np.ndarray:
    """Tokens entering the cache after one verification, per sequence: U{1 .. hi} (seeded)."""
    return rng_for(seed, _TID_PNEW).integers(1, hi + 1, size=batch).astype(np.int32)


# Projection workloads: Qwen3-8B KV geometry (8 KV heads x 128, d_kv = 1024), L_s = 3
# sampled layers (App. A), paged at 16 tokens, 64 sequences of 32K tokens (the
# long-range attention workload's cache).  The bench builds these on the device.
KVPROJ_WORKLOADS = {
    # building the whole projected cache of a 64 x 32K batch (prefill): 2,097,152 tokens
    "kvproj_prefill_b64_t32k": dict(batch=64, ctx=32768, new="all", seed=3101),
    # one verification's accepted tokens entering the cache: U{1..8} per sequence
    "kvproj_verify_b64_t32k": dict(batch=64, ctx=32768, new="verify", seed=3102),
}


def kvproj_algorithmic(n_tokens: int, layers: int = 3, d_kv: int = 1024) -> dict:
    """Unique bytes (bf16 source vectors, weights, projected output) and flops of one call."""
    src = 2 * n_tokens * layers * d_kv * 2
    weights = 2 * d_kv * layers * d_kv * 2
    out = 2 * n_tokens * d_kv * 2
    flops = 2 * 2 * n_tokens * d_kv * layers * d_kv
    return dict(bytes=src + weights + out, flops=flops, src=src, weights=weights, out=out)


# ---------------------------------------------------------------------------
# drafting metrics: per-verification accepted draft lengths
# ---------------------------------------------------------------------------

# Step-wise acceptance rates alpha_0 .. alpha_6 of the 1-layer gated KV drafter
# initialised from a checkpoint (App. C, table of complete step-wise rates).
GATED_KV_CKPT_RATES = (0.665, 0.603, 0.573, 0.553, 0.537, 0.525, 0.514)

ACCEPT_WORKLOADS = {
    # 64M verification records (one per sequence and verification), K = 7 draft steps: each
    # step accepted with probability alpha_k while the earlier ones were
    "accept_n64m_k7": dict(n=1 << 26, K=7, rates=GATED_KV_CKPT_RATES, seed=4101),
}


# ---------------------------------------------------------------------------
# draft-tree growth: drafter logits over the vocabulary
# ---------------------------------------------------------------------------

def draft_logits(seed: int, rows: int, vocab: int, *, dtype: str = "bf16", sigma: float = 2.0, peaks: int = 8,
                 peak_max: float = 12.0, grid: float = None, stream: int = 0) -> np.ndarray:
    """Seeded synthetic drafter logits [rows][vocab]: a sigma * N(0, 1) background with `peaks` random
    tokens per row raised by U(0, peak_max) -- a peaked next-token distribution whose top tokens carry
    most of the mass.  ``grid`` rounds every logit to a multiple of it (many equal logits); ``stream``
    selects an independent draw for the same seed (one per tree level)."""
    x = _normal(seed, _TID_LOGITS + 1000 * stream, (rows, vocab)) * np.float32(sigma)
    if peaks:
        g = rng_for(seed, _TID_PEAKS + 1000 * stream)
        idx = g.integers(0, vocab, size=(rows, peaks))
        x[np.arange(rows)[:, None], idx] += g.uniform(0.0, peak_max, size=(rows, peaks)).astype(np.float32)
    if grid:
        x = np.round(x / np.float32(grid)) * np.float32(grid)
    return _encode(x.astype(np.float32), dtype)


TREEGROW_WORKLOADS = {
    # tree (8, 10, 60) of Sec. 3.5 for a batch of 8 sequences over Qwen3-8B's vocabulary: level 0
    # expands the root (8 rows), levels 1..7 the 10-node frontiers (80 rows each), bf16 logits
    "treegrow_b8_v152k_d8k10n60": dict(batch=8, vocab=151936, depth=8, k=10, n=60, dtype="bf16", seed=5101),
}


def treegrow_levels(spec: dict, *, vocab: int = None, batch: int = None):
    """Per level d the logits [batch][F_d][vocab] (F_0 = 1, else k) of a tree-growth workload."""
    V = vocab or spec["vocab"]
    B = batch or spec["batch"]
    out = []
    for d in range(spec["depth"]):
        F = 1 if d == 0 else spec["k"]
        out.append(draft_logits(spec["seed"], B * F, V, dtype=spec["dtype"], stream=d).reshape(B, F, V))
    return out


def treegrow_algorithmic(spec: dict) -> dict:
    """Bytes one growth step must move: every level's logits once, plus the level outputs."""
    B, V, depth, k, n = spec["batch"], spec["vocab"], spec["depth"], spec["k"], spec["n"]
    eb = 2 if spec["dtype"] == "bf16" else 4
    rows = B * (1 + (depth - 1) * k)
    logits = rows * V * eb
    small = rows * k * 8 + depth * B * k * 12 + B * n * 16
    return dict(bytes=logits + small, logits=logits, rows=rows)
