"""Float64 reference for draft-step attention (test infrastructure; see package docstring).

Every function states the passage it follows.  Nothing here is blocked, fused
or reordered beyond the plain definition: gather the prefix, rotate, score,
mask, softmax, weighted sum.
"""
from __future__ import annotations

import math
from typing import Iterable, List, Optional, Sequence, Tuple

import numpy as np


# ---------------------------------------------------------------------------
# decoding
# ---------------------------------------------------------------------------

def decode(x: np.ndarray, dtype: str) -> np.ndarray:
    """Exact widening of stored values to float64.

    bf16 values are stored as raw uint16 bit patterns; a bf16 number is the
    float32 whose upper 16 bits are those bits and whose lower 16 bits are 0.
    """
    if dtype == "bf16":
        u = np.asarray(x, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
        return u.view(np.float32).astype(np.float64)
    if dtype == "fp32":
        return np.asarray(x, dtype=np.float32).astype(np.float64)
    raise ValueError(f"unknown dtype {dtype!r}")


# ---------------------------------------------------------------------------
# paged target KV (the target's per-token K/V, Sec. 2.2: "the full set of
# key/value pairs"; the paging is a storage layout, not part of the method)
# ---------------------------------------------------------------------------

def gather_prefix(pages: np.ndarray, table_row: np.ndarray, length: int, page_size: int) -> np.ndarray:
    """Logical prefix tokens 0..length-1 of one sequence, ``[length][Hkv][D]`` (stored dtype).

    Token t lives in slot ``t % page_size`` of physical page ``table_row[t // page_size]``;
    pages are laid out ``[page][kv_head][slot][D]``.  Table entries past the last
    used page are never read.
    """
    t = np.arange(int(length))
    pid = np.asarray(table_row)[t // page_size]
    return pages[pid, :, t % page_size, :]


def gather_dense(pages: np.ndarray, page_table: np.ndarray, ctx_lens: np.ndarray, page_size: int,
                 max_ctx: int, fill=0) -> np.ndarray:
    """``[B][max_ctx][Hkv][D]`` logical view of the paged pool (positions >= T_b hold ``fill``)."""
    B = page_table.shape[0]
    Hkv, D = pages.shape[1], pages.shape[3]
    out = np.full((B, max_ctx, Hkv, D), fill, dtype=pages.dtype)
    for b in range(B):
        T = int(ctx_lens[b])
        out[b, :T] = gather_prefix(pages, page_table[b], T, page_size)
    return out


# ---------------------------------------------------------------------------
# RoPE (Sec. 3.2: projected KV loses the position RoPE had encoded, so RoPE is
# re-applied; target keys in the cache are therefore already rotated, and the
# draft query / draft keys are rotated at their own positions)
# ---------------------------------------------------------------------------

def rope_inv_freq(head_dim: int, theta: float) -> np.ndarray:
    """theta_m = theta^(-2m/D), m = 0 .. D/2-1 (float64)."""
    m = np.arange(head_dim // 2, dtype=np.float64)
    return np.power(float(theta), -2.0 * m / head_dim)


def rope(x: np.ndarray, pos, theta: float) -> np.ndarray:
    """Rotate-half RoPE in float64.

    Channel m is paired with channel m + D/2 and the pair is rotated by the
    angle pos * theta_m:
        y_m       = x_m cos(a) - x_{m+D/2} sin(a)
        y_{m+D/2} = x_{m+D/2} cos(a) + x_m sin(a)
    ``pos`` broadcasts against ``x.shape[:-1]``.
    """
    x = np.asarray(x, dtype=np.float64)
    D = x.shape[-1]
    half = D // 2
    ang = np.asarray(pos, dtype=np.float64)[..., None] * rope_inv_freq(D, theta)
    c, s = np.cos(ang), np.sin(ang)
    x1, x2 = x[..., :half], x[..., half:]
    return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=-1)


# ---------------------------------------------------------------------------
# attention core (Sec. 2.2, Eq. 2: softmax re-attention of a query over K/V)
# ---------------------------------------------------------------------------

def masked_attention(q: np.ndarray, K: np.ndarray, V: np.ndarray, allowed: np.ndarray,
                     scale: float) -> Tuple[np.ndarray, np.ndarray]:
    """Softmax attention restricted to allowed columns.

    q ``[R][D]``, K/V ``[L][D]``, allowed ``[R][L]`` bool.  Returns (out ``[R][D]``,
    lse ``[R]`` natural log).  z = scale * q.k; masked scores are -inf; weights
    are exp(z - max) / sum exp(z - max); lse = max + log(sum exp(z - max)).
    Every row must have at least one allowed column.
    """
    allowed = np.asarray(allowed, dtype=bool)
    if not allowed.any(axis=1).all():
        raise ValueError("a query row has no allowed key")
    z = scale * (np.asarray(q, np.float64) @ np.asarray(K, np.float64).T)
    z = np.where(allowed, z, -np.inf)
    m = z.max(axis=1, keepdims=True)
    w = np.exp(z - m)
    s = w.sum(axis=1, keepdims=True)
    out = (w / s) @ np.asarray(V, np.float64)
    return out, m[:, 0] + np.log(s[:, 0])


# ---------------------------------------------------------------------------
# draft tree (Sec. 3.5: tree-structured drafting; a node sees its ancestors)
# ---------------------------------------------------------------------------

def tree_ancestry(parents: Sequence[int]) -> Tuple[List[set], np.ndarray]:
    """Ancestor-or-self sets and depths by walking parent links.

    parents[i] == -1 marks a root; otherwise 0 <= parents[i] < i.  Depth of a
    root is 0; depth of any node is the number of its strict ancestors.
    """
    n = len(parents)
    anc: List[set] = []
    depth = np.zeros(n, dtype=np.int64)
    for i in range(n):
        p = int(parents[i])
        if not (p == -1 or 0 <= p < i):
            raise ValueError(f"bad parent {p} for node {i}")
        s = {i}
        while p != -1:
            s.add(p)
            p = int(parents[p])
        anc.append(s)
        depth[i] = len(s) - 1
    return anc, depth


# ---------------------------------------------------------------------------
# the draft step (Sec. 3.4.1, Eq. 7 with memory M_i of App. B)
# ---------------------------------------------------------------------------

def _memory_attention(qrot, Kt, Vt, dk_rot, dv, allowed_draft, num_kv_heads, scale):
    """One sequence: qrot ``[rows][Hq][D]``, target ``[T][Hkv][D]``, draft ``[S][Hkv][D]``.

    allowed_draft ``[rows][S]``; every target column is allowed.  Query head h
    reads KV head floor(h / G), G = Hq / Hkv (grouped-query attention).
    """
    rows, Hq, D = qrot.shape
    G = Hq // num_kv_heads
    T = Kt.shape[0]
    out = np.empty((rows, Hq, D))
    lse = np.empty((rows, Hq))
    allowed = np.concatenate([np.ones((rows, T), dtype=bool), allowed_draft], axis=1)
    allowed = np.repeat(allowed, G, axis=0)          # row order (query, head in group)
    for g in range(num_kv_heads):
        K = np.concatenate([Kt[:, g], dk_rot[:, g]], axis=0)
        V = np.concatenate([Vt[:, g], dv[:, g]], axis=0)
        heads = slice(g * G, (g + 1) * G)
        o, l = masked_attention(qrot[:, heads].reshape(rows * G, D), K, V, allowed, scale)
        out[:, heads] = o.reshape(rows, G, D)
        lse[:, heads] = l.reshape(rows, G)
    return out, lse


def draft_attention_step(q, k_pages, v_pages, page_table, ctx_lens, draft_k, draft_v, step_offsets, *,
                         dtype: str, page_size: int, rope_theta: float = 1e6, softmax_scale: float = 0.0,
                         seqs: Optional[Iterable[int]] = None, pos_base=None):
    """Causal draft steps.  Returns (out ``[B][n][Hq][D]``, lse ``[B][n][Hq]``) in float64.

    Readings where the paper is silent:
      * positions are 0-based: the prefix occupies 0..T_b-1, query j of
        sequence b sits at draft step s0 + j (s0 = step_offsets[b]) and position
        T_b + s0 + j; draft key s sits at position T_b + s;
      * the draft keys are given un-rotated and are rotated at their own
        positions; target keys are already rotated and are used as stored;
      * query j sees every target key and draft keys s <= s0 + j (its own key
        included);
      * scale 1/sqrt(D) unless ``softmax_scale`` is non-zero.
    ``seqs`` restricts the computation to some sequences (other rows are NaN).
    ``pos_base[b]``, when given, replaces T_b as the position of draft step 0
    (the prefix keys are used as stored either way).
    """
    q = np.asarray(q)
    B, n, Hq, D = q.shape
    Hkv = k_pages.shape[1]
    scale = softmax_scale if softmax_scale != 0.0 else 1.0 / math.sqrt(D)
    out = np.full((B, n, Hq, D), np.nan)
    lse = np.full((B, n, Hq), np.nan)
    for b in (range(B) if seqs is None else seqs):
        T = int(ctx_lens[b])
        s0 = int(step_offsets[b])
        S = s0 + n
        Kt = decode(gather_prefix(k_pages, page_table[b], T, page_size), dtype)
        Vt = decode(gather_prefix(v_pages, page_table[b], T, page_size), dtype)
        base = T if pos_base is None else int(pos_base[b])
        qpos = base + s0 + np.arange(n)
        kpos = base + np.arange(S)
        qrot = rope(decode(q[b], dtype), qpos[:, None], rope_theta)
        dk = rope(decode(draft_k[b, :S], dtype), kpos[:, None], rope_theta)
        dv = decode(draft_v[b, :S], dtype)
        allowed = np.arange(S)[None, :] <= (s0 + np.arange(n))[:, None]
        out[b], lse[b] = _memory_attention(qrot, Kt, Vt, dk, dv, allowed, Hkv, scale)
    return out, lse


def draft_attention_tree(q, k_pages, v_pages, page_table, ctx_lens, draft_k, draft_v, parents, *,
                         dtype: str, page_size: int, rope_theta: float = 1e6, softmax_scale: float = 0.0,
                         seqs: Optional[Iterable[int]] = None, query_nodes=None, pos_base=None):
    """Tree drafting.  Returns (out ``[B][n_q][Hq][D]``, lse ``[B][n_q][Hq]``) in float64.

    Readings: node i of sequence b sits at position T_b + depth(i) (roots at
    T_b); draft key s (the key of node s) is rotated at T_b + depth(s); node i
    sees every target key and the keys of its ancestors and itself; parents[i]
    is -1 (root, forests allowed) or an earlier node.  ``parents`` is
    [B][N] over all N nodes; query row j is node ``query_nodes[b][j]`` when
    given (a tree grown level by level queries its newest level only), else
    node j.  ``pos_base[b]``, when given, replaces T_b as the position of depth 0.
    """
    q = np.asarray(q)
    B, nq, Hq, D = q.shape
    N = np.asarray(parents).shape[1]
    Hkv = k_pages.shape[1]
    scale = softmax_scale if softmax_scale != 0.0 else 1.0 / math.sqrt(D)
    out = np.full((B, nq, Hq, D), np.nan)
    lse = np.full((B, nq, Hq), np.nan)
    for b in (range(B) if seqs is None else seqs):
        T = int(ctx_lens[b])
        anc, depth = tree_ancestry(parents[b])
        nodes = np.arange(nq) if query_nodes is None else np.asarray(query_nodes[b], dtype=np.int64)
        Kt = decode(gather_prefix(k_pages, page_table[b], T, page_size), dtype)
        Vt = decode(gather_prefix(v_pages, page_table[b], T, page_size), dtype)
        base = T if pos_base is None else int(pos_base[b])
        qrot = rope(decode(q[b], dtype), (base + depth[nodes])[:, None], rope_theta)
        dk = rope(decode(draft_k[b, :N], dtype), (base + depth)[:, None], rope_theta)
        dv = decode(draft_v[b, :N], dtype)
        allowed = np.zeros((nq, N), dtype=bool)
        for j, i in enumerate(nodes):
            allowed[j, sorted(anc[int(i)])] = True
        out[b], lse[b] = _memory_attention(qrot, Kt, Vt, dk, dv, allowed, Hkv, scale)
    return out, lse


def draft_attention(case, seqs: Optional[Iterable[int]] = None):
    """Dispatch on a case object exposing the call's arrays as attributes."""
    common = dict(dtype=case.dtype, page_size=case.page_size, rope_theta=case.rope_theta,
                  softmax_scale=case.softmax_scale, seqs=seqs)
    pos_base = getattr(case, "pos_base", None)
    if case.mode == "step":
        return draft_attention_step(case.q, case.k_pages, case.v_pages, case.page_table, case.ctx_lens,
                                    case.draft_k, case.draft_v, case.step_offsets, pos_base=pos_base, **common)
    return draft_attention_tree(case.q, case.k_pages, case.v_pages, case.page_table, case.ctx_lens,
                                case.draft_k, case.draft_v, case.parents, pos_base=pos_base,
                                query_nodes=getattr(case, "query_nodes", None), **common)
