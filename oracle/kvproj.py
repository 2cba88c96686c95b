"""Float64 reference for the projected-KV cache builder (test infrastructure).

Sec. 3.2, KV-only reuse, the "linear projection" injection and its
"Proj + RoPE fix" variant; App. A ("Target KV layers"): L_s = 3 sampled
target layers.

For every token t that enters the drafter's cache (a prompt token at prefill,
a verified token after each verification), the K (and V) vectors of the L_s
sampled target layers are stacked into one vector of length L_s d_kv and mapped
back to one layer's width by a learned matrix in R^{d_kv x L_s d_kv}:

    k'_t = W_K^proj [k_t^(1); ...; k_t^(L_s)]      v'_t = W_V^proj [v_t^(1); ...; v_t^(L_s)]

and, in the RoPE-fix variant, k'_t is rotated at the token's position t
(values are never rotated).  The projected K/V are written into the drafter's
paged cache, which the draft-step attention then reads as its prefix.

Readings (the paper gives the matrices' shapes and the words above, not a
layout or a formula for the rotation):
  * stacking order: layer-major in the order the layers are given, each layer
    flattened head-major, so input index  l d_kv + h D + d  is channel d of KV
    head h of the l-th given layer; output index  h D + d  is channel d of
    head h of the projected cache.  Row c of W holds output channel c's
    weights (the usual linear-layer storage);
  * the rotation is the draft path's rotate-half RoPE at the token's absolute
    position, applied to the projected key as computed -- the source keys are
    used as stored (a target cache that keeps keys already rotated gives
    rotated-then-projected-then-rotated keys; one that keeps them unrotated
    gives a plain rotated projection);
  * pages: token t of sequence b is slot t % P of page page_table[b][t // P],
    pages laid out [page][kv_head][slot][D], for the source layers and for the
    destination alike.

Pins (tests/test_oracle_kvproj_pins.py): a selection matrix returns the chosen
layer's stored KV bit for bit (layer order and head layout); a scalar
brute-force loop on tiny shapes; the closed form of the rotation of a unit key;
values untouched by the RoPE flag; linearity in W; invariance under a
permutation of the physical pages; scatter-then-gather round trip; the paper's
shapes for Qwen3-8B (d_kv = 8 x 128, L_s = 3).
"""
from __future__ import annotations

from typing import Optional, Sequence, Tuple

import numpy as np

from .attention import decode, rope


def stacked_layers(pages: Sequence[np.ndarray], page_table: np.ndarray, token_seq: np.ndarray,
                   token_pos: np.ndarray, page_size: int, dtype: str = "bf16") -> np.ndarray:
    """``[N][L_s d_kv]`` float64: the L_s layers' vectors of each token, stacked layer-major.

    pages: L_s pools ``[num_pages][Hkv][P][D]`` (stored dtype); token i is
    position ``token_pos[i]`` of sequence ``token_seq[i]``.
    """
    seq = np.asarray(token_seq, dtype=np.int64)
    pos = np.asarray(token_pos, dtype=np.int64)
    pid = np.asarray(page_table)[seq, pos // page_size]
    slot = pos % page_size
    parts = []
    for pool in pages:
        x = decode(pool[pid, :, slot, :], dtype)           # [N][Hkv][D]
        parts.append(x.reshape(x.shape[0], -1))            # head-major flattening
    return np.concatenate(parts, axis=1)


def project_kv(k_pages: Sequence[np.ndarray], v_pages: Sequence[np.ndarray], page_table: np.ndarray,
               token_seq: np.ndarray, token_pos: np.ndarray, w_k: np.ndarray, w_v: np.ndarray, *,
               page_size: int, theta: float, rope_keys: bool = True, dtype: str = "bf16",
               w_dtype: Optional[str] = "bf16") -> Tuple[np.ndarray, np.ndarray]:
    """Projected keys and values ``[N][Hkv][D]`` in float64 (Sec. 3.2, linear projection).

    w_k, w_v: ``[d_kv][L_s d_kv]`` (stored dtype ``w_dtype``, or float arrays
    when ``w_dtype`` is None).  rope_keys: the RoPE-fix variant.
    """
    wk = decode(w_k, w_dtype) if w_dtype else np.asarray(w_k, dtype=np.float64)
    wv = decode(w_v, w_dtype) if w_dtype else np.asarray(w_v, dtype=np.float64)
    Hkv, D = k_pages[0].shape[1], k_pages[0].shape[3]
    d_kv = Hkv * D
    assert wk.shape == (d_kv, len(k_pages) * d_kv) and wv.shape == wk.shape
    xk = stacked_layers(k_pages, page_table, token_seq, token_pos, page_size, dtype)
    xv = stacked_layers(v_pages, page_table, token_seq, token_pos, page_size, dtype)
    kp = (xk @ wk.T).reshape(-1, Hkv, D)                   # W_K^proj [k^(1); ...; k^(L_s)]
    vp = (xv @ wv.T).reshape(-1, Hkv, D)                   # W_V^proj [v^(1); ...; v^(L_s)]
    if rope_keys:                                          # "Proj + RoPE fix": rotate the projected key at t
        kp = rope(kp, np.asarray(token_pos, dtype=np.float64)[:, None], theta)
    return kp, vp


def scatter_tokens(dst_pages: np.ndarray, page_table: np.ndarray, token_seq: np.ndarray, token_pos: np.ndarray,
                   values: np.ndarray, page_size: int) -> np.ndarray:
    """A copy of ``dst_pages`` with token i's ``[Hkv][D]`` vector written at its slot."""
    out = np.array(dst_pages, copy=True)
    seq = np.asarray(token_seq, dtype=np.int64)
    pos = np.asarray(token_pos, dtype=np.int64)
    pid = np.asarray(page_table)[seq, pos // page_size]
    out[pid, :, pos % page_size, :] = values
    return out
