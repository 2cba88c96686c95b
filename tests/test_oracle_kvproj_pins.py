"""Pins for the projected-KV cache builder oracle (Sec. 3.2, linear projection and
its RoPE-fix variant; App. A, L_s = 3 sampled target layers).

Chosen so that a plausible slip in the oracle fails at least one test:
  - wrong layer order or head-major/channel-major mix-up in the stacking -> selection pins;
  - a transposed W -> brute force (non-square W);
  - rotation at the wrong position, the wrong pairing or sign -> unit-key closed form
    and the relative-position test;
  - values rotated -> the values-untouched pin;
  - a page-table slip -> brute force (own page walk) and page-permutation invariance.
"""
import cmath
import math
import struct

import numpy as np
import pytest

from oracle.kvproj import project_kv, scatter_tokens, stacked_layers
from oracle.attention import rope
import workloads as W


def bf16_bits(x):
    return W.f32_to_bf16_bits(np.asarray(x, dtype=np.float32))


def tiny(seed=0, L=3, Hkv=2, D=4, P=2, pages=7, B=2, max_pages=3):
    rng = np.random.default_rng(seed)
    kp = [bf16_bits(rng.standard_normal((pages, Hkv, P, D))) for _ in range(L)]
    vp = [bf16_bits(rng.standard_normal((pages, Hkv, P, D))) for _ in range(L)]
    table = rng.permutation(pages)[:B * max_pages].reshape(B, max_pages).astype(np.int32)   # disjoint pages
    seq = np.array([0, 1, 1, 0, 1], np.int32)
    pos = np.array([5, 0, 3, 2, 4], np.int32)
    d_kv = Hkv * D
    wk = bf16_bits(rng.standard_normal((d_kv, L * d_kv)) / math.sqrt(L * d_kv))
    wv = bf16_bits(rng.standard_normal((d_kv, L * d_kv)) / math.sqrt(L * d_kv))
    return kp, vp, table, seq, pos, wk, wv


# --- an independent scalar walk: own bf16 decode, own page lookup, complex-form RoPE ---

def _f(bits):
    return struct.unpack("<f", struct.pack("<I", (int(bits) & 0xFFFF) << 16))[0]


def brute_project(pools, table, b, t, w, P, theta, rotate):
    L = len(pools)
    Hkv, D = len(pools[0][0]), len(pools[0][0][0][0])
    page = int(table[b][t // P])
    x = []
    for layer in range(L):
        for h in range(Hkv):
            for d in range(D):
                x.append(_f(pools[layer][page][h][t % P][d]))
    out = [math.fsum(_f(w[c][j]) * x[j] for j in range(len(x))) for c in range(Hkv * D)]
    if rotate:
        half = D // 2
        for h in range(Hkv):
            for m in range(half):
                z = complex(out[h * D + m], out[h * D + m + half]) * cmath.exp(1j * t * theta ** (-2.0 * m / D))
                out[h * D + m], out[h * D + m + half] = z.real, z.imag
    return out


@pytest.mark.parametrize("rotate", [False, True])
@pytest.mark.parametrize("L", [1, 3, 4])
def test_matches_scalar_brute_force(rotate, L):
    kp, vp, table, seq, pos, wk, wv = tiny(seed=L, L=L)
    theta = 10.0
    K, V = project_kv(kp, vp, table, seq, pos, wk, wv, page_size=2, theta=theta, rope_keys=rotate)
    for i in range(len(seq)):
        bk = brute_project(kp, table, int(seq[i]), int(pos[i]), wk, 2, theta, rotate)
        bv = brute_project(vp, table, int(seq[i]), int(pos[i]), wv, 2, theta, False)
        np.testing.assert_allclose(K[i].reshape(-1), bk, rtol=0, atol=1e-13)
        np.testing.assert_allclose(V[i].reshape(-1), bv, rtol=0, atol=1e-13)


@pytest.mark.parametrize("layer", [0, 1, 2])
def test_selection_matrix_returns_the_chosen_layer_bit_for_bit(layer):
    # W = [0 .. I .. 0] (identity in block `layer`) without rotation: k' is that layer's stored key
    kp, vp, table, seq, pos, _, _ = tiny(seed=5)
    d_kv = 8
    sel = np.zeros((d_kv, 3 * d_kv))
    sel[:, layer * d_kv:(layer + 1) * d_kv] = np.eye(d_kv)
    K, V = project_kv(kp, vp, table, seq, pos, sel, sel, page_size=2, theta=1e6, rope_keys=False, w_dtype=None)
    for i in range(len(seq)):
        page = table[seq[i], pos[i] // 2]
        want_k = W.bf16_bits_to_f32(kp[layer][page, :, pos[i] % 2, :]).astype(np.float64)
        want_v = W.bf16_bits_to_f32(vp[layer][page, :, pos[i] % 2, :]).astype(np.float64)
        assert np.array_equal(K[i], want_k)
        assert np.array_equal(V[i], want_v)


def test_head_permutation_matrix_moves_heads():
    # W maps head 0 of layer 2 to output head 1 and head 1 of layer 0 to output head 0
    kp, vp, table, seq, pos, _, _ = tiny(seed=6)
    D, d_kv = 4, 8
    sel = np.zeros((d_kv, 3 * d_kv))
    sel[D:2 * D, 2 * d_kv:2 * d_kv + D] = np.eye(D)
    sel[0:D, D:2 * D] = np.eye(D)
    K, _ = project_kv(kp, vp, table, seq, pos, sel, sel, page_size=2, theta=1e6, rope_keys=False, w_dtype=None)
    for i in range(len(seq)):
        page = table[seq[i], pos[i] // 2]
        assert np.array_equal(K[i, 1], W.bf16_bits_to_f32(kp[2][page, 0, pos[i] % 2]).astype(np.float64))
        assert np.array_equal(K[i, 0], W.bf16_bits_to_f32(kp[0][page, 1, pos[i] % 2]).astype(np.float64))


@pytest.mark.parametrize("m", [0, 1, 2, 3])
def test_rotation_of_a_unit_key_has_the_closed_form(m):
    # stored key e_m at position t, W selects layer 0: k' = cos(t w_m) e_m + sin(t w_m) e_{m+D/2}
    # (first half) or cos e_m - sin e_{m-D/2} (second half), w_m = theta^(-2 (m mod D/2) / D)
    D, P, t, theta = 4, 2, 5, 10.0
    pools = [np.zeros((3, 1, P, D), np.uint16) for _ in range(3)]
    pools[0][2, 0, t % P, m] = bf16_bits(1.0)
    table = np.array([[0, 1, 2]], np.int32)
    sel = np.zeros((D, 3 * D))
    sel[:, :D] = np.eye(D)
    K, _ = project_kv(pools, pools, table, [0], [t], sel, sel, page_size=P, theta=theta, rope_keys=True,
                      w_dtype=None)
    half = D // 2
    a = t * theta ** (-2.0 * (m % half) / D)
    want = np.zeros(D)
    if m < half:
        want[m], want[m + half] = math.cos(a), math.sin(a)
    else:
        want[m], want[m - half] = math.cos(a), -math.sin(a)
    np.testing.assert_allclose(K[0, 0], want, rtol=0, atol=1e-15)


def test_values_are_never_rotated():
    kp, vp, table, seq, pos, wk, wv = tiny(seed=7)
    _, v1 = project_kv(kp, vp, table, seq, pos, wk, wv, page_size=2, theta=10.0, rope_keys=True)
    _, v0 = project_kv(kp, vp, table, seq, pos, wk, wv, page_size=2, theta=10.0, rope_keys=False)
    assert np.array_equal(v0, v1)


def test_rotated_projection_gives_scores_that_depend_on_relative_position_only():
    # identical source KV at positions 1 and 4: a query at t + delta scores both keys alike
    rng = np.random.default_rng(8)
    D, P = 8, 2
    base = bf16_bits(rng.standard_normal((1, D)))
    pools = [np.zeros((4, 1, P, D), np.uint16) for _ in range(3)]
    for layer in range(3):
        for t in (1, 4):
            pools[layer][t // P, 0, t % P] = base[0] + layer       # distinct per layer, equal across t
    table = np.array([[0, 1, 2, 3]], np.int32)
    w = rng.standard_normal((D, 3 * D))
    K, _ = project_kv(pools, pools, table, [0, 0], [1, 4], w, w, page_size=P, theta=100.0, w_dtype=None)
    q = rng.standard_normal(D)
    for delta in (0, 1, 3):
        s1 = rope(q, 1 + delta, 100.0) @ K[0, 0]
        s2 = rope(q, 4 + delta, 100.0) @ K[1, 0]
        assert abs(s1 - s2) < 1e-12


def test_linear_in_the_projection_matrix():
    kp, vp, table, seq, pos, _, _ = tiny(seed=9)
    rng = np.random.default_rng(9)
    w1, w2 = rng.standard_normal((8, 24)), rng.standard_normal((8, 24))
    a = project_kv(kp, vp, table, seq, pos, w1 + w2, w1 - w2, page_size=2, theta=3.0, w_dtype=None)
    b = project_kv(kp, vp, table, seq, pos, w1, w1, page_size=2, theta=3.0, w_dtype=None)
    c = project_kv(kp, vp, table, seq, pos, w2, -w2, page_size=2, theta=3.0, w_dtype=None)
    np.testing.assert_allclose(a[0], b[0] + c[0], rtol=0, atol=1e-12)
    np.testing.assert_allclose(a[1], b[1] + c[1], rtol=0, atol=1e-12)


def test_invariant_under_a_permutation_of_physical_pages():
    kp, vp, table, seq, pos, wk, wv = tiny(seed=10)
    perm = np.random.default_rng(10).permutation(kp[0].shape[0])
    inv_kp, inv_vp = [], []
    for pool in kp:
        q = np.empty_like(pool)
        q[perm] = pool
        inv_kp.append(q)
    for pool in vp:
        q = np.empty_like(pool)
        q[perm] = pool
        inv_vp.append(q)
    a = project_kv(kp, vp, table, seq, pos, wk, wv, page_size=2, theta=10.0)
    b = project_kv(inv_kp, inv_vp, perm[table].astype(np.int32), seq, pos, wk, wv, page_size=2, theta=10.0)
    assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])


def test_scatter_then_gather_round_trip():
    kp, _, table, seq, pos, _, _ = tiny(seed=11)
    vals = np.random.default_rng(11).standard_normal((len(seq), 2, 4))
    dst = scatter_tokens(np.zeros((7, 2, 2, 4)), table, seq, pos, vals, 2)
    back = stacked_layers([dst], table, seq, pos, 2, dtype="fp32").reshape(len(seq), 2, 4)
    assert np.array_equal(back, vals.astype(np.float32).astype(np.float64))
    # slots no token maps to stay as they were
    touched = np.zeros(dst.shape[:1] + dst.shape[2:3], bool)
    touched[table[seq, pos // 2], pos % 2] = True
    assert np.all(dst[~touched[:, None, :].repeat(2, 1)] == 0)


def test_qwen3_8b_projection_shapes():
    # d_kv = 8 KV heads x 128 (Qwen3-8B, App. A), L_s = 3 (App. A): W in R^{1024 x 3072} (Sec. 3.2)
    c = W.kvproj_case(batch=1, ctx_lens=[16], new_tokens=[16], seed=1)
    assert len(c.k_src) == 3 and len(c.v_src) == 3
    assert c.w_k.shape == (1024, 3072) and c.w_v.shape == (1024, 3072)
