"""Pins for the CPU oracle: closed forms, invariants, brute force, library reductions.

Each test checks the oracle against something other than itself, chosen so
that a plausible slip (dropped term, wrong sign or index, transposed operand,
off-by-one position, wrong GQA mapping, mask off by one) fails at least one.
"""
import json
import math
import os

import numpy as np
import pytest

import oracle
import workloads as W
from tests import _bruteforce as BF

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def tiny(mode="step", **kw):
    base = dict(mode=mode, batch=2, ctx_lens=[5, 3], n_new=3, num_q_heads=4, num_kv_heads=2, head_dim=8,
                page_size=2, dtype="bf16", seed=7)
    base.update(kw)
    return W.make_case(**base)


def run(case, **kw):
    return oracle.draft_attention(case, **kw)


# ---------------------------------------------------------------------------
# attention core closed forms (Sec. 2.2, Eq. 2)
# ---------------------------------------------------------------------------

def test_single_key_returns_its_value_exactly():
    rng = np.random.default_rng(0)
    q, K, V = rng.standard_normal((3, 16)), rng.standard_normal((1, 16)), rng.standard_normal((1, 16))
    out, lse = oracle.masked_attention(q, K, V, np.ones((3, 1), bool), 0.25)
    assert np.array_equal(out, np.repeat(V, 3, axis=0))
    np.testing.assert_allclose(lse, 0.25 * (q @ K[0]), rtol=0, atol=1e-14)


def test_equal_scores_give_mean_of_allowed_values():
    rng = np.random.default_rng(1)
    V = rng.standard_normal((6, 5))
    allowed = np.array([[1, 1, 0, 1, 0, 0], [0, 0, 0, 0, 1, 1]], bool)
    out, lse = oracle.masked_attention(np.zeros((2, 5)), rng.standard_normal((6, 5)), V, allowed, 1.0)
    np.testing.assert_allclose(out[0], V[[0, 1, 3]].mean(0), atol=1e-15)
    np.testing.assert_allclose(out[1], V[[4, 5]].mean(0), atol=1e-15)
    np.testing.assert_allclose(lse, [math.log(3), math.log(2)], atol=1e-15)


def test_two_keys_give_logistic_weights():
    # q = (a, 0), k0 = (1, 0), k1 = 0: z = (scale*a, 0) -> weights sigma(+-scale*a)
    for a, scale in [(0.3, 1.0), (-2.0, 0.5), (7.0, 1 / math.sqrt(8))]:
        v0, v1 = np.array([1.0, -2.0]), np.array([3.0, 0.5])
        out, _ = oracle.masked_attention(np.array([[a, 0.0]]), np.array([[1.0, 0.0], [0.0, 0.0]]),
                                         np.stack([v0, v1]), np.ones((1, 2), bool), scale)
        w0 = 1.0 / (1.0 + math.exp(-scale * a))
        np.testing.assert_allclose(out[0], w0 * v0 + (1 - w0) * v1, rtol=1e-14, atol=1e-15)


def test_weights_sum_to_one():
    # with every value row equal to 1 the output equals the sum of the weights
    c = tiny()
    c.v_pages = np.where(np.isnan(W.bf16_bits_to_f32(c.v_pages)), c.v_pages, np.uint16(0x3F80))
    c.draft_v = np.where(np.isnan(W.bf16_bits_to_f32(c.draft_v)), c.draft_v, np.uint16(0x3F80))
    out, _ = run(c)
    np.testing.assert_allclose(out, 1.0, atol=1e-14)


def test_masked_scores_are_excluded():
    rng = np.random.default_rng(2)
    q, K, V = rng.standard_normal((1, 4)), rng.standard_normal((3, 4)), rng.standard_normal((3, 4))
    K2, V2 = K.copy(), V.copy()
    K2[1] = 1e6
    V2[1] = np.nan  # a masked column must not leak even NaN
    allowed = np.array([[True, False, True]])
    a, _ = oracle.masked_attention(q, K, V, allowed, 1.0)
    b, _ = oracle.masked_attention(q, K2, np.nan_to_num(V2, nan=123.0), allowed, 1.0)
    np.testing.assert_allclose(a, b, atol=1e-15)


# ---------------------------------------------------------------------------
# worked example with the paper's literal scale-free softmax (golden fixture)
# ---------------------------------------------------------------------------

def _golden_case(spec, mode, ln2):
    def arr(x):
        return np.array([[ln2 if v == "ln2_f32" else v for v in row] for row in x], dtype=np.float32)
    T = spec["ctx_len"]
    tk, tv = arr(spec["target_k"]), arr(spec["target_v"])
    kp = tk.reshape(1, T, 1, 2).transpose(0, 2, 1, 3).copy()
    vp = tv.reshape(1, T, 1, 2).transpose(0, 2, 1, 3).copy()
    q = arr(spec["q"])[None, :, None, :]
    dk = arr(spec["draft_k"])[None, :, None, :]
    dv = arr(spec["draft_v"])[None, :, None, :]
    common = dict(dtype="fp32", page_size=T, rope_theta=1e6, softmax_scale=1.0)
    if mode == "step":
        return oracle.draft_attention_step(q, kp, vp, np.array([[0]]), np.array([T]), dk, dv,
                                           np.array([spec["step_offset"]]), **common)
    return oracle.draft_attention_tree(q, kp, vp, np.array([[0]]), np.array([T]), dk, dv,
                                       np.array([spec["parents"]]), **common)


@pytest.mark.parametrize("mode", ["step", "tree"])
def test_golden_literal_scale_example(mode):
    g = json.load(open(os.path.join(GOLDEN, "literal_scale_memory_example.json")))
    out, lse = _golden_case(g[mode], mode, g["ln2_f32"])
    np.testing.assert_allclose(out[0, :, 0], np.array(g[mode]["expected_out"]), atol=g["tolerance"])
    np.testing.assert_allclose(lse[0, :, 0], np.array(g[mode]["expected_lse"]), atol=g["tolerance"])


# ---------------------------------------------------------------------------
# paging
# ---------------------------------------------------------------------------

def test_gather_inverts_scatter_bit_exactly():
    rng = np.random.default_rng(3)
    T, Hkv, D, P = 37, 2, 4, 8
    dense = rng.integers(0, 2 ** 16, size=(T, Hkv, D), dtype=np.uint16)
    pool = np.full((9, Hkv, P, D), 0xFFFF, np.uint16)
    table = rng.permutation(9)[:5].astype(np.int32)
    for t in range(T):  # scatter by an explicit loop
        pool[table[t // P], :, t % P, :] = dense[t]
    assert np.array_equal(oracle.gather_prefix(pool, np.append(table, -1), T, P), dense)


def test_physical_page_relocation_is_bit_invariant():
    c = tiny(ctx_lens=[9, 14], page_size=4)
    ref, ref_lse = run(c)
    perm = np.random.default_rng(4).permutation(c.num_pages)
    inv = np.argsort(perm)
    c.k_pages, c.v_pages = c.k_pages[perm], c.v_pages[perm]
    c.page_table = np.where(c.page_table >= 0, inv[np.maximum(c.page_table, 0)], -1).astype(np.int32)
    out, lse = run(c)
    assert np.array_equal(out, ref) and np.array_equal(lse, ref_lse)


def test_logical_prefix_order_does_not_matter_for_target_keys():
    # swapping two target tokens' K and V together leaves the output unchanged (target keys carry
    # their position inside the stored rotation; the kernel applies none)
    c = tiny(ctx_lens=[6, 6], page_size=2)
    ref, _ = run(c)
    for b in range(2):
        r = c.page_table[b]
        p0, p1 = r[0], r[2]
        for arr in (c.k_pages, c.v_pages):
            arr[[p0, p1]] = arr[[p1, p0]]
    out, _ = run(c)
    np.testing.assert_allclose(out, ref, atol=1e-13)


def test_page_table_padding_and_spare_pages_never_read():
    c = tiny(ctx_lens=[5, 3], page_size=4)
    assert (c.page_table == -1).any()
    out, _ = run(c)
    assert np.isfinite(out).all()   # spare pages / tail slots are NaN-poisoned


# ---------------------------------------------------------------------------
# RoPE
# ---------------------------------------------------------------------------

def test_rope_identity_at_zero_and_norm_preserving():
    x = np.random.default_rng(5).standard_normal((7, 128))
    assert np.array_equal(oracle.rope(x, 0, 1e6), x)
    y = oracle.rope(x, np.arange(7) * 4099 + 31, 1e6)
    np.testing.assert_allclose(np.linalg.norm(y, axis=1), np.linalg.norm(x, axis=1), rtol=1e-13)


def test_rope_scores_depend_only_on_relative_position():
    rng = np.random.default_rng(6)
    q, k = rng.standard_normal(128), rng.standard_normal(128)
    base = oracle.rope(q, 40, 1e6) @ oracle.rope(k, 33, 1e6)
    for shift in (1, 1000, 32000):
        np.testing.assert_allclose(oracle.rope(q, 40 + shift, 1e6) @ oracle.rope(k, 33 + shift, 1e6), base,
                                   rtol=1e-9, atol=1e-9)


def test_rope_matches_complex_form():
    rng = np.random.default_rng(7)
    D, theta = 128, 1e6
    x = rng.standard_normal(D)
    for p in (1, 17, 32767):
        y = oracle.rope(x, p, theta)
        z = (x[:D // 2] + 1j * x[D // 2:]) * np.exp(1j * p * theta ** (-np.arange(0, D, 2) / D))
        np.testing.assert_allclose(y, np.concatenate([z.real, z.imag]), atol=1e-12)


def test_rope_lowest_pair_rotates_by_position_radians():
    # theta_0 = theta^0 = 1: the pair (x_0, x_{D/2}) turns by exactly p radians
    x = np.zeros(8)
    x[0] = 1.0
    y = oracle.rope(x, 2, 1e6)
    np.testing.assert_allclose([y[0], y[4]], [math.cos(2), math.sin(2)], atol=1e-15)


# ---------------------------------------------------------------------------
# draft positions and masks
# ---------------------------------------------------------------------------

def test_first_draft_query_sees_only_target_and_itself_at_position_T():
    # T = 0, one query: the only key is its own; the output is that key's value exactly
    c = tiny(batch=1, ctx_lens=[0], n_new=1)
    out, lse = run(c)
    G = c.num_q_heads // c.num_kv_heads
    for h in range(c.num_q_heads):
        np.testing.assert_array_equal(out[0, 0, h], oracle.decode(c.draft_v[0, 0, h // G], "bf16"))


def test_step_by_step_equals_folded_call():
    c = tiny(step_offsets=[1, 0], n_new=3, max_draft=4)
    ref, ref_lse = run(c)
    for j in range(3):
        cj = W.DraftCase(**{**c.__dict__, "q": c.q[:, j:j + 1], "n_new": 1,
                            "step_offsets": c.step_offsets + j})
        o, l = run(cj)
        np.testing.assert_allclose(o[:, 0], ref[:, j], atol=1e-13)
        np.testing.assert_allclose(l[:, 0], ref_lse[:, j], atol=1e-13)


def test_query_does_not_see_later_draft_keys():
    c = tiny(n_new=3)
    ref, _ = run(c)
    c2 = W.DraftCase(**c.__dict__)
    c2.draft_k = c.draft_k.copy()
    c2.draft_v = c.draft_v.copy()
    c2.draft_v[:, 2] = W.f32_to_bf16_bits(np.full(c.draft_v[:, 2].shape, 50.0, np.float32))
    out, _ = run(c2)
    np.testing.assert_array_equal(out[:, :2], ref[:, :2])   # queries 0, 1 cannot see key 2
    assert not np.allclose(out[:, 2], ref[:, 2])            # query 2 sees its own key


def test_chain_tree_equals_causal_steps():
    N = 5
    c = tiny(n_new=N)
    ref, ref_lse = run(c)
    t = W.DraftCase(**{**c.__dict__, "mode": "tree", "step_offsets": None,
                       "parents": np.tile(np.arange(-1, N - 1, dtype=np.int32), (2, 1))})
    out, lse = run(t)
    np.testing.assert_allclose(out, ref, atol=1e-13)
    np.testing.assert_allclose(lse, ref_lse, atol=1e-13)


def test_star_forest_sees_target_and_self_only():
    N = 4
    c = tiny(mode="tree", n_new=N, parents=np.full((2, N), -1, np.int32))
    out, _ = run(c)
    for i in range(N):
        ci = W.DraftCase(**{**c.__dict__, "mode": "step", "parents": None, "n_new": 1,
                            "q": c.q[:, i:i + 1], "draft_k": c.draft_k[:, i:i + 1], "draft_v": c.draft_v[:, i:i + 1],
                            "step_offsets": np.zeros(2, np.int32), "max_draft": 1})
        o, _ = run(ci)
        np.testing.assert_allclose(out[:, i], o[:, 0], atol=1e-13)


def test_tree_ancestry_walk():
    anc, depth = oracle.tree_ancestry([-1, 0, 0, 1, -1, 4, 3])
    assert anc[6] == {6, 3, 1, 0} and anc[5] == {5, 4} and anc[2] == {2, 0}
    assert list(depth) == [0, 1, 1, 2, 0, 1, 3]
    with pytest.raises(ValueError):
        oracle.tree_ancestry([-1, 2, 0])


def test_siblings_are_mutually_invisible():
    c = tiny(mode="tree", n_new=3, parents=np.array([[-1, 0, 0]] * 2, np.int32))
    ref, _ = run(c)
    c2 = W.DraftCase(**c.__dict__)
    c2.draft_v = c.draft_v.copy()
    c2.draft_v[:, 2] = W.f32_to_bf16_bits(np.full(c.draft_v[:, 2].shape, -9.0, np.float32))
    out, _ = run(c2)
    np.testing.assert_array_equal(out[:, :2], ref[:, :2])


# ---------------------------------------------------------------------------
# grouped-query head mapping
# ---------------------------------------------------------------------------

def test_gqa_query_head_reads_kv_head_floor_h_over_g():
    c = tiny(num_q_heads=8, num_kv_heads=4, ctx_lens=[6, 2], page_size=2)
    for g in range(4):
        val = W.f32_to_bf16_bits(np.full(1, float(g + 1), np.float32))[0]
        live = ~np.isnan(W.bf16_bits_to_f32(c.v_pages[:, g]))
        c.v_pages[:, g][live] = val
        c.draft_v[:, :, g][~np.isnan(W.bf16_bits_to_f32(c.draft_v[:, :, g]))] = val
    out, _ = run(c)
    for h in range(8):
        np.testing.assert_allclose(out[:, :, h], h // 2 + 1, atol=1e-14)


# ---------------------------------------------------------------------------
# brute force and library reduction
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("dtype", ["bf16", "fp32"])
@pytest.mark.parametrize("heads", [(2, 1), (4, 2)])
def test_step_matches_bruteforce(dtype, heads):
    c = tiny(dtype=dtype, num_q_heads=heads[0], num_kv_heads=heads[1], ctx_lens=[7, 0], step_offsets=[2, 1],
             max_draft=5, rope_theta=100.0)
    out, _ = run(c)
    bf = np.array(BF.brute_step(c))
    np.testing.assert_allclose(out, bf, atol=1e-12, rtol=1e-12)


def test_tree_matches_bruteforce():
    c = tiny(mode="tree", n_new=6, parents=np.array([[-1, 0, 0, 1, 3, -1], [-1, 0, 1, 1, 0, 4]], np.int32),
             head_dim=4, rope_theta=50.0, ctx_lens=[4, 9], page_size=4)
    out, _ = run(c)
    np.testing.assert_allclose(out, np.array(BF.brute_tree(c)), atol=1e-12, rtol=1e-12)


def test_reduces_to_torch_sdpa_for_one_sequence():
    torch = pytest.importorskip("torch")
    c = tiny(batch=1, ctx_lens=[11], n_new=3, num_q_heads=8, num_kv_heads=2, head_dim=16, page_size=4,
             step_offsets=[2], max_draft=5)
    out, _ = run(c)
    T, s0, n, D, theta = 11, 2, 3, 16, c.rope_theta

    def rot(x, pos):  # complex form, independent of the oracle's rotate-half code
        x = torch.as_tensor(x, dtype=torch.float64)
        z = torch.complex(x[..., :D // 2], x[..., D // 2:])
        ang = torch.as_tensor(pos, dtype=torch.float64)[..., None] * theta ** (-torch.arange(0, D, 2, dtype=torch.float64) / D)
        z = z * torch.polar(torch.ones_like(ang), ang)
        return torch.cat([z.real, z.imag], -1)

    dec = lambda a: torch.as_tensor(W.bf16_bits_to_f32(a).astype(np.float64))
    Kt = dec(np.stack([c.k_pages[c.page_table[0][t // 4], :, t % 4] for t in range(T)]))
    Vt = dec(np.stack([c.v_pages[c.page_table[0][t // 4], :, t % 4] for t in range(T)]))
    S = s0 + n
    dk = rot(dec(c.draft_k[0, :S]).transpose(0, 1), (T + torch.arange(S))[None, :].expand(2, S)).transpose(0, 1)
    K = torch.cat([Kt, dk], 0).transpose(0, 1).repeat_interleave(4, 0)          # [Hq][L][D]
    V = torch.cat([Vt, dec(c.draft_v[0, :S])], 0).transpose(0, 1).repeat_interleave(4, 0)
    qpos = (T + s0 + torch.arange(n))[None, :].expand(8, n)
    Q = rot(dec(c.q[0]).transpose(0, 1), qpos)                                  # [Hq][n][D]
    mask = torch.cat([torch.ones(n, T, dtype=torch.bool),
                      torch.arange(S)[None, :] <= (s0 + torch.arange(n))[:, None]], 1)
    ref = torch.nn.functional.scaled_dot_product_attention(Q, K, V, attn_mask=mask, scale=1 / math.sqrt(D))
    np.testing.assert_allclose(out[0], ref.transpose(0, 1).numpy(), atol=1e-12)


# ---------------------------------------------------------------------------
# position base and query-node subset (general call: head-concatenated
# prefixes, level-wise tree growth)
# ---------------------------------------------------------------------------

def test_pos_base_equal_to_ctx_len_is_the_default_bit_for_bit():
    c = tiny(ctx_lens=[5, 3], step_offsets=[1, 0], max_draft=5)
    ref, _ = run(c)
    c.pos_base = c.ctx_lens.copy()
    out, _ = run(c)
    assert np.array_equal(out, ref)
    t = tiny(mode="tree", n_new=5, parents=np.array([[-1, 0, 0, 1, 2], [-1, 0, 1, -1, 3]], np.int32))
    ref, _ = run(t)
    t.pos_base = t.ctx_lens.copy()
    out, _ = run(t)
    assert np.array_equal(out, ref)


def test_empty_prefix_output_is_invariant_to_the_position_base():
    # with no prefix every score is draft-draft, and RoPE scores depend only on position differences
    c = tiny(ctx_lens=[0, 0], step_offsets=[2, 0], max_draft=6)
    ref, _ = run(c)
    c.pos_base = np.array([1000, 37], np.int32)
    out, _ = run(c)
    np.testing.assert_allclose(out, ref, atol=1e-12, rtol=0)


@pytest.mark.parametrize("mode", ["step", "tree"])
def test_pos_base_matches_bruteforce(mode):
    if mode == "step":
        c = tiny(ctx_lens=[6, 2], step_offsets=[1, 2], max_draft=6, head_dim=4, rope_theta=80.0)
    else:
        c = tiny(mode="tree", n_new=5, parents=np.array([[-1, 0, 1, 1, 0], [-1, -1, 0, 1, 2]], np.int32),
                 head_dim=4, rope_theta=60.0, ctx_lens=[5, 3], page_size=4)
    c.pos_base = np.array([2, 11], np.int32)          # not the prefix lengths
    out, _ = run(c)
    bf = np.array(BF.brute_step(c) if mode == "step" else BF.brute_tree(c))
    np.testing.assert_allclose(out, bf, atol=1e-12, rtol=1e-12)


def test_query_node_subset_selects_rows_of_the_full_tree():
    parents = np.array([[-1, 0, 0, 1, 1, 2, 3], [-1, 0, 1, 2, 0, 4, -1]], np.int32)
    full = tiny(mode="tree", n_new=7, parents=parents, ctx_lens=[6, 4])
    ref, ref_lse = run(full)
    nodes = np.array([[3, 4, 5], [6, 2, 5]], np.int32)      # e.g. the newest level of each tree
    sub = tiny(mode="tree", n_new=7, parents=parents, ctx_lens=[6, 4])
    sub.q = np.stack([full.q[b][nodes[b]] for b in range(2)])
    sub.query_nodes = nodes
    sub.n_new = 3
    out, lse = run(sub)
    for b in range(2):
        assert np.array_equal(out[b], ref[b][nodes[b]])
        assert np.array_equal(lse[b], ref_lse[b][nodes[b]])
    bf = np.array(BF.brute_tree(sub))
    np.testing.assert_allclose(out, bf, atol=1e-12, rtol=1e-12)
