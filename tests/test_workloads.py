"""The seeded input generators: determinism, bf16 rounding, page tables, trees, byte counts."""
import numpy as np
import pytest

import oracle
import workloads as W


def test_bf16_rounding_is_round_to_nearest_even_like_torch():
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(0)
    x = np.concatenate([rng.standard_normal(100000).astype(np.float32) * 10.0 ** rng.integers(-30, 30, 100000),
                        np.array([0.0, -0.0, 1.0, 65504.0, 3.4e38, -3.4e38, 1e-40, np.inf, -np.inf], np.float32)])
    # exact ties: mantissa low half == 0x8000 with even and odd kept parts
    ties = (np.array([0x3F808000, 0x3F818000, 0xBF808000, 0x40490000 | 0x8000], np.uint32)).view(np.float32)
    x = np.concatenate([x, ties]).astype(np.float32)
    mine = W.f32_to_bf16_bits(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(mine, ref)
    assert W.f32_to_bf16_bits(np.array([np.nan], np.float32))[0] == 0x7FC0


def test_oracle_decode_of_bf16_is_exact_widening():
    torch = pytest.importorskip("torch")
    bits = np.arange(0, 2 ** 16, dtype=np.uint16)
    bits = bits[~np.isnan(W.bf16_bits_to_f32(bits))]
    ref = torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16).to(torch.float64).numpy()
    assert np.array_equal(oracle.decode(bits, "bf16"), ref)


def test_generation_is_deterministic_per_seed():
    a = W.make_case(ctx_lens=[40, 17], n_new=3, num_q_heads=4, num_kv_heads=2, head_dim=8, seed=5)
    b = W.make_case(ctx_lens=[40, 17], n_new=3, num_q_heads=4, num_kv_heads=2, head_dim=8, seed=5)
    c = W.make_case(ctx_lens=[40, 17], n_new=3, num_q_heads=4, num_kv_heads=2, head_dim=8, seed=6)
    for f in ("q", "k_pages", "v_pages", "page_table", "draft_k", "draft_v"):
        assert np.array_equal(getattr(a, f), getattr(b, f))
    assert not np.array_equal(a.q, c.q)


def test_page_tables_are_disjoint_permutations_with_poisoned_rest():
    c = W.make_case(ctx_lens=[33, 16, 0, 1], n_new=2, num_q_heads=4, num_kv_heads=2, head_dim=8, page_size=16,
                    seed=9)
    used = c.page_table[c.page_table >= 0]
    assert len(np.unique(used)) == len(used)
    assert list((c.page_table >= 0).sum(1)) == [3, 1, 0, 1]
    spare = np.setdiff1d(np.arange(c.num_pages), used)
    assert len(spare) >= 1
    assert np.isnan(W.bf16_bits_to_f32(c.k_pages[spare])).all()
    # tail slots of the last page of sequence 0 (33 tokens -> slot 1.. of page 2) are NaN
    last = c.page_table[0, 2]
    assert np.isnan(W.bf16_bits_to_f32(c.k_pages[last, :, 1:])).all()
    assert not np.isnan(W.bf16_bits_to_f32(c.k_pages[last, :, 0])).any()


def test_logical_data_does_not_depend_on_the_page_table():
    a = W.make_case(ctx_lens=[50], n_new=2, num_q_heads=2, num_kv_heads=1, head_dim=8, seed=3, shuffle=True)
    b = W.make_case(ctx_lens=[50], n_new=2, num_q_heads=2, num_kv_heads=1, head_dim=8, seed=3, shuffle=False)
    ga = oracle.gather_prefix(a.k_pages, a.page_table[0], 50, 16)
    gb = oracle.gather_prefix(b.k_pages, b.page_table[0], 50, 16)
    assert np.array_equal(ga, gb)


def test_outlier_channels_scale_keys_only():
    a = W.make_case(ctx_lens=[64], n_new=1, num_q_heads=2, num_kv_heads=2, head_dim=16, seed=4, n_outlier=4)
    b = W.make_case(ctx_lens=[64], n_new=1, num_q_heads=2, num_kv_heads=2, head_dim=16, seed=4, n_outlier=0)
    ka = W.bf16_bits_to_f32(oracle.gather_prefix(a.k_pages, a.page_table[0], 64, 16))
    kb = W.bf16_bits_to_f32(oracle.gather_prefix(b.k_pages, b.page_table[0], 64, 16))
    for h in range(2):
        ratio = np.abs(ka[:, h]).mean(0) / np.abs(kb[:, h]).mean(0)
        assert (np.isclose(ratio, 8.0, rtol=0.02)).sum() == 4
        assert (np.isclose(ratio, 1.0)).sum() == 12
    assert np.array_equal(a.v_pages, b.v_pages)


@pytest.mark.parametrize("seed", [1005, 1, 2, 3])
def test_trees_respect_depth_and_branching(seed):
    for b in range(8):
        p = W.random_tree(seed, b, 60)
        assert p[0] == -1 and all(0 <= p[i] < i for i in range(1, 60))
        _, depth = oracle.tree_ancestry(p)
        assert depth.max() <= 7
        assert np.bincount(p[1:], minlength=60).max() <= 4


def test_ragged_workload_shape():
    lens = W.ragged_lengths(1003, 16, 512, 8192)
    offs = W.ragged_offsets(1003, 16, 8)
    assert lens.min() >= 512 and lens.max() <= 8192 and len(set(lens.tolist())) > 8
    assert offs.min() >= 0 and offs.max() <= 8


def test_long_range_byte_count():
    class Dims:
        head_dim, num_kv_heads, num_q_heads, page_size, batch, n_new, mode = 128, 8, 32, 16, 64, 8, "step"
        ctx_lens = np.full(64, 32768)
        step_offsets = np.zeros(64, np.int32)

        def draft_len(self, b):
            return 8
    kv = 64 * 32768 * 8 * 128 * 2 * 2
    assert kv == 8_589_934_592
    assert W.algorithmic_bytes(Dims()) == kv + 64 * 2048 * 4 + 64 * 2 * 8 * 8 * 128 * 2 + 2 * 64 * 8 * 32 * 128 * 2
