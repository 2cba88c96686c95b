"""GPU parity of level-wise draft-tree growth (Sec. 3.5, tree (8, 10, 60)) against the oracle.

- top-k: the token ids are integer work decided by comparing the logits
  themselves (bf16 or float32, exact in float64): bit-exact.  Log-probabilities
  are float32 z - logsumexp(z): |error| <= 5e-5 (the float32 log-sum-exp of up to
  152k terms, ~1e-6 relative, on values below 30).
- expansion and selection on scores and log-probabilities that are multiples
  of 1/64 below 64 in magnitude: every float32 sum is exact, so the decisions
  (ties included) are the oracle's: bit-exact, scores equal.
- whole growth from logits: the GPU's log-probabilities differ from float64 by
  ~1e-6, so a decision between two candidates closer than that may go either
  way.  Sequences whose oracle decisions all have a margin above 2e-4 must match
  exactly; every sequence must be a valid tree whose scores follow its logits
  and whose sorted scores match the oracle's within 1e-4.
"""
import numpy as np
import pytest

import oracle
import workloads as W
from tests import _gpu as G

pytestmark = pytest.mark.gpu

LP_ATOL = 5e-5


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def K():
    import paper_2604_26412_amd as m
    return m


def to_dev(host, dtype):
    t = G.torch()
    if dtype == "bf16":
        return t.from_numpy(np.ascontiguousarray(host).view(np.int16)).view(t.bfloat16).cuda()
    return t.from_numpy(np.ascontiguousarray(host)).cuda()


def as_f64(host, dtype):
    return (W.bf16_bits_to_f32(host) if dtype == "bf16" else host).astype(np.float64)


def check_topk(host, dtype, k, dev=None):
    t = G.torch()
    dev = to_dev(host, dtype) if dev is None else dev
    tok, lp = K().topk_logprobs(dev, k)
    t.cuda.synchronize()
    rt, rl = oracle.log_softmax_topk(as_f64(host, dtype), k)
    assert np.array_equal(tok.cpu().numpy(), rt)
    np.testing.assert_allclose(lp.cpu().numpy().astype(np.float64), rl, rtol=0, atol=LP_ATOL)


# ---------------------------------------------------------------- top-k


@pytest.mark.parametrize("dtype", ["bf16", "fp32"])
@pytest.mark.parametrize("vocab", [7, 8, 100, 16384, 16385, 40000, 151936])
@pytest.mark.parametrize("k", [1, 10, 16])
def test_topk_matches_the_oracle(dtype, vocab, k):
    if k > vocab:
        pytest.skip("k > vocab")
    host = W.draft_logits(7000 + vocab + k, 5, vocab, dtype=dtype)
    check_topk(host, dtype, k)


@pytest.mark.parametrize("dtype", ["bf16", "fp32"])
@pytest.mark.parametrize("sigma,grid,peaks", [(0.3, 1.0, 0), (1.0, 0.125, 8)])
@pytest.mark.parametrize("vocab", [3000, 151936])
def test_topk_ties_go_to_the_smaller_token(dtype, sigma, grid, peaks, vocab):
    # sigma 0.3 on a grid of 1: hundreds of logits of each chunk equal its maximum, past the
    # LDS list, so the workgroup arg-max rounds decide; grid 1/8 leaves a few ties
    host = W.draft_logits(7100, 4, vocab, dtype=dtype, sigma=sigma, peaks=peaks, grid=grid)
    check_topk(host, dtype, 16)
    check_topk(host, dtype, 10)


def test_topk_all_equal_row_and_single_winner():
    z = np.zeros((3, 20000), np.float32)
    z[1, 12345] = 1.0
    z[2, 19999] = -1.0                       # all equal but the last
    host = W.f32_to_bf16_bits(z)
    check_topk(host, "bf16", 16)
    t = G.torch()
    tok, _ = K().topk_logprobs(to_dev(host, "bf16"), 3)
    t.cuda.synchronize()
    assert tok.cpu().numpy().tolist() == [[0, 1, 2], [12345, 0, 1], [0, 1, 2]]


@pytest.mark.parametrize("dtype", ["bf16", "fp32"])
@pytest.mark.parametrize("vocab", [300, 40000])
def test_topk_treats_both_zeros_as_equal(dtype, vocab):
    # the 16th best logit falls among zeros of both signs: -0.0 and +0.0 tie, the smaller token wins
    z = np.full((2, vocab), -3.0, np.float32)
    z[:, :6] = 2.0
    zeros = np.arange(50, vocab, max(1, vocab // 40))[:30]
    z[0, zeros] = np.where(np.arange(len(zeros)) % 2 == 0, np.float32(-0.0), np.float32(0.0))
    z[1, zeros] = np.where(np.arange(len(zeros)) % 2 == 0, np.float32(0.0), np.float32(-0.0))
    host = W.f32_to_bf16_bits(z) if dtype == "bf16" else z
    check_topk(host, dtype, 16)


@pytest.mark.parametrize("dtype", ["bf16", "fp32"])
def test_topk_honours_the_row_stride(dtype):
    # rows of 151936 logits inside rows of 152000: the padding holds larger values that must be ignored
    vocab, stride = 151936, 152000
    host = W.draft_logits(7200, 6, vocab, dtype=dtype)
    pad = W.f32_to_bf16_bits(np.full((6, stride - vocab), 100.0, np.float32)) if dtype == "bf16" else \
        np.full((6, stride - vocab), 100.0, np.float32)
    full = to_dev(np.concatenate([host, pad], axis=1), dtype)
    check_topk(host, dtype, 10, dev=full[:, :vocab])


@pytest.mark.parametrize("dtype", ["bf16", "fp32"])
@pytest.mark.parametrize("offset", [1, 3])
def test_topk_rows_off_16_byte_boundaries(dtype, offset):
    # views starting a few elements into their rows: element loads
    vocab, stride = 40003, 40011
    host = W.draft_logits(7250 + offset, 5, stride, dtype=dtype)
    full = to_dev(host, dtype)
    check_topk(np.ascontiguousarray(host[:, offset:offset + vocab]), dtype, 10, dev=full[:, offset:offset + vocab])


def test_topk_large_row_count_and_largest_vocabulary():
    host = W.draft_logits(7300, 2, 64 * 16384, dtype="bf16")
    check_topk(host, "bf16", 16)
    host = W.draft_logits(7301, 700, 2048, dtype="fp32")
    check_topk(host, "fp32", 10)


def test_topk_workspace_may_be_reused_and_oversized():
    t = G.torch()
    host = W.draft_logits(7400, 12, 50000, dtype="bf16")
    ws = t.full((K().topk_workspace_bytes(12, 50000) + 4096,), 0x7F, dtype=t.uint8, device="cuda")
    dev = to_dev(host, "bf16")
    rt, rl = oracle.log_softmax_topk(as_f64(host, "bf16"), 10)
    for _ in range(2):
        tok, lp = K().topk_logprobs(dev, 10, workspace=ws)
        t.cuda.synchronize()
        assert np.array_equal(tok.cpu().numpy(), rt)
        np.testing.assert_allclose(lp.cpu().numpy(), rl, rtol=0, atol=LP_ATOL)


# ---------------------------------------------------------------- expansion and selection (exact inputs)


def grid_values(rng, shape, lo=-16.0):
    """Multiples of 1/64 in [lo, 0]: float32 sums of a few of them are exact."""
    return (rng.integers(int(lo * 64), 1, size=shape) / 64.0).astype(np.float32)


@pytest.mark.parametrize("F,P,k", [(1, 10, 10), (10, 10, 10), (16, 16, 16), (3, 5, 15), (7, 2, 1), (1, 1, 1),
                                   (16, 1, 16)])
def test_expand_matches_the_oracle_exactly(F, P, k):
    t = G.torch()
    rng = np.random.default_rng(F * 100 + P * 10 + k)
    B = 6
    scores = grid_values(rng, (B, F), lo=-8.0)
    lp = np.sort(grid_values(rng, (B, F, P), lo=-4.0), axis=-1)[..., ::-1].copy()   # best first, like top-k rows
    tokens = rng.integers(0, 151936, size=(B, F, P)).astype(np.int32)
    if F > 1:
        scores[:, 1] = scores[:, 0]                  # equal frontier scores: ties between frontier nodes
    par, tok, sc = K().tree_expand(t.from_numpy(scores).cuda(), t.from_numpy(tokens).cuda(),
                                   t.from_numpy(lp).cuda(), k)
    t.cuda.synchronize()
    for b in range(B):
        rp, rt, rs = oracle.grow_level(scores[b], tokens[b], lp[b], k)
        assert par[b].cpu().numpy().tolist() == rp.tolist()
        assert tok[b].cpu().numpy().tolist() == rt.tolist()
        assert np.array_equal(sc[b].cpu().numpy().astype(np.float64), rs)


def oracle_levels(rng, B, depth, k, lo=-3.0):
    """Per sequence, level records grown by the oracle from grid log-probabilities (ancestor-closed)."""
    seqs = []
    for _ in range(B):
        sc = np.zeros(1)
        levels = []
        for d in range(depth):
            F = 1 if d == 0 else k
            lp = np.sort(grid_values(rng, (F, k), lo=lo), axis=-1)[:, ::-1].astype(np.float64)
            tok = rng.integers(0, 1000, size=(F, k)).astype(np.int32)
            levels.append(oracle.grow_level(sc, tok, lp, k))
            sc = levels[-1][2]
        seqs.append(levels)
    return seqs


def stack_levels(seqs):
    depth = len(seqs[0])
    par = np.array([[seqs[b][d][0] for b in range(len(seqs))] for d in range(depth)], np.int32)
    tok = np.array([[seqs[b][d][1] for b in range(len(seqs))] for d in range(depth)], np.int32)
    sc = np.array([[seqs[b][d][2] for b in range(len(seqs))] for d in range(depth)], np.float32)
    return par, tok, sc


@pytest.mark.parametrize("depth,k,n", [(8, 10, 60), (8, 10, 80), (8, 10, 1), (1, 16, 16), (16, 16, 200),
                                       (5, 3, 7), (4, 1, 4)])
def test_select_matches_the_oracle_exactly(depth, k, n):
    t = G.torch()
    rng = np.random.default_rng(depth * 1000 + k * 10 + n)
    B = 5
    seqs = oracle_levels(rng, B, depth, k, lo=-2.0 if k > 1 else -0.5)
    par, tok, sc = stack_levels(seqs)
    out = K().tree_select(t.from_numpy(par).cuda(), t.from_numpy(tok).cuda(), t.from_numpy(sc).cuda(), n)
    t.cuda.synchronize()
    for b in range(B):
        ref = oracle.tree_finalize(seqs[b], n)
        for got, want in zip(out, ref):
            assert np.array_equal(got[b].cpu().numpy().astype(np.float64), np.asarray(want, np.float64))


def test_two_token_vocabulary_example():
    # the hand-derived tree of the oracle pins, grown on the GPU from float32 logits
    t = G.torch()
    row = np.log(np.array([0.9, 0.1], np.float32)).astype(np.float32)
    z = np.zeros((1, 8), np.float32) - 1e30
    z[0, :2] = row
    vocab = 8                                 # padded with effectively impossible tokens
    levels = [t.from_numpy(np.tile(z, (1, F, 1)).reshape(1, F, vocab)).cuda() for F in (1, 2, 2)]
    parents, tokens, depths, scores = K().grow_tree(levels, 2, 4)
    t.cuda.synchronize()
    assert parents.cpu().numpy().tolist() == [[-1, -1, 0, 2]]
    assert tokens.cpu().numpy().tolist() == [[0, 1, 0, 0]]
    assert depths.cpu().numpy().tolist() == [[0, 0, 1, 2]]


# ---------------------------------------------------------------- one level in one launch


def topk_then_expand(logits, scores, k):
    tok, lp = K().topk_logprobs(logits, k)
    return K().tree_expand(scores, tok, lp, k)


@pytest.mark.parametrize("dtype", ["bf16", "fp32"])
@pytest.mark.parametrize("B,F,V,k", [(8, 10, 151936, 10), (8, 1, 151936, 10), (3, 16, 40000, 16), (5, 7, 16384, 3),
                                     (2, 4, 5000, 1), (4, 2, 1000003, 16), (1, 3, 20, 16)])
def test_tree_level_equals_topk_then_expand(dtype, B, F, V, k):
    # the fused level and the two separate calls make the same float32 operations in the same order
    t = G.torch()
    host = W.draft_logits(7600 + V % 97 + F, B * F, V, dtype=dtype, stream=k).reshape(B, F, V)
    dev = to_dev(host, dtype)
    rng = np.random.default_rng(V + F)
    scores = t.from_numpy(-rng.uniform(0, 8, size=(B, F)).astype(np.float32)).cuda()
    got = K().tree_level(dev, scores, k)
    want = topk_then_expand(dev, scores, k)
    t.cuda.synchronize()
    for g, w in zip(got, want):
        assert np.array_equal(g.cpu().numpy(), w.cpu().numpy())


def test_tree_level_workspace_shared_by_frontier_sizes():
    # the root level (one frontier node) and full levels alternate on one workspace
    t = G.torch()
    B, V, k = 3, 40000, 10
    ws = K().tree_level_workspace(B, k, V)
    for i, F in enumerate([1, 10, 1, 10, 10, 1]):
        z = to_dev(W.draft_logits(7900 + i, B * F, V).reshape(B, F, V), "bf16")
        scores = t.full((B, F), -0.5 * i, device="cuda")
        got = K().tree_level(z, scores, k, workspace=ws)
        want = topk_then_expand(z, scores, k)
        t.cuda.synchronize()
        for g, w in zip(got, want):
            assert np.array_equal(g.cpu().numpy(), w.cpu().numpy()), (i, F)


def test_tree_level_ties_take_the_arg_max_rounds():
    # flat rows: more than 1024 logits of a chunk at the threshold
    t = G.torch()
    host = W.draft_logits(7700, 2 * 3, 40000, sigma=0.3, peaks=0, grid=1.0).reshape(2, 3, 40000)
    dev = to_dev(host, "bf16")
    scores = t.zeros((2, 3), device="cuda")
    scores[:, 1] = -1.0
    got = K().tree_level(dev, scores, 16)
    want = topk_then_expand(dev, scores, 16)
    t.cuda.synchronize()
    for g, w in zip(got, want):
        assert np.array_equal(g.cpu().numpy(), w.cpu().numpy())


def test_tree_level_workspace_is_left_clean_for_the_next_call_and_graph_replays():
    t = G.torch()
    B, F, V, k = 4, 10, 60000, 10
    ws = K().tree_level_workspace(B, F, V)
    levels = [to_dev(W.draft_logits(7800, B * F, V, stream=i).reshape(B, F, V), "bf16") for i in range(3)]
    scores = t.zeros((B, F), device="cuda")
    outs = [K().tree_level(z, scores, k, workspace=ws) for z in levels]
    t.cuda.synchronize()
    for z, o in zip(levels, outs):
        w = topk_then_expand(z, scores, k)
        for g, r in zip(o, w):
            assert np.array_equal(g.cpu().numpy(), r.cpu().numpy())
    assert int(ws[:256 * B * 17].view(t.int32).abs().sum()) == 0     # the counters are back at zero
    # captured once, replayed three times with eager work between the replays
    src = levels[0].clone()
    out = tuple(t.empty((B, k), dtype=dt, device="cuda") for dt in (t.int32, t.int32, t.float32))
    graph = t.cuda.CUDAGraph()
    side = t.cuda.Stream()
    side.wait_stream(t.cuda.current_stream())
    with t.cuda.stream(side):
        K().tree_level(src, scores, k, workspace=ws, out=out)
    t.cuda.current_stream().wait_stream(side)
    t.cuda.synchronize()
    with t.cuda.graph(graph):
        K().tree_level(src, scores, k, workspace=ws, out=out)
    for z in levels:
        src.copy_(z)
        t.cuda.synchronize()
        graph.replay()
        t.cuda.synchronize()
        w = topk_then_expand(z, scores, k)
        t.cuda.synchronize()
        for g, r in zip(out, w):
            assert np.array_equal(g.cpu().numpy(), r.cpu().numpy())


# ---------------------------------------------------------------- whole growth from logits


def oracle_tree(levels_f64, k, n):
    """The oracle's tree grown from each level's top-k rows, the smallest gap between two of its
    decisions (adjacent ranks among each level's k + 1 best candidates, and the n-th vs the
    (n + 1)-th node of the final selection), and the top-k rows themselves.

    Two children of one frontier node with equal logits tie exactly on both sides (one score plus
    one log-probability of the same row), and the tie rule orders them alike: such pairs are not
    decisions that rounding could flip, and are left out of the gaps."""
    sc = np.zeros(1)
    gaps, every, levels, rows = [], [], [], []
    for d, z in enumerate(levels_f64):
        tok, lp = oracle.log_softmax_topk(z, k)
        rows.append((tok, lp))
        cand = sorted(((float(sc[f] + lp[f, r]), f) for f in range(lp.shape[0]) for r in range(k)), reverse=True)
        for (a, fa), (b, fb) in zip(cand[:k], cand[1:k + 1]):
            if not (fa == fb and a == b):
                gaps.append(a - b)
        levels.append(oracle.grow_level(sc, tok, lp, k))
        sc = levels[-1][2]
        every += [(float(sc[i]), d, int(levels[-1][0][i])) for i in range(k)]
    every.sort(key=lambda e: -e[0])
    if n < len(every):
        (a, da, pa), (b, db, pb) = every[n - 1], every[n]
        if not (a == b and da == db and pa == pb):
            gaps.append(a - b)
    return oracle.tree_finalize(levels, n), min(gaps), rows


def check_valid_tree(rows, parents, tokens, depths, scores):
    """Parents precede children one level up; each token is among its parent row's top k, and its
    score is the parent's plus that token's log-probability."""
    n = len(parents)
    rank = np.zeros(n, np.int64)
    for i in range(n):
        rank[i] = np.sum(depths[:i] == depths[i])
        p = parents[i]
        assert (p == -1) == (depths[i] == 0)
        if depths[i] > 0:
            assert 0 <= p < i and depths[p] == depths[i] - 1
        top, lp = rows[depths[i]][0][0 if p < 0 else rank[p]], rows[depths[i]][1][0 if p < 0 else rank[p]]
        assert tokens[i] in top
        want = (0.0 if p < 0 else scores[p]) + lp[list(top).index(tokens[i])]
        assert abs(scores[i] - want) <= 1e-4


@pytest.mark.parametrize("vocab,B", [(151936, 4), (32000, 8)])
def test_grow_tree_matches_the_oracle(vocab, B):
    t = G.torch()
    spec = dict(W.TREEGROW_WORKLOADS["treegrow_b8_v152k_d8k10n60"])
    depth, k, n = spec["depth"], spec["k"], spec["n"]
    host = W.treegrow_levels(spec, vocab=vocab, batch=B)
    dev = [to_dev(h, "bf16") for h in host]
    parents, tokens, depths, scores = [a.cpu().numpy() for a in K().grow_tree(dev, k, n)]
    t.cuda.synchronize()
    exact = 0
    for b in range(B):
        lv = [W.bf16_bits_to_f32(h[b]).astype(np.float64) for h in host]
        (rp, rt, rd, rs), margin, rows = oracle_tree(lv, k, n)
        print(f"sequence {b}: smallest decision margin {margin:.2e}", flush=True)
        check_valid_tree(rows, parents[b], tokens[b], depths[b], scores[b])
        np.testing.assert_allclose(np.sort(scores[b].astype(np.float64)), np.sort(rs), rtol=0, atol=1e-4)
        if margin > 2e-4:
            exact += 1
            assert parents[b].tolist() == rp.tolist()
            assert tokens[b].tolist() == rt.tolist()
            assert depths[b].tolist() == rd.tolist()
            np.testing.assert_allclose(scores[b], rs, rtol=0, atol=1e-4)
    assert exact >= B // 2


def test_grow_tree_k1_is_the_greedy_chain():
    t = G.torch()
    host = [W.draft_logits(7500, 3, 30000, stream=d).reshape(3, 1, 30000) for d in range(6)]
    parents, tokens, depths, _ = K().grow_tree([to_dev(h, "bf16") for h in host], 1, 6)
    t.cuda.synchronize()
    for b in range(3):
        assert parents[b].cpu().numpy().tolist() == [-1, 0, 1, 2, 3, 4]
        want = [int(np.argmax(W.bf16_bits_to_f32(h[b, 0]))) for h in host]
        assert tokens[b].cpu().numpy().tolist() == want


# ---------------------------------------------------------------- argument errors


def test_binding_rejects_bad_arguments():
    t = G.torch()
    z = t.zeros((4, 100), dtype=t.bfloat16, device="cuda")
    with pytest.raises(K().KvshotError):
        K().topk_logprobs(z, 17)
    with pytest.raises(ValueError):
        K().topk_logprobs(z.to(t.float16), 4)
    big = t.zeros((4, 20000), dtype=t.bfloat16, device="cuda")
    with pytest.raises(K().KvshotError):
        K().topk_logprobs(big, 4, workspace=t.empty(16, dtype=t.uint8, device="cuda"))
    with pytest.raises((ValueError, K().KvshotError)):      # no workspace plan for 17 frontier nodes
        K().tree_level(t.zeros((2, 17, 100), dtype=t.bfloat16, device="cuda"), t.zeros((2, 17), device="cuda"), 4)
    with pytest.raises(K().KvshotError):
        K().tree_level(t.zeros((2, 17, 100), dtype=t.bfloat16, device="cuda"), t.zeros((2, 17), device="cuda"), 4,
                       workspace=t.zeros(1 << 16, dtype=t.uint8, device="cuda"))
    with pytest.raises(K().KvshotError):
        K().tree_level(t.zeros((2, 3, 20000), dtype=t.bfloat16, device="cuda"), t.zeros((2, 3), device="cuda"), 4,
                       workspace=t.zeros(256, dtype=t.uint8, device="cuda"))
    sc = t.zeros((2, 17), device="cuda")
    with pytest.raises(K().KvshotError):
        K().tree_expand(sc, t.zeros((2, 17, 4), dtype=t.int32, device="cuda"),
                        t.zeros((2, 17, 4), device="cuda"), 4)
