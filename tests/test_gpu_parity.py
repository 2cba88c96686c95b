"""GPU parity: the HIP library (through its C ABI) against the float64 oracle.

Bars: bf16 inputs max-abs <= 2e-2 and rel-L2 <= 5e-3; float32 inputs
max-abs <= 1e-4 and rel-L2 <= 2e-5 (see tests/_gpu.py); index work bit-exact.
"""
import sys

import numpy as np
import pytest

import oracle
import workloads as W
from tests import _gpu as G

pytestmark = pytest.mark.gpu


def _log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def small(mode="step", **kw):
    base = dict(mode=mode, batch=3, ctx_lens=[100, 37, 0], n_new=4, dtype="bf16", page_size=16, seed=11)
    base.update(kw)
    return W.make_case(**base)


# ---------------------------------------------------------------------------
# bit-exact index code
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("page_size", [16, 64, 256])
def test_gather_kv_is_bit_exact(page_size):
    c = small(ctx_lens=[300, 17, 0, 513], batch=4, page_size=page_size, seed=21)
    _log(f"gather page_size={page_size}")
    dc = G.DevCase(c)
    with G.handle_for(c) as att:
        kd, vd = att.debug_gather_kv(dc.k_pages, dc.v_pages, dc.page_table, dc.ctx_lens, max_ctx=520)
        import torch
        torch.cuda.synchronize()
        kd = kd.view(torch.int16).cpu().numpy().view(np.uint16)
        vd = vd.view(torch.int16).cpu().numpy().view(np.uint16)
    ref_k = oracle.gather_dense(c.k_pages, c.page_table, c.ctx_lens, page_size, 520, fill=0)
    ref_v = oracle.gather_dense(c.v_pages, c.page_table, c.ctx_lens, page_size, 520, fill=0)
    assert np.array_equal(kd, ref_k) and np.array_equal(vd, ref_v)


def test_tree_mask_is_bit_exact():
    B, N = 8, 60
    parents = np.stack([W.random_tree(1005, b, N) for b in range(B)])
    parents[3] = np.arange(-1, N - 1)                     # chain (depth 59)
    parents[4] = -1                                       # star forest
    c = small(mode="tree", batch=B, ctx_lens=[5] * B, n_new=N, parents=parents, max_draft=64)
    _log("tree mask")
    dc = G.DevCase(c)
    with G.handle_for(c) as att:
        anc, depth = att.debug_tree_mask(dc.extra)
        anc = anc.cpu().numpy().view(np.uint64)
        depth = depth.cpu().numpy()
    for b in range(B):
        sets, dref = oracle.tree_ancestry(parents[b])
        want = np.array([sum(1 << s for s in st) for st in sets], dtype=np.uint64)
        assert np.array_equal(anc[b], want), b
        assert np.array_equal(depth[b], dref), b


# ---------------------------------------------------------------------------
# the five workload shapes
# ---------------------------------------------------------------------------

def _check_case(c, *, sequential=False, splits=None, path=None, want_lse=True, what=""):
    dc = G.DevCase(c)
    ref, ref_lse = G.oracle_out(c)
    with G.handle_for(c) as att:
        if splits is not None:
            att.set_option(0, splits)
        if path is not None:
            att.set_option(1, path)
        if not sequential:
            out, lse = G.run(att, dc, want_lse=True)
        else:
            import torch
            outs, lses = [], []
            for j in range(c.n_new):
                offs = G.dev_array((c.step_offsets + j).astype(np.int32))
                o, l = G.run(att, dc, q=dc.q[:, j:j + 1].contiguous(), extra=offs, want_lse=True)
                outs.append(o)
                lses.append(l)
            out, lse = np.concatenate(outs, 1), np.concatenate(lses, 1)
    mx, rel = G.assert_parity(out, ref, c.dtype, what)
    if want_lse:
        bound = G.lse_tolerance(c)
        worst = float((np.abs(lse - ref_lse) / bound).max())
        assert worst <= 1.0, f"{what}: lse error exceeds its bound by {worst:.2f}x"
    _log(f"{what}: max_abs {mx:.3e} rel_l2 {rel:.3e}")
    return out


@pytest.mark.parametrize("sequential", [False, True])
def test_tiny_fp32_single_page(sequential):
    c = W.workload("tiny_fp32_ctx256")
    assert c.page_table.tolist() == [[0]]
    _check_case(c, sequential=sequential, what=f"tiny fp32 seq={sequential}")


def test_tiny_fp32_identity_table_page16():
    c = W.workload("tiny_fp32_ctx256", page_size=16)
    _check_case(c, what="tiny fp32 P=16")


def test_tiny_fp32_literal_scale():
    c = W.workload("tiny_fp32_ctx256", softmax_scale=1.0)
    _check_case(c, what="tiny fp32 scale=1")


@pytest.mark.parametrize("sequential", [False, True])
def test_single_ctx4096_k8(sequential):
    c = W.workload("single_ctx4096_k8")
    _check_case(c, sequential=sequential, what=f"ctx4096 k8 seq={sequential}")


@pytest.mark.parametrize("sequential", [False, True])
def test_ragged_b16_k6(sequential):
    c = W.workload("ragged_b16_k6")
    _check_case(c, sequential=sequential, what=f"ragged b16 seq={sequential}")


def test_tree_b8_ctx16k_n60():
    c = W.workload("tree_b8_ctx16k_n60")
    _check_case(c, what="tree b8 ctx16k n60")


# ---------------------------------------------------------------------------
# the 64 x 32768 workload the headline metric is quoted on (generated on the
# device; whole sampled sequences are copied back for the oracle)
# ---------------------------------------------------------------------------

LONG_SAMPLE = [0, 21, 42, 63]          # first, two interior, last


@pytest.fixture(scope="module")
def long_range():
    import torch

    import workloads.device as WD
    _log("generating the 64 x 32768 workload on the device")
    d = WD.long_range_on_device(torch, 1004)
    torch.cuda.synchronize()
    # the pool holds more than 2^31 elements per tensor, so 32-bit element offsets would wrap
    assert d["k_pages"].numel() > 2 ** 31
    host = WD.host_sample(torch, d, LONG_SAMPLE)
    ref, ref_lse = G.oracle_out(host)
    yield d, host, ref, ref_lse
    del d
    torch.cuda.empty_cache()


@pytest.mark.parametrize("sequential", [False, True])
def test_long_b64_ctx32k_k8(long_range, sequential):
    """Whole batch on the GPU in the bench's launch configuration (automatic plan); four whole
    sequences checked element by element, LSE included."""
    import torch

    from paper_2604_26412_amd import DraftAttention
    d, host, ref, ref_lse = long_range
    B, n, Hq, D = d["B"], d["n"], d["Hq"], d["D"]
    T = d["lens"][0]
    out = torch.empty((B, n, Hq, D), dtype=torch.bfloat16, device="cuda")
    lse = torch.empty((B, n, Hq), dtype=torch.float32, device="cuda")
    with DraftAttention(num_q_heads=Hq, num_kv_heads=d["Hkv"], head_dim=D, page_size=d["P"], dtype="bf16",
                        max_batch=B, max_draft=d["max_draft"], max_pages_per_seq=d["pps"],
                        num_pages=d["pool"]) as att:
        _log(f"64 x 32K sequential={sequential}: plan {att.plan(B, 1 if sequential else n, T)}")
        if not sequential:
            att.step(d["q"], d["k_pages"], d["v_pages"], d["page_table"], d["ctx_lens"], d["draft_k"],
                     d["draft_v"], d["extra"], max_ctx=T, out=out, lse=lse)
        else:
            for j in range(n):
                oj = torch.empty((B, 1, Hq, D), dtype=torch.bfloat16, device="cuda")
                lj = torch.empty((B, 1, Hq), dtype=torch.float32, device="cuda")
                att.step(d["q"][:, j:j + 1].contiguous(), d["k_pages"], d["v_pages"], d["page_table"],
                         d["ctx_lens"], d["draft_k"], d["draft_v"], (d["extra"] + j).contiguous(), max_ctx=T,
                         out=oj, lse=lj)
                out[:, j:j + 1] = oj
                lse[:, j:j + 1] = lj
        torch.cuda.synchronize()
    assert torch.isfinite(out.float()).all(), "non-finite output in the unsampled sequences"
    got = out[LONG_SAMPLE].float().cpu().numpy().astype(np.float64)
    got_lse = lse[LONG_SAMPLE].cpu().numpy().astype(np.float64)
    mx, rel = G.assert_parity(got, ref, "bf16", f"64 x 32K sequential={sequential}")
    worst = float((np.abs(got_lse - ref_lse) / G.lse_tolerance(host)).max())
    assert worst <= 1.0, f"lse error exceeds its bound by {worst:.2f}x"
    _log(f"64 x 32K sequential={sequential}: max_abs {mx:.3e} rel_l2 {rel:.3e} lse/bound {worst:.3f}")


# ---------------------------------------------------------------------------
# tall query tiles (more than 32 rows per (sequence, KV head)) on outlier keys:
# the recipe of the single-sequence workload (4 channels per KV head x 8) and
# a heavier one (2 channels x 32), which make scores sensitive to the query's
# rounding
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("outliers", [(4, 8.0), (2, 32.0)])
@pytest.mark.parametrize("n_new", [9, 16, 33, 64])
def test_tall_tiles_outlier_keys(n_new, outliers):
    no, sc = outliers
    c = small(n_new=n_new, max_draft=64, ctx_lens=[4096, 1500, 0], n_outlier=no, outlier_scale=sc,
              seed=151 + n_new)
    _check_case(c, what=f"tall tile n_new={n_new} outliers {no}x{sc:g}")


@pytest.mark.parametrize("page_size", [32, 64, 256])
def test_tall_tiles_page_sizes(page_size):
    """256-row tiles (40 draft queries x 4 heads) on pages of 32 to 256 slots: both 16-key halves of
    a block then sit in one page, and the prefix ends mid-page."""
    c = small(n_new=40, max_draft=64, ctx_lens=[3000, 517, 0], page_size=page_size, seed=181)
    with G.handle_for(c) as att:
        assert att.plan(c.batch, c.n_new, 3000)["path"] == 3
    _check_case(c, what=f"tall tile P={page_size}")


@pytest.mark.parametrize("lens", [[0, 1, 31, 33, 100], [16, 32, 0, 5000, 64]])
def test_tall_tree_short_prefixes(lens):
    """60-node trees over prefixes of 0 to a few blocks: splits whose target range is empty, a last
    split of draft blocks only, and a block ending mid-page, on the 256-row tile kernel."""
    parents = np.stack([W.random_tree(191, b, 60) for b in range(len(lens))])
    c = small(mode="tree", batch=len(lens), n_new=60, max_draft=64, parents=parents, ctx_lens=lens, seed=193)
    with G.handle_for(c) as att:
        assert att.plan(c.batch, c.n_new, int(max(lens)))["path"] == 3
    _check_case(c, what=f"tall tree prefixes {lens}")


@pytest.mark.parametrize("outliers", [(4, 8.0), (2, 32.0)])
def test_tree_b8_ctx16k_n60_outlier_keys(outliers):
    no, sc = outliers
    c = W.workload("tree_b8_ctx16k_n60", n_outlier=no, outlier_scale=sc)
    _check_case(c, what=f"tree b8 ctx16k n60 outliers {no}x{sc:g}")


@pytest.mark.parametrize("splits", [None, 1, 3])
def test_tall_tiles_on_the_general_kernel(splits):
    """256-row query tiles on the general MFMA kernel (path option 3; it also serves splits the
    tall-tile kernel cannot stage, more than 512 blocks), with outlier keys; same bars.  The tall-tile
    kernel raises a forced split count to its 512-block cap instead."""
    parents = np.stack([W.random_tree(181, b, 60) for b in range(2)])
    c = W.make_case(mode="tree", batch=2, ctx_lens=[17000, 3001], n_new=60, parents=parents, n_outlier=4,
                    seed=181)
    with G.handle_for(c) as att:
        att.set_option(1, 3)
        if splits:
            att.set_option(0, splits)
        plan = att.plan(2, 60, 17000)
        assert plan["path"] == 1, plan
        att.set_option(1, 1)
        assert att.plan(2, 60, 17000)["path"] == 3
        if splits == 1:
            assert att.plan(2, 60, 17000)["splits"] == 2      # 532 blocks: raised to the cap
    _check_case(c, splits=splits, path=3, what=f"tree on the general kernel, splits {splits}")


# ---------------------------------------------------------------------------
# edge cases
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("lens", [[0, 0], [1, 31], [32, 33], [15, 16], [17, 4095]])
def test_ragged_tails_and_empty_prefix(lens):
    c = small(batch=2, ctx_lens=lens, n_new=3, step_offsets=[2, 0], max_draft=6, seed=31)
    _check_case(c, what=f"tails {lens}")


_BALANCED_LENS = [
    # 32 sequences (the largest batch the balanced plan takes with 8 KV heads on 256 CUs): one long
    # prefix among empty, sub-block, block-edge and page-edge lengths
    [9000] + [0, 1, 31, 32, 33, 64, 65, 100, 511, 512, 513] * 2 + [7, 3, 2000, 4096, 0, 1, 15, 16, 17],
    # one prefix long enough that its share of the items hits the per-sequence cap of 64 splits
    [40000, 16],
    # every prefix shorter than one block (the handle sized for 1024-token prefixes, so that its
    # workspace holds the balanced plan's partials)
    [1] * 16,
]


@pytest.mark.parametrize("lens", _BALANCED_LENS, ids=["b32_mixed", "b2_capped", "b16_tiny"])
def test_balanced_schedule_extremes(lens):
    """Length-balanced split schedule (computed on the device from the lengths): every sequence's
    items, the per-sequence split cap, empty and sub-block prefixes, checked against the oracle."""
    c = small(batch=len(lens), ctx_lens=lens, n_new=3, seed=37, max_pages_per_seq=max(64, -(-max(lens) // 16)))
    with G.handle_for(c) as att:
        pl = att.plan(c.batch, c.n_new, int(max(lens)))
    # a balanced plan launches its items per KV head, independent of the batch (12 rows: one row tile)
    assert pl["row_tiles"] == 1 and pl["workgroups"] == pl["splits"] * c.num_kv_heads, pl
    _check_case(c, what=f"balanced {len(lens)} seqs, max {max(lens)}")


@pytest.mark.parametrize("page_size", [32, 64, 128, 256])
def test_page_sizes(page_size):
    c = small(ctx_lens=[700, 129, 3], page_size=page_size, seed=41)
    _check_case(c, what=f"P={page_size}")


@pytest.mark.parametrize("heads", [(8, 8), (16, 8), (64, 8), (32, 4)])
def test_group_sizes(heads):
    c = small(num_q_heads=heads[0], num_kv_heads=heads[1], seed=51)
    _check_case(c, what=f"heads {heads}")


@pytest.mark.parametrize("n_new", [1, 8, 9, 16, 33, 64])
def test_draft_lengths(n_new):
    c = small(n_new=n_new, max_draft=64, ctx_lens=[300, 40, 0], seed=61)
    _check_case(c, what=f"n_new {n_new}")


@pytest.mark.parametrize("splits", [1, 2, 7, 13, 64])
def test_split_invariance(splits):
    c = small(ctx_lens=[3000, 2100, 999], n_new=8, seed=71)
    _check_case(c, splits=splits, what=f"splits {splits}")


def test_generic_path_on_bf16():
    c = small(ctx_lens=[500, 260, 7], n_new=5, seed=81)
    _check_case(c, path=2, what="generic bf16")


def test_tree_shapes_small():
    parents = np.array([[-1, 0, 0, 1, 1, 2, -1, 6], [-1, -1, -1, -1, -1, -1, -1, -1], [-1, 0, 1, 2, 3, 4, 5, 6]],
                       np.int32)
    c = small(mode="tree", n_new=8, parents=parents, ctx_lens=[77, 0, 513], seed=91)
    _check_case(c, what="tree small")


def test_fp32_output_mode():
    c = small(ctx_lens=[999, 64, 5], n_new=6, seed=101)
    dc = G.DevCase(c)
    ref, _ = G.oracle_out(c)
    with G.handle_for(c, out_dtype="fp32") as att:
        out = G.run(att, dc)
    mx, rel = G.errors(out, ref)
    assert mx <= G.BF16_MAX_ABS and rel <= 3e-3, (mx, rel)


def test_determinism_bitwise():
    c = small(ctx_lens=[2000, 1500, 1], n_new=6, seed=111)
    dc = G.DevCase(c)
    with G.handle_for(c) as att:
        a = G.run(att, dc)
        b = G.run(att, dc)
    assert np.array_equal(a, b)


# ---------------------------------------------------------------------------
# probes through the production kernels
# ---------------------------------------------------------------------------

def test_hot_key_probe_returns_that_value_bitwise():
    """One logical target position gets a score far above the rest; the output is its V exactly."""
    torch = pytest.importorskip("torch")
    P = 16
    probes = [0, 15, 16, 31, 32, 100, 511, 1000, 1022]     # first/last page slots, tail, mid
    B = len(probes)
    lens = [1023] * B
    c = W.make_case(batch=B, ctx_lens=lens, n_new=2, page_size=P, seed=121)
    G_ = c.num_q_heads // c.num_kv_heads
    # zero every key; the probed key of each sequence points along its rotated query
    c.k_pages[...] = np.where(np.isnan(W.bf16_bits_to_f32(c.k_pages)), c.k_pages, np.uint16(0))
    c.draft_k[...] = np.where(np.isnan(W.bf16_bits_to_f32(c.draft_k)), c.draft_k, np.uint16(0))
    # same query for every head: a single channel
    qf = np.zeros(c.q.shape, np.float32)
    qf[..., 0] = 1.0
    c.q = W.f32_to_bf16_bits(qf)
    for b, t in enumerate(probes):
        # the query of row j sits at position T + j; target keys are used as stored, so put the key
        # along rope(q, T) for j = 0 with a large norm
        rq = oracle.rope(oracle.decode(c.q[b, 0, 0], "bf16"), lens[b], c.rope_theta)
        key = W.f32_to_bf16_bits((rq * 4000.0).astype(np.float32))
        pid = c.page_table[b, t // P]
        c.k_pages[pid, :, t % P] = key
    dc = G.DevCase(c)
    with G.handle_for(c) as att:
        out = G.run(att, dc)
    for b, t in enumerate(probes):
        pid = c.page_table[b, t // P]
        for hq in range(c.num_q_heads):
            want = oracle.decode(c.v_pages[pid, hq // G_, t % P], "bf16")
            assert np.array_equal(out[b, 0, hq], want), (b, t, hq)


def test_mask_probe_nonzero_pattern_is_the_allowed_set():
    """K = 0 (uniform scores), target V = 0, draft V of key s = one-hot channel s."""
    N = 40
    parents = np.stack([W.random_tree(7, b, N) for b in range(3)])
    for mode in ("tree", "step"):
        if mode == "tree":
            c = W.make_case(mode="tree", batch=3, ctx_lens=[50, 0, 33], n_new=N, parents=parents, max_draft=N,
                            seed=131)
        else:
            c = W.make_case(batch=3, ctx_lens=[50, 0, 33], n_new=12, step_offsets=[0, 5, 28], max_draft=N,
                            seed=131)
        live = ~np.isnan(W.bf16_bits_to_f32(c.k_pages))
        c.k_pages[live] = 0
        c.v_pages[live] = 0
        S = c.draft_k.shape[1]
        c.draft_k[...] = 0
        dv = np.zeros(c.draft_v.shape, np.float32)
        for s in range(S):
            dv[:, s, :, s] = 1.0
        c.draft_v = W.f32_to_bf16_bits(dv)
        dc = G.DevCase(c)
        with G.handle_for(c) as att:
            out = G.run(att, dc)
        for b in range(3):
            for i in range(c.n_new):
                if mode == "tree":
                    allowed = sorted(oracle.tree_ancestry(parents[b])[0][i])
                else:
                    allowed = list(range(int(c.step_offsets[b]) + i + 1))
                nz = np.nonzero(out[b, i, 0])[0].tolist()
                assert nz == allowed, (mode, b, i)


def test_hip_graph_replay_matches_eager():
    """A captured step replays to the eager result, with eager work and syncs between replays."""
    torch = pytest.importorskip("torch")
    c = small(ctx_lens=[3000, 700, 0], n_new=8, seed=141)
    dc = G.DevCase(c)
    with G.handle_for(c) as att:
        att.set_option(0, 3)                       # force split-K so the combine kernel is captured too
        out = torch.empty((3, 8, 32, 128), dtype=torch.bfloat16, device="cuda")
        lse = torch.empty((3, 8, 32), dtype=torch.float32, device="cuda")

        def step():
            att.step(dc.q, dc.k_pages, dc.v_pages, dc.page_table, dc.ctx_lens, dc.draft_k, dc.draft_v, dc.extra,
                     max_ctx=3000, out=out, lse=lse)
        step()
        torch.cuda.synchronize()
        eager, eager_lse = out.clone(), lse.clone()
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            step()
        torch.cuda.current_stream().wait_stream(side)
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            step()
        for rep in range(4):
            out.zero_()
            lse.zero_()
            torch.cuda.synchronize()
            g.replay()
            torch.cuda.synchronize()
            assert torch.equal(out, eager), rep
            assert torch.equal(lse, eager_lse), rep
            step()                                 # eager work between replays
            torch.cuda.synchronize()


@pytest.mark.parametrize("n,hq", [(40, 8), (30, 8), (40, 16)])
@pytest.mark.parametrize("lens", [[0, 5], [33, 0]])
def test_star_forest_blocks_fully_masked_for_some_rows(n, hq, lens):
    # every node is a root, so it sees only its own draft key: a key stream whose first block holds none
    # of a row's visible keys must leave that row's state empty (no -inf - -inf), not NaN
    parents = np.full((2, n), -1, np.int32)
    c = W.make_case(mode="tree", batch=2, ctx_lens=lens, n_new=n, num_q_heads=hq, parents=parents,
                    dtype="bf16", seed=60 + n)
    for splits in (None, 1):
        _check_case(c, splits=splits, what=f"star forest n={n} hq={hq} lens={lens} splits={splits}")
