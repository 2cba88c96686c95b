"""GPU parity of the general call: a position base separate from the prefix length
and a query-node subset of the tree.

These serve the variants that reuse the attention kernel:
- head concatenation of L_s target layers as one long prefix (Sec. 3.2);
- level-wise tree growth, where only the newest level's nodes query (Sec. 3.5);
- multi-layer drafters, one call per layer (Sec. 3.3);
- the hybrid self-attention branch over the drafter's own cache (Sec. 3.4.1, Eq. (self-attn)).

Bars as in test_gpu_parity.py.
"""
import sys

import numpy as np
import pytest

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


def check_lse(case, lse, ref_lse, what):
    bound = G.lse_tolerance(case)
    worst = float((np.abs(lse - ref_lse) / bound).max())
    assert worst <= 1.0, f"{what}: lse error exceeds its bound by {worst:.2f}x"


def run_call(att, c, dc, *, pos_base=None, query_nodes=None, max_ctx=None):
    t = G.torch()
    B, n = c.q.shape[0], c.q.shape[1]
    lse = t.empty((B, n, c.num_q_heads), dtype=t.float32, device="cuda")
    mc = int(c.ctx_lens.max()) if max_ctx is None else max_ctx
    pb = G.dev_array(np.asarray(pos_base, np.int32)) if pos_base is not None else None
    if c.mode == "step":
        out = att.step(dc.q, dc.k_pages, dc.v_pages, dc.page_table, dc.ctx_lens, dc.draft_k, dc.draft_v, dc.extra,
                       max_ctx=mc, lse=lse, pos_base=pb)
    else:
        qn = G.dev_array(np.asarray(query_nodes, np.int32)) if query_nodes is not None else None
        out = att.tree(dc.q, dc.k_pages, dc.v_pages, dc.page_table, dc.ctx_lens, dc.draft_k, dc.draft_v, dc.extra,
                       max_ctx=mc, lse=lse, pos_base=pb, query_nodes=qn)
    t.cuda.synchronize()
    return out.float().cpu().numpy().astype(np.float64), lse.cpu().numpy().astype(np.float64)


@pytest.mark.parametrize("mode", ["step", "tree"])
@pytest.mark.parametrize("splits", [0, 1, 5])
def test_position_base_matches_oracle(mode, splits):
    kw = dict(mode=mode, batch=3, ctx_lens=[300, 45, 0], dtype="bf16", page_size=16, seed=21)
    c = W.make_case(n_new=6 if mode == "step" else 20, step_offsets=[2, 0, 5] if mode == "step" else None,
                    max_draft=20, **kw)
    c.pos_base = np.array([17, 4000, 9], np.int32)
    ref, ref_lse = G.oracle_out(c)
    dc = G.DevCase(c)
    with G.handle_for(c, extra_positions=4100) as att:
        att.set_option(0, splits)
        out, lse = run_call(att, c, dc, pos_base=c.pos_base)
    mx, rel = G.assert_parity(out, ref, c.dtype, f"pos_base {mode} splits={splits}")
    check_lse(c, lse, ref_lse, f"pos_base {mode}")
    _log(f"pos_base {mode} splits={splits}: max_abs {mx:.2e} rel {rel:.2e}")


def test_position_base_equal_to_prefix_length_is_bitwise_the_default():
    c = W.make_case(mode="tree", batch=2, ctx_lens=[200, 33], n_new=30, dtype="bf16", seed=22)
    dc = G.DevCase(c)
    with G.handle_for(c) as att:
        a, _ = run_call(att, c, dc)
        b, _ = run_call(att, c, dc, pos_base=c.ctx_lens)
    assert np.array_equal(a, b)


@pytest.mark.parametrize("n_nodes,group", [(60, 4), (24, 8), (64, 1)])
def test_level_wise_tree_queries_only_the_newest_level(n_nodes, group):
    # the tree's keys are all n_nodes nodes; the queries are the nodes of its deepest level
    hq = 8 * group
    c = W.make_case(mode="tree", batch=4, ctx_lens=[1000, 64, 513, 7], n_new=n_nodes, num_q_heads=hq,
                    dtype="bf16", seed=23 + n_nodes)
    full = G.oracle_out(c)
    import oracle
    depth = [oracle.tree_ancestry(c.parents[b])[1] for b in range(4)]
    # a fixed-width query set: the deepest nodes of each tree (padded with the deepest node)
    width = 8
    nodes = np.zeros((4, width), np.int32)
    for b in range(4):
        order = np.argsort(-depth[b], kind="stable")[:width]
        nodes[b, :len(order)] = order
    sub = W.make_case(mode="tree", batch=4, ctx_lens=[1000, 64, 513, 7], n_new=n_nodes, num_q_heads=hq,
                      dtype="bf16", seed=23 + n_nodes)
    sub.q = np.stack([c.q[b][nodes[b]] for b in range(4)])
    sub.query_nodes = nodes
    sub.n_new = width
    ref, ref_lse = G.oracle_out(sub)
    for b in range(4):                            # the oracle's subset is the full call's rows (up to BLAS order)
        np.testing.assert_allclose(ref[b], full[0][b][nodes[b]], rtol=0, atol=1e-12)
    dc = G.DevCase(sub)
    with G.handle_for(sub) as att:
        out, lse = run_call(att, sub, dc, query_nodes=nodes)
    mx, rel = G.assert_parity(out, ref, "bf16", f"level-wise n={n_nodes} G={group}")
    check_lse(sub, lse, ref_lse, "level-wise")
    _log(f"level-wise n={n_nodes} G={group}: max_abs {mx:.2e} rel {rel:.2e}")


def test_head_concatenated_layers_as_one_prefix():
    # L_s = 3 sampled target layers' KV laid end to end in the page table (3T prefix keys), draft
    # positions continue from the real prefix length T (reading: one softmax over the 3T keys)
    Ls, T = 3, 320
    c = W.make_case(mode="step", batch=2, ctx_lens=[Ls * T, Ls * 48], n_new=8, dtype="bf16", seed=24)
    c.pos_base = np.array([T, 48], np.int32)
    ref, ref_lse = G.oracle_out(c)
    dc = G.DevCase(c)
    with G.handle_for(c) as att:
        out, lse = run_call(att, c, dc, pos_base=c.pos_base)
    G.assert_parity(out, ref, "bf16", "head concatenation")
    check_lse(c, lse, ref_lse, "head concatenation")


def test_multi_layer_drafter_one_call_per_layer():
    # two drafter layers: different queries and different (projected) target KV, one handle, same stream
    cases = [W.make_case(mode="step", batch=3, ctx_lens=[700, 70, 7], n_new=4, dtype="bf16", seed=30 + i)
             for i in range(2)]
    refs = [G.oracle_out(c) for c in cases]
    dcs = [G.DevCase(c) for c in cases]
    with G.handle_for(cases[0]) as att:
        outs = [run_call(att, c, dc) for c, dc in zip(cases, dcs)]
    for (o, l), (r, rl), c in zip(outs, refs, cases):
        G.assert_parity(o, r, "bf16", "multi-layer")
        check_lse(c, l, rl, "multi-layer")


def test_self_attention_branch_over_the_drafters_own_cache():
    # the hybrid drafter's self-attention path reads the drafter's own paged cache (here 64-token pages)
    c = W.make_case(mode="step", batch=2, ctx_lens=[900, 130], n_new=5, page_size=64, dtype="bf16", seed=40)
    ref, ref_lse = G.oracle_out(c)
    dc = G.DevCase(c)
    with G.handle_for(c) as att:
        out, lse = run_call(att, c, dc)
    G.assert_parity(out, ref, "bf16", "self-attention branch")
    check_lse(c, lse, ref_lse, "self-attention branch")


def test_validate_call_reports_query_nodes_and_positions():
    t = G.torch()
    c = W.make_case(mode="tree", batch=2, ctx_lens=[100, 50], n_new=10, dtype="bf16", seed=41)
    dc = G.DevCase(c)
    with G.handle_for(c) as att:
        import ctypes
        import paper_2604_26412_amd as K

        def validate(query_nodes, pos_base):
            call = K.KvshotCall()
            call.mode, call.batch, call.n_queries, call.n_nodes = K.MODE_TREE, 2, query_nodes.shape[1], 10
            call.max_ctx_len_hint = 100
            call.page_table, call.ctx_lens, call.parents = (dc.page_table.data_ptr(), dc.ctx_lens.data_ptr(),
                                                            dc.extra.data_ptr())
            qn = G.dev_array(query_nodes)
            call.query_nodes = qn.data_ptr()
            pb = G.dev_array(pos_base) if pos_base is not None else None
            call.pos_base = pb.data_ptr() if pb is not None else None
            bad = ctypes.c_int32(-1)
            st = att._lib.kvshot_draft_attn_validate_call(att._h, ctypes.byref(call), ctypes.byref(bad),
                                                          t.cuda.current_stream().cuda_stream)
            return st, bad.value

        good = np.array([[9, 8, 7], [0, 1, 2]], np.int32)
        assert validate(good, None) == (0, 0)
        assert validate(good, np.array([5, 5], np.int32)) == (0, 0)
        assert validate(np.array([[9, 10, 7], [0, 1, 2]], np.int32), None) == (5, 5)
        big = np.array([5, att.cfg.max_position], np.int32)
        assert validate(good, big) == (5, 6)
        assert validate(good, np.array([-1, 0], np.int32)) == (5, 6)


def test_call_rejects_inconsistent_arguments():
    import ctypes
    import paper_2604_26412_amd as K
    c = W.make_case(mode="tree", batch=1, ctx_lens=[40], n_new=6, dtype="bf16", seed=42)
    dc = G.DevCase(c)
    t = G.torch()
    out = t.zeros((1, 6, c.num_q_heads, c.head_dim), dtype=t.bfloat16, device="cuda")
    with G.handle_for(c) as att:
        def call(**kw):
            a = K.KvshotCall()
            a.mode, a.batch, a.n_queries, a.n_nodes, a.max_ctx_len_hint = K.MODE_TREE, 1, 6, 6, 40
            a.q, a.k_pages, a.v_pages = dc.q.data_ptr(), dc.k_pages.data_ptr(), dc.v_pages.data_ptr()
            a.page_table, a.ctx_lens = dc.page_table.data_ptr(), dc.ctx_lens.data_ptr()
            a.draft_k, a.draft_v, a.parents, a.out = (dc.draft_k.data_ptr(), dc.draft_v.data_ptr(),
                                                      dc.extra.data_ptr(), out.data_ptr())
            for k, v in kw.items():
                setattr(a, k, v)
            return att._lib.kvshot_draft_attn_call(att._h, ctypes.byref(a), None)
        assert call(n_nodes=5) == 1                  # nodes != queries without query_nodes
        assert call(mode=0, step_offsets=None) == 1  # step mode needs step offsets
        assert call(reserved=1) == 1
        assert call(mode=7) == 1
        assert call(n_nodes=65) == 1
        t.cuda.synchronize()
        assert float(out.float().abs().max()) == 0.0
