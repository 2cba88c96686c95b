"""kvshot_draft_attn_call_noalloc against kvshot_draft_attn_call.

Both run the same plan and kernels; the no-allocation call keeps the split
partials in the library's static scratch instead of the handle's workspace, so
the outputs (and LSE) must be bitwise equal.  Two calls in a row, the second
with a smaller input (the scratch still holds the first call's partials), both
also checked against the float64 oracle.  A call whose partials exceed the
scratch is rejected before anything is queued.
"""
import numpy as np
import pytest

import workloads as W
from tests import _gpu as G

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _both(att, dc, noalloc_first):
    import torch
    c = dc.case
    B, nq = c.q.shape[0], c.q.shape[1]
    res = {}
    for noalloc in ((True, False) if noalloc_first else (False, True)):
        out = torch.full((B, nq, c.num_q_heads, c.head_dim), float("nan"), dtype=torch.bfloat16, device="cuda")
        lse = torch.full((B, nq, c.num_q_heads), float("nan"), dtype=torch.float32, device="cuda")
        fn = att.step if c.mode == "step" else att.tree
        fn(dc.q, dc.k_pages, dc.v_pages, dc.page_table, dc.ctx_lens, dc.draft_k, dc.draft_v, dc.extra,
           max_ctx=int(c.ctx_lens.max()), out=out, lse=lse, noalloc=noalloc)
        torch.cuda.synchronize()
        res[noalloc] = (out, lse)
    return res


def test_noalloc_call_matches_the_workspace_call_twice_second_smaller():
    import torch
    # first call: a 60-node tree over three sequences, four splits (tall-tile kernel, partials used)
    c1 = W.make_case(mode="tree", batch=3, ctx_lens=[3000, 1200, 17], n_new=60, max_draft=64, seed=171,
                     max_pages_per_seq=192)
    # second call: smaller -- two sequences, five causal steps, the automatic plan (general kernel,
    # splits shared out by length); its page pool is smaller than the first one's, which sizes the handle
    c2 = W.make_case(batch=2, ctx_lens=[2500, 700], n_new=5, step_offsets=[3, 0], max_draft=64, seed=172,
                     max_pages_per_seq=192)
    assert c2.num_pages <= c1.num_pages
    # one pool size for both (the handle's): NaN pages pad the second pool
    pad = np.full((c1.num_pages - c2.num_pages,) + c2.k_pages.shape[1:], W.BF16_NAN, np.uint16)
    c2.k_pages = np.concatenate([c2.k_pages, pad])
    c2.v_pages = np.concatenate([c2.v_pages, pad])
    assert c2.num_pages == c1.num_pages and c2.max_pages_per_seq == c1.max_pages_per_seq
    with G.handle_for(c1) as att:
        for c, splits, first in ((c1, 4, True), (c2, 0, False)):
            print(f"noalloc case {c.mode} batch {c.batch} n {c.n_new} splits {splits or 'auto'}", flush=True)
            att.set_option(0, splits)
            plan = att.plan(c.batch, c.n_new, int(c.ctx_lens.max()))
            assert plan["splits"] == splits if splits else plan["splits"] > 1, plan
            # pools sized for this case; the handle's pool bound covers both
            dc = G.DevCase(c)
            res = _both(att, dc, noalloc_first=first)
            (o_na, l_na), (o_ws, l_ws) = res[True], res[False]
            assert torch.equal(o_na, o_ws), "outputs differ"
            assert torch.equal(l_na, l_ws), "LSE differs"
            got = o_na.float().cpu().numpy().astype(np.float64)
            ref, _ = G.oracle_out(c)
            mx, rel = G.assert_parity(got, ref, "bf16", f"noalloc {c.mode}")
            print(f"noalloc {c.mode}: bitwise equal to the workspace call; max_abs {mx:.3e} rel_l2 {rel:.3e}",
                  flush=True)


def test_noalloc_call_rejects_partials_beyond_the_scratch():
    import torch

    from paper_2604_26412_amd import KvshotError
    # 16 sequences x 8 KV heads x 256 rows x 64 splits of partials (about 1 GiB) exceed the 32 MiB scratch
    c = W.make_case(mode="tree", batch=16, ctx_lens=[2048] * 16, n_new=64, max_draft=64, seed=173)
    dc = G.DevCase(c)
    with G.handle_for(c) as att:
        att.set_option(0, 64)
        assert att.plan(16, 64, 2048)["splits"] == 64
        out = torch.full((16, 64, 32, 128), 7.0, dtype=torch.bfloat16, device="cuda")
        with pytest.raises(KvshotError) as ei:
            att.tree(dc.q, dc.k_pages, dc.v_pages, dc.page_table, dc.ctx_lens, dc.draft_k, dc.draft_v, dc.extra,
                     max_ctx=2048, out=out, noalloc=True)
        assert ei.value.status == 6
        torch.cuda.synchronize()
        assert bool((out == 7.0).all()), "a rejected call wrote its output"
        # the same call through the workspace entry point runs
        att.tree(dc.q, dc.k_pages, dc.v_pages, dc.page_table, dc.ctx_lens, dc.draft_k, dc.draft_v, dc.extra,
                 max_ctx=2048, out=out)
        torch.cuda.synchronize()
        assert bool(torch.isfinite(out.float()).all())
