"""GPU parity of the gated delta fusion (Sec. 3.4.1, Eqs. (delta), (fusion)) against the float64 oracle.

Error budget (bf16 activations and weights, float32 accumulation): Delta is
rounded to bf16 for the product (2^-9 relative per element, ~1e-3 of the
delta projection after the reduction averages it), the gate sees the same
rounding through W_g, and a bf16 output adds half an ulp, at most 2^-8 |h|.
Bars per element: |err| <= 2^-8 |h_ref| + 1e-2 (bf16 out) or <= 1e-2 (float32
out); rel-L2 <= 5e-3 (bf16 out) or 3e-3 (float32 out).
"""
import sys

import numpy as np
import pytest

from oracle.fusion import gated_delta_fusion
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


def dec(bits):
    return W.bf16_bits_to_f32(bits).astype(np.float64)


def reference(c, rows=None, cross_only=False):
    rows = np.arange(c.tokens) if rows is None else rows
    return gated_delta_fusion(dec(c.n[rows]), dec(c.o[rows]), dec(c.w_g), c.b_g.astype(np.float64),
                              dec(c.w_delta), cross_only=cross_only, return_gate=True)


def upload(c):
    return dict(n=G.dev_array(c.n), o=G.dev_array(c.o), w_g=G.dev_array(c.w_g), b_g=G.dev_array(c.b_g),
                w_delta=G.dev_array(c.w_delta))


def check(got, ref, fp32_out, what):
    got = np.asarray(got, dtype=np.float64)
    err = np.abs(got - ref)
    bound = (1e-2 if fp32_out else 2.0 ** -8 * np.abs(ref) + 1e-2)
    rel = np.linalg.norm(got - ref) / max(np.linalg.norm(ref), 1e-30)
    assert np.all(np.isfinite(got)), what
    worst = float(np.max(err - bound))
    assert worst <= 0, f"{what}: max excess over bound {worst:.3e}"
    assert rel <= (3e-3 if fp32_out else 5e-3), f"{what}: rel-L2 {rel:.3e}"
    return rel


def run(fz, dv, c, *, cross_only=False, out_dtype="bf16", gate=True):
    t = G.torch()
    g = t.empty((c.tokens, c.d), dtype=t.float32, device="cuda") if gate else None
    out = fz(None if cross_only else dv["n"], dv["o"], dv["w_g"], dv["b_g"], dv["w_delta"], gate=g,
             cross_only=cross_only, out_dtype=out_dtype)
    t.cuda.synchronize()
    return out.float().cpu().numpy(), (g.cpu().numpy() if gate else None)


@pytest.mark.parametrize("d", [256, 512])
@pytest.mark.parametrize("tokens", [1, 37, 64, 100])
@pytest.mark.parametrize("splits", [0, 1, 2, 4, 8, 16])
def test_fusion_matches_oracle(tokens, d, splits):
    from paper_2604_26412_amd import GatedDeltaFusion, OPT_SPLITS
    _log(f"fusion tokens={tokens} d={d} splits={splits}")
    c = W.fusion_case(tokens, d, seed=tokens * 7 + d)
    h_ref, g_ref = reference(c)
    with GatedDeltaFusion(d, max(tokens, 64)) as fz:
        fz.set_option(OPT_SPLITS, splits)
        h, g = run(fz, upload(c), c)
    check(h, h_ref, False, f"h tokens={tokens} d={d} splits={splits}")
    assert np.max(np.abs(g - g_ref)) <= 5e-3


@pytest.mark.parametrize("d", [256, 512, 768])
@pytest.mark.parametrize("tokens", [1, 100, 128, 200, 300])
@pytest.mark.parametrize("splits", [0, 1, 2, 4])
def test_fusion_128_token_tiles_match_oracle(tokens, d, splits):
    # 128-token tiles (KVSHOT_OPT_PATH 2): splits take parts of the reduction index range of all four
    # segments; ragged last tiles at 100, 200 and 300 tokens.  The main loop runs whole pairs of
    # 64-index chunks and then the rest: d = 256 with 4 splits has one chunk per split (no pair),
    # d = 768 with 4 splits three (one pair and one more)
    from paper_2604_26412_amd import GatedDeltaFusion, OPT_SPLITS, OPT_PATH
    _log(f"fusion 128-token tiles tokens={tokens} d={d} splits={splits}")
    c = W.fusion_case(tokens, d, seed=tokens * 11 + d + splits)
    h_ref, g_ref = reference(c)
    with GatedDeltaFusion(d, max(tokens, 64)) as fz:
        fz.set_option(OPT_SPLITS, splits)
        fz.set_option(OPT_PATH, 2)
        plan = fz.plan(tokens)
        assert plan["workgroups"] == -(-tokens // 128) * (d // 128) * plan["splits"], plan
        h, g = run(fz, upload(c), c)
    check(h, h_ref, False, f"h 128-token tiles tokens={tokens} d={d} splits={splits}")
    assert np.max(np.abs(g - g_ref)) <= 5e-3


@pytest.mark.parametrize("tokens", [128, 200, 256, 300, 480])
def test_fusion_automatic_plan_at_large_token_counts(tokens):
    from paper_2604_26412_amd import GatedDeltaFusion
    c = W.fusion_case(tokens, 512, seed=tokens + 3)
    h_ref, g_ref = reference(c)
    with GatedDeltaFusion(512, tokens) as fz:
        plan = fz.plan(tokens)
        h, g = run(fz, upload(c), c)
    check(h, h_ref, False, f"h automatic tokens={tokens} (plan {plan})")
    assert np.max(np.abs(g - g_ref)) <= 5e-3


@pytest.mark.parametrize("tile", [1, 2])
def test_fusion_tiles_agree_with_packed_weights_and_fp32_output(tile):
    from paper_2604_26412_amd import GatedDeltaFusion, OPT_PATH, OPT_SPLITS
    t = G.torch()
    c = W.fusion_case(150, 256, seed=41)
    h_ref, g_ref = reference(c)
    with GatedDeltaFusion(256, 150) as fz:
        fz.set_option(OPT_PATH, tile)
        dv = upload(c)
        packed = fz.pack_weights(dv["w_g"], dv["w_delta"])
        for splits in (1, 2):
            fz.set_option(OPT_SPLITS, splits)
            a = fz(dv["n"], dv["o"], dv["w_g"], dv["b_g"], dv["w_delta"], out_dtype="fp32")
            b = fz(dv["n"], dv["o"], None, dv["b_g"], None, packed=packed, out_dtype="fp32")
            t.cuda.synchronize()
            assert t.equal(a, b), (tile, splits)
            check(a.cpu().numpy(), h_ref, True, f"fp32 tile {64 * tile} splits {splits}")


@pytest.mark.parametrize("splits", [1, 8])
def test_fusion_float32_output_and_gate(splits):
    from paper_2604_26412_amd import GatedDeltaFusion, OPT_SPLITS
    c = W.fusion_case(70, 512, seed=5)
    h_ref, g_ref = reference(c)
    with GatedDeltaFusion(512, 70) as fz:
        fz.set_option(OPT_SPLITS, splits)
        h, g = run(fz, upload(c), c, out_dtype="fp32")
    check(h, h_ref, True, f"fp32 out splits={splits}")
    assert np.max(np.abs(g - g_ref)) <= 5e-3


@pytest.mark.parametrize("tile", [1, 2])
@pytest.mark.parametrize("splits", [1, 4])
def test_fusion_cross_only(splits, tile):
    # reading: the cross-only variant drops n (n = 0, Delta = o)
    from paper_2604_26412_amd import GatedDeltaFusion, OPT_SPLITS, OPT_PATH
    c = W.fusion_case(50, 256, seed=6)
    h_ref, g_ref = reference(c, cross_only=True)
    with GatedDeltaFusion(256, 64) as fz:
        fz.set_option(OPT_SPLITS, splits)
        fz.set_option(OPT_PATH, tile)
        h, g = run(fz, upload(c), c, cross_only=True)
    check(h, h_ref, False, f"cross-only splits={splits}")
    assert np.max(np.abs(g - g_ref)) <= 5e-3


@pytest.mark.parametrize("splits", [1, 8])
def test_fusion_shut_gate_returns_n_bit_exact(splits):
    # sigmoid saturates to exactly 0, so h = n + 0 * (W_Delta Delta) = n bit for bit
    from paper_2604_26412_amd import GatedDeltaFusion, OPT_SPLITS
    t = G.torch()
    c = W.fusion_case(64, 256, seed=8)
    c.b_g[:] = -1e4
    with GatedDeltaFusion(256, 64) as fz:
        fz.set_option(OPT_SPLITS, splits)
        dv = upload(c)
        g = t.empty((64, 256), dtype=t.float32, device="cuda")
        out = fz(dv["n"], dv["o"], dv["w_g"], dv["b_g"], dv["w_delta"], gate=g)
        t.cuda.synchronize()
    assert np.array_equal(out.cpu().view(t.int16).numpy().view(np.uint16), c.n)
    assert float(g.abs().max()) == 0.0


def test_fusion_is_deterministic_and_split_invariant():
    from paper_2604_26412_amd import GatedDeltaFusion, OPT_SPLITS
    c = W.fusion_case(64, 512, seed=9)
    with GatedDeltaFusion(512, 64) as fz:
        dv = upload(c)
        outs = {}
        for s in (1, 8):
            fz.set_option(OPT_SPLITS, s)
            a, _ = run(fz, dv, c, gate=False, out_dtype="fp32")
            b, _ = run(fz, dv, c, gate=False, out_dtype="fp32")
            assert np.array_equal(a, b), f"splits={s} not bitwise repeatable"
            outs[s] = a
    # the splits only reorder float32 sums
    assert np.max(np.abs(outs[1] - outs[8])) <= 1e-4 * (1 + np.max(np.abs(outs[1])))


@pytest.mark.parametrize("splits,tile", [(1, 1), (8, 1), (2, 2)])
def test_fusion_hip_graph_replay_matches_eager(splits, tile):
    """A captured call replays to the eager result, with eager work and syncs between replays
    (split path: the combine kernel is captured too)."""
    from paper_2604_26412_amd import GatedDeltaFusion, OPT_SPLITS, OPT_PATH
    t = G.torch()
    c = W.fusion_case(64, 512, seed=19)
    with GatedDeltaFusion(512, 64) as fz:
        fz.set_option(OPT_SPLITS, splits)
        fz.set_option(OPT_PATH, tile)
        dv = upload(c)
        out = t.empty((c.tokens, c.d), dtype=t.bfloat16, device="cuda")
        gate = t.empty((c.tokens, c.d), dtype=t.float32, device="cuda")

        def call():
            fz(dv["n"], dv["o"], dv["w_g"], dv["b_g"], dv["w_delta"], out=out, gate=gate)
        call()
        t.cuda.synchronize()
        eager, eager_gate = out.clone(), gate.clone()
        side = t.cuda.Stream()
        side.wait_stream(t.cuda.current_stream())
        with t.cuda.stream(side):
            call()
        t.cuda.current_stream().wait_stream(side)
        t.cuda.synchronize()
        g = t.cuda.CUDAGraph()
        with t.cuda.graph(g):
            call()
        for rep in range(4):
            out.zero_()
            gate.zero_()
            t.cuda.synchronize()
            g.replay()
            t.cuda.synchronize()
            assert t.equal(out, eager), rep
            assert t.equal(gate, eager_gate), rep
            call()                                  # eager work between replays
            t.cuda.synchronize()
    ref, _ = reference(c)
    check(eager.float().cpu().numpy(), ref, False, f"graph splits={splits}")


def packed_layout(c):
    """Expected packed copy, by index mapping only: piece (tile, seg, chunk, wave, s, lane) holds
    weights [channel tile*128 + wave*32 + lane%32][chunk*64 + 32*(lane/32) + 8s .. +7] of segment seg."""
    d = c.d
    segs = [c.w_g[:, 0:d], c.w_g[:, d:2 * d], c.w_g[:, 2 * d:3 * d], c.w_delta]
    tiles, chunks = d // 128, d // 64
    out = np.empty((tiles, 4, chunks, 4, 4, 64, 8), dtype=np.uint16)
    lane = np.arange(64)
    for seg in range(4):
        for w in range(4):
            rows = (np.arange(tiles)[:, None] * 128 + w * 32 + (lane % 32)[None, :])     # [tile][lane]
            for s in range(4):
                cols = (np.arange(chunks)[:, None] * 64 + 32 * (lane // 32)[None, :] + 8 * s)  # [chunk][lane]
                for e in range(8):
                    out[:, seg, :, w, s, :, e] = segs[seg][rows[:, None, :], cols[None, :, :] + e]
    return out.reshape(-1)


@pytest.mark.parametrize("d", [256, 512])
def test_fusion_pack_layout_is_exact(d):
    from paper_2604_26412_amd import GatedDeltaFusion
    t = G.torch()
    c = W.fusion_case(4, d, seed=12)
    with GatedDeltaFusion(d, 4) as fz:
        dv = upload(c)
        packed = fz.pack_weights(dv["w_g"], dv["w_delta"])
        t.cuda.synchronize()
    assert np.array_equal(packed.cpu().view(t.int16).numpy().view(np.uint16), packed_layout(c))


@pytest.mark.parametrize("tokens,d", [(1, 256), (64, 256), (100, 512), (200, 512)])
@pytest.mark.parametrize("splits", [0, 1, 2, 4, 8, 16])
def test_fusion_packed_equals_row_major_bitwise(tokens, d, splits):
    from paper_2604_26412_amd import GatedDeltaFusion, OPT_SPLITS
    t = G.torch()
    c = W.fusion_case(tokens, d, seed=13 + tokens)
    h_ref, _ = reference(c)
    with GatedDeltaFusion(d, max(tokens, 64)) as fz:
        fz.set_option(OPT_SPLITS, splits)
        dv = upload(c)
        packed = fz.pack_weights(dv["w_g"], dv["w_delta"])
        a = fz(dv["n"], dv["o"], dv["w_g"], dv["b_g"], dv["w_delta"])
        g = t.empty((tokens, d), dtype=t.float32, device="cuda")
        b = fz(dv["n"], dv["o"], None, dv["b_g"], None, packed=packed, gate=g)
        t.cuda.synchronize()
    assert t.equal(a.view(t.int16), b.view(t.int16))
    check(b.float().cpu().numpy(), h_ref, False, f"packed tokens={tokens} d={d} splits={splits}")


@pytest.mark.parametrize("name", sorted(W.FUSION_WORKLOADS))
def test_fusion_full_size_sampled_tokens(name):
    # the launch configuration the bench times, checked on 16 sampled tokens (tokens are independent)
    from paper_2604_26412_amd import GatedDeltaFusion
    spec = W.FUSION_WORKLOADS[name]
    _log(f"fusion workload {name}")
    c = W.fusion_case(spec["tokens"], spec["d"], seed=spec["seed"])
    rows = np.unique(np.concatenate([[0, c.tokens - 1],
                                     np.random.default_rng(0).choice(c.tokens, 14, replace=False)]))
    h_ref, g_ref = reference(c, rows)
    t = G.torch()
    with GatedDeltaFusion(c.d, c.tokens) as fz:
        plan = fz.plan(c.tokens)
        dv = upload(c)
        h, g = run(fz, dv, c)
        packed = fz.pack_weights(dv["w_g"], dv["w_delta"])
        hp = fz(dv["n"], dv["o"], None, dv["b_g"], None, packed=packed)
        t.cuda.synchronize()
    check(h[rows], h_ref, False, f"{name} plan={plan}")
    assert np.max(np.abs(g[rows] - g_ref)) <= 5e-3
    assert np.array_equal(hp.float().cpu().numpy(), h)


def test_fusion_rejects_bad_arguments():
    from paper_2604_26412_amd import GatedDeltaFusion, KvshotError
    t = G.torch()
    with GatedDeltaFusion(256, 8) as fz:
        c = W.fusion_case(9, 256, seed=1)
        dv = upload(c)
        with pytest.raises(KvshotError):          # more tokens than the handle was sized for
            fz(dv["n"], dv["o"], dv["w_g"], dv["b_g"], dv["w_delta"])
        out = t.zeros((4, 256), dtype=t.bfloat16, device="cuda")
        args = [dv["o"].data_ptr(), dv["w_g"].data_ptr(), dv["b_g"].data_ptr(), dv["w_delta"].data_ptr(),
                out.data_ptr(), None]
        assert fz._lib.kvshot_gated_delta_fusion(fz._h, 4, None, *args, 0, None) == 1     # n missing
        assert fz._lib.kvshot_gated_delta_fusion(fz._h, 4, dv["n"].data_ptr(), *args, 4, None) == 1  # bad flag
        assert fz._lib.kvshot_gated_delta_fusion(fz._h, 0, dv["n"].data_ptr(), *args, 0, None) == 1  # no tokens
        t.cuda.synchronize()
        assert float(out.float().abs().max()) == 0.0   # nothing was launched
