"""GPU parity of the projected-KV cache builder against the float64 oracle
(Sec. 3.2, linear projection of L_s sampled layers' KV, with and without the
RoPE re-application; App. A, L_s = 3).

Bar, derived from the arithmetic: bf16 products accumulate exactly in float32
(a bf16 x bf16 product has 16 significant bits), the float32 sum over
L_s d_kv = 3072 terms of unit-scale outputs errs by ~1e-5, the float32 RoPE
table by ~1e-7 relative, and the final rounding to bf16 by at most half an ulp
(2^-9 relative).  Elementwise |gpu - ref| <= 2^-8 |ref| + 1e-3, and relative L2
<= 5e-3 (the bf16 bar of the attention path).  Index work is bit-exact: every
destination slot that no listed token maps to keeps its bytes, and no listed
slot keeps the sentinel.
"""
import sys

import numpy as np
import pytest

import oracle
import workloads as W
from tests import _gpu as G

pytestmark = pytest.mark.gpu

SENTINEL = np.uint16(0x7FC1)   # a NaN payload the kernel never writes


def _log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def handle(case, *, dst_num_pages=None, max_tokens=None):
    from paper_2604_26412_amd import KvProjection
    return KvProjection(num_kv_heads=case.num_kv_heads, num_layers=case.layers, page_size=case.page_size,
                        max_pages_per_seq=case.max_pages_per_seq, num_pages=case.num_pages,
                        dst_num_pages=dst_num_pages or case.num_pages,
                        max_tokens=max_tokens or max(case.n_tokens, 1),
                        max_position=case.max_pages_per_seq * case.page_size, rope_theta=case.rope_theta)


class Dev:
    def __init__(self, case, dst_table=None, dst_pages=None):
        t = G.torch()
        self.k = [G.dev_array(x) for x in case.k_src]
        self.v = [G.dev_array(x) for x in case.v_src]
        self.table = G.dev_array(case.page_table)
        self.seq = G.dev_array(case.token_seq)
        self.pos = G.dev_array(case.token_pos)
        self.wk = G.dev_array(case.w_k)
        self.wv = G.dev_array(case.w_v)
        npages = dst_pages or case.num_pages
        shape = (npages, case.num_kv_heads, case.page_size, 128)
        self.kd = G.dev_array(np.full(shape, SENTINEL, np.uint16))
        self.vd = G.dev_array(np.full(shape, SENTINEL, np.uint16))
        self.dst_table_host = case.page_table if dst_table is None else dst_table
        self.dst_table = None if dst_table is None else G.dev_array(dst_table)
        self.t = t

    def host(self, x):
        return x.view(self.t.int16).cpu().numpy().view(np.uint16)


def run(proj, case, dev, *, rope=True, splits=0, path=0):
    proj.set_option(0, splits)
    proj.set_option(1, path)
    proj(dev.k, dev.v, dev.table, dev.seq, dev.pos, dev.wk, dev.wv, dev.kd, dev.vd, dst_page_table=dev.dst_table,
         rope=rope)
    G.torch().cuda.synchronize()
    return dev.host(dev.kd), dev.host(dev.vd)


def assert_close(gpu, ref, what):
    assert np.isfinite(gpu).all(), f"{what}: non-finite output"
    err = np.abs(gpu - ref)
    worst = float((err / (2.0 ** -8 * np.abs(ref) + 1e-3)).max())
    rel = float(np.linalg.norm((gpu - ref).ravel()) / np.linalg.norm(ref.ravel()))
    assert worst <= 1.0 and rel <= 5e-3, f"{what}: elementwise bound exceeded {worst:.2f}x, rel_l2 {rel:.2e}"
    return float(err.max()), rel


def check(case, dev, kd, vd, *, rope, what, sample=None):
    """Compare the listed tokens' slots with the oracle; untouched slots keep the sentinel."""
    idx = np.arange(case.n_tokens) if sample is None else np.asarray(sample)
    seq, pos = case.token_seq[idx], case.token_pos[idx]
    K, V = oracle.project_kv(case.k_src, case.v_src, case.page_table, seq, pos, case.w_k, case.w_v,
                             page_size=case.page_size, theta=case.rope_theta, rope_keys=rope)
    table = dev.dst_table_host
    P = case.page_size
    pid = table[seq, pos // P]
    gk = oracle.decode(kd[pid, :, pos % P, :], "bf16")
    gv = oracle.decode(vd[pid, :, pos % P, :], "bf16")
    mk = assert_close(gk, K, what + " K")
    mv = assert_close(gv, V, what + " V")
    # bit-exact index work over the whole pool: written exactly where a listed token maps
    written = np.zeros(kd.shape[:1] + kd.shape[2:3], bool)
    written[table[case.token_seq, case.token_pos // P], case.token_pos % P] = True
    for pool in (kd, vd):
        untouched = pool.transpose(0, 2, 1, 3)[~written]
        assert np.all(untouched == SENTINEL), f"{what}: a slot no token maps to was written"
        touched = pool.transpose(0, 2, 1, 3)[written]
        assert not np.any(touched == SENTINEL), f"{what}: a listed slot was not written"
    _log(f"{what}: K max_abs {mk[0]:.2e} rel {mk[1]:.2e}  V max_abs {mv[0]:.2e} rel {mv[1]:.2e}")


@pytest.mark.parametrize("rope", [True, False])
@pytest.mark.parametrize("path,splits", [(0, 0), (1, 0), (1, 1), (1, 2), (1, 5), (1, 16), (2, 0)])
def test_prefill_small_batch_matches_oracle(path, splits, rope):
    c = W.kvproj_case(batch=3, ctx_lens=[300, 45, 17], new_tokens=[300, 45, 17], seed=11)
    dev = Dev(c)
    with handle(c) as proj:
        kd, vd = run(proj, c, dev, rope=rope, splits=splits, path=path)
        plan = proj.plan(c.n_tokens)
    assert plan["path"] == (path or 2), plan     # 362 tokens: the tiled kernel would split, so auto is direct
    check(c, dev, kd, vd, rope=rope, what=f"prefill path={path} splits={splits} (plan {plan}) rope={rope}")


@pytest.mark.parametrize("path", [0, 1])
def test_verified_tokens_of_a_ragged_batch(path):
    c = W.kvproj_case(batch=4, ctx_lens=[1000, 64, 513, 7], new_tokens=[4, 1, 8, 7], seed=12)
    dev = Dev(c)
    with handle(c) as proj:
        kd, vd = run(proj, c, dev, path=path)
        plan = proj.plan(c.n_tokens)
    check(c, dev, kd, vd, rope=True, what=f"verify ragged (plan {plan})")


@pytest.mark.parametrize("counts", [[1], [40, 60], [100, 100], [64, 223], [240, 240], [7] * 64])
def test_direct_path_tile_heights(counts):
    # token counts whose direct plans take 16-, 32-, 48- and 64-token tiles (256 CUs), the last tile
    # ragged; [7] * 64 is one verification of 64 sequences at 7 accepted tokens each
    B = len(counts)
    c = W.kvproj_case(batch=B, ctx_lens=[max(n, 1) + 37 * b for b, n in enumerate(counts)], new_tokens=counts,
                      seed=30 + len(counts) + sum(counts))
    dev = Dev(c)
    with handle(c) as proj:
        kd, vd = run(proj, c, dev, path=0)
        plan = proj.plan(c.n_tokens)
    assert plan["path"] == 2 and plan["splits"] == 1, plan
    check(c, dev, kd, vd, rope=True, what=f"direct {c.n_tokens} tokens (plan {plan})")


def test_direct_path_forced_on_a_large_call_sampled():
    # 5000 tokens on the direct kernel: several workgroups per CU
    c = W.kvproj_case(batch=2, ctx_lens=[3000, 2600], new_tokens=[3000, 2000], seed=21)
    dev = Dev(c)
    with handle(c) as proj:
        kd, vd = run(proj, c, dev, path=2)
        plan = proj.plan(c.n_tokens)
    assert plan["path"] == 2 and plan["workgroups"] > 256, plan
    rng = np.random.default_rng(21)
    sample = np.concatenate([np.arange(200), rng.choice(c.n_tokens, 400, replace=False), [c.n_tokens - 1]])
    check(c, dev, kd, vd, rope=True, what=f"direct forced, 5000 tokens (plan {plan})", sample=sample)


@pytest.mark.parametrize("hkv,layers", [(1, 3), (2, 1), (3, 2), (8, 4), (16, 1), (5, 3), (1, 1)])
@pytest.mark.parametrize("path,splits", [(2, 0), (1, 0), (1, 1)])
def test_head_counts_and_layer_counts(hkv, layers, path, splits):
    c = W.kvproj_case(batch=2, ctx_lens=[130, 300], new_tokens=[130, 40], num_kv_heads=hkv, layers=layers,
                      seed=13 + hkv + 10 * layers)
    dev = Dev(c)
    with handle(c) as proj:
        kd, vd = run(proj, c, dev, splits=splits, path=path)
    check(c, dev, kd, vd, rope=True, what=f"Hkv={hkv} L={layers} path={path} splits={splits}")


def test_larger_pages_and_a_separate_destination_table():
    c = W.kvproj_case(batch=3, ctx_lens=[700, 64, 129], new_tokens=[700, 10, 129], page_size=64, seed=14)
    npages = c.num_pages + 9
    perm = np.random.default_rng(14).permutation(npages).astype(np.int32)
    dst = np.full_like(c.page_table, -1)
    used = 0
    for b in range(3):
        n = -(-int(c.ctx_lens[b]) // 64)
        dst[b, :n] = perm[used:used + n]
        used += n
    dev = Dev(c, dst_table=dst, dst_pages=npages)
    with handle(c, dst_num_pages=npages) as proj:
        kd, vd = run(proj, c, dev)
    check(c, dev, kd, vd, rope=True, what="P=64, own destination table")


def test_prefill_of_many_tiles_sampled():
    # 33,000 tokens: 130 token tiles x 4 channel tiles x 2 tensors, no split; oracle on a sample
    c = W.kvproj_case(batch=2, ctx_lens=[20000, 13000], new_tokens=[20000, 13000], seed=15)
    dev = Dev(c)
    with handle(c) as proj:
        assert proj.plan(c.n_tokens)["splits"] == 1
        kd, vd = run(proj, c, dev)
    rng = np.random.default_rng(15)
    sample = np.concatenate([np.arange(300), rng.choice(c.n_tokens, 500, replace=False), [c.n_tokens - 1]])
    check(c, dev, kd, vd, rope=True, what="33k tokens (sampled)", sample=sample)


@pytest.mark.parametrize("path", [1, 2])
def test_repeated_calls_are_bitwise_identical(path):
    c = W.kvproj_case(batch=2, ctx_lens=[600, 90], new_tokens=[8, 90], seed=16)
    dev = Dev(c)
    with handle(c) as proj:
        a = run(proj, c, dev, path=path)
        b = run(proj, c, dev, path=path)
    assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])


@pytest.mark.parametrize("path,splits", [(1, 1), (1, 5), (2, 0)])
def test_hip_graph_replay_matches_eager(path, splits):
    """A captured call replays to the eager result, with eager work and syncs between replays
    (split path: the combine kernel is captured too)."""
    t = G.torch()
    c = W.kvproj_case(batch=2, ctx_lens=[600, 90], new_tokens=[8, 90], seed=18)
    dev = Dev(c)
    with handle(c) as proj:
        proj.set_option(0, splits)
        proj.set_option(1, path)

        def call():
            proj(dev.k, dev.v, dev.table, dev.seq, dev.pos, dev.wk, dev.wv, dev.kd, dev.vd, rope=True)
        call()
        t.cuda.synchronize()
        eager_k, eager_v = dev.kd.clone(), dev.vd.clone()
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
            dev.kd.fill_(0)
            dev.vd.fill_(0)
            t.cuda.synchronize()
            g.replay()
            t.cuda.synchronize()
            # the call writes only the listed tokens' slots: compare those, through the oracle check
            kd, vd = dev.host(dev.kd), dev.host(dev.vd)
            pid = c.page_table[c.token_seq, c.token_pos // c.page_size]
            sl = c.token_pos % c.page_size
            ek, ev = dev.host(eager_k), dev.host(eager_v)
            assert np.array_equal(kd[pid, :, sl, :], ek[pid, :, sl, :]), rep
            assert np.array_equal(vd[pid, :, sl, :], ev[pid, :, sl, :]), rep
            call()                                  # eager work between replays
            t.cuda.synchronize()
    check(c, dev, dev.host(eager_k), dev.host(eager_v), rope=True, what=f"graph path={path} splits={splits}")


def test_validate_reports_the_first_bad_token():
    c = W.kvproj_case(batch=2, ctx_lens=[100, 50], new_tokens=[5, 5], seed=17)
    dev = Dev(c)
    t = G.torch()
    with handle(c) as proj:
        assert proj.validate(dev.table, dev.seq, dev.pos) == (0, -1, 0)

        def bad(seq=None, pos=None, table=None):
            s = G.dev_array(np.asarray(seq if seq is not None else c.token_seq, np.int32))
            p = G.dev_array(np.asarray(pos if pos is not None else c.token_pos, np.int32))
            tb = G.dev_array(np.asarray(table, np.int32)) if table is not None else dev.table
            return proj.validate(tb, s, p)
        seq = c.token_seq.copy()
        seq[3] = 2
        assert bad(seq=seq) == (5, 3, 1)
        pos = c.token_pos.copy()
        pos[7] = -1
        pos[9] = 10_000
        assert bad(pos=pos) == (5, 7, 2)
        table = c.page_table.copy()
        table[1, 45 // 16] = -3          # tokens 5 .. 9 are positions 45 .. 49 of sequence 1 (logical page 2)
        assert bad(table=table) == (5, 5, 3)
        st = proj.validate(dev.table, dev.seq, dev.pos, dst_page_table=G.dev_array(
            np.where(c.page_table >= 0, c.page_table + c.num_pages, -1).astype(np.int32)))
        assert st == (5, 0, 4)
    t.cuda.synchronize()


def test_rejects_bad_arguments_before_queueing():
    import ctypes
    import paper_2604_26412_amd as K
    c = W.kvproj_case(batch=1, ctx_lens=[40], new_tokens=[40], seed=18)
    dev = Dev(c)
    with handle(c) as proj:
        lib, h = proj._lib, proj._h
        L = c.layers
        ks = (ctypes.c_void_p * L)(*[x.data_ptr() for x in dev.k])
        vs = (ctypes.c_void_p * L)(*[x.data_ptr() for x in dev.v])

        def call(n=40, batch=1, flags=1, wk=None, kd=None):
            return lib.kvshot_kv_project(h, n, batch, ks, vs, dev.table.data_ptr(), dev.seq.data_ptr(),
                                         dev.pos.data_ptr(), wk if wk is not None else dev.wk.data_ptr(),
                                         dev.wv.data_ptr(), kd if kd is not None else dev.kd.data_ptr(),
                                         dev.vd.data_ptr(), None, flags, None)
        assert call(n=41) == 1          # above max_tokens
        assert call(n=0) == 1
        assert call(batch=0) == 1
        assert call(flags=2) == 1
        assert call(wk=dev.wk.data_ptr() + 2) == 1      # misaligned
        assert call(kd=0) == 1
        assert lib.kvshot_kvproj_set_option(h, 0, 17) == 1
        assert lib.kvshot_kvproj_set_option(h, 1, 3) == 1
        assert lib.kvshot_kvproj_set_option(h, 9, 0) == 1
        G.torch().cuda.synchronize()
        assert np.all(dev.host(dev.kd) == SENTINEL)
    assert K.KVPROJ_ROPE == 1


def test_projected_cache_feeds_the_draft_attention():
    # a KV-only drafter step: build the projected cache, then attend it (Sec. 3.2)
    c = W.kvproj_case(batch=2, ctx_lens=[200, 77], new_tokens=[200, 77], seed=19)
    dev = Dev(c)
    with handle(c) as proj:
        kd, vd = run(proj, c, dev)
    # the oracle's own projected cache, rounded to bf16 like the cache the kernel writes
    K, V = oracle.project_kv(c.k_src, c.v_src, c.page_table, c.token_seq, c.token_pos, c.w_k, c.w_v,
                             page_size=16, theta=c.rope_theta, rope_keys=True)
    shape = (c.num_pages, 8, 16, 128)
    ok = oracle.scatter_tokens(np.zeros(shape), c.page_table, c.token_seq, c.token_pos, K, 16)
    ov = oracle.scatter_tokens(np.zeros(shape), c.page_table, c.token_seq, c.token_pos, V, 16)
    a = W.make_case(mode="step", batch=2, ctx_lens=[200, 77], n_new=4, dtype="bf16", seed=20)
    a.k_pages, a.v_pages = W.f32_to_bf16_bits(ok.astype(np.float32)), W.f32_to_bf16_bits(ov.astype(np.float32))
    a.page_table = c.page_table
    ref, _ = G.oracle_out(a)
    a.k_pages, a.v_pages = kd, vd
    dc = G.DevCase(a)
    with G.handle_for(a) as att:
        out = G.run(att, dc)
    G.assert_parity(out, ref, "bf16", "attention over the projected cache")
