"""GPU parity of the drafting metrics (Sec. 3.1, Metrics) against the oracle.

Counts are integer work: bit-exact.  The rates are one float64 division of the
same two integers on both sides: bit-exact.  MAT and retention repeat the
oracle's float64 sequence; the compiler may fuse a multiply into the add, so
they are compared to 1e-14 relative.
"""
import json
import os

import numpy as np
import pytest

import oracle
from tests import _gpu as G

pytestmark = pytest.mark.gpu

GOLDEN = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "stepwise_acceptance_rates.json")))


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def run(accepted, K, rstep=None, offset=0):
    import paper_2604_26412_amd as Kmod
    t = G.torch()
    buf = t.from_numpy(np.concatenate([np.zeros(offset, np.int32), np.asarray(accepted, np.int32)])).cuda()
    dev = buf[offset:]
    counts, alpha, mat, ret = Kmod.acceptance_stats(dev, K, retention_step=rstep)
    t.cuda.synchronize()
    return (counts.cpu().numpy(), alpha.cpu().numpy(), float(mat.cpu()[0]),
            float(ret.cpu()[0]) if ret is not None else None)


def check(accepted, K, rstep=None, offset=0):
    c, a, m, r = run(accepted, K, rstep, offset)
    rc = oracle.acceptance_counts(accepted, K)
    ra = oracle.acceptance_rates(rc)
    assert np.array_equal(c, rc)
    assert np.array_equal(a, ra)
    rm = oracle.mat_from_alphas(ra)
    assert abs(m - rm) <= 1e-14 * rm
    if rstep is not None:
        rr = oracle.retention(ra, rstep) if ra[0] > 0 else 0.0
        assert abs(r - rr) <= 1e-14 * max(1.0, abs(rr))
    return c, a, m


@pytest.mark.parametrize("n", [1, 3, 4, 5, 1023, 4096, 100_003])
@pytest.mark.parametrize("offset", [0, 1])
def test_random_lengths_match_the_oracle(n, offset):
    rng = np.random.default_rng(n + offset)
    acc = rng.integers(-3, 11, size=n).astype(np.int32)      # out-of-range values are clamped into [0, 7]
    check(acc, 7, rstep=6, offset=offset)


@pytest.mark.parametrize("K", [1, 2, 8, 64, 255])
def test_step_counts(K):
    rng = np.random.default_rng(K)
    check(rng.integers(0, K + 1, size=20_000).astype(np.int32), K, rstep=K - 1)


def test_empty_input_gives_mat_one():
    c, a, m, r = run(np.zeros(0, np.int32), 7, 6)
    assert c.tolist() == [0] * 8 and a.tolist() == [0.0] * 7 and m == 1.0 and r == 0.0


def test_repeated_calls_restart_from_zero():
    acc = np.full(1000, 3, np.int32)
    for _ in range(3):
        c, a, m = check(acc, 7)
        assert c.tolist() == [1000] * 4 + [0] * 4 and m == 4.0


def test_hip_graph_replay_matches_eager():
    """A captured call replays to the eager result (its counts start from zero on every
    replay), with eager work and syncs between replays."""
    import paper_2604_26412_amd as Kmod
    t = G.torch()
    acc = np.random.default_rng(17).integers(0, 8, size=50_000).astype(np.int32)
    dev = t.from_numpy(acc).cuda()
    eager = [x.clone() for x in Kmod.acceptance_stats(dev, 7, retention_step=3)]
    t.cuda.synchronize()
    side = t.cuda.Stream()
    side.wait_stream(t.cuda.current_stream())
    with t.cuda.stream(side):
        Kmod.acceptance_stats(dev, 7, retention_step=3)
    t.cuda.current_stream().wait_stream(side)
    t.cuda.synchronize()
    g = t.cuda.CUDAGraph()
    with t.cuda.graph(g):
        outs = Kmod.acceptance_stats(dev, 7, retention_step=3)
    for rep in range(4):
        for x in outs:
            x.zero_()
        t.cuda.synchronize()
        g.replay()
        t.cuda.synchronize()
        for x, e in zip(outs, eager):
            assert t.equal(x, e), rep
        Kmod.acceptance_stats(dev, 7, retention_step=3)   # eager work between replays
        t.cuda.synchronize()
    assert np.array_equal(eager[0].cpu().numpy(), oracle.acceptance_counts(acc, 7))


@pytest.mark.parametrize("method", ["Proj + RoPE fix", "Gated KV (ckpt)"])
def test_ten_million_verifications_of_a_printed_row(method):
    row = [r for r in GOLDEN["rows"] if r["method"] == method][0]
    alpha = np.asarray(row["alpha"])
    rng = np.random.default_rng(5)
    n = 10_000_000
    acc = np.zeros(n, np.int32)
    alive = np.ones(n, bool)
    for k, ak in enumerate(alpha):            # step k accepted with probability alpha_k while all earlier were
        alive &= rng.random(n) < ak
        acc += alive
    c, a, m = check(acc, 7, rstep=6)
    assert np.all(np.abs(a - alpha) < 0.005)
    assert abs(m - row["mat"]) < 0.01
