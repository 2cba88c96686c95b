"""GPU checks of the two measurement probes the bench times beside its rooflines.

The streaming-read probe must read every 16-byte word of its buffer exactly once: each lane
folds what it reads with xor and each workgroup stores its fold, so the xor of all stored words
equals the xor of the buffer's words, for any grid.  The matrix-rate probe runs the same dense
products in every workgroup, so every workgroup stores the same word, run after run.
"""
import numpy as np
import pytest

from tests import _gpu as G

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("words16, workgroups", [(1, 1), (4096, 3), (1 << 20, 2048), ((1 << 20) + 7, 1024)])
def test_stream_read_reads_every_word_once(words16, workgroups):
    import paper_2604_26412_amd as K
    t = G.torch()
    print(f"stream read: {words16} words, {workgroups} workgroups", flush=True)
    rng = np.random.default_rng(words16 + workgroups)
    host = rng.integers(0, 2 ** 32, size=(words16, 4), dtype=np.uint32)
    src = t.from_numpy(host.view(np.int32)).cuda()
    sink = K.stream_read(src, workgroups=workgroups)
    t.cuda.synchronize()
    got = np.bitwise_xor.reduce(sink.cpu().numpy().view(np.uint32).reshape(workgroups, 4), axis=0)
    want = np.bitwise_xor.reduce(host, axis=0)
    assert np.array_equal(got, want)


def test_mfma_rate_probe_runs_the_same_products_everywhere():
    import paper_2604_26412_amd as K
    from paper_2604_26412_amd import KvshotError
    t = G.torch()
    print("mfma rate probe", flush=True)
    wgs = t.cuda.get_device_properties(0).multi_processor_count
    a = K.mfma_rate(64, wgs).clone()
    b = K.mfma_rate(64, wgs).clone()
    t.cuda.synchronize()
    wa = a.cpu().numpy().view(np.uint32).reshape(wgs, 4)
    wb = b.cpu().numpy().view(np.uint32).reshape(wgs, 4)
    assert np.array_equal(wa, wb)
    assert (wa[:, 0] == wa[0, 0]).all() and (wa[:, 1:] == 0).all()
    with pytest.raises(KvshotError):
        K.mfma_rate(0, wgs)
