"""Parity at full size: the 1,048,576-task x 2,048-variant transformer sweep
(32 chained iterations) in the launch configuration the benchmark times (one
batch, phase schedule, every variant in one dd_simulate_batch call).  Every
makespan and every finish column is compared exactly with the oracle; the
finish array (16 GiB) stays on the GPU and is compared in chunks of 128
variant columns."""
import time

import numpy as np
import pytest

from oracle import oracle as O
from paper_2006_03318_amd import batch as BT
from paper_2006_03318_amd import binding as B
from paper_2006_03318_amd import workloads as W
from tests.gpu_common import assert_equal_arrays, require_gpu, say

pytestmark = [pytest.mark.gpu, pytest.mark.timeout(1200)]

CHUNK = 128


@pytest.fixture(scope="module")
def config5():
    import torch
    require_gpu()
    g, vs = W.config(5)
    say("full size: config 5 n=%d V=%d" % (g.n, vs.n_variants))
    di = BT.to_device(g, vs)
    res = BT.simulate(di, mode=B.DD_PHASES, want_start=False)
    torch.cuda.synchronize()
    assert len(res) == 1
    v0, v1, fin, _, ms = res[0]
    del di
    yield dict(g=g, vs=vs, fin=fin, ms=ms.cpu().numpy())
    del fin, res
    torch.cuda.empty_cache()


def test_every_makespan_bit_exact(config5):
    g, vs = config5["g"], config5["vs"]
    t0 = time.time()
    _, _, oM, _ = O.run(g, vs, want_start=False, want_finish=False)
    say("oracle: 2048 makespans in %.1f s" % (time.time() - t0))
    assert config5["ms"].shape == (2048,)
    assert_equal_arrays("config 5 makespan", config5["ms"], oM)


def test_every_finish_column_bit_exact(config5):
    g, vs, fin = config5["g"], config5["vs"], config5["fin"]
    V = vs.n_variants
    for c0 in range(0, V, CHUNK):
        c1 = min(V, c0 + CHUNK)
        t0 = time.time()
        got = fin[:, c0:c1].t().contiguous().cpu().numpy()       # [c1-c0][N]
        _, oF, _, _ = O.run(g, vs, variants=range(c0, c1), want_start=False)
        assert_equal_arrays("config 5 finish, variants %d..%d" % (c0, c1 - 1), got, oF)
        say("finish columns %d..%d equal (%.1f s)" % (c0, c1 - 1, time.time() - t0))
        del got, oF
