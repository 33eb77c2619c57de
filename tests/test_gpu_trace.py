"""Graphs built from rocprofv3 traces through the HIP path: bit-exact with
the oracle on what-if sweeps of a real captured CNN training trace and of
the hand-written toy trace."""
import os

import numpy as np
import pytest

from oracle import oracle as O
from paper_2006_03318_amd import recipes as R
from paper_2006_03318_amd import trace as TR
from tests.gpu_common import assert_equal_arrays, gpu_run, require_gpu, say

pytestmark = pytest.mark.gpu
GOLD = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def _sweep(g, V, seed):
    rng = np.random.default_rng(seed)
    L = int(g.layer.max()) + 1 if g.n else 1
    sweep = [[]]
    for v in range(1, V):
        r = []
        if rng.random() < 0.5:
            r.append(R.AMP())
        if rng.random() < 0.5:
            r.append(R.ScaleLaunch(int(rng.integers(0, 3)), int(rng.integers(1, 4))))
        if rng.random() < 0.3 and L > 0:
            r.append(R.RemoveLayers([int(rng.integers(0, L))]))
        if rng.random() < 0.3:
            r.append(R.ScaleKernels(int(rng.integers(1, 5)), int(rng.integers(1, 5))))
        sweep.append(r)
    return R.compile_sweep(g, sweep)


@pytest.mark.parametrize("name,its", [("rocprof_cnn", [2, 3]), ("rocprof_cnn", [3]),
                                      ("trace_toy", None)])
def test_trace_sweep(name, its):
    require_gpu()
    tg = TR.build_graph(TR.read_rocprof_csv(os.path.join(GOLD, name)), iterations=its)
    g, vs = _sweep(tg.graph, 37, 5)
    say("trace", name, its, "n=%d V=%d" % (g.n, vs.n_variants))
    S, F, M = gpu_run(g, vs)
    oS, oF, oM, _ = O.run(g, vs)
    assert_equal_arrays("makespan", M, oM)
    assert_equal_arrays("finish", F, oF)
    assert_equal_arrays("start", S, oS)
