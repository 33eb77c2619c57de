"""Parity at full size: the 1,048,576-task x 2,048-variant transformer sweep
(32 chained iterations) in the launch configuration the benchmark times (one
batch, phase schedule, every variant in one dd_simulate_batch call).  The
oracle checks a sample of variant columns exactly (finish of every task and
the makespan); properties that hold for every variant are checked on all
2,048 columns."""
import numpy as np
import pytest

from oracle import oracle as O
from paper_2006_03318_amd import batch as BT
from paper_2006_03318_amd import binding as B
from paper_2006_03318_amd import workloads as W
from tests.gpu_common import assert_equal_arrays, require_gpu, say

pytestmark = pytest.mark.gpu

SAMPLE = [0, 1, 2, 7, 8, 15, 16, 1023, 1024, 2046, 2047]


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
    idx = torch.tensor(SAMPLE, device=fin.device)
    cols = fin.index_select(1, idx).cpu().numpy().T          # [len(SAMPLE)][N]
    last = fin.max(dim=0).values.cpu().numpy()               # max finish per variant
    out = dict(g=g, vs=vs, cols=cols, ms=ms.cpu().numpy(), last=last)
    del fin, res, di
    torch.cuda.empty_cache()
    return out


def test_sampled_variants_bit_exact(config5):
    g, vs = config5["g"], config5["vs"]
    _, oF, oM, _ = O.run(g, vs, variants=SAMPLE, want_start=False)
    assert_equal_arrays("config 5 makespan", config5["ms"][SAMPLE], oM)
    assert_equal_arrays("config 5 finish", config5["cols"], oF)


def test_every_variant_properties(config5):
    """Makespan = largest finish of a task kept in the variant; with removal
    (finish of a removed task equals its start) the largest finish overall
    can exceed it only through removed tasks, never fall below it."""
    ms, last = config5["ms"], config5["last"]
    assert ms.shape == (2048,)
    assert (ms > 0).all()
    assert (last >= ms).all()
    # variant 0 is the untransformed graph: identity scales, nothing removed
    _, _, o0, _ = O.run(config5["g"], config5["vs"], variants=[0], want_start=False,
                        want_finish=False)
    assert ms[0] == o0[0]
