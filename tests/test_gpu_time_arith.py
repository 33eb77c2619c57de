"""Parity of the uniform launch path with the oracle (start, finish and
makespan bit-exact), and of the launches that the same kind of input takes
past that path's bounds.

The uniform path (every edge class on in every variant, every scale p/q
with q a power of two, durations and gaps below 2^32) holds its times as
integers in doubles, biased by 2^52.  It is taken when every simulated time
stays below 2^51 (the sum of all scaled durations and gaps, bounded as
dur_sum * max(p/q) + gap_sum, below 2.0e15) and every duration times its
scale numerator stays below 2^53; otherwise the same inputs run on the
int64 path.  The cases below sit on either side of both bounds, at every
launch width, with and without start times, with thread carries (few
threads) and without (more than 64), with removals and with a wide fan-in.
"""
import numpy as np
import pytest

from oracle import oracle as O
from paper_2006_03318_amd import binding as B
from paper_2006_03318_amd import workloads as W
from paper_2006_03318_amd.workloads import VariantSet, pack_bits
from tests.gpu_common import assert_equal_arrays, gpu_run, require_gpu, say
from tests.test_gpu_coverage import _fan_in_graph

pytestmark = pytest.mark.gpu

FP_LIMIT = 2.0e15          # bound on the sum of weights for the double form


def _uniform_variants(rng, g, V, ratios, p_remove=0.2, p_scale=0.7):
    """Variant 0 the baseline; the others scale each task class by a ratio
    drawn from `ratios` (q a power of two) and remove tasks; every edge
    class on."""
    C = g.n_node_cls
    s = np.ones((C, V, 2), np.int32)
    for v in range(1, V):
        for c in range(C):
            if rng.random() < p_scale:
                s[c, v] = ratios[int(rng.integers(0, len(ratios)))]
    bits = rng.random((g.n, V)) < p_remove
    bits[:, 0] = False
    full = (1 << g.n_edge_cls) - 1
    eo = np.full((V, 1), np.uint64(full), np.uint64)
    return VariantSet(V, s, pack_bits(bits), eo, [(0, V, full)])


def _bounds(g, vs):
    """(weight-sum bound, largest duration times largest p), as the library
    bounds them."""
    r = vs.scale[..., 0].astype(np.float64) / vs.scale[..., 1].astype(np.float64)
    dsum = int(g.dur.astype(object).sum())
    gsum = int(g.gap.astype(object).sum())
    return dsum * float(r.max()) + gsum, int(g.dur.max()) * int(vs.scale[..., 0].max())


def _check(g, vs, label, width=0, want_start=True, fp=None):
    bound, dp = _bounds(g, vs)
    if fp is not None:   # the side of the bounds this case is built for
        assert (bound < FP_LIMIT and dp < 2**53) == fp, (bound, dp)
    say("time-arith", label, "n=%d threads=%d V=%d w=%d start=%d bound=%.3g dp=%.3g"
        % (g.n, g.n_threads, vs.n_variants, width, want_start, bound, dp))
    S, F, M = gpu_run(g, vs, variants_per_wg=width, want_start=want_start)
    oS, oF, oM, _ = O.run(g, vs, want_start=want_start)
    assert_equal_arrays(label + " makespan", M, oM)
    assert_equal_arrays(label + " finish", F, oF)
    if want_start:
        assert_equal_arrays(label + " start", S, oS)
    return oM


RATIOS = [(1, 1), (1, 2), (3, 4), (5, 8), (2, 1), (7, 16), (0, 1), (13, 4)]


@pytest.mark.parametrize("width", [0, 1, 2, 4, 8, 16])
@pytest.mark.parametrize("V", [37, 40])
@pytest.mark.parametrize("want_start", [True, False])
def test_uniform_every_width(width, V, want_start):
    """Few threads (thread carries in LDS), runs of tasks, phases of many
    rounds, two edge classes both on."""
    require_gpu()
    rng = np.random.default_rng(90_000 + 10 * width + V + (7 if want_start else 0))
    g = W.random_graph_sparse(rng, 6000, 3, mean_in=0.4, window=300, n_edge_cls=2,
                              n_node_cls=20, run_len=12)
    vs = _uniform_variants(rng, g, V, RATIOS)
    _check(g, vs, "uniform-w%d-V%d" % (width, V), width, want_start, fp=True)


@pytest.mark.parametrize("i", range(2))
def test_uniform_many_threads(i):
    """More than 64 threads: run heads gather their thread predecessor."""
    require_gpu()
    rng = np.random.default_rng(91_000 + i)
    g = W.random_graph_sparse(rng, 20000, 150 + 600 * i, mean_in=0.1, window=2000,
                              n_edge_cls=1, run_len=8)
    vs = _uniform_variants(rng, g, 24 + 9 * i, RATIOS, p_remove=0.25)
    _check(g, vs, "uniform-threads%d" % i, fp=True)


def _long_graph(rng, n=3000, T=4, lo=2**31, hi=2**32 - 1):
    """Durations close to 2^32 on few threads: simulated times reach
    hundreds of trillions."""
    g = W.random_graph_sparse(rng, n, T, mean_in=0.5, window=50, n_edge_cls=1,
                              n_node_cls=4, run_len=20)
    g.dur = rng.integers(lo, hi + 1, size=n).astype(np.int64)
    g.gap = (rng.integers(0, 2**32 - 1, size=n) * (rng.random(n) < 0.3)).astype(np.int64)
    return g


def test_times_near_the_bound():
    """Scales up to 128: times above 2^49, just inside the double form."""
    require_gpu()
    rng = np.random.default_rng(92_000)
    g = _long_graph(rng)
    vs = _uniform_variants(rng, g, 33, [(1, 1), (128, 1), (255, 2), (3, 256), (1, 2)],
                           p_remove=0.1)
    bound, _ = _bounds(g, vs)
    assert bound > 1.0e15
    oM = _check(g, vs, "near-bound", fp=True)
    assert int(oM.max()) > 2**49


def test_times_past_the_bound():
    """The same graph with scales up to 1024: the weight bound passes 2^51
    and the launch runs on int64 (times above 2^51 do occur)."""
    require_gpu()
    rng = np.random.default_rng(92_000)
    g = _long_graph(rng)
    vs = _uniform_variants(rng, g, 33, [(1, 1), (1024, 1), (2047, 2), (3, 256), (1, 2)],
                           p_remove=0.0, p_scale=0.9)
    oM = _check(g, vs, "past-bound", fp=False)
    assert int(oM.max()) > 2**51


@pytest.mark.parametrize("p,fp", [((1 << 20) + 1, True), ((1 << 21) + 1, False)])
def test_duration_times_numerator(p, fp):
    """Scale (2^k + 1) / 2^k on durations close to 2^32: the product d * p
    just below 2^53 (double form, exact floor) and just above (int64)."""
    require_gpu()
    rng = np.random.default_rng(93_000 + p % 7)
    g = _long_graph(rng, n=400, T=3, lo=2**32 - 2**20, hi=2**32 - 1)
    g.dur[7] = 2**32 - 1          # (2^32 - 1) * (2^21 + 1) > 2^53 > (2^32 - 1) * (2^20 + 1)
    q = 1 << ((p - 1).bit_length() - 1)
    vs = _uniform_variants(rng, g, 20, [(1, 1), (p, q), (q + 1, q * 2)], p_remove=0.1)
    _check(g, vs, "d*p-%s" % ("below" if fp else "above"), fp=fp)


def test_wide_fan_in_uniform():
    """A task waiting on 200 others inside a big round, with scaled
    classes and removals, at every width."""
    require_gpu()
    rng = np.random.default_rng(94_000)
    g, x, _ = _fan_in_graph(rng)
    g.node_cls = rng.integers(0, 5, size=g.n).astype(np.uint16)
    g.n_node_cls = 5
    vs = _uniform_variants(rng, g, 26, RATIOS, p_remove=0.25)
    for w in (0, 1, 4, 16):
        _check(g, vs, "fan-in-uniform-w%d" % w, w, fp=True)


def test_levels_mode_uniform():
    require_gpu()
    rng = np.random.default_rng(95_000)
    g = W.random_graph_sparse(rng, 5000, 5, mean_in=0.6, window=100, n_node_cls=6, run_len=4)
    vs = _uniform_variants(rng, g, 18, RATIOS)
    say("time-arith levels")
    S, F, M = gpu_run(g, vs, mode=B.DD_LEVELS)
    oS, oF, oM, _ = O.run(g, vs)
    assert_equal_arrays("levels makespan", M, oM)
    assert_equal_arrays("levels finish", F, oF)
    assert_equal_arrays("levels start", S, oS)
