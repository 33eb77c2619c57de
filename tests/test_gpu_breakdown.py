"""Parity of the runtime breakdown (Sec. 6.2, Fig. 6) computed on the GPU
(dd_runtime_breakdown after dd_simulate_batch, through the C-ABI) with the
oracle's breakdown of its own simulation: total, CPU-only, GPU-only and
CPU+GPU parallel time of every variant, bit-exact."""
import numpy as np
import pytest

from oracle import oracle as O
from paper_2006_03318_amd import batch as BT
from paper_2006_03318_amd import binding as B
from paper_2006_03318_amd import workloads as W
from tests.gpu_common import assert_equal_arrays, require_gpu, say

pytestmark = pytest.mark.gpu


def gpu_breakdown(g, vs, role, role_on_device=True):
    import torch
    di = BT.to_device(g, vs)
    res, gh, handles = BT.simulate(di, keep_handles=True)
    out = np.zeros((vs.n_variants, 4), np.int64)
    rl = torch.from_numpy(role).cuda() if role_on_device else np.ascontiguousarray(role)
    try:
        for (v0, v1, fin, _st, ms), (_sch, var) in zip(res, handles):
            d_out = torch.full((v1 - v0, 4), -7, dtype=torch.int64, device=fin.device)
            B.dd_runtime_breakdown(gh, var, rl, fin, ms, d_out)
            torch.cuda.synchronize()
            out[v0:v1] = d_out.cpu().numpy()
    finally:
        for sch, var in handles:
            B.dd_sched_free(sch)
            B.dd_variants_free(var)
        B.dd_graph_free(gh)
    return out


@pytest.mark.parametrize("k", [1, 2, 3, 4])
def test_breakdown_workloads(k):
    require_gpu()
    g, vs = W.config(k)
    role = W.task_roles(g)
    assert (role == 1).any() and (role == 2).any()
    say("breakdown config%d n=%d V=%d" % (k, g.n, vs.n_variants))
    got = gpu_breakdown(g, vs, role, role_on_device=k % 2 == 0)
    want = O.breakdown(g, vs, role)
    assert_equal_arrays("config%d breakdown" % k, got, want)
    assert (got[:, 1] + got[:, 2] + got[:, 3] == got[:, 0]).all()


@pytest.mark.parametrize("seed", range(12))
def test_breakdown_random(seed):
    """Random roles on random graphs: kernels and waiting calls anywhere,
    removal and scales per variant (chunks of 4,096 tasks, ragged ends)."""
    require_gpu()
    rng = np.random.default_rng(190_000 + seed)
    n = int(rng.integers(1, 9000)) if seed % 3 else int(rng.integers(1, 40))
    g = W.random_graph_sparse(rng, n, int(rng.integers(1, 6)), mean_in=0.6, window=200,
                              n_edge_cls=2, run_len=int(rng.integers(1, 30)))
    vs = W.random_variants(rng, g, int(rng.integers(1, 300)), p_remove=0.3)
    role = rng.integers(0, 4, size=g.n).astype(np.uint8)
    say("breakdown random%d n=%d V=%d" % (seed, g.n, vs.n_variants))
    got = gpu_breakdown(g, vs, role)
    want = O.breakdown(g, vs, np.where(role > 2, 0, role).astype(np.uint8))
    assert_equal_arrays("random breakdown", got, want)


@pytest.mark.parametrize("qs", [(1, 2, 4, 8), (1, 3, 5, 7)])
def test_breakdown_long_durations(qs):
    """Durations up to 2^40 (the 64-bit scaled-duration forms), with scales
    that shift only and with scales that need the multiply-high; many
    waiting calls, so the calls' blocks loop."""
    require_gpu()
    rng = np.random.default_rng(191_000 + qs[1])
    g = W.random_graph_sparse(rng, 3000, 4, mean_in=0.5, window=100, n_edge_cls=1, run_len=6)
    g.dur = rng.integers(0, 1 << 40, size=g.n).astype(np.int64)
    assert int(g.dur.max()) >= 1 << 32
    vs = W.random_variants(rng, g, 70, p_remove=0.2, qs=qs)
    role = rng.integers(0, 3, size=g.n).astype(np.uint8)
    assert (role == 2).sum() > 128
    say("breakdown long durations qs=%s" % (qs,))
    got = gpu_breakdown(g, vs, role)
    want = O.breakdown(g, vs, role)
    assert_equal_arrays("long-duration breakdown", got, want)


def test_breakdown_full_size_sample():
    """The 2,048-variant transformer sweep: every variant's breakdown."""
    require_gpu()
    g, vs = W.config(5)
    role = W.task_roles(g)
    got = gpu_breakdown(g, vs, role)
    want = O.breakdown(g, vs, role)
    assert_equal_arrays("config5 breakdown", got, want)


def test_breakdown_rejects_foreign_handles():
    import torch
    require_gpu()
    g1, vs1 = W.config(1)
    g2, vs2 = W.config(1, variants=8)
    d1 = BT.to_device(g1, vs1)
    res, gh, handles = BT.simulate(d1, keep_handles=True)
    d2 = BT.to_device(g2, vs2)
    gh2 = BT.load_graph(d2)
    try:
        fin, ms = res[0][2], res[0][4]
        out = torch.empty((vs1.n_variants, 4), dtype=torch.int64, device="cuda")
        with pytest.raises(B.DDError) as ei:
            B.dd_runtime_breakdown(gh2, handles[0][1], W.task_roles(g1), fin, ms, out)
        assert ei.value.code == B.DD_EMISMATCH
    finally:
        for sch, var in handles:
            B.dd_sched_free(sch)
            B.dd_variants_free(var)
        B.dd_graph_free(gh)
        B.dd_graph_free(gh2)
