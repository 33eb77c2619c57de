"""dd_simulate_batch_noalloc (the entry point that allocates nothing, its
working memory in the library's per-GPU scratch array) against
dd_simulate_batch on the same handles: finish, start and makespan bit-exact,
on two calls in a row, the second with a smaller input, and a batch too large
for the scratch array rejected before anything is launched."""
import numpy as np
import pytest

from paper_2006_03318_amd import batch as BT
from paper_2006_03318_amd import binding as B
from paper_2006_03318_amd import workloads as W
from tests.gpu_common import assert_equal_arrays, require_gpu, say

pytestmark = pytest.mark.gpu


def _both(g, vs, want_start):
    """Run every batch through both entry points; returns host arrays."""
    import torch
    di = BT.to_device(g, vs)
    gh = BT.load_graph(di)
    got, want = [], []
    try:
        for (v0, v1, mask, scale, rm, eon) in di.batches:
            Vb = v1 - v0
            sch, _ = B.dd_levelize(gh, mask, B.DD_PHASES)
            var = B.dd_apply_transforms(gh, Vb, di.n_cls, scale, rm, eon)
            try:
                outs = []
                for fn in (B.dd_simulate_batch_noalloc, B.dd_simulate_batch):
                    sent = 1 << 61
                    fin = torch.full((g.n, Vb), sent, dtype=torch.int64, device="cuda")
                    st = (torch.full((g.n, Vb), sent, dtype=torch.int64, device="cuda")
                          if want_start else None)
                    ms = torch.full((Vb,), sent, dtype=torch.int64, device="cuda")
                    fn(gh, sch, var, fin, st, ms)
                    torch.cuda.synchronize()
                    outs.append((fin.cpu().numpy(), None if st is None else st.cpu().numpy(),
                                 ms.cpu().numpy()))
                got.append(outs[0])
                want.append(outs[1])
            finally:
                B.dd_sched_free(sch)
                B.dd_variants_free(var)
    finally:
        B.dd_graph_free(gh)
    return got, want


def _compare(label, got, want):
    for (f0, s0, m0), (f1, s1, m1) in zip(got, want):
        assert_equal_arrays(label + " makespan", m0, m1)
        assert_equal_arrays(label + " finish", f0, f1)
        if s0 is not None:
            assert_equal_arrays(label + " start", s0, s1)


def test_no_alloc_matches_allocating_entry_point_twice():
    require_gpu()
    # first call: the larger input (32,768 tasks x 256 variants, start too)
    g, vs = W.config(2)
    say("no-alloc: call 1, n=%d V=%d" % (g.n, vs.n_variants))
    got, want = _both(g, vs, want_start=True)
    _compare("no-alloc call 1", got, want)
    # second call: a smaller input (the array keeps the first call's contents)
    g, vs = W.config(1, variants=37)
    say("no-alloc: call 2, n=%d V=%d" % (g.n, vs.n_variants))
    got, want = _both(g, vs, want_start=False)
    _compare("no-alloc call 2", got, want)


def test_no_alloc_several_batches_and_widths():
    """The four channel-order batches of the all-reduce workload."""
    require_gpu()
    g, vs = W.config(3, variants=64)
    got, want = _both(g, vs, want_start=True)
    _compare("no-alloc config 3", got, want)


def test_no_alloc_rejects_a_batch_beyond_the_scratch_array():
    import torch
    require_gpu()
    rng = np.random.default_rng(200_000)
    g = W.random_graph_sparse(rng, 300_000, 4, mean_in=0.3, window=500, run_len=100)
    vs = W.random_variants(rng, g, 2048, p_remove=0.1)
    di = BT.to_device(g, vs)
    gh = BT.load_graph(di)
    try:
        (v0, v1, mask, scale, rm, eon), = di.batches
        sch, _ = B.dd_levelize(gh, mask, B.DD_PHASES)
        var = B.dd_apply_transforms(gh, v1 - v0, di.n_cls, scale, rm, eon)
        try:
            fin = torch.empty((g.n, v1 - v0), dtype=torch.int64, device="cuda")
            ms = torch.empty((v1 - v0,), dtype=torch.int64, device="cuda")
            with pytest.raises(B.DDError) as ei:
                B.dd_simulate_batch_noalloc(gh, sch, var, fin, None, ms)
            assert ei.value.code == B.DD_EINVAL
            assert "scratch" in ei.value.msg
        finally:
            B.dd_sched_free(sch)
            B.dd_variants_free(var)
    finally:
        B.dd_graph_free(gh)
