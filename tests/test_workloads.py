"""Structure of the seeded synthetic workloads (input recipe checks)."""
import numpy as np
import pytest

from paper_2006_03318_amd import workloads as W


@pytest.mark.parametrize("k", [1, 2, 3, 4])
def test_deterministic(k):
    a = W.config(k, variants=8)
    b = W.config(k, variants=8)
    assert a[0].digest() == b[0].digest() and a[1].digest() == b[1].digest()


@pytest.mark.parametrize("k,n_lo,n_hi,V", [(1, 1500, 1700, 8), (2, 30000, 34000, 256),
                                          (3, 30000, 34000, 1024), (4, 240000, 270000, 64)])
def test_sizes(k, n_lo, n_hi, V):
    g, vs = W.config(k)
    assert n_lo <= g.n <= n_hi
    assert vs.n_variants == V
    assert vs.remove_bits.shape == (g.n, (V + 31) // 32)
    assert vs.scale.shape == (g.n_node_cls, V, 2)
    assert (vs.scale[..., 1] >= 1).all() and (vs.scale[..., 0] >= 0).all()


def test_large_sweep_size():
    g, vs = W.config(5, variants=32)
    assert g.n == 1 << 20                       # finish array = 2^20 * 2048 * 8 B = 16 GiB
    assert g.n * 2048 * 8 > 16e9
    assert g.n_edges + int((g.thread_prev >= 0).sum()) > 2_000_000


@pytest.mark.parametrize("k", [1, 2, 3, 4])
def test_chains_and_edges(k):
    g, vs = W.config(k, variants=8)
    # thread order: prev on the same thread, each task followed by at most one
    p = g.thread_prev
    has = p >= 0
    assert (g.thread_id[p[has]] == g.thread_id[has]).all()
    assert np.bincount(p[has], minlength=g.n).max() <= 1
    heads = np.bincount(g.thread_id[~has], minlength=g.n_threads)
    assert heads.max() == 1
    # ids are emission order: structural (class 0) edges go forward
    dst = np.repeat(np.arange(g.n), np.diff(g.in_ptr))
    c0 = g.edge_cls == 0
    assert (g.in_src[c0] < dst[c0]).all()
    assert (p[has] < np.nonzero(has)[0]).all()
    # device and communication tasks carry no gap
    assert (g.gap[~np.isin(g.kind, W.CPU_KINDS)] == 0).all()


@pytest.mark.parametrize("k,hi", [(2, 0.75), (4, 0.5)])
def test_removal_pairs(k, hi):
    """Config 2's upper bound is higher: a fused optimizer removes all but
    one of the 13,296 weight-update kernels (with their launch calls) of
    the 32,768-task iteration in about half of the variants."""
    g, vs = W.config(k)
    bits = W.unpack_bits(vs.remove_bits, vs.n_variants)
    k_ids = np.nonzero(g.launch_of >= 0)[0]
    assert (bits[k_ids] == bits[g.launch_of[k_ids]]).all()   # kernel removed with its launch
    assert not bits[:, 0].any()                               # variant 0 is the identity
    dens = bits[:, 1:].mean()
    assert 0.05 < dens < hi


def test_comm_batches():
    g, vs = W.config(3)
    assert len(vs.batches) == 4
    for v0, v1, mask in vs.batches:
        assert (vs.edge_on[v0:v1, 0] == np.uint64(mask)).all()
    ar = np.nonzero(g.kind == W.K_COMM)[0]
    assert 40 <= ar.size <= 70
    # the first weight-update kernel waits for every all-reduce
    wu = np.nonzero(g.kind == W.K_WU)[0][0]
    srcs = g.in_src[g.in_ptr[wu]:g.in_ptr[wu + 1]]
    assert set(ar.tolist()) <= set(srcs.tolist())


def test_pack_roundtrip():
    rng = np.random.default_rng(0)
    for V in (1, 5, 31, 32, 33, 64, 100):
        b = rng.random((17, V)) < 0.3
        assert (W.unpack_bits(W.pack_bits(b), V) == b).all()


def test_p3_workload_structure():
    g, vs, pp, prio = W.p3_workload(iters=3, variants=12)
    ch = np.isin(g.thread_id, (W.SEND, W.RECV))
    assert (g.kind[ch] == W.K_COMM).all() and (pp == ch).all()
    assert (g.thread_prev[ch] == -1).all()               # no recorded order on the channels
    prev = g.thread_prev[g.thread_prev >= 0]
    assert not ch[prev].any()
    assert (prio[ch] == -g.layer[ch]).all() and (prio[~ch] == 0).all()
    # every push follows the weight-gradient kernel of its layer, every pull its push
    dst = np.repeat(np.arange(g.n), np.diff(g.in_ptr))
    src = g.in_src
    comm_dst = ch[dst]
    assert (g.kind[src[comm_dst]] != W.K_LAUNCH).all()
    # pulls of iteration i feed the forward kernel of their layer in iteration i+1
    e = ch[src] & ~ch[dst]
    assert e.any()
    assert (g.layer[src[e]] == g.layer[dst[e]]).all()
    assert (g.iteration[dst[e]] == g.iteration[src[e]] + 1).all()
    # slice durations add up to each layer's gradient bytes at 10 Gbit/s
    params, fc = W.vgg19_layer_params()
    push = ch & (g.iteration == 0) & np.isin(np.arange(g.n), dst[ch[dst] & ~ch[src]])
    for l in range(19):
        tot = int(g.dur[push & (g.layer == l)].sum())
        assert abs(tot - 4 * params[l] * 8 // 10) <= int((push & (g.layer == l)).sum())
    assert len(params) == 19 and sum(params) > 140_000_000
    assert vs.n_variants == 12 and len(vs.batches) == 1
