"""Helpers for the GPU tests: run a workload through the C-ABI and through
the oracle on the same seeded inputs."""
from __future__ import annotations

import sys

import numpy as np
import pytest

from paper_2006_03318_amd import batch as BT
from paper_2006_03318_amd import binding as B


def require_gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.fail("GPU test run without a GPU")
    B.lib()   # raises if libdd.so is missing


def say(*a):
    print(*a, file=sys.stderr, flush=True)


def gpu_run(g, vs, mode=B.DD_PHASES, want_start=True, variants_per_wg=0):
    """All batches of a workload; returns host arrays start[V][N],
    finish[V][N], makespan[V] in variant order."""
    import torch
    di = BT.to_device(g, vs)
    res = BT.simulate(di, mode=mode, want_start=want_start, variants_per_wg=variants_per_wg)
    torch.cuda.synchronize()
    V = vs.n_variants
    fin = np.zeros((V, g.n), np.int64)
    st = np.zeros((V, g.n), np.int64) if want_start else None
    ms = np.zeros(V, np.int64)
    for v0, v1, f, s, m in res:
        fin[v0:v1] = f.cpu().numpy().T
        if want_start:
            st[v0:v1] = s.cpu().numpy().T
        ms[v0:v1] = m.cpu().numpy()
    return st, fin, ms


def assert_equal_arrays(name, got, want):
    if not np.array_equal(got, want):
        bad = np.argwhere(got != want)
        i = tuple(bad[0])
        raise AssertionError("%s differs at %d places; first %s: got %d want %d"
                             % (name, bad.shape[0], i, int(got[i]), int(want[i])))
