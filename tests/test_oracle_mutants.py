"""The pins are sensitive: each plausible mistake planted in a temporary copy
of the oracle (never in the oracle itself) makes at least one pin fail."""
import ctypes
import os
import subprocess
import tempfile

import numpy as np
import pytest

from oracle import oracle as O
from tests import test_oracle_pins as P

SRC = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))),
                   "oracle", "dd_oracle.c")

MUTANTS = {
    "gap_not_propagated": ("int64_t rel = s + w->dd[u] + w->gg[u];",
                           "int64_t rel = s + w->dd[u];"),
    "ceil_instead_of_floor": ("return (int64_t)(a / (__int128)q);",
                              "return (int64_t)((a + q - 1) / (__int128)q);"),
    "edge_classes_ignored": ("return (int)((w >> (cls % 64)) & 1u);", "return 1;"),
    "removed_task_in_makespan": ("if (!w->rm[u] && f > ms) ms = f;", "if (f > ms) ms = f;"),
    "removed_keeps_gap": ("w->gg[u] = r ? 0 : g->gap[u];", "w->gg[u] = g->gap[u];"),
    "finish_includes_gap": ("int64_t f = w->S[u] + w->dd[u];",
                            "int64_t f = w->S[u] + w->dd[u] + w->gg[u];"),
    "wrong_variant_bit": ("return (int)((vs->rm_bits[(int64_t)u * W + v / 32] >> (v % 32)) & 1u);",
                          "return (int)((vs->rm_bits[(int64_t)u * W + v / 32] >> ((v + 1) % 32)) & 1u);"),
    "removal_row_stride_slip": ("int32_t W = (vs->n_variants + 31) / 32;",
                                "int32_t W = vs->n_variants / 32 + 1;"),
    "removal_word_index_slip": ("return (int)((vs->rm_bits[(int64_t)u * W + v / 32] >> (v % 32)) & 1u);",
                                "return (int)((vs->rm_bits[(int64_t)u * W + v / 33] >> (v % 32)) & 1u);"),
}


def _build_mutant(name):
    old, new = MUTANTS_ALL[name]
    src = open(SRC).read()
    assert src.count(old) >= 1, name
    src = src.replace(old, new, 1)
    d = tempfile.mkdtemp(prefix="ddo_mut_")
    c = os.path.join(d, "m.c")
    so = os.path.join(d, "libm.so")
    open(c, "w").write(src)
    subprocess.check_call(["gcc", "-O1", "-std=gnu11", "-fPIC", "-shared", "-pthread",
                           "-w", "-o", so, c])
    return so


BREAKDOWN_MUTANTS = {
    "bd_wait_until_finish": ("wait += w->S[u] - reached;", "wait += w->S[u] + w->dd[u] - reached;"),
    "bd_reached_without_gap": ("int64_t reached = p >= 0 ? w->S[p] + w->dd[p] + w->gg[p] : 0;",
                               "int64_t reached = p >= 0 ? w->S[p] + w->dd[p] : 0;"),
    "bd_unscaled_kernel_time": ("if (role[u] == 1) gpu += w->dd[u];",
                                "if (role[u] == 1) gpu += g->dur[u];"),
    "bd_parallel_sign": ("out[3] = ms - out[1] - out[2];", "out[3] = ms - out[1] + out[2];"),
}
POLICY_MUTANTS = {
    "policy_priority_ignored": ("if (policy == 1 && tx == time && pp[x] && pp[best] && prio[x] > prio[best]) {",
                                "if (0) {"),
    "policy_priority_reversed": ("if (policy == 1 && tx == time && pp[x] && pp[best] && prio[x] > prio[best]) {",
                                 "if (policy == 1 && tx == time && pp[x] && pp[best] && prio[x] < prio[best]) {"),
    "policy_time_without_progress": ("int64_t tx = px > w->est[x] ? px : w->est[x];",
                                     "int64_t tx = w->est[x]; (void)px;"),
    "policy_last_of_equals": ("if (tx < time) { time = tx; best = x; bi = i; }",
                              "if (tx <= time) { time = tx; best = x; bi = i; }"),
    "policy_child_release_without_gap": ("int64_t rel = s + w->dd[u] + w->gg[u];\n        w->P[t] = rel;\n        dispatched++;",
                                         "int64_t rel = s + w->dd[u] + w->gg[u];\n        w->P[t] = rel;\n        rel -= w->gg[u];\n        dispatched++;"),
}
MUTANTS_ALL = dict(MUTANTS, **BREAKDOWN_MUTANTS, **POLICY_MUTANTS)


class _Mut:
    def __init__(self, so):
        lib = ctypes.CDLL(so)
        lib.ddo_run.restype = ctypes.c_int
        lib.ddo_run.argtypes = O._load().ddo_run.argtypes
        lib.ddo_breakdown.restype = ctypes.c_int
        lib.ddo_breakdown.argtypes = O._load().ddo_breakdown.argtypes
        lib.ddo_run_policy.restype = ctypes.c_int
        lib.ddo_run_policy.argtypes = O._load().ddo_run_policy.argtypes
        self.lib = lib
        self.OracleError = O.OracleError
        self.ECYCLE = O.ECYCLE

    def run(self, *a, **k):
        saved = O._lib
        O._lib = self.lib
        try:
            return O.run(*a, **k)
        finally:
            O._lib = saved

    def run_policy(self, *a, **k):
        saved = O._lib
        O._lib = self.lib
        try:
            return O.run_policy(*a, **k)
        finally:
            O._lib = saved

    def breakdown(self, *a, **k):
        saved = O._lib
        O._lib = self.lib
        try:
            return O.breakdown(*a, **k)
        finally:
            O._lib = saved


def _pins_fail(m):
    """Run a fast subset of the pins against the mutant; True if any fails."""
    checks = []
    for seed in range(60):
        g, vs = P._random_case(seed)
        try:
            S, F, ms, _ = m.run(g, vs)
        except Exception:
            return True
        for v in range(vs.n_variants):
            bS, bF, bms = P.brute_force(g, vs, v)
            if list(S[v]) != bS or list(F[v]) != bF or ms[v] != bms:
                return True
    for seed in range(40):
        rng = np.random.default_rng(50_000 + seed)
        n = int(rng.integers(2, 9))
        g = P.W.random_graph(rng, n, int(rng.integers(1, 4)), p_edge=float(rng.uniform(0.2, 0.6)),
                             n_edge_cls=int(rng.integers(3, 5)))
        V = int(rng.choice([33, 64, 65, 97]))
        vs = P.W.random_variants(rng, g, V, p_remove=0.3)
        try:
            S, F, ms, _ = m.run(g, vs)
        except Exception:
            return True
        for v in range(V):
            bS, bF, bms = P.brute_force(g, vs, v)
            if list(S[v]) != bS or list(F[v]) != bF or ms[v] != bms:
                return True
    for d, p, q, e in P._floor_rows():
        g = P.H.graph(1, [0], [], [d], [0])
        _, _, ms, _ = m.run(g, P.H.variants(g, scales=[{0: (p, q)}]))
        if ms[0] != e:
            return True
    return False


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_planted_mistake_is_caught(name):
    O.build(force=False)
    m = _Mut(_build_mutant(name))
    assert _pins_fail(m), "pins did not catch mutant " + name


def _breakdown_pins_fail(m):
    from tests import test_oracle_breakdown as BD
    g, role, expect = BD._read_toy()
    if list(m.breakdown(g, P.H.variants(g, V=1), role)[0]) != expect:
        return True
    for seed in range(60):
        rng = np.random.default_rng(170_000 + seed)
        g, role = BD._trace(rng, int(rng.integers(1, 6)), two_cpu=seed % 2 == 1)
        V = 4
        scales = [{}] + [{c: (int(rng.integers(0, 5)), int(rng.choice([1, 2, 3]))) for c in (0, 1)}
                         for _ in range(V - 1)]
        removed = [[]] + [[u for u in range(g.n) if rng.random() < 0.2] for _ in range(V - 1)]
        vs = P.H.variants(g, scales=scales, removed=removed, V=V)
        out = m.breakdown(g, vs, role)
        for v in range(V):
            if list(out[v]) != BD._stepwise(g, vs, v, role):
                return True
    return False


@pytest.mark.parametrize("name", sorted(BREAKDOWN_MUTANTS))
def test_planted_breakdown_mistake_is_caught(name):
    O.build(force=False)
    m = _Mut(_build_mutant(name))
    assert _breakdown_pins_fail(m), "breakdown pins did not catch mutant " + name


def _policy_pins_fail(m):
    from tests import test_oracle_schedule as SC
    try:
        for policy in (0, 1):
            g, pp, prio, exp = SC.load_p3_toy()
            S, _, M = m.run_policy(g, P.H.variants(g, V=1), policy, pp, prio)
            if S[0].tolist() != exp["start%d" % policy] or M[0] != exp["makespan%d" % policy][0]:
                return True
        for seed in range(25):
            g, vs, pp, prio = SC._shared_case(seed)
            for policy in (0, 1):
                S, _, _ = m.run_policy(g, vs, policy, pp, prio)
                for v in range(vs.n_variants):
                    SC._check_valid_run(g, vs, v, S[v], pp, prio, policy)
        for seed in range(10):
            g, vs, pp, prio = SC._chain_case(seed)
            S0, _, M0, _ = O.run(g, vs)
            s1, _, m1 = m.run_policy(g, vs, 1, pp, prio)
            if not (np.array_equal(S0, s1) and np.array_equal(M0, m1)):
                return True
    except AssertionError:
        return True
    return False


@pytest.mark.parametrize("name", sorted(POLICY_MUTANTS))
def test_planted_policy_mistake_is_caught(name):
    O.build(force=False)
    m = _Mut(_build_mutant(name))
    assert _policy_pins_fail(m), "schedule pins did not catch mutant " + name
