"""AddressSanitizer + UBSan builds of host code, run on the CPU:

* the oracle (plain C) on random graphs in both Remove readings, three tie
  rules and one or three worker threads; its outputs must equal those of the
  normal build;
* the C-ABI's host layer (argument checks, error messages per host thread,
  clean-up after a failed device call), linked alone with stubs for the
  device passes and run without a GPU.

Any sanitizer report ends the program with a non-zero status."""
import os
import shutil
import subprocess
import tempfile

import numpy as np
import pytest

from paper_2006_03318_amd import workloads as W

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HERE = os.path.join(ROOT, "tests", "sanitize")
CLANG = "/opt/rocm/lib/llvm/bin/clang"
CLANGXX = "/opt/rocm/lib/llvm/bin/clang++"
HIPCC = "/opt/rocm/bin/hipcc"
SAN_ENV = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0:halt_on_error=1",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")


def _need(tool):
    if not os.path.exists(tool):
        pytest.skip("%s not present" % tool)


@pytest.fixture(scope="module")
def tmpdir_mod():
    d = tempfile.mkdtemp(prefix="dd_san_")
    yield d
    shutil.rmtree(d, ignore_errors=True)


@pytest.fixture(scope="module")
def oracle_asan(tmpdir_mod):
    _need(CLANG)
    exe = os.path.join(tmpdir_mod, "oracle_asan")
    subprocess.check_call([CLANG, "-O1", "-g", "-std=gnu11", "-pthread",
                           "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
                           "-fno-omit-frame-pointer", "-o", exe,
                           os.path.join(ROOT, "oracle", "dd_oracle.c"),
                           os.path.join(HERE, "oracle_driver.c")])
    return exe


def _write_input(path, g, vs):
    K = vs.edge_on.shape[1]
    with open(path, "wb") as f:
        f.write(np.array([g.n, g.n_threads, vs.n_variants, vs.scale.shape[0], K], "<i4").tobytes())
        f.write(np.array([g.n_edges], "<i8").tobytes())
        for a, dt in ((g.in_ptr, "<i8"), (g.in_src, "<i4"), (g.edge_cls, "u1"),
                      (g.thread_prev, "<i4"), (g.thread_id, "<i4"), (g.dur, "<i8"),
                      (g.gap, "<i8"), (g.node_cls, "<u2"), (vs.scale, "<i4"),
                      (vs.remove_bits, "<u4"), (vs.edge_on, "<u8")):
            f.write(np.ascontiguousarray(a, dt).tobytes())


@pytest.mark.parametrize("seed", range(6))
def test_oracle_under_asan_ubsan(oracle_asan, tmpdir_mod, oracle_mod, seed):
    rng = np.random.default_rng(90_000 + seed)
    if seed < 4:
        g = W.random_graph(rng, int(rng.integers(1, 40)), int(rng.integers(1, 5)), p_edge=0.2,
                           n_edge_cls=3, max_dur=1000)
    else:
        g = W.random_graph_sparse(rng, 3000, 70, mean_in=0.5, window=100, n_edge_cls=2)
    vs = W.random_variants(rng, g, int(rng.choice([1, 7, 33, 40])), p_remove=0.3)
    inp = os.path.join(tmpdir_mod, "in%d.bin" % seed)
    out = os.path.join(tmpdir_mod, "out%d.bin" % seed)
    _write_input(inp, g, vs)
    r = subprocess.run([oracle_asan, inp, out], env=SAN_ENV, capture_output=True, text=True,
                       timeout=300)
    assert r.returncode == 0, r.stderr[-4000:]
    raw = open(out, "rb").read()
    n, V = g.n, vs.n_variants
    per = 8 * (2 * V * n + V)
    S0, F0, M0, _ = oracle_mod.run(g, vs)
    for k in range(12):                      # 2 modes x 3 ties x 2 worker counts
        blk = np.frombuffer(raw[k * per:(k + 1) * per], "<i8")
        assert np.array_equal(blk[:V * n].reshape(V, n), S0), k
        assert np.array_equal(blk[V * n:2 * V * n].reshape(V, n), F0), k
        assert np.array_equal(blk[2 * V * n:], M0), k
    steps = np.frombuffer(raw[12 * per:], "<i4")
    lv, ph = oracle_mod.steps(g)
    assert np.array_equal(steps[:n], lv) and np.array_equal(steps[n:], ph)


def test_abi_host_layer_under_asan_ubsan(tmpdir_mod):
    _need(HIPCC)
    _need(CLANGXX)
    csrc = os.path.join(ROOT, "paper_2006_03318_amd", "csrc")
    inc = ["-I", os.path.join(ROOT, "include"), "-I", csrc]
    obj = os.path.join(tmpdir_mod, "dd_api_host.o")
    # host code only (the API layer has no kernels); sanitizers on the host pass
    subprocess.check_call([HIPCC, "--offload-host-only", "-O1", "-g", "-std=c++17",
                           "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
                           "-fno-sanitize-recover=all", "-fno-omit-frame-pointer"] + inc +
                          ["-c", os.path.join(csrc, "dd_api.hip"), "-o", obj],
                          stdout=subprocess.DEVNULL, stderr=subprocess.DEVNULL)
    exe = os.path.join(tmpdir_mod, "abi_host")
    subprocess.check_call([CLANGXX, "-O1", "-g", "-std=c++17", "-fsanitize=address,undefined",
                           "-fno-sanitize-recover=all", "-D__HIP_PLATFORM_AMD__",
                           "-I/opt/rocm/include"] + inc +
                          [os.path.join(HERE, "abi_host_driver.cpp"), obj, "-L/opt/rocm/lib",
                           "-lamdhip64", "-Wl,-rpath,/opt/rocm/lib", "-pthread", "-o", exe])
    supp = os.path.join(tmpdir_mod, "lsan.supp")
    with open(supp, "w") as f:          # allocations the HIP runtime keeps for the process
        f.write("leak:libamdhip64\nleak:libhsa-runtime64\nleak:libhsakmt\nleak:libdrm\n")
    env = dict(SAN_ENV, LSAN_OPTIONS="suppressions=%s" % supp, HIP_VISIBLE_DEVICES="")
    r = subprocess.run([exe], env=env, capture_output=True, text=True, timeout=300)
    assert r.returncode == 0 and "ALL OK" in r.stdout, (r.stdout[-2000:], r.stderr[-4000:])
