"""Thin ctypes binding over libdd.so with the C-ABI's names (include/dd.h).

Arguments are numpy arrays or torch tensors (host or GPU); this module only
checks dtypes/shapes and passes raw pointers.  All computation happens in the
HIP library.  Importing works without a GPU; calling into the library needs
the built libdd.so and fails loudly if it is missing.
"""
from __future__ import annotations

import ctypes
import os
import re
from typing import Optional, Tuple

PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG, "libdd.so")
HEADER = os.path.join(os.path.dirname(PKG), "include", "dd.h")

DD_OK, DD_EINVAL, DD_ECYCLE, DD_ECHAIN, DD_ERANGE, DD_ENOMEM, DD_EHIP, DD_EMISMATCH, \
    DD_ELIMIT = range(9)
DD_LEVELS, DD_PHASES = 0, 1
DD_LOAD_SHARED_THREADS = 1
DD_POLICY_EARLIEST, DD_POLICY_PRIORITY = 0, 1
STATUS_NAMES = ["DD_OK", "DD_EINVAL", "DD_ECYCLE", "DD_ECHAIN", "DD_ERANGE", "DD_ENOMEM",
                "DD_EHIP", "DD_EMISMATCH", "DD_ELIMIT"]


class DDError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__("%s: %s" % (STATUS_NAMES[code] if 0 <= code < len(STATUS_NAMES)
                                     else code, msg))
        self.code = code
        self.msg = msg


_lib = None
_vp = ctypes.c_void_p
_i32, _i64, _u64 = ctypes.c_int32, ctypes.c_int64, ctypes.c_uint64


def declared_symbols():
    """Function names declared in include/dd.h."""
    txt = open(HEADER).read()
    return sorted(set(re.findall(r"\b(dd_[a-z_]+)\s*\(", txt)))


def lib():
    """Load libdd.so (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError("libdd.so not built: run __graft_entry__.build() "
                          "(hipcc --offload-arch=gfx950)")
    try:        # let torch bring up its HIP runtime first so both share one
        import torch  # noqa: F401
    except ImportError:
        pass
    L = ctypes.CDLL(LIB_PATH)
    sig = {
        "dd_graph_load": (_i32, [_i32, _i32, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp,
                                 ctypes.POINTER(_vp)]),
        "dd_graph_load_ex": (_i32, [_i32, _i32, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp,
                                    ctypes.c_uint32, _vp, ctypes.POINTER(_vp)]),
        "dd_levelize": (_i32, [_vp, _u64, _i32, _vp, ctypes.POINTER(_vp), ctypes.POINTER(_i64)]),
        "dd_simulate_policy": (_i32, [_vp, _vp, _i32, _vp, _vp, _vp, _vp, _vp, _vp]),
        "dd_apply_transforms": (_i32, [_vp, _i32, _i32, _vp, _vp, _vp, _vp, ctypes.POINTER(_vp)]),
        "dd_simulate_batch": (_i32, [_vp, _vp, _vp, _vp, _vp, _vp, _vp]),
        "dd_simulate_batch_vs": (_i32, [_vp, _vp, _vp, _vp, _vp, _vp, _i32, _vp]),
        "dd_set_lookback_polls": (None, [_i32]),
        "dd_simulate_plan": (_i32, [_vp, _vp, ctypes.POINTER(_i32)]),
        "dd_release_cache": (_i32, []),
        "dd_simulate_batch_noalloc": (_i32, [_vp, _vp, _vp, _vp, _vp, _vp, _vp]),
        "dd_runtime_breakdown": (_i32, [_vp, _vp, _vp, _vp, _vp, _vp, _vp]),
        "dd_sched_task_steps": (_i32, [_vp, _vp, _vp]),
        "dd_sched_info": (_i32, [_vp, ctypes.POINTER(_i64), ctypes.POINTER(_i64),
                                 ctypes.POINTER(_i64), ctypes.POINTER(_i64)]),
        "dd_graph_free": (None, [_vp]),
        "dd_sched_free": (None, [_vp]),
        "dd_variants_free": (None, [_vp]),
        "dd_status_str": (ctypes.c_char_p, [_i32]),
        "dd_last_error": (ctypes.c_char_p, []),
    }
    for name, (res, args) in sig.items():
        f = getattr(L, name)
        f.restype = res
        f.argtypes = args
    _lib = L
    return L


# ---------------------------------------------------------------------------
def _ptr(x, dtype_name: Optional[str] = None, count: Optional[int] = None):
    """Raw pointer of a numpy array / torch tensor (contiguous) or None."""
    if x is None:
        return None
    if hasattr(x, "data_ptr"):           # torch tensor
        if not x.is_contiguous():
            raise ValueError("tensor must be contiguous")
        if dtype_name is not None:
            tn = str(x.dtype).replace("torch.", "")
            if tn != dtype_name:
                raise TypeError("expected %s, got %s" % (dtype_name, tn))
        if count is not None and x.numel() < count:
            raise ValueError("expected at least %d elements, got %d" % (count, x.numel()))
        return x.data_ptr() if x.numel() else None
    import numpy as np
    if not x.flags["C_CONTIGUOUS"]:
        raise ValueError("array must be C-contiguous")
    if dtype_name is not None and x.dtype != np.dtype(dtype_name):
        raise TypeError("expected %s, got %s" % (dtype_name, x.dtype))
    if count is not None and x.size < count:
        raise ValueError("expected at least %d elements, got %d" % (count, x.size))
    return x.ctypes.data if x.size else None


def _stream(stream):
    if stream is None:
        return None
    if hasattr(stream, "cuda_stream"):
        return stream.cuda_stream
    return int(stream)


def _check(rc: int):
    if rc != DD_OK:
        raise DDError(rc, lib().dd_last_error().decode())


def dd_status_str(code: int) -> str:
    return lib().dd_status_str(code).decode()


def dd_last_error() -> str:
    return lib().dd_last_error().decode()


def dd_graph_load(n, n_threads, in_ptr, in_src, edge_cls, thread_prev, thread_id, dur_ns, gap_ns,
                  node_cls, stream=None):
    out = _vp()
    rc = lib().dd_graph_load(int(n), int(n_threads), _ptr(in_ptr, "int64", n + 1),
                             _ptr(in_src, "int32"), _ptr(edge_cls, "uint8"),
                             _ptr(thread_prev, "int32", n), _ptr(thread_id, "int32", n),
                             _ptr(dur_ns, "int64", n), _ptr(gap_ns, "int64", n),
                             _ptr(node_cls, "uint16", n), _stream(stream), ctypes.byref(out))
    _check(rc)
    return out


def dd_graph_load_ex(n, n_threads, in_ptr, in_src, edge_cls, thread_prev, thread_id, dur_ns,
                     gap_ns, node_cls, flags, stream=None):
    out = _vp()
    rc = lib().dd_graph_load_ex(int(n), int(n_threads), _ptr(in_ptr, "int64", n + 1),
                                _ptr(in_src, "int32"), _ptr(edge_cls, "uint8"),
                                _ptr(thread_prev, "int32", n), _ptr(thread_id, "int32", n),
                                _ptr(dur_ns, "int64", n), _ptr(gap_ns, "int64", n),
                                _ptr(node_cls, "uint16", n), ctypes.c_uint32(int(flags)),
                                _stream(stream), ctypes.byref(out))
    _check(rc)
    return out


def dd_simulate_policy(g, var, policy, pp, prio, d_finish, d_start, d_makespan, stream=None):
    rc = lib().dd_simulate_policy(g, var, int(policy), _ptr(pp, "uint8"), _ptr(prio, "int32"),
                                  _ptr(d_finish, "int64"), _ptr(d_start, "int64"),
                                  _ptr(d_makespan, "int64"), _stream(stream))
    _check(rc)


def dd_levelize(g, active_edge_classes: int, mode: int, stream=None) -> Tuple[object, int]:
    out = _vp()
    steps = _i64(0)
    rc = lib().dd_levelize(g, ctypes.c_uint64(active_edge_classes & (2 ** 64 - 1)), int(mode),
                           _stream(stream), ctypes.byref(out), ctypes.byref(steps))
    _check(rc)
    return out, int(steps.value)


def dd_apply_transforms(g, n_variants, n_cls, scale, remove_bits, edge_on, stream=None):
    out = _vp()
    rc = lib().dd_apply_transforms(g, int(n_variants), int(n_cls), _ptr(scale, "int32"),
                                   _ptr(remove_bits, "uint32"), _ptr(edge_on, "uint64"),
                                   _stream(stream), ctypes.byref(out))
    _check(rc)
    return out


def dd_simulate_batch(g, sched, var, d_finish, d_start, d_makespan, stream=None):
    rc = lib().dd_simulate_batch(g, sched, var, _ptr(d_finish, "int64"), _ptr(d_start, "int64"),
                                 _ptr(d_makespan, "int64"), _stream(stream))
    _check(rc)


def dd_simulate_batch_vs(g, sched, var, d_finish, d_start, d_makespan, variants_per_wg,
                         stream=None):
    rc = lib().dd_simulate_batch_vs(g, sched, var, _ptr(d_finish, "int64"),
                                    _ptr(d_start, "int64"), _ptr(d_makespan, "int64"),
                                    int(variants_per_wg), _stream(stream))
    _check(rc)


def dd_simulate_plan(sched, var) -> int:
    """Launch shape dd_simulate_batch takes: > 0 variants per workgroup of the
    strip kernel, < 0 the few-variant path (one launch per step)."""
    w = _i32()
    _check(lib().dd_simulate_plan(sched, var, ctypes.byref(w)))
    return int(w.value)


def dd_set_lookback_polls(polls: int):
    lib().dd_set_lookback_polls(int(polls))


def dd_runtime_breakdown(g, var, role, d_finish, d_makespan, d_out, stream=None):
    rc = lib().dd_runtime_breakdown(g, var, _ptr(role, "uint8"), _ptr(d_finish, "int64"),
                                    _ptr(d_makespan, "int64"), _ptr(d_out, "int64"),
                                    _stream(stream))
    _check(rc)


def dd_simulate_batch_noalloc(g, sched, var, d_finish, d_start, d_makespan, stream=None):
    rc = lib().dd_simulate_batch_noalloc(g, sched, var, _ptr(d_finish, "int64"),
                                         _ptr(d_start, "int64"), _ptr(d_makespan, "int64"),
                                         _stream(stream))
    _check(rc)


def dd_release_cache():
    _check(lib().dd_release_cache())


def dd_sched_task_steps(sched, out, stream=None):
    _check(lib().dd_sched_task_steps(sched, _ptr(out, "int32"), _stream(stream)))


def dd_sched_info(sched):
    a, b, c, d = _i64(), _i64(), _i64(), _i64()
    _check(lib().dd_sched_info(sched, ctypes.byref(a), ctypes.byref(b), ctypes.byref(c),
                               ctypes.byref(d)))
    return dict(n_steps=a.value, n_segments=b.value, max_step_width=c.value, n_gathers=d.value)


def dd_graph_free(g):
    if g:
        lib().dd_graph_free(g)


def dd_sched_free(s):
    if s:
        lib().dd_sched_free(s)


def dd_variants_free(v):
    if v:
        lib().dd_variants_free(v)
