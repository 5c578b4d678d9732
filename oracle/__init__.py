"""CPU oracle for NDVM -- TEST INFRASTRUCTURE ONLY.

Only the tests, the package smoke check and the benchmark's CPU-baseline leg
may import this package.  The GPU path never calls it.

``run`` evaluates a stack-bytecode program for L parameter vectors with the
plain C interpreter in ``ndvm_oracle.c`` (per-lane realized trace, Wengert
list, reverse sweep; paper Section 3.4 and Appendix C table tab:adjoints).
``run(..., extended=True)`` is the same source evaluated in x87 extended
precision, used to estimate how strongly rounding disturbs a lane's fp64
result.  ``run_ties`` also lists each lane's near-tie branch encounters, and
``run(..., flip=...)`` evaluates a lane with one of them decided the other
way (both are exact results of a realized trace, Section 4 Property 1).
``run(..., perturb=(seed, ulps))`` moves every library transcendental result
by a few ulps, to measure how strongly another math library's last-ulp
differences move a lane's result.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
import threading

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "ndvm_oracle.c")
LIB = os.path.join(HERE, "liboracle.so")
LIB_LD = os.path.join(HERE, "liboracle_ld.so")
_lock = threading.Lock()
_libs = {}


def build(force: bool = True) -> None:
    """Compile the oracle (fp64 and extended-precision copies) in-tree."""
    base = ["gcc", "-O2", "-std=gnu11", "-ffp-contract=off", "-fno-fast-math",
            "-fPIC", "-shared", "-pthread", SRC, "-lm"]
    for out, extra in ((LIB, []), (LIB_LD, ["-DORACLE_LONG_DOUBLE"])):
        if force or not os.path.exists(out) or os.path.getmtime(out) < os.path.getmtime(SRC):
            tmp = out + ".tmp"
            subprocess.check_call(base[:-2] + extra + [SRC, "-o", tmp, "-lm"])
            os.replace(tmp, out)


def _lib(ld: bool):
    with _lock:
        key = "ld" if ld else "d"
        if key not in _libs:
            path = LIB_LD if ld else LIB
            if not os.path.exists(path) or os.path.getmtime(path) < os.path.getmtime(SRC):
                build(force=True)
            lib = ctypes.CDLL(path)
            fn = getattr(lib, "ndvm_oracle_run_ld" if ld else "ndvm_oracle_run")
            fn.restype = ctypes.c_int
            fn.argtypes = [ctypes.c_char_p, ctypes.c_size_t, ctypes.c_void_p, ctypes.c_int64,
                           ctypes.c_int64, ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p,
                           ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p, ctypes.c_void_p,
                           ctypes.c_double, ctypes.c_void_p, ctypes.c_uint64, ctypes.c_int, ctypes.c_int]
            err = getattr(lib, "ndvm_oracle_error_ld" if ld else "ndvm_oracle_error")
            err.restype = ctypes.c_char_p
            _libs[key] = (lib, fn, err)
        return _libs[key]


class OracleError(RuntimeError):
    def __init__(self, code, msg):
        super().__init__(f"oracle error {code}: {msg}")
        self.code = code


def _ptr(a):
    return a.ctypes.data if a is not None else None


MAX_TIES = 8


def run(bytecode: bytes, params, obs, grad: bool = True, threads: int = 0,
        margin: bool = False, extended: bool = False, flip=None, perturb=None):
    """Return (loss[L], grad[L, P] or None, margin[L] or None).

    flip: optional int array [L]; lane l inverts the decision of its
    flip[l]-th IFLT encounter (counted from 0 in walk order; -1: none).
    perturb: optional (seed, ulps); every library transcendental result is
    moved by a pseudo-random whole number of ulps in [-ulps, ulps]."""
    loss, g, m, _ = _run(bytecode, params, obs, grad, threads, margin, extended, flip, None, perturb)
    return loss, g, m


def run_ties(bytecode: bytes, params, obs, tie_tol: float = 1e-9, grad: bool = True,
             threads: int = 0, extended: bool = False):
    """Return (loss, grad, margin, ties): ties[L, 8] lists per lane the IFLT
    encounters whose relative gap |a-b|/max(|a|,|b|) is at most tie_tol,
    closest first, -1 padded."""
    return _run(bytecode, params, obs, grad, threads, True, extended, None, tie_tol, None)


def _run(bytecode, params, obs, grad, threads, margin, extended, flip, tie_tol, perturb):
    _, fn, err = _lib(extended)
    params = np.ascontiguousarray(params, dtype=np.float64)
    if params.ndim == 1:
        params = params[None, :]
    obs = np.ascontiguousarray(obs, dtype=np.float64)
    L, P = params.shape
    loss = np.empty(L)
    g = np.empty((L, P)) if grad else None
    m = np.empty(L) if margin else None
    ties = np.empty((L, MAX_TIES), dtype=np.int64) if tie_tol is not None else None
    if flip is not None:
        flip = np.ascontiguousarray(flip, dtype=np.int64)
        if flip.shape != (L,):
            raise ValueError("flip must have one entry per lane")
    if threads <= 0:
        threads = max(1, min(os.cpu_count() or 1, 16))
    rc = fn(bytecode, len(bytecode), _ptr(params), L, P, _ptr(obs), obs.size,
            _ptr(loss), _ptr(g), P, _ptr(m), _ptr(ties), float(tie_tol or 0.0), _ptr(flip),
            int(perturb[0]) if perturb else 0, int(perturb[1]) if perturb else 0, threads)
    if rc != 0:
        raise OracleError(rc, err().decode(errors="replace"))
    return loss, g, m, ties
