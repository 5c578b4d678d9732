"""ctypes wrapper of libndvm_emu.so (host emulator of device programs; a
scheduler-checking tool used by the CPU tests only)."""
import ctypes
import os

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PATH = os.path.join(ROOT, "paper_2607_03574_amd", "libndvm_emu.so")

_lib = None


def lib():
    global _lib
    if _lib is None:
        _lib = ctypes.CDLL(PATH)
        f = _lib.ndvm_emu_run
        vp, i64 = ctypes.c_void_p, ctypes.c_int64
        f.restype = ctypes.c_int
        f.argtypes = [ctypes.c_char_p, ctypes.c_size_t, ctypes.c_int, ctypes.c_uint32, ctypes.c_uint32, vp, i64,
                      i64, vp, i64, vp, vp, i64, vp]
        _lib.ndvm_emu_error.restype = ctypes.c_char_p
        g = _lib.ndvm_emu_program
        g.restype = ctypes.c_int64
        g.argtypes = [ctypes.c_char_p, ctypes.c_size_t, ctypes.c_int, ctypes.c_uint32, ctypes.c_uint32, vp,
                      ctypes.c_size_t, vp]
    return _lib


STATS = ["n_regs", "n_ckpt_rows", "n_segments", "n_instr", "fwd_ops", "recompute_ops", "rev_ops",
         "ckpt_stored", "n_uops", "slots_used", "n_skips"]


_ARMS = {False: 0, None: 0, "option": 8, "all": 16}


def run(tape: bytes, params, obs, with_grad=True, budget=320, slots=4, save=False, arms=False, skip=True):
    """with_grad: gradient program (loss and grad); save: the save policy
    (values the adjoint rules read are stored, nothing recomputed); arms:
    branch arms laid out behind skip tests, "option" as the BRANCH_SKIP
    option lays them out, "all" every arm however small; skip: then each lane
    skips the arms it does not take (else every arm runs)."""
    params = np.ascontiguousarray(params, dtype=np.float64)
    obs = np.ascontiguousarray(obs, dtype=np.float64)
    L, P = params.shape
    loss = np.empty(L)
    grad = np.empty((L, P)) if with_grad else None
    stats = (ctypes.c_uint64 * 11)()
    mode = ((2 if save else 1) if with_grad else 0) | (0 if skip else 4) | _ARMS[arms]
    rc = lib().ndvm_emu_run(tape, len(tape), mode, budget, slots, params.ctypes.data, L, P,
                            obs.ctypes.data, obs.size, loss.ctypes.data,
                            grad.ctypes.data if grad is not None else None, P, stats)
    if rc != 0:
        raise RuntimeError(f"emulator rc={rc}: {lib().ndvm_emu_error().decode()}")
    return loss, grad, dict(zip(STATS, list(stats)))


def program(tape: bytes, with_grad=True, budget=320, slots=4, save=False, arms=False):
    """The scheduled device program in instruction order: (headers[n_instr],
    words[n_instr, 4 rows, 4]) as uint32 arrays (padding after END included).
    The device layout is chunk-major ([chunk][row][instr][4] words), then the
    header words."""
    mode = ((2 if save else 1) if with_grad else 0) | _ARMS[arms]
    n = lib().ndvm_emu_program(tape, len(tape), mode, budget, slots, None, 0, None)
    assert n >= 0, lib().ndvm_emu_error()
    out = np.empty(n, dtype=np.uint32)
    hdr_off = ctypes.c_uint32(0)
    lib().ndvm_emu_program(tape, len(tape), mode, budget, slots, out.ctypes.data, n,
                           ctypes.byref(hdr_off))
    k = hdr_off.value
    words = out[:k].reshape(-1, 4, 4, 4).transpose(0, 2, 1, 3).reshape(-1, 4, 4)
    headers = out[k:k + words.shape[0]]
    return headers, words
