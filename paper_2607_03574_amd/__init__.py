"""Python binding of libndvm (the C ABI declared in include/ndvm.h).

Argument marshalling only: every step of the hot path (trace production,
scheduling, forward replay, reverse sweep) runs inside libndvm.so.  Torch is
used for device memory and streams.  If the library has not been built the
import fails: there is no fallback implementation.
"""
from __future__ import annotations

import ctypes
import os
import sys
from typing import Optional, Sequence

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libndvm.so")

OK, E_ARG, E_BYTECODE, E_STRUCT_DIVERGE, E_TAPE, E_NOMEM, E_DEVICE, E_UNSUPPORTED, E_INTERNAL = range(9)
STATUS_NAMES = {0: "NDVM_OK", 1: "NDVM_E_ARG", 2: "NDVM_E_BYTECODE", 3: "NDVM_E_STRUCT_DIVERGE",
                4: "NDVM_E_TAPE", 5: "NDVM_E_NOMEM", 6: "NDVM_E_DEVICE", 7: "NDVM_E_UNSUPPORTED",
                8: "NDVM_E_INTERNAL"}
POLICY_SAVE = 1        # store what the reverse sweep reads, recompute nothing
POLICY_RECOMPUTE = 2   # store segment inputs, recompute inside segments
BRANCH_SKIP = 0x100    # option OR'd into the policy: waves skip branch arms none of their lanes takes
NOALLOC_SCRATCH_BYTES = 64 << 20    # NDVM_NOALLOC_SCRATCH_BYTES

# exported symbols of include/ndvm.h
EXPORTS = ["ndvm_tape_build", "ndvm_tape_upload", "ndvm_tape_upload_many", "ndvm_tape_info_get", "ndvm_workspace_bytes",
           "ndvm_forward", "ndvm_grad", "ndvm_grad_many", "ndvm_workspace_bytes_many",
           "ndvm_tape_free", "ndvm_free", "ndvm_last_error", "ndvm_adam_step", "ndvm_grad_noalloc",
           "ndvm_grad_points", "ndvm_workspace_bytes_points", "ndvm_walk_prepare", "ndvm_walk_measure", "ndvm_walk_workspace_bytes",
           "ndvm_walk_grad", "ndvm_walk_status", "ndvm_walk_free"]

if not os.path.exists(LIB_PATH):
    raise ImportError(f"{LIB_PATH} is missing: build it with paper_2607_03574_amd/build.py "
                      "(or __graft_entry__.build()); there is no fallback path")

_lib = ctypes.CDLL(LIB_PATH)
_vp, _i64, _sz, _int = ctypes.c_void_p, ctypes.c_int64, ctypes.c_size_t, ctypes.c_int


class _Info(ctypes.Structure):
    _fields_ = [("n_params", ctypes.c_uint32), ("n_obs", ctypes.c_uint32), ("n_ops", ctypes.c_uint32),
                ("n_consts", ctypes.c_uint32), ("loss_slot", ctypes.c_uint32),
                ("n_selects", ctypes.c_uint32), ("tape_bytes", ctypes.c_uint64)]


def _sig(name, res, args):
    f = getattr(_lib, name)
    f.restype = res
    f.argtypes = args
    return f


_tape_build = _sig("ndvm_tape_build", _int, [ctypes.c_char_p, _sz, ctypes.POINTER(_vp), ctypes.POINTER(_sz)])
_tape_upload = _sig("ndvm_tape_upload", _int, [ctypes.c_char_p, _sz, _int, _vp, ctypes.POINTER(_vp)])
_tape_upload_many = _sig("ndvm_tape_upload_many", _int, [ctypes.POINTER(ctypes.c_char_p), ctypes.POINTER(_sz), _int,
                                                         _int, _vp, ctypes.POINTER(_vp)])
_tape_info = _sig("ndvm_tape_info_get", _int, [_vp, ctypes.POINTER(_Info)])
_ws_bytes = _sig("ndvm_workspace_bytes", _int, [_vp, _i64, _int, ctypes.POINTER(_sz)])
_ws_bytes_many = _sig("ndvm_workspace_bytes_many", _int, [ctypes.POINTER(_vp), _int, _i64, ctypes.POINTER(_sz)])
_forward = _sig("ndvm_forward", _int, [_vp, _vp, _i64, _i64, _vp, _i64, _vp, _vp, _sz, _vp])
_grad = _sig("ndvm_grad", _int, [_vp, _vp, _i64, _i64, _vp, _i64, _vp, _vp, _i64, _vp, _sz, _vp])
_grad_noalloc = _sig("ndvm_grad_noalloc", _int, [_vp, _vp, _i64, _i64, _vp, _i64, _vp, _vp, _i64, _vp])
_grad_points = _sig("ndvm_grad_points", _int, [_vp, _vp, _i64, _i64, _vp, _i64, _i64, ctypes.c_double, _vp, _vp,
                                                _i64, _vp, _sz, _vp])
_ws_bytes_points = _sig("ndvm_workspace_bytes_points", _int, [_vp, _i64, _i64, ctypes.POINTER(_sz)])
_grad_many = _sig("ndvm_grad_many", _int, [ctypes.POINTER(_vp), _int, _vp, _i64, _i64, _i64, _vp, _i64, _vp,
                                            _vp, _i64, _i64, _vp, _sz, _vp])
_walk_prepare = _sig("ndvm_walk_prepare", _int, [ctypes.POINTER(ctypes.c_char_p), ctypes.POINTER(_sz), _int, _vp,
                                                  ctypes.POINTER(_vp)])
_walk_ws_bytes = _sig("ndvm_walk_workspace_bytes", _int, [_vp, _i64, ctypes.POINTER(_sz)])
_walk_grad = _sig("ndvm_walk_grad", _int, [_vp, _vp, _i64, _i64, _i64, _vp, _i64, _vp, _vp, _i64, _i64, _vp, _sz,
                                            _vp])
_walk_status = _sig("ndvm_walk_status", _int, [_vp, _vp])
_walk_free = _sig("ndvm_walk_free", None, [_vp])


class _WalkInfo(ctypes.Structure):
    _fields_ = [("n_params", ctypes.c_uint32), ("n_obs", ctypes.c_uint32), ("n_nodes", ctypes.c_uint64),
                ("depth", ctypes.c_uint32), ("n_locals", ctypes.c_uint32), ("n_frames", ctypes.c_uint32),
                ("n_loops", ctypes.c_uint32)]


_walk_measure = _sig("ndvm_walk_measure", _int, [ctypes.c_char_p, _sz, ctypes.POINTER(_WalkInfo)])
_tape_free = _sig("ndvm_tape_free", None, [_vp])
_free = _sig("ndvm_free", None, [_vp])
_last_error = _sig("ndvm_last_error", ctypes.c_char_p, [])
_f64 = ctypes.c_double
_adam = _sig("ndvm_adam_step", _int, [_vp, _vp, _vp, _vp, _i64, _i64, _i64, _i64, _i64, _f64, _f64, _f64, _f64,
                                      _vp])


class NdvmError(RuntimeError):
    def __init__(self, status: int, where: str):
        msg = (_last_error() or b"").decode(errors="replace")
        super().__init__(f"{where}: {STATUS_NAMES.get(status, status)}: {msg}")
        self.status = status


def _check(st: int, where: str):
    if st != OK:
        raise NdvmError(st, where)


def last_error() -> str:
    return (_last_error() or b"").decode(errors="replace")


def tape_build(bytecode: bytes) -> bytes:
    """Trace producer: stack bytecode -> serialized lane-invariant tape."""
    out, n = _vp(), _sz()
    _check(_tape_build(bytecode, len(bytecode), ctypes.byref(out), ctypes.byref(n)), "ndvm_tape_build")
    try:
        return ctypes.string_at(out, n.value)
    finally:
        _free(out)


class Tape:
    """Owner of an uploaded tape handle."""

    def __init__(self, handle: int):
        self.handle = handle

    def __del__(self, _free_fn=_tape_free, _finalizing=sys.is_finalizing):
        # at interpreter exit the device runtime may already be gone: leave
        # the handle to the process teardown then
        h, self.handle = getattr(self, "handle", None), None
        if h and not _finalizing():
            _free_fn(h)

    @property
    def info(self) -> dict:
        return tape_info(self)


def _stream_ptr(stream):
    import torch
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    return getattr(stream, "cuda_stream", stream)


def _launch_stream(stream, device):
    """The torch stream a call launches on: the current stream when `stream`
    is None, else `stream` (a torch stream or a raw hipStream_t handle).
    Temporaries a call allocates (workspace, default outputs) are allocated
    and filled under this stream, so the caching allocator orders their reuse
    after the launch and a fill cannot land after the kernel's writes.  Inputs
    the caller produced on another stream are the caller's to order (as for
    any torch kernel launched on a side stream)."""
    import torch
    if stream is None:
        return torch.cuda.current_stream(device)
    if isinstance(stream, torch.cuda.Stream):
        return stream
    return torch.cuda.ExternalStream(int(stream), device=device)


def tape_upload(tape_bytes: bytes, policy: int = POLICY_RECOMPUTE, stream=None) -> Tape:
    h = _vp()
    _check(_tape_upload(tape_bytes, len(tape_bytes), policy, _stream_ptr(stream), ctypes.byref(h)),
           "ndvm_tape_upload")
    return Tape(h.value)


def tape_upload_many(tapes: Sequence[bytes], policy: int = POLICY_RECOMPUTE, stream=None) -> list:
    """tape_upload for a population of tapes (one library call)."""
    n = len(tapes)
    arr = (ctypes.c_char_p * n)(*tapes)
    lens = (_sz * n)(*[len(t) for t in tapes])
    hs = (_vp * n)()
    _check(_tape_upload_many(arr, lens, n, policy, _stream_ptr(stream), hs), "ndvm_tape_upload_many")
    return [Tape(h) for h in hs]


def tape_info(tape: Tape) -> dict:
    info = _Info()
    _check(_tape_info(tape.handle, ctypes.byref(info)), "ndvm_tape_info_get")
    return {k: getattr(info, k) for k, _ in _Info._fields_}


def workspace_bytes(tape: Tape, L: int, with_grad: bool = True) -> int:
    n = _sz()
    _check(_ws_bytes(tape.handle, L, int(with_grad), ctypes.byref(n)), "ndvm_workspace_bytes")
    return n.value


def workspace_bytes_many(tapes: Sequence[Tape], L: int) -> int:
    arr = (_vp * len(tapes))(*[t.handle for t in tapes])
    n = _sz()
    _check(_ws_bytes_many(arr, len(tapes), L, ctypes.byref(n)), "ndvm_workspace_bytes_many")
    return n.value


def _dev_f64(t, name):
    import torch
    if not isinstance(t, torch.Tensor) or t.dtype != torch.float64 or not t.is_cuda:
        raise TypeError(f"{name} must be a float64 CUDA/ROCm tensor")
    return t


def _ld(t, dim=0):
    """Leading dimension of a row-major 2-D view: its row stride, or the row
    length when there is only one row (torch reports any stride for a
    dimension of size one)."""
    return t.stride(dim) if t.shape[dim] > 1 else max(t.shape[dim + 1], 1)


def _workspace(tape_or_bytes, device, workspace):
    import torch
    need = tape_or_bytes
    if workspace is None:
        return torch.empty(max(need, 8), dtype=torch.uint8, device=device), need
    if workspace.numel() * workspace.element_size() < need:
        raise ValueError("workspace too small")
    return workspace, workspace.numel() * workspace.element_size()


def forward(tape: Tape, params, obs, loss=None, workspace=None, stream=None):
    """loss[L] for params[L, P] (rows may be padded: params.stride(0) >= P)."""
    import torch
    _dev_f64(params, "params")
    _dev_f64(obs, "obs")
    if params.dim() != 2 or params.stride(1) != 1 or not obs.is_contiguous():
        raise ValueError("params must be [L, P] with unit inner stride; obs contiguous")
    L = params.shape[0]
    if workspace is not None and loss is not None:     # nothing to allocate: launch directly
        _check(_forward(tape.handle, params.data_ptr(), L, _ld(params), obs.data_ptr(), obs.numel(),
                        loss.data_ptr(), workspace.data_ptr(), workspace.numel() * workspace.element_size(),
                        _stream_ptr(stream)), "ndvm_forward")
        return loss
    need = workspace_bytes(tape, L, False)
    s = _launch_stream(stream, params.device)
    with torch.cuda.stream(s):
        if loss is None:
            loss = torch.empty(L, dtype=torch.float64, device=params.device)
        ws, nbytes = _workspace(need, params.device, workspace)
        _check(_forward(tape.handle, params.data_ptr(), L, _ld(params), obs.data_ptr(), obs.numel(),
                        loss.data_ptr(), ws.data_ptr(), nbytes, s.cuda_stream), "ndvm_forward")
    return loss


def grad(tape: Tape, params, obs, loss=None, grad_out=None, workspace=None, stream=None):
    """(loss[L], grad[L, P]) for params[L, P]."""
    import torch
    _dev_f64(params, "params")
    _dev_f64(obs, "obs")
    if params.dim() != 2 or params.stride(1) != 1 or not obs.is_contiguous():
        raise ValueError("params must be [L, P] with unit inner stride; obs contiguous")
    L, P = params.shape
    if workspace is not None and loss is not None and grad_out is not None:   # launch directly
        _check(_grad(tape.handle, params.data_ptr(), L, _ld(params), obs.data_ptr(), obs.numel(),
                     loss.data_ptr(), grad_out.data_ptr(), _ld(grad_out), workspace.data_ptr(),
                     workspace.numel() * workspace.element_size(), _stream_ptr(stream)), "ndvm_grad")
        return loss, grad_out
    need = workspace_bytes(tape, L, True)
    s = _launch_stream(stream, params.device)
    with torch.cuda.stream(s):
        if loss is None:
            loss = torch.empty(L, dtype=torch.float64, device=params.device)
        if grad_out is None:
            grad_out = torch.empty((L, P), dtype=torch.float64, device=params.device)
        ws, nbytes = _workspace(need, params.device, workspace)
        _check(_grad(tape.handle, params.data_ptr(), L, _ld(params), obs.data_ptr(), obs.numel(),
                     loss.data_ptr(), grad_out.data_ptr(), _ld(grad_out), ws.data_ptr(), nbytes,
                     s.cuda_stream), "ndvm_grad")
    return loss, grad_out


def grad_noalloc(tape: Tape, params, obs, loss, grad_out, stream=None):
    """ndvm_grad_noalloc: (loss[L], grad[L, P]) into the caller's buffers with
    no workspace (the library's static scratch array serves).  The lane count
    must have been prepared with workspace_bytes(tape, L, True)."""
    for name, x in (("params", params), ("obs", obs), ("loss", loss), ("grad", grad_out)):
        _dev_f64(x, name)
    if params.dim() != 2 or params.stride(1) != 1 or not obs.is_contiguous() or grad_out.stride(1) != 1:
        raise ValueError("params and grad must be [L, P] with unit inner stride; obs contiguous")
    L = params.shape[0]
    if loss.numel() < L or grad_out.shape[0] < L:
        raise ValueError("loss and grad must hold L rows")
    _check(_grad_noalloc(tape.handle, params.data_ptr(), L, _ld(params), obs.data_ptr(), obs.numel(),
                         loss.data_ptr(), grad_out.data_ptr(), _ld(grad_out), _stream_ptr(stream)),
           "ndvm_grad_noalloc")
    return loss, grad_out


def workspace_bytes_points(tape: Tape, L: int, n_points: int) -> int:
    n = _sz()
    _check(_ws_bytes_points(tape.handle, L, n_points, ctypes.byref(n)), "ndvm_workspace_bytes_points")
    return n.value


def grad_points(tape: Tape, params, points, scale: float, loss=None, grad_out=None, workspace=None, stream=None):
    """Flattened data axis (ndvm_grad_points): `tape` is the per-point term
    program; points[N, D] holds each data point's observation row; returns
    (loss[L], grad[L, P]) of scale * sum over points of the term."""
    import torch
    _dev_f64(params, "params")
    _dev_f64(points, "points")
    if params.dim() != 2 or params.stride(1) != 1 or points.dim() != 2 or points.stride(1) != 1:
        raise ValueError("params [L, P] and points [N, D] need unit inner stride")
    L, P = params.shape
    N = points.shape[0]
    if workspace is not None and loss is not None and grad_out is not None:   # launch directly
        _check(_grad_points(tape.handle, params.data_ptr(), L, _ld(params), points.data_ptr(), N, _ld(points),
                            float(scale), loss.data_ptr(), grad_out.data_ptr(), _ld(grad_out), workspace.data_ptr(),
                            workspace.numel() * workspace.element_size(), _stream_ptr(stream)), "ndvm_grad_points")
        return loss, grad_out
    need = workspace_bytes_points(tape, L, N)
    s = _launch_stream(stream, params.device)
    with torch.cuda.stream(s):
        if loss is None:
            loss = torch.empty(L, dtype=torch.float64, device=params.device)
        if grad_out is None:
            grad_out = torch.empty((L, P), dtype=torch.float64, device=params.device)
        ws, nbytes = _workspace(need, params.device, workspace)
        _check(_grad_points(tape.handle, params.data_ptr(), L, _ld(params), points.data_ptr(), N,
                            _ld(points), float(scale), loss.data_ptr(), grad_out.data_ptr(), _ld(grad_out),
                            ws.data_ptr(), nbytes, s.cuda_stream), "ndvm_grad_points")
    return loss, grad_out


def grad_many(tapes: Sequence[Tape], params, obs, loss=None, grad_out=None, workspace=None, stream=None):
    """Many programs in one launch: params[n_prog, L, Pmax] -> loss[n_prog, L],
    grad[n_prog, L, Pmax] (entries beyond a program's own P are left as is)."""
    import torch
    _dev_f64(params, "params")
    _dev_f64(obs, "obs")
    if params.dim() != 3 or params.stride(2) != 1 or not obs.is_contiguous():
        raise ValueError("params must be [n_prog, L, Pmax] with unit inner stride")
    n_prog, L, P = params.shape
    if n_prog != len(tapes):
        raise ValueError("one tape per program row")
    need = workspace_bytes_many(tapes, L)
    s = _launch_stream(stream, params.device)
    with torch.cuda.stream(s):
        if loss is None:
            loss = torch.empty((n_prog, L), dtype=torch.float64, device=params.device)
        if grad_out is None:
            grad_out = torch.zeros((n_prog, L, P), dtype=torch.float64, device=params.device)
        ws, nbytes = _workspace(need, params.device, workspace)
        arr = (_vp * n_prog)(*[t.handle for t in tapes])
        ldp, ldg = _ld(params, 1), _ld(grad_out, 1)
        sp = params.stride(0) if n_prog > 1 else L * ldp
        sg = grad_out.stride(0) if n_prog > 1 else L * ldg
        _check(_grad_many(arr, n_prog, params.data_ptr(), L, ldp, sp, obs.data_ptr(),
                          obs.numel(), loss.data_ptr(), grad_out.data_ptr(), ldg,
                          sg, ws.data_ptr(), nbytes, s.cuda_stream), "ndvm_grad_many")
    return loss, grad_out


class WalkSet:
    """Owner of a program set prepared for the device walker."""

    def __init__(self, handle: int, n_prog: int):
        self.handle = handle
        self.n_prog = n_prog

    def __del__(self, _free_fn=_walk_free, _finalizing=sys.is_finalizing):
        h, self.handle = getattr(self, "handle", None), None
        if h and not _finalizing():
            _free_fn(h)


def walk_prepare(bytecodes: Sequence[bytes], stream=None) -> WalkSet:
    """Validate stack-bytecode programs and copy them to the GPU for the
    device walker (ndvm_walk_prepare): no tape, no scheduling."""
    n = len(bytecodes)
    arr = (ctypes.c_char_p * n)(*bytecodes)
    lens = (_sz * n)(*[len(b) for b in bytecodes])
    h = _vp()
    _check(_walk_prepare(arr, lens, n, _stream_ptr(stream), ctypes.byref(h)), "ndvm_walk_prepare")
    return WalkSet(h.value, n)


def walk_measure(bytecode: bytes) -> dict:
    """Host-only validation and structural measurement of one program for the
    device walker (ndvm_walk_measure)."""
    info = _WalkInfo()
    _check(_walk_measure(bytecode, len(bytecode), ctypes.byref(info)), "ndvm_walk_measure")
    return {k: getattr(info, k) for k, _ in _WalkInfo._fields_}


def walk_workspace_bytes(ws: WalkSet, L: int) -> int:
    n = _sz()
    _check(_walk_ws_bytes(ws.handle, int(L), ctypes.byref(n)), "ndvm_walk_workspace_bytes")
    return n.value


def walk_grad(ws: WalkSet, params, obs, loss=None, grad_out=None, workspace=None, stream=None):
    """The device walk of every program of the set: params[n_prog, L, Pmax]
    (or [L, P] for one program) -> loss, grad of the same leading shape
    (entries beyond a program's own P are left as is)."""
    import torch
    _dev_f64(params, "params")
    _dev_f64(obs, "obs")
    single = params.dim() == 2
    p3 = params.unsqueeze(0) if single else params
    if p3.dim() != 3 or p3.stride(2) != 1 or not obs.is_contiguous():
        raise ValueError("params must be [n_prog, L, Pmax] (or [L, P]) with unit inner stride")
    n_prog, L, P = p3.shape
    if n_prog != ws.n_prog:
        raise ValueError("one parameter block per program of the set")
    need = walk_workspace_bytes(ws, L)
    s = _launch_stream(stream, params.device)
    with torch.cuda.stream(s):
        if loss is None:
            loss = torch.empty((n_prog, L) if not single else (L,), dtype=torch.float64, device=params.device)
        if grad_out is None:
            grad_out = torch.zeros(tuple(params.shape), dtype=torch.float64, device=params.device)
        g3 = grad_out.unsqueeze(0) if single else grad_out
        work, nbytes = _workspace(need, params.device, workspace)
        ldp, ldg = _ld(p3, 1), _ld(g3, 1)
        sp = p3.stride(0) if n_prog > 1 else L * ldp
        sg = g3.stride(0) if n_prog > 1 else L * ldg
        _check(_walk_grad(ws.handle, p3.data_ptr(), L, ldp, sp, obs.data_ptr(), obs.numel(), loss.data_ptr(),
                          g3.data_ptr(), ldg, sg, work.data_ptr(), nbytes, s.cuda_stream), "ndvm_walk_grad")
    return loss, grad_out


def walk_status(workspace, stream=None):
    """Synchronise `stream` and raise if a walk that used `workspace` met a
    bound its validation should have excluded (ndvm_walk_status)."""
    _check(_walk_status(workspace.data_ptr(), _stream_ptr(stream)), "ndvm_walk_status")


def adam_step(params, grad_in, m, v, t: int, lr: float, beta1: float = 0.9, beta2: float = 0.999,
              eps: float = 1e-8, stream=None):
    """One Adam step for params[L, P] in place (ndvm_adam_step); m and v are
    [L, P] contiguous moment buffers, zero before step t = 1."""
    for name, x in (("params", params), ("grad", grad_in), ("m", m), ("v", v)):
        _dev_f64(x, name)
    if params.dim() != 2 or params.stride(1) != 1 or grad_in.stride(1) != 1:
        raise ValueError("params and grad must be [L, P] with unit inner stride")
    L, P = params.shape
    if tuple(grad_in.shape) != (L, P) or tuple(m.shape) != (L, P) or tuple(v.shape) != (L, P) \
            or not m.is_contiguous() or not v.is_contiguous():
        raise ValueError("grad, m and v must match params [L, P]; m and v contiguous")
    _check(_adam(params.data_ptr(), grad_in.data_ptr(), m.data_ptr(), v.data_ptr(), L, P, _ld(params),
                 _ld(grad_in), int(t), float(lr), float(beta1), float(beta2), float(eps),
                 _stream_ptr(stream)), "ndvm_adam_step")
    return params
