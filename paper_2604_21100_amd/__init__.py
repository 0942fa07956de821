"""Chunkwise preconditioned delta rule (PDN / PGDN / PKDA) on MI355X.

Thin ctypes binding of libpdn.so, the C ABI declared in include/pdn.h.  The
binding only marshals arguments: it maps torch tensors to device pointers,
allocates outputs and the workspace when the caller does not pass them, and
turns status codes into exceptions.  Every step of the computation runs in
the library's HIP kernels; there is no fallback.  Importing this package
fails loudly if the library has not been built.
"""
from __future__ import annotations

import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libpdn.so")

if not os.path.exists(LIB_PATH):
    raise ImportError(
        f"{LIB_PATH} is missing: build the HIP library first "
        "(python -c 'import __graft_entry__ as g; g.build()' or "
        "python paper_2604_21100_amd/_build.py)")

# The library and torch must share one HIP runtime.  torch ships its own
# libamdhip64 / libhsa-runtime64 under the same sonames as the system ROCm
# that libpdn.so is linked against: if libpdn.so were loaded first, torch
# would later map a second pair, and two HSA runtimes in one process make
# every HIP call undefined.  Loading torch first makes libpdn.so bind to the
# runtime already in the process.
try:
    import torch  # noqa: F401
except ImportError:   # no torch: the C ABI alone, nothing else maps HIP
    torch = None
_lib = ctypes.CDLL(LIB_PATH)


def loaded_hip_runtimes():
    """Paths of the HIP runtime libraries mapped into this process."""
    try:
        with open("/proc/self/maps") as f:
            maps = f.read()
    except OSError:
        return []
    return sorted({ln.split()[-1] for ln in maps.splitlines()
                   if "libamdhip64" in ln and "/" in ln})


if len(loaded_hip_runtimes()) > 1:
    raise ImportError(
        "two HIP runtimes are mapped into this process "
        f"({loaded_hip_runtimes()}); import torch before anything that "
        "loads the system ROCm runtime")

# ---------------------------------------------------------------- enums
PDN_OK, PDN_ERR_NULL, PDN_ERR_SHAPE, PDN_ERR_DTYPE, PDN_ERR_UNSUPPORTED, \
    PDN_ERR_ALIGN, PDN_ERR_ALIAS, PDN_ERR_WORKSPACE, PDN_ERR_VALUE, \
    PDN_ERR_HIP, PDN_ERR_SCRATCH = range(11)
PDN_F32, PDN_BF16 = 0, 1
PDN_GATE_NONE, PDN_GATE_SCALAR, PDN_GATE_CHANNEL = 0, 1, 2
PDN_PRECOND_SQUASH, PDN_PRECOND_IDENTITY, PDN_PRECOND_EXTERNAL, \
    PDN_PRECOND_DIAG_SM, PDN_PRECOND_ATQ = 0, 1, 2, 3, 4

GATES = {"none": PDN_GATE_NONE, "scalar": PDN_GATE_SCALAR,
         "channel": PDN_GATE_CHANNEL}
PRECONDS = {"squash": PDN_PRECOND_SQUASH, "identity": PDN_PRECOND_IDENTITY,
            "external": PDN_PRECOND_EXTERNAL, "diag_sm": PDN_PRECOND_DIAG_SM,
            "atq": PDN_PRECOND_ATQ}
# modes driven by the diagonal key-Gram recurrence (they take beta_p, g_p,
# A0 and return A_T)
GRAM_PRECONDS = ("squash", "diag_sm", "atq")
# write-key normalisation of the squash mode (pdn_knorm)
KNORMS = {"none": 0, "m": 1, "1pm": 2, "beta": 3}

_vp = ctypes.c_void_p


class Problem(ctypes.Structure):
    _fields_ = [("B", ctypes.c_int64), ("T", ctypes.c_int64),
                ("H", ctypes.c_int64), ("dk", ctypes.c_int32),
                ("dv", ctypes.c_int32), ("chunk", ctypes.c_int32),
                ("io", ctypes.c_int), ("gate", ctypes.c_int),
                ("precond", ctypes.c_int), ("x", ctypes.c_float),
                ("scale", ctypes.c_float), ("ridge", ctypes.c_float),
                ("knorm", ctypes.c_int)]


class Inputs(ctypes.Structure):
    _fields_ = [(n, _vp) for n in ("q", "k", "v", "beta", "g", "beta_p",
                                   "g_p", "log_a_scale", "A0", "S0",
                                   "ktilde")]


class FwdOut(ctypes.Structure):
    _fields_ = [("o", _vp), ("S_T", _vp), ("A_T", _vp)]


class BwdOut(ctypes.Structure):
    _fields_ = [(n, _vp) for n in ("dq", "dk", "dv", "dbeta", "dg", "dS0",
                                   "dbeta_p", "dg_p", "dlog_a_scale", "dA0",
                                   "dktilde")]


_lib.pdn_workspace_size.argtypes = [ctypes.POINTER(Problem), ctypes.c_int,
                                    ctypes.POINTER(ctypes.c_size_t)]
_lib.pdn_workspace_size.restype = ctypes.c_int
_lib.pdn_chunk_fwd.argtypes = [ctypes.POINTER(Problem), ctypes.POINTER(Inputs),
                               ctypes.POINTER(FwdOut), _vp, ctypes.c_size_t,
                               _vp]
_lib.pdn_chunk_fwd.restype = ctypes.c_int
_lib.pdn_chunk_fwd_events.argtypes = [
    ctypes.POINTER(Problem), ctypes.POINTER(Inputs), ctypes.POINTER(FwdOut),
    _vp, ctypes.c_size_t, _vp, ctypes.POINTER(_vp), ctypes.c_int]
_lib.pdn_chunk_fwd_events.restype = ctypes.c_int
_lib.pdn_chunk_bwd.argtypes = [ctypes.POINTER(Problem), ctypes.POINTER(Inputs),
                               _vp, _vp, ctypes.POINTER(BwdOut), _vp,
                               ctypes.c_size_t, _vp]
_lib.pdn_chunk_bwd.restype = ctypes.c_int
_lib.pdn_chunk_bwd_events.argtypes = [
    ctypes.POINTER(Problem), ctypes.POINTER(Inputs), _vp, _vp,
    ctypes.POINTER(BwdOut), _vp, ctypes.c_size_t, _vp, ctypes.POINTER(_vp),
    ctypes.c_int]
_lib.pdn_chunk_bwd_events.restype = ctypes.c_int
_lib.pdn_chunk_fwd_train.argtypes = [
    ctypes.POINTER(Problem), ctypes.POINTER(Inputs), ctypes.POINTER(FwdOut),
    _vp, ctypes.c_size_t, _vp, ctypes.POINTER(_vp), ctypes.c_int]
_lib.pdn_chunk_fwd_train.restype = ctypes.c_int
_lib.pdn_chunk_bwd_train.argtypes = [
    ctypes.POINTER(Problem), ctypes.POINTER(Inputs), _vp, _vp,
    ctypes.POINTER(BwdOut), _vp, ctypes.c_size_t, _vp, ctypes.POINTER(_vp),
    ctypes.c_int]
_lib.pdn_chunk_bwd_train.restype = ctypes.c_int
_lib.pdn_chunk_fwd_noalloc.argtypes = [
    ctypes.POINTER(Problem), ctypes.POINTER(Inputs), ctypes.POINTER(FwdOut),
    _vp]
_lib.pdn_chunk_fwd_noalloc.restype = ctypes.c_int
_lib.pdn_noalloc_scratch_bytes.argtypes = []
_lib.pdn_noalloc_scratch_bytes.restype = ctypes.c_size_t
_lib.pdn_status_string.argtypes = [ctypes.c_int]
_lib.pdn_status_string.restype = ctypes.c_char_p
_lib.pdn_abi_version.argtypes = []
_lib.pdn_abi_version.restype = ctypes.c_int
_lib.pdn_scan_segments.argtypes = [ctypes.POINTER(Problem),
                                   ctypes.POINTER(ctypes.c_int)]
_lib.pdn_scan_segments.restype = ctypes.c_int

ABI_VERSION = 5   # PDN_ABI_VERSION: the struct layouts mirrored above
if _lib.pdn_abi_version() != ABI_VERSION:
    raise ImportError(f"{LIB_PATH} implements ABI version "
                      f"{_lib.pdn_abi_version()}, this binding mirrors "
                      f"version {ABI_VERSION}: rebuild the library")

EXPORTED = ("pdn_workspace_size", "pdn_chunk_fwd", "pdn_chunk_fwd_events",
            "pdn_chunk_bwd", "pdn_chunk_bwd_events", "pdn_chunk_fwd_train",
            "pdn_chunk_bwd_train", "pdn_chunk_fwd_noalloc",
            "pdn_noalloc_scratch_bytes", "pdn_status_string",
            "pdn_abi_version", "pdn_scan_segments")
FWD_STAGE_EVENTS = 4   # PDN_FWD_STAGE_EVENTS
BWD_STAGE_EVENTS = 7   # PDN_BWD_STAGE_EVENTS
FWD_STAGES = ("precond", "chunk_prep", "chunk_scan")
BWD_STAGES = ("bwd_precond_recompute", "bwd_chunk_prep", "bwd_state_save_scan",
              "bwd_state_adjoint_scan", "bwd_chunk_grads", "bwd_precond_reverse")


class PdnError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: {pdn_status_string(status)} "
                         f"(status {status})")


def pdn_status_string(status: int) -> str:
    return _lib.pdn_status_string(int(status)).decode()


def pdn_abi_version() -> int:
    return _lib.pdn_abi_version()


def make_problem(B, T, H, dk, dv, *, io="bf16", gate="none",
                 precond="squash", x=1.5, scale=1.0, chunk=64,
                 ridge=1.0, knorm="none") -> Problem:
    return Problem(B, T, H, dk, dv, chunk,
                   PDN_BF16 if io == "bf16" else PDN_F32,
                   GATES[gate] if isinstance(gate, str) else int(gate),
                   PRECONDS[precond] if isinstance(precond, str)
                   else int(precond), x, scale, ridge,
                   KNORMS[knorm] if isinstance(knorm, str) else int(knorm))


def pdn_workspace_size(problem: Problem, with_bwd: bool = False) -> int:
    n = ctypes.c_size_t(0)
    st = _lib.pdn_workspace_size(ctypes.byref(problem), int(with_bwd),
                                 ctypes.byref(n))
    if st != PDN_OK:
        raise PdnError(st, "pdn_workspace_size")
    return n.value


def pdn_scan_segments(problem: Problem) -> int:
    n = ctypes.c_int(0)
    st = _lib.pdn_scan_segments(ctypes.byref(problem), ctypes.byref(n))
    if st != PDN_OK:
        raise PdnError(st, "pdn_scan_segments")
    return n.value


# ------------------------------------------------------- raw pointer calls
def pdn_chunk_fwd_raw(problem: Problem, inputs: Inputs, out: FwdOut, ws: int,
                      ws_bytes: int, stream: int) -> int:
    """Direct call with raw pointers; returns the status code."""
    return _lib.pdn_chunk_fwd(ctypes.byref(problem), ctypes.byref(inputs),
                              ctypes.byref(out), ws, ws_bytes, stream)


def pdn_chunk_fwd_events_raw(problem: Problem, inputs: Inputs, out: FwdOut,
                             ws: int, ws_bytes: int, stream: int,
                             events) -> int:
    """pdn_chunk_fwd_events with raw hipEvent_t handles (ints)."""
    arr = (_vp * len(events))(*events)
    return _lib.pdn_chunk_fwd_events(ctypes.byref(problem),
                                     ctypes.byref(inputs), ctypes.byref(out),
                                     ws, ws_bytes, stream, arr, len(events))


def pdn_chunk_fwd_noalloc_raw(problem: Problem, inputs: Inputs, out: FwdOut,
                              stream: int) -> int:
    """pdn_chunk_fwd_noalloc with raw pointers; returns the status code."""
    return _lib.pdn_chunk_fwd_noalloc(ctypes.byref(problem),
                                      ctypes.byref(inputs), ctypes.byref(out),
                                      stream)


def pdn_noalloc_scratch_bytes() -> int:
    return _lib.pdn_noalloc_scratch_bytes()


def pdn_chunk_bwd_raw(problem: Problem, inputs: Inputs, dO: int, dS_T: int,
                      out: BwdOut, ws: int, ws_bytes: int,
                      stream: int) -> int:
    return _lib.pdn_chunk_bwd(ctypes.byref(problem), ctypes.byref(inputs), dO,
                              dS_T, ctypes.byref(out), ws, ws_bytes, stream)


# ------------------------------------------------------- torch marshalling
def _ptr(t):
    if t is None:
        return None
    if not t.is_contiguous():
        raise ValueError("tensors passed to libpdn must be contiguous")
    return t.data_ptr()


def _io_of(t):
    import torch
    if t.dtype == torch.bfloat16:
        return "bf16"
    if t.dtype == torch.float32:
        return "f32"
    raise TypeError(f"q/k/v must be float32 or bfloat16, got {t.dtype}")


def _stream(stream, device):
    import torch
    s = stream if stream is not None else torch.cuda.current_stream(device)
    return s.cuda_stream


def _inputs(q, k, v, beta, g, beta_p, g_p, log_a_scale, A0, S0, ktilde):
    return Inputs(*[_ptr(t) for t in (q, k, v, beta, g, beta_p, g_p,
                                      log_a_scale, A0, S0, ktilde)])


def pdn_chunk_fwd(q, k, v, beta, *, g=None, gate="none", precond="squash",
                  beta_p=None, g_p=None, log_a_scale=None, A0=None, S0=None,
                  ktilde=None, x=1.5, scale=1.0, chunk=64, ridge=1.0,
                  knorm="none", o=None, S_T=None, A_T=None, want_state=True,
                  workspace=None, stream=None, stage_events=None,
                  train=False):
    """Forward pass on torch device tensors in the ABI layouts of pdn.h.

    Returns (o, S_T, A_T); S_T / A_T are None when not requested.  Outputs and
    the workspace are allocated with torch when not given.  stage_events: 4
    recorded-at-stage-boundary torch.cuda.Event objects (see
    pdn_chunk_fwd_events), or None.  train=True runs pdn_chunk_fwd_train:
    the workspace (then of the backward's size, and required) keeps the
    intermediates pdn_chunk_bwd(..., saved=True) reads."""
    import torch
    B, T, H, dk = q.shape
    dv = v.shape[-1]
    io = _io_of(q)
    prob = make_problem(B, T, H, dk, dv, io=io, gate=gate, precond=precond,
                        x=x, scale=scale, chunk=chunk, ridge=ridge,
                        knorm=knorm)
    dev = q.device
    if o is None:
        o = torch.empty((B, T, H, dv), dtype=q.dtype, device=dev)
    if S_T is None and want_state:
        S_T = torch.empty((B, H, dk, dv), dtype=torch.float32, device=dev)
    if A_T is None and want_state and precond in GRAM_PRECONDS:
        A_T = torch.empty((B, H, dk), dtype=torch.float32, device=dev)
    nbytes = pdn_workspace_size(prob, train)
    if workspace is None:
        if train:
            raise ValueError("train=True needs the caller's workspace (it "
                             "carries the intermediates to the backward)")
        workspace = torch.empty(max(nbytes, 1), dtype=torch.uint8, device=dev)
    inp = _inputs(q, k, v, beta, g, beta_p, g_p, log_a_scale, A0, S0, ktilde)
    out = FwdOut(_ptr(o), _ptr(S_T), _ptr(A_T))
    if train:
        evs = [_event_handle(e) if e is not None else None
               for e in (stage_events or [])]
        arr = (_vp * len(evs))(*evs) if evs else None
        st = _lib.pdn_chunk_fwd_train(
            ctypes.byref(prob), ctypes.byref(inp), ctypes.byref(out),
            _ptr(workspace), workspace.numel(), _stream(stream, dev), arr,
            len(evs))
    elif stage_events is None:
        st = pdn_chunk_fwd_raw(prob, inp, out, _ptr(workspace),
                               workspace.numel(), _stream(stream, dev))
    else:
        st = pdn_chunk_fwd_events_raw(
            prob, inp, out, _ptr(workspace), workspace.numel(),
            _stream(stream, dev),
            [_event_handle(e) if e is not None else None for e in stage_events])
    if st != PDN_OK:
        raise PdnError(st, "pdn_chunk_fwd")
    return o, S_T, A_T


def pdn_chunk_fwd_noalloc(q, k, v, beta, *, o, g=None, gate="none",
                          precond="squash", beta_p=None, g_p=None,
                          log_a_scale=None, A0=None, S0=None, ktilde=None,
                          x=1.5, scale=1.0, chunk=64, ridge=1.0,
                          knorm="none", S_T=None, A_T=None, stream=None):
    """pdn_chunk_fwd through the no-allocation entry point: the caller passes
    every output (o required, S_T / A_T optional) and no workspace; the
    library uses its fixed per-device scratch.  Returns (o, S_T, A_T)."""
    B, T, H, dk = q.shape
    dv = v.shape[-1]
    prob = make_problem(B, T, H, dk, dv, io=_io_of(q), gate=gate,
                        precond=precond, x=x, scale=scale, chunk=chunk,
                        ridge=ridge, knorm=knorm)
    inp = _inputs(q, k, v, beta, g, beta_p, g_p, log_a_scale, A0, S0, ktilde)
    out = FwdOut(_ptr(o), _ptr(S_T), _ptr(A_T))
    st = pdn_chunk_fwd_noalloc_raw(prob, inp, out, _stream(stream, q.device))
    if st != PDN_OK:
        raise PdnError(st, "pdn_chunk_fwd_noalloc")
    return o, S_T, A_T


def _event_handle(ev):
    """Raw hipEvent_t of a torch.cuda.Event (created on first use)."""
    if ev.cuda_event == 0:
        import torch
        ev.record(torch.cuda.current_stream())   # forces creation
    return ev.cuda_event


def pdn_chunk_bwd(q, k, v, beta, dO, *, g=None, gate="none", precond="squash",
                  beta_p=None, g_p=None, log_a_scale=None, A0=None, S0=None,
                  ktilde=None, dS_T=None, x=1.5, scale=1.0, chunk=64,
                  outputs=None, want_optional=True, workspace=None,
                  stream=None, stage_events=None, saved=False):
    """Backward pass on torch device tensors (layouts of pdn.h).

    Returns a dict with dq, dk, dv, dbeta and, when present, dg, dS0 and the
    preconditioner gradients dbeta_p, dg_p, dlog_a_scale, dA0 (squash) or
    dktilde (external).  Outputs and the workspace are allocated with torch
    when not given (``outputs``: dict of preallocated tensors).  saved=True
    runs pdn_chunk_bwd_train on the intermediates a preceding
    pdn_chunk_fwd(..., train=True) left in ``workspace``."""
    import torch
    B, T, H, dk = q.shape
    dv = v.shape[-1]
    io = _io_of(q)
    prob = make_problem(B, T, H, dk, dv, io=io, gate=gate, precond=precond,
                        x=x, scale=scale, chunk=chunk)
    dev = q.device
    f32 = torch.float32
    out = dict(outputs or {})

    def need(name, shape, dtype):
        if name not in out:
            out[name] = torch.empty(shape, dtype=dtype, device=dev)

    need("dq", (B, T, H, dk), q.dtype)
    need("dk", (B, T, H, dk), q.dtype)
    need("dv", (B, T, H, dv), q.dtype)
    need("dbeta", (B, T, H), f32)
    if gate != "none":
        need("dg", tuple(g.shape), f32)
    if want_optional:
        need("dS0", (B, H, dk, dv), f32)
        if precond == "squash":
            need("dbeta_p", (B, T, H), f32)
            need("dg_p", (B, T, H), f32)
            need("dlog_a_scale", (H,), f32)
            need("dA0", (B, H, dk), f32)
        if precond == "external":
            need("dktilde", (B, T, H, dk), q.dtype)
    nbytes = pdn_workspace_size(prob, True)
    if workspace is None:
        if saved:
            raise ValueError("saved=True needs the training forward's workspace")
        workspace = torch.empty(max(nbytes, 1), dtype=torch.uint8, device=dev)
    inp = _inputs(q, k, v, beta, g, beta_p, g_p, log_a_scale, A0, S0, ktilde)
    bo = BwdOut(*[_ptr(out.get(n)) for n, _ in BwdOut._fields_])
    if saved:
        evs = [_event_handle(e) if e is not None else None
               for e in (stage_events or [])]
        arr = (_vp * len(evs))(*evs) if evs else None
        st = _lib.pdn_chunk_bwd_train(
            ctypes.byref(prob), ctypes.byref(inp), _ptr(dO), _ptr(dS_T),
            ctypes.byref(bo), _ptr(workspace), workspace.numel(),
            _stream(stream, dev), arr, len(evs))
    elif stage_events is None:
        st = pdn_chunk_bwd_raw(prob, inp, _ptr(dO), _ptr(dS_T), bo,
                               _ptr(workspace), workspace.numel(),
                               _stream(stream, dev))
    else:
        evs = [_event_handle(e) if e is not None else None
               for e in stage_events]
        arr = (_vp * len(evs))(*evs)
        st = _lib.pdn_chunk_bwd_events(
            ctypes.byref(prob), ctypes.byref(inp), _ptr(dO), _ptr(dS_T),
            ctypes.byref(bo), _ptr(workspace), workspace.numel(),
            _stream(stream, dev), arr, len(evs))
    if st != PDN_OK:
        raise PdnError(st, "pdn_chunk_bwd")
    return out
