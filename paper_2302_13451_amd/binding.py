"""Thin ctypes binding of libsa.so (include/sa.h) for torch tensors.

Argument marshalling only: every function checks shapes, allocates outputs
with torch when the caller does not pass them, and calls the C entry point of
the same name on the current HIP stream. All the arithmetic runs in the HIP
kernels; if the library is missing, every call raises.
"""

from __future__ import annotations

import ctypes
import os
from typing import Optional, Tuple

import torch

SA_OK = 0
SA_ERR_NULL = 1
SA_ERR_INVALID = 2
SA_ERR_UNSUPPORTED = 3
SA_ERR_HIP = 4

SA_F32 = 0
SA_BF16 = 1
SA_STREAM_MAX_WINDOW = 1024

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "libsa.so")

_lib = None

_vp = ctypes.c_void_p
_i = ctypes.c_int

_SIGNATURES = {
    "sa_forward": [_vp, _vp, _vp, _vp, _vp, _i, _i, _i, _i, _i, _i, _vp, _i, _vp],
    "sa_backward": [_vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _i, _i, _i, _i, _i, _i, _vp,
                    _i, _vp],
    "llsa_forward": [_vp, _vp, _vp, _vp, _vp, _i, _i, _i, _i, _i, _i, _vp, _i, _vp],
    "llsa_paper_forward": [_vp, _vp, _vp, _vp, _vp, _i, _i, _i, _i, _i, _i, _vp, _i, _vp],
    "llsa_paper_backward": [_vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _i, _i, _i, _i, _i, _i,
                            _vp, _i, _vp],
    "llsa_backward": [_vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _i, _i, _i, _i, _i, _i, _vp,
                      _i, _vp],
    "sa_stream_step": [_vp, _vp, _vp, _vp, _vp, _vp, _vp, _i, _vp, _vp, _i, _i, _i, _i, _i, _vp,
                       _i, _vp],
    "llsa_stream_step": [_vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _i, _vp,
                         _vp, _vp, _i, _i, _i, _i, _i, _vp, _i, _vp],
    "sa_copy_reference": [_vp, _vp, ctypes.c_longlong, _i, _vp],
    "sa_last_error": [],
    "sa_abi_version": [],
}


class SAError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__("status %d: %s" % (status, message))
        self.status = status


def library_path() -> str:
    return _LIB_PATH


def load_library():
    """Load libsa.so (built by ``python -m paper_2302_13451_amd.build``)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        raise SAError(-1, "libsa.so not built at %s; run python -m paper_2302_13451_amd.build"
                      % _LIB_PATH)
    lib = ctypes.CDLL(_LIB_PATH)
    for name, args in _SIGNATURES.items():
        fn = getattr(lib, name)
        fn.argtypes = args
        fn.restype = ctypes.c_char_p if name == "sa_last_error" else ctypes.c_int
    _lib = lib
    return lib


class _Recorder:
    """Stands in for the loaded library while one binding call runs, and
    records the entry points it calls with their marshalled arguments."""

    def __init__(self, lib):
        self.lib = lib
        self.calls = []

    def __getattr__(self, name):
        fn = getattr(self.lib, name)

        def call(*args):
            self.calls.append((fn, args))
            return fn(*args)
        return call


def prepared(fn, *args, **kwargs):
    """Runs ``fn(*args, **kwargs)`` (a binding call, or a function making
    several) once and returns a function of no arguments that repeats the same
    calls of the C entry points with the same marshalled arguments: no shape
    checks, no allocation, the stream of the first call. For timing loops, in
    which the per-call checks would otherwise cost more host time than a short
    kernel takes. Outputs must be passed in (not allocated by the call), and
    every tensor must stay alive while the function is used."""
    global _lib
    lib = load_library()
    rec = _Recorder(lib)
    _lib = rec
    try:
        fn(*args, **kwargs)
    finally:
        _lib = lib
    calls = [(f, a) for f, a in rec.calls if f is not lib.sa_last_error]

    def run():
        for f, a in calls:
            rc = f(*a)
            if rc != SA_OK:
                _check(rc)
    return run


def _check(rc: int):
    if rc != SA_OK:
        raise SAError(rc, load_library().sa_last_error().decode(errors="replace"))


def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.bfloat16:
        return SA_BF16
    if t.dtype == torch.float32:
        return SA_F32
    raise SAError(SA_ERR_UNSUPPORTED, "tensors must be bfloat16 or float32, got %s" % t.dtype)


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(device, stream) -> ctypes.c_void_p:
    s = stream if stream is not None else torch.cuda.current_stream(device)
    return ctypes.c_void_p(s.cuda_stream)


def _require(t: torch.Tensor, name: str, shape, dtype, device):
    if not t.is_cuda:
        raise SAError(SA_ERR_INVALID, "%s must be a GPU tensor" % name)
    if tuple(t.shape) != tuple(shape):
        raise SAError(SA_ERR_INVALID, "%s has shape %s, expected %s" % (name, tuple(t.shape),
                                                                         tuple(shape)))
    if t.dtype != dtype:
        raise SAError(SA_ERR_INVALID, "%s has dtype %s, expected %s" % (name, t.dtype, dtype))
    if t.device != device:
        raise SAError(SA_ERR_INVALID, "%s is on %s, expected %s" % (name, t.device, device))
    if not t.is_contiguous():
        raise SAError(SA_ERR_INVALID, "%s must be contiguous" % name)


def _lengths(lengths, n, device):
    if lengths is None:
        return None
    _require(lengths, "lengths", (n,), torch.int32, device)
    return lengths


def sa_forward(q, k, v, Lb: int, La: int, lengths=None, out=None, lse=None, *,
               want_lse: bool = True, stream=None) -> Tuple[torch.Tensor, Optional[torch.Tensor]]:
    """SA forward. q, k, v: [B][T][H][d] (bf16 or f32); lengths: int32 [B] or
    None. Returns (out, lse) with lse float32 [B][H][T] (None if not wanted)."""
    B, T, H, d = q.shape
    for n, t in (("q", q), ("k", k), ("v", v)):
        _require(t, n, (B, T, H, d), q.dtype, q.device)
    code = _dtype_code(q)
    out = torch.empty_like(q) if out is None else out
    _require(out, "out", (B, T, H, d), q.dtype, q.device)
    if lse is None and want_lse:
        lse = torch.empty((B, H, T), dtype=torch.float32, device=q.device)
    if lse is not None:
        _require(lse, "lse", (B, H, T), torch.float32, q.device)
    lengths = _lengths(lengths, B, q.device)
    _check(load_library().sa_forward(_ptr(q), _ptr(k), _ptr(v), _ptr(out), _ptr(lse), B, T, H, d,
                                     int(Lb), int(La), _ptr(lengths), code,
                                     _stream(q.device, stream)))
    return out, lse


def sa_backward(q, k, v, out, lse, dout, Lb: int, La: int, lengths=None, dq=None, dk=None,
                dv=None, *, stream=None):
    """SA backward. Returns (dq, dk, dv), each [B][T][H][d]."""
    B, T, H, d = q.shape
    for n, t in (("q", q), ("k", k), ("v", v), ("out", out), ("dout", dout)):
        _require(t, n, (B, T, H, d), q.dtype, q.device)
    _require(lse, "lse", (B, H, T), torch.float32, q.device)
    code = _dtype_code(q)
    dq = torch.empty_like(q) if dq is None else dq
    dk = torch.empty_like(q) if dk is None else dk
    dv = torch.empty_like(q) if dv is None else dv
    for n, t in (("dq", dq), ("dk", dk), ("dv", dv)):
        _require(t, n, (B, T, H, d), q.dtype, q.device)
    lengths = _lengths(lengths, B, q.device)
    _check(load_library().sa_backward(_ptr(q), _ptr(k), _ptr(v), _ptr(out), _ptr(lse),
                                      _ptr(dout), _ptr(dq), _ptr(dk), _ptr(dv), B, T, H, d,
                                      int(Lb), int(La), _ptr(lengths), code,
                                      _stream(q.device, stream)))
    return dq, dk, dv


def llsa_forward(q, k, v, Lb: int, La: int, lengths=None, out=None, lse=None, *,
                 want_lse: bool = True, stream=None):
    """Two-branch LLSA forward. q, k, v: [2][B][T][H][d], index 0 = causal
    branch, 1 = look-ahead branch. Returns (out [2][B][T][H][d], lse
    [2][B][H][T] or None)."""
    two, B, T, H, d = q.shape
    if two != 2:
        raise SAError(SA_ERR_INVALID, "LLSA tensors must have a leading dimension of 2")
    for n, t in (("q", q), ("k", k), ("v", v)):
        _require(t, n, (2, B, T, H, d), q.dtype, q.device)
    code = _dtype_code(q)
    out = torch.empty_like(q) if out is None else out
    _require(out, "out", (2, B, T, H, d), q.dtype, q.device)
    if lse is None and want_lse:
        lse = torch.empty((2, B, H, T), dtype=torch.float32, device=q.device)
    if lse is not None:
        _require(lse, "lse", (2, B, H, T), torch.float32, q.device)
    lengths = _lengths(lengths, B, q.device)
    _check(load_library().llsa_forward(_ptr(q), _ptr(k), _ptr(v), _ptr(out), _ptr(lse), B, T, H,
                                       d, int(Lb), int(La), _ptr(lengths), code,
                                       _stream(q.device, stream)))
    return out, lse


def llsa_paper_forward(q, k, v, Lb: int, La: int, lengths=None, out=None, lse=None, *,
                       stream=None):
    """The paper's (La+1)-channel LLSA forward. q, k, v: [La+1][B][T][H][d],
    channel c computed with its own query. Returns (out [La+1][B][T][H][d],
    lse [La+1][B][H][T])."""
    C, B, T, H, d = q.shape
    if C != La + 1:
        raise SAError(SA_ERR_INVALID, "paper LLSA tensors must have La + 1 = %d channels" % (La + 1))
    for n, t in (("q", q), ("k", k), ("v", v)):
        _require(t, n, (C, B, T, H, d), q.dtype, q.device)
    code = _dtype_code(q)
    out = torch.empty_like(q) if out is None else out
    _require(out, "out", (C, B, T, H, d), q.dtype, q.device)
    lse = torch.empty((C, B, H, T), dtype=torch.float32, device=q.device) if lse is None else lse
    _require(lse, "lse", (C, B, H, T), torch.float32, q.device)
    lengths = _lengths(lengths, B, q.device)
    _check(load_library().llsa_paper_forward(_ptr(q), _ptr(k), _ptr(v), _ptr(out), _ptr(lse), B,
                                             T, H, d, int(Lb), int(La), _ptr(lengths), code,
                                             _stream(q.device, stream)))
    return out, lse


def llsa_paper_backward(q, k, v, out, lse, dout, Lb: int, La: int, lengths=None, dq=None,
                        dk=None, dv=None, *, stream=None):
    """Backward of llsa_paper_forward. Every tensor is [La+1][B][T][H][d],
    lse [La+1][B][H][T] from the forward. Returns (dq, dk, dv)."""
    C, B, T, H, d = q.shape
    if C != La + 1:
        raise SAError(SA_ERR_INVALID, "paper LLSA tensors must have La + 1 = %d channels" % (La + 1))
    for n, t in (("q", q), ("k", k), ("v", v), ("out", out), ("dout", dout)):
        _require(t, n, (C, B, T, H, d), q.dtype, q.device)
    _require(lse, "lse", (C, B, H, T), torch.float32, q.device)
    code = _dtype_code(q)
    dq = torch.empty_like(q) if dq is None else dq
    dk = torch.empty_like(q) if dk is None else dk
    dv = torch.empty_like(q) if dv is None else dv
    for n, t in (("dq", dq), ("dk", dk), ("dv", dv)):
        _require(t, n, (C, B, T, H, d), q.dtype, q.device)
    lengths = _lengths(lengths, B, q.device)
    _check(load_library().llsa_paper_backward(_ptr(q), _ptr(k), _ptr(v), _ptr(out), _ptr(lse),
                                              _ptr(dout), _ptr(dq), _ptr(dk), _ptr(dv), B, T, H,
                                              d, int(Lb), int(La), _ptr(lengths), code,
                                              _stream(q.device, stream)))
    return dq, dk, dv


def llsa_backward(q, k, v, out, lse, dout, Lb: int, La: int, lengths=None, dq=None, dk=None,
                  dv=None, *, stream=None):
    """Two-branch LLSA backward. Every tensor is [2][B][T][H][d] (index 0 =
    causal branch, 1 = look-ahead branch), lse [2][B][H][T] from
    llsa_forward. Returns (dq, dk, dv)."""
    two, B, T, H, d = q.shape
    if two != 2:
        raise SAError(SA_ERR_INVALID, "LLSA tensors must have a leading dimension of 2")
    for n, t in (("q", q), ("k", k), ("v", v), ("out", out), ("dout", dout)):
        _require(t, n, (2, B, T, H, d), q.dtype, q.device)
    _require(lse, "lse", (2, B, H, T), torch.float32, q.device)
    code = _dtype_code(q)
    dq = torch.empty_like(q) if dq is None else dq
    dk = torch.empty_like(q) if dk is None else dk
    dv = torch.empty_like(q) if dv is None else dv
    for n, t in (("dq", dq), ("dk", dk), ("dv", dv)):
        _require(t, n, (2, B, T, H, d), q.dtype, q.device)
    lengths = _lengths(lengths, B, q.device)
    _check(load_library().llsa_backward(_ptr(q), _ptr(k), _ptr(v), _ptr(out), _ptr(lse),
                                        _ptr(dout), _ptr(dq), _ptr(dk), _ptr(dv), B, T, H, d,
                                        int(Lb), int(La), _ptr(lengths), code,
                                        _stream(q.device, stream)))
    return dq, dk, dv


class StreamState:
    """Caller-owned ring buffers and counters of ``sa_stream_step`` for S
    streams (allocated here with torch; the library never allocates)."""

    def __init__(self, S: int, H: int, d: int, Lb: int, La: int, R: Optional[int] = None,
                 lengths=None, dtype=torch.bfloat16, device="cuda"):
        self.S, self.H, self.d, self.Lb, self.La = S, H, d, Lb, La
        self.R = R if R is not None else Lb + La + 1
        self.q_ring = torch.zeros((S, La + 1, H, d), dtype=dtype, device=device)
        self.k_ring = torch.zeros((S, self.R, H, d), dtype=dtype, device=device)
        self.v_ring = torch.zeros((S, self.R, H, d), dtype=dtype, device=device)
        self.step_ctr = torch.zeros((S,), dtype=torch.int32, device=device)
        self.emitted = torch.full((S,), -1, dtype=torch.int32, device=device)
        self.lengths = None if lengths is None else torch.as_tensor(
            lengths, dtype=torch.int32).to(device)


def sa_stream_step(state: StreamState, q, k, v, out=None, *, stream=None):
    """One streaming step: q, k, v are the new frames [S][H][d]. Returns
    (out [S][H][d], emitted [S]); emitted[s] = -1 when stream s emitted
    nothing. ``state`` is advanced on the device."""
    S, H, d = state.S, state.H, state.d
    dt = state.k_ring.dtype
    dev = state.k_ring.device
    for n, t in (("q", q), ("k", k), ("v", v)):
        _require(t, n, (S, H, d), dt, dev)
    out = torch.empty_like(q) if out is None else out
    _require(out, "out", (S, H, d), dt, dev)
    code = _dtype_code(state.k_ring)
    _check(load_library().sa_stream_step(
        _ptr(q), _ptr(k), _ptr(v), _ptr(out), _ptr(state.q_ring), _ptr(state.k_ring),
        _ptr(state.v_ring), state.R, _ptr(state.step_ctr), _ptr(state.emitted), S, H, d,
        state.Lb, state.La, _ptr(state.lengths), code, _stream(dev, stream)))
    return out, state.emitted


class LlsaStreamState:
    """Caller-owned rings and counters of ``llsa_stream_step`` for S streams:
    key/value rings of branch C and of branch L (allocated here with torch;
    the library never allocates)."""

    def __init__(self, S: int, H: int, d: int, Lb: int, La: int, R: Optional[int] = None,
                 lengths=None, dtype=torch.bfloat16, device="cuda"):
        self.S, self.H, self.d, self.Lb, self.La = S, H, d, Lb, La
        self.R = R if R is not None else Lb + La + 1
        self.rings = [torch.zeros((S, self.R, H, d), dtype=dtype, device=device)
                      for _ in range(4)]  # k, v of branch C; k, v of branch L
        self.step_ctr = torch.zeros((S,), dtype=torch.int32, device=device)
        self.emitted_c = torch.full((S,), -1, dtype=torch.int32, device=device)
        self.emitted_l = torch.full((S,), -1, dtype=torch.int32, device=device)
        self.lengths = None if lengths is None else torch.as_tensor(
            lengths, dtype=torch.int32).to(device)


def llsa_stream_step(state: LlsaStreamState, qc, kc, vc, ql, kl, vl, out_c=None, out_l=None, *,
                     stream=None):
    """One streaming step: branch C's frame u (qc, kc, vc) and branch L's
    frame u - La (ql, kl, vl), each [S][H][d]. Returns (out_c, emitted_c,
    out_l, emitted_l): the causal output of frame u and the look-ahead output
    of frame u - La; emitted = -1 where nothing was emitted."""
    S, H, d = state.S, state.H, state.d
    dt = state.rings[0].dtype
    dev = state.rings[0].device
    for n, t in (("qc", qc), ("kc", kc), ("vc", vc), ("ql", ql), ("kl", kl), ("vl", vl)):
        _require(t, n, (S, H, d), dt, dev)
    out_c = torch.empty_like(qc) if out_c is None else out_c
    out_l = torch.empty_like(qc) if out_l is None else out_l
    _require(out_c, "out_c", (S, H, d), dt, dev)
    _require(out_l, "out_l", (S, H, d), dt, dev)
    code = _dtype_code(state.rings[0])
    _check(load_library().llsa_stream_step(
        _ptr(qc), _ptr(kc), _ptr(vc), _ptr(ql), _ptr(kl), _ptr(vl), _ptr(out_c), _ptr(out_l),
        *[_ptr(r) for r in state.rings], state.R, _ptr(state.step_ctr), _ptr(state.emitted_c),
        _ptr(state.emitted_l), S, H, d, state.Lb, state.La, _ptr(state.lengths), code,
        _stream(dev, stream)))
    return out_c, state.emitted_c, out_l, state.emitted_l


def copy_reference(src: torch.Tensor, dst: torch.Tensor, mode: int = 0, *, stream=None):
    """Device-copy reference for measurement (not part of the method): copies
    src into dst (same size in bytes, contiguous, GPU) with 16-byte vector
    loads (mode 0) or direct global->LDS copies (mode 1)."""
    if not (src.is_cuda and dst.is_cuda and src.is_contiguous() and dst.is_contiguous()):
        raise SAError(SA_ERR_INVALID, "src and dst must be contiguous GPU tensors")
    n = src.numel() * src.element_size()
    if dst.numel() * dst.element_size() != n:
        raise SAError(SA_ERR_INVALID, "src and dst differ in size")
    _check(load_library().sa_copy_reference(_ptr(src), _ptr(dst), n, int(mode),
                                            _stream(src.device, stream)))
    return dst
