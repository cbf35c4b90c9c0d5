"""CPU oracle for band attention (SA and LLSA) -- TEST INFRASTRUCTURE ONLY.

Only the test suite, the package smoke check and the CPU-baseline leg of the
benchmark import this package. The GPU library never imports, links or calls
it, and it shares no code with the GPU library.

The arithmetic lives in ``sa_oracle.c`` (plain C, double precision, explicit
per-frame windows written from Eq. 4-15 of the paper). This module compiles it
with gcc (no fast-math) on first use and wraps each entry point for NumPy
float64 arrays:

* :func:`sa_forward`   -- Eq. 4-6 (scores over the band, softmax, weighted sum)
* :func:`sa_backward`  -- Eq. 7-13 (explicit softmax Jacobian, M_n for the keys)
* :func:`llsa_forward` -- Eq. 14/15, general channel form with an alias map
* :func:`llsa_two_branch` / :func:`llsa_paper` -- the two instances used here
* :func:`llsa_backward` / :func:`llsa_two_branch_backward` -- the exact adjoint
  of the LLSA forward (Eq. 16 gives only its value part)
* :class:`StreamOracle` -- the streaming step as a literal ring-buffer simulation

Layouts: frame tensors are ``[B][T][H][d]``; log-sum-exp is ``[B][H][T]``.
"""

from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "sa_oracle.c")
_BUILD_DIR = os.path.join(_HERE, "_build")
_LIB_PATH = os.path.join(_BUILD_DIR, "liboracle.so")

_lib = None

_DP = ctypes.POINTER(ctypes.c_double)
_IP = ctypes.POINTER(ctypes.c_int32)


def build(force: bool = True) -> str:
    """Compile ``sa_oracle.c`` into ``_build/liboracle.so`` (gcc -O2, OpenMP)."""
    global _lib
    if not force and os.path.exists(_LIB_PATH):
        return _LIB_PATH
    os.makedirs(_BUILD_DIR, exist_ok=True)
    tmp = _LIB_PATH + ".tmp%d" % os.getpid()
    cmd = ["gcc", "-O2", "-std=c11", "-fopenmp", "-fPIC", "-shared", "-Wall", "-Wextra",
           "-o", tmp, _SRC, "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(tmp, _LIB_PATH)
    _lib = None
    return _LIB_PATH


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH) or os.path.getmtime(_LIB_PATH) < os.path.getmtime(_SRC):
        build(force=True)
    lib = ctypes.CDLL(_LIB_PATH)
    i = ctypes.c_int
    lib.oracle_sa_forward.argtypes = [_DP, _DP, _DP, _DP, _DP, i, i, i, i, i, i, _IP, i]
    lib.oracle_sa_backward.argtypes = [_DP, _DP, _DP, _DP, _DP, _DP, _DP, _DP, i, i, i, i, i, i, _IP,
                                       i]
    lib.oracle_llsa_forward.argtypes = [_DP, _DP, _DP, i, _IP, i, _IP, _IP, i, _DP, _DP,
                                        i, i, i, i, i, i, _IP, i]
    lib.oracle_llsa_backward.argtypes = [_DP, _DP, _DP, _DP, _DP, i, _IP, i, _IP, _IP, i, _DP, _DP,
                                         _DP, i, i, i, i, i, i, _IP, i]
    lib.oracle_sa_stream_step.argtypes = [_DP, _DP, _DP, _DP, _DP, _DP, _DP, i, _IP, _IP,
                                          i, i, i, i, i, _IP]
    lib.oracle_llsa_stream_step.argtypes = [_DP, _DP, _DP, _DP, _DP, _DP, _DP, _DP, _DP, _DP,
                                            _DP, _DP, i, _IP, _IP, _IP, i, i, i, i, i, _IP]
    for fn in (lib.oracle_sa_forward, lib.oracle_sa_backward, lib.oracle_llsa_forward,
               lib.oracle_llsa_backward, lib.oracle_sa_stream_step, lib.oracle_llsa_stream_step):
        fn.restype = ctypes.c_int
    _lib = lib
    return lib


def _f64(x) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(x, dtype=np.float64))


def _dp(a):
    return None if a is None else a.ctypes.data_as(_DP)


def _lengths(lengths, n):
    if lengths is None:
        return None
    arr = np.ascontiguousarray(np.asarray(lengths, dtype=np.int32))
    if arr.shape != (n,):
        raise ValueError("lengths must have shape (%d,)" % n)
    return arr


def _ip(a):
    return None if a is None else a.ctypes.data_as(_IP)


def _check(rc, name):
    if rc != 0:
        raise RuntimeError("%s failed with status %d" % (name, rc))


def default_threads() -> int:
    return os.cpu_count() or 1


def sa_forward(q, k, v, Lb: int, La: int, lengths=None, threads: int = 0):
    """SA forward (Eq. 4-6). Returns ``(y [B][T][H][d], lse [B][H][T])``."""
    q, k, v = _f64(q), _f64(k), _f64(v)
    B, T, H, d = q.shape
    if k.shape != q.shape or v.shape != q.shape:
        raise ValueError("q, k, v must share one shape")
    ln = _lengths(lengths, B)
    y = np.empty_like(q)
    lse = np.empty((B, H, T), dtype=np.float64)
    rc = _load().oracle_sa_forward(_dp(q), _dp(k), _dp(v), _dp(y), _dp(lse), B, T, H, d,
                                   int(Lb), int(La), _ip(ln), threads or default_threads())
    _check(rc, "oracle_sa_forward")
    return y, lse


def sa_backward(q, k, v, dy, Lb: int, La: int, lengths=None, threads: int = 0, y=None):
    """SA backward (Eq. 7-13). Returns ``(dq, dk, dv)``, each ``[B][T][H][d]``.

    ``y`` (optional, ``[B][T][H][d]``): a supplied forward output. Without it
    the gradient is exact (explicit softmax Jacobian); with it the term
    ``sum_i a_i g_i = dy_n . y_n`` of the Jacobian product takes ``y_n`` from
    the supplied output, which is what a backward given a stored (rounded)
    output computes."""
    q, k, v, dy = _f64(q), _f64(k), _f64(v), _f64(dy)
    B, T, H, d = q.shape
    for x in (k, v, dy):
        if x.shape != q.shape:
            raise ValueError("q, k, v, dy must share one shape")
    if y is not None:
        y = _f64(y)
        if y.shape != q.shape:
            raise ValueError("y must have the shape of q")
    ln = _lengths(lengths, B)
    dq, dk, dv = np.empty_like(q), np.empty_like(q), np.empty_like(q)
    rc = _load().oracle_sa_backward(_dp(q), _dp(k), _dp(v), _dp(dy), _dp(y), _dp(dq), _dp(dk),
                                    _dp(dv),
                                    B, T, H, d, int(Lb), int(La), _ip(ln),
                                    threads or default_threads())
    _check(rc, "oracle_sa_backward")
    return dq, dk, dv


def llsa_forward(q, k, v, alias, out_channels, q_branches, Lb: int, La: int, lengths=None,
                 convention: str = "text", threads: int = 0):
    """LLSA forward in the general channel form (Eq. 14/15).

    ``q, k, v``: ``[nbranch][B][T][H][d]``. ``alias[c]`` (c = 0..La) is the
    branch holding input channel c. Output ``o`` computes channel
    ``out_channels[o]`` with the query of branch ``q_branches[o]``.
    ``convention`` is ``"text"`` (Fig. 4: c counts look-ahead frames) or
    ``"eq14"`` (the literal index form of Eq. 14).
    Returns ``(y [nout][B][T][H][d], lse [nout][B][H][T])``.
    """
    q, k, v = _f64(q), _f64(k), _f64(v)
    nb, B, T, H, d = q.shape
    if k.shape != q.shape or v.shape != q.shape:
        raise ValueError("q, k, v must share one shape")
    alias = np.ascontiguousarray(np.asarray(alias, dtype=np.int32))
    outc = np.ascontiguousarray(np.asarray(out_channels, dtype=np.int32))
    qb = np.ascontiguousarray(np.asarray(q_branches, dtype=np.int32))
    if alias.shape != (La + 1,):
        raise ValueError("alias must have La + 1 entries")
    if outc.shape != qb.shape:
        raise ValueError("out_channels and q_branches must have the same length")
    conv = {"text": 0, "eq14": 1}[convention]
    ln = _lengths(lengths, B)
    nout = outc.shape[0]
    y = np.empty((nout, B, T, H, d), dtype=np.float64)
    lse = np.empty((nout, B, H, T), dtype=np.float64)
    rc = _load().oracle_llsa_forward(_dp(q), _dp(k), _dp(v), nb, _ip(alias), nout, _ip(outc),
                                     _ip(qb), conv, _dp(y), _dp(lse), B, T, H, d, int(Lb),
                                     int(La), _ip(ln), threads or default_threads())
    _check(rc, "oracle_llsa_forward")
    return y, lse


def llsa_backward(q, k, v, dy, alias, out_channels, q_branches, Lb: int, La: int, lengths=None,
                  convention: str = "text", threads: int = 0, y=None):
    """Gradient of the LLSA forward (same arguments as :func:`llsa_forward`)
    for the output gradient ``dy [nout][B][T][H][d]``: the exact adjoint of
    the forward's gather. Returns ``(dq, dk, dv)``, each
    ``[nbranch][B][T][H][d]``. ``y`` (optional, ``[nout][B][T][H][d]``): a
    supplied forward output, used as in :func:`sa_backward`."""
    q, k, v, dy = _f64(q), _f64(k), _f64(v), _f64(dy)
    nb, B, T, H, d = q.shape
    if k.shape != q.shape or v.shape != q.shape:
        raise ValueError("q, k, v must share one shape")
    alias = np.ascontiguousarray(np.asarray(alias, dtype=np.int32))
    outc = np.ascontiguousarray(np.asarray(out_channels, dtype=np.int32))
    qb = np.ascontiguousarray(np.asarray(q_branches, dtype=np.int32))
    if alias.shape != (La + 1,):
        raise ValueError("alias must have La + 1 entries")
    if outc.shape != qb.shape:
        raise ValueError("out_channels and q_branches must have the same length")
    nout = outc.shape[0]
    if dy.shape != (nout, B, T, H, d):
        raise ValueError("dy must have shape %s" % ((nout, B, T, H, d),))
    if y is not None:
        y = _f64(y)
        if y.shape != dy.shape:
            raise ValueError("y must have the shape of dy")
    conv = {"text": 0, "eq14": 1}[convention]
    ln = _lengths(lengths, B)
    dq, dk, dv = np.empty_like(q), np.empty_like(q), np.empty_like(q)
    rc = _load().oracle_llsa_backward(_dp(q), _dp(k), _dp(v), _dp(dy), _dp(y), nb, _ip(alias), nout,
                                      _ip(outc), _ip(qb), conv, _dp(dq), _dp(dk), _dp(dv), B, T,
                                      H, d, int(Lb), int(La), _ip(ln),
                                      threads or default_threads())
    _check(rc, "oracle_llsa_backward")
    return dq, dk, dv


# Branch indices of the two-branch LLSA tensors.
CAUSAL = 0
LOOKAHEAD = 1


def llsa_two_branch(q, k, v, Lb: int, La: int, lengths=None, threads: int = 0):
    """Two-branch LLSA: branch 0 = causal (C), branch 1 = look-ahead (L).

    The paper's LLSA with input channels 0..La-1 held by the causal branch and
    channel La held by the look-ahead branch; output 0 is channel 0 with the
    causal query, output 1 is channel La with the look-ahead query. For La = 1
    this is exactly the paper's two-channel module.
    """
    alias = [CAUSAL] * La + [LOOKAHEAD]
    return llsa_forward(q, k, v, alias, [0, La], [CAUSAL, LOOKAHEAD], Lb, La, lengths,
                        "text", threads)


def llsa_two_branch_backward(q, k, v, dy, Lb: int, La: int, lengths=None, threads: int = 0,
                             y=None):
    """Gradient of :func:`llsa_two_branch` for ``dy [2][B][T][H][d]``;
    returns ``(dq, dk, dv)``, each ``[2][B][T][H][d]`` (index 0 = causal
    branch, 1 = look-ahead branch)."""
    alias = [CAUSAL] * La + [LOOKAHEAD]
    return llsa_backward(q, k, v, dy, alias, [0, La], [CAUSAL, LOOKAHEAD], Lb, La, lengths,
                         "text", threads, y)


def llsa_paper(q, k, v, Lb: int, La: int, lengths=None, convention: str = "text",
               threads: int = 0):
    """The paper's (La+1)-channel LLSA: channel c of every tensor is its own
    branch, and every channel is computed with its own query."""
    chans = list(range(La + 1))
    return llsa_forward(q, k, v, chans, chans, chans, Lb, La, lengths, convention, threads)


def llsa_paper_backward(q, k, v, dy, Lb: int, La: int, lengths=None, convention: str = "text",
                        threads: int = 0, y=None):
    """Gradient of :func:`llsa_paper` for ``dy [La+1][B][T][H][d]``; returns
    ``(dq, dk, dv)``, each ``[La+1][B][T][H][d]``."""
    chans = list(range(La + 1))
    return llsa_backward(q, k, v, dy, chans, chans, chans, Lb, La, lengths, convention, threads,
                         y)


class StreamOracle:
    """Per-stream ring buffers driven one frame at a time (SA streaming step).

    ``R`` must be at least ``Lb + La + 1``. ``lengths[s]`` (or None for
    open-ended streams) bounds the frames each stream accepts.
    """

    def __init__(self, S: int, H: int, d: int, Lb: int, La: int, R: int, lengths=None):
        if R < Lb + La + 1:
            raise ValueError("the ring must hold at least Lb + La + 1 frames")
        self.S, self.H, self.d, self.Lb, self.La, self.R = S, H, d, Lb, La, R
        self.q_ring = np.zeros((S, La + 1, H, d), dtype=np.float64)
        self.k_ring = np.zeros((S, R, H, d), dtype=np.float64)
        self.v_ring = np.zeros((S, R, H, d), dtype=np.float64)
        self.step_ctr = np.zeros((S,), dtype=np.int32)
        self.lengths = _lengths(lengths, S)

    def step(self, q, k, v):
        """Feed one frame per stream (``[S][H][d]`` each); returns
        ``(out [S][H][d], emitted [S])`` with ``emitted[s] = -1`` when stream s
        emitted nothing this step."""
        q, k, v = _f64(q), _f64(k), _f64(v)
        shape = (self.S, self.H, self.d)
        for x in (q, k, v):
            if x.shape != shape:
                raise ValueError("frames must have shape %s" % (shape,))
        out = np.empty(shape, dtype=np.float64)
        emitted = np.empty((self.S,), dtype=np.int32)
        rc = _load().oracle_sa_stream_step(
            _dp(q), _dp(k), _dp(v), _dp(out), _dp(self.q_ring), _dp(self.k_ring),
            _dp(self.v_ring), self.R, _ip(self.step_ctr), _ip(emitted), self.S, self.H,
            self.d, self.Lb, self.La, _ip(self.lengths))
        _check(rc, "oracle_sa_stream_step")
        return out, emitted


class LlsaStreamOracle:
    """Two-branch LLSA streaming step: per-stream key/value rings of the
    causal branch C and the look-ahead branch L, driven one step at a time.
    At step u a stream takes branch C's frame u and branch L's frame u - La
    and emits the causal output of frame u and the look-ahead output of frame
    u - La. ``R`` must be at least ``Lb + La + 1``."""

    def __init__(self, S: int, H: int, d: int, Lb: int, La: int, R: int, lengths=None):
        if R < Lb + La + 1:
            raise ValueError("the rings must hold at least Lb + La + 1 frames")
        self.S, self.H, self.d, self.Lb, self.La, self.R = S, H, d, Lb, La, R
        self.rings = [np.zeros((S, R, H, d), dtype=np.float64) for _ in range(4)]
        self.step_ctr = np.zeros((S,), dtype=np.int32)
        self.lengths = _lengths(lengths, S)

    def step(self, qc, kc, vc, ql, kl, vl):
        """Feed branch C's frame u and branch L's frame u - La of every stream
        (``[S][H][d]`` each); returns ``(out_c, emitted_c, out_l, emitted_l)``
        with ``emitted[s] = -1`` where stream s emitted nothing."""
        xs = [_f64(x) for x in (qc, kc, vc, ql, kl, vl)]
        shape = (self.S, self.H, self.d)
        for x in xs:
            if x.shape != shape:
                raise ValueError("frames must have shape %s" % (shape,))
        out_c = np.empty(shape, dtype=np.float64)
        out_l = np.empty(shape, dtype=np.float64)
        em_c = np.empty((self.S,), dtype=np.int32)
        em_l = np.empty((self.S,), dtype=np.int32)
        rc = _load().oracle_llsa_stream_step(
            *[_dp(x) for x in xs], _dp(out_c), _dp(out_l), *[_dp(r) for r in self.rings], self.R,
            _ip(self.step_ctr), _ip(em_c), _ip(em_l), self.S, self.H, self.d, self.Lb, self.La,
            _ip(self.lengths))
        _check(rc, "oracle_llsa_stream_step")
        return out_c, em_c, out_l, em_l
