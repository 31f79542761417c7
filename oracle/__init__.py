"""fp64 CPU oracle for the resettable memoroid scan -- TEST INFRASTRUCTURE.

Only the tests, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package.  The product library never does, and the
two share no code: the arithmetic lives in ``oracle.c`` (plain sequential fp64
loops, compiled with gcc), this module only marshals numpy arrays through
ctypes.

Each wrapper takes numpy arrays already decoded exactly to float64 / complex128
(fp32 and complex64 widen exactly; bf16 is decoded by the input generator) and
returns float64 / complex128 results together with the magnitude companions
described in ``oracle.h``.
"""
from __future__ import annotations

import contextlib
import ctypes
import os
import shutil
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
_lib = None


def _compile(src: str, out: str) -> None:
    """gcc, plain -O2, no fast-math and no FP contraction, so every
    expression is evaluated as written."""
    cmd = ["gcc", "-std=c99", "-O2", "-ffp-contract=off", "-fno-fast-math",
           "-fPIC", "-shared", "-Wall", "-o", out, src, "-lm"]
    subprocess.run(cmd, check=True)


def build(force: bool = True) -> str:
    """Compile oracle.c into liboracle.so."""
    if force or not os.path.exists(_LIB_PATH):
        tmp = _LIB_PATH + ".tmp%d" % os.getpid()
        _compile(_SRC, tmp)
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def _bind(lib):
    """Declare the argument and result types of every oracle function."""
    P, I64 = ctypes.c_void_p, ctypes.c_int64
    lib.oracle_episode_idx.argtypes = [P, I64, I64, P]
    for name in ("oracle_diag_fwd", "oracle_diag_fwd_c"):
        getattr(lib, name).argtypes = [P, I64, P, P, I64, I64, I64, P, P]
    for name in ("oracle_diag_bwd", "oracle_diag_bwd_c"):
        getattr(lib, name).argtypes = [P, I64, P, P, P, I64, I64, I64, P, P, P, P]
    lib.oracle_phi.argtypes = [ctypes.c_double]
    lib.oracle_phi.restype = ctypes.c_double
    lib.oracle_linattn.argtypes = [P, P, P, P, I64, I64, I64, I64, P, P]
    D = ctypes.c_double
    lib.oracle_discounted_return.argtypes = [P, P, D, I64, I64, P, P]
    lib.oracle_gae.argtypes = [P, P, P, P, P, D, D, I64, I64, P, P, P, P]
    lib.oracle_ffm.argtypes = [P, P, P, P, I64, I64, I64, I64, P, P]
    lib.oracle_linattn_bwd.argtypes = [P, P, P, P, P, I64, I64, I64, I64, P, P, P, P, P, P]
    lib.oracle_ffm_bwd.argtypes = [P, P, P, P, P, I64, I64, I64, I64, P, P, P, P, P, P]
    lib.oracle_ffm_bwd.restype = None
    lib.oracle_linattn_bwd.restype = None
    lib.oracle_tbb_begin_indices.argtypes = [P, I64, I64, P]
    lib.oracle_tbb_begin_indices.restype = I64
    lib.oracle_tbb_sample.argtypes = [P, I64, I64, P, I64, P, I64, I64, P, P, P]
    lib.oracle_tbb_sample.restype = I64
    for name in ("oracle_episode_idx", "oracle_diag_fwd", "oracle_diag_fwd_c",
                 "oracle_diag_bwd", "oracle_diag_bwd_c", "oracle_linattn",
                 "oracle_discounted_return", "oracle_gae", "oracle_ffm"):
        getattr(lib, name).restype = None
    return lib


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            build(force=True)
        _lib = _bind(ctypes.CDLL(_LIB_PATH))
    return _lib


def source() -> str:
    """Text of oracle.c (for tests that compile altered copies of it)."""
    with open(_SRC) as f:
        return f.read()


@contextlib.contextmanager
def variant(src_text: str, workdir: str):
    """Compile `src_text` (an altered copy of oracle.c, e.g. with a mistake
    planted on purpose) into `workdir` and route every wrapper of this
    module through it for the duration of the block.  Used by the tests
    that check the pins fail on a wrong oracle."""
    global _lib
    src = os.path.join(workdir, "oracle_variant.c")
    with open(src, "w") as f:
        f.write(src_text)
    shutil.copy(os.path.join(_HERE, "oracle.h"), os.path.join(workdir, "oracle.h"))
    out = os.path.join(workdir, "liboracle_variant.so")
    _compile(src, out)
    saved = _lib
    _lib = _bind(ctypes.CDLL(out))
    try:
        yield
    finally:
        _lib = saved


def _ptr(arr):
    return None if arr is None else arr.ctypes.data_as(ctypes.c_void_p)


def _flags(start, B, T):
    s = np.ascontiguousarray(start, dtype=np.uint8)
    if s.size != B * T:
        raise ValueError("start must hold B*T flags")
    return s.reshape(B, T)


def episode_idx(start) -> np.ndarray:
    """Per-step episode index; start is [B, T] (or [T])."""
    s = np.asarray(start, dtype=np.uint8)
    s2 = s.reshape(1, -1) if s.ndim == 1 else s
    B, T = s2.shape
    s2 = _flags(s2, B, T)
    out = np.empty((B, T), dtype=np.int32)
    _load().oracle_episode_idx(_ptr(s2), B, T, _ptr(out))
    return out.reshape(s.shape)


def _diag_shapes(a, x, start):
    x = np.asarray(x)
    if x.ndim == 2:
        x = x[None]
    B, T, d = x.shape
    cplx = np.iscomplexobj(x) or np.iscomplexobj(a)
    dt = np.complex128 if cplx else np.float64
    x = np.ascontiguousarray(x, dtype=dt)
    a = np.asarray(a)
    if a.ndim == 1:
        if a.shape[0] != d:
            raise ValueError("time-invariant a must have shape [d]")
        stride = 0
    else:
        a = a.reshape(B, T, d)
        stride = d
    a = np.ascontiguousarray(a, dtype=dt)
    s = _flags(start, B, T)
    return a, x, s, B, T, d, stride, cplx, dt


def diag_fwd(a, x, start):
    """h_t = x_t at a begin step, else a_t h_{t-1} + x_t.

    a: [B,T,d] (per step) or [d] (time-invariant); x: [B,T,d]; start: [B,T].
    Returns (h, m) with m the magnitude companion (float64)."""
    a, x, s, B, T, d, stride, cplx, dt = _diag_shapes(a, x, start)
    h = np.empty((B, T, d), dtype=dt)
    m = np.empty((B, T, d), dtype=np.float64)
    fn = _load().oracle_diag_fwd_c if cplx else _load().oracle_diag_fwd
    fn(_ptr(a), stride, _ptr(x), _ptr(s), B, T, d, _ptr(h), _ptr(m))
    return h, m


def diag_bwd(a, start, h, g):
    """Reverse scan: returns (dx, da, m_dx, m_da); da is [B,T,d] for per-step a
    and [d] (summed) for time-invariant a."""
    a, g, s, B, T, d, stride, cplx, dt = _diag_shapes(a, g, start)
    h = np.ascontiguousarray(np.asarray(h).reshape(B, T, d), dtype=dt)
    dx = np.empty((B, T, d), dtype=dt)
    m_dx = np.empty((B, T, d), dtype=np.float64)
    da_shape = (B, T, d) if stride else (d,)
    da = np.empty(da_shape, dtype=dt)
    m_da = np.empty(da_shape, dtype=np.float64)
    fn = _load().oracle_diag_bwd_c if cplx else _load().oracle_diag_bwd
    fn(_ptr(a), stride, _ptr(s), _ptr(h), _ptr(g), B, T, d,
       _ptr(dx), _ptr(da), _ptr(m_dx), _ptr(m_da))
    return dx, da, m_dx, m_da


def phi(u: float) -> float:
    return _load().oracle_phi(float(u))


def linattn(q, k, v, start):
    """Linear-transformer memoroid readout over one tape.

    q, k: [T,H,dk]; v: [T,H,dv]; start: [T].  Returns (out, m), both
    [T,H,dv] float64."""
    q = np.ascontiguousarray(q, dtype=np.float64)
    k = np.ascontiguousarray(k, dtype=np.float64)
    v = np.ascontiguousarray(v, dtype=np.float64)
    T, H, dk = q.shape
    dv = v.shape[2]
    if k.shape != (T, H, dk) or v.shape[:2] != (T, H):
        raise ValueError("q, k must be [T,H,dk] and v [T,H,dv]")
    s = _flags(start, 1, T)
    out = np.empty((T, H, dv), dtype=np.float64)
    m = np.empty((T, H, dv), dtype=np.float64)
    _load().oracle_linattn(_ptr(q), _ptr(k), _ptr(v), _ptr(s), T, H, dk, dv,
                           _ptr(out), _ptr(m))
    return out, m


def _tape2(x, B=None, T=None):
    x = np.asarray(x)
    x2 = x.reshape(1, -1) if x.ndim == 1 else x
    return np.ascontiguousarray(x2, dtype=np.float64)


def discounted_return(r, start, gamma):
    """G_t = discounted sum of rewards to the end of t's episode.

    r, start: [B,T] (or [T]).  Returns (G, m) shaped like r."""
    shape = np.shape(r)
    r2 = _tape2(r)
    B, T = r2.shape
    s = _flags(start, B, T)
    G = np.empty((B, T), dtype=np.float64)
    m = np.empty((B, T), dtype=np.float64)
    _load().oracle_discounted_return(_ptr(r2), _ptr(s), float(gamma), B, T, _ptr(G), _ptr(m))
    return G.reshape(shape), m.reshape(shape)


def gae(r, v, start, gamma, lam, vn=None, done=None):
    """Generalized advantage estimate over a tape.

    r, v, start (and vn, done if given): [B,T] (or [T]).  Returns
    (adv, target, m_adv, m_target) shaped like r; target = adv + v."""
    shape = np.shape(r)
    r2 = _tape2(r)
    B, T = r2.shape
    v2 = _tape2(v).reshape(B, T)
    vn2 = None if vn is None else _tape2(vn).reshape(B, T)
    d2 = None if done is None else _flags(done, B, T)
    s = _flags(start, B, T)
    out = [np.empty((B, T), dtype=np.float64) for _ in range(4)]
    _load().oracle_gae(_ptr(r2), _ptr(v2), _ptr(vn2), _ptr(d2), _ptr(s), float(gamma), float(lam), B, T,
                       *[_ptr(o) for o in out])
    return tuple(o.reshape(shape) for o in out)


def ffm(alpha, omega, x, start):
    """FFM aggregator state.  alpha [m], omega [c], x [B,T,m] (or [T,m]) real,
    start [B,T].  Returns (S, m) with S complex128 [B,T,m,c] and m its
    magnitude companion (float64, same shape)."""
    x = np.asarray(x, dtype=np.float64)
    squeeze = x.ndim == 2
    if squeeze:
        x = x[None]
    B, T, m = x.shape
    alpha = np.ascontiguousarray(alpha, dtype=np.float64)
    omega = np.ascontiguousarray(omega, dtype=np.float64)
    if alpha.shape != (m,):
        raise ValueError("alpha must have shape [m]")
    c = omega.shape[0]
    x = np.ascontiguousarray(x)
    s = _flags(start, B, T)
    S = np.empty((B, T, m, c), dtype=np.complex128)
    mo = np.empty((B, T, m, c), dtype=np.float64)
    _load().oracle_ffm(_ptr(alpha), _ptr(omega), _ptr(x), _ptr(s), B, T, m, c, _ptr(S), _ptr(mo))
    if squeeze:
        return S[0], mo[0]
    return S, mo


def tbb_begin_indices(start, offset=0):
    """I = offset + where(start != 0) (Alg. 1); step 0 is not forced."""
    s = np.ascontiguousarray(start, dtype=np.uint8).reshape(-1)
    out = np.empty(max(s.size, 1), dtype=np.int64)
    k = _load().oracle_tbb_begin_indices(_ptr(s), s.size, int(offset), _ptr(out))
    return out[:k].copy()


def tbb_sample(D, I, draws, batch):
    """Alg. 2 batch: D is [n_D, ...] (any dtype; rows are its first axis), I
    the begin indices, draws the sampled positions in I.  Returns (out,
    out_start, out_src, filled) with out shaped [batch, ...] like D's rows."""
    D = np.ascontiguousarray(D)
    n_D = D.shape[0]
    row_shape = D.shape[1:]
    row_bytes = int(D.dtype.itemsize * int(np.prod(row_shape, dtype=np.int64)))
    I = np.ascontiguousarray(I, dtype=np.int64)
    draws = np.ascontiguousarray(draws, dtype=np.int64)
    if draws.size and (draws.min() < 0 or draws.max() >= I.size):
        raise ValueError("draws must index I")
    out = np.empty((batch,) + row_shape, dtype=D.dtype)
    out_start = np.empty(batch, dtype=np.uint8)
    out_src = np.empty(batch, dtype=np.int64)
    filled = _load().oracle_tbb_sample(D.ctypes.data_as(ctypes.c_void_p), n_D, row_bytes, _ptr(I), I.size,
                                       _ptr(draws), draws.size, int(batch),
                                       out.ctypes.data_as(ctypes.c_void_p), _ptr(out_start), _ptr(out_src))
    return out, out_start, out_src, int(filled)


def linattn_bwd(q, k, v, start, g):
    """Gradient of the linear-attention readout w.r.t. the raw q, k, v.

    q, k: [T,H,dk]; v, g: [T,H,dv]; start: [T].  Returns (dq, dk, dv, m_dq,
    m_dk, m_dv), all float64, the last three the magnitude companions."""
    q = np.ascontiguousarray(q, dtype=np.float64)
    k = np.ascontiguousarray(k, dtype=np.float64)
    v = np.ascontiguousarray(v, dtype=np.float64)
    g = np.ascontiguousarray(g, dtype=np.float64)
    T, H, dk = q.shape
    dv = v.shape[2]
    if k.shape != (T, H, dk) or v.shape[:2] != (T, H) or g.shape != v.shape:
        raise ValueError("q, k must be [T,H,dk]; v, g [T,H,dv]")
    s = _flags(start, 1, T)
    outs = [np.empty((T, H, dk)), np.empty((T, H, dk)), np.empty((T, H, dv)),
            np.empty((T, H, dk)), np.empty((T, H, dk)), np.empty((T, H, dv))]
    _load().oracle_linattn_bwd(_ptr(q), _ptr(k), _ptr(v), _ptr(s), _ptr(g), T, H, dk, dv,
                               *[_ptr(o) for o in outs])
    return tuple(outs)


def ffm_bwd(alpha, omega, start, S, G):
    """Gradient of the FFM aggregator: S (forward output) and G = dL/dS are
    complex [B,T,m,c] (or [T,m,c]).  Returns (dx [B,T,m], dalpha [m],
    domega [c], m_dx, m_dalpha, m_domega), all float64."""
    S = np.asarray(S)
    squeeze = S.ndim == 3
    S = np.ascontiguousarray(S[None] if squeeze else S, dtype=np.complex128)
    G = np.ascontiguousarray(np.asarray(G).reshape(S.shape), dtype=np.complex128)
    B, T, m, c = S.shape
    alpha = np.ascontiguousarray(alpha, dtype=np.float64)
    omega = np.ascontiguousarray(omega, dtype=np.float64)
    s = _flags(start, B, T)
    dx, mdx = np.empty((B, T, m)), np.empty((B, T, m))
    da, mda, dw, mdw = np.empty(m), np.empty(m), np.empty(c), np.empty(c)
    _load().oracle_ffm_bwd(_ptr(alpha), _ptr(omega), _ptr(s), _ptr(S), _ptr(G), B, T, m, c,
                           _ptr(dx), _ptr(da), _ptr(dw), _ptr(mdx), _ptr(mda), _ptr(mdw))
    if squeeze:
        dx, mdx = dx[0], mdx[0]
    return dx, da, dw, mdx, mda, mdw
