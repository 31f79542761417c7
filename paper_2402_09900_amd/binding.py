"""Python binding of libmemoroid.so (C ABI in include/memoroid.h).

Two layers, both argument marshalling only -- every step of the computation
runs in the library's HIP kernels:

* ``memoroid_*`` functions with the C names and signatures (plain integers
  for pointers), for callers that manage device memory themselves;
* ``scan_diag``, ``scan_diag_bwd``, ``scan_linattn`` ... taking torch CUDA
  tensors: they check shapes, dtypes and contiguity, allocate outputs with
  ``torch.empty`` and launch on the current torch stream.  Without a
  ``workspace`` argument they call the ``*_prepared`` entry points (one
  kernel per call, see include/memoroid.h) on a workspace from a small cache
  of prepared workspaces, one per (device, stream, entry point, sizes,
  flags, operand alignment).  A workspace tensor passed in explicitly goes
  to the self-initialising entry point (which fills what it needs on the
  stream).  ``DiagScan`` wraps the diagonal pair as a
  ``torch.autograd.Function``.

Loading fails loudly (``MemoroidError``) if the shared library is missing:
there is no fallback implementation.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Tuple

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libmemoroid.so")

OK, EINVAL, EUNSUPPORTED, EWORKSPACE, EHIP, ETIMEOUT, EMISMATCH = 0, -1, -2, -3, -4, -5, -6
F32, BF16, C64 = 0, 1, 2
(OP_DIAG, OP_DIAG_BWD, OP_LINATTN, OP_LINATTN_BWD, OP_FFM, OP_FFM_BWD, OP_RETURN, OP_GAE,
 OP_TBB_BEGIN_INDICES, OP_TBB_SAMPLE) = range(10)

_lib = None


class MemoroidError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__("%s failed: %s (status %d)" % (where, status_string(status), status))


def lib() -> ctypes.CDLL:
    """The loaded library (loaded on first use)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise MemoroidError(EHIP, "loading %s (not built: run python -m paper_2402_09900_amd.build)"
                                % LIB_PATH)
        L = ctypes.CDLL(LIB_PATH)
        P, I64, I32, SZ = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int, ctypes.c_size_t
        L.memoroid_abi_version.restype = I32
        L.memoroid_abi_version.argtypes = []
        L.memoroid_status_string.restype = ctypes.c_char_p
        L.memoroid_status_string.argtypes = [I32]
        L.memoroid_scan_diag_workspace_bytes.restype = SZ
        L.memoroid_scan_diag_workspace_bytes.argtypes = [I64, I64, I64, I32, I32]
        L.memoroid_scan_diag.restype = I32
        L.memoroid_scan_diag.argtypes = [P, I64, P, P, P, P, I64, I64, I64, I32, I32, P, SZ, P]
        L.memoroid_scan_diag_bwd_workspace_bytes.restype = SZ
        L.memoroid_scan_diag_bwd_workspace_bytes.argtypes = [I64, I64, I64, I32, I64]
        L.memoroid_scan_diag_bwd.restype = I32
        L.memoroid_scan_diag_bwd.argtypes = [P, I64, P, P, P, P, P, I64, I64, I64, I32, P, SZ, P]
        L.memoroid_scan_linattn_workspace_bytes.restype = SZ
        L.memoroid_scan_linattn_workspace_bytes.argtypes = [I64, I64, I64, I64, I64]
        L.memoroid_scan_linattn.restype = I32
        L.memoroid_scan_linattn.argtypes = [P, P, P, P, P, P, I64, I64, I64, I64, I64, P, SZ, P]
        L.memoroid_scan_linattn_bwd_workspace_bytes.restype = SZ
        L.memoroid_scan_linattn_bwd_workspace_bytes.argtypes = [I64, I64, I64, I64, I64]
        L.memoroid_scan_linattn_bwd.restype = I32
        L.memoroid_scan_linattn_bwd.argtypes = [P, P, P, P, P, P, P, P, P, I64, I64, I64, I64, I64, P, SZ, P]
        L.memoroid_scan_ffm_bwd_workspace_bytes.restype = SZ
        L.memoroid_scan_ffm_bwd_workspace_bytes.argtypes = [I64, I64, I64, I64]
        L.memoroid_scan_ffm_bwd.restype = I32
        L.memoroid_scan_ffm_bwd.argtypes = [P, P, P, P, P, P, P, P, I64, I64, I64, I64, P, SZ, P]
        L.memoroid_scan_ffm_workspace_bytes.restype = SZ
        L.memoroid_scan_ffm_workspace_bytes.argtypes = [I64, I64, I64, I64]
        L.memoroid_scan_ffm.restype = I32
        L.memoroid_scan_ffm.argtypes = [P, P, P, P, P, P, I64, I64, I64, I64, P, SZ, P]
        L.memoroid_tbb_begin_indices_workspace_bytes.restype = SZ
        L.memoroid_tbb_begin_indices_workspace_bytes.argtypes = [I64]
        L.memoroid_tbb_begin_indices.restype = I32
        L.memoroid_tbb_begin_indices.argtypes = [P, I64, I64, P, P, P, SZ, P]
        L.memoroid_tbb_sample_workspace_bytes.restype = SZ
        L.memoroid_tbb_sample_workspace_bytes.argtypes = [I64, I64]
        L.memoroid_tbb_sample.restype = I32
        L.memoroid_tbb_sample.argtypes = [P, I64, I64, P, I64, P, I64, I64, P, P, P, P, P, SZ, P]
        L.memoroid_discount_workspace_bytes.restype = SZ
        L.memoroid_discount_workspace_bytes.argtypes = [I64, I64]
        L.memoroid_discounted_return.restype = I32
        L.memoroid_discounted_return.argtypes = [P, P, ctypes.c_float, P, I64, I64, P, SZ, P]
        L.memoroid_gae.restype = I32
        L.memoroid_gae.argtypes = [P, P, P, P, P, ctypes.c_float, ctypes.c_float, P, P, I64, I64, P, SZ, P]
        L.memoroid_workspace_status.restype = I32
        L.memoroid_workspace_status.argtypes = [P, SZ, P]
        L.memoroid_workspace_prepare.restype = I32
        L.memoroid_workspace_prepare.argtypes = [P, SZ, P]
        for name in ("memoroid_scan_diag", "memoroid_scan_diag_bwd", "memoroid_scan_ffm", "memoroid_scan_ffm_bwd",
                     "memoroid_discounted_return", "memoroid_gae", "memoroid_tbb_begin_indices",
                     "memoroid_tbb_sample"):
            fp = getattr(L, name + "_prepared")
            fp.restype = I32
            fp.argtypes = getattr(L, name).argtypes
        L.memoroid_scan_diag_noalloc.restype = I32
        L.memoroid_scan_diag_noalloc.argtypes = [P, I64, P, P, P, P, I64, I64, I64, I32, I32, P]
        L.memoroid_workspace_bytes.restype = SZ
        L.memoroid_workspace_bytes.argtypes = [I32, I64, I64, I64, I64, I64, I64]
        L.memoroid_testing_set_fallback_polls.restype = I64
        L.memoroid_testing_set_fallback_polls.argtypes = [I64]
        L.memoroid_testing_tile_steps.restype = I64
        L.memoroid_testing_tile_steps.argtypes = [I32, I64, I64, I64, I32, I64, I32]
        _lib = L
    return _lib


# ------------------------------------------------------------ C-named layer

def memoroid_abi_version() -> int:
    return lib().memoroid_abi_version()


def status_string(status: int) -> str:
    try:
        return lib().memoroid_status_string(status).decode()
    except MemoroidError:
        return "status %d" % status


def memoroid_status_string(status: int) -> str:
    return status_string(status)


def memoroid_workspace_bytes(op, B, T, d_or_H, dk, dv, chunk) -> int:
    return lib().memoroid_workspace_bytes(op, B, T, d_or_H, dk, dv, chunk)


def memoroid_testing_set_fallback_polls(polls) -> int:
    return lib().memoroid_testing_set_fallback_polls(polls)


def memoroid_testing_tile_steps(reverse, B, T, d, dtype, a_stride_t, vectorised) -> int:
    return lib().memoroid_testing_tile_steps(reverse, B, T, d, dtype, a_stride_t, vectorised)


def memoroid_scan_diag_workspace_bytes(B, T, d, in_dtype, out_dtype) -> int:
    return lib().memoroid_scan_diag_workspace_bytes(B, T, d, in_dtype, out_dtype)


def memoroid_scan_diag(a, a_stride_t, x, start, h, episode_idx, B, T, d, in_dtype, out_dtype,
                       workspace, workspace_bytes, stream) -> int:
    return lib().memoroid_scan_diag(a, a_stride_t, x, start, h, episode_idx, B, T, d, in_dtype,
                                    out_dtype, workspace, workspace_bytes, stream)


def memoroid_scan_diag_prepared(a, a_stride_t, x, start, h, episode_idx, B, T, d, in_dtype, out_dtype,
                                workspace, workspace_bytes, stream) -> int:
    return lib().memoroid_scan_diag_prepared(a, a_stride_t, x, start, h, episode_idx, B, T, d, in_dtype,
                                             out_dtype, workspace, workspace_bytes, stream)


def memoroid_scan_diag_noalloc(a, a_stride_t, x, start, h, episode_idx, B, T, d, in_dtype, out_dtype,
                               stream) -> int:
    return lib().memoroid_scan_diag_noalloc(a, a_stride_t, x, start, h, episode_idx, B, T, d, in_dtype,
                                            out_dtype, stream)


NOALLOC_SCRATCH_BYTES = 64 << 20    # MEMOROID_NOALLOC_SCRATCH_BYTES


def memoroid_scan_diag_bwd_workspace_bytes(B, T, d, dtype, a_stride_t) -> int:
    return lib().memoroid_scan_diag_bwd_workspace_bytes(B, T, d, dtype, a_stride_t)


def memoroid_scan_diag_bwd(a, a_stride_t, start, h, grad_h, grad_x, grad_a, B, T, d, dtype,
                           workspace, workspace_bytes, stream) -> int:
    return lib().memoroid_scan_diag_bwd(a, a_stride_t, start, h, grad_h, grad_x, grad_a, B, T, d,
                                        dtype, workspace, workspace_bytes, stream)


def memoroid_scan_diag_bwd_prepared(a, a_stride_t, start, h, grad_h, grad_x, grad_a, B, T, d, dtype,
                                    workspace, workspace_bytes, stream) -> int:
    return lib().memoroid_scan_diag_bwd_prepared(a, a_stride_t, start, h, grad_h, grad_x, grad_a, B, T, d,
                                                 dtype, workspace, workspace_bytes, stream)


def memoroid_scan_linattn_workspace_bytes(T, H, dk, dv, chunk) -> int:
    return lib().memoroid_scan_linattn_workspace_bytes(T, H, dk, dv, chunk)


def memoroid_scan_linattn(q, k, v, start, out, episode_idx, T, H, dk, dv, chunk,
                          workspace, workspace_bytes, stream) -> int:
    return lib().memoroid_scan_linattn(q, k, v, start, out, episode_idx, T, H, dk, dv, chunk,
                                       workspace, workspace_bytes, stream)


def memoroid_scan_linattn_bwd_workspace_bytes(T, H, dk, dv, chunk) -> int:
    return lib().memoroid_scan_linattn_bwd_workspace_bytes(T, H, dk, dv, chunk)


def memoroid_scan_linattn_bwd(q, k, v, start, out, grad_out, grad_q, grad_k, grad_v, T, H, dk, dv, chunk,
                              workspace, workspace_bytes, stream) -> int:
    return lib().memoroid_scan_linattn_bwd(q, k, v, start, out, grad_out, grad_q, grad_k, grad_v, T, H, dk, dv,
                                           chunk, workspace, workspace_bytes, stream)


def memoroid_scan_ffm_workspace_bytes(B, T, m, c) -> int:
    return lib().memoroid_scan_ffm_workspace_bytes(B, T, m, c)


def memoroid_scan_ffm(alpha, omega, x, start, S, episode_idx, B, T, m, c, workspace, workspace_bytes,
                      stream) -> int:
    return lib().memoroid_scan_ffm(alpha, omega, x, start, S, episode_idx, B, T, m, c, workspace,
                                   workspace_bytes, stream)


def memoroid_scan_ffm_prepared(alpha, omega, x, start, S, episode_idx, B, T, m, c, workspace, workspace_bytes,
                               stream) -> int:
    return lib().memoroid_scan_ffm_prepared(alpha, omega, x, start, S, episode_idx, B, T, m, c, workspace,
                                            workspace_bytes, stream)


def memoroid_tbb_begin_indices_workspace_bytes(n) -> int:
    return lib().memoroid_tbb_begin_indices_workspace_bytes(n)


def memoroid_tbb_begin_indices(start, n, offset, indices, count, workspace, workspace_bytes, stream) -> int:
    return lib().memoroid_tbb_begin_indices(start, n, offset, indices, count, workspace, workspace_bytes, stream)


def memoroid_tbb_begin_indices_prepared(start, n, offset, indices, count, workspace, workspace_bytes,
                                        stream) -> int:
    return lib().memoroid_tbb_begin_indices_prepared(start, n, offset, indices, count, workspace,
                                                     workspace_bytes, stream)


def memoroid_tbb_sample_workspace_bytes(n_draws, batch) -> int:
    return lib().memoroid_tbb_sample_workspace_bytes(n_draws, batch)


def memoroid_tbb_sample(D, n_D, row_bytes, I, n_I, draws, n_draws, batch, out, out_start, out_src, filled,
                        workspace, workspace_bytes, stream) -> int:
    return lib().memoroid_tbb_sample(D, n_D, row_bytes, I, n_I, draws, n_draws, batch, out, out_start, out_src,
                                     filled, workspace, workspace_bytes, stream)


def memoroid_tbb_sample_prepared(D, n_D, row_bytes, I, n_I, draws, n_draws, batch, out, out_start, out_src,
                                 filled, workspace, workspace_bytes, stream) -> int:
    return lib().memoroid_tbb_sample_prepared(D, n_D, row_bytes, I, n_I, draws, n_draws, batch, out, out_start,
                                              out_src, filled, workspace, workspace_bytes, stream)


def memoroid_scan_ffm_bwd_workspace_bytes(B, T, m, c) -> int:
    return lib().memoroid_scan_ffm_bwd_workspace_bytes(B, T, m, c)


def memoroid_scan_ffm_bwd(alpha, omega, start, S, grad_S, grad_x, grad_alpha, grad_omega, B, T, m, c, workspace,
                          workspace_bytes, stream) -> int:
    return lib().memoroid_scan_ffm_bwd(alpha, omega, start, S, grad_S, grad_x, grad_alpha, grad_omega, B, T, m, c,
                                       workspace, workspace_bytes, stream)


def memoroid_scan_ffm_bwd_prepared(alpha, omega, start, S, grad_S, grad_x, grad_alpha, grad_omega, B, T, m, c,
                                   workspace, workspace_bytes, stream) -> int:
    return lib().memoroid_scan_ffm_bwd_prepared(alpha, omega, start, S, grad_S, grad_x, grad_alpha, grad_omega,
                                                B, T, m, c, workspace, workspace_bytes, stream)


def memoroid_discount_workspace_bytes(B, T) -> int:
    return lib().memoroid_discount_workspace_bytes(B, T)


def memoroid_discounted_return(r, start, gamma, G, B, T, workspace, workspace_bytes, stream) -> int:
    return lib().memoroid_discounted_return(r, start, gamma, G, B, T, workspace, workspace_bytes, stream)


def memoroid_discounted_return_prepared(r, start, gamma, G, B, T, workspace, workspace_bytes, stream) -> int:
    return lib().memoroid_discounted_return_prepared(r, start, gamma, G, B, T, workspace, workspace_bytes, stream)


def memoroid_gae(r, value, value_next, done, start, gamma, lam, adv, target, B, T,
                 workspace, workspace_bytes, stream) -> int:
    return lib().memoroid_gae(r, value, value_next, done, start, gamma, lam, adv, target, B, T,
                              workspace, workspace_bytes, stream)


def memoroid_gae_prepared(r, value, value_next, done, start, gamma, lam, adv, target, B, T,
                          workspace, workspace_bytes, stream) -> int:
    return lib().memoroid_gae_prepared(r, value, value_next, done, start, gamma, lam, adv, target, B, T,
                                       workspace, workspace_bytes, stream)


def memoroid_workspace_status(workspace, workspace_bytes, stream) -> int:
    return lib().memoroid_workspace_status(workspace, workspace_bytes, stream)


def memoroid_workspace_prepare(workspace, workspace_bytes, stream) -> int:
    return lib().memoroid_workspace_prepare(workspace, workspace_bytes, stream)


# ------------------------------------------------------------- torch layer

def _torch():
    import torch
    return torch


def _dtype_code(t) -> int:
    torch = _torch()
    if t.dtype == torch.float32:
        return F32
    if t.dtype == torch.bfloat16:
        return BF16
    if t.dtype == torch.complex64:
        return C64
    raise TypeError("unsupported dtype %s (float32, bfloat16 or complex64)" % t.dtype)


def _stream_ptr(device) -> int:
    torch = _torch()
    return torch.cuda.current_stream(device).cuda_stream


def _check_cuda(*ts):
    dev = None
    for t in ts:
        if t is None:
            continue
        if not t.is_cuda:
            raise ValueError("tensors must live on a CUDA (HIP) device")
        if not t.is_contiguous():
            raise ValueError("tensors must be contiguous")
        if dev is None:
            dev = t.device
        elif t.device != dev:
            raise ValueError("tensors must live on one device")
    return dev


def _raise(status: int, where: str):
    if status != OK:
        raise MemoroidError(status, where)


def _workspace(nbytes: int, device, workspace=None):
    """Workspace of a self-initialising entry point."""
    torch = _torch()
    if workspace is not None and workspace.numel() >= nbytes:
        return workspace
    return torch.empty(max(nbytes, 256), dtype=torch.uint8, device=device)


_PREPARED = None            # OrderedDict: key -> prepared workspace tensor
_PREPARED_MAX = 32


def _prepared(nbytes: int, device, key, operands, workspace=None, entry=None):
    """Workspace and entry point of a call.  With no workspace given: a
    prepared workspace from the cache and the `entry`_prepared function.
    `key` names the entry point and the sizes and flags its layout depends
    on; the alignment of the operands (which selects the vectorised kernels)
    is added here.  A workspace given by the caller goes to the
    self-initialising `entry` (a smaller one raises EWORKSPACE there)."""
    global _PREPARED
    torch = _torch()
    stream = _stream_ptr(device)
    if workspace is not None:
        return workspace, getattr(lib(), entry)
    import collections
    if _PREPARED is None:
        _PREPARED = collections.OrderedDict()
    full = (device.index, stream, key, tuple(t.data_ptr() % 16 == 0 for t in operands if t is not None))
    ws = _PREPARED.get(full)
    if ws is None or ws.numel() < nbytes:
        ws = torch.empty(max(nbytes, 256), dtype=torch.uint8, device=device)
        _raise(lib().memoroid_workspace_prepare(ws.data_ptr(), ws.numel(), stream), "memoroid_workspace_prepare")
        _PREPARED[full] = ws
        while len(_PREPARED) > _PREPARED_MAX:
            _PREPARED.popitem(last=False)
    _PREPARED.move_to_end(full)
    return ws, getattr(lib(), entry + "_prepared")


def _diag_shapes(a, x, start):
    if x.dim() == 2:
        x = x.unsqueeze(0)
    if x.dim() != 3:
        raise ValueError("x must be [B, T, d] or [T, d]")
    B, T, d = x.shape
    if a.dim() == 1:
        if a.shape[0] != d:
            raise ValueError("time-invariant a must have shape [d]")
        stride = 0
    else:
        a = a.reshape(B, T, d)
        stride = d
    start = start.reshape(B, T)
    return a, x, start, B, T, d, stride


def scan_diag(a, x, start, out_dtype=None, episode_idx: bool = False, workspace=None):
    """h_t = x_t at a begin step, else a_t * h_{t-1} + x_t (per feature).

    a: [B,T,d] per step or [d] time-invariant; x: [B,T,d] (or [T,d]);
    start: uint8 [B,T].  Dtypes: float32, bfloat16 (fp32 state; out_dtype
    bfloat16 by default, or float32) or complex64.  Returns h, plus the int32
    episode index [B,T] when episode_idx is true."""
    torch = _torch()
    a, x, start, B, T, d, stride = _diag_shapes(a, x, start)
    dev = _check_cuda(a, x, start)
    if start.dtype != torch.uint8:
        raise TypeError("start must be uint8")
    if a.dtype != x.dtype:
        raise TypeError("a and x must share a dtype")
    in_dt = _dtype_code(x)
    out_torch = x.dtype if out_dtype is None else out_dtype
    out_dt = _dtype_code(torch.empty(0, dtype=out_torch))
    h = torch.empty((B, T, d), dtype=out_torch, device=dev)
    idx = torch.empty((B, T), dtype=torch.int32, device=dev) if episode_idx else None
    nbytes = lib().memoroid_scan_diag_workspace_bytes(B, T, d, in_dt, out_dt)
    ws, fn = _prepared(nbytes, dev, ("diag", B, T, d, in_dt, out_dt, stride), (a, x, h), workspace,
                       "memoroid_scan_diag")
    st = fn(a.data_ptr(), stride, x.data_ptr(), start.data_ptr(), h.data_ptr(),
                                  idx.data_ptr() if idx is not None else None, B, T, d, in_dt, out_dt,
                                  ws.data_ptr(), ws.numel(), _stream_ptr(dev))
    _raise(st, "memoroid_scan_diag")
    return (h, idx) if episode_idx else h


def scan_diag_bwd(a, start, h, grad_h, need_grad_a: bool = True, workspace=None):
    """Reverse scan: returns (grad_x, grad_a); grad_a is [B,T,d] for per-step
    a, [d] for time-invariant a, None if not requested."""
    torch = _torch()
    a, grad_h, start, B, T, d, stride = _diag_shapes(a, grad_h, start)
    h = h.reshape(B, T, d) if h is not None else None
    dev = _check_cuda(a, grad_h, start, h)
    if start.dtype != torch.uint8:
        raise TypeError("start must be uint8")
    dt = _dtype_code(grad_h)
    if dt == BF16:
        raise TypeError("the reverse scan takes float32 or complex64")
    for t in (a, h):
        if t is not None and t.dtype != grad_h.dtype:
            raise TypeError("a, h and grad_h must share a dtype")
    gx = torch.empty((B, T, d), dtype=grad_h.dtype, device=dev)
    ga = None
    if need_grad_a:
        ga = torch.empty((B, T, d) if stride else (d,), dtype=grad_h.dtype, device=dev)
    nbytes = lib().memoroid_scan_diag_bwd_workspace_bytes(B, T, d, dt, stride)
    ws, fn = _prepared(nbytes, dev, ("diag_bwd", B, T, d, dt, stride, need_grad_a), (a, h, grad_h, gx, ga),
                       workspace, "memoroid_scan_diag_bwd")
    st = fn(a.data_ptr(), stride, start.data_ptr(),
                                      h.data_ptr() if h is not None else None, grad_h.data_ptr(),
                                      gx.data_ptr(), ga.data_ptr() if ga is not None else None,
                                      B, T, d, dt, ws.data_ptr(), ws.numel(), _stream_ptr(dev))
    _raise(st, "memoroid_scan_diag_bwd")
    return gx, ga


def scan_linattn(q, k, v, start, episode_idx: bool = False, chunk: int = 64, workspace=None):
    """Linear-transformer memoroid readout phi(q)^T S / (phi(q)^T z) over one
    tape.  q, k: [T,H,dk]; v: [T,H,dv] float32; start: uint8 [T]."""
    torch = _torch()
    dev = _check_cuda(q, k, v, start)
    T, H, dk = q.shape
    dv = v.shape[2]
    if k.shape != q.shape or v.shape[:2] != (T, H):
        raise ValueError("q, k must be [T,H,dk] and v [T,H,dv]")
    for t in (q, k, v):
        if t.dtype != torch.float32:
            raise TypeError("q, k, v must be float32")
    if start.dtype != torch.uint8 or start.numel() != T:
        raise TypeError("start must be uint8 [T]")
    out = torch.empty((T, H, dv), dtype=torch.float32, device=dev)
    idx = torch.empty((T,), dtype=torch.int32, device=dev) if episode_idx else None
    nbytes = lib().memoroid_scan_linattn_workspace_bytes(T, H, dk, dv, chunk)
    ws = _workspace(nbytes, dev, workspace)
    st = lib().memoroid_scan_linattn(q.data_ptr(), k.data_ptr(), v.data_ptr(), start.data_ptr(),
                                     out.data_ptr(), idx.data_ptr() if idx is not None else None,
                                     T, H, dk, dv, chunk, ws.data_ptr(), ws.numel(), _stream_ptr(dev))
    _raise(st, "memoroid_scan_linattn")
    return (out, idx) if episode_idx else out


def scan_ffm(alpha, omega, x, start, episode_idx: bool = False, workspace=None):
    """FFM aggregator state.  alpha float32 [m], omega float32 [c], x float32
    [B,T,m] (or [T,m]), start uint8 [B,T].  Returns S complex64 [B,T,m,c]
    (and the int32 episode index [B,T] when asked)."""
    torch = _torch()
    squeeze = x.dim() == 2
    if squeeze:
        x = x.unsqueeze(0)
    B, T, m = x.shape
    c = omega.shape[0]
    if alpha.shape != (m,):
        raise ValueError("alpha must have shape [m]")
    start = start.reshape(B, T)
    dev = _check_cuda(alpha, omega, x, start)
    for t in (alpha, omega, x):
        if t.dtype != torch.float32:
            raise TypeError("alpha, omega and x must be float32")
    if start.dtype != torch.uint8:
        raise TypeError("start must be uint8")
    S = torch.empty((B, T, m, c), dtype=torch.complex64, device=dev)
    idx = torch.empty((B, T), dtype=torch.int32, device=dev) if episode_idx else None
    ws, fn = _prepared(lib().memoroid_scan_ffm_workspace_bytes(B, T, m, c), dev, ("ffm", B, T, m, c), (S,),
                       workspace, "memoroid_scan_ffm")
    st = fn(alpha.data_ptr(), omega.data_ptr(), x.data_ptr(), start.data_ptr(), S.data_ptr(),
                                 idx.data_ptr() if idx is not None else None, B, T, m, c, ws.data_ptr(), ws.numel(),
                                 _stream_ptr(dev))
    _raise(st, "memoroid_scan_ffm")
    if squeeze:
        S = S[0]
        idx = idx[0] if idx is not None else None
    return (S, idx) if episode_idx else S


def tbb_begin_indices(start, offset: int = 0, workspace=None):
    """Alg. 1's I = offset + where(start) of a rollout (step 0 not forced).
    start: uint8 [n].  Returns (indices int64 [n] of which the first `count`
    are valid, count int64 [1]); both stay on the device."""
    torch = _torch()
    dev = _check_cuda(start)
    if start.dtype != torch.uint8:
        raise TypeError("start must be uint8")
    n = start.numel()
    idx = torch.empty(max(n, 1), dtype=torch.int64, device=dev)
    count = torch.empty(1, dtype=torch.int64, device=dev)
    ws, fn = _prepared(lib().memoroid_tbb_begin_indices_workspace_bytes(n), dev, ("tbb_begins", n), (),
                       workspace, "memoroid_tbb_begin_indices")
    st = fn(start.data_ptr(), n, int(offset), idx.data_ptr(), count.data_ptr(),
                                          ws.data_ptr(), ws.numel(), _stream_ptr(dev))
    _raise(st, "memoroid_tbb_begin_indices")
    return idx, count


def tbb_sample(D, I, draws, batch: int, workspace=None):
    """Alg. 2 batch: D [n_D, ...] (rows on the first axis, any dtype), I int64
    begin indices, draws int64 positions in I.  Returns (out [batch, ...],
    out_start uint8 [batch], out_src int64 [batch], filled int64 [1])."""
    torch = _torch()
    dev = _check_cuda(D, I, draws)
    if I.dtype != torch.int64 or draws.dtype != torch.int64:
        raise TypeError("I and draws must be int64")
    n_D = D.shape[0]
    row_bytes = D.element_size() * (D[0].numel() if n_D else int(torch.tensor(D.shape[1:]).prod().item()))
    out = torch.empty((batch,) + tuple(D.shape[1:]), dtype=D.dtype, device=dev)
    out_start = torch.empty(batch, dtype=torch.uint8, device=dev)
    out_src = torch.empty(batch, dtype=torch.int64, device=dev)
    filled = torch.empty(1, dtype=torch.int64, device=dev)
    nd = draws.numel()
    ws, fn = _prepared(lib().memoroid_tbb_sample_workspace_bytes(nd, batch), dev, ("tbb_sample", nd, batch), (),
                       workspace, "memoroid_tbb_sample")
    st = fn(D.data_ptr(), n_D, row_bytes, I.data_ptr(), I.numel(), draws.data_ptr(), nd,
                                   batch, out.data_ptr(), out_start.data_ptr(), out_src.data_ptr(),
                                   filled.data_ptr(), ws.data_ptr(), ws.numel(), _stream_ptr(dev))
    _raise(st, "memoroid_tbb_sample")
    return out, out_start, out_src, filled


def scan_ffm_bwd(alpha, omega, start, S, grad_S, params: bool = True, workspace=None):
    """Gradient of the FFM aggregator: returns (grad_x [B,T,m], grad_alpha [m],
    grad_omega [c]); the parameter gradients are None when params is false."""
    torch = _torch()
    squeeze = grad_S.dim() == 3
    if squeeze:
        grad_S = grad_S.unsqueeze(0)
        S = S.unsqueeze(0) if S is not None else None
    B, T, m, c = grad_S.shape
    start = start.reshape(B, T)
    dev = _check_cuda(alpha, omega, start, S, grad_S)
    if grad_S.dtype != torch.complex64 or (S is not None and S.dtype != torch.complex64):
        raise TypeError("S and grad_S must be complex64")
    gx = torch.empty((B, T, m), dtype=torch.float32, device=dev)
    ga = torch.empty(m, dtype=torch.float32, device=dev) if params else None
    gw = torch.empty(c, dtype=torch.float32, device=dev) if params else None
    ws, fn = _prepared(lib().memoroid_scan_ffm_bwd_workspace_bytes(B, T, m, c), dev,
                       ("ffm_bwd", B, T, m, c, params), (S, grad_S), workspace, "memoroid_scan_ffm_bwd")
    st = fn(alpha.data_ptr(), omega.data_ptr(), start.data_ptr(),
                                     S.data_ptr() if S is not None else None, grad_S.data_ptr(), gx.data_ptr(),
                                     ga.data_ptr() if ga is not None else None,
                                     gw.data_ptr() if gw is not None else None, B, T, m, c, ws.data_ptr(),
                                     ws.numel(), _stream_ptr(dev))
    _raise(st, "memoroid_scan_ffm_bwd")
    return (gx[0] if squeeze else gx), ga, gw


def _tape_shapes(r, *others):
    if r.dim() == 1:
        r = r.unsqueeze(0)
    if r.dim() != 2:
        raise ValueError("tape tensors must be [B, T] or [T]")
    B, T = r.shape
    return r, [None if o is None else o.reshape(B, T) for o in others], B, T


def discounted_return(r, start, gamma: float, workspace=None):
    """Discounted return of every step to the end of its episode (episodes end
    before each begin step and at the tape end).  r: float32 [B,T] (or [T]);
    start: uint8, same shape.  Returns G shaped like r."""
    torch = _torch()
    shape = r.shape
    r, (start,), B, T = _tape_shapes(r, start)
    dev = _check_cuda(r, start)
    if r.dtype != torch.float32 or start.dtype != torch.uint8:
        raise TypeError("r must be float32 and start uint8")
    G = torch.empty((B, T), dtype=torch.float32, device=dev)
    ws, fn = _prepared(lib().memoroid_discount_workspace_bytes(B, T), dev, ("return", B, T), (), workspace,
                       "memoroid_discounted_return")
    st = fn(r.data_ptr(), start.data_ptr(), float(gamma), G.data_ptr(), B, T,
                                          ws.data_ptr(), ws.numel(), _stream_ptr(dev))
    _raise(st, "memoroid_discounted_return")
    return G.reshape(shape)


def gae(r, value, start, gamma: float, lam: float, value_next=None, done=None, target: bool = True,
        workspace=None):
    """Generalized advantage estimate over a tape.  r, value (and value_next)
    float32 [B,T] (or [T]); start (and done) uint8 of the same shape.
    Returns (adv, target) with target = adv + value (None if not asked)."""
    torch = _torch()
    shape = r.shape
    r, (value, value_next, done, start), B, T = _tape_shapes(r, value, value_next, done, start)
    dev = _check_cuda(r, value, value_next, done, start)
    for t in (r, value, value_next):
        if t is not None and t.dtype != torch.float32:
            raise TypeError("r, value and value_next must be float32")
    for t in (start, done):
        if t is not None and t.dtype != torch.uint8:
            raise TypeError("start and done must be uint8")
    adv = torch.empty((B, T), dtype=torch.float32, device=dev)
    tg = torch.empty((B, T), dtype=torch.float32, device=dev) if target else None
    ws, fn = _prepared(lib().memoroid_discount_workspace_bytes(B, T), dev, ("gae", B, T), (), workspace,
                       "memoroid_gae")
    st = fn(r.data_ptr(), value.data_ptr(),
                            value_next.data_ptr() if value_next is not None else None,
                            done.data_ptr() if done is not None else None, start.data_ptr(),
                            float(gamma), float(lam), adv.data_ptr(), tg.data_ptr() if tg is not None else None,
                            B, T, ws.data_ptr(), ws.numel(), _stream_ptr(dev))
    _raise(st, "memoroid_gae")
    return adv.reshape(shape), (tg.reshape(shape) if tg is not None else None)


def scan_linattn_bwd(q, k, v, start, out, grad_out, chunk: int = 64, workspace=None):
    """Gradient of the linear-attention readout: (dq, dk, dv), each like q /
    k / v.  out is the forward output for the same inputs."""
    torch = _torch()
    dev = _check_cuda(q, k, v, start, out, grad_out)
    T, H, dk = q.shape
    dv = v.shape[2]
    for t in (q, k, v, out, grad_out):
        if t.dtype != torch.float32:
            raise TypeError("q, k, v, out and grad_out must be float32")
    if out.shape != v.shape or grad_out.shape != v.shape or k.shape != q.shape:
        raise ValueError("q, k must be [T,H,dk]; v, out, grad_out [T,H,dv]")
    gq, gk, gv = torch.empty_like(q), torch.empty_like(k), torch.empty_like(v)
    ws = _workspace(lib().memoroid_scan_linattn_bwd_workspace_bytes(T, H, dk, dv, chunk), dev, workspace)
    st = lib().memoroid_scan_linattn_bwd(q.data_ptr(), k.data_ptr(), v.data_ptr(), start.data_ptr(), out.data_ptr(),
                                         grad_out.data_ptr(), gq.data_ptr(), gk.data_ptr(), gv.data_ptr(), T, H,
                                         dk, dv, chunk, ws.data_ptr(), ws.numel(), _stream_ptr(dev))
    _raise(st, "memoroid_scan_linattn_bwd")
    return gq, gk, gv


def workspace_status(workspace) -> int:
    """Synchronise and report OK, ETIMEOUT (a cross-tile wait gave up) or
    EMISMATCH (a prepared workspace was bound to another call) for the calls
    that used `workspace` since it was prepared (self-initialising calls:
    the last call)."""
    return lib().memoroid_workspace_status(workspace.data_ptr(), workspace.numel(),
                                           _stream_ptr(workspace.device))


def _make_autograd():
    torch = _torch()

    class DiagScan(torch.autograd.Function):
        """Differentiable diagonal resettable scan (float32 / complex64)."""

        @staticmethod
        def forward(ctx, a, x, start):
            h = scan_diag(a, x, start)
            ctx.save_for_backward(a, start, h)
            ctx.x_shape = x.shape
            return h.reshape(x.shape)

        @staticmethod
        def backward(ctx, grad_h):
            a, start, h = ctx.saved_tensors
            gx, ga = scan_diag_bwd(a, start, h, grad_h.contiguous(), need_grad_a=ctx.needs_input_grad[0])
            if ga is not None:
                ga = ga.reshape(a.shape)
            return ga, gx.reshape(ctx.x_shape), None

    return DiagScan


_DiagScan = None


def diag_scan(a, x, start):
    """Autograd-aware scan_diag."""
    global _DiagScan
    if _DiagScan is None:
        _DiagScan = _make_autograd()
    return _DiagScan.apply(a, x, start)


def _make_linattn_autograd():
    torch = _torch()

    class LinAttn(torch.autograd.Function):
        """Differentiable linear-attention readout over a tape with resets."""

        @staticmethod
        def forward(ctx, q, k, v, start):
            out = scan_linattn(q, k, v, start)
            ctx.save_for_backward(q, k, v, start, out)
            return out

        @staticmethod
        def backward(ctx, grad_out):
            q, k, v, start, out = ctx.saved_tensors
            gq, gk, gv = scan_linattn_bwd(q, k, v, start, out, grad_out.contiguous())
            return gq, gk, gv, None

    return LinAttn


_LinAttn = None


def linattn(q, k, v, start):
    """Autograd-aware scan_linattn."""
    global _LinAttn
    if _LinAttn is None:
        _LinAttn = _make_linattn_autograd()
    return _LinAttn.apply(q, k, v, start)
