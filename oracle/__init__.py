"""Plain CPU reference (the oracle) for the affine-recurrence hot path.

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import this package.  The product
package never imports it, and it shares no code with the HIP sources.

The arithmetic lives in ``sw_oracle.c`` (plain C, fp64 and uint32 loops).  This
module only compiles that file with gcc and marshals numpy arrays to it.

What each routine computes (see ``sw_oracle.c`` for the loops):

* ``affine_scan`` / ``affine_scan_i32``: the recurrence of Sec. 3.1, Eq. (3),
  ``h_t = a_t h_{t-1} + bx_t``, as a sequential loop; all inclusive states.
* ``affine_prefix`` / ``affine_prefix_i32``: the inclusive prefix compositions
  of Sec. 3.2 built with the operator of Eq. (7), and the state rebuilt from
  them, ``h_t = A_{1:t} h_0 + U_{1:t}``.
* ``compose`` / ``compose_u32``: Eq. (7) itself.
* ``selective_scan``: the Mamba-style fused form (Sec. 1, Sec. 3.1) with
  ``a = exp(delta A)``, ``u = delta B x``, ``y = sum_n C h + Dskip x``, and
  the optional pieces of a Mamba block (delta bias and softplus, initial
  state, output gate).
* ``selective_scan_seq32``: the same as a plain fp32 sequential loop.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
import threading

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "sw_oracle.c")
_HDR = os.path.join(_HERE, "sw_oracle.h")
_LIB_PATH = os.path.join(_HERE, "libsw_oracle.so")
_lock = threading.Lock()
_lib = None

_f32p = np.ctypeslib.ndpointer(dtype=np.float32, flags="C_CONTIGUOUS")
_f64p = np.ctypeslib.ndpointer(dtype=np.float64, flags="C_CONTIGUOUS")
_u32p = np.ctypeslib.ndpointer(dtype=np.uint32, flags="C_CONTIGUOUS")
_i64p = np.ctypeslib.ndpointer(dtype=np.int64, flags="C_CONTIGUOUS")
_vp = ctypes.c_void_p
_i64 = ctypes.c_int64


def build(force: bool = False) -> str:
    """Compile sw_oracle.c into libsw_oracle.so (gcc, -O2, no fast-math)."""
    stale = (not os.path.exists(_LIB_PATH)) or any(
        os.path.getmtime(p) > os.path.getmtime(_LIB_PATH) for p in (_SRC, _HDR))
    if force or stale:
        tmp = _LIB_PATH + ".tmp%d" % os.getpid()
        cmd = ["gcc", "-O2", "-fno-fast-math", "-std=c11", "-Wall", "-Wextra", "-fPIC",
               "-shared", "-pthread", "-o", tmp, _SRC, "-lm"]
        subprocess.run(cmd, check=True, cwd=_HERE)
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def _load():
    global _lib
    with _lock:
        if _lib is not None:
            return _lib
        build()
        lib = ctypes.CDLL(_LIB_PATH)
        lib.swo_threads_used.argtypes = [ctypes.c_int, _i64]
        lib.swo_threads_used.restype = ctypes.c_int
        lib.swo_compose_f64.argtypes = [ctypes.c_double] * 4 + [ctypes.POINTER(ctypes.c_double)] * 2
        lib.swo_compose_f64.restype = None
        lib.swo_compose_u32.argtypes = [ctypes.c_uint32] * 4 + [ctypes.POINTER(ctypes.c_uint32)] * 2
        lib.swo_compose_u32.restype = None
        lib.swo_affine_scan_f64.argtypes = [_vp] * 6 + [_i64, _i64, ctypes.c_int]
        lib.swo_affine_scan_f64.restype = ctypes.c_int
        lib.swo_affine_scan_u32.argtypes = [_vp] * 4 + [_i64, _i64, ctypes.c_int]
        lib.swo_affine_scan_u32.restype = ctypes.c_int
        lib.swo_affine_proj_f64.argtypes = [_vp] * 9 + [_i64, _i64, ctypes.c_int]
        lib.swo_affine_proj_f64.restype = ctypes.c_int
        lib.swo_affine_proj_u32.argtypes = [_vp] * 7 + [_i64, _i64, ctypes.c_int]
        lib.swo_affine_proj_u32.restype = ctypes.c_int
        lib.swo_affine_prefix_f64.argtypes = [_vp] * 6 + [_i64, _i64]
        lib.swo_affine_prefix_f64.restype = ctypes.c_int
        lib.swo_affine_prefix_u32.argtypes = [_vp] * 6 + [_i64, _i64]
        lib.swo_affine_prefix_u32.restype = ctypes.c_int
        lib.swo_selective_scan_f64.argtypes = [_vp] * 13 + [_i64, _i64, _i64, ctypes.c_int,
                                                            ctypes.c_int]
        lib.swo_selective_scan_f64.restype = ctypes.c_int
        lib.swo_selective_scan_ex_f64.argtypes = ([_vp] * 10 + [ctypes.c_int] + [_vp] * 6
                                                  + [_i64, _i64, _i64, ctypes.c_int, ctypes.c_int])
        lib.swo_selective_scan_ex_f64.restype = ctypes.c_int
        lib.swo_selective_scan_bwd_f64.argtypes = ([_vp] * 10 + [ctypes.c_int] + [_vp] * 12
                                                   + [_i64] * 4 + [ctypes.c_int])
        lib.swo_selective_scan_bwd_f64.restype = ctypes.c_int
        lib.swo_selective_scan_f32seq.argtypes = [_vp] * 9 + [_i64, _i64, _i64, ctypes.c_int]
        lib.swo_selective_scan_f32seq.restype = ctypes.c_int
        _lib = lib
        return lib


def _p(arr):
    return None if arr is None else arr.ctypes.data_as(ctypes.c_void_p)


def _as(arr, dtype):
    return None if arr is None else np.ascontiguousarray(arr, dtype=dtype)


def threads_used(requested: int, rows: int) -> int:
    """Threads a call with ``requested`` threads (<=0: all CPUs) over ``rows`` uses."""
    return int(_load().swo_threads_used(int(requested), int(rows)))


def compose(p2, p1):
    """Eq. (7) in fp64: ``(A2,U2) (+) (A1,U1) = (A2 A1, A2 U1 + U2)``."""
    A = ctypes.c_double()
    U = ctypes.c_double()
    _load().swo_compose_f64(float(p2[0]), float(p2[1]), float(p1[0]), float(p1[1]),
                            ctypes.byref(A), ctypes.byref(U))
    return (A.value, U.value)


def compose_u32(p2, p1):
    """Eq. (7) in Z/2^32 (operands and results as uint32)."""
    A = ctypes.c_uint32()
    U = ctypes.c_uint32()
    m = 0xFFFFFFFF
    _load().swo_compose_u32(int(p2[0]) & m, int(p2[1]) & m, int(p1[0]) & m, int(p1[1]) & m,
                            ctypes.byref(A), ctypes.byref(U))
    return (A.value, U.value)


def _rows_L(a):
    L = a.shape[-1] if a.ndim else 0
    rows = int(np.prod(a.shape[:-1])) if a.ndim > 1 else 1
    return rows, L


def affine_scan(a, bx, h0=None, bounds: bool = False, threads: int = 0):
    """Sequential fp64 evaluation of Eq. (3) over the last axis.

    ``a`` and ``bx`` are fp32 arrays of shape (..., L); ``h0`` has shape (...)
    or is None (zero).  Returns ``h`` (fp64, same shape), and with
    ``bounds=True`` also ``(mag, sens)`` (see sw_oracle.c).
    """
    a = _as(a, np.float32)
    bx = _as(bx, np.float32)
    if a.shape != bx.shape:
        raise ValueError("a and bx must have the same shape")
    rows, L = _rows_L(a)
    h0 = _as(h0, np.float32)
    if h0 is not None and h0.size != rows:
        raise ValueError("h0 must hold one value per row")
    h = np.empty(a.shape, np.float64)
    mag = np.empty(a.shape, np.float64) if bounds else None
    sens = np.empty(a.shape, np.float64) if bounds else None
    rc = _load().swo_affine_scan_f64(_p(a), _p(bx), _p(h0), _p(h), _p(mag), _p(sens), rows, L,
                                     int(threads))
    if rc != 0:
        raise ValueError("oracle rejected the arguments")
    return (h, mag, sens) if bounds else h


def affine_scan_i32(a, bx, h0=None, threads: int = 0):
    """Eq. (3) in the int32 wraparound ring; int32 in, int32 out."""
    a = _as(a, np.int32).view(np.uint32)
    bx = _as(bx, np.int32).view(np.uint32)
    if a.shape != bx.shape:
        raise ValueError("a and bx must have the same shape")
    rows, L = _rows_L(a)
    h0 = None if h0 is None else _as(h0, np.int32).view(np.uint32)
    if h0 is not None and h0.size != rows:
        raise ValueError("h0 must hold one value per row")
    h = np.empty(a.shape, np.uint32)
    rc = _load().swo_affine_scan_u32(_p(a), _p(bx), _p(h0), _p(h), rows, L, int(threads))
    if rc != 0:
        raise ValueError("oracle rejected the arguments")
    return h.view(np.int32)


def _proj_args(a, b, x, c, h0, dtype):
    a, b = _as(a, dtype), _as(b, dtype)
    x, c = _as(x, dtype), _as(c, dtype)
    for v, name in ((b, "b"), (x, "x"), (c, "c")):
        if v is not None and v.shape != a.shape:
            raise ValueError(f"{name} must have the shape of a")
    rows, L = _rows_L(a)
    h0 = _as(h0, dtype)
    if h0 is not None and h0.size != rows:
        raise ValueError("h0 must hold one value per row")
    return a, b, x, c, h0, rows, L


def affine_proj(a, b, x=None, c=None, h0=None, bounds: bool = False, threads: int = 0):
    """Eq. (3)-(4) with input and output projections, fp64: per row
    h_t = a_t h_{t-1} + b_t x_t and y_t = c_t h_t (x, c None: ones).

    fp32 arrays of shape (..., L); ``h0`` has shape (...) or is None.  Returns
    ``(y, h_last)`` and with ``bounds=True`` also ``(y_mag, y_sens)``.
    """
    a, b, x, c, h0, rows, L = _proj_args(a, b, x, c, h0, np.float32)
    y = np.empty(a.shape, np.float64)
    h_last = np.empty(a.shape[:-1], np.float64)
    ym = np.empty(a.shape, np.float64) if bounds else None
    ys = np.empty(a.shape, np.float64) if bounds else None
    rc = _load().swo_affine_proj_f64(_p(a), _p(b), _p(x), _p(c), _p(h0), _p(y), _p(h_last),
                                     _p(ym), _p(ys), rows, L, int(threads))
    if rc != 0:
        raise ValueError("oracle rejected the arguments")
    return (y, h_last, ym, ys) if bounds else (y, h_last)


def affine_proj_i32(a, b, x=None, c=None, h0=None, threads: int = 0):
    """Eq. (3)-(4) with projections in the int32 wraparound ring; returns
    ``(y, h_last)`` as int32."""
    cv = (lambda v: None if v is None else _as(v, np.int32).view(np.uint32))
    a, b, x, c, h0 = (cv(v) for v in (a, b, x, c, h0))
    a, b, x, c, h0, rows, L = _proj_args(a, b, x, c, h0, np.uint32)
    y = np.empty(a.shape, np.uint32)
    h_last = np.empty(a.shape[:-1], np.uint32)
    rc = _load().swo_affine_proj_u32(_p(a), _p(b), _p(x), _p(c), _p(h0), _p(y), _p(h_last),
                                     rows, L, int(threads))
    if rc != 0:
        raise ValueError("oracle rejected the arguments")
    return y.view(np.int32), h_last.view(np.int32)


def affine_prefix(a, bx, h0=None):
    """Sec. 3.2 prefix compositions (fp64): returns ``(A_pre, U_pre, h)``."""
    a = _as(a, np.float32)
    bx = _as(bx, np.float32)
    rows, L = _rows_L(a)
    h0 = _as(h0, np.float32)
    A = np.empty(a.shape, np.float64)
    U = np.empty(a.shape, np.float64)
    h = np.empty(a.shape, np.float64)
    if _load().swo_affine_prefix_f64(_p(a), _p(bx), _p(h0), _p(A), _p(U), _p(h), rows, L):
        raise ValueError("oracle rejected the arguments")
    return A, U, h


def affine_prefix_i32(a, bx, h0=None):
    """Sec. 3.2 prefix compositions in Z/2^32: returns int32 ``(A_pre, U_pre, h)``."""
    a = _as(a, np.int32).view(np.uint32)
    bx = _as(bx, np.int32).view(np.uint32)
    rows, L = _rows_L(a)
    h0 = None if h0 is None else _as(h0, np.int32).view(np.uint32)
    A = np.empty(a.shape, np.uint32)
    U = np.empty(a.shape, np.uint32)
    h = np.empty(a.shape, np.uint32)
    if _load().swo_affine_prefix_u32(_p(a), _p(bx), _p(h0), _p(A), _p(U), _p(h), rows, L):
        raise ValueError("oracle rejected the arguments")
    return A.view(np.int32), U.view(np.int32), h.view(np.int32)


def _selective_rows(x, delta, A, Bm, Cm, Dskip, rows, z=None, delta_bias=None, h0=None):
    """Flatten the fused-scan inputs to the per-row layout of the C loops."""
    x = np.asarray(x)
    Bsz, D, L = x.shape
    N = np.asarray(A).shape[1]
    x2 = x.reshape(Bsz * D, L)
    d2 = np.asarray(delta).reshape(Bsz * D, L)
    if rows is None:
        ridx = None
        xs = _as(x2, np.float32)
        ds = _as(d2, np.float32)
        R = Bsz * D
        row_b = np.repeat(np.arange(Bsz, dtype=np.int64), D)
        As = _as(np.tile(np.asarray(A, np.float32), (Bsz, 1)), np.float32)
        Ds = None if Dskip is None else _as(np.tile(np.asarray(Dskip, np.float32), Bsz),
                                            np.float32)
    else:
        ridx = np.asarray(rows, dtype=np.int64).reshape(-1)
        if ridx.size and (ridx.min() < 0 or ridx.max() >= Bsz * D):
            raise ValueError("row index out of range")
        R = ridx.size
        xs = _as(x2[ridx], np.float32)
        ds = _as(d2[ridx], np.float32)
        row_b = np.ascontiguousarray(ridx // D, dtype=np.int64)
        As = _as(np.asarray(A, np.float32)[ridx % D], np.float32)
        Ds = None if Dskip is None else _as(np.asarray(Dskip, np.float32)[ridx % D], np.float32)
    Bs = _as(Bm, np.float32)
    Cs = _as(Cm, np.float32)
    if Bs.shape != (Bsz, L, N) or Cs.shape != (Bsz, L, N):
        raise ValueError("Bm and Cm must have shape (B, L, N)")
    sel = slice(None) if ridx is None else ridx
    zs = None if z is None else _as(np.asarray(z).reshape(Bsz * D, L)[sel], np.float32)
    h0s = None if h0 is None else _as(np.asarray(h0).reshape(Bsz * D, N)[sel], np.float32)
    if delta_bias is None:
        dbs = None
    else:
        db = np.asarray(delta_bias, np.float32)
        dbs = _as(np.tile(db, Bsz) if ridx is None else db[ridx % D], np.float32)
    return dict(Bsz=Bsz, D=D, L=L, N=N, R=R, ridx=ridx, xs=xs, ds=ds, row_b=row_b, As=As,
                Ds=Ds, Bs=Bs, Cs=Cs, zs=zs, dbs=dbs, h0s=h0s)


def _unflatten(out, f):
    if f["ridx"] is None:
        for k in list(out):
            out[k] = out[k].reshape((f["Bsz"], f["D"]) + out[k].shape[1:])
    return out


def selective_scan(x, delta, A, Bm, Cm, Dskip=None, rows=None, a_mode: int = 0,
                   bounds: bool = False, threads: int = 0, z=None, delta_bias=None, h0=None,
                   delta_softplus: bool = False):
    """Fused selective scan in fp64.

    Shapes: ``x, delta`` (B, D, L); ``A`` (D, N); ``Bm, Cm`` (B, L, N);
    ``Dskip`` (D,) or None.  All values are taken as given (fp32, or bf16
    values already widened exactly to fp32).

    ``rows``: optional 1-D array of flat row indices ``b*D + d``; only those
    rows are evaluated and results have a leading axis of len(rows) instead
    of (B, D).

    ``a_mode=1`` rounds every ``a = exp(delta A)`` to fp32 before use.

    Optional inputs of a Mamba block: ``delta_bias`` (D,) is added to delta,
    ``delta_softplus`` then applies log(1 + exp(.)), ``h0`` (B, D, N) is the
    initial state, and ``z`` (B, D, L) gates the output, y * z / (1 + e^-z).

    Returns a dict with ``y`` and ``h_last``; with ``bounds=True`` also
    ``y_mag, y_sens, h_mag, h_sens``.
    """
    f = _selective_rows(x, delta, A, Bm, Cm, Dskip, rows, z, delta_bias, h0)
    R, N, L = f["R"], f["N"], f["L"]
    y = np.empty((R, L), np.float64)
    h_last = np.empty((R, N), np.float64)
    ym = np.empty((R, L), np.float64) if bounds else None
    ys = np.empty((R, L), np.float64) if bounds else None
    hm = np.empty((R, N), np.float64) if bounds else None
    hs = np.empty((R, N), np.float64) if bounds else None
    rc = _load().swo_selective_scan_ex_f64(_p(f["xs"]), _p(f["ds"]), _p(f["As"]), _p(f["Bs"]),
                                           _p(f["Cs"]), _p(f["row_b"]), _p(f["Ds"]),
                                           _p(f["zs"]), _p(f["dbs"]), _p(f["h0s"]),
                                           int(bool(delta_softplus)), _p(y), _p(h_last),
                                           _p(ym), _p(ys), _p(hm), _p(hs), R, N, L,
                                           int(a_mode), int(threads))
    if rc != 0:
        raise ValueError("oracle rejected the arguments")
    out = {"y": y, "h_last": h_last}
    if bounds:
        out.update(y_mag=ym, y_sens=ys, h_mag=hm, h_sens=hs)
    return _unflatten(out, f)


def selective_scan_seq32(x, delta, A, Bm, Cm, Dskip=None, rows=None, threads: int = 0):
    """The fused form as a plain fp32 sequential loop (every operation rounded
    to fp32 in the written order, libm ``expf``, no FMA).  Same arguments and
    layout as :func:`selective_scan`; returns fp32 ``y`` and ``h_last``.  It
    measures what a direct fp32 evaluation incurs against the fp64 loop."""
    f = _selective_rows(x, delta, A, Bm, Cm, Dskip, rows)
    R, N, L = f["R"], f["N"], f["L"]
    y = np.empty((R, L), np.float32)
    h_last = np.empty((R, N), np.float32)
    rc = _load().swo_selective_scan_f32seq(_p(f["xs"]), _p(f["ds"]), _p(f["As"]), _p(f["Bs"]),
                                           _p(f["Cs"]), _p(f["row_b"]), _p(f["Ds"]), _p(y),
                                           _p(h_last), R, N, L, int(threads))
    if rc != 0:
        raise ValueError("oracle rejected the arguments")
    return _unflatten({"y": y, "h_last": h_last}, f)


def selective_scan_bwd(x, delta, A, Bm, Cm, Dskip=None, dy=None, dh_last=None, *, z=None,
                       delta_bias=None, h0=None, delta_softplus: bool = False, rows=None,
                       bounds: bool = False, threads: int = 0):
    """Backward of the fused selective scan in fp64 (chain rule through the
    forward loop; see sw_oracle.c): gradients of sum(dy * y) + sum(dh_last *
    h_last) with respect to every input.

    Inputs as for :func:`selective_scan`; ``dy`` (B, D, L), ``dh_last``
    (B, D, N) or None.  Returns a dict with ``dx, ddelta`` (and ``dz`` when z
    is given) of shape (B, D, L), ``dh0`` (B, D, N), ``dA`` (D, N), ``dDskip``
    and ``ddelta_bias`` (D,), ``dB, dC`` (B, L, N).  With ``rows`` (flat row
    indices b*D + d) only those rows are evaluated: per-row outputs get a
    leading axis of len(rows), ``dA_rows`` (R, N), ``dDskip_rows`` and
    ``ddelta_bias_rows`` (R,) hold each row's share, and ``dB, dC`` are summed
    over the given rows only.  With ``bounds=True`` every output ``k`` also
    has ``m_k``, the magnitude (sum of absolute values of its terms).
    """
    f = _selective_rows(x, delta, A, Bm, Cm, Dskip, rows, z=z, delta_bias=delta_bias, h0=h0)
    Bsz, D, L, N, R = f["Bsz"], f["D"], f["L"], f["N"], f["R"]
    sel = slice(None) if f["ridx"] is None else f["ridx"]
    dys = _as(np.asarray(dy, np.float32).reshape(Bsz * D, L)[sel], np.float32)
    dhl = None if dh_last is None else _as(
        np.asarray(dh_last, np.float32).reshape(Bsz * D, N)[sel], np.float32)
    out = {k: np.zeros((R, L)) for k in ("dx", "ddelta")}
    out["dz"] = np.zeros((R, L)) if z is not None else None
    out["dh0"] = np.zeros((R, N))
    out["dA_rows"] = np.zeros((R, N))
    out["dDskip_rows"] = np.zeros(R)
    out["ddelta_bias_rows"] = np.zeros(R)
    out["dB"] = np.zeros((Bsz, L, N))
    out["dC"] = np.zeros((Bsz, L, N))
    names = ["dx", "ddelta", "dz", "dA_rows", "dDskip_rows", "ddelta_bias_rows", "dh0", "dB", "dC"]
    mags = None
    if bounds:
        for k in names:
            out["m_" + k] = None if out[k] is None else np.zeros_like(out[k])
        mags = (ctypes.c_void_p * 9)(*[_p(out["m_" + k]) for k in names])
    rc = _load().swo_selective_scan_bwd_f64(
        _p(f["xs"]), _p(f["ds"]), _p(f["As"]), _p(f["Bs"]), _p(f["Cs"]), _p(f["row_b"]),
        _p(f["Ds"]), _p(f["zs"]), _p(f["dbs"]), _p(f["h0s"]), int(bool(delta_softplus)),
        _p(dys), _p(dhl), _p(out["dx"]), _p(out["ddelta"]), _p(out["dz"]), _p(out["dA_rows"]),
        _p(out["dDskip_rows"]), _p(out["ddelta_bias_rows"]), _p(out["dh0"]), _p(out["dB"]),
        _p(out["dC"]), mags, Bsz, R, N, L, int(threads))
    if rc != 0:
        raise ValueError("oracle rejected the arguments")
    if f["ridx"] is None:
        for k in ("dx", "ddelta", "dz", "dh0"):
            for kk in (k, "m_" + k):
                if out.get(kk) is not None:
                    out[kk] = out[kk].reshape((Bsz, D) + out[kk].shape[1:])
        for src, dst in (("dA_rows", "dA"), ("dDskip_rows", "dDskip"),
                         ("ddelta_bias_rows", "ddelta_bias")):
            for pre in ("", "m_"):
                if (pre + src) in out:
                    v = out.pop(pre + src)
                    out[pre + dst] = v.reshape((Bsz, D) + v.shape[1:]).sum(axis=0)
    return out
