"""MI355X-native forward affine scan and fused selective scan.

Thin Python binding over libscanweaver.so (C ABI in include/scanweaver.h).
Each function only checks and marshals its torch tensors (device, dtype,
contiguity), hands the current HIP stream to the library and raises on a
non-OK status; every step of the computation runs in the HIP kernels.  The
calls go through a small CPython extension (csrc/swcall.c) that mirrors the
C ABI one function per entry point; ``lib()`` is the same ABI through ctypes.

* ``affine_scan(a, bx, h0=None)``: h_t = a_t h_{t-1} + bx_t over the last
  axis of (B, D, L) fp32 tensors (ScanWeaver Sec. 3.1, Eq. (3)).
* ``affine_scan_i32(a, bx, h0=None)``: the same in the int32 wraparound ring.
* ``affine_scan_proj(a, b, x=None, c=None, h0=None)`` (and ``_i32``): the
  elementwise form of Eq. (3)-(4), u = b x and y = c h, returning
  ``(y, h_last)``; with x = c = None it is the weighted prefix of Eq. (10).
* ``affine_scan_schedule(a, bx, h0=None, schedule=...)`` (and ``_i32``): the
  bare scan with the library's schedule or the paper's Blelloch tree
  (Sec. 3.3), for the schedule ablation.
* ``selective_scan_fwd(x, delta, A, Bm, Cm, Dskip=None, ...)``: the
  Mamba-style fused form, returning ``(y, h_last)``; x/delta/Bm/Cm may be fp32
  or bf16, with optional output gate, delta bias and softplus, initial state
  and bf16 y; with ``ckpt=new_ckpt(x, N)`` it also keeps the 8-step
  checkpoints the backward can reuse.
* ``selective_scan_fwd_schedule(...)``: the plain fused form with either
  schedule.
* ``selective_scan_bwd(x, delta, A, Bm, Cm, Dskip, dy, dh_last=None, ...)``:
  every gradient of the fused form (fp32), deterministic.
* ``selective_scan_fn(...)``: the fused form as a torch autograd function
  (forward with checkpoints, the library's backward).
* ``selective_scan_plan(B, D, N, L, ...)``: the kernels, segments and form
  the fused forward would take for those sizes, without launching anything.
"""
from __future__ import annotations

import torch

from ._lib import (SW_DELTA_SOFTPLUS, SW_DTYPE_BF16, SW_DTYPE_F32,  # noqa: F401
                   ScanWeaverError, check, fast, last_error, lib, status_string)

__all__ = ["last_launch", "selective_scan_plan", "affine_scan", "affine_scan_noalloc", "affine_scan_i32", "affine_scan_schedule", "affine_scan_schedule_i32",
           "affine_scan_proj", "affine_scan_proj_i32",
           "selective_scan_fwd", "selective_scan_fwd_schedule", "selective_scan_bwd", "new_ckpt",
           "selective_scan_fn",
           "ScanWeaverError",
           "version"]


def version() -> int:
    return int(lib().sw_version())


def last_launch() -> str:
    """Which kernels this thread's last fused forward or backward call
    enqueued (forward: layout, segment count and form; backward: where its
    checkpoints came from); for tuning and benchmarks, not a stable format."""
    return lib().sw_last_launch().decode()


_FORMS = {0: "whole", 1: "records", 2: "correction"}


def selective_scan_plan(B, D, N, L, dtype="f32", y_dtype=None, train=False, cus=0) -> dict:
    """The kernels the fused forward would take for these sizes (16-byte
    aligned arrays) on a part with ``cus`` compute units (0: the current
    device's), without launching anything: ``layout`` 16, 4, 8 (or 0: nothing
    to launch), ``segments`` and ``segment_steps`` (the last segment takes
    the rest) and ``form`` ("whole", "records" or "correction")."""
    import ctypes
    codes = {"f32": SW_DTYPE_F32, "bf16": SW_DTYPE_BF16}
    layout, form = ctypes.c_int(), ctypes.c_int()
    nseg, lseg = ctypes.c_int64(), ctypes.c_int64()
    check(lib().sw_selective_scan_plan(
        B, D, N, L, codes[dtype], codes[y_dtype or "f32"], int(bool(train)), int(cus),
        ctypes.byref(layout), ctypes.byref(nseg), ctypes.byref(lseg), ctypes.byref(form)),
        "sw_selective_scan_plan")
    return {"layout": layout.value, "segments": nseg.value, "segment_steps": lseg.value,
            "form": _FORMS[form.value]}


def _ptr(t):
    return None if t is None else t.data_ptr()


def _need(t, name, dtype, shape=None):
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if not t.is_cuda:
        raise ValueError(f"{name} must be on a GPU (got {t.device})")
    if t.dtype is not dtype:  # dtypes are singletons
        raise TypeError(f"{name} must be {dtype} (got {t.dtype})")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if shape is not None and t.shape != shape:  # torch.Size compares as a tuple
        raise ValueError(f"{name} must have shape {tuple(shape)} (got {tuple(t.shape)})")


_raw_stream = getattr(torch._C, "_cuda_getCurrentRawStream", None)
_get_device = getattr(torch._C, "_cuda_getDevice", None)


def _current_device():
    # the binding only runs once a GPU tensor exists, so torch's GPU state is
    # initialised and its raw query is enough
    if _get_device is not None:
        return _get_device()
    return torch.cuda.current_device()


def _stream_handle(idx):
    """torch's current HIP stream on GPU idx, as a raw handle."""
    if _raw_stream is not None:
        return _raw_stream(idx)
    return torch.cuda.current_stream(idx).cuda_stream


class _on:
    """``with _on(device):`` makes the tensor's GPU current (switching only when
    another one is) and hands torch's current stream on it to the library, for
    the library calls inside the block."""

    __slots__ = ("idx", "prev")

    def __init__(self, device):
        idx = device.index
        self.idx = idx if idx is not None else _current_device()
        self.prev = -1

    def __enter__(self):
        cur = _current_device()
        if cur != self.idx:
            torch.cuda.set_device(self.idx)
            self.prev = cur
        fast().sw_set_stream(_stream_handle(self.idx))
        return self

    def __exit__(self, *exc):
        if self.prev >= 0:
            torch.cuda.set_device(self.prev)
        return False


def _affine(fn, where, dtype, a, bx, h0, out):
    _need(a, "a", dtype)
    if a.dim() != 3:
        raise ValueError("a must have shape (B, D, L)")
    B, D, L = a.shape
    _need(bx, "bx", dtype, a.shape)
    if h0 is not None:
        _need(h0, "h0", dtype, (B, D))
    if out is None:
        out = torch.empty_like(a)
    else:
        _need(out, "out", dtype, a.shape)
    with _on(a.device):
        check(fn(_ptr(a), _ptr(bx), _ptr(h0), _ptr(out), B, D, L), where)
    return out


def affine_scan(a, bx, h0=None, out=None):
    """Inclusive states of h_t = a_t h_{t-1} + bx_t (fp32, shape (B, D, L))."""
    return _affine(fast().sw_affine_scan, "sw_affine_scan", torch.float32, a, bx, h0, out)


def affine_scan_noalloc(a, bx, h0=None, out=None):
    """:func:`affine_scan` through the entry point that allocates no device
    memory (its look-back scratch is a fixed array in the library; calls with
    more than ``SW_NOALLOC_MAX_CHUNKS`` look-back chunks are refused).  With
    ``out`` given, the call itself allocates nothing."""
    return _affine(fast().sw_affine_scan_noalloc, "sw_affine_scan_noalloc", torch.float32, a, bx,
                   h0, out)


def affine_scan_i32(a, bx, h0=None, out=None):
    """The recurrence in Z/2^32 on int32 tensors (bit-exact for any schedule)."""
    return _affine(fast().sw_affine_scan_i32, "sw_affine_scan_i32", torch.int32, a, bx, h0, out)


_SCHEDULES = {"default": 0, "blelloch": 1}


def affine_scan_schedule(a, bx, h0=None, out=None, *, schedule="default"):
    """:func:`affine_scan` with an explicit scan schedule ("default" or
    "blelloch", the paper's upsweep / downsweep tree)."""
    sched = _SCHEDULES[schedule]
    fn = lambda *args: fast().sw_affine_scan_schedule(*args, sched)  # noqa: E731
    return _affine(fn, "sw_affine_scan_schedule", torch.float32, a, bx, h0, out)


def affine_scan_schedule_i32(a, bx, h0=None, out=None, *, schedule="default"):
    """:func:`affine_scan_i32` with an explicit scan schedule."""
    sched = _SCHEDULES[schedule]
    fn = lambda *args: fast().sw_affine_scan_schedule_i32(*args, sched)  # noqa: E731
    return _affine(fn, "sw_affine_scan_schedule_i32", torch.int32, a, bx, h0, out)


def _affine_proj(fn, where, dtype, a, b, x, c, h0, y, want_h_last):
    _need(a, "a", dtype)
    if a.dim() != 3:
        raise ValueError("a must have shape (B, D, L)")
    B, D, L = a.shape
    _need(b, "b", dtype, a.shape)
    for t, name in ((x, "x"), (c, "c")):
        if t is not None:
            _need(t, name, dtype, a.shape)
    if h0 is not None:
        _need(h0, "h0", dtype, (B, D))
    if y is None:
        y = torch.empty_like(a)
    else:
        _need(y, "y", dtype, a.shape)
    h_last = torch.empty((B, D), dtype=dtype, device=a.device) if want_h_last else None
    with _on(a.device):
        check(fn(_ptr(a), _ptr(b), _ptr(x), _ptr(c), _ptr(h0), _ptr(y), _ptr(h_last), B, D, L),
              where)
    return y, h_last


def affine_scan_proj(a, b, x=None, c=None, h0=None, *, y=None, want_h_last=True):
    """Eq. (3)-(4) elementwise: h_t = a_t h_{t-1} + b_t x_t, y_t = c_t h_t (fp32,
    shape (B, D, L); x, c None mean ones).  Returns ``(y, h_last)``."""
    return _affine_proj(fast().sw_affine_scan_proj, "sw_affine_scan_proj", torch.float32, a, b,
                        x, c, h0, y, want_h_last)


def affine_scan_proj_i32(a, b, x=None, c=None, h0=None, *, y=None, want_h_last=True):
    """The projection form in Z/2^32 on int32 tensors (bit-exact)."""
    return _affine_proj(fast().sw_affine_scan_proj_i32, "sw_affine_scan_proj_i32", torch.int32,
                        a, b, x, c, h0, y, want_h_last)


def selective_scan_fwd(x, delta, A, Bm, Cm, Dskip=None, *, y=None, h_last=None,
                       want_h_last=True, z=None, delta_bias=None, h0=None,
                       delta_softplus=False, y_dtype=torch.float32, ckpt=None, s_pre=None):
    """Fused selective scan forward; returns ``(y, h_last)`` (h_last None if not wanted).

    x, delta: (B, D, L); A: (D, N) fp32; Bm, Cm: (B, L, N); Dskip: (D,) fp32 or None.
    x, delta, Bm, Cm (and z) are all fp32 or all bf16; h_last is fp32; y is
    fp32 or bf16 (``y_dtype``).  Optional inputs of a Mamba block: ``z``
    (B, D, L) gates the output by silu(z); ``delta_bias`` (D,) fp32 is added to
    delta, then ``delta_softplus`` applies softplus; ``h0`` (B, D, N) fp32 is
    the initial state (e.g. the h_last of the previous chunk).  Training:
    ``ckpt=new_ckpt(x, N)`` (N <= 16) receives the 8-step checkpoints and
    ``s_pre`` (B, D, L) fp32 (with ckpt) the output before the gate, both for
    :func:`selective_scan_bwd`.
    """
    if not isinstance(x, torch.Tensor) or x.dim() != 3:
        raise ValueError("x must be a (B, D, L) tensor")
    dt = x.dtype
    if dt not in (torch.float32, torch.bfloat16):
        raise TypeError("x must be float32 or bfloat16")
    if s_pre is not None and ckpt is None:
        raise ValueError("s_pre is written by the training forward: pass ckpt too")
    if y_dtype not in (torch.float32, torch.bfloat16):
        raise TypeError("y_dtype must be float32 or bfloat16")
    B, D, L = x.shape
    _need(x, "x", dt)
    _need(delta, "delta", dt, (B, D, L))
    _need(A, "A", torch.float32)
    if A.dim() != 2 or A.shape[0] != D:
        raise ValueError("A must have shape (D, N)")
    N = A.shape[1]
    _need(Bm, "Bm", dt, (B, L, N))
    _need(Cm, "Cm", dt, (B, L, N))
    if Dskip is not None:
        _need(Dskip, "Dskip", torch.float32, (D,))
    if z is not None:
        _need(z, "z", dt, (B, D, L))
    if delta_bias is not None:
        _need(delta_bias, "delta_bias", torch.float32, (D,))
    if h0 is not None:
        _need(h0, "h0", torch.float32, (B, D, N))
    if y is None:
        y = torch.empty((B, D, L), dtype=y_dtype, device=x.device)
    else:
        _need(y, "y", y_dtype, (B, D, L))
    if want_h_last:
        if h_last is None:
            h_last = torch.empty((B, D, N), dtype=torch.float32, device=x.device)
        else:
            _need(h_last, "h_last", torch.float32, (B, D, N))
    else:
        h_last = None
    in_dt = SW_DTYPE_F32 if dt == torch.float32 else SW_DTYPE_BF16
    out_dt = SW_DTYPE_F32 if y_dtype == torch.float32 else SW_DTYPE_BF16
    flags = SW_DELTA_SOFTPLUS if delta_softplus else 0
    if ckpt is not None:
        _need(ckpt, "ckpt", torch.float32, (B, D, (L + 7) // 8, 16))
    if s_pre is not None:
        _need(s_pre, "s_pre", torch.float32, (B, D, L))
    with _on(x.device):
        if ckpt is not None:
            check(fast().sw_selective_scan_fwd_train(
                _ptr(x), _ptr(delta), _ptr(A), _ptr(Bm), _ptr(Cm), _ptr(Dskip), _ptr(z),
                _ptr(delta_bias), _ptr(h0), _ptr(y), _ptr(h_last), _ptr(ckpt), _ptr(s_pre),
                B, D, N, L, in_dt, out_dt, flags), "sw_selective_scan_fwd_train")
        elif z is None and delta_bias is None and h0 is None and not flags \
                and out_dt == SW_DTYPE_F32:
            fn = fast().sw_selective_scan_fwd if dt == torch.float32 \
                else fast().sw_selective_scan_fwd_bf16
            where = "sw_selective_scan_fwd" if dt == torch.float32 \
                else "sw_selective_scan_fwd_bf16"
            check(fn(_ptr(x), _ptr(delta), _ptr(A), _ptr(Bm), _ptr(Cm), _ptr(Dskip), _ptr(y),
                     _ptr(h_last), B, D, N, L), where)
        else:
            check(fast().sw_selective_scan_fwd_ex(
                _ptr(x), _ptr(delta), _ptr(A), _ptr(Bm), _ptr(Cm), _ptr(Dskip), _ptr(z),
                _ptr(delta_bias), _ptr(h0), _ptr(y), _ptr(h_last), B, D, N, L, in_dt, out_dt,
                flags), "sw_selective_scan_fwd_ex")
    return y, h_last


def selective_scan_fwd_schedule(x, delta, A, Bm, Cm, Dskip=None, *, schedule="default",
                                want_h_last=True):
    """The plain fused forward (fp32 y) with an explicit scan schedule
    ("default" or "blelloch", the paper's tree); returns ``(y, h_last)``."""
    if not isinstance(x, torch.Tensor) or x.dim() != 3:
        raise ValueError("x must be a (B, D, L) tensor")
    dt = x.dtype
    if dt not in (torch.float32, torch.bfloat16):
        raise TypeError("x must be float32 or bfloat16")
    B, D, L = x.shape
    _need(x, "x", dt)
    _need(delta, "delta", dt, (B, D, L))
    _need(A, "A", torch.float32)
    if A.dim() != 2 or A.shape[0] != D:
        raise ValueError("A must have shape (D, N)")
    N = A.shape[1]
    _need(Bm, "Bm", dt, (B, L, N))
    _need(Cm, "Cm", dt, (B, L, N))
    if Dskip is not None:
        _need(Dskip, "Dskip", torch.float32, (D,))
    y = torch.empty((B, D, L), dtype=torch.float32, device=x.device)
    h_last = torch.empty((B, D, N), dtype=torch.float32, device=x.device) if want_h_last else None
    in_dt = SW_DTYPE_F32 if dt == torch.float32 else SW_DTYPE_BF16
    with _on(x.device):
        check(fast().sw_selective_scan_fwd_schedule(
            _ptr(x), _ptr(delta), _ptr(A), _ptr(Bm), _ptr(Cm), _ptr(Dskip), _ptr(y),
            _ptr(h_last), B, D, N, L, in_dt, _SCHEDULES[schedule]),
            "sw_selective_scan_fwd_schedule")
    return y, h_last


def new_ckpt(x, N):
    """An empty checkpoint buffer for :func:`selective_scan_fwd` (``ckpt=``)
    and :func:`selective_scan_bwd`: (B, D, ceil(L/8), 16) fp32."""
    B, D, L = x.shape
    return torch.empty((B, D, (L + 7) // 8, 16), dtype=torch.float32, device=x.device)


def selective_scan_bwd(x, delta, A, Bm, Cm, Dskip, dy, dh_last=None, *, z=None, delta_bias=None,
                       h0=None, delta_softplus=False, want_dh0=True, ckpt=None, s_pre=None):
    """Backward of :func:`selective_scan_fwd`: gradients of sum(dy * y) +
    sum(dh_last * h_last) with respect to every input.

    Inputs as for the forward; ``dy`` (B, D, L) fp32 or bf16, ``dh_last``
    (B, D, N) fp32 or None.  Returns a dict of fp32 tensors ``dx, ddelta``
    (B, D, L), ``dA`` (D, N), ``dB, dC`` (B, L, N), ``dDskip`` and
    ``ddelta_bias`` (D,) when Dskip / delta_bias are given, ``dz`` (B, D, L)
    when z is given, and ``dh0`` (B, D, N) when ``want_dh0``.
    """
    if not isinstance(x, torch.Tensor) or x.dim() != 3:
        raise ValueError("x must be a (B, D, L) tensor")
    dt = x.dtype
    if dt not in (torch.float32, torch.bfloat16):
        raise TypeError("x must be float32 or bfloat16")
    B, D, L = x.shape
    _need(x, "x", dt)
    _need(delta, "delta", dt, (B, D, L))
    _need(A, "A", torch.float32)
    if A.dim() != 2 or A.shape[0] != D:
        raise ValueError("A must have shape (D, N)")
    N = A.shape[1]
    _need(Bm, "Bm", dt, (B, L, N))
    _need(Cm, "Cm", dt, (B, L, N))
    if Dskip is not None:
        _need(Dskip, "Dskip", torch.float32, (D,))
    if z is not None:
        _need(z, "z", dt, (B, D, L))
    if delta_bias is not None:
        _need(delta_bias, "delta_bias", torch.float32, (D,))
    if h0 is not None:
        _need(h0, "h0", torch.float32, (B, D, N))
    if not isinstance(dy, torch.Tensor) or dy.dtype not in (torch.float32, torch.bfloat16):
        raise TypeError("dy must be a float32 or bfloat16 tensor")
    _need(dy, "dy", dy.dtype, (B, D, L))
    if dh_last is not None:
        _need(dh_last, "dh_last", torch.float32, (B, D, N))
    if ckpt is not None:
        _need(ckpt, "ckpt", torch.float32, (B, D, (L + 7) // 8, 16))
    if s_pre is not None:
        _need(s_pre, "s_pre", torch.float32, (B, D, L))
    dev = x.device
    f32 = dict(dtype=torch.float32, device=dev)
    out = {"dx": torch.empty((B, D, L), **f32), "ddelta": torch.empty((B, D, L), **f32),
           "dA": torch.empty((D, N), **f32), "dB": torch.empty((B, L, N), **f32),
           "dC": torch.empty((B, L, N), **f32)}
    out["dDskip"] = torch.empty((D,), **f32) if Dskip is not None else None
    out["ddelta_bias"] = torch.empty((D,), **f32) if delta_bias is not None else None
    out["dz"] = torch.empty((B, D, L), **f32) if z is not None else None
    out["dh0"] = torch.empty((B, D, N), **f32) if want_dh0 else None
    in_dt = SW_DTYPE_F32 if dt == torch.float32 else SW_DTYPE_BF16
    dy_dt = SW_DTYPE_F32 if dy.dtype == torch.float32 else SW_DTYPE_BF16
    with _on(dev):
        check(fast().sw_selective_scan_bwd(
            _ptr(x), _ptr(delta), _ptr(A), _ptr(Bm), _ptr(Cm), _ptr(Dskip), _ptr(z),
            _ptr(delta_bias), _ptr(h0), _ptr(dy), _ptr(dh_last), _ptr(ckpt), _ptr(s_pre),
            _ptr(out["dx"]),
            _ptr(out["ddelta"]), _ptr(out["dA"]), _ptr(out["dB"]), _ptr(out["dC"]),
            _ptr(out["dDskip"]), _ptr(out["dz"]), _ptr(out["ddelta_bias"]), _ptr(out["dh0"]),
            B, D, N, L, in_dt, dy_dt, SW_DELTA_SOFTPLUS if delta_softplus else 0),
            "sw_selective_scan_bwd")
    return {k: v for k, v in out.items() if v is not None}


class _SelectiveScanFn(torch.autograd.Function):
    """Autograd glue: the forward keeps its 8-step checkpoints (N <= 16) and,
    with a gate, its output before the gate; the backward runs
    sw_selective_scan_bwd on them; no arithmetic happens here."""

    @staticmethod
    def forward(ctx, x, delta, A, Bm, Cm, Dskip, z, delta_bias, h0, delta_softplus):
        N = A.shape[1]
        ck = new_ckpt(x, N) if N <= 16 else None
        sp = (torch.empty(x.shape, dtype=torch.float32, device=x.device)
              if ck is not None and z is not None else None)
        y, h_last = selective_scan_fwd(x, delta, A, Bm, Cm, Dskip, z=z, delta_bias=delta_bias,
                                       h0=h0, delta_softplus=delta_softplus, ckpt=ck,
                                       s_pre=sp, y_dtype=torch.float32)
        ctx.save_for_backward(x, delta, A, Bm, Cm, Dskip, z, delta_bias, h0, ck, sp)
        ctx.delta_softplus = delta_softplus
        ctx.set_materialize_grads(False)
        return y, h_last

    @staticmethod
    def backward(ctx, dy, dh_last):
        x, delta, A, Bm, Cm, Dskip, z, delta_bias, h0, ck, sp = ctx.saved_tensors
        if dy is None:  # only h_last reached the loss
            dy = torch.zeros(x.shape, dtype=torch.float32, device=x.device)
        dy = dy.contiguous().to(torch.float32)
        if dh_last is not None:
            dh_last = dh_last.contiguous().to(torch.float32)
        g = selective_scan_bwd(x, delta, A, Bm, Cm, Dskip, dy, dh_last, z=z, delta_bias=delta_bias,
                               h0=h0, delta_softplus=ctx.delta_softplus,
                               want_dh0=h0 is not None and h0.requires_grad, ckpt=ck,
                               s_pre=sp)
        cast = lambda t, like: None if t is None else t.to(like.dtype)  # noqa: E731
        return (cast(g["dx"], x), cast(g["ddelta"], delta), g["dA"], cast(g["dB"], Bm),
                cast(g["dC"], Cm), g.get("dDskip"), cast(g.get("dz"), z) if z is not None else None,
                g.get("ddelta_bias"), g.get("dh0"), None)


def selective_scan_fn(x, delta, A, Bm, Cm, Dskip=None, z=None, delta_bias=None, h0=None,
                      delta_softplus=False, return_last_state=False):
    """Differentiable fused selective scan (fp32 y): :func:`selective_scan_fwd`
    forward, :func:`selective_scan_bwd` backward through torch autograd.
    Gradients come back in each input's dtype.  With ``return_last_state``
    the final state h_last is differentiable too, so segments chained through
    ``h0`` = the previous segment's h_last train end to end."""
    y, h_last = _SelectiveScanFn.apply(x, delta, A, Bm, Cm, Dskip, z, delta_bias, h0,
                                       bool(delta_softplus))
    return (y, h_last) if return_last_state else y
