"""fp64 CPU oracle for the SS2D selective-scan path (ctypes over ``oracle.c``).

TEST INFRASTRUCTURE ONLY: imported by the test suite, the smoke check and the
benchmark's CPU-baseline leg, never by the product path. It shares no code with
the HIP kernels; see ``oracle.c`` for what each function computes and which
passage of the paper it follows.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from typing import Optional, Sequence

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")

_lib = None


def build(force: bool = True) -> str:
    """Compile ``oracle.c`` with gcc (fp64, no FP contraction, OpenMP)."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp"
        cmd = ["gcc", "-O2", "-std=c11", "-ffp-contract=off", "-fno-fast-math", "-fopenmp",
               "-shared", "-fPIC", "-o", tmp, _SRC, "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB):
        build(force=False)
    lib = ctypes.CDLL(_LIB)
    P = ctypes.c_void_p
    I64 = ctypes.c_int64
    scan_args = [P, P, P, P, P, P, P, ctypes.c_int, I64, I64, I64, I64, I64, P, I64, P, ctypes.c_int]
    lib.oracle_full_scan.argtypes = scan_args
    lib.oracle_full_scan.restype = None
    lib.oracle_full_scan_opt.argtypes = scan_args[:15] + [ctypes.c_int] + scan_args[15:]
    lib.oracle_full_scan_opt.restype = None
    lib.oracle_mean_scan.argtypes = scan_args
    lib.oracle_mean_scan.restype = None
    lib.oracle_mean_scan_opt.argtypes = scan_args[:15] + [ctypes.c_int] + scan_args[15:]
    lib.oracle_mean_scan_opt.restype = None
    lib.oracle_mean_scan_pooled.argtypes = scan_args[:13] + [P, ctypes.c_int]
    lib.oracle_mean_scan_pooled.restype = None
    lib.oracle_cross_scan.argtypes = [P, P, I64, I64, I64, I64, I64]
    lib.oracle_cross_merge_f64.argtypes = [P, P, I64, I64, I64, I64]
    lib.oracle_cross_merge_f32.argtypes = [P, P, I64, I64, I64, I64]
    lib.oracle_cross_merge_bf16.argtypes = [P, P, I64, I64, I64, I64]
    lib.oracle_f32_to_bf16.argtypes = [P, P, I64]
    lib.oracle_discrete_scan.argtypes = [P, P, P, P, I64, I64, I64, P, ctypes.c_int]
    lib.oracle_discrete_scan.restype = None
    lib.oracle_channel_mean.argtypes = [P, I64, I64, I64, P, ctypes.c_int]
    lib.oracle_channel_mean.restype = None
    lib.oracle_max_threads.restype = ctypes.c_int
    _lib = lib
    return lib


def _f32(a: Optional[np.ndarray]) -> Optional[np.ndarray]:
    if a is None:
        return None
    return np.ascontiguousarray(a, dtype=np.float32)


def _ptr(a: Optional[np.ndarray]):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def max_threads() -> int:
    return int(_load().oracle_max_threads())


# reading variants of the mean scan (bit flags of oracle_mean_scan_opt)
MEAN_SKIP_PER_CHANNEL = 1  # D u outside T, added per channel after the broadcast
MEAN_RAW = 2               # T averages Delta, u and A before the discretisation
MEAN_NO_BROADCAST = 4      # T^-1 left out: one reduced row per (batch, k)
# zero-order-hold B-bar (eq. 4, second line as (delta A)^-1 (exp(delta A) - I) delta B),
# for full_scan and mean_scan alike
ZOH = 16


def _scan(fn_name, per_seq, u, delta, A, B, C, D, dt_bias, softplus, sel, nthreads,
          options=None, rows=None):
    lib = _load()
    u, delta, A, B, C = map(_f32, (u, delta, A, B, C))
    D, dt_bias = _f32(D), _f32(dt_bias)
    batch, K, Dc, L = u.shape
    N = A.shape[1]
    assert delta.shape == u.shape and A.shape == (K * Dc, N)
    assert B.shape == (batch, K, N, L) and C.shape == B.shape
    if sel is None:
        sel_arr = None
        nsel = batch * K * (Dc if per_seq else 1)
    else:
        sel_arr = np.ascontiguousarray(np.asarray(sel, dtype=np.int64))
        nsel = int(sel_arr.size)
    shape = (nsel, L) if per_seq else (nsel, Dc if rows is None else rows, L)
    y = np.empty(shape, dtype=np.float64)
    args = [_ptr(u), _ptr(delta), _ptr(A), _ptr(B), _ptr(C), _ptr(D), _ptr(dt_bias),
            int(bool(softplus)), batch, K, Dc, L, N, _ptr(sel_arr), nsel]
    if options is not None:
        args.append(int(options))
    getattr(lib, fn_name)(*args, _ptr(y), int(nthreads))
    return y


def full_scan(u, delta, A, B, C, D=None, dt_bias=None, softplus=True,
              sel: Optional[Sequence[int]] = None, nthreads: int = 0,
              options: int = 0) -> np.ndarray:
    """Full selective scan in fp64.

    u, delta: [batch, K, Dc, L]; A: [K*Dc, N]; B, C: [batch, K, N, L];
    D, dt_bias: [K*Dc] or None. Returns [batch, K, Dc, L] (sel None) or
    [len(sel), L] for the flat sequence indices (b*K + k)*Dc + d in ``sel``.
    ``options`` ZOH selects the zero-order-hold B-bar.
    """
    if options:
        y = _scan("oracle_full_scan_opt", True, u, delta, A, B, C, D, dt_bias, softplus, sel,
                  nthreads, options=options)
    else:
        y = _scan("oracle_full_scan", True, u, delta, A, B, C, D, dt_bias, softplus, sel,
                  nthreads)
    if sel is None:
        return y.reshape(np.shape(u))
    return y


def mean_scan(u, delta, A, B, C, D=None, dt_bias=None, softplus=True,
              sel: Optional[Sequence[int]] = None, nthreads: int = 0,
              options: int = 0) -> np.ndarray:
    """VMeanba channel-mean scan in fp64, output broadcast over channels.

    Returns [batch, K, Dc, L] (sel None) or [len(sel), Dc, L] for the flat
    direction indices b*K + k in ``sel``; with MEAN_NO_BROADCAST in
    ``options`` one row per direction instead of Dc ([batch, K, 1, L]).
    ``options`` 0 is the reading of the main path (means of the discretised
    terms, the skip term reduced with them, broadcast output).
    """
    if options == 0:
        y = _scan("oracle_mean_scan", False, u, delta, A, B, C, D, dt_bias, softplus, sel,
                  nthreads)
    else:
        assert not (options & MEAN_NO_BROADCAST and options & MEAN_SKIP_PER_CHANNEL)
        rows = 1 if options & MEAN_NO_BROADCAST else None
        y = _scan("oracle_mean_scan_opt", False, u, delta, A, B, C, D, dt_bias, softplus, sel,
                  nthreads, options=options, rows=rows)
    if sel is None:
        batch, K, Dc, L = np.shape(u)
        return y.reshape(batch, K, y.shape[1], L)
    return y


def mean_scan_pooled(u, delta, A, B, C, D=None, dt_bias=None, softplus=True,
                     nthreads: int = 0) -> np.ndarray:
    """VMeanba scan with T over all K*Dc channels of each batch element, fp64.

    Inputs as for mean_scan. Returns the reduced output [batch, L]; the
    method's output is this row broadcast to every (direction, channel).
    """
    lib = _load()
    u, delta, A, B, C = map(_f32, (u, delta, A, B, C))
    D, dt_bias = _f32(D), _f32(dt_bias)
    batch, K, Dc, L = u.shape
    N = A.shape[1]
    assert delta.shape == u.shape and A.shape == (K * Dc, N)
    assert B.shape == (batch, K, N, L) and C.shape == B.shape
    y = np.empty((batch, L), dtype=np.float64)
    lib.oracle_mean_scan_pooled(_ptr(u), _ptr(delta), _ptr(A), _ptr(B), _ptr(C), _ptr(D),
                                _ptr(dt_bias), int(bool(softplus)), batch, K, Dc, L, N, _ptr(y),
                                int(nthreads))
    return y


def projections(u, W, W_dt=None, N: int = 16):
    """Selection projections of eq. 6 (Linear_N for B and C, Linear then the
    channel expansion for the timescale), fp64, per direction k:
      x_dbl[b,k,r,t] = sum_d W[k,r,d] u[b,k,d,t]          (R + 2N rows)
      B = x_dbl[:, :, R:R+N],  C = x_dbl[:, :, R+N:R+2N]
      delta[b,k,d,t] = sum_r W_dt[k,d,r] x_dbl[b,k,r,t]   (W_dt None, R = 1:
                       x_dbl[b,k,0,t] for every d, the broadcast of eq. 6)
    u [batch, K, Dc, L]; W [K, R+2N, Dc]; W_dt [K, Dc, R] or None.
    Returns (delta, B, C) as float64 arrays. Each product is numpy's matmul.
    """
    u = np.asarray(u, dtype=np.float64)
    W = np.asarray(W, dtype=np.float64)
    batch, K, Dc, L = u.shape
    R = W.shape[1] - 2 * N
    assert W.shape == (K, R + 2 * N, Dc) and R >= 1
    x_dbl = np.matmul(W[None], u)                     # [batch, K, R+2N, L]
    B = x_dbl[:, :, R:R + N]
    C = x_dbl[:, :, R + N:R + 2 * N]
    if W_dt is None:
        assert R == 1
        delta = np.broadcast_to(x_dbl[:, :, :1], (batch, K, Dc, L)).copy()
    else:
        W_dt = np.asarray(W_dt, dtype=np.float64)
        assert W_dt.shape == (K, Dc, R)
        delta = np.matmul(W_dt[None], x_dbl[:, :, :R])  # [batch, K, Dc, L]
    return delta, np.ascontiguousarray(B), np.ascontiguousarray(C)


def out_norm_gate(y, z=None, gamma=None, beta=None, eps: float = 1e-5):
    """The step after the cross-merge in VMamba's SS2D block (not in the
    paper's text): a layer normalisation over the channels of each pixel,
    then, with z given, the gate z * sigmoid(z) (SiLU), fp64:
      mu[b,p]    = mean_d y[b,d,p]
      var[b,p]   = mean_d (y[b,d,p] - mu[b,p])^2          (biased)
      out[b,d,p] = (y[b,d,p] - mu[b,p]) / sqrt(var[b,p] + eps) * gamma[d] + beta[d]
      out[b,d,p] *= z[b,d,p] / (1 + exp(-z[b,d,p]))        (z given)
    y, z [batch, Dc, P] (P = H*W, the 2-D layout); gamma, beta [Dc] or None
    (1 and 0). Returns out [batch, Dc, P] as float64.
    """
    y = np.asarray(y, dtype=np.float64)
    mu = y.mean(axis=1, keepdims=True)
    var = ((y - mu) ** 2).mean(axis=1, keepdims=True)
    out = (y - mu) / np.sqrt(var + eps)
    if gamma is not None:
        out = out * np.asarray(gamma, dtype=np.float64)[None, :, None]
    if beta is not None:
        out = out + np.asarray(beta, dtype=np.float64)[None, :, None]
    if z is not None:
        z = np.asarray(z, dtype=np.float64)
        out = out * (z / (1.0 + np.exp(-z)))
    return out


def discrete_scan(abar, bu, C, skip=None, nthreads: int = 0) -> np.ndarray:
    """One-state scan on materialised inputs in fp64.

    abar, bu, skip: [batch, Dc, L] (skip may be None); C: [batch, L].
    Returns y [batch, Dc, L] with h_t = abar_t h_{t-1} + bu_t, y_t = C_t h_t + skip_t.
    """
    lib = _load()
    abar, bu, C, skip = _f32(abar), _f32(bu), _f32(C), _f32(skip)
    batch, Dc, L = abar.shape
    assert bu.shape == abar.shape and C.shape == (batch, L)
    assert skip is None or skip.shape == abar.shape
    y = np.empty((batch, Dc, L), dtype=np.float64)
    lib.oracle_discrete_scan(_ptr(abar), _ptr(bu), _ptr(C), _ptr(skip), batch, Dc, L, _ptr(y),
                             int(nthreads))
    return y


def channel_mean(x, nthreads: int = 0) -> np.ndarray:
    """T of eq. 9 on a materialised input: x [batch, Dc, L] -> [batch, L] (fp64)."""
    lib = _load()
    x = _f32(x)
    batch, Dc, L = x.shape
    xm = np.empty((batch, L), dtype=np.float64)
    lib.oracle_channel_mean(_ptr(x), batch, Dc, L, _ptr(xm), int(nthreads))
    return xm


def cross_scan(x: np.ndarray) -> np.ndarray:
    """x [batch, Dc, H, W] -> [batch, 4, Dc, H*W] (any element type)."""
    lib = _load()
    x = np.ascontiguousarray(x)
    batch, Dc, H, W = x.shape
    xs = np.empty((batch, 4, Dc, H * W), dtype=x.dtype)
    lib.oracle_cross_scan(_ptr(x), _ptr(xs), batch, Dc, H, W, x.dtype.itemsize)
    return xs


def cross_merge(ys: np.ndarray, H: int, W: int, precision: str = "f64") -> np.ndarray:
    """ys [batch, 4, Dc, H*W] -> [batch, Dc, H, W].

    precision "f64": double sums; "f32": binary32 sums in the fixed
    association; "bf16": ys given as uint16 bfloat16 patterns, binary32 sums,
    one nearest-even rounding (returns uint16 patterns).
    """
    lib = _load()
    batch, K, Dc, L = ys.shape
    assert K == 4 and L == H * W
    if precision == "f64":
        ys = np.ascontiguousarray(ys, dtype=np.float64)
        y = np.empty((batch, Dc, H, W), dtype=np.float64)
        lib.oracle_cross_merge_f64(_ptr(ys), _ptr(y), batch, Dc, H, W)
    elif precision == "f32":
        ys = np.ascontiguousarray(ys, dtype=np.float32)
        y = np.empty((batch, Dc, H, W), dtype=np.float32)
        lib.oracle_cross_merge_f32(_ptr(ys), _ptr(y), batch, Dc, H, W)
    elif precision == "bf16":
        ys = np.ascontiguousarray(ys, dtype=np.uint16)
        y = np.empty((batch, Dc, H, W), dtype=np.uint16)
        lib.oracle_cross_merge_bf16(_ptr(ys), _ptr(y), batch, Dc, H, W)
    else:
        raise ValueError(precision)
    return y


def to_bf16_bits(a: np.ndarray) -> np.ndarray:
    """binary32 -> bfloat16 bit patterns, nearest-even (a bf16 store)."""
    lib = _load()
    a = np.ascontiguousarray(a, dtype=np.float32)
    out = np.empty(a.shape, dtype=np.uint16)
    lib.oracle_f32_to_bf16(_ptr(a), _ptr(out), a.size)
    return out
