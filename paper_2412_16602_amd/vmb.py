"""Python binding of libvmb (ctypes). Argument marshalling only.

Each function takes torch tensors that already live on the GPU, checks that
they are contiguous CUDA (HIP) tensors of the expected element type, and
passes raw device pointers, sizes and the current HIP stream to the C entry
point of the same name; every step of the computation runs in the HIP
kernels. A non-OK status raises ``VmbError``. There is no CPU fallback: if
the library is missing or was not built, loading fails loudly.
"""
from __future__ import annotations

import ctypes
import os
import re
from typing import Optional

import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libvmb.so")
HEADER_PATH = os.path.join(os.path.dirname(_PKG), "include", "vmb.h")

VMB_F32, VMB_BF16 = 0, 1
VMB_LAYOUT_SEQ, VMB_LAYOUT_2D = 0, 1
# vmb_mean_option bits (vmb_mean_scan_fwd_ex)
VMB_MEAN_SKIP_PER_CHANNEL, VMB_MEAN_RAW, VMB_MEAN_NO_BROADCAST, VMB_MEAN_POOLED = 1, 2, 4, 8
# test hook of the mean scan's error report (see include/vmb.h)
VMB_MEAN_TEST_GIVE_UP = 1 << 30
# vmb_scan_option bits (vmb_selective_scan_fwd_ex; vmb_mean_scan_fwd_ex takes them too)
VMB_SCAN_ZOH = 16

STATUS = {0: "VMB_OK", 1: "VMB_ERR_NULL", 2: "VMB_ERR_SHAPE", 3: "VMB_ERR_DTYPE",
          4: "VMB_ERR_ALIGN", 5: "VMB_ERR_ALIAS", 6: "VMB_ERR_UNSUPPORTED",
          7: "VMB_ERR_WORKSPACE", 8: "VMB_ERR_HIP", 9: "VMB_ERR_INCOMPLETE"}
VMB_OK, VMB_ERR_UNSUPPORTED, VMB_ERR_WORKSPACE, VMB_ERR_INCOMPLETE = 0, 6, 7, 9


class VmbError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: {STATUS.get(status, status)} ({status_string(status)})")


_lib = None


def load_library():
    """Load libvmb.so (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"libvmb.so not found at {LIB_PATH}; run __graft_entry__.build()")
    lib = ctypes.CDLL(LIB_PATH)
    P, I64, I = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int
    cross = [P, P, I64, I64, I64, I64, I, P]
    for name in ("vmb_cross_scan", "vmb_cross_merge"):
        fn = getattr(lib, name)
        fn.argtypes = cross
        fn.restype = I
    scan = [P, P, P, P, P, P, P, I, P, I64, I64, I64, I64, I64, I, I, I, I64, I64, P,
            ctypes.c_size_t, P]
    for name in ("vmb_selective_scan_fwd", "vmb_mean_scan_fwd"):
        fn = getattr(lib, name)
        fn.argtypes = scan
        fn.restype = I
    for name in ("vmb_selective_scan_fwd_ex", "vmb_mean_scan_fwd_ex"):
        fn = getattr(lib, name)
        fn.argtypes = scan[:-1] + [ctypes.c_uint, P]
        fn.restype = I
    lib.vmb_ss2d_projections.argtypes = [P, P, P, P, P, P, I64, I64, I64, I64, I64, I64, I, P]
    lib.vmb_ss2d_projections.restype = I
    lib.vmb_ss2d_out_norm.argtypes = [P, P, P, P, ctypes.c_float, P, I64, I64, I64, I, P]
    lib.vmb_ss2d_out_norm.restype = I
    lib.vmb_discrete_scan.argtypes = [P, P, P, P, P, I64, I64, I64, P]
    lib.vmb_discrete_scan.restype = I
    lib.vmb_channel_mean.argtypes = [P, P, I64, I64, I64, P]
    lib.vmb_channel_mean.restype = I
    lib.vmb_scan_workspace_bytes.argtypes = [I, I64, I64, I64, I64, I64, I]
    lib.vmb_scan_workspace_bytes.restype = ctypes.c_size_t
    lib.vmb_mean_scan_fwd_noalloc.argtypes = scan[:-3] + [P]
    lib.vmb_mean_scan_fwd_noalloc.restype = I
    lib.vmb_mean_scan_status.argtypes = [P, P]
    lib.vmb_mean_scan_status.restype = I
    lib.vmb_status_string.argtypes = [I]
    lib.vmb_status_string.restype = ctypes.c_char_p
    lib.vmb_abi_version.argtypes = []
    lib.vmb_abi_version.restype = I
    _lib = lib
    return lib


def declared_symbols() -> list[str]:
    """Function names declared in include/vmb.h."""
    with open(HEADER_PATH) as f:
        text = f.read()
    return sorted(set(re.findall(r"\b(vmb_[a-z_0-9]+)\s*\(", text)))


def status_string(status: int) -> str:
    try:
        return load_library().vmb_status_string(int(status)).decode()
    except Exception:  # the message is best-effort; the code is in the exception
        return "?"


def abi_version() -> int:
    return int(load_library().vmb_abi_version())


# ---------------------------------------------------------------- helpers

_DT = {torch.float32: VMB_F32, torch.bfloat16: VMB_BF16}


def _dev(t: Optional[torch.Tensor], name: str):
    if t is None:
        return None
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if not t.is_cuda:
        raise ValueError(f"{name} must be a GPU tensor (got {t.device})")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return ctypes.c_void_p(t.data_ptr())


def _dtype(t: torch.Tensor, name: str) -> int:
    if t.dtype not in _DT:
        raise ValueError(f"{name}: unsupported dtype {t.dtype}")
    return _DT[t.dtype]


def _f32(t: Optional[torch.Tensor], name: str):
    if t is not None and t.dtype != torch.float32:
        raise ValueError(f"{name} must be float32")
    return _dev(t, name)


def _stream(stream) -> ctypes.c_void_p:
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(int(stream.cuda_stream))


def _check(status: int, where: str):
    if status != 0:
        raise VmbError(status, where)


# ---------------------------------------------------------------- entry points

def vmb_cross_scan(x: torch.Tensor, xs: torch.Tensor, stream=None) -> torch.Tensor:
    """x [batch, channels, H, W] -> xs [batch, 4, channels, H*W] (same dtype)."""
    lib = load_library()
    batch, channels, H, W = x.shape
    dt = _dtype(x, "x")
    if xs.dtype != x.dtype:
        raise ValueError("xs must have the dtype of x")
    if tuple(xs.shape) != (batch, 4, channels, H * W):
        raise ValueError(f"xs shape {tuple(xs.shape)} != {(batch, 4, channels, H * W)}")
    _check(lib.vmb_cross_scan(_dev(x, "x"), _dev(xs, "xs"), batch, channels, H, W, dt,
                              _stream(stream)), "vmb_cross_scan")
    return xs


def vmb_cross_merge(ys: torch.Tensor, y: torch.Tensor, stream=None) -> torch.Tensor:
    """ys [batch, 4, channels, H*W] -> y [batch, channels, H, W] (same dtype)."""
    lib = load_library()
    batch, channels, H, W = y.shape
    dt = _dtype(ys, "ys")
    if y.dtype != ys.dtype:
        raise ValueError("y must have the dtype of ys")
    if tuple(ys.shape) != (batch, 4, channels, H * W):
        raise ValueError(f"ys shape {tuple(ys.shape)} != {(batch, 4, channels, H * W)}")
    _check(lib.vmb_cross_merge(_dev(ys, "ys"), _dev(y, "y"), batch, channels, H, W, dt,
                               _stream(stream)), "vmb_cross_merge")
    return y


def vmb_scan_workspace_bytes(mean_variant: bool, batch: int, K: int, channels: int, L: int,
                             N: int, layout: int = VMB_LAYOUT_SEQ) -> int:
    return int(load_library().vmb_scan_workspace_bytes(int(bool(mean_variant)), batch, K,
                                                       channels, L, N, layout))


def _scan(name, mean_variant, u, delta, A, B, C, D, dt_bias, delta_softplus, y, layout,
          workspace, stream, options=None):
    lib = load_library()
    batch, K, channels, L = delta.shape
    N = A.shape[1]
    in_dt = _dtype(delta, "delta")
    out_dt = _dtype(y, "y")
    for t, nm in ((u, "u"), (B, "B"), (C, "C")):
        if t.dtype != delta.dtype:
            raise ValueError(f"{nm} must have the dtype of delta")
    if layout == VMB_LAYOUT_2D:
        if u.dim() != 4 or u.shape[0] != batch or u.shape[1] != channels:
            raise ValueError("2-D layout: u must be x [batch, channels, H, W]")
        H, W = int(u.shape[2]), int(u.shape[3])
        y_shape = (batch, channels, H, W)
    else:
        H, W = 1, L
        if tuple(u.shape) != (batch, K, channels, L):
            raise ValueError(f"u shape {tuple(u.shape)} != {(batch, K, channels, L)}")
        rows = 1 if options and options & VMB_MEAN_NO_BROADCAST else channels
        y_shape = (batch, K, rows, L)
    if tuple(y.shape) != y_shape:
        raise ValueError(f"y shape {tuple(y.shape)} != {y_shape}")
    for t, nm in ((B, "B"), (C, "C")):
        if tuple(t.shape) != (batch, K, N, L):
            raise ValueError(f"{nm} shape {tuple(t.shape)} != {(batch, K, N, L)}")
    if tuple(A.shape) != (K * channels, N):
        raise ValueError(f"A shape {tuple(A.shape)} != {(K * channels, N)}")
    for t, nm in ((D, "D"), (dt_bias, "dt_bias")):
        if t is not None and t.numel() != K * channels:
            raise ValueError(f"{nm} must hold K * channels = {K * channels} values")
    args = [_dev(u, "u"), _dev(delta, "delta"), _f32(A, "A"), _dev(B, "B"), _dev(C, "C"),
            _f32(D, "D"), _f32(dt_bias, "dt_bias"), int(bool(delta_softplus)), _dev(y, "y"),
            batch, K, channels, L, N, in_dt, out_dt, layout, H, W]
    if workspace is not False:  # False: the entry point takes no workspace
        if workspace is None:
            need = vmb_scan_workspace_bytes(mean_variant, batch, K, channels, L, N, layout)
            workspace = (torch.empty(max(need, 1), dtype=torch.uint8, device=delta.device)
                         if need else None)
        ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
        args += [_dev(workspace, "workspace"), ws_bytes]
    if options is not None:
        args.append(int(options))
    status = getattr(lib, name)(*args, _stream(stream))
    _check(status, name)
    return y


def vmb_selective_scan_fwd(u, delta, A, B, C, D, dt_bias, delta_softplus, y,
                           layout: int = VMB_LAYOUT_SEQ, workspace=None, stream=None):
    """Full selective scan; shapes as in include/vmb.h. Returns y."""
    return _scan("vmb_selective_scan_fwd", False, u, delta, A, B, C, D, dt_bias, delta_softplus,
                 y, layout, workspace, stream)


def vmb_selective_scan_fwd_ex(u, delta, A, B, C, D, dt_bias, delta_softplus, y, options: int,
                              layout: int = VMB_LAYOUT_SEQ, workspace=None, stream=None):
    """Full selective scan with options (VMB_SCAN_* bits). Returns y."""
    return _scan("vmb_selective_scan_fwd_ex", False, u, delta, A, B, C, D, dt_bias,
                 delta_softplus, y, layout, workspace, stream, options=options)


def vmb_mean_scan_fwd(u, delta, A, B, C, D, dt_bias, delta_softplus, y,
                      layout: int = VMB_LAYOUT_SEQ, workspace=None, stream=None):
    """VMeanba channel-mean scan; shapes as in include/vmb.h. Returns y."""
    return _scan("vmb_mean_scan_fwd", True, u, delta, A, B, C, D, dt_bias, delta_softplus,
                 y, layout, workspace, stream)


def vmb_mean_scan_fwd_ex(u, delta, A, B, C, D, dt_bias, delta_softplus, y, options: int,
                         layout: int = VMB_LAYOUT_SEQ, workspace=None, stream=None):
    """VMeanba scan with a reading of T chosen by ``options`` (VMB_MEAN_* bits;
    y is [batch, K, 1, L] with VMB_MEAN_NO_BROADCAST). Returns y."""
    return _scan("vmb_mean_scan_fwd_ex", True, u, delta, A, B, C, D, dt_bias, delta_softplus,
                 y, layout, workspace, stream, options=options)


def vmb_mean_scan_fwd_noalloc(u, delta, A, B, C, D, dt_bias, delta_softplus, y,
                              layout: int = VMB_LAYOUT_SEQ, stream=None):
    """VMeanba scan without a workspace argument (the library's fixed 8 MiB
    per-device scratch array; calls overlapping on one GPU race). Returns y."""
    return _scan("vmb_mean_scan_fwd_noalloc", True, u, delta, A, B, C, D, dt_bias,
                 delta_softplus, y, layout, False, stream)


def vmb_mean_scan_status(workspace: torch.Tensor, stream=None) -> int:
    """Completion status of the last mean-scan call that used ``workspace``
    (waits for the stream): VMB_OK, VMB_ERR_INCOMPLETE (a bounded wait gave up,
    outputs partly NaN) or VMB_ERR_WORKSPACE (no call recorded). Returns the
    code; other codes raise."""
    status = int(load_library().vmb_mean_scan_status(_dev(workspace, "workspace"),
                                                     _stream(stream)))
    if status not in (VMB_OK, VMB_ERR_WORKSPACE, VMB_ERR_INCOMPLETE):
        raise VmbError(status, "vmb_mean_scan_status")
    return status


def vmb_ss2d_projections(u: torch.Tensor, W: torch.Tensor, W_dt: Optional[torch.Tensor],
                         delta: torch.Tensor, B: torch.Tensor, C: torch.Tensor,
                         stream=None):
    """Selection projections of eq. 6: u [batch, K, channels, L] ->
    delta [batch, K, channels, L], B, C [batch, K, N, L]; W float32
    [K, R + 2N, channels], W_dt float32 [K, channels, R] or None (R = 1,
    broadcast). Returns (delta, B, C)."""
    lib = load_library()
    batch, K, channels, L = u.shape
    N = B.shape[2]
    R = W.shape[1] - 2 * N
    if tuple(W.shape) != (K, R + 2 * N, channels):
        raise ValueError(f"W shape {tuple(W.shape)} != {(K, R + 2 * N, channels)}")
    if W_dt is not None and tuple(W_dt.shape) != (K, channels, R):
        raise ValueError(f"W_dt shape {tuple(W_dt.shape)} != {(K, channels, R)}")
    if tuple(delta.shape) != tuple(u.shape):
        raise ValueError("delta must have the shape of u")
    for t, nm in ((B, "B"), (C, "C")):
        if tuple(t.shape) != (batch, K, N, L):
            raise ValueError(f"{nm} shape {tuple(t.shape)} != {(batch, K, N, L)}")
    for t, nm in ((delta, "delta"), (B, "B"), (C, "C")):
        if t.dtype != u.dtype:
            raise ValueError(f"{nm} must have the dtype of u")
    _check(lib.vmb_ss2d_projections(_dev(u, "u"), _f32(W, "W"), _f32(W_dt, "W_dt"),
                                    _dev(delta, "delta"), _dev(B, "B"), _dev(C, "C"), batch, K,
                                    channels, L, N, R, _dtype(u, "u"), _stream(stream)),
           "vmb_ss2d_projections")
    return delta, B, C


def vmb_ss2d_out_norm(y: torch.Tensor, z: Optional[torch.Tensor], gamma: Optional[torch.Tensor],
                      beta: Optional[torch.Tensor], eps: float, out: torch.Tensor, stream=None):
    """Channel layer normalisation per pixel, then the SiLU gate by z (None:
    no gate): y, z, out [batch, channels, H, W] (or [batch, channels, P]) of
    one dtype; gamma, beta float32 [channels] or None. Returns out."""
    lib = load_library()
    batch, channels = y.shape[0], y.shape[1]
    P = y.numel() // max(1, batch * channels)
    if y.dim() < 3 or batch * channels * P != y.numel():
        raise ValueError(f"y shape {tuple(y.shape)} is not [batch, channels, ...]")
    for t, nm in ((z, "z"), (out, "out")):
        if t is not None and (tuple(t.shape) != tuple(y.shape) or t.dtype != y.dtype):
            raise ValueError(f"{nm} must have the shape and dtype of y")
    for t, nm in ((gamma, "gamma"), (beta, "beta")):
        if t is not None and t.numel() != channels:
            raise ValueError(f"{nm} must have {channels} elements")
    _check(lib.vmb_ss2d_out_norm(_dev(y, "y"), _dev(z, "z"), _f32(gamma, "gamma"),
                                 _f32(beta, "beta"), float(eps), _dev(out, "out"), batch,
                                 channels, P, _dtype(y, "y"), _stream(stream)),
           "vmb_ss2d_out_norm")
    return out


def vmb_discrete_scan(abar: torch.Tensor, bu: torch.Tensor, C: torch.Tensor,
                      skip: Optional[torch.Tensor], y: torch.Tensor, stream=None) -> torch.Tensor:
    """One-state scan on materialised inputs (float32).

    abar, bu, skip, y: [batch, channels, L] (skip may be None); C: [batch, L].
    h_t = abar_t h_{t-1} + bu_t, y_t = C_t h_t + skip_t.
    """
    lib = load_library()
    batch, channels, L = abar.shape
    for t, name in ((bu, "bu"), (y, "y")) + (((skip, "skip"),) if skip is not None else ()):
        if tuple(t.shape) != (batch, channels, L):
            raise ValueError(f"{name} shape {tuple(t.shape)} != {(batch, channels, L)}")
    if tuple(C.shape) != (batch, L):
        raise ValueError(f"C shape {tuple(C.shape)} != {(batch, L)}")
    _check(lib.vmb_discrete_scan(_f32(abar, "abar"), _f32(bu, "bu"), _f32(C, "C"),
                                 _f32(skip, "skip"), _f32(y, "y"), batch, channels, L,
                                 _stream(stream)), "vmb_discrete_scan")
    return y


def vmb_channel_mean(x: torch.Tensor, xm: torch.Tensor, stream=None) -> torch.Tensor:
    """T of eq. 9: x [batch, channels, L] -> xm [batch, L], the channel mean (float32)."""
    lib = load_library()
    batch, channels, L = x.shape
    if tuple(xm.shape) != (batch, L):
        raise ValueError(f"xm shape {tuple(xm.shape)} != {(batch, L)}")
    _check(lib.vmb_channel_mean(_f32(x, "x"), _f32(xm, "xm"), batch, channels, L,
                                _stream(stream)), "vmb_channel_mean")
    return xm
