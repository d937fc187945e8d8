"""Helpers shared by the GPU parity tests: device upload, tolerance checks,
and one call of the HIP path through the C ABI binding."""
from __future__ import annotations

import sys

import numpy as np
import torch

import oracle
import workloads
from paper_2412_16602_amd import vmb

# Tolerances: |got - ref| <= atol + rtol * |ref| elementwise, ref = fp64 oracle.
FP32_TOL = dict(rtol=1e-4, atol=1e-5)
BF16_TOL = dict(rtol=2e-2, atol=1e-4)


def dev():
    return torch.device("cuda:0")


def log(msg: str):
    print(msg, flush=True)
    sys.stdout.flush()


def upload_f32(a):
    return None if a is None else torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(dev())


def upload_stream(inp: workloads.Inputs, name: str):
    """Upload one streamed tensor (x, u, delta, B, C) in the workload dtype."""
    a = getattr(inp, {"B": "B", "C": "C"}.get(name, name))
    if inp.shape.dtype == "bf16":
        bits = inp.bits[name]
        return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).to(dev()).view(torch.bfloat16)
    return upload_f32(a)


def to_f64(t: torch.Tensor) -> np.ndarray:
    t = t.detach()
    if t.dtype == torch.bfloat16:
        t = t.float()
    return t.cpu().numpy().astype(np.float64)


def excess(got, ref, rtol, atol, scale=None):
    """max over elements of |got-ref| - (atol + rtol*|scale|) (<= 0 passes)."""
    scale = np.abs(ref) if scale is None else scale
    return float(np.max(np.abs(got - ref) - (atol + rtol * scale))) if got.size else -1.0


def assert_close(got, ref, rtol, atol, what="", scale=None):
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert got.shape == ref.shape, (got.shape, ref.shape)
    assert np.all(np.isfinite(got)), f"{what}: non-finite output"
    sc = np.abs(ref) if scale is None else scale
    bad = np.abs(got - ref) > (atol + rtol * sc)
    if bad.any():
        idx = np.unravel_index(np.argmax(np.abs(got - ref) - (atol + rtol * sc)), got.shape)
        raise AssertionError(f"{what}: {int(bad.sum())}/{got.size} outside tol (rtol={rtol}, "
                             f"atol={atol}); worst at {idx}: got {got[idx]!r} ref {ref[idx]!r}")


def run_scan(inp: workloads.Inputs, variant: str, layout: str, out_dtype=None, softplus=True,
             use_bias=True, use_d=True, delta=None, workspace=None, options=None):
    """One call of vmb_selective_scan_fwd / vmb_mean_scan_fwd on cuda:0
    (vmb_mean_scan_fwd_ex when ``options`` is given)."""
    s = inp.shape
    lay = vmb.VMB_LAYOUT_2D if layout == "2d" else vmb.VMB_LAYOUT_SEQ
    u = upload_stream(inp, "x" if layout == "2d" else "u")
    if delta is None:
        dl = upload_stream(inp, "delta")
    else:
        dl = upload_f32(delta) if s.dtype == "f32" else delta
    B, C = upload_stream(inp, "B"), upload_stream(inp, "C")
    A = upload_f32(inp.A)
    D = upload_f32(inp.D) if use_d else None
    bias = upload_f32(inp.dt_bias) if use_bias else None
    if out_dtype is None:
        out_dtype = torch.bfloat16 if s.dtype == "bf16" else torch.float32
    b = inp.delta.shape[0]
    shape = (b, s.channels, s.H, s.W) if layout == "2d" else tuple(inp.delta.shape)
    if options is not None and options & vmb.VMB_MEAN_NO_BROADCAST and layout == "seq":
        shape = shape[:2] + (1,) + shape[3:]
    y = torch.empty(shape, dtype=out_dtype, device=dev())
    if options is not None and variant == "full":
        vmb.vmb_selective_scan_fwd_ex(u, dl, A, B, C, D, bias, softplus, y, options, layout=lay,
                                      workspace=workspace)
    elif options is not None:
        vmb.vmb_mean_scan_fwd_ex(u, dl, A, B, C, D, bias, softplus, y, options, layout=lay,
                                 workspace=workspace)
    else:
        fn = vmb.vmb_selective_scan_fwd if variant == "full" else vmb.vmb_mean_scan_fwd
        fn(u, dl, A, B, C, D, bias, softplus, y, layout=lay, workspace=workspace)
    torch.cuda.synchronize()
    return y


def oracle_seq(inp: workloads.Inputs, variant: str, layout: str, softplus=True, use_bias=True,
               use_d=True, delta=None, sel=None, options=0):
    """fp64 oracle on the same inputs (per-direction sequence outputs);
    ``options`` are the oracle's mean-scan reading bits."""
    u = oracle.cross_scan(inp.x) if layout == "2d" else inp.u
    dl = inp.delta if delta is None else delta
    args = (u, dl, inp.A, inp.B, inp.C, inp.D if use_d else None,
            inp.dt_bias if use_bias else None, softplus)
    if variant == "full":
        return oracle.full_scan(*args, sel=sel, options=options)
    return oracle.mean_scan(*args, sel=sel, options=options)
