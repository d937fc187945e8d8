"""The pooled reading of the VMeanba scan (VMB_MEAN_POOLED: T over all
K*channels sequences of an image, one scan per batch element, broadcast to
every direction and channel) against the fp64 oracle's pooled scan; both
layouts, fp32 and bf16, several lengths (chunk tails) and state counts."""
import numpy as np
import pytest
import torch

import oracle
import workloads
from gpu_util import BF16_TOL, FP32_TOL, assert_close, log, run_scan, to_f64
from paper_2412_16602_amd import vmb

pytestmark = pytest.mark.gpu


def shape(b, H, W, c, N, dtype="f32", seed=0):
    return workloads.custom_shape(b, H, W, c, N, dtype, seed, True)


def pooled_ref(inp, u=None, use_d=True, use_bias=True, softplus=True):
    u = inp.u if u is None else u
    return oracle.mean_scan_pooled(u, inp.delta, inp.A, inp.B, inp.C,
                                   inp.D if use_d else None,
                                   inp.dt_bias if use_bias else None, softplus)


def vary_params(inp):
    """A and D differing per channel (the generator's are channel-constant)."""
    import dataclasses
    c = np.arange(inp.A.shape[0], dtype=np.float64)
    A = (inp.A * (1.0 + 0.5 * np.modf(c * 0.37)[0])[:, None]).astype(np.float32)
    D = (inp.D * (0.5 + np.modf(c * 0.61)[0])).astype(np.float32)
    return dataclasses.replace(inp, A=A, D=D)


SEQ = [("b2_c24_L100_n16", shape(2, 10, 10, 24, 16, seed=81)),
       ("b1_c7_L65_n4", shape(1, 5, 13, 7, 4, seed=82)),
       ("b3_c5_L9_n1", shape(3, 3, 3, 5, 1, seed=83)),
       ("b1_c192_L3136_n16", shape(1, 56, 56, 192, 16, seed=84))]


@pytest.mark.parametrize("name,shp", SEQ, ids=[c[0] for c in SEQ])
def test_seq_f32(name, shp):
    log(f"pooled seq f32 {name}")
    inp = vary_params(workloads.make_inputs(shp, "seq"))
    y = to_f64(run_scan(inp, "mean", "seq", options=vmb.VMB_MEAN_POOLED))
    ref = pooled_ref(inp)
    b, K, Dc, L = y.shape
    assert_close(y, np.broadcast_to(ref[:, None, None, :], y.shape), **FP32_TOL,
                 what=f"pooled seq {name}")


@pytest.mark.parametrize("use_bias,use_d", [(False, True), (True, False)])
def test_optional_parameters(use_bias, use_d):
    log(f"pooled seq bias={use_bias} D={use_d}")
    inp = vary_params(workloads.make_inputs(shape(2, 6, 9, 12, 8, seed=85), "seq"))
    y = to_f64(run_scan(inp, "mean", "seq", options=vmb.VMB_MEAN_POOLED, use_bias=use_bias,
                        use_d=use_d))
    ref = pooled_ref(inp, use_d=use_d, use_bias=use_bias)
    assert_close(y, np.broadcast_to(ref[:, None, None, :], y.shape), **FP32_TOL,
                 what="pooled optional parameters")


@pytest.mark.parametrize("out", ["bf16", "f32"])
def test_seq_bf16(out):
    log(f"pooled seq bf16 -> {out}")
    inp = workloads.make_inputs(shape(2, 8, 12, 20, 16, "bf16", seed=86), "seq")
    y = run_scan(inp, "mean", "seq", options=vmb.VMB_MEAN_POOLED,
                 out_dtype=torch.bfloat16 if out == "bf16" else torch.float32)
    ref = pooled_ref(inp)
    got = to_f64(y)
    assert_close(got, np.broadcast_to(ref[:, None, None, :], got.shape),
                 **(BF16_TOL if out == "bf16" else FP32_TOL), what=f"pooled bf16 -> {out}")


TWO_D = [("7x7_c32_n4", shape(1, 7, 7, 32, 4, seed=87)),
         ("5x9_c3_n16", shape(2, 5, 9, 3, 16, seed=88)),
         ("56x56_c192_n16", shape(1, 56, 56, 192, 16, seed=89))]


@pytest.mark.parametrize("name,shp", TWO_D, ids=[c[0] for c in TWO_D])
def test_2d_f32(name, shp):
    log(f"pooled 2d f32 {name}")
    inp = vary_params(workloads.make_inputs(shp, "2d"))
    got = to_f64(run_scan(inp, "mean", "2d", options=vmb.VMB_MEAN_POOLED))
    u = oracle.cross_scan(inp.x)
    ref_seq = pooled_ref(inp, u=u)  # [b, L]
    b, Dc = got.shape[0], got.shape[1]
    seq = np.ascontiguousarray(np.broadcast_to(ref_seq[:, None, None, :], (b, 4, Dc, shp.L)))
    ref = oracle.cross_merge(seq, shp.H, shp.W, "f64")
    scale = oracle.cross_merge(np.abs(seq), shp.H, shp.W, "f64")
    assert_close(got, ref, rtol=FP32_TOL["rtol"], atol=4 * FP32_TOL["atol"], scale=scale,
                 what=f"pooled 2d {name}")


def test_pooled_with_other_bits_raises():
    inp = workloads.make_inputs(shape(1, 4, 4, 8, 4, seed=90), "seq")
    for other in (vmb.VMB_MEAN_SKIP_PER_CHANNEL, vmb.VMB_MEAN_RAW, vmb.VMB_MEAN_NO_BROADCAST):
        with pytest.raises(vmb.VmbError):
            run_scan(inp, "mean", "seq", options=vmb.VMB_MEAN_POOLED | other)
