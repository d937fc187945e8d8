"""The channel normalisation and SiLU gate after the cross-merge
(vmb_ss2d_out_norm) against the fp64 oracle: the stage shapes, tiles of 16
flattened pixels crossing image boundaries, a mean offset far from zero,
one channel (zero variance), one pixel per image, no gate / no affine, bf16,
and the whole SS2D output step (2-D scan, then the norm)."""
import numpy as np
import pytest
import torch

import oracle
import workloads
from gpu_util import BF16_TOL, FP32_TOL, assert_close, dev, log, to_f64, upload_f32
from paper_2412_16602_amd import vmb

pytestmark = pytest.mark.gpu


def upload(a, dtype):
    if dtype == "bf16":
        r, bits = workloads.bf16_round(np.ascontiguousarray(a, dtype=np.float32))
        t = torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).to(dev()).view(torch.bfloat16)
        return r.astype(np.float64), t
    a = np.ascontiguousarray(a, dtype=np.float32)
    return a.astype(np.float64), upload_f32(a)


def run(y, z, g, be, eps, dtype="f32"):
    yr, yt = upload(y, dtype)
    zr, zt = (None, None) if z is None else upload(z, dtype)
    out = torch.empty_like(yt)
    vmb.vmb_ss2d_out_norm(yt, zt, None if g is None else upload_f32(g),
                          None if be is None else upload_f32(be), eps, out)
    torch.cuda.synchronize()
    ref = oracle.out_norm_gate(yr, zr, g, be, eps)
    return to_f64(out), ref


CASES = [  # batch, channels, pixels
    ("stage1_1x192x3136", 1, 192, 3136),
    ("stage4_32x1536x49", 32, 1536, 49),
    ("b3_c70_p45", 3, 70, 45),       # 135 pixels: tiles straddle images
    ("b2_c17_p1", 2, 17, 1),         # one pixel per image
    ("b5_c1_p20", 5, 1, 20),         # one channel: zero variance, out = beta
    # tile widths: 16 pixels from 8192 pixels or with few channels, 8 from
    # 4096 pixels (and 512 channels), 4 below (and 1024 channels)
    ("tile16_b2_c40_p4500", 2, 40, 4500),
    ("tile8_b1_c600_p5000", 1, 600, 5000),
    ("tile4_b3_c1100_p300", 3, 1100, 300),
]


@pytest.mark.parametrize("gate", [True, False])
@pytest.mark.parametrize("name,b,c,p", CASES, ids=[c[0] for c in CASES])
def test_out_norm_f32(name, b, c, p, gate):
    log(f"out norm {name} gate={gate}")
    rng = np.random.default_rng(b * 1000 + c + p)
    y = rng.standard_normal((b, c, p)).astype(np.float32)
    z = (rng.standard_normal((b, c, p)) * 2).astype(np.float32) if gate else None
    g = (1 + 0.1 * rng.standard_normal(c)).astype(np.float32)
    be = (0.1 * rng.standard_normal(c)).astype(np.float32)
    got, ref = run(y, z, g, be, 1e-5)
    assert_close(got, ref, **FP32_TOL, what=f"out norm {name}")


def test_out_norm_offset_mean():
    """y = 10 + N(0, 1): the centred second pass keeps the variance exact."""
    log("out norm offset mean")
    rng = np.random.default_rng(5)
    y = (10.0 + rng.standard_normal((2, 384, 100))).astype(np.float32)
    got, ref = run(y, None, None, None, 1e-6)
    assert_close(got, ref, **FP32_TOL, what="offset mean")


def test_out_norm_no_affine_eps0():
    log("out norm no affine, eps 0")
    rng = np.random.default_rng(6)
    y = rng.standard_normal((4, 96, 49)).astype(np.float32)
    z = rng.standard_normal((4, 96, 49)).astype(np.float32)
    got, ref = run(y, z, None, None, 0.0)
    assert_close(got, ref, **FP32_TOL, what="no affine")


# tiles 32 (16384 pixels), 16 (few channels), 8 (2048 channels, 392 pixels)
@pytest.mark.parametrize("b,c,p", [(2, 96, 196), (1, 24, 9000), (4, 24, 4100), (2, 2048, 196)])
def test_out_norm_bf16(b, c, p):
    log(f"out norm bf16 {b}x{c}x{p}")
    rng = np.random.default_rng(7 + p)
    y = rng.standard_normal((b, c, p))
    z = rng.standard_normal((b, c, p))
    g = (1 + 0.1 * rng.standard_normal(c)).astype(np.float32)
    got, ref = run(y, z, g, None, 1e-5, dtype="bf16")
    assert_close(got, ref, **BF16_TOL, what="bf16")


def test_out_norm_deterministic():
    rng = np.random.default_rng(8)
    y = upload_f32(rng.standard_normal((3, 200, 77)).astype(np.float32))
    a, b = torch.empty_like(y), torch.empty_like(y)
    vmb.vmb_ss2d_out_norm(y, None, None, None, 1e-5, a)
    vmb.vmb_ss2d_out_norm(y, None, None, None, 1e-5, b)
    torch.cuda.synchronize()
    assert torch.equal(a, b)


def test_ss2d_then_out_norm():
    """The SS2D output step: the 2-D full scan (cross-scan, scan, merge) then
    the norm, against the oracle's merged scan then its norm. The scan's
    error bound e (4 atol + rtol times the merge of |y_k|) reaches the
    normalised output at most as 2 max(e) / std of each pixel, times gamma."""
    from test_gpu_scan import merged_oracle

    log("ss2d then out norm, 14x14 c96")
    shp = workloads.custom_shape(2, 14, 14, 96, 16, "f32", 9, True)
    inp = workloads.make_inputs(shp, "2d")
    ref_y, scale = merged_oracle(inp, "full")
    lay = vmb.VMB_LAYOUT_2D
    ws_n = vmb.vmb_scan_workspace_bytes(False, 2, 4, 96, 196, 16, lay)
    ws = torch.empty(max(ws_n, 1), dtype=torch.uint8, device=dev())
    y = torch.empty((2, 96, 14, 14), device=dev())
    vmb.vmb_selective_scan_fwd(upload_f32(inp.x), upload_f32(inp.delta), upload_f32(inp.A),
                               upload_f32(inp.B), upload_f32(inp.C), upload_f32(inp.D),
                               upload_f32(inp.dt_bias), True, y, layout=lay, workspace=ws)
    rng = np.random.default_rng(10)
    z = rng.standard_normal((2, 96, 14, 14)).astype(np.float32)
    out = torch.empty_like(y)
    vmb.vmb_ss2d_out_norm(y, upload_f32(z), None, None, 1e-5, out)
    torch.cuda.synchronize()
    ref_y = ref_y.reshape(2, 96, 196)
    ref = oracle.out_norm_gate(ref_y, z.reshape(2, 96, 196).astype(np.float64), eps=1e-5)
    e = 4 * FP32_TOL["atol"] + FP32_TOL["rtol"] * scale.reshape(2, 96, 196)
    std = ref_y.std(axis=1, keepdims=True)
    silu = np.abs(z.reshape(2, 96, 196) / (1 + np.exp(-z.reshape(2, 96, 196).astype(np.float64))))
    bound = 2 * e.max(axis=1, keepdims=True) / std * np.maximum(silu, 1.0) + 1e-5
    err = np.abs(to_f64(out).reshape(2, 96, 196) - ref)
    assert np.all(err <= bound), float((err / bound).max())
