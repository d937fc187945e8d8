"""VMeanba scan on long sequences: many chunks (separate carry pass), chunk
boundaries that do not align with the 64-position finish blocks, 2-D layout."""
import pytest
import torch

import workloads
from gpu_util import FP32_TOL, assert_close, log, oracle_seq, run_scan, to_f64
from test_gpu_scan import merged_oracle

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("L,channels,batch", [(2049, 8, 1), (3136, 5, 1), (4097, 3, 2),
                                              (8193, 4, 1), (65536, 2, 1)])
def test_mean_long(L, channels, batch):
    log(f"mean long L={L} channels={channels} batch={batch}")
    shp = workloads.custom_shape(batch, 1, L, channels, 16, "f32", L + channels, True)
    inp = workloads.make_inputs(shp, "seq", d_value=0.0)
    got = to_f64(run_scan(inp, "mean", "seq"))
    ref = oracle_seq(inp, "mean", "seq")
    assert_close(got, ref, **FP32_TOL, what=f"mean L={L}")


# 64x130 and 97x101 (L > 6144) take the 32 x 32 tile transpose of the planes;
# 97x101 has ragged tiles at both edges and L % 4 != 0
@pytest.mark.parametrize("H,W,batch", [(64, 130, 1), (56, 56, 1), (97, 101, 2)])
def test_mean_2d_long(H, W, batch):
    log(f"mean 2d {H}x{W} batch={batch}")
    shp = workloads.custom_shape(batch, H, W, 6, 16, "f32", H + W, True)
    inp = workloads.make_inputs(shp, "2d")
    got = to_f64(run_scan(inp, "mean", "2d"))
    ref, scale = merged_oracle(inp, "mean")
    assert_close(got, ref, rtol=FP32_TOL["rtol"], atol=4 * FP32_TOL["atol"], scale=scale,
                 what=f"mean 2d {H}x{W}")


# bf16 planes beyond LDS (the transpose in bf16), fp32 output at the fp32 bound:
# the bf16 inputs are exact values the oracle reads as they are
def test_mean_2d_long_bf16():
    H, W = 72, 100
    log(f"mean 2d bf16 {H}x{W}")
    shp = workloads.custom_shape(1, H, W, 5, 16, "bf16", 7, True)
    inp = workloads.make_inputs(shp, "2d")
    got = to_f64(run_scan(inp, "mean", "2d", out_dtype=torch.float32))
    ref, scale = merged_oracle(inp, "mean")
    assert_close(got, ref, rtol=FP32_TOL["rtol"], atol=4 * FP32_TOL["atol"], scale=scale,
                 what=f"mean 2d bf16 {H}x{W}")
