"""Full scan on short sequences (whole sequences in segments of 16 or 32 lanes
of one wave, N = 16): segment and run boundaries, channel-slot tails, dtypes
and the 2-D layout."""
import numpy as np
import pytest
import torch

import workloads
from gpu_util import BF16_TOL, FP32_TOL, assert_close, log, oracle_seq, run_scan, to_f64
from test_gpu_scan import merged_oracle

pytestmark = pytest.mark.gpu


def shape(b, H, W, c, dtype="f32", seed=0):
    return workloads.custom_shape(b, H, W, c, 16, dtype, seed, True)


# segment shapes 16 x 4 (L <= 64), 16 x 13 (L <= 208), 32 x 13 (L <= 416)
LENGTHS = [1, 2, 15, 16, 17, 63, 64, 65, 100, 207, 208, 209, 300, 415, 416, 417, 500]


@pytest.mark.parametrize("L", LENGTHS)
def test_lengths(L):
    log(f"short full L={L}")
    inp = workloads.make_inputs(shape(1, 1, L, 5, seed=L), "seq", d_value=0.0)
    got = to_f64(run_scan(inp, "full", "seq"))
    ref = oracle_seq(inp, "full", "seq")
    assert_close(got, ref, **FP32_TOL, what=f"short L={L}")


# 32 channels per workgroup for 16-lane segments, 16 for 32-lane ones
@pytest.mark.parametrize("L", [49, 196, 300])
@pytest.mark.parametrize("channels", [1, 3, 15, 16, 17, 31, 32, 33, 70])
def test_channel_slot_tails(L, channels):
    log(f"short full L={L} channels={channels}")
    inp = workloads.make_inputs(shape(2, 1, L, channels, seed=100 + channels + L), "seq")
    got = to_f64(run_scan(inp, "full", "seq"))
    ref = oracle_seq(inp, "full", "seq")
    assert_close(got, ref, **FP32_TOL, what=f"short L={L} channels={channels}")


@pytest.mark.parametrize("out", ["bf16", "f32"])
@pytest.mark.parametrize("H,W", [(7, 7), (14, 14), (16, 20)])
def test_bf16(H, W, out):
    log(f"short full bf16 {H}x{W} -> {out}")
    inp = workloads.make_inputs(shape(2, H, W, 40, "bf16", seed=200 + H), "seq")
    y = run_scan(inp, "full", "seq", out_dtype=torch.bfloat16 if out == "bf16" else torch.float32)
    ref = oracle_seq(inp, "full", "seq")
    assert_close(to_f64(y), ref, **(BF16_TOL if out == "bf16" else FP32_TOL), what=f"bf16->{out}")


@pytest.mark.parametrize("H,W", [(7, 7), (14, 14), (1, 200), (200, 1), (13, 17), (20, 20)])
def test_2d_layout(H, W):
    log(f"short full 2d {H}x{W}")
    inp = workloads.make_inputs(shape(1, H, W, 36, seed=H * 1000 + W), "2d")
    got = to_f64(run_scan(inp, "full", "2d"))
    ref, scale = merged_oracle(inp, "full")
    assert_close(got, ref, rtol=FP32_TOL["rtol"], atol=4 * FP32_TOL["atol"], scale=scale,
                 what=f"2d {H}x{W}")


def test_softplus_off_and_no_bias():
    log("short full softplus off")
    inp = workloads.make_inputs(shape(1, 12, 12, 20, seed=300), "seq")
    delta = (np.abs(inp.delta) * 0.05 + 1e-3).astype(np.float32)
    got = to_f64(run_scan(inp, "full", "seq", softplus=False, use_bias=False, delta=delta))
    ref = oracle_seq(inp, "full", "seq", softplus=False, use_bias=False, delta=delta)
    assert_close(got, ref, **FP32_TOL, what="softplus off")
