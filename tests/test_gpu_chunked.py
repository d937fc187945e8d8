"""Full scan on long sequences (the positions-over-lanes kernel): chunk and
run boundaries, channel-group tails, dtypes and the 2-D layout."""
import numpy as np
import pytest
import torch

import workloads
from paper_2412_16602_amd import vmb
from gpu_util import BF16_TOL, FP32_TOL, assert_close, log, oracle_seq, run_scan, to_f64
from test_gpu_scan import merged_oracle

pytestmark = pytest.mark.gpu


def shape(b, H, W, c, dtype="f32", seed=0):
    return workloads.custom_shape(b, H, W, c, 16, dtype, seed, True)


# L chosen around the run / wave / chunk boundaries (runs of 13 or 16 positions,
# 64 lanes per wave, 1, 2 or 4 waves per channel)
LENGTHS = [417, 500, 512, 831, 832, 833, 1663, 1664, 1665, 3136, 3327, 3328, 3329, 4096, 4097,
           8193]


@pytest.mark.parametrize("L", LENGTHS)
def test_lengths(L):
    log(f"chunked full L={L}")
    inp = workloads.make_inputs(shape(1, 1, L, 5, seed=L), "seq", d_value=0.0)
    got = to_f64(run_scan(inp, "full", "seq"))
    ref = oracle_seq(inp, "full", "seq")
    assert_close(got, ref, **FP32_TOL, what=f"chunked L={L}")


@pytest.mark.parametrize("channels", [1, 2, 3, 4, 7, 13])
def test_channel_group_tails(channels):
    log(f"chunked full channels={channels}")
    inp = workloads.make_inputs(shape(2, 40, 50, channels, seed=100 + channels), "seq")
    got = to_f64(run_scan(inp, "full", "seq"))
    ref = oracle_seq(inp, "full", "seq")
    assert_close(got, ref, **FP32_TOL, what=f"chunked channels={channels}")


# bf16 rows of 16-byte pieces (L % 8 == 0), of 4-byte pieces (L even) and of
# odd length (not on 4-byte boundaries: the lane-per-channel kernel takes them)
@pytest.mark.parametrize("out", ["bf16", "f32"])
@pytest.mark.parametrize("H,W", [(32, 64), (33, 62), (33, 61)])
def test_bf16(out, H, W):
    log(f"chunked full bf16 {H}x{W} -> {out}")
    inp = workloads.make_inputs(shape(1, H, W, 6, "bf16", seed=200 + W), "seq")
    y = run_scan(inp, "full", "seq", out_dtype=torch.bfloat16 if out == "bf16" else torch.float32)
    ref = oracle_seq(inp, "full", "seq")
    assert_close(to_f64(y), ref, **(BF16_TOL if out == "bf16" else FP32_TOL), what=f"bf16->{out}")


# one chunk (56x56, 29x31, 1x700, 700x1) and several (64x130; 61x67 and 57x64 with whole and
# partial row-major runs read as vectors, the column-major directions from the plane copies)
@pytest.mark.parametrize("H,W", [(56, 56), (29, 31), (1, 700), (700, 1), (64, 130), (61, 67), (57, 64)])
def test_2d_layout(H, W):
    log(f"chunked full 2d {H}x{W}")
    inp = workloads.make_inputs(shape(1, H, W, 4, seed=H * 1000 + W), "2d")
    got = to_f64(run_scan(inp, "full", "2d"))
    ref, scale = merged_oracle(inp, "full")
    assert_close(got, ref, rtol=FP32_TOL["rtol"], atol=4 * FP32_TOL["atol"], scale=scale,
                 what=f"2d {H}x{W}")


# bf16 inputs in the 2-D layout, one chunk and several
@pytest.mark.parametrize("H,W", [(40, 50), (60, 70)])
def test_2d_layout_bf16(H, W):
    log(f"chunked full 2d bf16 {H}x{W}")
    inp = workloads.make_inputs(shape(1, H, W, 3, "bf16", seed=H * 1000 + W + 7), "2d")
    got = to_f64(run_scan(inp, "full", "2d", out_dtype=torch.float32))
    ref, scale = merged_oracle(inp, "full")
    assert_close(got, ref, rtol=FP32_TOL["rtol"], atol=4 * FP32_TOL["atol"], scale=scale,
                 what=f"2d bf16 {H}x{W}")


def test_softplus_off_and_no_bias():
    log("chunked full softplus off")
    inp = workloads.make_inputs(shape(1, 20, 60, 3, seed=300), "seq")
    delta = (np.abs(inp.delta) * 0.05 + 1e-3).astype(np.float32)
    got = to_f64(run_scan(inp, "full", "seq", softplus=False, use_bias=False, delta=delta))
    ref = oracle_seq(inp, "full", "seq", softplus=False, use_bias=False, delta=delta)
    assert_close(got, ref, **FP32_TOL, what="softplus off")


def test_2d_map_beyond_the_merge_grid_is_refused():
    # a 1 x 2^21 map has 65536 tiles of 32 columns, more than the merge and
    # transpose kernels' grid takes: the call returns VMB_ERR_UNSUPPORTED from
    # its host checks and writes nothing
    log("chunked full 2d 1x2097152 refused")
    W = 1 << 21
    f = torch.float32
    x = torch.zeros(1, 1, 1, W, dtype=f, device="cuda")
    delta = torch.zeros(1, 4, 1, W, dtype=f, device="cuda")
    Bm = torch.zeros(1, 4, 16, W, dtype=f, device="cuda")
    A = -torch.ones(4, 16, dtype=f, device="cuda")
    y = torch.full((1, 1, 1, W), 7.0, dtype=f, device="cuda")
    with pytest.raises(vmb.VmbError) as err:
        vmb.vmb_selective_scan_fwd(x, delta, A, Bm, Bm, None, None, True, y,
                                   layout=vmb.VMB_LAYOUT_2D)
    assert err.value.status == vmb.VMB_ERR_UNSUPPORTED
    torch.cuda.synchronize()
    assert bool((y == 7.0).all())
