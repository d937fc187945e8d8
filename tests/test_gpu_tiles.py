"""Full scan on grids with many channel rows (channels over lanes, the 16
states over the four waves of a workgroup, positions in tiles of 16): tile
boundaries and the partial last tile, unaligned lengths, channel counts that
leave lanes idle, bf16 in / out, the 2-D layout, optional parameters, and
both sides of the row threshold that selects this path.

A and D are made to differ per channel (the generator's A rows and D are the
same for every channel), so a wrong channel index in either shows up."""
import dataclasses

import numpy as np
import pytest
import torch

import workloads
from gpu_util import BF16_TOL, FP32_TOL, assert_close, log, oracle_seq, run_scan, to_f64
from test_gpu_scan import merged_oracle

pytestmark = pytest.mark.gpu

MIN_ROWS = 16384  # batch * 4 * channels from which the tile path runs


def inputs(batch, H, W, channels, layout="seq", dtype="f32", seed=0, d_value=1.0):
    shp = workloads.custom_shape(batch, H, W, channels, 16, dtype, seed, True)
    inp = workloads.make_inputs(shp, layout, d_value=d_value)
    c = np.arange(4 * channels, dtype=np.float64)
    scale = 1.0 + 0.5 * np.modf(c * 0.37)[0]
    A = (inp.A * scale[:, None]).astype(np.float32)
    D = (inp.D * (0.5 + np.modf(c * 0.61)[0])).astype(np.float32)
    return dataclasses.replace(inp, A=A, D=D)


# partial last tile, L % 4 != 0 (element loads and stores), one tile, several
LENGTHS = [1, 3, 4, 15, 16, 17, 31, 33, 49, 50, 64, 100]


@pytest.mark.parametrize("L", LENGTHS)
def test_lengths(L):
    log(f"tiles full L={L}")
    inp = inputs(4, 1, L, 1024, seed=L)
    got = to_f64(run_scan(inp, "full", "seq"))
    ref = oracle_seq(inp, "full", "seq")
    assert_close(got, ref, **FP32_TOL, what=f"tiles L={L}")


@pytest.mark.parametrize("batch,channels", [(5, 1000), (4, 1025), (3, 1400), (4096, 1), (66, 63)])
def test_channel_tails(batch, channels):
    assert batch * 4 * channels >= MIN_ROWS
    log(f"tiles full batch={batch} channels={channels}")
    inp = inputs(batch, 1, 20, channels, seed=batch + channels)
    got = to_f64(run_scan(inp, "full", "seq"))
    ref = oracle_seq(inp, "full", "seq")
    assert_close(got, ref, **FP32_TOL, what=f"tiles channels={channels}")


@pytest.mark.parametrize("out", ["bf16", "f32"])
@pytest.mark.parametrize("L", [36, 50, 49])  # 49: odd, bf16 takes the other path
def test_bf16(L, out):
    log(f"tiles full bf16 L={L} -> {out}")
    inp = inputs(4, 1, L, 1024, dtype="bf16", seed=500 + L)
    y = run_scan(inp, "full", "seq", out_dtype=torch.bfloat16 if out == "bf16" else torch.float32)
    ref = oracle_seq(inp, "full", "seq")
    assert_close(to_f64(y), ref, **(BF16_TOL if out == "bf16" else FP32_TOL), what=f"bf16->{out}")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("H,W", [(7, 7), (5, 9), (14, 14)])
def test_2d_layout(H, W, dtype):
    log(f"tiles full 2d {H}x{W} {dtype}")
    inp = inputs(4, H, W, 1024, layout="2d", dtype=dtype, seed=H * 100 + W)
    got = to_f64(run_scan(inp, "full", "2d", out_dtype=torch.float32))
    ref, scale = merged_oracle(inp, "full")
    tol = BF16_TOL if dtype == "bf16" else FP32_TOL
    # fp32 output: the inputs are exact, only the fp32 arithmetic differs
    assert_close(got, ref, rtol=FP32_TOL["rtol"], atol=4 * FP32_TOL["atol"], scale=scale,
                 what=f"2d {H}x{W} {dtype}")
    del tol


@pytest.mark.parametrize("use_bias,use_d,softplus", [(False, True, True), (True, False, True),
                                                     (False, False, False)])
def test_optional_parameters(use_bias, use_d, softplus):
    log(f"tiles full bias={use_bias} D={use_d} softplus={softplus}")
    inp = inputs(4, 1, 40, 1024, seed=77)
    delta = None
    if not softplus:
        delta = (np.abs(inp.delta) * 0.05 + 1e-3).astype(np.float32)
    got = to_f64(run_scan(inp, "full", "seq", use_bias=use_bias, use_d=use_d, softplus=softplus,
                          delta=delta))
    ref = oracle_seq(inp, "full", "seq", use_bias=use_bias, use_d=use_d, softplus=softplus,
                     delta=delta)
    assert_close(got, ref, **FP32_TOL, what="optional parameters")


@pytest.mark.parametrize("channels", [1023, 1024])  # 16368 rows: other path; 16384: tiles
def test_row_threshold(channels):
    log(f"tiles threshold channels={channels}")
    inp = inputs(4, 1, 60, channels, seed=channels)
    got = to_f64(run_scan(inp, "full", "seq"))
    ref = oracle_seq(inp, "full", "seq")
    assert_close(got, ref, **FP32_TOL, what=f"threshold channels={channels}")


def test_deterministic():
    log("tiles deterministic")
    inp = inputs(4, 1, 33, 1024, seed=5)
    a = run_scan(inp, "full", "seq")
    b = run_scan(inp, "full", "seq")
    assert torch.equal(a, b)


def test_2d_long_gather():
    """L > 6144: the 2-D tile path reads directions 1 and 3 straight from the
    plane (no column-major copy); sampled channels against the oracle."""
    import oracle

    H, W, Dc = 80, 80, 4096  # L 6400, 16384 rows
    log(f"tiles full 2d gather {H}x{W} channels={Dc}")
    inp = inputs(1, H, W, Dc, layout="2d", seed=9)
    got = to_f64(run_scan(inp, "full", "2d"))
    ds = [0, 1, 63, 64, 2047, 4095]
    u = oracle.cross_scan(inp.x)
    rows = [k * Dc + d for k in range(4) for d in ds]
    seq = oracle.full_scan(u, inp.delta, inp.A, inp.B, inp.C, inp.D, inp.dt_bias, True,
                           sel=rows).reshape(1, 4, len(ds), H * W)
    seq = np.ascontiguousarray(seq)
    ref = oracle.cross_merge(seq, H, W, "f64")
    scale = oracle.cross_merge(np.abs(seq), H, W, "f64")
    assert_close(got[:, ds], ref, rtol=FP32_TOL["rtol"], atol=4 * FP32_TOL["atol"], scale=scale,
                 what="2d gather")
