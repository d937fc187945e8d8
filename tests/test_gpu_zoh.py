"""The zero-order-hold B-bar option (VMB_SCAN_ZOH: eq. 4's second line as
(Delta A)^-1 (exp(Delta A) - I) Delta B) of the full scan against the fp64
oracle's ZOH scan: the tile kernel (N = 16, any number of rows, tile
boundaries, bf16), the lane kernel (other N, and N = 16 below one tile), the
2-D layout; D = 0 cases show the B term alone. A and D differ per channel, and
the timescale reaches both sides of the series/direct switch at |Delta A| =
0.02 (softplus(dt_bias) spans 1e-3 .. 1e-1, A = -(n + 1) scaled per channel)."""
import dataclasses

import numpy as np
import pytest
import torch

import oracle
import workloads
from gpu_util import BF16_TOL, FP32_TOL, assert_close, log, oracle_seq, run_scan, to_f64
from paper_2412_16602_amd import vmb
from test_gpu_scan import merged_oracle

pytestmark = pytest.mark.gpu

LIB_ZOH, ORA_ZOH = vmb.VMB_SCAN_ZOH, oracle.ZOH  # set independently on each side


def inputs(b, H, W, c, N, layout="seq", dtype="f32", seed=0, d_value=1.0):
    shp = workloads.custom_shape(b, H, W, c, N, dtype, seed, True)
    inp = workloads.make_inputs(shp, layout, d_value=d_value)
    ch = np.arange(4 * c, dtype=np.float64)
    A = (inp.A * (1.0 + 0.5 * np.modf(ch * 0.37)[0])[:, None]).astype(np.float32)
    D = (inp.D * (0.5 + np.modf(ch * 0.61)[0])).astype(np.float32)
    return dataclasses.replace(inp, A=A, D=D)


CASES = [
    # tile kernel (N = 16, L >= 16): few rows, many rows, tails, odd lengths
    ("tiles_b1_c24_L100", dict(b=1, H=10, W=10, c=24, N=16)),
    ("tiles_b4_c1024_L40", dict(b=4, H=5, W=8, c=1024, N=16)),
    ("tiles_b2_c70_L33", dict(b=2, H=3, W=11, c=70, N=16)),
    ("tiles_b1_c8_L3136", dict(b=1, H=56, W=56, c=8, N=16)),
    # lane kernel: other N, and N = 16 below one tile
    ("lanes_n4_L49", dict(b=2, H=7, W=7, c=40, N=4)),
    ("lanes_n1_L60", dict(b=1, H=6, W=10, c=9, N=1)),
    ("lanes_n8_L200", dict(b=1, H=10, W=20, c=65, N=8)),
    ("lanes_n16_L9", dict(b=2, H=3, W=3, c=30, N=16)),
]


@pytest.mark.parametrize("dval", [1.0, 0.0])
@pytest.mark.parametrize("name,kw", CASES, ids=[c[0] for c in CASES])
def test_seq_f32(name, kw, dval):
    log(f"zoh full seq {name} D={dval}")
    inp = inputs(layout="seq", seed=len(name), d_value=dval, **kw)
    got = to_f64(run_scan(inp, "full", "seq", options=LIB_ZOH))
    ref = oracle_seq(inp, "full", "seq", options=ORA_ZOH)
    assert_close(got, ref, **FP32_TOL, what=f"zoh {name} D={dval}")


def test_zoh_differs_from_first_order():
    """The option changes the result by more than the tolerance (it is not a no-op)."""
    inp = inputs(1, 10, 10, 24, 16, seed=3, d_value=0.0)
    z = to_f64(run_scan(inp, "full", "seq", options=LIB_ZOH))
    e = to_f64(run_scan(inp, "full", "seq"))
    assert np.max(np.abs(z - e)) > 100 * (FP32_TOL["atol"] + FP32_TOL["rtol"] * np.max(np.abs(e)))


@pytest.mark.parametrize("out", ["bf16", "f32"])
@pytest.mark.parametrize("L", [48, 49])  # 49: odd, bf16 takes the lane kernel
def test_bf16(L, out):
    log(f"zoh full bf16 L={L} -> {out}")
    inp = inputs(2, 1, L, 40, 16, dtype="bf16", seed=600 + L)
    y = run_scan(inp, "full", "seq", options=LIB_ZOH,
                 out_dtype=torch.bfloat16 if out == "bf16" else torch.float32)
    ref = oracle_seq(inp, "full", "seq", options=ORA_ZOH)
    assert_close(to_f64(y), ref, **(BF16_TOL if out == "bf16" else FP32_TOL), what=f"bf16->{out}")


@pytest.mark.parametrize("H,W,c,N", [(7, 7, 32, 16), (14, 14, 1024, 16), (5, 9, 12, 4)])
def test_2d(H, W, c, N):
    log(f"zoh full 2d {H}x{W} c={c} N={N}")
    inp = inputs(2 if c < 1024 else 4, H, W, c, N, layout="2d", seed=H * 10 + N)
    got = to_f64(run_scan(inp, "full", "2d", options=LIB_ZOH))
    ref, scale = merged_oracle(inp, "full", options=ORA_ZOH)
    assert_close(got, ref, rtol=FP32_TOL["rtol"], atol=4 * FP32_TOL["atol"], scale=scale,
                 what=f"zoh 2d {H}x{W}")


# ---------------------------------------------------------------- under the mean (T of eq. 9)

MEAN_CASES = [
    ("b2_c24_L100_n16", dict(b=2, H=10, W=10, c=24, N=16)),
    ("b1_c7_L200_n4", dict(b=1, H=8, W=25, c=7, N=4)),
    ("b1_c5_L4500_n16", dict(b=1, H=1, W=4500, c=5, N=16)),  # 71 chunks: carry pass
    ("b3_c3_L9_n1", dict(b=3, H=3, W=3, c=3, N=1)),
]
MEAN_OPTS = {"main": (0, 0),
             "skip1": (vmb.VMB_MEAN_SKIP_PER_CHANNEL, oracle.MEAN_SKIP_PER_CHANNEL),
             "nobc": (vmb.VMB_MEAN_NO_BROADCAST, oracle.MEAN_NO_BROADCAST)}


@pytest.mark.parametrize("opt", list(MEAN_OPTS))
@pytest.mark.parametrize("name,kw", MEAN_CASES, ids=[c[0] for c in MEAN_CASES])
def test_mean_seq(name, kw, opt):
    log(f"zoh mean seq {name} {opt}")
    inp = inputs(layout="seq", seed=7 + len(name), **kw)
    lib_o, ora_o = MEAN_OPTS[opt]
    got = to_f64(run_scan(inp, "mean", "seq", options=LIB_ZOH | lib_o))
    ref = oracle_seq(inp, "mean", "seq", options=ORA_ZOH | ora_o)
    assert_close(got, ref, **FP32_TOL, what=f"zoh mean {name} {opt}")


def test_mean_bf16():
    log("zoh mean seq bf16")
    inp = inputs(2, 8, 12, 20, 16, dtype="bf16", seed=31)
    y = run_scan(inp, "mean", "seq", options=LIB_ZOH)
    ref = oracle_seq(inp, "mean", "seq", options=ORA_ZOH)
    assert_close(to_f64(y), ref, **BF16_TOL, what="zoh mean bf16")


@pytest.mark.parametrize("H,W,c,N", [(7, 7, 32, 4), (12, 10, 24, 16)])
def test_mean_2d(H, W, c, N):
    log(f"zoh mean 2d {H}x{W}")
    inp = inputs(2, H, W, c, N, layout="2d", seed=H + W)
    got = to_f64(run_scan(inp, "mean", "2d", options=LIB_ZOH))
    ref, scale = merged_oracle(inp, "mean", options=ORA_ZOH)
    assert_close(got, ref, rtol=FP32_TOL["rtol"], atol=4 * FP32_TOL["atol"], scale=scale,
                 what=f"zoh mean 2d {H}x{W}")


# positions-over-lanes kernel (N = 16, L > 416, few rows): 1, 2 and 4 waves per
# channel, several chunks (L > 3328)
CHUNKED = [("chunked_L500", dict(b=1, H=20, W=25, c=6, N=16)),
           ("chunked_L1000", dict(b=1, H=25, W=40, c=5, N=16)),
           ("chunked_L3136", dict(b=1, H=56, W=56, c=12, N=16)),
           ("chunked_L4000", dict(b=1, H=40, W=100, c=3, N=16))]


@pytest.mark.parametrize("name,kw", CHUNKED, ids=[c[0] for c in CHUNKED])
def test_chunked_seq(name, kw):
    log(f"zoh full {name}")
    inp = inputs(layout="seq", seed=11 + len(name), **kw)
    got = to_f64(run_scan(inp, "full", "seq", options=LIB_ZOH))
    ref = oracle_seq(inp, "full", "seq", options=ORA_ZOH)
    assert_close(got, ref, **FP32_TOL, what=f"zoh {name}")


def test_chunked_bf16_and_2d():
    log("zoh full chunked bf16 seq, f32 2-D")
    inp = inputs(1, 28, 28, 8, 16, dtype="bf16", seed=21)
    y = run_scan(inp, "full", "seq", options=LIB_ZOH)
    ref = oracle_seq(inp, "full", "seq", options=ORA_ZOH)
    assert_close(to_f64(y), ref, **BF16_TOL, what="zoh chunked bf16")
    inp = inputs(1, 30, 30, 6, 16, layout="2d", seed=22)
    got = to_f64(run_scan(inp, "full", "2d", options=LIB_ZOH))
    ref, scale = merged_oracle(inp, "full", options=ORA_ZOH)
    assert_close(got, ref, rtol=FP32_TOL["rtol"], atol=4 * FP32_TOL["atol"], scale=scale,
                 what="zoh chunked 2d")
