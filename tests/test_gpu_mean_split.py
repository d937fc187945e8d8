"""VMeanba scan with the channels of a chunk split over several reduce
workgroups (few chunk-sequences: 7x7 and 14x14 maps, short sequences at small
batch), whose partial sums a combine pass adds: group counts from 4 to the
maximum 16, channel slices of unequal size, several chunks per sequence,
every reading option, bf16, the 2-D layout."""
import pytest
import torch

import oracle
import workloads
from gpu_util import BF16_TOL, FP32_TOL, assert_close, log, oracle_seq, run_scan, to_f64
from paper_2412_16602_amd import vmb
from test_gpu_scan import merged_oracle

pytestmark = pytest.mark.gpu


def groups(batch, channels, L, K=4):
    """The library's split rule, restated to check that a case splits."""
    wgs = -(-L // 64) * K * batch
    if wgs >= 160:
        return 1
    return max(1, min(-(-512 // wgs), 16, channels // 64))


def shape(b, H, W, c, dtype="f32", seed=0):
    return workloads.custom_shape(b, H, W, c, 16, dtype, seed, True)


SEQ = [("b2_7x7_c256", shape(2, 7, 7, 256, seed=81), 4),
       ("b1_L200_c1024", shape(1, 1, 200, 1024, seed=82), 16),
       ("b1_L130_c1000", shape(1, 1, 130, 1000, seed=83), 15),
       ("b1_L2000_c256", shape(1, 1, 2000, 256, seed=84), 4)]


@pytest.mark.parametrize("name,shp,g", SEQ, ids=[c[0] for c in SEQ])
def test_split_seq(name, shp, g):
    assert groups(shp.batch, shp.channels, shp.L) == g
    log(f"mean split seq {name} groups={g}")
    inp = workloads.make_inputs(shp, "seq")
    got = to_f64(run_scan(inp, "mean", "seq"))
    ref = oracle_seq(inp, "mean", "seq")
    assert_close(got, ref, **FP32_TOL, what=f"mean split {name}")


OPTS = {"skip1": (vmb.VMB_MEAN_SKIP_PER_CHANNEL, oracle.MEAN_SKIP_PER_CHANNEL),
        "raw": (vmb.VMB_MEAN_RAW, oracle.MEAN_RAW),
        "nobc": (vmb.VMB_MEAN_NO_BROADCAST, oracle.MEAN_NO_BROADCAST),
        "zoh": (vmb.VMB_SCAN_ZOH, oracle.ZOH)}


@pytest.mark.parametrize("opt", list(OPTS))
@pytest.mark.parametrize("name,shp,g", SEQ[:3], ids=[c[0] for c in SEQ[:3]])
def test_split_options(name, shp, g, opt):
    log(f"mean split {name} option {opt}")
    lib_opt, ora_opt = OPTS[opt]
    inp = workloads.make_inputs(shp, "seq")
    got = to_f64(run_scan(inp, "mean", "seq", options=lib_opt))
    ref = oracle_seq(inp, "mean", "seq", options=ora_opt)
    assert_close(got, ref, **FP32_TOL, what=f"mean split {name} {opt}")


@pytest.mark.parametrize("out", ["bf16", "f32"])
def test_split_bf16(out):
    shp = shape(2, 7, 7, 256, dtype="bf16", seed=85)
    assert groups(2, 256, 49) > 1
    log(f"mean split bf16 -> {out}")
    inp = workloads.make_inputs(shp, "seq")
    y = run_scan(inp, "mean", "seq", out_dtype=torch.bfloat16 if out == "bf16" else torch.float32)
    ref = oracle_seq(inp, "mean", "seq")
    assert_close(to_f64(y), ref, **(BF16_TOL if out == "bf16" else FP32_TOL), what=f"bf16->{out}")


@pytest.mark.parametrize("H,W,c,b", [(7, 7, 256, 2), (14, 14, 512, 1)])
def test_split_2d(H, W, c, b):
    assert groups(b, c, H * W) > 1
    log(f"mean split 2d {H}x{W} c{c} b{b}")
    inp = workloads.make_inputs(shape(b, H, W, c, seed=H + c), "2d")
    got = to_f64(run_scan(inp, "mean", "2d"))
    ref, scale = merged_oracle(inp, "mean")
    assert_close(got, ref, rtol=FP32_TOL["rtol"], atol=4 * FP32_TOL["atol"], scale=scale,
                 what=f"mean split 2d {H}x{W}")


def test_split_deterministic():
    inp = workloads.make_inputs(shape(1, 1, 200, 1024, seed=86), "seq")
    log("mean split deterministic")
    a = run_scan(inp, "mean", "seq")
    b = run_scan(inp, "mean", "seq")
    assert torch.equal(a, b)
