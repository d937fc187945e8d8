"""Full and VMeanba scans on the GPU against the fp64 oracle (small and
ragged shapes, every dtype combination, both layouts, degenerate sizes)."""
import numpy as np
import pytest
import torch

import oracle
import workloads
from gpu_util import (BF16_TOL, FP32_TOL, assert_close, log, oracle_seq, run_scan, to_f64,
                      upload_f32)

pytestmark = pytest.mark.gpu

VARIANTS = ["full", "mean"]


def shape(b, H, W, c, N, dtype="f32", seed=0, lowvar=True):
    return workloads.custom_shape(b, H, W, c, N, dtype, seed, lowvar)


SEQ_CASES = [
    # (name, shape, d_value)
    ("tiny_7x7", workloads.TINY, 1.0),
    ("tiny_7x7_D0", workloads.TINY, 0.0),
    ("ragged_b2_c65_L130_n16", shape(2, 10, 13, 65, 16, seed=1), 1.0),
    ("ragged_b2_c65_L130_n16_D0", shape(2, 10, 13, 65, 16, seed=1), 0.0),
    ("L1_c1_n1", shape(1, 1, 1, 1, 1, seed=2), 1.0),
    ("L2_c3_n2", shape(1, 1, 2, 3, 2, seed=3), 0.0),
    ("c1_n8_L200", shape(1, 8, 25, 1, 8, seed=4), 0.0),
    ("c130_n16_L64", shape(1, 8, 8, 130, 16, seed=5), 1.0),
    ("c192_n16_L257", shape(1, 1, 257, 192, 16, seed=6), 0.0),
]


@pytest.mark.parametrize("variant", VARIANTS)
@pytest.mark.parametrize("name,shp,dval", SEQ_CASES, ids=[c[0] for c in SEQ_CASES])
def test_seq_f32(variant, name, shp, dval):
    log(f"{variant} seq f32 {name}")
    inp = workloads.make_inputs(shp, "seq", d_value=dval)
    got = to_f64(run_scan(inp, variant, "seq"))
    ref = oracle_seq(inp, variant, "seq")
    assert_close(got, ref, **FP32_TOL, what=f"{variant} {name}")


@pytest.mark.parametrize("variant", VARIANTS)
@pytest.mark.parametrize("use_bias,use_d", [(False, True), (True, False), (False, False)])
def test_optional_parameters(variant, use_bias, use_d):
    log(f"{variant} optional bias={use_bias} D={use_d}")
    inp = workloads.make_inputs(shape(1, 6, 11, 40, 4, seed=8), "seq")
    got = to_f64(run_scan(inp, variant, "seq", use_bias=use_bias, use_d=use_d))
    ref = oracle_seq(inp, variant, "seq", use_bias=use_bias, use_d=use_d)
    assert_close(got, ref, **FP32_TOL, what=f"{variant} bias={use_bias} D={use_d}")


@pytest.mark.parametrize("variant", VARIANTS)
def test_softplus_off(variant):
    log(f"{variant} softplus off")
    inp = workloads.make_inputs(shape(1, 9, 9, 33, 8, seed=9), "seq")
    # without softplus Delta is used as given: keep it positive and small
    delta = (np.abs(inp.delta) * 0.05 + 1e-3).astype(np.float32)
    got = to_f64(run_scan(inp, variant, "seq", softplus=False, use_bias=False, delta=delta))
    ref = oracle_seq(inp, variant, "seq", softplus=False, use_bias=False, delta=delta)
    assert_close(got, ref, **FP32_TOL, what=f"{variant} softplus off")


@pytest.mark.parametrize("variant", VARIANTS)
@pytest.mark.parametrize("out", ["bf16", "f32"])
def test_bf16_inputs(variant, out):
    log(f"{variant} bf16 in, {out} out")
    inp = workloads.make_inputs(shape(2, 7, 9, 48, 16, "bf16", seed=10), "seq")
    y = run_scan(inp, variant, "seq", out_dtype=torch.bfloat16 if out == "bf16" else torch.float32)
    ref = oracle_seq(inp, variant, "seq")
    tol = BF16_TOL if out == "bf16" else FP32_TOL
    assert_close(to_f64(y), ref, **tol, what=f"{variant} bf16->{out}")


def merged_oracle(inp, variant, **kw):
    """fp64 oracle of the 2-D layout: per-direction outputs folded by the
    oracle's merge; also returns the merge of |y_k| for the tolerance."""
    seq = oracle_seq(inp, variant, "2d", **kw)
    H, W = inp.shape.H, inp.shape.W
    return oracle.cross_merge(seq, H, W, "f64"), oracle.cross_merge(np.abs(seq), H, W, "f64")


TWO_D_CASES = [("7x7_c32_n4", shape(1, 7, 7, 32, 4, lowvar=False)),
               ("5x9_c3_n16", shape(2, 5, 9, 3, 16, seed=11)),
               ("1x1_c2_n2", shape(1, 1, 1, 2, 2, seed=12)),
               ("1x13_c4_n4", shape(1, 1, 13, 4, 4, seed=13)),
               ("13x1_c4_n4", shape(1, 13, 1, 4, 4, seed=14)),
               ("33x40_c8_n16", shape(1, 33, 40, 8, 16, seed=15))]


@pytest.mark.parametrize("variant", VARIANTS)
@pytest.mark.parametrize("name,shp", TWO_D_CASES, ids=[c[0] for c in TWO_D_CASES])
def test_2d_layout_f32(variant, name, shp):
    log(f"{variant} 2d f32 {name}")
    inp = workloads.make_inputs(shp, "2d")
    got = to_f64(run_scan(inp, variant, "2d"))
    ref, scale = merged_oracle(inp, variant)
    # a sum of four per-direction results: their tolerances add
    assert_close(got, ref, rtol=FP32_TOL["rtol"], atol=4 * FP32_TOL["atol"], scale=scale,
                 what=f"{variant} 2d {name}")


@pytest.mark.parametrize("variant", VARIANTS)
def test_2d_layout_bf16(variant):
    log(f"{variant} 2d bf16")
    inp = workloads.make_inputs(shape(2, 12, 10, 24, 16, "bf16", seed=16), "2d")
    got = to_f64(run_scan(inp, variant, "2d"))
    ref, scale = merged_oracle(inp, variant)
    assert_close(got, ref, rtol=BF16_TOL["rtol"], atol=4 * BF16_TOL["atol"], scale=scale,
                 what=f"{variant} 2d bf16")


@pytest.mark.parametrize("variant", VARIANTS)
@pytest.mark.parametrize("layout", ["seq", "2d"])
def test_deterministic(variant, layout):
    log(f"{variant} determinism {layout}")
    inp = workloads.make_inputs(shape(1, 14, 14, 96, 16, seed=17), layout)
    a = run_scan(inp, variant, layout).cpu()
    b = run_scan(inp, variant, layout).cpu()
    assert torch.equal(a.view(torch.int32), b.view(torch.int32))


def test_mean_broadcasts_and_equals_full_on_identical_channels():
    """Identical channels within each direction: VMeanba equals the full scan."""
    log("mean == full on identical channels")
    inp = workloads.make_inputs(shape(1, 9, 9, 16, 16, seed=18), "seq")
    inp.u[...] = inp.u[:, :, :1]
    inp.delta[...] = inp.delta[:, :, :1]
    inp.dt_bias.reshape(4, 16)[...] = inp.dt_bias.reshape(4, 16)[:, :1]
    ym = to_f64(run_scan(inp, "mean", "seq"))
    yf = to_f64(run_scan(inp, "full", "seq"))
    assert np.all(ym == ym[:, :, :1])
    assert_close(ym, yf, **FP32_TOL, what="mean vs full, identical channels")
