"""Parity at the full workload sizes, in the configuration the benchmark
launches, on sampled outputs.

The GPU runs the whole call at full size. The fp64 oracle then recomputes
sampled sequences (full scan) or sampled (batch, direction) pairs (mean scan)
from the same inputs and compares them elementwise. Batch items are
independent, so the oracle runs on the sampled batch items only.
"""
import functools

import numpy as np
import pytest
import torch

import oracle
import workloads
from gpu_util import BF16_TOL, FP32_TOL, assert_close, log, run_scan, to_f64

pytestmark = pytest.mark.gpu

CONFIGS = [workloads.TINY, workloads.STAGE1, workloads.STAGE2, workloads.STAGE3, workloads.STAGE4,
           workloads.BATCHED_BF16, workloads.HIRES]
IDS = [s.name for s in CONFIGS]


@functools.lru_cache(maxsize=2)
def inputs(name, layout):
    shp = {s.name: s for s in CONFIGS}[name]
    return workloads.make_inputs(shp, layout)


def tol(shp):
    return BF16_TOL if shp.dtype == "bf16" else FP32_TOL


def sample_batches(shp):
    b = shp.batch
    return sorted({0, b - 1, b // 2})


def sub_batch(inp, bs):
    """The same inputs restricted to batch items bs (parameters unchanged)."""
    pick = lambda a: None if a is None else np.ascontiguousarray(a[bs])
    return workloads.Inputs(inp.shape, pick(inp.x), pick(inp.u), pick(inp.delta), inp.A,
                            pick(inp.B), pick(inp.C), inp.D, inp.dt_bias, None)


def sample_rows(shp, nb, rng):
    """Flat sequence indices (b*K + k)*Dc + d over nb batch items: the first
    and last channel of every direction plus random ones."""
    Dc = shp.channels
    rows = set()
    for b in range(nb):
        for k in range(4):
            base = (b * 4 + k) * Dc
            rows.update({base, base + Dc - 1})
            rows.update(int(base + d) for d in rng.choice(Dc, size=min(Dc, 4), replace=False))
    return sorted(rows)


# D = 1 (the workloads' skip) and D = 0: with D = 1 the skip term D u ~ N(0, 1)
# dominates y while the scan term C h is a few hundredths, so only the D = 0
# runs check the recurrence itself at the workload's tolerance.
SKIPS = [True, False]
SKIP_IDS = ["d1", "d0"]


@pytest.mark.parametrize("use_d", SKIPS, ids=SKIP_IDS)
@pytest.mark.parametrize("shp", CONFIGS, ids=IDS)
def test_full_seq(shp, use_d):
    log(f"full seq {shp.name} D={'1' if use_d else '0'}")
    inp = inputs(shp.name, "seq")
    y = to_f64(run_scan(inp, "full", "seq", use_d=use_d))
    bs = sample_batches(shp)
    sub = sub_batch(inp, bs)
    rows = sample_rows(shp, len(bs), np.random.default_rng(1))
    ref = oracle.full_scan(sub.u, sub.delta, sub.A, sub.B, sub.C, sub.D if use_d else None,
                           sub.dt_bias, True, sel=rows)
    got = y[bs].reshape(-1, shp.L)[rows]
    assert_close(got, ref, **tol(shp), what=f"full seq {shp.name} use_d={use_d}")


@pytest.mark.parametrize("use_d", SKIPS, ids=SKIP_IDS)
@pytest.mark.parametrize("shp", CONFIGS, ids=IDS)
def test_mean_seq(shp, use_d):
    log(f"mean seq {shp.name} D={'1' if use_d else '0'}")
    inp = inputs(shp.name, "seq")
    y = to_f64(run_scan(inp, "mean", "seq", use_d=use_d))
    bs = sample_batches(shp)
    sub = sub_batch(inp, bs)
    ref = oracle.mean_scan(sub.u, sub.delta, sub.A, sub.B, sub.C, sub.D if use_d else None,
                           sub.dt_bias, True)
    assert_close(y[bs], ref, **tol(shp), what=f"mean seq {shp.name} use_d={use_d}")


# The batched bf16 workload with fp32 output: the bf16 inputs are exact values
# the oracle reads as they are and the state is binary32, so the fp32
# tolerance applies (no output rounding). Checks the tile kernel's carry over
# the whole 3136-position sequence at that bound.
@pytest.mark.parametrize("variant", ["full", "mean"])
@pytest.mark.parametrize("use_d", SKIPS, ids=SKIP_IDS)
def test_batched_bf16_inputs_f32_output(variant, use_d):
    shp = workloads.BATCHED_BF16
    log(f"{variant} seq {shp.name} f32 out D={'1' if use_d else '0'}")
    inp = inputs(shp.name, "seq")
    y = to_f64(run_scan(inp, variant, "seq", out_dtype=torch.float32, use_d=use_d))
    bs = sample_batches(shp)
    sub = sub_batch(inp, bs)
    Dv = sub.D if use_d else None
    if variant == "full":
        rows = sample_rows(shp, len(bs), np.random.default_rng(3))
        ref = oracle.full_scan(sub.u, sub.delta, sub.A, sub.B, sub.C, Dv, sub.dt_bias, True,
                               sel=rows)
        got = y[bs].reshape(-1, shp.L)[rows]
    else:
        ref = oracle.mean_scan(sub.u, sub.delta, sub.A, sub.B, sub.C, Dv, sub.dt_bias, True)
        got = y[bs]
    assert_close(got, ref, **FP32_TOL, what=f"{variant} {shp.name} f32 out use_d={use_d}")


def merged_reference(sub, variant, shp, ds, use_d=True):
    """Oracle 2-D output for channels ds of the sampled batch items: every
    direction of those channels, folded by the oracle's merge."""
    u = oracle.cross_scan(sub.x)
    nb, Dc = u.shape[0], shp.channels
    Dv = sub.D if use_d else None
    if variant == "full":
        rows = [(b * 4 + k) * Dc + d for b in range(nb) for k in range(4) for d in ds]
        seq = oracle.full_scan(u, sub.delta, sub.A, sub.B, sub.C, Dv, sub.dt_bias, True,
                               sel=rows).reshape(nb, 4, len(ds), shp.L)
    else:
        seq = oracle.mean_scan(u, sub.delta, sub.A, sub.B, sub.C, Dv, sub.dt_bias,
                               True)[:, :, ds]
    seq = np.ascontiguousarray(seq)
    return (oracle.cross_merge(seq, shp.H, shp.W, "f64"),
            oracle.cross_merge(np.abs(seq), shp.H, shp.W, "f64"))


TWO_D = CONFIGS


@pytest.mark.parametrize("use_d", SKIPS, ids=SKIP_IDS)
@pytest.mark.parametrize("variant", ["full", "mean"])
@pytest.mark.parametrize("shp", TWO_D, ids=[s.name for s in TWO_D])
def test_2d(shp, variant, use_d):
    log(f"{variant} 2d {shp.name} D={'1' if use_d else '0'}")
    inp = inputs(shp.name, "2d")
    y = to_f64(run_scan(inp, variant, "2d", use_d=use_d))
    bs = sample_batches(shp)
    sub = sub_batch(inp, bs)
    rng = np.random.default_rng(2)
    Dc = shp.channels
    ds = sorted({0, Dc - 1, *(int(d) for d in rng.choice(Dc, size=min(Dc, 6), replace=False))})
    ref, scale = merged_reference(sub, variant, shp, ds, use_d)
    t = tol(shp)
    got = y[bs][:, ds]
    assert_close(got, ref, rtol=t["rtol"], atol=4 * t["atol"], scale=scale,
                 what=f"{variant} 2d {shp.name} use_d={use_d}")
