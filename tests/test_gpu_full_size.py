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


@functools.lru_cache(maxsize=1)
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


@pytest.mark.parametrize("shp", CONFIGS, ids=IDS)
def test_full_seq(shp):
    log(f"full seq {shp.name}")
    inp = inputs(shp.name, "seq")
    y = to_f64(run_scan(inp, "full", "seq"))
    bs = sample_batches(shp)
    sub = sub_batch(inp, bs)
    rows = sample_rows(shp, len(bs), np.random.default_rng(1))
    ref = oracle.full_scan(sub.u, sub.delta, sub.A, sub.B, sub.C, sub.D, sub.dt_bias, True,
                           sel=rows)
    got = y[bs].reshape(-1, shp.L)[rows]
    assert_close(got, ref, **tol(shp), what=f"full seq {shp.name}")


@pytest.mark.parametrize("shp", CONFIGS, ids=IDS)
def test_mean_seq(shp):
    log(f"mean seq {shp.name}")
    inp = inputs(shp.name, "seq")
    y = to_f64(run_scan(inp, "mean", "seq"))
    bs = sample_batches(shp)
    sub = sub_batch(inp, bs)
    ref = oracle.mean_scan(sub.u, sub.delta, sub.A, sub.B, sub.C, sub.D, sub.dt_bias, True)
    assert_close(y[bs], ref, **tol(shp), what=f"mean seq {shp.name}")


def merged_reference(sub, variant, shp, ds):
    """Oracle 2-D output for channels ds of the sampled batch items: every
    direction of those channels, folded by the oracle's merge."""
    u = oracle.cross_scan(sub.x)
    nb, Dc = u.shape[0], shp.channels
    if variant == "full":
        rows = [(b * 4 + k) * Dc + d for b in range(nb) for k in range(4) for d in ds]
        seq = oracle.full_scan(u, sub.delta, sub.A, sub.B, sub.C, sub.D, sub.dt_bias, True,
                               sel=rows).reshape(nb, 4, len(ds), shp.L)
    else:
        seq = oracle.mean_scan(u, sub.delta, sub.A, sub.B, sub.C, sub.D, sub.dt_bias,
                               True)[:, :, ds]
    seq = np.ascontiguousarray(seq)
    return (oracle.cross_merge(seq, shp.H, shp.W, "f64"),
            oracle.cross_merge(np.abs(seq), shp.H, shp.W, "f64"))


TWO_D = [workloads.TINY, workloads.STAGE1, workloads.STAGE2, workloads.BATCHED_BF16, workloads.HIRES]


@pytest.mark.parametrize("variant", ["full", "mean"])
@pytest.mark.parametrize("shp", TWO_D, ids=[s.name for s in TWO_D])
def test_2d(shp, variant):
    log(f"{variant} 2d {shp.name}")
    inp = inputs(shp.name, "2d")
    y = to_f64(run_scan(inp, variant, "2d"))
    bs = sample_batches(shp)
    sub = sub_batch(inp, bs)
    rng = np.random.default_rng(2)
    Dc = shp.channels
    ds = sorted({0, Dc - 1, *(int(d) for d in rng.choice(Dc, size=min(Dc, 6), replace=False))})
    ref, scale = merged_reference(sub, variant, shp, ds)
    t = tol(shp)
    got = y[bs][:, ds]
    assert_close(got, ref, rtol=t["rtol"], atol=4 * t["atol"], scale=scale,
                 what=f"{variant} 2d {shp.name}")
