"""VMeanba scan in one launch (reduce, carry and finish together, chunks of a
sequence waiting on the flags of the earlier chunks).

The flags live in the caller's workspace, so the results must not depend on
what the workspace held before the call (zeros, all-ones bytes, random bytes,
the flags of an earlier call), and repeated calls must agree bit for bit.
Grids on both sides of the single-launch limit (eight rounds of co-resident
workgroups: 2048 with one 1024-thread workgroup per compute unit) are checked
against the oracle, so the one-launch and the three-pass paths are both
covered at the same sequence length."""
import numpy as np
import pytest
import torch

import workloads
from gpu_util import FP32_TOL, assert_close, dev, log, oracle_seq, run_scan, to_f64
from paper_2412_16602_amd import vmb

pytestmark = pytest.mark.gpu


def _workspace(shp, fill: str) -> torch.Tensor:
    need = vmb.vmb_scan_workspace_bytes(1, shp.batch, 4, shp.channels, shp.H * shp.W, shp.N,
                                        vmb.VMB_LAYOUT_SEQ)
    ws = torch.empty(max(need, 1), dtype=torch.uint8, device=dev())
    if fill == "zeros":
        ws.zero_()
    elif fill == "ones":
        ws.fill_(0xFF)
    else:
        g = torch.Generator(device="cpu").manual_seed(7)
        ws.copy_(torch.randint(0, 256, (ws.numel(),), dtype=torch.uint8, generator=g))
    return ws


@pytest.mark.parametrize("fill", ["zeros", "ones", "random"])
def test_fused_any_workspace_contents(fill):
    # 49 chunks of 64 positions per sequence, 196 workgroups: one launch
    log(f"mean fused workspace={fill}")
    shp = workloads.custom_shape(1, 1, 3136, 8, 16, "f32", 11, True)
    inp = workloads.make_inputs(shp, "seq")
    ref = oracle_seq(inp, "mean", "seq")
    ws = _workspace(shp, fill)
    first = run_scan(inp, "mean", "seq", workspace=ws)
    assert_close(to_f64(first), ref, **FP32_TOL, what=f"mean fused ({fill})")
    # the flags of the first call are still in the workspace
    for i in range(2):
        again = run_scan(inp, "mean", "seq", workspace=ws)
        assert torch.equal(again, first), f"call {i + 2} differs from the first"


@pytest.mark.parametrize("batch", [10, 11])
def test_fused_grid_limit(batch):
    # 4 x 49 chunks per batch element: 1960 workgroups (one launch) and 2156
    # (reduce, finish as separate passes)
    log(f"mean grid limit batch={batch}")
    shp = workloads.custom_shape(batch, 1, 3136, 2, 16, "f32", 12 + batch, True)
    inp = workloads.make_inputs(shp, "seq")
    got = to_f64(run_scan(inp, "mean", "seq"))
    ref = oracle_seq(inp, "mean", "seq")
    assert_close(got, ref, **FP32_TOL, what=f"mean batch={batch}")


@pytest.mark.parametrize("N", [1, 4, 8])
def test_fused_fewer_states(N):
    # fewer states than waves: the spare waves sit out the scans
    log(f"mean fused N={N}")
    shp = workloads.custom_shape(1, 1, 700, 24, N, "f32", 30 + N, True)
    inp = workloads.make_inputs(shp, "seq")
    got = to_f64(run_scan(inp, "mean", "seq"))
    ref = oracle_seq(inp, "mean", "seq")
    assert_close(got, ref, **FP32_TOL, what=f"mean N={N}")
    assert np.all(np.isfinite(got))


# ---------------------------------------------------------------- error report
# The one-launch path's waits are bounded. VMB_MEAN_TEST_GIVE_UP makes them
# give up from the host side: the first chunk of every sequence withholds its
# flag and the others poll 8 times, so every kernel still ends normally. A
# chunk that gives up must not pass stale aggregates off as results: its
# outputs are NaN and vmb_mean_scan_status reports the call as incomplete.

def _stage1_like(batch=1, channels=8, seed=41):
    # 49 chunks of 64 positions per sequence: the one-launch path
    return workloads.custom_shape(batch, 56, 56, channels, 16, "f32", seed, True)


@pytest.mark.parametrize("fill", ["zeros", "ones"])
def test_status_of_unused_workspace(fill):
    log(f"mean status unused workspace={fill}")
    ws = _workspace(_stage1_like(), fill)
    torch.cuda.synchronize()
    assert vmb.vmb_mean_scan_status(ws) == vmb.VMB_ERR_WORKSPACE


def test_give_up_is_reported_and_poisons_only_the_unfinished_chunks():
    log("mean give-up (sequence layout)")
    shp = _stage1_like()
    inp = workloads.make_inputs(shp, "seq")
    ref = oracle_seq(inp, "mean", "seq")
    ws = _workspace(shp, "random")
    y = to_f64(run_scan(inp, "mean", "seq", workspace=ws, options=vmb.VMB_MEAN_TEST_GIVE_UP))
    assert vmb.vmb_mean_scan_status(ws) == vmb.VMB_ERR_INCOMPLETE
    # chunk 0 of every sequence waits for nothing and is exact; every later
    # chunk gave up and is NaN in every channel
    assert_close(y[..., :64], ref[..., :64], **FP32_TOL, what="chunk 0 after give-up")
    assert np.all(np.isnan(y[..., 64:])), "chunks after a give-up must be NaN"
    # the next ordinary call on the same workspace completes and says so
    again = to_f64(run_scan(inp, "mean", "seq", workspace=ws))
    assert vmb.vmb_mean_scan_status(ws) == vmb.VMB_OK
    assert_close(again, ref, **FP32_TOL, what="mean after a give-up call")


def test_give_up_2d_layout():
    log("mean give-up (2-D layout)")
    shp = _stage1_like(seed=42)
    inp = workloads.make_inputs(shp, "2d")
    need = vmb.vmb_scan_workspace_bytes(1, 1, 4, shp.channels, shp.L, 16, vmb.VMB_LAYOUT_2D)
    ws = torch.zeros(need, dtype=torch.uint8, device=dev())
    y = to_f64(run_scan(inp, "mean", "2d", workspace=ws, options=vmb.VMB_MEAN_TEST_GIVE_UP))
    assert vmb.vmb_mean_scan_status(ws) == vmb.VMB_ERR_INCOMPLETE
    # every pixel of a 56x56 map lies past position 63 in some direction
    assert np.all(np.isnan(y))
    ok = to_f64(run_scan(inp, "mean", "2d", workspace=ws))
    assert vmb.vmb_mean_scan_status(ws) == vmb.VMB_OK
    assert np.all(np.isfinite(ok))


@pytest.mark.parametrize("case", ["three_pass_long", "zoh", "pooled"])
def test_status_of_other_paths(case):
    # the separate passes never wait; they record the call all the same, so
    # a give-up left by an earlier call on the workspace is not reported again
    log(f"mean status {case}")
    if case == "three_pass_long":
        shp = workloads.custom_shape(1, 1, 64 * 70, 8, 16, "f32", 43, True)  # 70 chunks
        opts = vmb.VMB_MEAN_TEST_GIVE_UP  # ignored off the one-launch path
    else:
        shp = _stage1_like(seed=44)
        opts = vmb.VMB_SCAN_ZOH if case == "zoh" else vmb.VMB_MEAN_POOLED
    inp = workloads.make_inputs(shp, "seq")
    ws = _workspace(shp, "zeros")
    if case != "three_pass_long":
        fail_shp = _stage1_like(seed=45)
        run_scan(workloads.make_inputs(fail_shp, "seq"), "mean", "seq", workspace=ws,
                 options=vmb.VMB_MEAN_TEST_GIVE_UP)
        assert vmb.vmb_mean_scan_status(ws) == vmb.VMB_ERR_INCOMPLETE
    y = to_f64(run_scan(inp, "mean", "seq", workspace=ws, options=opts))
    assert vmb.vmb_mean_scan_status(ws) == vmb.VMB_OK
    assert np.all(np.isfinite(y))
