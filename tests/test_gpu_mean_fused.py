"""VMeanba scan in one launch (reduce, carry and finish together, chunks of a
sequence waiting on the flags of the earlier chunks).

The flags live in the caller's workspace, so the results must not depend on
what the workspace held before the call (zeros, all-ones bytes, random bytes,
the flags of an earlier call), and repeated calls must agree bit for bit.
Grids on both sides of the single-launch limit (2048 workgroups) are checked
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
