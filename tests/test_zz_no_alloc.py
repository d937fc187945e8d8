"""The allocation-free VMeanba entry point (vmb_mean_scan_fwd_noalloc) against
vmb_mean_scan_fwd with a caller workspace: same kernels, so the outputs must
agree bit for bit, and both must meet the fp32 bound against the oracle. Two
calls in a row share the library's scratch array, the second on a smaller
input; a shape whose workspace exceeds the array is refused before launch."""
import numpy as np
import pytest
import torch

import workloads
from gpu_util import FP32_TOL, assert_close, dev, log, oracle_seq, run_scan, to_f64, upload_f32, \
    upload_stream
from paper_2412_16602_amd import vmb

pytestmark = pytest.mark.gpu


def _noalloc(inp, layout):
    s = inp.shape
    lay = vmb.VMB_LAYOUT_2D if layout == "2d" else vmb.VMB_LAYOUT_SEQ
    u = upload_stream(inp, "x" if layout == "2d" else "u")
    shape = (s.batch, s.channels, s.H, s.W) if layout == "2d" else tuple(inp.delta.shape)
    y = torch.full(shape, float("nan"), dtype=torch.float32, device=dev())
    vmb.vmb_mean_scan_fwd_noalloc(u, upload_stream(inp, "delta"), upload_f32(inp.A),
                                  upload_stream(inp, "B"), upload_stream(inp, "C"),
                                  upload_f32(inp.D), upload_f32(inp.dt_bias), True, y, layout=lay)
    torch.cuda.synchronize()
    return y


@pytest.mark.parametrize("layout", ["seq", "2d"])
def test_noalloc_matches_workspace_entry_point(layout):
    # the 56x56 stage-1 map at 192 channels (one launch), then a smaller
    # 28x28 map at 32 channels that reuses the scratch array
    big = workloads.custom_shape(1, 56, 56, 192, 16, "f32", 61, True)
    small = workloads.custom_shape(1, 28, 28, 32, 16, "f32", 62, True)
    for shp in (big, small):
        log(f"noalloc mean {layout} {shp.H}x{shp.W} c{shp.channels}")
        inp = workloads.make_inputs(shp, layout)
        got = _noalloc(inp, layout)
        ref_ws = run_scan(inp, "mean", layout)
        assert torch.equal(got, ref_ws), "no-alloc output differs from the workspace entry point"
        ref = oracle_seq(inp, "mean", layout)
        if layout == "2d":
            import oracle
            ref = oracle.cross_merge(np.ascontiguousarray(ref), shp.H, shp.W, "f64")
            assert_close(to_f64(got), ref, rtol=FP32_TOL["rtol"], atol=4 * FP32_TOL["atol"],
                         what=f"noalloc mean 2d {shp.name}")
        else:
            assert_close(to_f64(got), ref, **FP32_TOL, what=f"noalloc mean seq {shp.name}")


def test_noalloc_refuses_shapes_beyond_the_scratch_array():
    # 4 x 16 x 65536 positions of chunk scans alone need 32 MiB > 8 MiB
    log("noalloc refuses an oversized shape")
    L, Dc = 65536, 8
    t = lambda *s: torch.zeros(s, dtype=torch.float32, device=dev())
    u, dl, y = t(1, 4, Dc, L), t(1, 4, Dc, L), t(1, 4, Dc, L)
    A, B, C = t(4 * Dc, 16), t(1, 4, 16, L), t(1, 4, 16, L)
    assert vmb.vmb_scan_workspace_bytes(True, 1, 4, Dc, L, 16) > 8 << 20
    with pytest.raises(vmb.VmbError) as e:
        vmb.vmb_mean_scan_fwd_noalloc(u, dl, A, B, C, None, None, True, y)
    assert e.value.status == vmb.VMB_ERR_WORKSPACE
