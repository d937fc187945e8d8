"""Scan calls captured in a HIP graph and replayed on new inputs.

Between replays the program copies another input set into the captured
tensors (its own eager work) and synchronizes; every replay must compute the
result for the inputs it finds. The mean scan's one-launch form waits on
per-call flag values, which a captured call would carry into every replay;
while a stream is capturing the library takes the separate passes instead.
The sequences here have 15 chunks of 64 positions, where an eager call takes
the one-launch form.
"""
import numpy as np
import pytest
import torch

import workloads
from gpu_util import FP32_TOL, assert_close, dev, log, oracle_seq, to_f64
from paper_2412_16602_amd import vmb
from test_gpu_scan import merged_oracle

pytestmark = pytest.mark.gpu

H, W, DC = 24, 40, 16  # L = 960


def make(seed, layout):
    return workloads.make_inputs(workloads.custom_shape(1, H, W, DC, 16, "f32", seed, True), layout)


def fields(inp, layout):
    return [inp.x if layout == "2d" else inp.u, inp.delta, inp.A, inp.B, inp.C, inp.D, inp.dt_bias]


def reference(inp, variant, layout):
    if layout == "2d":
        return merged_oracle(inp, variant)
    return oracle_seq(inp, variant, "seq"), None


@pytest.mark.parametrize("layout", ["seq", "2d"])
@pytest.mark.parametrize("variant", ["mean", "mean_noalloc", "full"])
def test_graph_replays_on_new_inputs(variant, layout):
    log(f"graph replay {variant} {layout}")
    sets = [make(71, layout), make(72, layout)]
    lay = vmb.VMB_LAYOUT_2D if layout == "2d" else vmb.VMB_LAYOUT_SEQ
    tensors = [torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(dev())
               for a in fields(sets[0], layout)]
    u, delta, A, B, C, D, bias = tensors
    y = torch.empty((1, DC, H, W) if layout == "2d" else tuple(sets[0].delta.shape), device=dev())
    base = "full" if variant == "full" else "mean"
    if variant == "mean_noalloc":
        call = lambda: vmb.vmb_mean_scan_fwd_noalloc(u, delta, A, B, C, D, bias, True, y,
                                                     layout=lay)
    else:
        fn = vmb.vmb_selective_scan_fwd if base == "full" else vmb.vmb_mean_scan_fwd
        need = vmb.vmb_scan_workspace_bytes(base == "mean", 1, 4, DC, H * W, 16, lay)
        ws = torch.empty(max(need, 1), dtype=torch.uint8, device=dev()) if need else None
        call = lambda: fn(u, delta, A, B, C, D, bias, True, y, layout=lay, workspace=ws)
    # warm up on a side stream, then capture one call
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        call()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        call()
    torch.cuda.synchronize()
    refs = [reference(s, base, layout) for s in sets]
    eager_y = []
    for i in range(4):
        s = i % 2
        for t, a in zip(tensors, fields(sets[s], layout)):
            t.copy_(torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)))
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        got = to_f64(y)
        ref, scale = refs[s]
        if layout == "2d":
            assert_close(got, ref, rtol=FP32_TOL["rtol"], atol=4 * FP32_TOL["atol"], scale=scale,
                         what=f"replay {i} {variant} {layout}")
        else:
            assert_close(got, ref, **FP32_TOL, what=f"replay {i} {variant} {layout}")
        if base == "full":
            # the full scan has no per-call state: replays match eager calls bit for bit
            call()
            torch.cuda.synchronize()
            eager_y.append(y.clone())
            assert np.array_equal(to_f64(eager_y[-1]), got), f"replay {i} differs from eager"
