"""One-state scan on materialised inputs and the channel mean (the paper's
kernel-experiment decomposition) against the fp64 oracle: small shapes that
span several chunks and ragged tails, and every Table 1 shape at full size
on sampled sequences."""
import numpy as np
import pytest
import torch

import oracle
import workloads
from gpu_util import FP32_TOL, assert_close, dev, log
from paper_2412_16602_amd import vmb

pytestmark = pytest.mark.gpu


def _up(a):
    return None if a is None else torch.from_numpy(np.ascontiguousarray(a)).to(dev())


def _run_scan(inp: workloads.DiscreteInputs):
    a, b, c, k = map(_up, (inp.abar, inp.bu, inp.C, inp.skip))
    y = torch.empty_like(a)
    vmb.vmb_discrete_scan(a, b, c, k, y)
    torch.cuda.synchronize()
    return y.cpu().numpy().astype(np.float64)


# sequences under 8 positions take a 16-lane row each; up to 256 positions
# several whole sequences share a wave as one flat run (Q of them: 2 for
# (2, 2048, 100), 6 for (1, 12288, 28), 4 for the small odd L, crossing batch
# elements when Q does not divide the channels); longer ones take one wave
# each when there are at least 2048 of them ((4, 1024, 600)), else one
# workgroup each with the chunks spread over up to 16 waves (one to three
# groups of 16 chunks)
@pytest.mark.parametrize("batch,channels,L", [
    (1, 1, 1), (2, 3, 7), (5, 3, 4), (1, 1, 8), (3, 5, 9), (4, 3, 30), (3, 3, 50), (2, 7, 49),
    (1, 2, 512), (1, 2, 513), (2, 3, 1000), (1, 1, 3136), (3, 2, 49), (2, 5, 196), (1, 3, 1026),
    (1, 1, 4099), (5, 7, 64), (3, 11, 65), (2, 9, 256), (2, 13, 100), (1, 1, 257),
    (2, 2048, 100), (1, 12288, 28), (4, 1024, 600), (1, 2, 20000), (2, 1, 8193)])
@pytest.mark.parametrize("with_skip", [False, True])
def test_discrete_scan_small(batch, channels, L, with_skip):
    log(f"discrete scan {batch}x{channels}x{L} skip={with_skip}")
    inp = workloads.make_discrete_inputs(batch, channels, L, seed=L + channels, with_skip=with_skip)
    got = _run_scan(inp)
    ref = oracle.discrete_scan(inp.abar, inp.bu, inp.C, inp.skip)
    assert_close(got, ref, **FP32_TOL, what=f"discrete scan {batch}x{channels}x{L}")


# rows of lcm(L, 4) elements (one tile folded to positions for L = 49, 98,
# 50; whole position rows for L % 4 == 0), element rows otherwise; 1 to 16
# waves splitting the rows, with and without a remainder
@pytest.mark.parametrize("batch,channels,L", [
    (1, 1, 5), (2, 7, 33), (3, 64, 1000), (1, 9, 4096), (2, 12, 49), (3, 6, 98), (2, 5, 130),
    (2, 40, 50), (1, 3, 1001), (4, 700, 49), (2, 16, 3136), (2, 333, 196), (1, 6, 2)])
def test_channel_mean_small(batch, channels, L):
    log(f"channel mean {batch}x{channels}x{L}")
    rng = np.random.default_rng(batch * 1000 + L)
    x = rng.standard_normal((batch, channels, L), dtype=np.float32)
    xm = torch.empty(batch, L, device=dev())
    vmb.vmb_channel_mean(_up(x), xm)
    torch.cuda.synchronize()
    assert_close(xm.cpu().numpy(), oracle.channel_mean(x), **FP32_TOL,
                 what=f"channel mean {batch}x{channels}x{L}")


def test_mean_path_matches_oracle():
    """VMeanba path: T on both inputs, then the scan at one channel."""
    inp = workloads.make_discrete_inputs(2, 48, 784, seed=5)
    a, b, c = map(_up, (inp.abar, inp.bu, inp.C))
    am = torch.empty(2, 784, device=dev())
    bm = torch.empty(2, 784, device=dev())
    vmb.vmb_channel_mean(a, am)
    vmb.vmb_channel_mean(b, bm)
    y = torch.empty(2, 1, 784, device=dev())
    vmb.vmb_discrete_scan(am.view(2, 1, 784), bm.view(2, 1, 784), c, None, y)
    torch.cuda.synchronize()
    ref_a = oracle.channel_mean(inp.abar).astype(np.float32)[:, None, :]
    ref_b = oracle.channel_mean(inp.bu).astype(np.float32)[:, None, :]
    ref = oracle.discrete_scan(ref_a, ref_b, inp.C)
    assert_close(y.cpu().numpy(), ref, **FP32_TOL, what="mean path")


@pytest.mark.parametrize("backbone,channels,L", workloads.TABLE1_SHAPES)
def test_table1_shapes_sampled(backbone, channels, L):
    """Full Table 1 shape (batch 128) on the GPU; 24 sampled (b, d) sequences
    checked against the oracle on the same inputs."""
    batch = workloads.TABLE1_BATCH
    log(f"table 1 {backbone} channels={channels} L={L}")
    inp = workloads.make_discrete_inputs(batch, channels, L, seed=channels + L)
    a, b_, c = map(_up, (inp.abar, inp.bu, inp.C))
    y = torch.empty_like(a)
    vmb.vmb_discrete_scan(a, b_, c, None, y)
    torch.cuda.synchronize()
    assert bool(torch.isfinite(y).all())
    rng = np.random.default_rng(channels)
    picks = [(int(b), int(d)) for b, d in zip(rng.integers(0, batch, 24),
                                              rng.integers(0, channels, 24))]
    picks += [(0, 0), (batch - 1, channels - 1)]
    for b, d in picks:
        ref = oracle.discrete_scan(inp.abar[b:b + 1, d:d + 1], inp.bu[b:b + 1, d:d + 1],
                                   inp.C[b:b + 1])
        assert_close(y[b, d].cpu().numpy(), ref[0, 0], **FP32_TOL, what=f"({b}, {d})")


def test_graph_replay_matches_eager():
    """The calls captured in a HIP graph (as the Table 1 timing does): every
    replay, with eager work between, equals the eager result bit for bit."""
    inp = workloads.make_discrete_inputs(2, 40, 196, seed=9)
    a, b, c = map(_up, (inp.abar, inp.bu, inp.C))
    y_ref = torch.empty_like(a)
    am_ref = torch.empty(2, 196, device=dev())
    vmb.vmb_discrete_scan(a, b, c, None, y_ref)
    vmb.vmb_channel_mean(a, am_ref)
    torch.cuda.synchronize()
    y = torch.empty_like(a)
    am = torch.empty(2, 196, device=dev())
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        st = torch.cuda.current_stream()
        vmb.vmb_discrete_scan(a, b, c, None, y, stream=st)
        vmb.vmb_channel_mean(a, am, stream=st)
    for i in range(3):
        y.fill_(float("nan"))
        am.fill_(float("nan"))
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(y, y_ref), f"replay {i}: scan"
        assert torch.equal(am, am_ref), f"replay {i}: channel mean"
        vmb.vmb_discrete_scan(b, a, c, None, y_ref.clone())  # eager work in between
        torch.cuda.synchronize()
