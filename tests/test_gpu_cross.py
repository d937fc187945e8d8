"""Cross-scan / cross-merge on the GPU: bit-exact against the oracle."""
import numpy as np
import pytest
import torch

import oracle
import workloads
from gpu_util import dev, log
from paper_2412_16602_amd import vmb

pytestmark = pytest.mark.gpu

# whole-plane path (16-byte vectors, or single elements when L is not a
# multiple of the vector) and 32 x 32 tiles for planes larger than LDS; the
# last two have enough mid-size planes for the cross-scan to take three per
# workgroup (the second with a part-filled last workgroup and an odd L)
SHAPES = [(1, 32, 7, 7), (2, 3, 56, 56), (1, 5, 1, 1), (1, 2, 1, 33), (2, 3, 33, 1),
          (1, 4, 40, 70), (3, 2, 64, 32), (1, 192, 56, 56), (1, 3, 6, 10), (1, 2, 128, 160),
          (1, 2, 96, 127), (2, 1536, 40, 40), (1, 3073, 33, 35)]


def _x(shape, seed, dtype):
    rng = np.random.default_rng(seed)
    x = rng.standard_normal(shape).astype(np.float32)
    if dtype == "bf16":
        vals, bits = workloads.bf16_round(x)
        return vals, bits, torch.from_numpy(bits.view(np.int16)).to(dev()).view(torch.bfloat16)
    return x, None, torch.from_numpy(x).to(dev())


def _bits(t):
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).cpu().numpy().view(np.uint16)
    return t.cpu().numpy().view(np.uint32)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("shape", SHAPES)
def test_cross_scan_bit_exact(shape, dtype):
    log(f"cross_scan {shape} {dtype}")
    vals, bits, xd = _x(shape, sum(shape), dtype)
    b, c, H, W = shape
    xs = torch.empty((b, 4, c, H * W), dtype=xd.dtype, device=dev())
    vmb.vmb_cross_scan(xd, xs)
    torch.cuda.synchronize()
    ref = oracle.cross_scan(bits if dtype == "bf16" else vals)
    np.testing.assert_array_equal(_bits(xs), ref.view(np.uint16 if dtype == "bf16" else np.uint32))


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("shape", SHAPES)
def test_cross_merge_bit_exact(shape, dtype):
    log(f"cross_merge {shape} {dtype}")
    b, c, H, W = shape
    rng = np.random.default_rng(7 + sum(shape))
    ys = (rng.standard_normal((b, 4, c, H * W)) * 10.0 ** rng.integers(-3, 4, (b, 4, c, 1))).astype(np.float32)
    if dtype == "bf16":
        _, ybits = workloads.bf16_round(ys)
        yd = torch.from_numpy(ybits.view(np.int16)).to(dev()).view(torch.bfloat16)
        ref = oracle.cross_merge(ybits, H, W, "bf16")
    else:
        yd = torch.from_numpy(ys).to(dev())
        ref = oracle.cross_merge(ys, H, W, "f32").view(np.uint32)
    y = torch.empty((b, c, H, W), dtype=yd.dtype, device=dev())
    vmb.vmb_cross_merge(yd, y)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(_bits(y), ref)


@pytest.mark.parametrize("shape", [(2, 3, 56, 56), (1, 7, 13, 5)])
def test_round_trip_is_four_x(shape):
    log(f"round trip {shape}")
    vals, _, xd = _x(shape, 3, "f32")
    b, c, H, W = shape
    xs = torch.empty((b, 4, c, H * W), device=dev())
    y = torch.empty_like(xd)
    vmb.vmb_cross_scan(xd, xs)
    vmb.vmb_cross_merge(xs, y)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(y.cpu().numpy(), 4 * vals)
