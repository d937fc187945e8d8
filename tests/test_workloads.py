"""The seeded input generator: both layouts draw the same values, and the
sequence layout's u is the feature map in the four scan orders."""
import numpy as np

import oracle
import workloads


def test_layouts_draw_the_same_values():
    s = workloads.custom_shape(2, 5, 7, 3, 4, "f32", 3, True)
    a, b = workloads.make_inputs(s, "seq"), workloads.make_inputs(s, "2d")
    for name in ("x", "delta", "A", "B", "C", "D", "dt_bias"):
        assert np.array_equal(getattr(a, name), getattr(b, name)), name
    assert b.u is None


def test_sequence_u_is_the_cross_scan_of_x():
    for dtype in ("f32", "bf16"):
        s = workloads.custom_shape(2, 6, 9, 3, 4, dtype, 5, True)
        inp = workloads.make_inputs(s, "seq")
        assert np.array_equal(inp.u, oracle.cross_scan(inp.x))
        if dtype == "bf16":
            widened = (inp.bits["u"].astype(np.uint32) << 16).view(np.float32)
            assert np.array_equal(widened, inp.u)
