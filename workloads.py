"""Seeded synthetic inputs for the SS2D selective-scan path.

This module only draws random numbers and lays them out; it holds none of the
method's arithmetic. Both the fp64 oracle (under ``oracle/``) and the HIP path
consume what it produces, so neither side feeds the other.

Shapes follow the VMamba-T SS2D stages the paper evaluates (224x224 ImageNet
inputs give 56x56 / 28x28 / 14x14 / 7x7 stage maps; a 512x2048 ADE20k-sized
input at stride 4 gives 128x512). The datasets and trained weights are not
available, so values are synthetic, with the low cross-channel variance the
paper reports for the scan's activations (Section 2.1, Fig. 3): every channel
of a position shares a N(0,1) base value plus N(0, 0.05^2) channel noise.

Distributions (fixed draw order, numpy PCG64, float32 draws):
  x      : tiny case N(0,1); other cases base + 0.05 * noise, [batch, channels, H, W]
  u      : (sequence layout) x laid out in the four scan orders, [batch, K, channels, L]:
           row by row, column by column, and both reversed (a permutation of
           the drawn values, so both layouts see the same data)
  delta  : N(0, 0.5) (variance 0.5), shape [batch, K, channels, L]
  dt     : log-uniform in [1e-3, 1e-1] per (k, d); dt_bias = log(expm1(dt)),
           so softplus(dt_bias) = dt (the usual Mamba dt initialisation)
  B, C   : N(0,1), shape [batch, K, N, L]
  A      : A[c, n] = -(n + 1)   (S4D-real initialisation), shape [K*channels, N]
  D      : 1 (or 0 for the scan-term-only parity case), shape [K*channels]
"""
from __future__ import annotations

import dataclasses
import math
from typing import Optional

import numpy as np

K_DIRS = 4


@dataclasses.dataclass(frozen=True)
class Shape:
    name: str
    batch: int
    H: int
    W: int
    channels: int
    N: int
    dtype: str = "f32"          # "f32" or "bf16" for u, delta, B, C
    seed: int = 0
    low_variance: bool = True   # base + 0.05 noise (False: plain N(0,1))

    @property
    def L(self) -> int:
        return self.H * self.W


# The five workloads: tiny, VMamba-T stage 1, later stages at batch 32,
# batched stage 1 in bf16, high-resolution segmentation stage 1.
TINY = Shape("tiny_7x7_c32_n4", 1, 7, 7, 32, 4, "f32", 0, low_variance=False)
STAGE1 = Shape("vmamba_t_stage1_56x56_c192_n16", 1, 56, 56, 192, 16, "f32", 10)
STAGE2 = Shape("vmamba_t_stage2_b32_28x28_c384_n16", 32, 28, 28, 384, 16, "f32", 20)
STAGE3 = Shape("vmamba_t_stage3_b32_14x14_c768_n16", 32, 14, 14, 768, 16, "f32", 21)
STAGE4 = Shape("vmamba_t_stage4_b32_7x7_c1536_n16", 32, 7, 7, 1536, 16, "f32", 22)
BATCHED_BF16 = Shape("vmamba_t_stage1_b128_56x56_c192_n16_bf16", 128, 56, 56, 192, 16, "bf16", 30)
HIRES = Shape("seg_stage1_b2_128x512_c192_n16", 2, 128, 512, 192, 16, "f32", 40)

ALL_SHAPES = [TINY, STAGE1, STAGE2, STAGE3, STAGE4, BATCHED_BF16, HIRES]


def bf16_round(a: np.ndarray) -> tuple[np.ndarray, np.ndarray]:
    """Round float32 values to bfloat16, nearest-even on the bit pattern.

    Returns (values widened back to float32, uint16 bit patterns). This is an
    input-storage conversion: both sides then read exactly these values.
    """
    a = np.ascontiguousarray(a, dtype=np.float32)
    bits = a.view(np.uint32).astype(np.uint64)
    lsb = (bits >> 16) & 1
    r = ((bits + 0x7FFF + lsb) >> 16).astype(np.uint16)
    nan = np.isnan(a)
    if nan.any():
        r[nan] = ((bits[nan] >> 16) | 0x40).astype(np.uint16)
    widened = (r.astype(np.uint32) << 16).view(np.float32)
    return widened, r


@dataclasses.dataclass
class Inputs:
    shape: Shape
    x: Optional[np.ndarray]      # [batch, channels, H, W] (2-D layout input)
    u: Optional[np.ndarray]      # [batch, K, channels, L] (sequence layout input)
    delta: np.ndarray            # [batch, K, channels, L]
    A: np.ndarray                # [K*channels, N] float32
    B: np.ndarray                # [batch, K, N, L]
    C: np.ndarray                # [batch, K, N, L]
    D: np.ndarray                # [K*channels] float32
    dt_bias: np.ndarray          # [K*channels] float32
    # bf16 bit patterns of the four streamed tensors when shape.dtype == "bf16"
    bits: Optional[dict] = None


def _normal(rng: np.random.Generator, shape, scale: float = 1.0) -> np.ndarray:
    out = rng.standard_normal(size=shape, dtype=np.float32)
    if scale != 1.0:
        out *= np.float32(scale)
    return out


def scan_orders(x: np.ndarray) -> np.ndarray:
    """A feature map [batch, channels, H, W] laid out in the four scan orders,
    [batch, 4, channels, H*W]: row by row, column by column, then the same
    two reversed. A permutation of x's elements (no arithmetic)."""
    b, c, H, W = x.shape
    rows = x.reshape(b, c, H * W)
    cols = np.ascontiguousarray(np.swapaxes(x, 2, 3)).reshape(b, c, H * W)
    return np.ascontiguousarray(np.stack([rows, cols, rows[..., ::-1], cols[..., ::-1]], axis=1))


def make_inputs(shape: Shape, layout: str = "seq", *, batch: Optional[int] = None,
                d_value: float = 1.0, seed: Optional[int] = None) -> Inputs:
    """Draw one seeded input set.

    The feature map x [batch, channels, H, W] is drawn for both layouts.
    layout "2d" : x is the input.
    layout "seq": u = x in the four scan orders, [batch, K, channels, L], is
    the input (x is kept too). Both layouts draw the same values for a seed.
    ``batch`` overrides the shape's batch (used to draw a bounded sample of a
    large workload); ``d_value`` sets the skip vector D.
    """
    if layout not in ("2d", "seq"):
        raise ValueError(f"unknown layout {layout!r}")
    b = shape.batch if batch is None else batch
    s = shape.seed if seed is None else seed
    rng = np.random.Generator(np.random.PCG64(s))
    Dc, L, N, H, W = shape.channels, shape.L, shape.N, shape.H, shape.W
    if shape.low_variance:
        base = _normal(rng, (b, 1, H, W))
        noise = _normal(rng, (b, Dc, H, W), 0.05)
        x = base + noise
    else:
        x = _normal(rng, (b, Dc, H, W))
    delta = _normal(rng, (b, K_DIRS, Dc, L), math.sqrt(0.5))
    lo, hi = math.log(1e-3), math.log(1e-1)
    dt = np.exp(rng.uniform(lo, hi, size=(K_DIRS * Dc,))).astype(np.float64)
    dt_bias = np.log(np.expm1(dt)).astype(np.float32)
    Bm = _normal(rng, (b, K_DIRS, N, L))
    Cm = _normal(rng, (b, K_DIRS, N, L))
    A = -np.tile(np.arange(1, N + 1, dtype=np.float32), (K_DIRS * Dc, 1))
    Dv = np.full((K_DIRS * Dc,), d_value, dtype=np.float32)
    bits = None
    if shape.dtype == "bf16":
        bits = {}
        x, bits["x"] = bf16_round(x)
        delta, bits["delta"] = bf16_round(delta)
        Bm, bits["B"] = bf16_round(Bm)
        Cm, bits["C"] = bf16_round(Cm)
    u = None
    if layout == "seq":
        u = scan_orders(x)
        if bits is not None:
            bits["u"] = scan_orders(bits["x"])
    return Inputs(shape, x, u, np.ascontiguousarray(delta), np.ascontiguousarray(A),
                  np.ascontiguousarray(Bm), np.ascontiguousarray(Cm), Dv, dt_bias, bits)


def custom_shape(batch: int, H: int, W: int, channels: int, N: int, dtype: str = "f32",
                 seed: int = 0, low_variance: bool = True, name: str = "custom") -> Shape:
    return Shape(name, batch, H, W, channels, N, dtype, seed, low_variance)


# ------------------------------------------------ materialised scan inputs
# The shapes of the paper's kernel experiments (Appendix D, Table 1): batch
# 128, one state, (inner dimension, sequence length) per VMamba stage, for the
# Tiny/Small and Base backbones.
TABLE1_SHAPES = [
    ("tiny_small", 384, 3136), ("tiny_small", 768, 784), ("tiny_small", 1536, 196),
    ("tiny_small", 3072, 49),
    ("base", 512, 3136), ("base", 1024, 784), ("base", 2048, 196), ("base", 4096, 49),
]
TABLE1_BATCH = 128


@dataclasses.dataclass
class DiscreteInputs:
    abar: np.ndarray  # [batch, channels, L]
    bu: np.ndarray    # [batch, channels, L]
    C: np.ndarray     # [batch, L]
    skip: Optional[np.ndarray]  # [batch, channels, L] or None


def make_discrete_inputs(batch: int, channels: int, L: int, seed: int,
                         with_skip: bool = False) -> DiscreteInputs:
    """Materialised one-state scan inputs, drawn directly (no discretisation
    is computed here): abar uniform in [e^-0.1, e^-0.001] (the decays exp(-dt)
    of dt in [1e-3, 1e-1] with A = -1), bu ~ N(0, 0.05^2) with the low
    cross-channel variance of the SS2D activations (a per-(b, t) base plus
    channel noise of one tenth its size), C ~ N(0, 1), skip ~ N(0, 1).
    Draw order: abar, bu base, bu noise, C, skip (PCG64, float32)."""
    rng = np.random.default_rng(seed)
    lo, hi = math.exp(-0.1), math.exp(-0.001)
    abar = rng.uniform(lo, hi, size=(batch, channels, L)).astype(np.float32)
    base = rng.standard_normal((batch, 1, L), dtype=np.float32)
    noise = rng.standard_normal((batch, channels, L), dtype=np.float32)
    bu = (np.float32(0.05) * (base + np.float32(0.1) * noise)).astype(np.float32)
    C = rng.standard_normal((batch, L), dtype=np.float32)
    skip = rng.standard_normal((batch, channels, L), dtype=np.float32) if with_skip else None
    return DiscreteInputs(abar=abar, bu=bu, C=C, skip=skip)


# ------------------------------------------------ selection projections (eq. 6)
@dataclasses.dataclass
class ProjectionWeights:
    W: np.ndarray               # [K, R + 2N, channels]: R timescale rows, N rows for B, N for C
    W_dt: Optional[np.ndarray]  # [K, channels, R], or None for the broadcast (R = 1)


def make_projection_weights(K: int, channels: int, N: int, R: int, seed: int,
                            broadcast: bool = False) -> ProjectionWeights:
    """Random projection weights of the shapes eq. 6 implies, drawn directly
    (PCG64, float32; W then W_dt): W ~ N(0, 1/channels) (unit-variance
    outputs for unit-variance inputs), W_dt ~ N(0, 1/R). ``broadcast`` (R = 1)
    leaves W_dt out: the timescale projection is Broadcast_D(Linear_1(u))."""
    rng = np.random.default_rng(seed)
    W = (rng.standard_normal((K, R + 2 * N, channels), dtype=np.float32)
         * np.float32(1.0 / math.sqrt(channels))).astype(np.float32)
    W_dt = None
    if not broadcast:
        W_dt = (rng.standard_normal((K, channels, R), dtype=np.float32)
                * np.float32(1.0 / math.sqrt(R))).astype(np.float32)
    else:
        assert R == 1
    return ProjectionWeights(W=W, W_dt=W_dt)
