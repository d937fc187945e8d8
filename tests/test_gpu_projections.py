"""Selection projections of eq. 6 (vmb_ss2d_projections, on the matrix
cores) against the fp64 oracle's matmuls: VMamba's rank (channels / 16), the
paper's broadcast timescale (R = 1), the largest rank and row count, channel
chunks and position tiles with tails, bf16; then projections feeding the
scan, end to end."""
import numpy as np
import pytest
import torch

import oracle
import workloads
from gpu_util import BF16_TOL, FP32_TOL, assert_close, dev, log, to_f64, upload_f32
from paper_2412_16602_amd import vmb

pytestmark = pytest.mark.gpu


def draw_u(batch, K, Dc, L, seed, dtype="f32"):
    rng = np.random.default_rng(seed)
    u = (rng.standard_normal((batch, K, 1, L), dtype=np.float32)
         + np.float32(0.05) * rng.standard_normal((batch, K, Dc, L), dtype=np.float32))
    if dtype == "bf16":
        u, bits = workloads.bf16_round(u)
        t = torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).to(dev()).view(torch.bfloat16)
        return u, t
    return u.astype(np.float32), upload_f32(u)


def run(ut, pw, N):
    batch, K, Dc, L = ut.shape
    delta = torch.empty_like(ut)
    B = torch.empty((batch, K, N, L), dtype=ut.dtype, device=dev())
    C = torch.empty_like(B)
    W_dt = None if pw.W_dt is None else upload_f32(pw.W_dt)
    vmb.vmb_ss2d_projections(ut, upload_f32(pw.W), W_dt, delta, B, C)
    torch.cuda.synchronize()
    return delta, B, C


CASES = [  # batch, K, Dc, L, N, R, broadcast
    ("stage1_R12", 1, 4, 192, 3136, 16, 12, False),
    ("c70_L100_R5", 2, 4, 70, 100, 16, 5, False),
    ("c33_L49_bcast", 1, 4, 33, 49, 4, 1, True),
    ("c17_L10_n1_R3", 1, 2, 17, 10, 1, 3, False),
    ("c64_L64_R32_n16", 1, 1, 64, 64, 16, 32, False),
    ("c130_L65_n8_R1", 1, 3, 130, 65, 8, 1, False),
    ("c1536_L49_R48", 2, 4, 1536, 49, 16, 48, False),   # VMamba-T stage 4 rank
    ("c200_L70_R64_n16", 1, 2, 200, 70, 16, 64, False),  # largest rank, six row blocks
    ("c40_L30_R9_n2", 1, 4, 40, 30, 2, 9, False),
    # flattened positions over (batch, t): tiles of 64 (>= 8192 positions at
    # K = 4) and of 32 (>= 4065), tiles crossing batch boundaries, ragged tails
    ("tile64_b3_L2900_c70_R5", 3, 4, 70, 2900, 16, 5, False),
    ("tile64_b3_L2900_c100_R48", 3, 4, 100, 2900, 16, 48, False),
    ("tile64_b3_L2900_c65_bcast", 3, 4, 65, 2900, 16, 1, True),
    ("tile32_b5_L900_c130_R7", 5, 4, 130, 900, 16, 7, False),
    ("tile32_b5_L900_c64_bcast_n8", 5, 4, 64, 900, 8, 1, True),
]


@pytest.mark.parametrize("name,batch,K,Dc,L,N,R,bcast", CASES, ids=[c[0] for c in CASES])
def test_projections_f32(name, batch, K, Dc, L, N, R, bcast):
    log(f"projections {name}")
    u, ut = draw_u(batch, K, Dc, L, seed=len(name))
    pw = workloads.make_projection_weights(K, Dc, N, R, seed=7 + R, broadcast=bcast)
    d, B, C = run(ut, pw, N)
    rd, rB, rC = oracle.projections(u, pw.W, pw.W_dt, N=N)
    assert_close(to_f64(B), rB, **FP32_TOL, what=f"{name} B")
    assert_close(to_f64(C), rC, **FP32_TOL, what=f"{name} C")
    assert_close(to_f64(d), rd, **FP32_TOL, what=f"{name} delta")


@pytest.mark.parametrize("batch,L", [(2, 200), (5, 900), (3, 2900)])  # tiles of 16, 32, 64
def test_projections_bf16(batch, L):
    log(f"projections bf16 batch={batch} L={L}")
    u, ut = draw_u(batch, 4, 96, L, seed=3 + L, dtype="bf16")
    pw = workloads.make_projection_weights(4, 96, 16, 6, seed=4)
    d, B, C = run(ut, pw, 16)
    rd, rB, rC = oracle.projections(u, pw.W, pw.W_dt, N=16)
    for got, ref, nm in ((B, rB, "B"), (C, rC, "C"), (d, rd, "delta")):
        assert_close(to_f64(got), ref, **BF16_TOL, what=f"bf16 {nm}")


def test_rejects_bad_arguments():
    _, ut = draw_u(1, 4, 16, 8, seed=5)
    pw = workloads.make_projection_weights(4, 16, 4, 2, seed=6)
    with pytest.raises(vmb.VmbError):  # no W_dt with R = 2
        vmb.vmb_ss2d_projections(ut, upload_f32(pw.W), None, torch.empty_like(ut),
                                 torch.empty((1, 4, 4, 8), device=dev()),
                                 torch.empty((1, 4, 4, 8), device=dev()))
    B = torch.empty((1, 4, 4, 8), device=dev())
    with pytest.raises(vmb.VmbError):  # B and C the same buffer
        vmb.vmb_ss2d_projections(ut, upload_f32(pw.W), upload_f32(pw.W_dt), torch.empty_like(ut),
                                 B, B)


def test_projections_then_scan():
    """Eq. 6 feeding eqs. 3-4: the projections' delta, B and C go straight into
    the full and mean scans (the layouts agree); compared with the oracle's
    scan of the oracle's projections."""
    log("projections then scan, 28x28 c96")
    batch, K, Dc, L, N, R = 1, 4, 96, 784, 16, 6
    u, ut = draw_u(batch, K, Dc, L, seed=8)
    pw = workloads.make_projection_weights(K, Dc, N, R, seed=9)
    d, B, C = run(ut, pw, N)
    rd, rB, rC = oracle.projections(u, pw.W, pw.W_dt, N=N)
    shp = workloads.custom_shape(batch, 28, 28, Dc, N, "f32", 10, True)
    inp = workloads.make_inputs(shp, "seq")  # A, D, dt_bias of the workload recipe
    A, Dv, bias = upload_f32(inp.A), upload_f32(inp.D), upload_f32(inp.dt_bias)
    for variant, fn, ofn in (("full", vmb.vmb_selective_scan_fwd, oracle.full_scan),
                             ("mean", vmb.vmb_mean_scan_fwd, oracle.mean_scan)):
        ws_n = vmb.vmb_scan_workspace_bytes(variant == "mean", batch, K, Dc, L, N,
                                            vmb.VMB_LAYOUT_SEQ)
        ws = torch.empty(max(ws_n, 1), dtype=torch.uint8, device=dev()) if ws_n else None
        y = torch.empty_like(ut)
        fn(ut, d, A, B, C, Dv, bias, True, y, workspace=ws)
        torch.cuda.synchronize()
        ref = ofn(u, rd.astype(np.float32), inp.A, rB.astype(np.float32), rC.astype(np.float32),
                  inp.D, inp.dt_bias, True)
        # y is bilinear in (B, C) given u: the projections' fp32 rounding
        # (about 1e-6 of sum |W||u|) reaches y relative to the scan of the
        # absolute values, which bounds every term's magnitude
        scale = ofn(np.abs(u), rd.astype(np.float32), inp.A, np.abs(rB).astype(np.float32),
                    np.abs(rC).astype(np.float32), np.abs(inp.D), inp.dt_bias, True)
        assert_close(to_f64(y), ref, rtol=FP32_TOL["rtol"], atol=4 * FP32_TOL["atol"],
                     scale=scale, what=f"projections + {variant} scan")
