"""The C ABI on the CPU: the library loads, exports every function the
header declares, and rejects bad arguments with the documented status before
launching anything (the pointers below are never dereferenced)."""
import ctypes

import pytest
import torch

from paper_2412_16602_amd import vmb

OK, NULL, SHAPE, DTYPE, ALIGN, ALIAS, UNSUP, WS = 0, 1, 2, 3, 4, 5, 6, 7
F32, BF16 = 0, 1
SEQ, TWO_D = 0, 1


@pytest.fixture(scope="module")
def lib():
    # The calls below pass fake device addresses that validation must reject
    # before any launch. Never run them where a GPU could execute a kernel.
    import torch
    if torch.cuda.device_count() > 0:
        pytest.skip("fake-pointer validation tests run on CPU-only hosts")
    return vmb.load_library()


def test_exports_every_declared_symbol(lib):
    names = vmb.declared_symbols()
    assert set(names) >= {"vmb_cross_scan", "vmb_cross_merge", "vmb_selective_scan_fwd",
                          "vmb_mean_scan_fwd", "vmb_scan_workspace_bytes", "vmb_status_string",
                          "vmb_abi_version", "vmb_discrete_scan", "vmb_channel_mean",
                          "vmb_mean_scan_fwd_ex", "vmb_selective_scan_fwd_ex"}
    for name in names:
        assert hasattr(lib, name), name


def test_version_and_status_strings(lib):
    assert vmb.abi_version() == 2
    for s in range(10):
        assert lib.vmb_status_string(s) != b"unknown status"
    assert lib.vmb_status_string(OK) == b"ok"
    assert lib.vmb_status_string(10) == b"unknown status"


def test_mean_status_rejects(lib):
    # validation before any HIP call: NULL and misaligned workspaces
    assert lib.vmb_mean_scan_status(None, None) == NULL
    assert lib.vmb_mean_scan_status(ctypes.c_void_p(BASE + 8), None) == ALIGN
    with open(vmb.HEADER_PATH) as f:
        text = f.read()
    assert "VMB_ERR_INCOMPLETE = 9" in text and vmb.VMB_ERR_INCOMPLETE == 9
    assert "VMB_MEAN_TEST_GIVE_UP = 1 << 30" in text
    assert vmb.VMB_MEAN_TEST_GIVE_UP == 1 << 30


# A call that passes validation goes on to launch its kernels. With the fake
# addresses below that is harmless only on a host without a GPU, where the
# launch fails (VMB_ERR_HIP) and the status shows that validation let the call
# through; on a GPU host such calls are skipped.
NO_GPU = torch.cuda.device_count() == 0


def passes(call):
    """Assert that ``call()`` passes validation (only run without a GPU)."""
    if NO_GPU:
        assert call() in (OK, 8)


# fake, well-separated, 256-aligned "device" addresses
BASE = 1 << 40
STEP = 1 << 36


def P(i, off=0):
    return ctypes.c_void_p(BASE + i * STEP + off)


def scan_call(lib, fn="vmb_selective_scan_fwd", **kw):
    a = dict(u=P(0), delta=P(1), A=P(2), B=P(3), C=P(4), D=P(5), dt_bias=P(6), sp=1, y=P(7),
             batch=1, K=4, channels=8, L=12, N=4, in_dt=F32, out_dt=F32, layout=SEQ, H=3, W=4,
             ws=P(8), ws_bytes=1 << 30, stream=None)
    a.update(kw)
    args = [a["u"], a["delta"], a["A"], a["B"], a["C"], a["D"], a["dt_bias"], a["sp"], a["y"],
            a["batch"], a["K"], a["channels"], a["L"], a["N"], a["in_dt"], a["out_dt"],
            a["layout"], a["H"], a["W"], a["ws"], a["ws_bytes"]]
    if fn in ("vmb_mean_scan_fwd_ex", "vmb_selective_scan_fwd_ex"):
        args.append(a.get("options", 0))
    return getattr(lib, fn)(*args, a["stream"])


@pytest.mark.parametrize("fn", ["vmb_selective_scan_fwd", "vmb_mean_scan_fwd",
                                "vmb_mean_scan_fwd_ex", "vmb_selective_scan_fwd_ex"])
@pytest.mark.parametrize("kw,expect", [
    (dict(u=None), NULL), (dict(delta=None), NULL), (dict(A=None), NULL), (dict(B=None), NULL),
    (dict(C=None), NULL), (dict(y=None), NULL),
    (dict(batch=0), SHAPE), (dict(K=0), SHAPE), (dict(channels=-1), SHAPE), (dict(L=0), SHAPE),
    (dict(N=0), SHAPE), (dict(layout=7), SHAPE),
    (dict(layout=TWO_D, K=3), SHAPE), (dict(layout=TWO_D, H=5, W=4), SHAPE),
    (dict(N=3), UNSUP), (dict(N=32), UNSUP),
    (dict(in_dt=2), DTYPE), (dict(out_dt=5), DTYPE), (dict(in_dt=F32, out_dt=BF16), DTYPE),
    (dict(u=P(0, 4)), ALIGN), (dict(y=P(7, 8)), ALIGN), (dict(B=P(3, 2)), ALIGN),
    (dict(A=P(2, 2)), ALIGN),
    (dict(y=P(0, 16)), ALIAS), (dict(y=P(3)), ALIAS), (dict(y=P(2)), ALIAS),
])
def test_scan_rejects(lib, fn, kw, expect):
    assert scan_call(lib, fn, **kw) == expect


def test_mean_options_rules(lib):
    ex = "vmb_mean_scan_fwd_ex"
    SKIP1, RAW, NOBC = vmb.VMB_MEAN_SKIP_PER_CHANNEL, vmb.VMB_MEAN_RAW, vmb.VMB_MEAN_NO_BROADCAST
    POOL = vmb.VMB_MEAN_POOLED
    # the descriptions of include/vmb.h carry the same values
    with open(vmb.HEADER_PATH) as f:
        text = f.read()
    for name, val in (("VMB_MEAN_SKIP_PER_CHANNEL", SKIP1), ("VMB_MEAN_RAW", RAW),
                      ("VMB_MEAN_NO_BROADCAST", NOBC), ("VMB_MEAN_POOLED", POOL)):
        assert f"{name} = {val}" in text
    for opt in (0, SKIP1, RAW, NOBC, SKIP1 | RAW, RAW | NOBC):
        passes(lambda: scan_call(lib, ex, options=opt))
    # the test hook of the error report goes with every reading but the pooled one
    GIVE = vmb.VMB_MEAN_TEST_GIVE_UP
    for opt in (GIVE, GIVE | SKIP1, GIVE | RAW):
        passes(lambda: scan_call(lib, ex, options=opt))
    assert scan_call(lib, ex, options=GIVE | POOL) == UNSUP
    assert scan_call(lib, "vmb_selective_scan_fwd_ex", options=GIVE) == UNSUP
    assert scan_call(lib, ex, options=32) == UNSUP
    # the pooled reading only on its own, in either layout
    passes(lambda: scan_call(lib, ex, options=POOL))
    passes(lambda: scan_call(lib, ex, options=POOL, layout=TWO_D))
    for other in (SKIP1, RAW, NOBC):
        assert scan_call(lib, ex, options=POOL | other) == UNSUP
    assert scan_call(lib, ex, options=NOBC | SKIP1) == UNSUP
    # the zero-order-hold B: with the main reading, D1 and no-broadcast, not with R2 or pooled
    ZOH = vmb.VMB_SCAN_ZOH
    assert "VMB_SCAN_ZOH = 16" in text and ZOH == 16
    for opt in (ZOH, ZOH | SKIP1, ZOH | NOBC):
        passes(lambda: scan_call(lib, ex, options=opt))
    for opt in (ZOH | RAW, ZOH | POOL):
        assert scan_call(lib, ex, options=opt) == UNSUP
    full = "vmb_selective_scan_fwd_ex"
    passes(lambda: scan_call(lib, full, options=0))
    passes(lambda: scan_call(lib, full, options=ZOH))
    passes(lambda: scan_call(lib, full, options=ZOH, layout=TWO_D))
    for opt in (SKIP1, RAW, NOBC, POOL, 32):
        assert scan_call(lib, full, options=opt) == UNSUP
    assert scan_call(lib, ex, options=NOBC, layout=TWO_D) == UNSUP
    passes(lambda: scan_call(lib, ex, options=SKIP1 | RAW, layout=TWO_D))
    # without the broadcast y holds batch*K*L elements: [P(7), +4*12*4 B) overlaps
    # nothing here, and y placed just past the end of u (4*8*12 floats) is fine
    passes(lambda: scan_call(lib, ex, options=NOBC, y=P(0, 4 * 8 * 12 * 4)))
    passes(lambda: scan_call(lib, ex, options=0, y=P(0, 4 * 8 * 12 * 4)))
    assert scan_call(lib, ex, options=NOBC, y=P(0, 4 * 8 * 12 * 4 - 16)) == ALIAS


def test_workspace_rules(lib):
    need_full_2d = lib.vmb_scan_workspace_bytes(0, 1, 4, 8, 12, 4, TWO_D)
    need_mean = lib.vmb_scan_workspace_bytes(1, 1, 4, 8, 12, 4, SEQ)
    assert lib.vmb_scan_workspace_bytes(0, 1, 4, 8, 12, 4, SEQ) == 0
    assert need_full_2d >= 4 * 8 * 12 * 4 and need_mean > 0
    assert scan_call(lib, layout=TWO_D, ws=None) == WS
    assert scan_call(lib, layout=TWO_D, ws_bytes=need_full_2d - 1) == WS
    assert scan_call(lib, "vmb_mean_scan_fwd", ws=None) == WS
    assert scan_call(lib, "vmb_mean_scan_fwd", ws_bytes=need_mean - 1) == WS
    assert scan_call(lib, "vmb_mean_scan_fwd", ws=P(8, 8)) == ALIGN
    # workspace overlapping the output or an input
    assert scan_call(lib, "vmb_mean_scan_fwd", ws=P(7)) == ALIAS
    assert scan_call(lib, "vmb_mean_scan_fwd", ws=P(1)) == ALIAS
    assert lib.vmb_scan_workspace_bytes(1, 0, 4, 8, 12, 4, SEQ) == ctypes.c_size_t(-1).value


def test_shape_limits(lib):
    # 2-D maps beyond the merge pass's grid (65536 tiles of 32 columns) are
    # refused before any launch; one tile fewer passes
    for fn in ("vmb_selective_scan_fwd", "vmb_mean_scan_fwd"):
        assert scan_call(lib, fn, layout=TWO_D, channels=1, N=16, H=1, W=1 << 21,
                         L=1 << 21) == UNSUP
        passes(lambda: scan_call(lib, fn, layout=TWO_D, channels=1, N=16, H=1,
                                 W=(1 << 21) - 32, L=(1 << 21) - 32, ws_bytes=1 << 34))
    assert scan_call(lib, L=1 << 31) == SHAPE
    assert scan_call(lib, batch=1 << 20, channels=1 << 20) == SHAPE
    assert scan_call(lib, N=16, L=(1 << 31) // 8) == SHAPE


@pytest.mark.parametrize("fn,unfold", [("vmb_cross_scan", True), ("vmb_cross_merge", False)])
def test_cross_rejects(lib, fn, unfold):
    f = getattr(lib, fn)
    assert f(None, P(1), 1, 2, 3, 4, F32, None) == NULL
    assert f(P(0), None, 1, 2, 3, 4, F32, None) == NULL
    assert f(P(0), P(1), 0, 2, 3, 4, F32, None) == SHAPE
    assert f(P(0), P(1), 1, 2, 0, 4, F32, None) == SHAPE
    assert f(P(0), P(1), 1, 2, 3, 4, 9, None) == DTYPE
    assert f(P(0, 2), P(1), 1, 2, 3, 4, BF16, None) == ALIGN
    assert f(P(0), P(1, 4), 1, 2, 3, 4, F32, None) == ALIGN
    # overlap: map is 1*2*12 floats = 96 B, sequences 4x that
    assert f(P(0), P(0, 64), 1, 2, 3, 4, F32, None) == ALIAS
    if not unfold:
        # merge input is the 4-direction tensor (384 B): an output 256 B in overlaps it
        assert f(P(0), P(0, 256), 1, 2, 3, 4, F32, None) == ALIAS


def test_discrete_scan_rejects(lib):
    f = lib.vmb_discrete_scan
    # abar, bu, skip: [2, 3, 8] floats (192 B); C: [2, 8]
    ok = dict(a=P(0), b=P(1), c=P(2), k=P(3), y=P(4), batch=2, ch=3, L=8)

    def call(**kw):
        a = dict(ok)
        a.update(kw)
        return f(a["a"], a["b"], a["c"], a["k"], a["y"], a["batch"], a["ch"], a["L"], None)

    assert call(a=None) == NULL and call(b=None) == NULL and call(c=None) == NULL
    assert call(y=None) == NULL
    assert call(batch=0) == SHAPE and call(ch=0) == SHAPE and call(L=-1) == SHAPE
    assert call(L=1 << 31) == SHAPE
    assert call(a=P(0, 4)) == ALIGN and call(k=P(3, 8)) == ALIGN and call(y=P(4, 4)) == ALIGN
    assert call(y=P(0, 64)) == ALIAS and call(y=P(2, 48)) == ALIAS and call(y=P(3)) == ALIAS
    # skip is optional
    assert lib.vmb_discrete_scan(P(0), P(1), P(2), None, None, 2, 3, 8, None) == NULL


def test_channel_mean_rejects(lib):
    f = lib.vmb_channel_mean
    assert f(None, P(1), 2, 3, 8, None) == NULL and f(P(0), None, 2, 3, 8, None) == NULL
    assert f(P(0), P(1), 0, 3, 8, None) == SHAPE and f(P(0), P(1), 2, 3, 0, None) == SHAPE
    assert f(P(0, 4), P(1), 2, 3, 8, None) == ALIGN and f(P(0), P(1, 8), 2, 3, 8, None) == ALIGN
    assert f(P(0), P(0, 128), 2, 3, 8, None) == ALIAS


def test_projections_rejects(lib):
    f = lib.vmb_ss2d_projections
    # u, delta: [1, 4, 8, 12]; W [4, 2 + 8, 8]; W_dt [4, 8, 2]; B, C [1, 4, 4, 12]; R = 2, N = 4
    ok = dict(u=P(0), W=P(1), Wd=P(2), d=P(3), B=P(4), C=P(5), b=1, K=4, ch=8, L=12, N=4, R=2,
              dt=F32)

    def call(**kw):
        a = dict(ok)
        a.update(kw)
        return f(a["u"], a["W"], a["Wd"], a["d"], a["B"], a["C"], a["b"], a["K"], a["ch"], a["L"],
                 a["N"], a["R"], a["dt"], None)

    passes(call)
    assert call(u=None) == NULL and call(W=None) == NULL and call(C=None) == NULL
    assert call(b=0) == SHAPE and call(R=0) == SHAPE and call(L=0) == SHAPE
    assert call(dt=3) == DTYPE
    assert call(N=3) == UNSUP and call(R=65) == UNSUP and call(Wd=None) == UNSUP
    passes(lambda: call(Wd=None, R=1))  # the broadcast form
    assert call(u=P(0, 8)) == ALIGN and call(W=P(1, 2)) == ALIGN and call(B=P(4, 4)) == ALIGN
    assert call(d=P(0, 64)) == ALIAS and call(B=P(1)) == ALIAS and call(C=P(4, 16)) == ALIAS


def test_out_norm_rejects(lib):
    f = lib.vmb_ss2d_out_norm
    # y, z, out: [2, 8, 12] floats (768 B); gamma, beta [8]
    ok = dict(y=P(0), z=P(1), g=P(2), be=P(3), eps=1e-5, o=P(4), b=2, ch=8, p=12, dt=F32)

    def call(**kw):
        a = dict(ok)
        a.update(kw)
        return f(a["y"], a["z"], a["g"], a["be"], a["eps"], a["o"], a["b"], a["ch"], a["p"],
                 a["dt"], None)

    passes(call)
    assert call(y=None) == NULL and call(o=None) == NULL
    passes(lambda: call(z=None, g=None, be=None))  # all optional
    assert call(b=0) == SHAPE and call(ch=0) == SHAPE and call(p=-1) == SHAPE
    assert call(eps=-1.0) == SHAPE and call(eps=float("nan")) == SHAPE
    assert call(eps=float("inf")) == SHAPE
    assert call(dt=9) == DTYPE
    assert call(y=P(0, 2)) == ALIGN and call(g=P(2, 2)) == ALIGN
    passes(lambda: call(y=P(0, 2), o=P(4, 2), z=None, dt=BF16))  # bf16: 2-byte alignment
    assert call(o=P(0, 512)) == ALIAS and call(o=P(1)) == ALIAS and call(o=P(2, 4)) == ALIAS


def test_python_binding_refuses_cpu_tensors():
    import torch
    x = torch.zeros(1, 2, 3, 4)
    xs = torch.zeros(1, 4, 2, 12)
    with pytest.raises(ValueError):
        vmb.vmb_cross_scan(x, xs)


def test_python_binding_checks_new_entry_points():
    """Shape and dtype checks of the projection and norm bindings raise
    before any device work (CPU tensors, no GPU needed)."""
    import torch
    y = torch.zeros(2, 8, 12)
    with pytest.raises(ValueError):  # out of another shape
        vmb.vmb_ss2d_out_norm(y, None, None, None, 1e-5, torch.zeros(2, 8, 11))
    with pytest.raises(ValueError):  # gamma of the wrong length
        vmb.vmb_ss2d_out_norm(y, None, torch.ones(7), None, 1e-5, torch.zeros_like(y))
    with pytest.raises(ValueError):  # z of another dtype
        vmb.vmb_ss2d_out_norm(y, torch.zeros(2, 8, 12, dtype=torch.bfloat16), None, None, 1e-5,
                              torch.zeros_like(y))
    u = torch.zeros(1, 4, 8, 12)
    B = torch.zeros(1, 4, 4, 12)
    with pytest.raises(ValueError):  # W rows != R + 2N for the N of B
        vmb.vmb_ss2d_projections(u, torch.zeros(4, 9, 7), None, torch.zeros_like(u), B,
                                 torch.zeros_like(B))
    with pytest.raises(ValueError):  # W_dt of the wrong rank
        vmb.vmb_ss2d_projections(u, torch.zeros(4, 10, 8), torch.zeros(4, 8, 3),
                                 torch.zeros_like(u), B, torch.zeros_like(B))
    with pytest.raises(ValueError):  # C of another shape
        vmb.vmb_ss2d_projections(u, torch.zeros(4, 10, 8), torch.zeros(4, 8, 2),
                                 torch.zeros_like(u), B, torch.zeros(1, 4, 4, 11))
