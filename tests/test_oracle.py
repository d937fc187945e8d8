"""Pins for the fp64 oracle: each test checks it against something other than
itself -- a hand-worked example, a closed form, a library routine, or an
invariant the method implies. CPU only."""
import json
import math
import os

import numpy as np
import pytest
import scipy.signal

import oracle
import workloads

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def rand_case(seed, batch=1, K=2, Dc=3, L=9, N=3, softplus=True, with_d=True, with_bias=True):
    rng = np.random.default_rng(seed)
    f = lambda *s: rng.standard_normal(s).astype(np.float32)
    u = f(batch, K, Dc, L)
    delta = (0.5 * f(batch, K, Dc, L)).astype(np.float32)
    A = (-rng.uniform(0.2, 2.0, size=(K * Dc, N))).astype(np.float32)
    B = f(batch, K, N, L)
    C = f(batch, K, N, L)
    D = f(K * Dc) if with_d else None
    bias = (0.3 * f(K * Dc)).astype(np.float32) if with_bias else None
    return dict(u=u, delta=delta, A=A, B=B, C=C, D=D, dt_bias=bias, softplus=softplus)


def timescale_np(delta, bias, softplus, K, Dc):
    """Delta = softplus(delta + bias) with numpy's logaddexp as the softplus."""
    v = delta.astype(np.float64)
    if bias is not None:
        v = v + bias.astype(np.float64).reshape(1, K, Dc, 1)
    return np.logaddexp(0.0, v) if softplus else v


def closed_form_full(c):
    """Cumulative-product closed form of eq. 3 (no recurrence):
    h[n,t] = sum_{s<=t} exp(A_n * sum_{r=s+1..t} Delta_r) * Delta_s * B[n,s] * u_s."""
    u, A, B, C = c["u"], c["A"], c["B"], c["C"]
    batch, K, Dc, L = u.shape
    N = A.shape[1]
    dl = timescale_np(c["delta"], c["dt_bias"], c["softplus"], K, Dc)
    y = np.zeros((batch, K, Dc, L))
    for b in range(batch):
        for k in range(K):
            for d in range(Dc):
                ch = k * Dc + d
                for t in range(L):
                    acc = 0.0
                    for n in range(N):
                        h = 0.0
                        for s in range(t + 1):
                            decay = math.exp(float(A[ch, n]) * float(np.sum(dl[b, k, d, s + 1:t + 1])))
                            h += decay * dl[b, k, d, s] * float(B[b, k, n, s]) * float(u[b, k, d, s])
                        acc += float(C[b, k, n, t]) * h
                    dskip = 0.0 if c["D"] is None else float(c["D"][ch])
                    y[b, k, d, t] = acc + dskip * float(u[b, k, d, t])
    return y


def run_full(c, **kw):
    return oracle.full_scan(c["u"], c["delta"], c["A"], c["B"], c["C"], c["D"], c["dt_bias"],
                            c["softplus"], **kw)


def run_mean(c, **kw):
    return oracle.mean_scan(c["u"], c["delta"], c["A"], c["B"], c["C"], c["D"], c["dt_bias"],
                            c["softplus"], **kw)


# ---------------------------------------------------------------- golden

def _golden(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


def _golden_case(g):
    i = g["inputs"]
    a = lambda key: np.asarray(i[key], dtype=np.float32)
    if "A_over_ln2" in i:
        A = (np.asarray(i["A_over_ln2"], dtype=np.float64) * math.log(2.0)).astype(np.float32)
    else:
        A = a("A")
    return dict(u=a("u"), delta=a("delta"), A=A, B=a("B"), C=a("C"), D=a("D"),
                dt_bias=a("dt_bias"), softplus=g["softplus"])


@pytest.mark.parametrize("name", ["hand_two_channel.json", "hand_softplus.json"])
def test_golden_full(name):
    g = _golden(name)
    c = _golden_case(g)
    np.testing.assert_allclose(run_full(c), np.asarray(g["expected_full"]), rtol=g["rtol"], atol=0)


def test_golden_mean():
    g = _golden("hand_two_channel.json")
    c = _golden_case(g)
    np.testing.assert_allclose(run_mean(c), np.asarray(g["expected_mean"]), rtol=g["rtol"], atol=0)


# ---------------------------------------------------------------- P1 closed form

@pytest.mark.parametrize("seed,softplus,with_d,with_bias,N", [
    (0, True, True, True, 3), (1, False, True, False, 2), (2, True, False, True, 1),
    (3, True, True, False, 4), (4, False, False, True, 3)])
def test_full_matches_cumulative_product_closed_form(seed, softplus, with_d, with_bias, N):
    c = rand_case(seed, batch=2, K=2, Dc=2, L=8, N=N, softplus=softplus, with_d=with_d,
                  with_bias=with_bias)
    np.testing.assert_allclose(run_full(c), closed_form_full(c), rtol=1e-10, atol=1e-12)


# ---------------------------------------------------------------- P2 LTI forms

def _lti_case(seed, L=40, N=3, Dc=2, const_u=False):
    rng = np.random.default_rng(seed)
    K = 1
    u = rng.standard_normal((1, K, Dc, L)).astype(np.float32)
    if const_u:
        u[...] = u[..., :1]
    delta = np.repeat(rng.uniform(0.05, 0.4, size=(1, K, Dc, 1)), L, axis=3).astype(np.float32)
    A = (-rng.uniform(0.3, 1.5, size=(K * Dc, N))).astype(np.float32)
    Bn = rng.standard_normal((N,)).astype(np.float32)
    Cn = rng.standard_normal((N,)).astype(np.float32)
    B = np.broadcast_to(Bn.reshape(1, 1, N, 1), (1, K, N, L)).copy()
    C = np.broadcast_to(Cn.reshape(1, 1, N, 1), (1, K, N, L)).copy()
    D = rng.standard_normal((K * Dc,)).astype(np.float32)
    return dict(u=u, delta=delta, A=A, B=B, C=C, D=D, dt_bias=None, softplus=False), Bn, Cn


def test_lti_equals_iir_filter_per_state():
    """Time-invariant Delta, B, C: each state is the first-order IIR filter
    h_t = a h_{t-1} + (Delta B) u_t, i.e. scipy.signal.lfilter([Delta B], [1, -a])."""
    c, Bn, Cn = _lti_case(7)
    y = run_full(c)
    Dc, L, N = c["u"].shape[2], c["u"].shape[3], c["A"].shape[1]
    for d in range(Dc):
        dl = float(c["delta"][0, 0, d, 0])
        u = c["u"][0, 0, d].astype(np.float64)
        ref = float(c["D"][d]) * u
        for n in range(N):
            a = math.exp(dl * float(c["A"][d, n]))
            ref = ref + float(Cn[n]) * scipy.signal.lfilter([dl * float(Bn[n])], [1.0, -a], u)
        np.testing.assert_allclose(y[0, 0, d], ref, rtol=1e-11, atol=1e-12)


def test_lti_equals_convolution_kernel():
    """eq. 5: with time-invariant parameters y = u * Kbar + D u, where
    Kbar_j = sum_n C_n Abar_n^j Bbar_n."""
    c, Bn, Cn = _lti_case(8, L=30)
    y = run_full(c)
    Dc, L, N = c["u"].shape[2], c["u"].shape[3], c["A"].shape[1]
    j = np.arange(L)
    for d in range(Dc):
        dl = float(c["delta"][0, 0, d, 0])
        kbar = np.zeros(L)
        for n in range(N):
            a = math.exp(dl * float(c["A"][d, n]))
            kbar += float(Cn[n]) * a ** j * dl * float(Bn[n])
        u = c["u"][0, 0, d].astype(np.float64)
        ref = np.convolve(u, kbar)[:L] + float(c["D"][d]) * u
        np.testing.assert_allclose(y[0, 0, d], ref, rtol=1e-11, atol=1e-12)


def test_constant_input_geometric_series():
    """Constant u, Delta, B: h_t = Delta B u (1 - a^(t+1)) / (1 - a)."""
    c, Bn, Cn = _lti_case(9, L=25, const_u=True)
    c["D"] = None
    y = run_full(c)
    N = c["A"].shape[1]
    t = np.arange(c["u"].shape[3])
    for d in range(c["u"].shape[2]):
        dl = float(c["delta"][0, 0, d, 0])
        uu = float(c["u"][0, 0, d, 0])
        ref = np.zeros_like(t, dtype=np.float64)
        for n in range(N):
            a = math.exp(dl * float(c["A"][d, n]))
            ref += float(Cn[n]) * dl * float(Bn[n]) * uu * (1 - a ** (t + 1)) / (1 - a)
        np.testing.assert_allclose(y[0, 0, d], ref, rtol=1e-11, atol=1e-12)


# ---------------------------------------------------------------- P3 N = 1, superposition

def test_states_superpose():
    """The output is linear in the states: the N-state run equals the sum of
    N one-state runs minus the N-1 extra copies of the skip term."""
    c = rand_case(11, batch=1, K=2, Dc=3, L=12, N=4)
    y = run_full(c)
    acc = np.zeros_like(y)
    N = c["A"].shape[1]
    for n in range(N):
        cn = dict(c)
        cn["A"] = np.ascontiguousarray(c["A"][:, n:n + 1])
        cn["B"] = np.ascontiguousarray(c["B"][:, :, n:n + 1])
        cn["C"] = np.ascontiguousarray(c["C"][:, :, n:n + 1])
        acc += run_full(cn)
    skip = c["D"].reshape(1, 2, 3, 1).astype(np.float64) * c["u"].astype(np.float64)
    np.testing.assert_allclose(y, acc - (N - 1) * skip, rtol=1e-11, atol=1e-12)


def test_n1_scalar_recurrence_by_hand_loop():
    c = rand_case(12, batch=1, K=1, Dc=1, L=15, N=1, with_bias=False)
    y = run_full(c)[0, 0, 0]
    dl = np.logaddexp(0.0, c["delta"][0, 0, 0].astype(np.float64))
    a = np.exp(dl * float(c["A"][0, 0]))
    # unrolled closed form for N = 1: h_t = sum_s (prod_{r=s+1..t} a_r) bu_s
    bu = dl * c["B"][0, 0, 0].astype(np.float64) * c["u"][0, 0, 0].astype(np.float64)
    for t in range(15):
        h = sum(np.prod(a[s + 1:t + 1]) * bu[s] for s in range(t + 1))
        ref = float(c["C"][0, 0, 0, t]) * h + float(c["D"][0]) * float(c["u"][0, 0, 0, t])
        assert abs(y[t] - ref) <= 1e-12 * max(1.0, abs(ref))


# ---------------------------------------------------------------- P4 / P5 mean variant

def test_mean_equals_full_when_channels_identical():
    """Identical channels within a direction: the channel mean of the
    discretised inputs is each channel's own, so VMeanba = the full scan."""
    c = rand_case(13, batch=2, K=2, Dc=4, L=11, N=3)
    for key in ("u", "delta"):
        c[key][...] = c[key][:, :, :1, :]
    A = c["A"].reshape(2, 4, 3)
    A[...] = A[:, :1, :]
    for key in ("D", "dt_bias"):
        v = c[key].reshape(2, 4)
        v[...] = v[:, :1]
    np.testing.assert_allclose(run_mean(c), run_full(c), rtol=1e-13, atol=1e-14)


def test_mean_is_channel_mean_of_full_when_timescale_shared():
    """If Delta and A do not vary over channels, the recurrence is linear in u,
    so under T = mean of (Abar, Bbar u, D u) the reduced output is exactly the
    channel mean of the full outputs, even with per-channel u and D."""
    c = rand_case(14, batch=1, K=3, Dc=5, L=10, N=3)
    c["delta"][...] = c["delta"][:, :, :1, :]
    A = c["A"].reshape(3, 5, 3)
    A[...] = A[:, :1, :]
    v = c["dt_bias"].reshape(3, 5)
    v[...] = v[:, :1]
    ym = run_mean(c)
    yf = run_full(c)
    ref = np.broadcast_to(yf.mean(axis=2, keepdims=True), yf.shape)
    np.testing.assert_allclose(ym, ref, rtol=1e-12, atol=1e-13)


def test_mean_single_channel_is_full():
    c = rand_case(15, batch=1, K=2, Dc=1, L=9, N=2)
    np.testing.assert_allclose(run_mean(c), run_full(c), rtol=1e-13, atol=1e-14)


def test_mean_output_is_broadcast():
    c = rand_case(16, batch=1, K=2, Dc=4, L=7, N=2)
    y = run_mean(c)
    assert np.all(y == y[:, :, :1, :])


# ---------------------------------------------------------------- mean-scan reading variants

SKIP1, RAW, NOBC = oracle.MEAN_SKIP_PER_CHANNEL, oracle.MEAN_RAW, oracle.MEAN_NO_BROADCAST


def _identical_channels(c, K, Dc, N):
    for key in ("u", "delta"):
        c[key][...] = c[key][:, :, :1, :]
    A = c["A"].reshape(K, Dc, N)
    A[...] = A[:, :1, :]
    for key in ("D", "dt_bias"):
        v = c[key].reshape(K, Dc)
        v[...] = v[:, :1]


@pytest.mark.parametrize("options", [SKIP1, RAW, SKIP1 | RAW])
def test_mean_variants_equal_full_when_channels_identical(options):
    """With identical channels every reading of T is the identity on them:
    each variant equals the full scan."""
    c = rand_case(40 + options, batch=2, K=2, Dc=4, L=12, N=3)
    _identical_channels(c, 2, 4, 3)
    np.testing.assert_allclose(run_mean(c, options=options), run_full(c), rtol=1e-12, atol=1e-13)


def test_mean_raw_is_full_scan_of_averaged_inputs():
    """Mean before discretisation, softplus off: Delta is affine in delta, so
    the mean timescale is that of the mean delta and mean bias; with D equal
    over a direction's channels, mean(D u) = D mean(u). The reduced scan is
    then the full scan of one channel fed the averaged u, delta, bias, A."""
    K, Dc, N, L = 3, 5, 4, 14
    c = rand_case(46, batch=2, K=K, Dc=Dc, L=L, N=N, softplus=False)
    D = c["D"].reshape(K, Dc)
    D[...] = D[:, :1]
    y = run_mean(c, options=RAW)
    avg = lambda a, axis: a.astype(np.float64).mean(axis=axis, keepdims=True)
    one = dict(u=avg(c["u"], 2).astype(np.float32), delta=avg(c["delta"], 2).astype(np.float32),
               A=avg(c["A"].reshape(K, Dc, N), 1).reshape(K, N).astype(np.float32),
               B=c["B"], C=c["C"], D=D[:, 0].copy(),
               dt_bias=avg(c["dt_bias"].reshape(K, Dc), 1).reshape(K).astype(np.float32),
               softplus=False)
    ref = run_full(one)  # [batch, K, 1, L]
    # the averages are rounded to float32 to feed the full scan
    np.testing.assert_allclose(y, np.broadcast_to(ref, y.shape), rtol=2e-5, atol=2e-6)


def test_mean_raw_softplus_averages_the_timescales():
    """Mean before discretisation with softplus on and delta varying over the
    channels: T averages the timescales Delta_d = softplus(delta_d + bias_d)
    themselves (the mean of the raw Delta of eq. 6), not softplus of the mean
    biased delta. The reduced scan is then the full scan of one channel fed
    that mean timescale as delta, with softplus off and no bias, the mean u and
    the mean A; D is shared over a direction's channels, so mean(D u) = D mean(u).
    The other order of softplus and mean is checked to fail the same comparison,
    so this pin tells the two readings apart."""
    K, Dc, N, L = 2, 6, 3, 13
    c = rand_case(49, batch=2, K=K, Dc=Dc, L=L, N=N, softplus=True)
    c["delta"] = (2.0 * c["delta"]).astype(np.float32)  # spread over softplus' curved part
    D = c["D"].reshape(K, Dc)
    D[...] = D[:, :1]
    y = run_mean(c, options=RAW)
    avg = lambda a, axis: a.astype(np.float64).mean(axis=axis, keepdims=True)
    v = c["delta"].astype(np.float64) + c["dt_bias"].astype(np.float64).reshape(1, K, Dc, 1)
    assert np.ptp(v, axis=2).min() > 0.5  # the channels really differ

    def one_channel(timescale):
        one = dict(u=avg(c["u"], 2).astype(np.float32), delta=timescale.astype(np.float32),
                   A=avg(c["A"].reshape(K, Dc, N), 1).reshape(K, N).astype(np.float32),
                   B=c["B"], C=c["C"], D=D[:, 0].copy(), dt_bias=None, softplus=False)
        return np.broadcast_to(run_full(one), y.shape)

    ref = one_channel(np.logaddexp(0.0, v).mean(axis=2, keepdims=True))
    np.testing.assert_allclose(y, ref, rtol=2e-5, atol=2e-6)
    wrong = one_channel(np.logaddexp(0.0, v.mean(axis=2, keepdims=True)))
    assert np.max(np.abs(wrong - y) - (2e-6 + 2e-5 * np.abs(y))) > 1e-3


def test_mean_raw_equals_discretised_mean_when_timescale_shared():
    """If Delta and A do not vary over channels, exp(Delta A) is the same for
    every channel and mean(Delta u) = Delta mean(u): both readings of T give
    the same reduced scan."""
    c = rand_case(47, batch=1, K=3, Dc=6, L=13, N=3)
    c["delta"][...] = c["delta"][:, :, :1, :]
    A = c["A"].reshape(3, 6, 3)
    A[...] = A[:, :1, :]
    v = c["dt_bias"].reshape(3, 6)
    v[...] = v[:, :1]
    np.testing.assert_allclose(run_mean(c, options=RAW), run_mean(c), rtol=1e-12, atol=1e-13)


@pytest.mark.parametrize("raw", [0, RAW])
def test_mean_skip_per_channel_averages_to_reduced_skip(raw):
    """The per-channel skip D[c] u_d averages over the channels to r_mean, so
    the channel mean of the per-channel-skip output is the reduced-skip output,
    and the two differ channel by channel by D[c] u_d - r_mean."""
    K, Dc = 2, 5
    c = rand_case(48 + raw, batch=2, K=K, Dc=Dc, L=11, N=3)
    y1 = run_mean(c, options=SKIP1 | raw)
    y2 = run_mean(c, options=raw)
    np.testing.assert_allclose(y1.mean(axis=2, keepdims=True), y2[:, :, :1], rtol=1e-12,
                               atol=1e-13)
    du = c["D"].astype(np.float64).reshape(1, K, Dc, 1) * c["u"].astype(np.float64)
    np.testing.assert_allclose(y1 - du, y2 - du.mean(axis=2, keepdims=True), rtol=1e-12,
                               atol=1e-13)


@pytest.mark.parametrize("raw", [0, RAW])
def test_mean_no_broadcast_is_one_row(raw):
    c = rand_case(50 + raw, batch=2, K=2, Dc=4, L=10, N=2)
    y = run_mean(c, options=NOBC | raw)
    assert y.shape == (2, 2, 1, 10)
    assert np.array_equal(y, run_mean(c, options=raw)[:, :, :1])


# ---------------------------------------------------------------- P6 permutations

@pytest.mark.parametrize("H,W", [(1, 1), (1, 5), (4, 1), (3, 3), (4, 6), (7, 7)])
def test_cross_scan_maps(H, W):
    rng = np.random.default_rng(H * 10 + W)
    x = rng.standard_normal((2, 3, H, W)).astype(np.float32)
    xs = oracle.cross_scan(x)
    assert xs.shape == (2, 4, 3, H * W)
    np.testing.assert_array_equal(xs[:, 0], x.reshape(2, 3, H * W))
    np.testing.assert_array_equal(xs[:, 1], np.swapaxes(x, 2, 3).reshape(2, 3, H * W))
    np.testing.assert_array_equal(xs[:, 2], xs[:, 0, :, ::-1])
    np.testing.assert_array_equal(xs[:, 3], xs[:, 1, :, ::-1])
    # every direction is a bijection of the positions
    idx = np.arange(H * W, dtype=np.int64).reshape(1, 1, H, W)
    p = oracle.cross_scan(idx)
    for k in range(4):
        assert sorted(p[0, k, 0].tolist()) == list(range(H * W))


@pytest.mark.parametrize("H,W", [(1, 1), (2, 5), (5, 3), (7, 7), (8, 16)])
def test_merge_of_scan_is_four_times_exact(H, W):
    rng = np.random.default_rng(3)
    x = rng.standard_normal((2, 3, H, W)).astype(np.float32)
    xs = oracle.cross_scan(x)
    np.testing.assert_array_equal(oracle.cross_merge(xs, H, W, "f32"), 4 * x)
    np.testing.assert_array_equal(oracle.cross_merge(xs.astype(np.float64), H, W, "f64"), 4 * x.astype(np.float64))
    xb = workloads.bf16_round(x)[1]
    yb = oracle.cross_merge(oracle.cross_scan(xb), H, W, "bf16")
    widened = (yb.astype(np.uint32) << 16).view(np.float32)
    np.testing.assert_array_equal(widened, 4 * workloads.bf16_round(x)[0])


def test_merge_is_adjoint_of_scan():
    """<cross_scan(x), ys> = <x, cross_merge(ys)>: the merge sums exactly the
    positions the scan copied to."""
    rng = np.random.default_rng(4)
    H, W = 5, 6
    x = rng.standard_normal((2, 3, H, W))
    ys = rng.standard_normal((2, 4, 3, H * W))
    lhs = float(np.sum(oracle.cross_scan(x) * ys))
    rhs = float(np.sum(x * oracle.cross_merge(ys, H, W, "f64")))
    assert abs(lhs - rhs) <= 1e-12 * max(1.0, abs(lhs))


def test_merge_association_f32():
    """binary32 merge = (y0 + y2) + (y1 + y3) in single precision, checked
    against numpy float32 adds on the scan-order gathered values."""
    rng = np.random.default_rng(5)
    H, W = 4, 5
    ys = (rng.standard_normal((1, 4, 2, H * W)) * np.array([1, 1e4, 1e-4, 3e3]).reshape(1, 4, 1, 1)).astype(np.float32)
    y = oracle.cross_merge(ys, H, W, "f32")
    L = H * W
    hh, ww = np.meshgrid(np.arange(H), np.arange(W), indexing="ij")
    p0 = hh * W + ww
    p1 = ww * H + hh
    g = [ys[0, 0][:, p0], ys[0, 1][:, p1], ys[0, 2][:, L - 1 - p0], ys[0, 3][:, L - 1 - p1]]
    ref = (g[0] + g[2]) + (g[1] + g[3])
    np.testing.assert_array_equal(y[0], ref)


def test_bf16_rounding_matches_torch():
    import torch
    rng = np.random.default_rng(6)
    a = (rng.standard_normal(4096) * 10.0 ** rng.integers(-20, 20, 4096)).astype(np.float32)
    a[:4] = [0.0, -0.0, np.inf, -np.inf]
    ours = oracle.to_bf16_bits(a)
    ref = torch.from_numpy(a).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    np.testing.assert_array_equal(ours, ref)


# ---------------------------------------------------------------- P7 combine algebra

def _combine(p, q):
    (a1, b1), (a2, b2) = p, q
    return (a1 * a2, a2 * b1 + b2)


def test_associative_combine_matches_sequential_scan():
    """The (a, b) combine used by a parallel scan, applied over random
    chunkings and tree orders, reproduces the oracle's sequential states."""
    rng = np.random.default_rng(17)
    L = 64
    c = rand_case(17, batch=1, K=1, Dc=1, L=L, N=1, with_d=False)
    c["C"][...] = 1.0
    h_ref = run_full(c)[0, 0, 0]
    dl = np.logaddexp(0.0, c["delta"][0, 0, 0].astype(np.float64) + float(c["dt_bias"][0]))
    a = np.exp(dl * float(c["A"][0, 0]))
    b = dl * c["B"][0, 0, 0].astype(np.float64) * c["u"][0, 0, 0].astype(np.float64)
    for trial in range(20):
        cuts = np.sort(rng.choice(np.arange(1, L), size=rng.integers(1, 12), replace=False))
        chunks = np.split(np.arange(L), cuts)
        aggs = []
        for ch in chunks:  # chunk aggregate, combined in a random tree order
            items = [(a[i], b[i]) for i in ch]
            while len(items) > 1:
                j = int(rng.integers(0, len(items) - 1))
                items[j:j + 2] = [_combine(items[j], items[j + 1])]
            aggs.append(items[0])
        carry = (1.0, 0.0)
        for ch, agg in zip(chunks, aggs):
            h = carry[1]
            for i in ch:
                h = a[i] * h + b[i]
                assert abs(h - h_ref[i]) <= 1e-12 * max(1.0, abs(h_ref[i]))
            carry = _combine(carry, agg)
            assert abs(carry[1] - h_ref[ch[-1]]) <= 1e-12 * max(1.0, abs(h_ref[ch[-1]]))


# ---------------------------------------------------------------- P8 softplus / timescale

def test_timescale_is_softplus_of_biased_delta():
    """One step, A = 0, B = C = u = 1, D = 0: y = Delta = softplus(delta + bias)."""
    v = np.concatenate([np.linspace(-30, 30, 61), [-80.0, 80.0, 1e-6, -1e-6]]).astype(np.float32)
    n = v.size
    u = np.ones((1, 1, n, 1), np.float32)
    c = dict(u=u, delta=v.reshape(1, 1, n, 1), A=np.zeros((n, 1), np.float32),
             B=np.ones((1, 1, 1, 1), np.float32), C=np.ones((1, 1, 1, 1), np.float32), D=None,
             dt_bias=np.zeros(n, np.float32), softplus=True)
    y = run_full(c)[0, 0, :, 0]
    np.testing.assert_allclose(y, np.logaddexp(0.0, v.astype(np.float64)), rtol=1e-14, atol=0)
    c["softplus"] = False
    np.testing.assert_array_equal(run_full(c)[0, 0, :, 0], v.astype(np.float64))


def test_dt_bias_inverts_softplus():
    """The generator's dt_bias = softplus^-1(dt): with delta = 0 the oracle's
    timescale is dt, log-uniform in [1e-3, 1e-1]."""
    inp = workloads.make_inputs(workloads.TINY, "seq")
    n = inp.dt_bias.size
    c = dict(u=np.ones((1, 1, n, 1), np.float32), delta=np.zeros((1, 1, n, 1), np.float32),
             A=np.zeros((n, 1), np.float32), B=np.ones((1, 1, 1, 1), np.float32),
             C=np.ones((1, 1, 1, 1), np.float32), D=None, dt_bias=inp.dt_bias, softplus=True)
    dt = run_full(c)[0, 0, :, 0]
    assert dt.min() >= 1e-3 * (1 - 1e-5) and dt.max() <= 1e-1 * (1 + 1e-5)


# ---------------------------------------------------------------- selection / threads

def test_selected_sequences_match_full_output():
    c = rand_case(18, batch=2, K=4, Dc=3, L=6, N=2)
    y = run_full(c)
    sel = [0, 5, 23, 11]
    ys = run_full(c, sel=sel)
    flat = y.reshape(-1, 6)
    np.testing.assert_array_equal(ys, flat[sel])
    ym = run_mean(c)
    selm = [7, 2]
    np.testing.assert_array_equal(run_mean(c, sel=selm), ym.reshape(8, 3, 6)[selm])


def test_thread_count_does_not_change_results():
    c = rand_case(19, batch=2, K=4, Dc=5, L=20, N=3)
    np.testing.assert_array_equal(run_full(c, nthreads=1), run_full(c, nthreads=4))
    np.testing.assert_array_equal(run_mean(c, nthreads=1), run_mean(c, nthreads=4))


def test_degenerate_sizes():
    c = rand_case(20, batch=1, K=1, Dc=1, L=1, N=1)
    y = run_full(c)
    dl = float(np.logaddexp(0.0, float(c["delta"].ravel()[0]) + float(c["dt_bias"][0])))
    ref = float(c["C"].ravel()[0]) * dl * float(c["B"].ravel()[0]) * float(c["u"].ravel()[0]) \
        + float(c["D"][0]) * float(c["u"].ravel()[0])
    assert abs(y.ravel()[0] - ref) <= 1e-14 * max(1.0, abs(ref))


# ------------------------------------------- scan on materialised inputs (N = 1)
# The decomposition of the paper's kernel experiments (Appendix D, Table 1):
# discretisation outside, a one-state scan inside; T applied beforehand.

def _discrete_case(seed, batch=2, Dc=3, L=17, with_skip=True):
    rng = np.random.default_rng(seed)
    abar = rng.uniform(0.3, 1.0, size=(batch, Dc, L)).astype(np.float32)
    bu = rng.standard_normal((batch, Dc, L)).astype(np.float32)
    C = rng.standard_normal((batch, L)).astype(np.float32)
    skip = rng.standard_normal((batch, Dc, L)).astype(np.float32) if with_skip else None
    return abar, bu, C, skip


def test_discrete_scan_is_full_scan_with_one_state():
    """With abar = exp(Delta A), bu = Delta B u and skip = D u formed outside,
    the one-state scan is the (independently pinned) full scan at N = 1."""
    c = rand_case(40, batch=2, K=1, Dc=3, L=13, N=1)
    y_full = run_full(c)[:, 0]  # [batch, Dc, L]
    dl = timescale_np(c["delta"], c["dt_bias"], c["softplus"], 1, 3)[:, 0]
    A = c["A"][:, 0].astype(np.float64).reshape(1, 3, 1)
    abar = np.exp(dl * A).astype(np.float32)
    bu = (dl * c["B"][:, 0, 0][:, None, :] * c["u"][:, 0]).astype(np.float32)
    skip = (c["D"].astype(np.float64).reshape(1, 3, 1) * c["u"][:, 0]).astype(np.float32)
    y = oracle.discrete_scan(abar, bu, c["C"][:, 0, 0], skip)
    # inputs rounded to fp32 on the way in: agreement to fp32 input precision
    np.testing.assert_allclose(y, y_full, rtol=2e-6, atol=2e-6)


def test_discrete_scan_geometric_series():
    """Constant a, b, C = 1, no skip: h_t = b (1 - a^{t+1}) / (1 - a)."""
    L = 40
    a, b = 0.8125, 0.375  # exact in fp32
    abar = np.full((1, 2, L), a, np.float32)
    bu = np.full((1, 2, L), b, np.float32)
    C = np.ones((1, L), np.float32)
    y = oracle.discrete_scan(abar, bu, C)
    t = np.arange(L)
    ref = b * (1.0 - a ** (t + 1)) / (1.0 - a)
    np.testing.assert_allclose(y[0, 0], ref, rtol=1e-14, atol=0)
    np.testing.assert_allclose(y[0, 1], ref, rtol=1e-14, atol=0)


def test_discrete_scan_product_form_brute_force():
    """h_t = sum_{s<=t} (prod_{r=s+1..t} a_r) b_s, y_t = C_t h_t + skip_t."""
    abar, bu, C, skip = _discrete_case(41, batch=2, Dc=2, L=11)
    y = oracle.discrete_scan(abar, bu, C, skip)
    a64, b64 = abar.astype(np.float64), bu.astype(np.float64)
    for bb in range(2):
        for d in range(2):
            for t in range(11):
                h = sum(np.prod(a64[bb, d, s + 1:t + 1]) * b64[bb, d, s] for s in range(t + 1))
                ref = float(C[bb, t]) * h + float(skip[bb, d, t])
                assert abs(y[bb, d, t] - ref) <= 1e-12 * max(1.0, abs(ref))


def test_channel_mean_matches_numpy():
    rng = np.random.default_rng(42)
    x = rng.standard_normal((3, 7, 19)).astype(np.float32)
    np.testing.assert_allclose(oracle.channel_mean(x), x.astype(np.float64).mean(axis=1),
                               rtol=1e-14, atol=1e-15)


def test_scan_of_channel_means_is_mean_of_scans_when_decay_shared():
    """Linearity: with abar the same on every channel, the one-channel scan of
    T(bu) (and T(skip)) is the channel mean of the per-channel scans."""
    abar, bu, C, skip = _discrete_case(43, batch=2, Dc=5, L=23)
    abar[...] = abar[:, :1, :]
    y = oracle.discrete_scan(abar, bu, C, skip)
    am = oracle.channel_mean(abar).astype(np.float32)[:, None, :]
    bm = oracle.channel_mean(bu).astype(np.float32)[:, None, :]
    sm = oracle.channel_mean(skip).astype(np.float32)[:, None, :]
    ym = oracle.discrete_scan(am, bm, C, sm)[:, 0]
    np.testing.assert_allclose(ym, y.mean(axis=1), rtol=1e-6, atol=1e-6)


def test_discrete_scan_degenerate_sizes():
    abar, bu, C, _ = _discrete_case(44, batch=1, Dc=1, L=1, with_skip=False)
    y = oracle.discrete_scan(abar, bu, C)
    assert y.shape == (1, 1, 1) and y[0, 0, 0] == float(C[0, 0]) * float(bu[0, 0, 0])


# ---------------------------------------------------------------- pooled reading (T over K*Dc)

def run_pooled(c):
    return oracle.mean_scan_pooled(c["u"], c["delta"], c["A"], c["B"], c["C"], c["D"],
                                   c["dt_bias"], c["softplus"])


def test_pooled_one_direction_is_direction_mean():
    """K = 1: the image's channels are the direction's, so pooling changes nothing."""
    c = rand_case(40, batch=2, K=1, Dc=5, L=9, N=3)
    ref = run_mean(c)[:, 0, 0, :]
    np.testing.assert_allclose(run_pooled(c), ref, rtol=1e-13, atol=1e-14)


def test_pooled_identical_directions_is_direction_mean():
    """Four identical directions (inputs, parameters, B and C): the mean over
    all K*Dc channels is the mean over one direction's."""
    c = rand_case(41, batch=2, K=4, Dc=3, L=8, N=3)
    for key in ("u", "delta", "B", "C"):
        c[key][...] = c[key][:, :1]
    A = c["A"].reshape(4, 3, 3)
    A[...] = A[:1]
    for key in ("D", "dt_bias"):
        v = c[key].reshape(4, 3)
        v[...] = v[:1]
    ref = run_mean(c)[:, 0, 0, :]
    np.testing.assert_allclose(run_pooled(c), ref, rtol=1e-13, atol=1e-14)


def test_pooled_identical_channels_is_full():
    """Every channel of every direction identical, B and C shared by the
    directions: the pooled scan is each channel's own full scan."""
    c = rand_case(42, batch=1, K=4, Dc=3, L=10, N=2)
    for key in ("u", "delta"):
        c[key][...] = c[key][:, :1, :1]
    for key in ("B", "C"):
        c[key][...] = c[key][:, :1]
    c["A"][...] = c["A"][:1]
    for key in ("D", "dt_bias"):
        c[key][...] = c[key][:1]
    ref = run_full(c)[:, 0, 0, :]
    np.testing.assert_allclose(run_pooled(c), ref, rtol=1e-13, atol=1e-14)


def test_pooled_is_mean_of_full_when_timescale_and_c_shared():
    """Delta and A shared by all K*Dc channels, C by the directions; u, D and
    B (per direction) free. The recurrence is then linear in Delta u B with a
    common decay, so the pooled output is exactly the mean of the full scan's
    outputs over all K*Dc channels: this fixes how B, u and D enter."""
    c = rand_case(43, batch=2, K=4, Dc=3, L=9, N=3)
    c["delta"][...] = c["delta"][:, :1, :1]
    c["A"][...] = c["A"][:1]
    c["dt_bias"][...] = c["dt_bias"][:1]
    c["C"][...] = c["C"][:, :1]
    yf = run_full(c)
    ref = yf.reshape(2, -1, 9).mean(axis=1)
    np.testing.assert_allclose(run_pooled(c), ref, rtol=1e-12, atol=1e-13)


def test_pooled_is_mean_of_full_when_only_c_differs():
    """All channels identical except C, which differs per direction: every
    channel has the same state, so the pooled output (the mean of C applied to
    it) is the mean of the full outputs: this fixes how C enters."""
    c = rand_case(44, batch=1, K=4, Dc=2, L=8, N=3)
    for key in ("u", "delta"):
        c[key][...] = c[key][:, :1, :1]
    c["B"][...] = c["B"][:, :1]
    c["A"][...] = c["A"][:1]
    for key in ("D", "dt_bias"):
        c[key][...] = c[key][:1]
    yf = run_full(c)
    ref = yf.reshape(1, -1, 8).mean(axis=1)
    np.testing.assert_allclose(run_pooled(c), ref, rtol=1e-12, atol=1e-13)


# ---------------------------------------------------------------- zero-order hold (eq. 4)

def test_zoh_is_exact_step_of_the_ode():
    """With u, B and Delta held over a step, ZOH is the exact solution of
    h' = A h + B u (eq. 1): each step equals the matrix exponential of the
    augmented system [[A, B u], [0, 0]] * Delta (Van Loan), by scipy."""
    import scipy.linalg
    c = rand_case(50, batch=1, K=1, Dc=2, L=6, N=3)
    y = oracle.full_scan(c["u"], c["delta"], c["A"], c["B"], c["C"], c["D"], c["dt_bias"],
                         True, options=oracle.ZOH)
    dl = timescale_np(c["delta"], c["dt_bias"], True, 1, 2)
    for d in range(2):
        h = np.zeros(3)
        for t in range(6):
            acc = 0.0
            for n in range(3):
                a = float(c["A"][d, n])
                bu = float(c["B"][0, 0, n, t]) * float(c["u"][0, 0, d, t])
                M = np.array([[a, bu], [0.0, 0.0]]) * dl[0, 0, d, t]
                E = scipy.linalg.expm(M)
                h[n] = E[0, 0] * h[n] + E[0, 1]
                acc += float(c["C"][0, 0, n, t]) * h[n]
            ref = acc + float(c["D"][d]) * float(c["u"][0, 0, d, t])
            assert abs(y[0, 0, d, t] - ref) <= 1e-12 * max(1.0, abs(ref))


def test_zoh_constant_inputs_closed_form():
    """Constant Delta, A, B, u: h_t = a h_{t-1} + (a - 1) B u / A sums to
    h_t = (a^(t+1) - 1) B u / A, which tends to the steady state -B u / A."""
    L = 40
    u = np.full((1, 1, 1, L), 0.7, np.float32)
    delta = np.full((1, 1, 1, L), 0.25, np.float32)
    A = np.array([[-1.5]], np.float32)
    B = np.full((1, 1, 1, L), 1.3, np.float32)
    C = np.ones((1, 1, 1, L), np.float32)
    y = oracle.full_scan(u, delta, A, B, C, None, None, False, options=oracle.ZOH)[0, 0, 0]
    a = math.exp(0.25 * -1.5)
    bu_over_a = float(np.float32(1.3)) * float(np.float32(0.7)) / -1.5
    for t in range(L):
        ref = (a ** (t + 1) - 1.0) * bu_over_a
        assert abs(y[t] - ref) <= 1e-13
    assert abs(y[-1] + bu_over_a) < 1e-6  # steady state -B u / A


def test_zoh_tends_to_euler_as_a_vanishes():
    """phi(x) = (e^x - 1)/x -> 1 as x -> 0: with a tiny A the two B-bar forms agree."""
    c = rand_case(51, batch=1, K=2, Dc=2, L=8, N=2)
    c["A"][...] = -1e-7
    ze = oracle.full_scan(c["u"], c["delta"], c["A"], c["B"], c["C"], c["D"], c["dt_bias"],
                          True, options=oracle.ZOH)
    eu = run_full(c)
    np.testing.assert_allclose(ze, eu, rtol=1e-6, atol=1e-9)
    assert not np.array_equal(ze, eu)


def test_zoh_mean_equals_full_when_channels_identical():
    c = rand_case(52, batch=2, K=2, Dc=4, L=9, N=3)
    for key in ("u", "delta"):
        c[key][...] = c[key][:, :, :1, :]
    A = c["A"].reshape(2, 4, 3)
    A[...] = A[:, :1, :]
    for key in ("D", "dt_bias"):
        v = c[key].reshape(2, 4)
        v[...] = v[:, :1]
    ym = run_mean(c, options=oracle.ZOH)
    yf = oracle.full_scan(c["u"], c["delta"], c["A"], c["B"], c["C"], c["D"], c["dt_bias"],
                          True, options=oracle.ZOH)
    np.testing.assert_allclose(ym, yf, rtol=1e-13, atol=1e-14)


def test_zoh_mean_is_channel_mean_of_full_when_timescale_shared():
    """Delta and A shared by a direction's channels: the ZOH gain is then
    common too, the recurrence linear in u, and the reduced output the channel
    mean of the full ZOH outputs."""
    c = rand_case(53, batch=1, K=3, Dc=5, L=10, N=3)
    c["delta"][...] = c["delta"][:, :, :1, :]
    A = c["A"].reshape(3, 5, 3)
    A[...] = A[:, :1, :]
    v = c["dt_bias"].reshape(3, 5)
    v[...] = v[:, :1]
    ym = run_mean(c, options=oracle.ZOH)
    yf = oracle.full_scan(c["u"], c["delta"], c["A"], c["B"], c["C"], c["D"], c["dt_bias"],
                          True, options=oracle.ZOH)
    ref = np.broadcast_to(yf.mean(axis=2, keepdims=True), yf.shape)
    np.testing.assert_allclose(ym, ref, rtol=1e-12, atol=1e-13)


# ---------------------------------------------------------------- selection projections (eq. 6)

def test_projections_brute_force():
    """Triple loops on a tiny case: x_dbl = W u per direction, B and C its rows
    R.. and R+N.., delta the rank-R expansion of its first R rows."""
    rng = np.random.default_rng(60)
    batch, K, Dc, L, N, R = 2, 3, 4, 5, 2, 3
    u = rng.standard_normal((batch, K, Dc, L)).astype(np.float32)
    pw = workloads.make_projection_weights(K, Dc, N, R, seed=61)
    delta, B, C = oracle.projections(u, pw.W, pw.W_dt, N=N)
    for b in range(batch):
        for k in range(K):
            for t in range(L):
                xd = [sum(float(pw.W[k, r, d]) * float(u[b, k, d, t]) for d in range(Dc))
                      for r in range(R + 2 * N)]
                for n in range(N):
                    assert abs(B[b, k, n, t] - xd[R + n]) < 1e-12
                    assert abs(C[b, k, n, t] - xd[R + N + n]) < 1e-12
                for d in range(Dc):
                    ref = sum(float(pw.W_dt[k, d, r]) * xd[r] for r in range(R))
                    assert abs(delta[b, k, d, t] - ref) < 1e-12


def test_projections_one_hot_input_reads_weight_columns():
    """u = e_j at one position: B, C there are column j of W's B and C rows,
    and zero elsewhere (a transposed W fails this)."""
    K, Dc, L, N, R = 2, 6, 4, 3, 2
    pw = workloads.make_projection_weights(K, Dc, N, R, seed=62)
    u = np.zeros((1, K, Dc, L), np.float32)
    u[0, 1, 4, 2] = 1.0
    delta, B, C = oracle.projections(u, pw.W, pw.W_dt, N=N)
    np.testing.assert_array_equal(B[0, 1, :, 2], pw.W[1, R:R + N, 4].astype(np.float64))
    np.testing.assert_array_equal(C[0, 1, :, 2], pw.W[1, R + N:, 4].astype(np.float64))
    mask = np.ones(L, bool)
    mask[2] = False
    assert not B[0, 1][:, mask].any() and not B[0, 0].any()
    ref = pw.W_dt[1].astype(np.float64) @ pw.W[1, :R, 4].astype(np.float64)
    np.testing.assert_allclose(delta[0, 1, :, 2], ref, rtol=1e-15, atol=0)


def test_projections_broadcast_timescale():
    """R = 1 without W_dt (Broadcast_D(Linear_1(u)) of eq. 6): delta is the
    same for every channel and equals the single timescale row of W times u."""
    rng = np.random.default_rng(63)
    u = rng.standard_normal((1, 2, 5, 7)).astype(np.float32)
    pw = workloads.make_projection_weights(2, 5, 4, 1, seed=64, broadcast=True)
    delta, _, _ = oracle.projections(u, pw.W, None, N=4)
    for k in range(2):
        ref = pw.W[k, 0].astype(np.float64) @ u[0, k].astype(np.float64)
        for d in range(5):
            np.testing.assert_allclose(delta[0, k, d], ref, rtol=1e-14, atol=1e-15)


# ---- the post-merge channel normalisation and gate (VMamba's SS2D step after
# the cross-merge; not in the paper's text, so pinned by definition and a
# library routine, not by paper values)

def test_out_norm_matches_torch_layer_norm():
    """Channel LayerNorm per pixel = torch's layer_norm over the last axis of
    the channel-last transpose (an independent library routine), fp64."""
    import torch

    rng = np.random.default_rng(70)
    b, Dc, P = 2, 9, 13
    y = rng.standard_normal((b, Dc, P)) * 3.0 + 1.5
    g = rng.standard_normal(Dc)
    be = rng.standard_normal(Dc)
    got = oracle.out_norm_gate(y, None, g, be, eps=1e-3)
    ref = torch.nn.functional.layer_norm(torch.from_numpy(y).permute(0, 2, 1), (Dc,),
                                         torch.from_numpy(g), torch.from_numpy(be), 1e-3)
    np.testing.assert_allclose(got, ref.permute(0, 2, 1).numpy(), rtol=1e-12, atol=1e-12)


def test_out_norm_hand_example():
    """One pixel, channels (1, 2, 3), eps 0: mean 2, biased variance 2/3, so the
    output is (-sqrt(3/2), 0, sqrt(3/2)); gamma (2, 2, 2) and beta (1, 1, 1)
    map it to 1 -+ sqrt(6)."""
    y = np.array([1.0, 2.0, 3.0]).reshape(1, 3, 1)
    got = oracle.out_norm_gate(y, eps=0.0)[0, :, 0]
    np.testing.assert_allclose(got, [-np.sqrt(1.5), 0.0, np.sqrt(1.5)], rtol=1e-15, atol=1e-15)
    got = oracle.out_norm_gate(y, None, np.full(3, 2.0), np.ones(3), eps=0.0)[0, :, 0]
    np.testing.assert_allclose(got, [1 - np.sqrt(6), 1.0, 1 + np.sqrt(6)], rtol=1e-15)


def test_out_norm_invariants():
    """gamma 1, beta 0, eps 0: every pixel's output has mean 0 and variance 1,
    and is unchanged by a positive scale and a per-pixel shift of y (the
    normalisation runs over channels, not pixels: a per-channel shift would
    change it)."""
    rng = np.random.default_rng(71)
    y = rng.standard_normal((3, 11, 7))
    out = oracle.out_norm_gate(y, eps=0.0)
    np.testing.assert_allclose(out.mean(axis=1), 0.0, atol=1e-14)
    np.testing.assert_allclose((out ** 2).mean(axis=1), 1.0, rtol=1e-13)
    shift = rng.standard_normal((3, 1, 7))
    np.testing.assert_allclose(oracle.out_norm_gate(2.5 * y + shift, eps=0.0), out, atol=1e-12)
    per_channel = rng.standard_normal((1, 11, 1))
    assert not np.allclose(oracle.out_norm_gate(y + per_channel, eps=0.0), out, atol=1e-3)


def test_out_gate_silu():
    """The gate is z * sigmoid(z). Textbook values: silu(1) = e / (1 + e),
    silu(-1) = -(1 - e / (1 + e)), silu(2) = 2 e^2 / (1 + e^2), silu(0) = 0; the mirrored form
    z * sigmoid(-z) gives 1 / (1 + e) at z = 1 and fails. The odd part
    silu(z) - silu(-z) = z holds for any z."""
    e = np.e
    y = np.array([1.0, 2.0, 3.0]).reshape(1, 3, 1)  # normalises to (-a, 0, a), a = sqrt(3/2)
    a = np.sqrt(1.5)
    for zv, silu in ((1.0, e / (1 + e)), (-1.0, -(1 - e / (1 + e))), (2.0, 2 * e * e / (1 + e * e))):
        z = np.full((1, 3, 1), zv)
        got = oracle.out_norm_gate(y, z, eps=0.0)[0, :, 0]
        np.testing.assert_allclose(got, [-a * silu, 0.0, a * silu], rtol=1e-14, atol=1e-15)
    rng = np.random.default_rng(72)
    y = rng.standard_normal((1, 5, 6))
    z = rng.standard_normal((1, 5, 6)) * 4.0
    n = oracle.out_norm_gate(y, eps=1e-5)
    diff = oracle.out_norm_gate(y, z, eps=1e-5) - oracle.out_norm_gate(y, -z, eps=1e-5)
    np.testing.assert_allclose(diff, n * z, rtol=1e-12, atol=1e-12)
    np.testing.assert_array_equal(oracle.out_norm_gate(y, np.zeros_like(y)), 0.0)
