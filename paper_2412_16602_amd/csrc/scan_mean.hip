// scan_mean.hip -- VMeanba channel-mean selective scan.
//
// Section 2.2, eq. 9: y = T^-1(Mamba(T(Abar, Bbar u, C))), T the mean over the
// inner channel axis, T^-1 the broadcast back. Per (batch, direction k) and
// position t, over the channels d of that direction (c = k*channels + d):
//   Abar_mean[n,t] = mean_d exp(Delta_{d,t} A[c,n])
//   s_mean[t]      = mean_d Delta_{d,t} u_{d,t}      (Bbar u reduced = B[n,t] s_mean[t])
//   r_mean[t]      = mean_d D[c] u_{d,t}             (skip term, reduced with the scan)
// then one N-state recurrence per (batch, k) and the broadcast of its output.
//
// Three passes over chunks of kMeanChunk positions:
//   1. reduce : lanes own positions, each of the 4 waves sums a fixed quarter
//               of the channels (coalesced loads along t, channel parameters
//               wave-uniform), the quarters are added in a fixed order; the
//               reduced tile is written to the workspace together with each
//               chunk's scan aggregate (prod Abar, local end state) from a
//               wave-level inclusive scan of the (a, b) pairs;
//   2. carry  : one lane per (batch, k, n) walks the chunk aggregates and
//               stores each chunk's incoming state;
//   3. finish : re-runs the chunk's wave-level scan from its incoming state,
//               forms ytilde and broadcasts it to every channel (sequence
//               layout) or stores it for the merge-and-broadcast pass (2-D).
// The (a, b) combine is (a1, b1) then (a2, b2) -> (a1 a2, a2 b1 + b2).
#include "vmb_internal.h"

namespace vmb {
namespace {

constexpr int kC = kMeanChunk;  // positions per chunk = lanes per wave
constexpr int kWaves = 4;

// Inclusive scan over the 64 lanes of a wave of the (a, b) pairs, in lane
// order: on return lane i holds the composition of lanes 0..i.
__device__ __forceinline__ void wave_scan(float& a, float& b, int lane) {
#pragma unroll
    for (int off = 1; off < kC; off <<= 1) {
        const float pa = __shfl_up(a, off, kC);
        const float pb = __shfl_up(b, off, kC);
        if (lane >= off) {
            b = __builtin_fmaf(a, pb, b);
            a = a * pa;
        }
    }
}

template <int N, typename Tin, bool kTwoD>
__global__ __launch_bounds__(kC* kWaves) void k_mean_reduce(
    const Tin* __restrict__ u, const Tin* __restrict__ delta, const float* __restrict__ A,
    const Tin* __restrict__ Bm, const float* __restrict__ D, const float* __restrict__ dt_bias,
    float* __restrict__ red, float* __restrict__ agg, int K, int Dc, int L, int H, int W,
    int nchunks, int softplus) {
    __shared__ float part[kWaves][N + 2][kC];
    const int chunk = blockIdx.x, k = blockIdx.y, b = blockIdx.z;
    const int lane = threadIdx.x % kC, wv = threadIdx.x / kC;
    const int t = chunk * kC + lane;
    const bool valid = t < L;
    const int tc = valid ? t : L - 1;  // clamped: every address below stays in bounds
    const size_t bk = static_cast<size_t>(b) * K + k;
    const bool sp = softplus != 0;
    const int src = kTwoD ? pixel_of(k, tc, H, W) : tc;

    float acc[N];
#pragma unroll
    for (int n = 0; n < N; ++n) acc[n] = 0.0f;
    float s = 0.0f, r = 0.0f;
    const int d0 = (wv * Dc) / kWaves, d1 = ((wv + 1) * Dc) / kWaves;
    for (int d = d0; d < d1; ++d) {
        const int c = k * Dc + d;
        const size_t row = (bk * Dc + d) * static_cast<size_t>(L);
        const size_t urow = kTwoD ? (static_cast<size_t>(b) * Dc + d) * L : row;
        const float dv = valid ? to_f32(delta[row + tc]) : 0.0f;
        const float uv = valid ? to_f32(u[urow + src]) : 0.0f;
        const float bias = dt_bias ? dt_bias[c] : 0.0f;
        const float dl = timescale(dv + bias, sp);
        const float dl2 = dl * kLog2e;
#pragma unroll
        for (int n = 0; n < N; ++n) acc[n] += fast_exp2(dl2 * A[static_cast<size_t>(c) * N + n]);
        s = __builtin_fmaf(dl, uv, s);
        r = __builtin_fmaf(D ? D[c] : 0.0f, uv, r);
    }
#pragma unroll
    for (int n = 0; n < N; ++n) part[wv][n][lane] = acc[n];
    part[wv][N][lane] = s;
    part[wv][N + 1][lane] = r;
    __syncthreads();
    if (wv != 0) return;

    const float inv = 1.0f / static_cast<float>(Dc);
    float* redbk = red + bk * (N + 2) * L;
    float sm = 0.0f;
    for (int w = 0; w < kWaves; ++w) sm += part[w][N][lane];
    sm *= inv;
    float rm = 0.0f;
    for (int w = 0; w < kWaves; ++w) rm += part[w][N + 1][lane];
    rm *= inv;
    if (valid) {
        redbk[static_cast<size_t>(N) * L + t] = sm;
        redbk[static_cast<size_t>(N + 1) * L + t] = rm;
    }
    float* aggc = agg + (bk * nchunks + chunk) * N * 2;
#pragma unroll
    for (int n = 0; n < N; ++n) {
        float am = 0.0f;
        for (int w = 0; w < kWaves; ++w) am += part[w][n][lane];
        am *= inv;
        if (valid) redbk[static_cast<size_t>(n) * L + t] = am;
        float a = valid ? am : 1.0f;
        float bb = valid ? to_f32(Bm[(bk * N + n) * L + tc]) * sm : 0.0f;
        wave_scan(a, bb, lane);
        if (lane == kC - 1) {
            aggc[2 * n] = a;
            aggc[2 * n + 1] = bb;
        }
    }
}

__global__ __launch_bounds__(64) void k_mean_carry(const float* __restrict__ agg,
                                                   float* __restrict__ carry, int lanes, int N,
                                                   int nchunks) {
    const int i = blockIdx.x * 64 + threadIdx.x;
    if (i >= lanes) return;
    const size_t bk = i / N;
    const int n = i - static_cast<int>(bk) * N;
    float h = 0.0f;
    for (int c = 0; c < nchunks; ++c) {
        const size_t o = (bk * nchunks + c) * N + n;
        carry[o] = h;
        h = __builtin_fmaf(agg[2 * o], h, agg[2 * o + 1]);
    }
}

template <int N, typename Tin, typename Tout, bool kTwoD>
__global__ __launch_bounds__(kC* kWaves) void k_mean_finish(
    const float* __restrict__ red, const float* __restrict__ carry, const Tin* __restrict__ Bm,
    const Tin* __restrict__ Cm, Tout* __restrict__ y, float* __restrict__ ytil, int K, int Dc,
    int L, int nchunks) {
    __shared__ float ybuf[kC];
    const int chunk = blockIdx.x, k = blockIdx.y, b = blockIdx.z;
    const int lane = threadIdx.x % kC, wv = threadIdx.x / kC;
    const int t = chunk * kC + lane;
    const bool valid = t < L;
    const int tc = valid ? t : L - 1;  // clamped: every address below stays in bounds
    const size_t bk = static_cast<size_t>(b) * K + k;
    if (wv == 0) {
        const float* redbk = red + bk * (N + 2) * L;
        const float* carc = carry + (bk * nchunks + chunk) * N;
        const float sm = valid ? redbk[static_cast<size_t>(N) * L + tc] : 0.0f;
        float acc = valid ? redbk[static_cast<size_t>(N + 1) * L + tc] : 0.0f;
#pragma unroll
        for (int n = 0; n < N; ++n) {
            float a = valid ? redbk[static_cast<size_t>(n) * L + tc] : 1.0f;
            float bb = valid ? to_f32(Bm[(bk * N + n) * L + tc]) * sm : 0.0f;
            wave_scan(a, bb, lane);
            const float h = __builtin_fmaf(a, carc[n], bb);
            const float cv = valid ? to_f32(Cm[(bk * N + n) * L + tc]) : 0.0f;
            acc = __builtin_fmaf(cv, h, acc);
        }
        ybuf[lane] = acc;
        if (kTwoD && valid) ytil[bk * L + t] = acc;
    }
    if (kTwoD) return;
    __syncthreads();
    if (!valid) return;
    const float v = ybuf[lane];
    const Tout o = from_f32<Tout>(v);
    for (int d = wv; d < Dc; d += kWaves) y[(bk * Dc + d) * static_cast<size_t>(L) + t] = o;
}

// 2-D layout: fold the four reduced sequences of each batch element into one
// map, (y0 + y2) + (y1 + y3) per pixel, and broadcast it to every channel.
template <typename Tout>
__global__ __launch_bounds__(256) void k_mean_merge_broadcast(const float* __restrict__ ytil,
                                                              Tout* __restrict__ y, int Dc, int H,
                                                              int W) {
    const int L = H * W;
    const int p = blockIdx.x * 256 + threadIdx.x;
    const int b = blockIdx.y;
    if (p >= L) return;
    const int hh = p / W, ww = p - hh * W;
    const int q = ww * H + hh;
    const float* yb = ytil + static_cast<size_t>(b) * 4 * L;
    const float s02 = yb[p] + yb[2 * static_cast<size_t>(L) + (L - 1 - p)];
    const float s13 = yb[static_cast<size_t>(L) + q] + yb[3 * static_cast<size_t>(L) + (L - 1 - q)];
    const Tout o = from_f32<Tout>(s02 + s13);
    Tout* yp = y + static_cast<size_t>(b) * Dc * L + p;
    for (int d = 0; d < Dc; ++d) yp[static_cast<size_t>(d) * L] = o;
}

template <int N, typename Tin, typename Tout, bool kTwoD>
vmb_status run(const ScanArgs& a) {
    const int nchunks = static_cast<int>((a.L + kC - 1) / kC);
    const size_t bkn = static_cast<size_t>(a.batch * a.K);
    auto round_up = [](size_t v) { return (v + 255) & ~size_t{255}; };
    char* ws = static_cast<char*>(a.ws);
    float* red = reinterpret_cast<float*>(ws);
    ws += round_up(bkn * (N + 2) * a.L * 4);
    float* agg = reinterpret_cast<float*>(ws);
    ws += round_up(bkn * nchunks * N * 2 * 4);
    float* carry = reinterpret_cast<float*>(ws);
    ws += round_up(bkn * nchunks * N * 4);
    float* ytil = kTwoD ? reinterpret_cast<float*>(ws) : nullptr;

    const dim3 grid(nchunks, static_cast<unsigned>(a.K), static_cast<unsigned>(a.batch));
    const dim3 block(kC * kWaves);
    const int K = int(a.K), Dc = int(a.channels), L = int(a.L), H = int(a.H), W = int(a.W);
    hipLaunchKernelGGL((k_mean_reduce<N, Tin, kTwoD>), grid, block, 0, a.stream,
                       static_cast<const Tin*>(a.u), static_cast<const Tin*>(a.delta), a.A,
                       static_cast<const Tin*>(a.B), a.D, a.dt_bias, red, agg, K, Dc, L, H, W,
                       nchunks, a.softplus);
    vmb_status st = check_launch();
    if (st != VMB_OK) return st;
    const int lanes = static_cast<int>(bkn * N);
    hipLaunchKernelGGL(k_mean_carry, dim3((lanes + 63) / 64), dim3(64), 0, a.stream, agg, carry,
                       lanes, N, nchunks);
    st = check_launch();
    if (st != VMB_OK) return st;
    hipLaunchKernelGGL((k_mean_finish<N, Tin, Tout, kTwoD>), grid, block, 0, a.stream, red, carry,
                       static_cast<const Tin*>(a.B), static_cast<const Tin*>(a.C),
                       static_cast<Tout*>(a.y), ytil, K, Dc, L, nchunks);
    st = check_launch();
    if (st != VMB_OK || !kTwoD) return st;
    hipLaunchKernelGGL(k_mean_merge_broadcast<Tout>, dim3((L + 255) / 256, unsigned(a.batch)),
                       dim3(256), 0, a.stream, ytil, static_cast<Tout*>(a.y), Dc, H, W);
    return check_launch();
}

template <int N, typename Tin, typename Tout>
vmb_status dispatch_layout(const ScanArgs& a) {
    return a.layout == VMB_LAYOUT_SEQ ? run<N, Tin, Tout, false>(a) : run<N, Tin, Tout, true>(a);
}

template <int N>
vmb_status dispatch_dtype(const ScanArgs& a) {
    if (a.in_dt == VMB_F32) return dispatch_layout<N, float, float>(a);
    if (a.out_dt == VMB_BF16) return dispatch_layout<N, bf16_t, bf16_t>(a);
    return dispatch_layout<N, bf16_t, float>(a);
}

}  // namespace

vmb_status launch_mean_scan(const ScanArgs& a) {
    if (a.batch > 65535 || a.K > 65535) return VMB_ERR_UNSUPPORTED;
    switch (a.N) {
        case 1: return dispatch_dtype<1>(a);
        case 2: return dispatch_dtype<2>(a);
        case 4: return dispatch_dtype<4>(a);
        case 8: return dispatch_dtype<8>(a);
        case 16: return dispatch_dtype<16>(a);
        default: return VMB_ERR_UNSUPPORTED;
    }
}

}  // namespace vmb
