// scan_full.hip -- full (per-channel) selective scan.
//
// Appendix A: eq. 3 recurrence h_t = Abar h_{t-1} + Bbar u_t, y_t = C h_t + D u_t,
// with Abar = exp(Delta A) (eq. 4, first line), Bbar u_t = Delta B_t u_t and
// Delta = softplus(delta + dt_bias) (eq. 6). One independent recurrence per
// (batch, direction k, channel d, state n); c = k*channels + d.
//
// Lane-per-channel kernel: each lane owns one channel and keeps all N states
// in registers while it walks the sequence. B[n, t] and C[n, t] are shared by
// every channel of a direction, so inside a wave (64 consecutive channels of
// one direction) their addresses are uniform and the compiler serves them
// from the scalar cache into SGPRs; the per-element work is then
// mul (Delta*A), exp2, mul (Delta*u*B), fma (state), fma (output).
// exp(Delta*A) is evaluated as exp2((Delta*log2 e) * A) so the log2 e scaling
// is paid once per (channel, position), not once per state.
#include "vmb_internal.h"

namespace vmb {
namespace {

constexpr int kWave = 64;

template <int N, typename Tin, typename Tout, bool kTwoD, bool kZoh>
__global__ __launch_bounds__(kWave) void k_full_scan_lanes(
    const Tin* __restrict__ u, const Tin* __restrict__ delta, const float* __restrict__ A,
    const Tin* __restrict__ Bm, const Tin* __restrict__ Cm, const float* __restrict__ D,
    const float* __restrict__ dt_bias, Tout* __restrict__ y, int K, int Dc, int L, int H, int W,
    int softplus) {
    const int d = blockIdx.x * kWave + threadIdx.x;
    const int k = blockIdx.y;
    const int b = blockIdx.z;
    if (d >= Dc) return;
    const int c = k * Dc + d;
    const size_t bk = static_cast<size_t>(b) * K + k;
    const size_t row = (bk * Dc + d) * static_cast<size_t>(L);

    float a_row[N], inv_a[N];
#pragma unroll
    for (int n = 0; n < N; ++n) {
        a_row[n] = A[static_cast<size_t>(c) * N + n];
        inv_a[n] = kZoh ? 1.0f / a_row[n] : 0.0f;
    }
    const float bias = dt_bias ? dt_bias[c] : 0.0f;
    const float dskip = D ? D[c] : 0.0f;
    const bool sp = softplus != 0;

    const Tin* drow = delta + row;
    const Tin* urow = kTwoD ? u + (static_cast<size_t>(b) * Dc + d) * L : u + row;
    const Tin* Bb = Bm + bk * N * L;
    const Tin* Cb = Cm + bk * N * L;
    Tout* yrow = y + row;

    float h[N];
#pragma unroll
    for (int n = 0; n < N; ++n) h[n] = 0.0f;

    for (int t = 0; t < L; ++t) {
        const int src = kTwoD ? pixel_of(k, t, H, W) : t;
        const float ut = to_f32(urow[src]);
        const float dl = timescale(to_f32(drow[t]) + bias, sp);
        const float dl2 = dl * kLog2e;
        const float du = dl * ut;
        float acc = dskip * ut;
#pragma unroll
        for (int n = 0; n < N; ++n) {
            const float x2 = dl2 * a_row[n];
            const float a = fast_exp2(x2);
            const float q = kZoh ? zoh_q(x2, a, du, ut, inv_a[n]) : du;
            const float bu = q * to_f32(Bb[n * L + t]);
            h[n] = __builtin_fmaf(a, h[n], bu);
            acc = __builtin_fmaf(to_f32(Cb[n * L + t]), h[n], acc);
        }
        yrow[t] = from_f32<Tout>(acc);
    }
}

template <int N, typename Tin, typename Tout, bool kTwoD, bool kZoh>
vmb_status launch_lanes_zoh(const ScanArgs& a, Tout* y) {
    const dim3 grid(static_cast<unsigned>((a.channels + kWave - 1) / kWave),
                    static_cast<unsigned>(a.K), static_cast<unsigned>(a.batch));
    hipLaunchKernelGGL((k_full_scan_lanes<N, Tin, Tout, kTwoD, kZoh>), grid, dim3(kWave), 0, a.stream,
                       static_cast<const Tin*>(a.u), static_cast<const Tin*>(a.delta), a.A,
                       static_cast<const Tin*>(a.B), static_cast<const Tin*>(a.C), a.D, a.dt_bias,
                       y, int(a.K), int(a.channels), int(a.L), int(a.H), int(a.W), a.softplus);
    return check_launch();
}

template <int N, typename Tin, typename Tout, bool kTwoD>
vmb_status launch_lanes(const ScanArgs& a, Tout* y) {
    return (a.options & VMB_SCAN_ZOH) ? launch_lanes_zoh<N, Tin, Tout, kTwoD, true>(a, y)
                                      : launch_lanes_zoh<N, Tin, Tout, kTwoD, false>(a, y);
}

template <int N, typename Tin, typename Tout>
vmb_status dispatch_layout(const ScanArgs& a) {
    if (a.layout == VMB_LAYOUT_SEQ) return launch_lanes<N, Tin, Tout, false>(a, static_cast<Tout*>(a.y));
    // 2-D: per-direction fp32 outputs into the workspace, then the merge pass
    float* ys = static_cast<float*>(a.ws);
    vmb_status st = launch_lanes<N, Tin, float, true>(a, ys);
    if (st != VMB_OK) return st;
    return launch_cross_merge(ys, a.y, a.batch, a.channels, a.H, a.W, VMB_F32, a.out_dt, a.stream);
}

template <int N>
vmb_status dispatch_dtype(const ScanArgs& a) {
    if (a.in_dt == VMB_F32) return dispatch_layout<N, float, float>(a);
    if (a.out_dt == VMB_BF16) return dispatch_layout<N, bf16_t, bf16_t>(a);
    return dispatch_layout<N, bf16_t, float>(a);
}

}  // namespace

// The chunked kernel copies B and C rows into LDS in pieces of 4 or 16
// bytes; a bf16 row of odd length has neither its start nor its end on a
// 4-byte boundary, so those shapes take the lane-per-channel kernel.
bool use_chunked_full(const ScanArgs& a) {
    return a.N == 16 && a.L > kShortMaxL && !(a.in_dt == VMB_BF16 && (a.L & 1));
}

vmb_status launch_full_scan(const ScanArgs& a) {
    // the zero-order-hold B runs in the tile, positions-over-lanes and lane
    // kernels (not the short-sequence one: those shapes take the tile kernel)
    const bool zoh = (a.options & VMB_SCAN_ZOH) != 0;
    const bool tiles =
        use_tiles_full(a) || (zoh && !use_chunked_full(a) && tiles_take(a));
    if (tiles || use_chunked_full(a) || (!zoh && use_short_full(a))) {
        auto run = [&](void* y_seq, const void* xt) {
            if (tiles) return launch_full_tiles(a, y_seq, xt);
            return use_short_full(a) ? launch_full_short(a, y_seq) : launch_full_chunked(a, y_seq, xt);
        };
        if (a.layout == VMB_LAYOUT_SEQ) return run(a.y, nullptr);
        // 2-D: the tile path, and the positions-over-lanes path on sequences of
        // several chunks, read directions 1 and 3 from column-major plane
        // copies in the workspace
        const void* xt = nullptr;
        const bool chunked_long = !tiles && !use_short_full(a) && a.L > kChunkedOneChunkMaxL;
        if ((tiles || chunked_long) && full_ws_has_xt(a.batch, a.K, a.channels, a.L, a.N)) {
            void* xtw = static_cast<char*>(a.ws) + full_ws_xt_offset(a.batch, a.K, a.channels, a.L);
            vmb_status st = launch_transpose_planes(a.u, xtw, a.batch, a.channels, a.H, a.W,
                                                    a.in_dt, a.stream);
            if (st != VMB_OK) return st;
            xt = xtw;
        }
        vmb_status st = run(a.ws, xt);
        if (st != VMB_OK) return st;
        return launch_cross_merge(a.ws, a.y, a.batch, a.channels, a.H, a.W, VMB_F32, a.out_dt,
                                  a.stream);
    }
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
