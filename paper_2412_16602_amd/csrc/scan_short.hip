// scan_short.hip -- full selective scan for short sequences (the 14 x 14 and
// 7 x 7 stages of VMamba), N = 16.
//
// Same recurrence as scan_full.hip (Appendix A: eq. 3, eq. 4 first line,
// eq. 6). A wave holds 64 / S channels; each channel's whole sequence lies in
// one segment of S lanes, each lane owning a run of T consecutive positions
// (L <= S * T). Per state a lane forms exp(Delta A) and Delta B u for its run
// (registers), composes them into the run aggregate, and an inclusive scan of
// the aggregates over the segment's lanes (DPP within rows of 16 lanes, plus
// the row broadcast for S = 32) gives the state entering each run; the lane
// then re-walks its run accumulating y += C h. The combine is
// (a1, b1) then (a2, b2) -> (a1 a2, a2 b1 + b2).
//
// Every sequence is a single chunk, so waves never exchange state: the only
// workgroup barrier follows the copy of the direction's B and C rows (all
// states, all positions) into LDS. Outputs leave through a per-wave LDS slice
// and are stored lane-contiguous.
#include "vmb_internal.h"

namespace vmb {
namespace {

constexpr int kWave = 64;
constexpr int kShortWaves = 8;
constexpr int kShortThreads = kShortWaves * kWave;
constexpr int kWaveShr1 = 0x138;  // DPP wave_shr:1 (GFX9 encoding)

__device__ __forceinline__ float shr1(float old, float v) {
    return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(__builtin_bit_cast(int, old),
                                                                 __builtin_bit_cast(int, v),
                                                                 kWaveShr1, 0xf, 0xf, false));
}

// T consecutive elements from p (first cnt valid, the rest 0).
template <int T, typename Tin>
__device__ __forceinline__ void load_seq(const Tin* p, float (&v)[T], int cnt) {
#pragma unroll
    for (int i = 0; i < T; ++i) v[i] = i < cnt ? to_f32(p[i]) : 0.0f;
}

// u values of a run in the 2-D layout: position t of direction k reads pixel
// pixel_of(k, t); rows are walked incrementally for the column-major maps.
template <int T, typename Tin>
__device__ __forceinline__ void load_seq_2d(const Tin* plane, int k, int t0, int H, int W, int L,
                                            float (&v)[T], int cnt) {
    const int tt = (k >= 2) ? (L - 1 - t0) : t0;
    if ((k & 1) == 0) {
        const int step = (k >= 2) ? -1 : 1;
#pragma unroll
        for (int i = 0; i < T; ++i) v[i] = i < cnt ? to_f32(plane[tt + step * i]) : 0.0f;
        return;
    }
    int w = tt / H;
    int h = tt - w * H;
    const bool rev = k >= 2;
#pragma unroll
    for (int i = 0; i < T; ++i) {
        v[i] = i < cnt ? to_f32(plane[h * W + w]) : 0.0f;
        if (!rev) {
            if (++h == H) { h = 0; ++w; }
        } else {
            if (--h < 0) { h = H - 1; --w; }
        }
    }
}

template <int N, int S, int T, typename Tin, typename Tout, bool kTwoD>
__global__ __launch_bounds__(kShortThreads) void k_full_scan_short(
    const Tin* __restrict__ u, const Tin* __restrict__ delta, const float* __restrict__ A,
    const Tin* __restrict__ Bm, const Tin* __restrict__ Cm, const float* __restrict__ D,
    const float* __restrict__ dt_bias, Tout* __restrict__ y, int K, int Dc, int L, int H, int W,
    int softplus) {
    constexpr int kCpw = kWave / S;            // channels per wave
    constexpr int G = kShortWaves * kCpw;     // channels per workgroup
    constexpr int kSeg = S * T;               // positions one segment covers (>= L)
    __shared__ Tin bst[N * kSeg], cst[N * kSeg];  // B, C rows [n][t] of this (batch, k)
    __shared__ __align__(16) float ystage[kShortWaves][kWave * T];

    const int k = blockIdx.y, b = blockIdx.z;
    const size_t bk = static_cast<size_t>(b) * K + k;
    const int tid = threadIdx.x;
    const int lane = tid % kWave;
    const int wv = __builtin_amdgcn_readfirstlane(tid / kWave);

    // B and C of this direction: N rows of L, packed with row stride L
    {
        const Tin* Bg = Bm + bk * N * L;
        const Tin* Cg = Cm + bk * N * L;
        const int total = N * L;
        constexpr int kBatch = 8;  // loads in flight per thread before their stores
        for (int base = tid; base < total; base += kBatch * kShortThreads) {
            Tin bv[kBatch], cv[kBatch];
#pragma unroll
            for (int j = 0; j < kBatch; ++j) {
                const int idx = base + j * kShortThreads;
                if (idx < total) {
                    bv[j] = Bg[idx];
                    cv[j] = Cg[idx];
                }
            }
#pragma unroll
            for (int j = 0; j < kBatch; ++j) {
                const int idx = base + j * kShortThreads;
                if (idx < total) {
                    bst[idx] = bv[j];
                    cst[idx] = cv[j];
                }
            }
        }
    }

    // this lane: channel slot cw of the wave, run sl of the segment
    const int cw = lane / S, sl = lane % S;
    const int d_raw = blockIdx.x * G + wv * kCpw + cw;
    const int d = d_raw < Dc ? d_raw : Dc - 1;  // slots past Dc compute a copy, not stored
    const int c = k * Dc + d;
    const int run = sl * T;
    const int cnt = L - run < T ? (L - run > 0 ? L - run : 0) : T;
    const size_t row = (bk * Dc + d) * static_cast<size_t>(L);
    float dv[T], uv[T];
    load_seq<T>(delta + row + (cnt > 0 ? run : 0), dv, cnt);
    if constexpr (kTwoD)
        load_seq_2d<T>(u + (static_cast<size_t>(b) * Dc + d) * L, k, cnt > 0 ? run : 0, H, W, L, uv,
                       cnt);
    else
        load_seq<T>(u + row + (cnt > 0 ? run : 0), uv, cnt);
    float an[N];
#pragma unroll
    for (int n = 0; n < N; ++n) an[n] = A[static_cast<size_t>(c) * N + n];
    const float bias = dt_bias ? dt_bias[c] : 0.0f;
    const float dskip = D ? D[c] : 0.0f;
    const bool sp = softplus != 0;

    float dl2[T], du[T], yv[T];
    float s2 = 0.0f;
#pragma unroll
    for (int i = 0; i < T; ++i) {
        // positions past the end act as the identity: a = 1, b = 0
        float dl = sp ? timescale(dv[i] + bias, true) : dv[i] + bias;
        dl = i < cnt ? dl : 0.0f;
        dl2[i] = dl * kLog2e;
        du[i] = dl * uv[i];
        yv[i] = dskip * uv[i];
        s2 += dl2[i];
    }
    __syncthreads();  // B, C staged

    const int rb = cnt > 0 ? run : 0;  // keep LDS reads in range for empty runs
#pragma unroll 1
    for (int n = 0; n < N; ++n) {
        const Tin* bsrc = bst + n * L + rb;
        const Tin* csrc = cst + n * L + rb;
        float a[T], bu[T];
        float agg = 0.0f;
#pragma unroll
        for (int i = 0; i < T; ++i) {
            a[i] = fast_exp2(dl2[i] * an[n]);
            bu[i] = du[i] * (i < cnt ? to_f32(bsrc[i]) : 0.0f);
            agg = __builtin_fmaf(a[i], agg, bu[i]);
        }
        float P = fast_exp2(s2 * an[n]);
        float Hs = agg;
        seg_scan<S>(P, Hs);
        // state entering this run: the inclusive value of lane - 1 in the
        // segment (the segment's first lane starts from h = 0)
        const float hex = shr1(0.0f, Hs);
        float h = sl == 0 ? 0.0f : hex;
#pragma unroll
        for (int i = 0; i < T; ++i) {
            h = __builtin_fmaf(a[i], h, bu[i]);
            yv[i] = __builtin_fmaf(i < cnt ? to_f32(csrc[i]) : 0.0f, h, yv[i]);
        }
    }

    // outputs through the wave's LDS slice: segment cw's row is contiguous
    float* slice = ystage[wv];
#pragma unroll
    for (int i = 0; i < T; ++i) slice[lane * T + i] = yv[i];
#pragma unroll
    for (int r = 0; r < kCpw; ++r) {
        const int dr = blockIdx.x * G + wv * kCpw + r;
        if (dr >= Dc) break;
        Tout* yrow = y + (bk * Dc + dr) * static_cast<size_t>(L);
        const float* src = slice + r * kSeg;
        for (int j = lane; j < L; j += kWave) yrow[j] = from_f32<Tout>(src[j]);
    }
}

template <int N, int S, int T, typename Tin, typename Tout, bool kTwoD>
vmb_status launch_short_st(const ScanArgs& a, Tout* y) {
    constexpr int G = kShortWaves * (kWave / S);
    const long long groups = (a.channels + G - 1) / G;
    if (groups > 0x7fffffffLL || a.K > 65535 || a.batch > 65535) return VMB_ERR_UNSUPPORTED;
    const dim3 grid(static_cast<unsigned>(groups), static_cast<unsigned>(a.K),
                    static_cast<unsigned>(a.batch));
    hipLaunchKernelGGL((k_full_scan_short<N, S, T, Tin, Tout, kTwoD>), grid, dim3(kShortThreads), 0,
                       a.stream, static_cast<const Tin*>(a.u), static_cast<const Tin*>(a.delta),
                       a.A, static_cast<const Tin*>(a.B), static_cast<const Tin*>(a.C), a.D,
                       a.dt_bias, y, int(a.K), int(a.channels), int(a.L), int(a.H), int(a.W),
                       a.softplus);
    return check_launch();
}

// Segment shape from L: 16 lanes x 4 positions up to 64, 16 x 13 up to 208,
// 32 x 13 up to 416.
template <int N, typename Tin, typename Tout, bool kTwoD>
vmb_status launch_short_impl(const ScanArgs& a, Tout* y) {
    if (a.L <= 16 * 4) return launch_short_st<N, 16, 4, Tin, Tout, kTwoD>(a, y);
    if (a.L <= 16 * 13) return launch_short_st<N, 16, 13, Tin, Tout, kTwoD>(a, y);
    return launch_short_st<N, 32, 13, Tin, Tout, kTwoD>(a, y);
}

}  // namespace

bool use_short_full(const ScanArgs& a) { return a.N == 16 && a.L <= kShortMaxL; }

vmb_status launch_full_short(const ScanArgs& a, void* y_seq) {
    if (a.N != 16 || a.L > kShortMaxL) return VMB_ERR_UNSUPPORTED;
    const bool two_d = a.layout == VMB_LAYOUT_2D;
    if (a.in_dt == VMB_F32)
        return two_d ? launch_short_impl<16, float, float, true>(a, static_cast<float*>(y_seq))
                     : launch_short_impl<16, float, float, false>(a, static_cast<float*>(y_seq));
    if (two_d) return launch_short_impl<16, bf16_t, float, true>(a, static_cast<float*>(y_seq));
    if (a.out_dt == VMB_BF16)
        return launch_short_impl<16, bf16_t, bf16_t, false>(a, static_cast<bf16_t*>(y_seq));
    return launch_short_impl<16, bf16_t, float, false>(a, static_cast<float*>(y_seq));
}

}  // namespace vmb
