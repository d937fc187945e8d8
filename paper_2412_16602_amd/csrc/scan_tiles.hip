// scan_tiles.hip -- full selective scan for grids with many channel rows
// (the batched VMamba stages), N = 16.
//
// Same recurrence as scan_full.hip (Appendix A: eq. 3, eq. 4 first line,
// eq. 6): h_t = exp(Delta_t A_n) h_{t-1} + Delta_t B_t u_t from h_{-1} = 0,
// y_t = sum_n C_t h_t + D u_t, Delta = softplus(delta + dt_bias).
//
// Work decomposition. A workgroup owns 64 channels of one (batch, direction)
// and walks the sequence in tiles of 16 positions. Lanes are channels; the
// 16 states are split over the four waves, four each, so every lane runs four
// independent recurrences straight along the sequence: no cross-lane scan,
// no re-walk. Per (channel, state, position): mul, exp2, mul, fma, fma.
//   - B[n, t] and C[n, t] are the same for every channel of a direction, so a
//     wave's four rows are wave-uniform: they are read with scalar loads into
//     SGPRs and used as the scalar operand of the VALU instructions.
//   - delta and u arrive in coalesced row pieces (each thread 4 positions of
//     one channel), are discretized once per (channel, position) by the
//     thread that loaded them (Delta log2 e, Delta u, D u) and transposed
//     through LDS for the channel-per-lane walk.
//   - Each wave's partial output (its four states' C h) goes back through LDS
//     and the loading threads add the four partials and D u, then store y
//     with row-contiguous vectors.
// Two workgroup barriers per tile; the next tile's delta / u loads, and one
// load per B / C row segment that brings those lines into L2, are in flight
// while the current tile is scanned.
//
// Workgroups are numbered so that those sharing a (batch, direction), and
// therefore B and C, land on the same XCD and its L2.
#include <type_traits>

#include "vmb_internal.h"

namespace vmb {
namespace {

constexpr int kWave = 64;
constexpr int kTileWaves = 4;                     // four states per wave
constexpr int kTileThreads = kTileWaves * kWave;  // 256
constexpr int kTP = 16;                           // positions per tile
constexpr int kStride = kTP + 1;                  // LDS row stride (words): conflict-free columns

// Four consecutive elements of a row starting at p: vector load when vec
// (16-byte fp32 / 8-byte bf16 aligned and all in range), else cnt guarded
// element loads, the rest 0.
__device__ __forceinline__ void load4(const float* p, float (&v)[4], bool vec, int cnt) {
    if (vec) {
        const float4 q = *reinterpret_cast<const float4*>(p);
        v[0] = q.x;
        v[1] = q.y;
        v[2] = q.z;
        v[3] = q.w;
    } else {
#pragma unroll
        for (int e = 0; e < 4; ++e) v[e] = e < cnt ? p[e] : 0.0f;
    }
}
__device__ __forceinline__ void load4(const bf16_t* p, float (&v)[4], bool vec, int cnt) {
    if (vec) {
        const uint2 q = *reinterpret_cast<const uint2*>(p);
        v[0] = __uint_as_float(q.x << 16);
        v[1] = __uint_as_float(q.x & 0xffff0000u);
        v[2] = __uint_as_float(q.y << 16);
        v[3] = __uint_as_float(q.y & 0xffff0000u);
    } else {
#pragma unroll
        for (int e = 0; e < 4; ++e) v[e] = e < cnt ? to_f32(p[e]) : 0.0f;
    }
}

template <bool kNt>
__device__ __forceinline__ void store4(float* p, const float (&v)[4], bool vec, int cnt) {
    if (vec) {
        if constexpr (kNt)
            store_out<true>(reinterpret_cast<float4*>(p), make_float4(v[0], v[1], v[2], v[3]));
        else
            *reinterpret_cast<float4*>(p) = make_float4(v[0], v[1], v[2], v[3]);
    } else {
#pragma unroll
        for (int e = 0; e < 4; ++e)
            if (e < cnt) p[e] = v[e];
    }
}
template <bool kNt>
__device__ __forceinline__ void store4(bf16_t* p, const float (&v)[4], bool vec, int cnt) {
    if (vec) {
        bf16_t o[4] = {from_f32<bf16_t>(v[0]), from_f32<bf16_t>(v[1]), from_f32<bf16_t>(v[2]),
                       from_f32<bf16_t>(v[3])};
        if constexpr (kNt) {
            unsigned long long q;
            __builtin_memcpy(&q, o, sizeof(o));
            store_out<true>(reinterpret_cast<unsigned long long*>(p), q);
        } else {
            __builtin_memcpy(p, o, sizeof(o));
        }
    } else {
#pragma unroll
        for (int e = 0; e < 4; ++e)
            if (e < cnt) p[e] = from_f32<bf16_t>(v[e]);
    }
}

// Eight consecutive elements of a wave-uniform B or C row from element
// offset off (scalar loads). bf16: off is even (even L, even tile starts),
// so the elements are four whole 32-bit words.
__device__ __forceinline__ void row8(const float* r, int off, float (&v)[8]) {
#pragma unroll
    for (int e = 0; e < 8; ++e) v[e] = r[off + e];
}
__device__ __forceinline__ void row8(const bf16_t* r, int off, float (&v)[8]) {
    const uint32_t* w = reinterpret_cast<const uint32_t*>(r) + (off >> 1);
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        const uint32_t x = w[q];
        v[2 * q] = __uint_as_float(x << 16);
        v[2 * q + 1] = __uint_as_float(x & 0xffff0000u);
    }
}

template <typename Tin, typename Tout, bool kTwoD, bool kZoh, bool kNt>
__global__ __launch_bounds__(kTileThreads) void k_full_scan_tiles(
    const Tin* __restrict__ u, const Tin* __restrict__ delta, const float* __restrict__ A,
    const Tin* __restrict__ Bm, const Tin* __restrict__ Cm, const float* __restrict__ D,
    const float* __restrict__ dt_bias, Tout* __restrict__ y, const Tin* __restrict__ xt, int K,
    int Dc, int L, int H, int W, int softplus, int n_cg, int n_wg) {
    constexpr int N = 16;
    __shared__ float s_dl2[kWave][kStride];               // Delta * log2 e
    __shared__ float s_du[kWave][kStride];                // Delta * u
    __shared__ float s_y[kTileWaves][kWave][kStride];     // per wave: its states' C h
    __shared__ float s_u[kZoh ? kWave : 1][kStride];      // u itself (zero-order-hold B only)

    // XCD-aware numbering: hardware places workgroup i on XCD i % 8
    const int bid = blockIdx.x;
    const int per = n_wg / 8, rem = n_wg % 8;
    const int xcd = bid % 8, slot = bid / 8;
    const int logical = xcd < rem ? xcd * (per + 1) + slot : rem * (per + 1) + (xcd - rem) * per + slot;
    const int cg = logical % n_cg;
    const int bk = logical / n_cg;  // b * K + k
    const int k = bk % K;
    const int b = bk / K;
    const int d0 = cg * kWave;

    const int tid = threadIdx.x;
    const int lane = tid % kWave;
    const int wv = __builtin_amdgcn_readfirstlane(tid / kWave);
    const bool sp = softplus != 0;

    // Loader role: row lr (channel d0 + lr), positions 4 lq .. 4 lq + 3 of each tile.
    const int lr = tid >> 2, lq = tid & 3;
    const bool ld_ok = d0 + lr < Dc;
    const int ld_d = ld_ok ? d0 + lr : Dc - 1;  // rows past the end repeat a valid one, unstored
    const int ld_c = k * Dc + ld_d;
    const float ld_bias = dt_bias ? dt_bias[ld_c] : 0.0f;
    const float ld_skip = D ? D[ld_c] : 0.0f;
    const size_t ld_row = (static_cast<size_t>(bk) * Dc + ld_d) * static_cast<size_t>(L);
    const Tin* drow = delta + ld_row;
    const Tin* urow = kTwoD ? u + (static_cast<size_t>(b) * Dc + ld_d) * L : u + ld_row;
    // 2-D layout: direction k's sequence is the plane read row-major (k even)
    // or column-major (k odd: the transposed copy xt when given), forwards
    // for k < 2 and backwards for k >= 2
    const Tin* srow = (kTwoD && (k & 1) && xt) ? xt + (static_cast<size_t>(b) * Dc + ld_d) * L : urow;
    const bool gather = kTwoD && (k & 1) && !xt;
    Tout* yrow = y + ld_row;
    // every row starts on a 4-element boundary: 4-element pieces are 16-byte
    // (fp32) or 8-byte (bf16) aligned vectors
    const bool in_aligned = (L % 4) == 0;

    // Scan role: lane = channel d0 + lane, states 4 wv .. 4 wv + 3.
    const int sd = d0 + lane < Dc ? d0 + lane : Dc - 1;
    const int sc = k * Dc + sd;
    float an[4], h[4], inv_a[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        an[j] = A[static_cast<size_t>(sc) * N + 4 * wv + j];
        inv_a[j] = kZoh ? 1.0f / an[j] : 0.0f;
        h[j] = 0.0f;
    }
    // the wave's four B and C rows: one base each, rows L elements apart
    const size_t r0 = (static_cast<size_t>(bk) * N + 4 * wv) * static_cast<size_t>(L);
    const Tin* bbase = Bm + r0;
    const Tin* cbase = Cm + r0;

    // Tile j covers positions [ts, ts + 16) with ts = 16 j, except the last,
    // which starts at L - 16 (L >= 16) so that every tile is whole: its
    // positions below 16 j were done by the previous tile and are run here
    // as identity steps (Delta = 0: a = 1, b = 0) and not stored again.
    const int ntiles = (L + kTP - 1) / kTP;
    auto tile_start = [&](int tile) { return tile * kTP + kTP <= L ? tile * kTP : L - kTP; };
    float dv[4], uv[4];
    auto load_tile = [&](int tile) {
        const int t = tile_start(tile) + 4 * lq;
        load4(drow + t, dv, in_aligned, 4);
        if constexpr (kTwoD) {
            if (gather) {
#pragma unroll
                for (int e = 0; e < 4; ++e) uv[e] = to_f32(urow[pixel_of(k, t + e, H, W)]);
            } else if (k < 2) {
                load4(srow + t, uv, in_aligned, 4);
            } else {
                float r[4];
                load4(srow + (L - 4 - t), r, in_aligned, 4);
#pragma unroll
                for (int e = 0; e < 4; ++e) uv[e] = r[3 - e];
            }
        } else {
            load4(urow + t, uv, in_aligned, 4);
        }
    };
    load_tile(0);
    // L2 prefetch of the next tile's B and C segments (16 + 16 rows of the
    // direction, one line each), so that the scan's scalar loads of them do
    // not wait for HBM: threads 0..31 each touch one row and hold the value
    // until the following tile, where it is consumed (a precise vmcnt wait
    // long after the load completed).
    const Tin* pf_row = (tid < 16 ? Bm : Cm) +
                        (static_cast<size_t>(bk) * N + (tid & 15)) * static_cast<size_t>(L);
    float pf = 0.0f;

    for (int tile = 0; tile < ntiles; ++tile) {
        const int t0 = tile_start(tile);
        const int tnew = tile * kTP;  // positions below tnew belong to the previous tile
        // 1. discretize this thread's four positions
        float skip[4];
        {
            const int t = t0 + 4 * lq;
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const float dl = t + e >= tnew ? timescale(dv[e] + ld_bias, sp) : 0.0f;
                s_dl2[lr][4 * lq + e] = dl * kLog2e;
                s_du[lr][4 * lq + e] = dl * uv[e];
                if constexpr (kZoh) s_u[lr][4 * lq + e] = uv[e];
                skip[e] = ld_skip * uv[e];
            }
        }
        __syncthreads();
        // 2. the next tile's delta / u (and its B, C lines), in flight during the scan
        if (tile + 1 < ntiles) {
            load_tile(tile + 1);
            asm volatile("" ::"v"(pf));
            if (tid < 2 * N) pf = to_f32(pf_row[tile_start(tile + 1)]);
        }
        // 3. scan the tile: four recurrences per lane, straight along the
        //    positions, in two halves of 8. Each half first issues all its B
        //    and C scalar loads (4 states x 8 consecutive positions each) and
        //    waits once: scalar loads complete out of order, so every wait is
        //    for all of them.
        float yp[kTP];
#pragma unroll
        for (int hh = 0; hh < 2; ++hh) {
            float bq[4][kTP / 2], cq[4][kTP / 2];
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                row8(bbase, j * L + t0 + 8 * hh, bq[j]);
                row8(cbase, j * L + t0 + 8 * hh, cq[j]);
            }
            __builtin_amdgcn_sched_barrier(0);
#pragma unroll
            for (int e = 0; e < kTP / 2; ++e) {
                const int i = 8 * hh + e;
                const float dl2 = s_dl2[lane][i];
                const float du = s_du[lane][i];
                const float ui = kZoh ? s_u[lane][i] : 0.0f;
                float acc = 0.0f;
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    const float x2 = dl2 * an[j];
                    const float a = fast_exp2(x2);
                    const float q = kZoh ? zoh_q(x2, a, du, ui, inv_a[j]) : du;
                    h[j] = __builtin_fmaf(a, h[j], q * bq[j][e]);
                    acc = __builtin_fmaf(cq[j][e], h[j], acc);
                }
                yp[i] = acc;
            }
        }
#pragma unroll
        for (int i = 0; i < kTP; ++i) s_y[wv][lane][i] = yp[i];
        __syncthreads();
        // 4. y = D u + the four waves' partial sums, stored row-contiguous
        //    (a piece that straddles the previous tile stores its new part)
        {
            const int t = t0 + 4 * lq;
            float o[4];
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const int i = 4 * lq + e;
                o[e] = skip[e] + ((s_y[0][lr][i] + s_y[1][lr][i]) + (s_y[2][lr][i] + s_y[3][lr][i]));
            }
            if (ld_ok) {
                if (t >= tnew) {
                    store4<kNt>(yrow + t, o, in_aligned, 4);
                } else {
#pragma unroll
                    for (int e = 0; e < 4; ++e)
                        if (t + e >= tnew)
                            store4<false>(yrow + t + e, {o[e], 0.0f, 0.0f, 0.0f}, false, 1);
                }
            }
        }
    }
}

template <typename Tin, typename Tout, bool kTwoD, bool kZoh>
vmb_status launch_tiles_zoh(const ScanArgs& a, Tout* y, const void* xt) {
    const int n_cg = int((a.channels + kWave - 1) / kWave);
    const long long n_wg = static_cast<long long>(n_cg) * a.K * a.batch;
    if (n_wg > 0x7fffffffLL) return VMB_ERR_UNSUPPORTED;
    // non-temporal output stores for rows of whole cache lines
    if (whole_lines(a.L, sizeof(Tout)))
        hipLaunchKernelGGL((k_full_scan_tiles<Tin, Tout, kTwoD, kZoh, true>),
                           dim3(static_cast<unsigned>(n_wg)), dim3(kTileThreads), 0, a.stream,
                           static_cast<const Tin*>(a.u), static_cast<const Tin*>(a.delta), a.A,
                           static_cast<const Tin*>(a.B), static_cast<const Tin*>(a.C), a.D,
                           a.dt_bias, y, static_cast<const Tin*>(xt), int(a.K), int(a.channels),
                           int(a.L), int(a.H), int(a.W), a.softplus, n_cg, int(n_wg));
    else
        hipLaunchKernelGGL((k_full_scan_tiles<Tin, Tout, kTwoD, kZoh, false>),
                           dim3(static_cast<unsigned>(n_wg)), dim3(kTileThreads), 0, a.stream,
                           static_cast<const Tin*>(a.u), static_cast<const Tin*>(a.delta), a.A,
                           static_cast<const Tin*>(a.B), static_cast<const Tin*>(a.C), a.D,
                           a.dt_bias, y, static_cast<const Tin*>(xt), int(a.K), int(a.channels),
                           int(a.L), int(a.H), int(a.W), a.softplus, n_cg, int(n_wg));
    return check_launch();
}

template <typename Tin, typename Tout, bool kTwoD>
vmb_status launch_tiles_impl(const ScanArgs& a, Tout* y, const void* xt) {
    return (a.options & VMB_SCAN_ZOH) ? launch_tiles_zoh<Tin, Tout, kTwoD, true>(a, y, xt)
                                      : launch_tiles_zoh<Tin, Tout, kTwoD, false>(a, y, xt);
}

}  // namespace

// Whether the tile kernel takes this shape at all (N = 16, whole tiles; bf16
// rows of even length): the zero-order-hold option runs here whatever the
// number of rows.
bool tiles_take(const ScanArgs& a) {
    return a.N == 16 && a.L >= kTP && !(a.in_dt == VMB_BF16 && (a.L % 2) != 0);
}

// Many channel rows (each sequence's channels split into 64-channel
// workgroups still give several waves per SIMD), N = 16, L >= 16; bf16 rows
// need an even length for the word-wise scalar reads of B and C.
bool use_tiles_full(const ScanArgs& a) {
    if (a.N != 16) return false;
    if (a.L < kTP) return false;  // the last tile starts at L - 16
    if (a.in_dt == VMB_BF16 && (a.L % 2) != 0) return false;
    const int64_t rows = a.batch * a.K * a.channels;
    return rows >= kTilesMinRows;
}

vmb_status launch_full_tiles(const ScanArgs& a, void* y_seq, const void* xt) {
    const bool two_d = a.layout == VMB_LAYOUT_2D;
    if (a.in_dt == VMB_F32)
        return two_d ? launch_tiles_impl<float, float, true>(a, static_cast<float*>(y_seq), xt)
                     : launch_tiles_impl<float, float, false>(a, static_cast<float*>(y_seq), xt);
    if (two_d) return launch_tiles_impl<bf16_t, float, true>(a, static_cast<float*>(y_seq), xt);
    if (a.out_dt == VMB_BF16)
        return launch_tiles_impl<bf16_t, bf16_t, false>(a, static_cast<bf16_t*>(y_seq), xt);
    return launch_tiles_impl<bf16_t, float, false>(a, static_cast<float*>(y_seq), xt);
}

}  // namespace vmb
