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
// Passes over chunks of C = 64 positions:
//   1. reduce : a workgroup owns one chunk of one (batch, k); lanes own
//               positions (coalesced loads along t), each of its 16 waves sums
//               a fixed share of the channels (their parameters staged in
//               the wave's LDS slice and read as broadcasts; delta / u of the
//               next channels in flight), and the shares are added in a
//               fixed order in LDS. Each state's
//               chunk-local inclusive scan of the pairs (Abar_mean, B s_mean),
//               composed with (a1, b1) then (a2, b2) -> (a1 a2, a2 b1 + b2), is
//               stored per position together with r_mean; the chunk's
//               aggregate is its last position's value.
//   2. carry  : (only with more than 64 chunks) one wave per (batch, k, n)
//               scans the chunk aggregates across lanes (DPP) and stores the
//               state entering each chunk; with at most 64 chunks the finish
//               pass does this scan itself.
//   3. finish : h[n,t] = P[n,t] * carry[n] + H[n,t], ytilde = sum_n C h + r,
//               broadcast to every channel (sequence layout), or stored and
//               then folded and broadcast by the merge pass (2-D layout).
// In the 2-D layout directions 1 and 3 read column-major copies of the input
// planes (made first, one transpose pass) so that every reduce load stays
// coalesced.
// All sums run in a fixed order, so results are deterministic.
#include <atomic>
#include <chrono>
#include <mutex>
#include <random>
#include <vector>

#include "vmb_internal.h"

namespace vmb {
namespace {

constexpr int kWave = 64;
constexpr int kC = kMeanChunk;  // positions per chunk = lanes per wave
constexpr int kRedWaves = 16;   // channel split of the reduce pass
// Channel shares of the reduce waves by age on their SIMD (waves w, w + 4,
// w + 8, w + 12 share SIMD w): the SIMD issues the oldest ready wave first,
// so with equal shares the youngest waves finish last and run alone at the
// end. Older waves take more channels (15 : 13 : 11 : 9 of every 48); the
// split is fixed, so the sums keep their order from call to call.
constexpr int kShareW[4] = {15, 13, 11, 9};
constexpr int kShareTot = 4 * (kShareW[0] + kShareW[1] + kShareW[2] + kShareW[3]);
static_assert(kRedWaves == 16, "four waves of each age rank, one per SIMD");
constexpr int kAhead = 4;       // channels of delta / u in flight per wave
// The reduce and one-launch kernels whose LDS lets two workgroups share a CU
// (at most 80 KB each: all but the zero-order-hold reduce and the one-launch
// raw-means form) are built for 8 waves per SIMD, i.e. at most 64 VGPRs,
// with two channels in flight per wave instead of four (the ring of four
// does not fit 64 registers without spills). Mean calls then take 0.80-0.86
// of the time at 128 x 56x56 (three passes), 0.85 at 32 x 28x28 (one
// launch) and 0.88-0.91 at 2 x 128x512; at 1 x 56x56 (196 workgroups)
// there is no second workgroup to place and the time is unchanged.
constexpr int kAheadPaired = 2;
constexpr int kWavesPaired = 8;  // waves per SIMD: two 16-wave workgroups per CU

__device__ float g_zero = 0.0f;  // stands in for an absent dt_bias / D (never written)
constexpr int kFinWaves = 4;    // waves of a finish workgroup

// Workspace layout, per (batch, k) = bk, for L positions and nch chunks:
//   scan[bk][n][t][2] : chunk-local inclusive (P, H) of state n at position t
//   rmean[bk][t]      : r_mean
//   agg[bk][n][c][2]  : chunk aggregates (copy of the last position's scan)
//   carry[bk][c][n]   : state entering chunk c
struct MeanWs {
    float* scan;
    float* rmean;
    float* agg;
    float* carry;
    float* ytil;  // 2-D layout: reduced output ytilde[bk][t]
    float* gpart; // channel-group partial sums (split reduce)
};

// How the reduced output leaves (sequence layout): skip_own adds each
// channel's own D[c] u[d, t] to the broadcast value (which then holds no
// r_mean); no_bcast stores one row per (batch, k) instead of broadcasting.
struct StoreOpts {
    int skip_own;
    int no_bcast;
};

// Store ytilde at position t for the channels d0 + wv, d0 + wv + step, ...
// below d1 of sequence bk (sequence layout).
template <typename Tin, typename Tout, bool kNt = false>
__device__ __forceinline__ void store_reduced(float yt, Tout* __restrict__ y,
                                              const Tin* __restrict__ u,
                                              const float* __restrict__ D, StoreOpts so,
                                              size_t bk, int k, int Dc, int L, int t, int wv,
                                              int step, int d0, int d1) {
    if (so.no_bcast) {
        if (wv == 0 && d0 == 0) store_out<kNt>(y + bk * L + t, from_f32<Tout>(yt));
        return;
    }
    if (so.skip_own && D) {
        for (int d = d0 + wv; d < d1; d += step) {
            const size_t off = (bk * Dc + d) * static_cast<size_t>(L) + t;
            store_out<kNt>(y + off, from_f32<Tout>(__builtin_fmaf(
                                        D[static_cast<size_t>(k) * Dc + d], to_f32(u[off]), yt)));
        }
        return;
    }
    const Tout o = from_f32<Tout>(yt);
    for (int d = d0 + wv; d < d1; d += step)
        store_out<kNt>(y + (bk * Dc + d) * static_cast<size_t>(L) + t, o);
}

// Reduce stage of one chunk (chunk blockIdx.x / groups of sequence
// (blockIdx.z, blockIdx.y), channel group blockIdx.x % groups): every wave's
// partial sums over its channels (a 1 / (16 groups) slice of the sequence's
// channels), for the lanes' positions, left in part[wv][0..N+2) (exp sums
// per state, s, r).
// A wave's partial sums fill N + 2 rows (exp sums per state, s, r), one more
// (the input sum) when T averages the raw terms, N more (the sums of the
// zero-order-hold terms phi(Delta A_n) Delta u, rows N + 2 ..) with kZoh.
template <int N, bool kRaw, bool kZoh>
constexpr int part_rows() {
    return N + 2 + (kRaw ? 1 : 0) + (kZoh ? N : 0);
}

template <int N, typename Tin, bool kTwoD, bool kRaw, bool kZoh = false, int kAh = kAhead>
__device__ __forceinline__ void reduce_partials(
    float (*part)[(part_rows<N, kRaw, kZoh>())][kC], const Tin* __restrict__ u, const Tin* __restrict__ delta,
    const float* __restrict__ A, const float* __restrict__ D, const float* __restrict__ dt_bias,
    const Tin* __restrict__ xt, int K, int Dc, int L, int H, int W, int C, int softplus,
    int groups = 1) {
    // Each wave's slice part[wv] first holds its channel parameters (two
    // buffers of kAh rows: A[c, 0..N) log2(e), dt_bias[c], D[c], and with
    // kZoh 1 / A[c, 0..N)), read back as wave-uniform broadcasts, and
    // afterwards its partial sums.
    constexpr int kPS = (N + 2 + (kZoh ? N : 0) + 3) & ~3;  // parameter row stride (16-byte rows)
    static_assert(2 * kAh * kPS <= (N + 2) * kC, "parameter buffers fit a wave's slice");
    static_assert(kAh <= 32, "parameter row layout");
    const int chunk = blockIdx.x / groups, grp = blockIdx.x % groups;
    const int k = blockIdx.y, b = blockIdx.z;
    const int lane = threadIdx.x % kC;
    const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x / kC);
    const int t = chunk * C + lane;
    const bool valid = lane < C && t < L;
    const int tc = valid ? t : L - 1;  // clamped: every address below stays in bounds
    const size_t bk = static_cast<size_t>(b) * K + k;
    const bool sp = softplus != 0;
    // 2-D layout: directions 0 / 2 read x at t / L - 1 - t; directions 1 / 3
    // read the column-major copies xt (when given) at the same positions, or
    // gather x through the cross-scan map
    const bool use_xt = kTwoD && xt != nullptr && (k & 1);
    const int src = !kTwoD ? tc : (use_xt ? (k == 3 ? L - 1 - tc : tc) : pixel_of(k, tc, H, W));
    const Tin* usrc = use_xt ? xt : u;
    // byte offsets of this lane within a row (32-bit, non-negative)
    const unsigned toff = static_cast<unsigned>(tc) * sizeof(Tin);
    const unsigned soff = static_cast<unsigned>(src) * sizeof(Tin);
    float acc[N], zacc[kZoh ? N : 1];
#pragma unroll
    for (int n = 0; n < N; ++n) acc[n] = 0.0f;
#pragma unroll
    for (int n = 0; n < (kZoh ? N : 1); ++n) zacc[n] = 0.0f;
    float s = 0.0f, r = 0.0f, q = 0.0f;
    // channels [d0, d1) of this wave: with one group the age-weighted shares
    // (kShareW), with several (the split reduce) equal shares of the group
    int d0, d1;
    if (groups == 1) {
        const int rank = wv / 4;
        int cum = (wv % 4) * kShareW[rank];
        for (int r = 0; r < rank; ++r) cum += 4 * kShareW[r];
        d0 = (cum * Dc) / kShareTot;
        d1 = ((cum + kShareW[rank]) * Dc) / kShareTot;
    } else {
        const int slice = grp * kRedWaves + wv, nslices = kRedWaves * groups;
        d0 = (slice * Dc) / nslices;
        d1 = ((slice + 1) * Dc) / nslices;
    }
    const int nw = d1 - d0;  // channels of this wave
    float* prm = &part[wv][0][0];
    const size_t cw = static_cast<size_t>(k) * Dc + d0;  // parameter row of the wave's first channel
    // absent dt_bias / D read as zeros (a select, not a branch)
    const float* pbias = dt_bias ? dt_bias : &g_zero;
    const float* pskip = D ? D : &g_zero;
    const int bias_stride = dt_bias ? 1 : 0, skip_stride = D ? 1 : 0;

    // delta / u of wave channel i (clamped to the wave's last channel)
    auto load_ch = [&](int i, float& dv, float& uv) {
        // wave-uniform row bases (scalar registers), one lane offset each
        const int d = d0 + (i < nw ? i : nw - 1);
        const size_t row = (bk * Dc + d) * static_cast<size_t>(L);
        const size_t urow = kTwoD ? (static_cast<size_t>(b) * Dc + d) * L : row;
        const char* dp = reinterpret_cast<const char*>(delta + row);
        const char* up = reinterpret_cast<const char*>(usrc + urow);
        dv = to_f32(*reinterpret_cast<const Tin*>(dp + toff));
        uv = to_f32(*reinterpret_cast<const Tin*>(up + soff));
    };
    // parameters of wave channels i0 .. i0 + kAh - 1 (clamped): global
    // loads into registers, later written to LDS buffer buf
    constexpr int kPA = (kAh * N + kC - 1) / kC;
    auto load_par = [&](int i0, float (&pa)[kPA], float& pbd) {
#pragma unroll
        for (int m = 0; m < kPA; ++m) {
            const int idx = (lane + m * kC) % (kAh * N);
            const int i = i0 + idx / N;
            pa[m] = A[(cw + (i < nw ? i : nw - 1)) * N + idx % N];
        }
        const int i = i0 + (lane % kAh);
        const size_t c = cw + (i < nw ? i : nw - 1);
        pbd = lane < 32 ? pbias[c * bias_stride] : pskip[c * skip_stride];
    };
    auto write_par = [&](int buf, const float (&pa)[kPA], float pbd) {
        float* base = prm + buf * kAh * kPS;
#pragma unroll
        for (int m = 0; m < kPA; ++m) {
            const int idx = lane + m * kC;
            if (idx < kAh * N) {
                base[(idx / N) * kPS + idx % N] = pa[m] * kLog2e;
                if constexpr (kZoh) base[(idx / N) * kPS + N + 2 + idx % N] = 1.0f / pa[m];
            }
        }
        if (lane < kAh) base[lane * kPS + N] = pbd;
        else if (lane >= 32 && lane < 32 + kAh) base[(lane - 32) * kPS + N + 1] = pbd;
    };
    auto read_par = [&](int buf, int i, float (&an)[N], float& bias, float& dskip) {
        const float* row = prm + buf * kAh * kPS + i * kPS;
#pragma unroll
        for (int n = 0; n < N; ++n) an[n] = row[n];
        bias = row[N];
        dskip = row[N + 1];
    };
    // 1 / A of the same channel (kZoh)
    auto read_inv = [&](int buf, int i, int n) {
        return prm[buf * kAh * kPS + i * kPS + N + 2 + n];
    };
    auto channel = [&](const float (&an)[N], float bias, float dskip, float dv, float uv, int buf,
                       int i) {
        const float dl = valid ? timescale(dv + bias, sp) : 0.0f;
        if constexpr (kZoh) {
            // means of exp(Delta A_n) and of the zero-order-hold terms per state
            const float du = dl * uv;
#pragma unroll
            for (int n = 0; n < N; ++n) {
                const float x2 = dl * an[n];  // an = A log2(e)
                const float a = fast_exp2(x2);
                acc[n] += a;
                zacc[n] += zoh_q(x2, a, du, uv, read_inv(buf, i, n));
            }
            s = __builtin_fmaf(dl, uv, s);
        } else if constexpr (kRaw) {
            // sums of A log2(e) (the same in every lane), Delta and u
#pragma unroll
            for (int n = 0; n < N; ++n) acc[n] += an[n];
            s += dl;
            q += uv;
        } else {
#pragma unroll
            for (int n = 0; n < N; ++n) acc[n] += fast_exp2(dl * an[n]);  // an = A log2(e)
            s = __builtin_fmaf(dl, uv, s);
        }
        r = __builtin_fmaf(dskip, uv, r);
        // the sums are formed here, not sunk towards their next use (which
        // would keep every channel's parameters live)
#pragma unroll
        for (int n = 0; n < N; ++n) asm volatile("" : "+v"(acc[n]));
        if constexpr (kZoh) {
#pragma unroll
            for (int n = 0; n < N; ++n) asm volatile("" : "+v"(zacc[n]));
        }
        if constexpr (kRaw)
            asm volatile("" : "+v"(s), "+v"(r), "+v"(q));
        else
            asm volatile("" : "+v"(s), "+v"(r));
    };

    if (nw > 0) {
        // parameters of the first block, then delta / u of its kAh
        // channels: a ring refilled kAh channels ahead of use
        float pa[kPA], pbd;
        load_par(0, pa, pbd);
        // issued before the ring's loads, so that writing them out waits for
        // them alone
        __builtin_amdgcn_sched_barrier(0);
        float dv[kAh], uv[kAh];
#pragma unroll
        for (int j = 0; j < kAh; ++j) load_ch(j, dv[j], uv[j]);
        write_par(0, pa, pbd);
        const int nb = nw / kAh;  // full blocks; the rest is the tail
        for (int blk = 0; blk < nb; ++blk) {
            const int buf = blk & 1, i0 = blk * kAh;
            load_par(i0 + kAh, pa, pbd);
            __builtin_amdgcn_sched_barrier(0);
#pragma unroll
            for (int j = 0; j < kAh; ++j) {
                // one channel at a time (no hoisting across channels, which
                // would cost registers the load ring needs)
                __builtin_amdgcn_sched_barrier(0);
                float an[N], bias, dskip;
                read_par(buf, j, an, bias, dskip);
                channel(an, bias, dskip, dv[j], uv[j], buf, j);
                load_ch(i0 + kAh + j, dv[j], uv[j]);
            }
            __builtin_amdgcn_sched_barrier(0);
            write_par(buf ^ 1, pa, pbd);
        }
        const int rem = nw - nb * kAh;
#pragma unroll
        for (int j = 0; j < kAh - 1; ++j) {
            if (j < rem) {
                float an[N], bias, dskip;
                read_par(nb & 1, j, an, bias, dskip);
                channel(an, bias, dskip, dv[j], uv[j], nb & 1, j);
            }
        }
    }
#pragma unroll
    for (int n = 0; n < N; ++n) part[wv][n][lane] = acc[n];
    part[wv][N][lane] = s;
    part[wv][N + 1][lane] = r;
    if constexpr (kRaw) part[wv][N + 2][lane] = q;
    if constexpr (kZoh) {
#pragma unroll
        for (int n = 0; n < N; ++n) part[wv][N + 2 + n][lane] = zacc[n];
    }
}

// The pair (a, b) of state n at one position from the channel-group sums:
// the means of the discretised terms, (mean exp(Delta A), B mean(Delta u)),
// or with kRaw the discretisation of the means, (exp(mean Delta mean A),
// mean Delta B mean u).
template <int N, bool kRaw, bool kZoh = false>
__device__ __forceinline__ void reduced_pair(const float (*part)[(part_rows<N, kRaw, kZoh>())][kC],
                                             int n, int lane, float inv, float bval, float& a,
                                             float& bb) {
    float sm = 0.0f, am = 0.0f;
    // zero-order hold: the state's own mean of phi(Delta A_n) Delta u
    const int srow = kZoh ? N + 2 + n : N;
    for (int w = 0; w < kRedWaves; ++w) sm += part[w][srow][lane];
    for (int w = 0; w < kRedWaves; ++w) am += part[w][n][lane];
    sm *= inv;
    am *= inv;
    if constexpr (kRaw) {
        float um = 0.0f;
        for (int w = 0; w < kRedWaves; ++w) um += part[w][N + 2][lane];
        um *= inv;
        a = fast_exp2(sm * am);  // am = mean A log2(e)
        bb = sm * bval * um;
    } else {
        a = am;
        bb = bval * sm;
    }
}

// Chunk-local scan of one chunk from the channel sums in part (slots added
// in slot order): r_mean, then wave w scans states w, w + 16, ... and stores
// the per-position pairs and the chunk aggregate.
template <int N, typename Tin, bool kRaw, bool kZoh>
__device__ __forceinline__ void scan_chunk(const float (*part)[(part_rows<N, kRaw, kZoh>())][kC],
                                           const Tin* __restrict__ Bm, MeanWs ws, int K, int Dc,
                                           int L, int C, int nchunks, int chunk) {
    const int k = blockIdx.y, b = blockIdx.z;
    const int lane = threadIdx.x % kC;
    const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x / kC);
    const int t = chunk * C + lane;
    const bool valid = lane < C && t < L;
    const int tc = valid ? t : L - 1;
    const size_t bk = static_cast<size_t>(b) * K + k;

    const float inv = 1.0f / static_cast<float>(Dc);
    if (wv == 0) {
        float rm = 0.0f;
        for (int w = 0; w < kRedWaves; ++w) rm += part[w][N + 1][lane];
        if (valid) ws.rmean[bk * L + t] = rm * inv;
    }
    float* scan_bk = ws.scan + bk * N * L * 2;
    float* agg_bk = ws.agg + bk * N * nchunks * 2;
    for (int n = wv; n < N; n += kRedWaves) {
        float a, bb;
        reduced_pair<N, kRaw, kZoh>(part, n, lane, inv, to_f32(Bm[(bk * N + n) * L + tc]), a, bb);
        // positions past the end act as the identity (1, 0)
        a = valid ? a : 1.0f;
        bb = valid ? bb : 0.0f;
        wave_scan(a, bb);
        if (valid) {
            float2 v = make_float2(a, bb);
            *reinterpret_cast<float2*>(scan_bk + (static_cast<size_t>(n) * L + t) * 2) = v;
        }
        if (lane == kC - 1)
            *reinterpret_cast<float2*>(agg_bk + (static_cast<size_t>(n) * nchunks + chunk) * 2) =
                make_float2(a, bb);
    }
}

// The first workgroup of the call's first mean kernel records the call's tag
// in the workspace's completion record (word 0, and its complement in word 2,
// so that no fill pattern reads as a recorded call).
__device__ __forceinline__ void record_call(const MeanStatus& st) {
    if (threadIdx.x == 0 && blockIdx.x == 0 && blockIdx.y == 0 && blockIdx.z == 0) {
        __hip_atomic_store(st.words, st.epoch, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        __hip_atomic_store(st.words + 2, ~st.epoch, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
}

// With groups == 1 the reduce scans its chunk itself; otherwise each of the
// groups workgroups of a chunk stores its channel group's sums (its waves
// added in wave order) for k_mean_combine.
template <int N, typename Tin, bool kTwoD, bool kRaw, bool kZoh>
__global__ __launch_bounds__(kC* kRedWaves)
__attribute__((amdgpu_waves_per_eu(kZoh ? 1 : kWavesPaired))) void k_mean_reduce(
    const Tin* __restrict__ u, const Tin* __restrict__ delta, const float* __restrict__ A,
    const Tin* __restrict__ Bm, const float* __restrict__ D, const float* __restrict__ dt_bias,
    const Tin* __restrict__ xt, MeanWs ws, int K, int Dc, int L, int H, int W, int C, int nchunks,
    int softplus, int groups, MeanStatus st) {
    constexpr int kRows = part_rows<N, kRaw, kZoh>();
    __shared__ __align__(16) float part[kRedWaves][kRows][kC];
    record_call(st);
    reduce_partials<N, Tin, kTwoD, kRaw, kZoh, kZoh ? kAhead : kAheadPaired>(
        part, u, delta, A, D, dt_bias, xt, K, Dc, L, H, W, C, softplus, groups);
    __syncthreads();
    if (groups == 1) {
        scan_chunk<N, Tin, kRaw, kZoh>(part, Bm, ws, K, Dc, L, C, nchunks, blockIdx.x);
        return;
    }
    const int chunk = blockIdx.x / groups, grp = blockIdx.x % groups;
    const int lane = threadIdx.x % kC;
    const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x / kC);
    const size_t bkc = (static_cast<size_t>(blockIdx.z) * K + blockIdx.y) * nchunks + chunk;
    float* gp = ws.gpart + ((bkc * groups + grp) * kRows) * kC;
    for (int r = wv; r < kRows; r += kRedWaves) {
        float sum = 0.0f;
        for (int w = 0; w < kRedWaves; ++w) sum += part[w][r][lane];
        gp[r * kC + lane] = sum;
    }
}

// Combine of the split reduce: chunk blockIdx.x of sequence (blockIdx.z,
// blockIdx.y) takes its groups' sums as the first slots of part (the other
// slots zero), then scans the chunk as the unsplit reduce does.
template <int N, typename Tin, bool kRaw, bool kZoh>
__global__ __launch_bounds__(kC* kRedWaves) void k_mean_combine(const Tin* __restrict__ Bm,
                                                                MeanWs ws, int K, int Dc, int L,
                                                                int C, int nchunks, int groups) {
    constexpr int kRows = part_rows<N, kRaw, kZoh>();
    __shared__ __align__(16) float part[kRedWaves][kRows][kC];
    const size_t bkc =
        (static_cast<size_t>(blockIdx.z) * K + blockIdx.y) * nchunks + blockIdx.x;
    const float* gp = ws.gpart + bkc * groups * kRows * kC;
    float* pf = &part[0][0][0];
    for (int i = threadIdx.x; i < kRedWaves * kRows * kC; i += kC * kRedWaves)
        pf[i] = i < groups * kRows * kC ? gp[i] : 0.0f;
    __syncthreads();
    scan_chunk<N, Tin, kRaw, kZoh>(part, Bm, ws, K, Dc, L, C, nchunks, blockIdx.x);
}

// One wave per (batch, k, n): exclusive scan of the chunk aggregates.
__global__ __launch_bounds__(kWave) void k_mean_carry(MeanWs ws, int N, int nchunks) {
    const int lane = threadIdx.x;
    const size_t bk = blockIdx.x / N;
    const int n = blockIdx.x % N;
    float carry = 0.0f;  // state entering the current block of 64 chunks
    for (int c0 = 0; c0 < nchunks; c0 += kWave) {
        const int c = c0 + lane;
        float a = 1.0f, bb = 0.0f;
        if (c < nchunks) {
            const float2 g = *reinterpret_cast<const float2*>(
                ws.agg + ((bk * N + n) * nchunks + c) * 2);
            a = g.x;
            bb = g.y;
        }
        wave_scan(a, bb);
        // state entering chunk c = carry composed with the chunks before c
        const float pa = __shfl_up(a, 1, kWave), pb = __shfl_up(bb, 1, kWave);
        const float cin = lane == 0 ? carry : __builtin_fmaf(pa, carry, pb);
        if (c < nchunks) ws.carry[(bk * nchunks + c) * N + n] = cin;
        const float la = __shfl(a, kWave - 1, kWave), lb = __shfl(bb, kWave - 1, kWave);
        carry = __builtin_fmaf(la, carry, lb);
    }
}

// All three passes in one launch, for sequences of at most 64 chunks. After
// its reduce, each workgroup publishes its chunk aggregates and, once those
// stores are performed, raises its flag (the call's epoch: a 64-bit value
// never reused, so flags left by earlier calls, or never written, do not
// match); it then waits for the
// flags of the earlier chunks of its sequence, scans their aggregates into
// the state entering its own chunk, and forms and stores its outputs.
// Workgroups wait only on lower-numbered workgroups of their own sequence
// (chunk is the fastest grid dimension), which are dispatched no later, so
// the lowest unfinished workgroup never waits; every wait is also bounded
// by a spin limit, so the kernel ends whatever happens. A workgroup whose
// wait gives up does not read aggregates it has not seen announced: it
// records the call's failure in the workspace (word 1 of the completion
// record) and stores NaN for its chunk, so the caller finds out from
// vmb_mean_scan_status and no stale value is ever passed off as a result.
constexpr int kSpinLimit = 1 << 16;
constexpr int kTestSpinLimit = 8;  // VMB_MEAN_TEST_GIVE_UP
// Grid bound of the one-launch path, in rounds of co-resident workgroups:
// progress does not depend on co-residency (a workgroup waits only on
// lower-numbered ones, dispatched no later), but beyond a few rounds the
// waiting workgroups hold compute units that the separate passes keep busy
// (batch 128 at 56x56: 1.42 ms fused against 1.21 ms in three passes).
constexpr int kFusedRounds = 8;

// (a, b) pairs exchanged between workgroups: 64-bit device-scope atomic
// accesses, coherent across the chip's L2 caches without cache-wide
// write-back or invalidation.
__device__ __forceinline__ void put_pair(float* p, float a, float b) {
    const unsigned long long v = (static_cast<unsigned long long>(__float_as_uint(b)) << 32) |
                                 __float_as_uint(a);
    __hip_atomic_store(reinterpret_cast<unsigned long long*>(p), v, __ATOMIC_RELAXED,
                       __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void get_pair(float* p, float& a, float& b) {
    const unsigned long long v = __hip_atomic_load(reinterpret_cast<unsigned long long*>(p),
                                                   __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    a = __uint_as_float(static_cast<unsigned>(v));
    b = __uint_as_float(static_cast<unsigned>(v >> 32));
}

template <int N, typename Tin, typename Tout, bool kTwoD, bool kRaw, bool kNt>
__global__ __launch_bounds__(kC* kRedWaves)
__attribute__((amdgpu_waves_per_eu(kRaw ? 1 : kWavesPaired))) void k_mean_fused(
    const Tin* __restrict__ u, const Tin* __restrict__ delta, const float* __restrict__ A,
    const Tin* __restrict__ Bm, const Tin* __restrict__ Cm, const float* __restrict__ D,
    const float* __restrict__ dt_bias, const Tin* __restrict__ xt, MeanWs ws,
    unsigned long long* __restrict__ flags, MeanStatus st, int spin_limit, int withhold,
    Tout* __restrict__ y, int K, int Dc, int L, int H, int W, int nchunks, int softplus,
    StoreOpts so) {
    static_assert(N <= kRedWaves, "one state per wave");
    __shared__ __align__(16) float part[kRedWaves][N + 2 + int(kRaw)][kC];
    __shared__ float yst[kRedWaves][kC];  // C h of state n at each position
    __shared__ float rsh[kC];             // r_mean at each position
    __shared__ int gave_up;
    const unsigned long long epoch = st.epoch;
    record_call(st);
    reduce_partials<N, Tin, kTwoD, kRaw, false, kRaw ? kAhead : kAheadPaired>(
        part, u, delta, A, D, dt_bias, xt, K, Dc, L, H, W, kC, softplus);
    __syncthreads();
    const int chunk = blockIdx.x, k = blockIdx.y, b = blockIdx.z;
    const int lane = threadIdx.x % kC;
    const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x / kC);
    const int t = chunk * kC + lane;
    const bool valid = t < L;
    const int tc = valid ? t : L - 1;
    const size_t bk = static_cast<size_t>(b) * K + k;
    const float inv = 1.0f / static_cast<float>(Dc);
    float* agg_bk = ws.agg + bk * N * nchunks * 2;

    // channel groups added in a fixed order; wave n scans state n
    float a = 1.0f, bb = 0.0f, cv = 0.0f;
    if (wv < N) {
        const int n = wv;
        cv = valid ? to_f32(Cm[(bk * N + n) * L + tc]) : 0.0f;
        reduced_pair<N, kRaw>(part, n, lane, inv, to_f32(Bm[(bk * N + n) * L + tc]), a, bb);
        // positions past the end act as the identity (1, 0)
        a = valid ? a : 1.0f;
        bb = valid ? bb : 0.0f;
        wave_scan(a, bb);
        if (lane == kC - 1) put_pair(agg_bk + (static_cast<size_t>(n) * nchunks + chunk) * 2, a, bb);
    } else if (wv == N) {
        float rm = 0.0f;
        for (int w = 0; w < kRedWaves; ++w) rm += part[w][N + 1][lane];
        rsh[lane] = rm * inv;
    }
    if (N == kRedWaves && wv == 0) {  // no spare wave: wave 0 sums r_mean too
        float rm = 0.0f;
        for (int w = 0; w < kRedWaves; ++w) rm += part[w][N + 1][lane];
        rsh[lane] = rm * inv;
    }
    // publish: the aggregates (device-coherent stores) are performed before
    // the flag is stored
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    if (threadIdx.x == 0 && !(withhold && chunk == 0))
        __hip_atomic_store(flags + bk * nchunks + chunk, epoch, __ATOMIC_RELAXED,
                           __HIP_MEMORY_SCOPE_AGENT);
    // wait for the earlier chunks (lanes = chunks) of this sequence
    if (wv == 0) {
        bool ready = lane >= chunk;
        for (int spin = 0; spin < spin_limit; ++spin) {
            if (!ready)
                ready = __hip_atomic_load(flags + bk * nchunks + lane, __ATOMIC_RELAXED,
                                          __HIP_MEMORY_SCOPE_AGENT) == epoch;
            if (__all(ready)) break;
            __builtin_amdgcn_s_sleep(2);
        }
        const bool failed = !__all(ready);
        if (lane == 0) {
            gave_up = failed ? 1 : 0;
            if (failed)
                __hip_atomic_store(st.words + 1, epoch ^ kFailTag, __ATOMIC_RELAXED,
                                   __HIP_MEMORY_SCOPE_AGENT);
        }
    }
    __syncthreads();
    if (gave_up) {
        // the state entering this chunk is unknown: NaN outputs, no stale sums
        if (wv < N) yst[wv][lane] = __builtin_nanf("");
    } else if (wv < N) {
        const int n = wv;
        // state entering this chunk: scan of the earlier chunks' aggregates
        // (device-coherent loads, issued after the flags were seen)
        float ga = 1.0f, gb = 0.0f;
        if (lane < chunk) get_pair(agg_bk + (static_cast<size_t>(n) * nchunks + lane) * 2, ga, gb);
        wave_scan(ga, gb);
        const float prev = __shfl(gb, chunk > 0 ? chunk - 1 : 0, kWave);
        const float cin = chunk > 0 ? prev : 0.0f;
        yst[n][lane] = cv * __builtin_fmaf(a, cin, bb);
    }
    __syncthreads();
    if (!valid) return;
    float yt = so.skip_own ? 0.0f : rsh[lane];
#pragma unroll
    for (int n = 0; n < N; ++n) yt += yst[n][lane];
    if constexpr (kTwoD) {
        if (wv == 0) ws.ytil[bk * L + t] = yt;
    } else {
        store_reduced<Tin, Tout, kNt>(yt, y, u, D, so, bk, k, Dc, L, t, wv, kRedWaves, 0, Dc);
    }
}

// C h summed over the states n = wv, wv + kFinWaves, ... of each of kDirs
// sequences bk[i] at positions t[i] (chunk-local scan composed with the state
// entering the position's chunk). The entering state comes, with at most 64
// chunks per sequence, from an exclusive scan of the chunk aggregates done
// here (lanes = chunks, then lane ch - 1's inclusive value), otherwise from
// the carry pass. All loads are issued before any of the scans.
template <int N, int kDirs, typename Tin>
__device__ __forceinline__ void ch_partials(const MeanWs& ws, const Tin* __restrict__ Cm,
                                            const size_t (&bk)[kDirs], int L, const int (&t)[kDirs],
                                            int C, int nchunks, bool inline_carry, int lane,
                                            int wv, float (&acc)[kDirs]) {
    constexpr int kPer = N / kFinWaves > 0 ? N / kFinWaves : 1;
    float ga[kDirs][kPer], gb[kDirs][kPer], cv[kDirs][kPer];
    float2 ph[kDirs][kPer];
#pragma unroll
    for (int i = 0; i < kDirs; ++i) {
        const float* scan_bk = ws.scan + bk[i] * N * L * 2;
        const int ch = t[i] / C;
#pragma unroll
        for (int j = 0; j < kPer; ++j) {
            const int n = wv + j * kFinWaves;
            const bool on = n < N;
            const int nn = on ? n : 0;
            ga[i][j] = 1.0f;
            gb[i][j] = 0.0f;
            if (inline_carry) {
                if (on && lane < nchunks) {
                    const float2 g = *reinterpret_cast<const float2*>(
                        ws.agg + ((bk[i] * N + nn) * nchunks + lane) * 2);
                    ga[i][j] = g.x;
                    gb[i][j] = g.y;
                }
            } else {
                gb[i][j] = ws.carry[(bk[i] * nchunks + ch) * N + nn];
            }
            ph[i][j] = *reinterpret_cast<const float2*>(scan_bk +
                                                        (static_cast<size_t>(nn) * L + t[i]) * 2);
            cv[i][j] = on ? to_f32(Cm[(bk[i] * N + nn) * L + t[i]]) : 0.0f;
        }
    }
#pragma unroll
    for (int i = 0; i < kDirs; ++i) {
        const int ch = t[i] / C;
        acc[i] = 0.0f;
#pragma unroll
        for (int j = 0; j < kPer; ++j) {
            float cin = gb[i][j];
            if (inline_carry) {
                float a = ga[i][j], bb = gb[i][j];
                wave_scan(a, bb);
                const float prev = __shfl(bb, ch > 0 ? ch - 1 : 0, kWave);
                cin = ch > 0 ? prev : 0.0f;
            }
            const float h = __builtin_fmaf(ph[i][j].x, cin, ph[i][j].y);
            acc[i] = __builtin_fmaf(cv[i][j], h, acc[i]);
        }
    }
}

// Sequence layout. grid: (block of 64 positions, k * groups, batch). The
// four waves form the C h partials of their states, the partials and r_mean
// are added in a fixed order, and every wave writes its share of the group's
// channels (lane-contiguous rows).
// With kTwoD the reduced sequence itself is stored (to ws.ytil) for the
// merge-and-broadcast pass.
template <int N, typename Tin, typename Tout, bool kTwoD, bool kNt>
__global__ __launch_bounds__(kC* kFinWaves) void k_mean_finish_seq(
    MeanWs ws, const Tin* __restrict__ Cm, Tout* __restrict__ y, const Tin* __restrict__ u,
    const float* __restrict__ D, int K, int Dc, int L, int C, int nchunks, int groups,
    int inline_carry, StoreOpts so) {
    __shared__ float part[kFinWaves][kC];
    const int blk = blockIdx.x, k = blockIdx.y / groups, grp = blockIdx.y % groups;
    const int b = blockIdx.z;
    const int lane = threadIdx.x % kC;
    const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x / kC);
    const int t = blk * kC + lane;
    const bool valid = t < L;
    const int tc = valid ? t : L - 1;
    const size_t bk = static_cast<size_t>(b) * K + k;
    const size_t bks[1] = {bk};
    const int ts[1] = {tc};
    float acc[1];
    ch_partials<N, 1>(ws, Cm, bks, L, ts, C, nchunks, inline_carry != 0, lane, wv, acc);
    part[wv][lane] = acc[0];
    __syncthreads();
    if (!valid) return;
    float yt = so.skip_own ? 0.0f : ws.rmean[bk * L + tc];
#pragma unroll
    for (int w = 0; w < kFinWaves; ++w) yt += part[w][lane];
    if constexpr (kTwoD) {
        if (wv == 0) ws.ytil[bk * L + t] = yt;
        return;
    }
    const int dg0 = (grp * Dc) / groups, dg1 = ((grp + 1) * Dc) / groups;
    store_reduced<Tin, Tout, kNt>(yt, y, u, D, so, bk, k, Dc, L, t, wv, kFinWaves, dg0, dg1);
}

// 2-D layout: fold the four reduced sequences of each batch element into one
// map, (y0 + y2) + (y1 + y3) per pixel (the cross-merge, same association as
// the standalone merge), and broadcast it to the channels of group blockIdx.y.
// With a per-channel skip (x given) each channel adds the merge of its four
// directions' D[k, d] x[b, d, pixel] terms, (D0 + D2) + (D1 + D3) times x.
// grid: (block of 256 pixels, channel groups, batch).
template <typename Tin, typename Tout, bool kNt>
__global__ __launch_bounds__(256) void k_mean_merge_broadcast(const float* __restrict__ ytil,
                                                              Tout* __restrict__ y,
                                                              const Tin* __restrict__ x,
                                                              const float* __restrict__ D, int Dc,
                                                              int H, int W, int groups) {
    const int L = H * W;
    const int p = blockIdx.x * 256 + threadIdx.x;
    const int grp = blockIdx.y, b = blockIdx.z;
    if (p >= L) return;
    const int hh = p / W, ww = p - hh * W;
    const int q = ww * H + hh;
    const float* yb = ytil + static_cast<size_t>(b) * 4 * L;
    const float s02 = yb[p] + yb[2 * static_cast<size_t>(L) + (L - 1 - p)];
    const float s13 = yb[static_cast<size_t>(L) + q] + yb[3 * static_cast<size_t>(L) + (L - 1 - q)];
    const float ym = s02 + s13;
    const int dg0 = (grp * Dc) / groups, dg1 = ((grp + 1) * Dc) / groups;
    Tout* yp = y + static_cast<size_t>(b) * Dc * L + p;
    if (x) {
        const Tin* xp = x + static_cast<size_t>(b) * Dc * L + p;
        for (int d = dg0; d < dg1; ++d) {
            const float dsum = (D[d] + D[2 * Dc + d]) + (D[Dc + d] + D[3 * Dc + d]);
            store_out<kNt>(yp + static_cast<size_t>(d) * L,
                           from_f32<Tout>(__builtin_fmaf(dsum, to_f32(xp[static_cast<size_t>(d) * L]),
                                                         ym)));
        }
        return;
    }
    const Tout o = from_f32<Tout>(ym);
    for (int d = dg0; d < dg1; ++d) store_out<kNt>(yp + static_cast<size_t>(d) * L, o);
}

// Channel groups for a broadcast pass: the wanted count, at least 1 and at
// most one group per 16 channels.
inline int clamp_groups(long long want, int Dc) {
    const long long most = Dc >= 16 ? Dc / 16 : 1;
    return static_cast<int>(want < 1 ? 1 : (want > most ? most : want));
}

template <typename Tin, typename Tout>
vmb_status launch_merge_broadcast(const float* ytil, const ScanArgs& a) {
    const int Dc = int(a.channels), H = int(a.H), W = int(a.W), L = H * W;
    const int pblk = (L + 255) / 256;
    const long long mwant = (512 + pblk * a.batch - 1) / (pblk * a.batch);
    const int mgroups = clamp_groups(mwant, Dc);
    // per-channel skip: x and D (an absent D makes it the reduced output alone)
    const bool own = (a.options & VMB_MEAN_SKIP_PER_CHANNEL) && a.D;
    // non-temporal stores for planes of whole cache lines
    auto kernel = whole_lines(L, sizeof(Tout)) ? k_mean_merge_broadcast<Tin, Tout, true>
                                               : k_mean_merge_broadcast<Tin, Tout, false>;
    hipLaunchKernelGGL(kernel, dim3(pblk, static_cast<unsigned>(mgroups), unsigned(a.batch)),
                       dim3(256), 0, a.stream, ytil, static_cast<Tout*>(a.y),
                       own ? static_cast<const Tin*>(a.u) : nullptr, a.D, Dc, H, W, mgroups);
    return check_launch();
}

// Flag value of one call of the fused pass: a process-wide counter started
// at a random 64-bit value (never 0), so that no flag left in a workspace by
// an earlier call, or by whatever the memory held before, can match it.
unsigned long long next_epoch() {
    static std::atomic<unsigned long long> counter{[] {
        std::random_device rd;
        const unsigned long long seed =
            (static_cast<unsigned long long>(rd()) << 32) ^ rd() ^
            static_cast<unsigned long long>(
                std::chrono::steady_clock::now().time_since_epoch().count());
        return seed | 1ull;
    }()};
    unsigned long long e = counter.fetch_add(2, std::memory_order_relaxed);
    return e ? e : counter.fetch_add(2, std::memory_order_relaxed);
}

// The completion record of this call: the workspace base and a fresh tag.
MeanStatus call_status(const ScanArgs& a) {
    MeanStatus st;
    st.words = static_cast<unsigned long long*>(a.ws);
    st.epoch = next_epoch();
    return st;
}

// Workgroups of `kernel` (block threads each) that the current device holds
// at once: occupancy per compute unit times the compute units, read once per
// (kernel, device) and kept; 0 if HIP cannot say.
long long resident_workgroups(const void* kernel, int threads) {
    struct Entry {
        const void* kernel;
        int dev;
        long long value;
    };
    static std::mutex mu;
    static std::vector<Entry> cache;
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) return 0;
    {
        std::lock_guard<std::mutex> lock(mu);
        for (const Entry& e : cache)
            if (e.kernel == kernel && e.dev == dev) return e.value;
    }
    int per_cu = 0, cus = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kernel, threads, 0) != hipSuccess)
        return 0;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
        return 0;
    const long long v = static_cast<long long>(per_cu) * cus;
    if (v > 0) {
        std::lock_guard<std::mutex> lock(mu);
        cache.push_back(Entry{kernel, dev, v});
    }
    return v;
}

// ---------------------------------------------------------------- pooled reading
// T over all K * channels sequences of an image (VMB_MEAN_POOLED). The
// reduce of the main reading gives, per (b, k) and position, the sums over
// the direction's channels of exp(Delta A_n), Delta u and D u; a direction's
// B and C multiply its own sums, so the pooled means combine the directions:
//   abar[n] = sum_k E_k[n] / M,  bu[n] = sum_k B_k[n] S_k / M,
//   cbar[n] = sum_k C_k[n] / K,  r = sum_k R_k / M      (M = K * channels),
// then one N-state scan per image (the one-state scan, states as channels)
// and ytilde = sum_n cbar h + r, broadcast to every (k, d).

// Pass 1: per chunk of one (b, k), the channel sums (fixed order over the
// 16 channel groups), stored raw in psum[bk][row][t], rows 0..N-1 the exp
// sums, N the Delta u sum, N + 1 the D u sum.
template <int N, typename Tin, bool kTwoD>
__global__ __launch_bounds__(kC* kRedWaves) void k_pooled_sums(
    const Tin* __restrict__ u, const Tin* __restrict__ delta, const float* __restrict__ A,
    const float* __restrict__ D, const float* __restrict__ dt_bias, const Tin* __restrict__ xt,
    float* __restrict__ psum, int K, int Dc, int L, int H, int W, int C, int softplus,
    MeanStatus st) {
    __shared__ __align__(16) float part[kRedWaves][N + 2][kC];
    record_call(st);
    reduce_partials<N, Tin, kTwoD, false>(part, u, delta, A, D, dt_bias, xt, K, Dc, L, H, W, C,
                                          softplus);
    __syncthreads();
    const int chunk = blockIdx.x, k = blockIdx.y, b = blockIdx.z;
    const int lane = threadIdx.x % kC;
    const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x / kC);
    const int t = chunk * C + lane;
    if (lane >= C || t >= L) return;
    const size_t bk = static_cast<size_t>(b) * K + k;
    for (int row = wv; row < N + 2; row += kRedWaves) {
        float sum = 0.0f;
        for (int w = 0; w < kRedWaves; ++w) sum += part[w][row][lane];
        psum[(bk * (N + 2) + row) * static_cast<size_t>(L) + t] = sum;
    }
}

// Pass 2: the pooled scan inputs per (b, n, t) (state n = blockIdx.y),
// directions added in order; the state-0 threads also form r and the ones.
template <int N, typename Tin>
__global__ __launch_bounds__(256) void k_pooled_combine(
    const float* __restrict__ psum, const Tin* __restrict__ Bm, const Tin* __restrict__ Cm,
    float* __restrict__ abar, float* __restrict__ bu, float* __restrict__ cbar,
    float* __restrict__ ones, float* __restrict__ rbar, int K, int Dc, int L) {
    const int t = blockIdx.x * 256 + threadIdx.x;
    const int n = blockIdx.y, b = blockIdx.z;
    if (t >= L) return;
    const float inv = 1.0f / (static_cast<float>(K) * static_cast<float>(Dc));
    const float invk = 1.0f / static_cast<float>(K);
    const size_t l = static_cast<size_t>(L);
    float e = 0.0f, bs = 0.0f, cs = 0.0f, r = 0.0f;
    for (int k = 0; k < K; ++k) {
        const size_t bk = static_cast<size_t>(b) * K + k;
        const float* ps = psum + bk * (N + 2) * l;
        e += ps[n * l + t];
        bs = __builtin_fmaf(to_f32(Bm[(bk * N + n) * l + t]), ps[N * l + t], bs);
        cs += to_f32(Cm[(bk * N + n) * l + t]);
        if (n == 0) r += ps[(N + 1) * l + t];
    }
    const size_t o = (static_cast<size_t>(b) * N + n) * l + t;
    abar[o] = e * inv;
    bu[o] = bs * inv;
    cbar[o] = cs * invk;
    if (n == 0) {
        rbar[static_cast<size_t>(b) * l + t] = r * inv;
        ones[static_cast<size_t>(b) * l + t] = 1.0f;
    }
}

// Pass 4: ytilde = sum_n cbar h + r. Sequence layout: broadcast to the rows
// (k, d) of row group blockIdx.y; 2-D layout (ytil4 given): the same value
// written once per direction for the merge-and-broadcast pass.
template <int N, typename Tout>
__global__ __launch_bounds__(256) void k_pooled_out(const float* __restrict__ cbar,
                                                    const float* __restrict__ h,
                                                    const float* __restrict__ rbar,
                                                    Tout* __restrict__ y,
                                                    float* __restrict__ ytil4, int rows, int L,
                                                    int groups) {
    const int t = blockIdx.x * 256 + threadIdx.x;
    const int grp = blockIdx.y, b = blockIdx.z;
    if (t >= L) return;
    const size_t l = static_cast<size_t>(L);
    float acc = rbar[static_cast<size_t>(b) * l + t];
    for (int n = 0; n < N; ++n) {
        const size_t o = (static_cast<size_t>(b) * N + n) * l + t;
        acc = __builtin_fmaf(cbar[o], h[o], acc);
    }
    if (ytil4) {
        for (int k = 0; k < 4; ++k) ytil4[(static_cast<size_t>(b) * 4 + k) * l + t] = acc;
        return;
    }
    const int r0 = (grp * rows) / groups, r1 = ((grp + 1) * rows) / groups;
    const Tout o = from_f32<Tout>(acc);
    Tout* yb = y + static_cast<size_t>(b) * rows * l + t;
    for (int r = r0; r < r1; ++r) yb[static_cast<size_t>(r) * l] = o;
}

template <int N, typename Tin, typename Tout, bool kTwoD>
vmb_status run_pooled(const ScanArgs& a) {
    const PooledWsLayout lay = pooled_ws_layout(a.batch, a.K, a.channels, a.L, N, kTwoD);
    char* p = static_cast<char*>(a.ws);
    auto f = [&](size_t off) { return reinterpret_cast<float*>(p + off); };
    const int K = int(a.K), Dc = int(a.channels), L = int(a.L), H = int(a.H), W = int(a.W);
    const int C = kC;
    const int nchunks = (L + C - 1) / C;
    const Tin* xt = nullptr;
    if (kTwoD && mean_transposes(a.L, true) && cross_fits(a.batch, a.channels, a.H, a.W)) {
        vmb_status s0 = launch_transpose_planes(a.u, p + lay.xt, a.batch, a.channels, a.H, a.W,
                                                a.in_dt, a.stream);
        if (s0 != VMB_OK) return s0;
        xt = reinterpret_cast<const Tin*>(p + lay.xt);
    }
    hipLaunchKernelGGL((k_pooled_sums<N, Tin, kTwoD>),
                       dim3(nchunks, static_cast<unsigned>(a.K), static_cast<unsigned>(a.batch)),
                       dim3(kC * kRedWaves), 0, a.stream, static_cast<const Tin*>(a.u),
                       static_cast<const Tin*>(a.delta), a.A, a.D, a.dt_bias, xt, f(lay.psum), K,
                       Dc, L, H, W, C, a.softplus, call_status(a));
    vmb_status st = check_launch();
    if (st != VMB_OK) return st;
    const unsigned pblk = static_cast<unsigned>((L + 255) / 256);
    hipLaunchKernelGGL((k_pooled_combine<N, Tin>), dim3(pblk, N, static_cast<unsigned>(a.batch)),
                       dim3(256), 0, a.stream, f(lay.psum), static_cast<const Tin*>(a.B),
                       static_cast<const Tin*>(a.C), f(lay.abar), f(lay.bu), f(lay.cbar),
                       f(lay.ones), f(lay.rbar), K, Dc, L);
    st = check_launch();
    if (st != VMB_OK) return st;
    // the states of the pooled scan: one-state scans with the states as channels
    st = launch_discrete_scan(f(lay.abar), f(lay.bu), f(lay.ones), nullptr, f(lay.h), a.batch, N,
                              a.L, a.stream);
    if (st != VMB_OK) return st;
    const int rows = K * Dc;
    if (kTwoD) {
        hipLaunchKernelGGL((k_pooled_out<N, Tout>), dim3(pblk, 1, static_cast<unsigned>(a.batch)),
                           dim3(256), 0, a.stream, f(lay.cbar), f(lay.h), f(lay.rbar),
                           static_cast<Tout*>(nullptr), f(lay.ytil), rows, L, 1);
        st = check_launch();
        if (st != VMB_OK) return st;
        return launch_merge_broadcast<Tin, Tout>(f(lay.ytil), a);
    }
    const long long want = (1024 + pblk * a.batch - 1) / (pblk * a.batch);
    const int groups = clamp_groups(want, rows);
    hipLaunchKernelGGL((k_pooled_out<N, Tout>),
                       dim3(pblk, static_cast<unsigned>(groups), static_cast<unsigned>(a.batch)),
                       dim3(256), 0, a.stream, f(lay.cbar), f(lay.h), f(lay.rbar),
                       static_cast<Tout*>(a.y), static_cast<float*>(nullptr), rows, L, groups);
    return check_launch();
}

template <int N, typename Tin, typename Tout, bool kTwoD, bool kRaw, bool kZoh>
vmb_status run(const ScanArgs& a) {
    const size_t bkn = static_cast<size_t>(a.batch * a.K);
    const MeanWsLayout lay = mean_ws_layout(a.batch, a.K, a.channels, a.L, N, kTwoD);
    char* p = static_cast<char*>(a.ws);
    MeanWs ws;
    ws.scan = reinterpret_cast<float*>(p + lay.scan);
    ws.rmean = reinterpret_cast<float*>(p + lay.rmean);
    ws.agg = reinterpret_cast<float*>(p + lay.agg);
    ws.carry = reinterpret_cast<float*>(p + lay.carry);
    ws.ytil = kTwoD ? reinterpret_cast<float*>(p + lay.ytil) : nullptr;
    ws.gpart = reinterpret_cast<float*>(p + lay.gpart);

    const int K = int(a.K), Dc = int(a.channels), L = int(a.L), H = int(a.H), W = int(a.W);
    const int C = mean_chunk(a.batch, a.K, a.L);
    const int nchunks = (L + C - 1) / C;
    // One launch for all passes when every sequence has at most 64 chunks and
    // the grid is small (up to 8 workgroups per compute unit): with many more
    // rounds of workgroups, time spent waiting for an earlier chunk would
    // hold a compute unit that the separate passes keep busy.
    const long long wgs = static_cast<long long>(nchunks) * a.K * a.batch;
    // (the zero-order-hold sums need more LDS than the one-launch kernel has
    // room for next to its other buffers: those calls take the three passes)
    const int rgroups = mean_groups(a.batch, a.K, a.channels, a.L);  // reduce channel groups
    bool fused = !kZoh && rgroups == 1 && C == kC && nchunks <= kWave;
    if constexpr (!kZoh) {
        if (fused && nchunks > 1) {
            // A call captured into a HIP graph keeps its arguments, this
            // call's flag value included, for every replay: a workgroup could
            // take an earlier chunk's flag left by the previous replay for this
            // one's and read that replay's aggregates. Captured calls take the
            // separate passes, which kernel boundaries alone order.
            hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
            if (hipStreamIsCapturing(a.stream, &cs) != hipSuccess) {
                (void)hipGetLastError();  // the separate passes are safe either way
                cs = hipStreamCaptureStatusActive;
            }
            if (cs != hipStreamCaptureStatusNone) fused = false;
        }
        if (fused && nchunks > 1) {
            const long long cap = resident_workgroups(
                reinterpret_cast<const void*>(&k_mean_fused<N, Tin, Tout, kTwoD, kRaw, false>),
                kC * kRedWaves);
            if (cap < 1) return VMB_ERR_HIP;
            fused = wgs <= kFusedRounds * cap;
        }
    }
    const MeanStatus stat = call_status(a);
    const dim3 grid(nchunks, static_cast<unsigned>(a.K), static_cast<unsigned>(a.batch));
    // 2-D layout: column-major copies of the planes first, so that every
    // direction's reduce reads stay coalesced
    const Tin* xt = nullptr;
    if (kTwoD && mean_transposes(a.L, true) && cross_fits(a.batch, a.channels, a.H, a.W)) {
        vmb_status s0 = launch_transpose_planes(a.u, p + lay.xt, a.batch, a.channels, a.H, a.W,
                                                a.in_dt, a.stream);
        if (s0 != VMB_OK) return s0;
        xt = reinterpret_cast<const Tin*>(p + lay.xt);
    }
    StoreOpts so;
    so.skip_own = (a.options & VMB_MEAN_SKIP_PER_CHANNEL) ? 1 : 0;
    so.no_bcast = (a.options & VMB_MEAN_NO_BROADCAST) ? 1 : 0;
    if constexpr (!kZoh) if (fused) {
        // non-temporal broadcast stores for rows of whole cache lines (N = 16)
        auto kernel = (N == 16 && !kTwoD && whole_lines(L, sizeof(Tout)))
                          ? k_mean_fused<N, Tin, Tout, kTwoD, kRaw, N == 16 && !kTwoD>
                          : k_mean_fused<N, Tin, Tout, kTwoD, kRaw, false>;
        hipLaunchKernelGGL(kernel, grid, dim3(kC * kRedWaves), 0, a.stream,
                           static_cast<const Tin*>(a.u),
                           static_cast<const Tin*>(a.delta), a.A, static_cast<const Tin*>(a.B),
                           static_cast<const Tin*>(a.C), a.D, a.dt_bias, xt, ws,
                           reinterpret_cast<unsigned long long*>(p + lay.flags), stat,
                           (a.options & VMB_MEAN_TEST_GIVE_UP) ? kTestSpinLimit : kSpinLimit,
                           (a.options & VMB_MEAN_TEST_GIVE_UP) ? 1 : 0, static_cast<Tout*>(a.y),
                           K, Dc, L, H, W, nchunks, a.softplus, so);
        const vmb_status sf = check_launch();
        if (sf != VMB_OK || !kTwoD) return sf;
        return launch_merge_broadcast<Tin, Tout>(ws.ytil, a);
    }
    hipLaunchKernelGGL((k_mean_reduce<N, Tin, kTwoD, kRaw, kZoh>),
                       dim3(nchunks * rgroups, static_cast<unsigned>(a.K), static_cast<unsigned>(a.batch)),
                       dim3(kC * kRedWaves), 0, a.stream,
                       static_cast<const Tin*>(a.u), static_cast<const Tin*>(a.delta), a.A,
                       static_cast<const Tin*>(a.B), a.D, a.dt_bias, xt, ws, K, Dc, L, H, W, C,
                       nchunks, a.softplus, rgroups, stat);
    vmb_status st = check_launch();
    if (st != VMB_OK) return st;
    if (rgroups > 1) {
        hipLaunchKernelGGL((k_mean_combine<N, Tin, kRaw, kZoh>), grid, dim3(kC * kRedWaves), 0,
                           a.stream, static_cast<const Tin*>(a.B), ws, K, Dc, L, C, nchunks,
                           rgroups);
        st = check_launch();
        if (st != VMB_OK) return st;
    }
    const int inline_carry = nchunks <= kWave ? 1 : 0;
    if (!inline_carry) {
        hipLaunchKernelGGL(k_mean_carry, dim3(static_cast<unsigned>(bkn * N)), dim3(kWave), 0,
                           a.stream, ws, N, nchunks);
        st = check_launch();
        if (st != VMB_OK) return st;
    }
    // channel groups of the finish pass: enough workgroups to spread the
    // broadcast stores (each group recomputes the reduced output it stores);
    // the 2-D layout stores the reduced sequences once and broadcasts them in
    // the merge pass
    const int nblk = (L + kC - 1) / kC;
    const long long seqs = a.batch * a.K;
    const long long want = (512 + nblk * seqs - 1) / (nblk * seqs);
    const int groups = kTwoD || so.no_bcast ? 1 : clamp_groups(want, Dc);
    auto fin = (N == 16 && !kTwoD && whole_lines(L, sizeof(Tout)))
                   ? k_mean_finish_seq<N, Tin, Tout, kTwoD, N == 16 && !kTwoD>
                   : k_mean_finish_seq<N, Tin, Tout, kTwoD, false>;
    hipLaunchKernelGGL(fin, dim3(nblk, static_cast<unsigned>(a.K * groups), unsigned(a.batch)),
                       dim3(kC * kFinWaves), 0, a.stream, ws, static_cast<const Tin*>(a.C),
                       static_cast<Tout*>(a.y), static_cast<const Tin*>(a.u), a.D, K, Dc, L, C,
                       nchunks, groups, inline_carry, so);
    st = check_launch();
    if (st != VMB_OK || !kTwoD) return st;
    return launch_merge_broadcast<Tin, Tout>(ws.ytil, a);
}

template <int N, typename Tin, typename Tout, bool kRaw, bool kZoh = false>
vmb_status dispatch_layout(const ScanArgs& a) {
    return a.layout == VMB_LAYOUT_SEQ ? run<N, Tin, Tout, false, kRaw, kZoh>(a)
                                      : run<N, Tin, Tout, true, kRaw, kZoh>(a);
}

template <int N, typename Tin, typename Tout>
vmb_status dispatch_reading(const ScanArgs& a) {
    if (a.options & VMB_MEAN_POOLED)
        return a.layout == VMB_LAYOUT_SEQ ? run_pooled<N, Tin, Tout, false>(a)
                                          : run_pooled<N, Tin, Tout, true>(a);
    if (a.options & VMB_SCAN_ZOH) return dispatch_layout<N, Tin, Tout, false, true>(a);
    return (a.options & VMB_MEAN_RAW) ? dispatch_layout<N, Tin, Tout, true>(a)
                                      : dispatch_layout<N, Tin, Tout, false>(a);
}

template <int N>
vmb_status dispatch_dtype(const ScanArgs& a) {
    if (a.in_dt == VMB_F32) return dispatch_reading<N, float, float>(a);
    if (a.out_dt == VMB_BF16) return dispatch_reading<N, bf16_t, bf16_t>(a);
    return dispatch_reading<N, bf16_t, float>(a);
}

}  // namespace

vmb_status mean_scan_status(const void* ws, hipStream_t s) {
    if (hipStreamSynchronize(s) != hipSuccess) return VMB_ERR_HIP;
    unsigned long long rec[3] = {0, 0, 0};
    if (hipMemcpy(rec, ws, sizeof(rec), hipMemcpyDeviceToHost) != hipSuccess) return VMB_ERR_HIP;
    // tags are odd and stored with their complement: otherwise no call is recorded
    if ((rec[0] & 1ull) == 0 || rec[2] != ~rec[0]) return VMB_ERR_WORKSPACE;
    return rec[1] == (rec[0] ^ kFailTag) ? VMB_ERR_INCOMPLETE : VMB_OK;
}

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
