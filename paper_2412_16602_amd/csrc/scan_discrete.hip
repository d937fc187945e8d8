// scan_discrete.hip -- the decomposition of the paper's kernel experiments
// (Appendix D, Table 1): a scan kernel that only walks the recurrence of
// eq. 3 with one state on materialised inputs (discretisation outside), and
// the transform T of eq. 9 (mean over the inner channel axis) that reduces
// those inputs for the VMeanba kernel (the same scan at one channel).
//
// Scan: one wave per (b, d) sequence, walking L in chunks of 64 x 8
// positions. A lane owns 8 consecutive positions (two 16-byte loads per
// input), folds them into its run aggregate (prod a, h from 0), the 64 runs
// are combined by a DPP scan of (a1, b1) then (a2, b2) -> (a1 a2, a2 b1 + b2),
// the state entering the chunk is applied, and the lane re-walks its run to
// form y. The state leaving the chunk (lane 63) carries into the next one.
// Sequences of at most half a chunk are packed several to a wave as one flat
// run (the state reset at each sequence start), so short rows do not leave
// most of a wave idle; fewer than 2048 long sequences take a workgroup each,
// their chunks spread over its waves.
// Per element the kernel reads 8 bytes (12 with skip) and writes 4, with
// about six VALU slots of work: bound by HBM.
//
// Channel mean: each batch element's [channels][L] slab is read as rows of
// lcm(L, 4) elements (16 bytes a lane below 2048 positions, 4 above), the
// block's waves split the rows, and the partial sums meet in LDS.
#include "vmb_internal.h"

namespace vmb {
namespace {

constexpr int kWave = 64;
constexpr int kRun = 8;                   // positions per lane
constexpr int kChunk = kWave * kRun;      // positions per wave step
constexpr int kScanWaves = 4;             // sequences per workgroup

template <int kCtrl, int kRowMask>
__device__ __forceinline__ float dpp(float old, float v) {
    return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(__builtin_bit_cast(int, old),
                                                                 __builtin_bit_cast(int, v), kCtrl,
                                                                 kRowMask, 0xf, false));
}

// kRun values starting at element p of a row: two 16-byte loads when the row
// is 16-byte aligned and the run lies inside it, else element loads of the
// first cnt (the rest 0).
template <bool kVec>
__device__ __forceinline__ void load_run8(const float* p, int cnt, float (&v)[kRun]) {
    if (kVec && cnt == kRun) {
        const float4 a = *reinterpret_cast<const float4*>(p);
        const float4 b = *reinterpret_cast<const float4*>(p + 4);
        v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
        v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
        return;
    }
#pragma unroll
    for (int i = 0; i < kRun; ++i) v[i] = i < cnt ? p[i] : 0.0f;
}

template <bool kVec>
__device__ __forceinline__ void store_run8(float* p, int cnt, const float (&v)[kRun]) {
    if (kVec && cnt == kRun) {
        *reinterpret_cast<float4*>(p) = make_float4(v[0], v[1], v[2], v[3]);
        *reinterpret_cast<float4*>(p + 4) = make_float4(v[4], v[5], v[6], v[7]);
        return;
    }
#pragma unroll
    for (int i = 0; i < kRun; ++i)
        if (i < cnt) p[i] = v[i];
}

// A wave scans Q whole consecutive sequences (Q L positions, fewer in the
// last wave) as one flat run: a = 0 at each sequence start drops the state
// carried in from the previous sequence, so the flat scan gives every
// sequence's own scan (inputs are taken to be finite: 0 * inf would not
// drop it). Q > 1 (kMulti) packs short sequences so a wave's lanes and loads
// stay full; the host picks Q so that Q L is a multiple of 4, which keeps
// every run start 16-byte aligned, and L >= 8, so a run of 8 crosses at most
// one sequence start. kCVec: L % 4 == 0, C is read in 16-byte pieces (a run
// can only cross a sequence start at its midpoint then).
template <bool kMulti, bool kCVec>
__global__ __launch_bounds__(kWave* kScanWaves) void k_discrete_scan(
    const float* __restrict__ abar, const float* __restrict__ bu, const float* __restrict__ C,
    const float* __restrict__ skip, float* __restrict__ y, int64_t nseq, int channels, int L,
    int Q) {
    constexpr bool kVec = kMulti || kCVec;
    const int lane = threadIdx.x % kWave;
    const int64_t s0 = (static_cast<int64_t>(blockIdx.x) * kScanWaves + threadIdx.x / kWave) * Q;
    if (s0 >= nseq) return;  // whole waves: s0 is wave-uniform
    const int nq = nseq - s0 < Q ? static_cast<int>(nseq - s0) : Q;
    const int n = nq * L;
    const size_t row = static_cast<size_t>(s0) * L;
    const float* ap = abar + row;
    const float* bp = bu + row;
    const float* sp = skip ? skip + row : nullptr;
    float* yp = y + row;
    const int64_t b0 = s0 / channels;  // batch element of the first sequence
    const unsigned r0 = static_cast<unsigned>(s0 - b0 * channels);
    float carry = 0.0f;  // state entering the chunk
    for (int c0 = 0; c0 < n; c0 += kChunk) {
        const int t0 = c0 + lane * kRun;
        const int cnt = n - t0 < kRun ? (n - t0 > 0 ? n - t0 : 0) : kRun;
        const int tl = cnt > 0 ? t0 : 0;  // in range for empty runs
        float a[kRun], x[kRun], cv[kRun], kv[kRun];
        load_run8<kVec>(ap + tl, cnt, a);
        load_run8<kVec>(bp + tl, cnt, x);
        if (sp) {
            load_run8<kVec>(sp + tl, cnt, kv);
        } else {
#pragma unroll
            for (int i = 0; i < kRun; ++i) kv[i] = 0.0f;
        }
        if constexpr (!kMulti) {
            load_run8<kVec>(C + static_cast<size_t>(b0) * L + tl, cnt, cv);
        } else {
            // run start: sequence s0 + q, position t; positions t + i >= L
            // belong to sequence s0 + q + 1 (and its batch element's C row)
            const int q = tl / L;
            const int t = tl - q * L;
            const unsigned rq = r0 + static_cast<unsigned>(q);
            const float* ca = C + static_cast<size_t>(b0 + rq / channels) * L;
            const float* cb = C + static_cast<size_t>(b0 + (rq + 1) / channels) * L;
            auto cload = [&](int i) { return t + i < L ? ca[t + i] : cb[t + i - L]; };
            if constexpr (kCVec) {
                if (cnt == kRun) {
                    const float4 lo = *reinterpret_cast<const float4*>(ca + t);
                    const float4 hi = *reinterpret_cast<const float4*>(
                        t + 4 < L ? ca + t + 4 : cb + (t + 4 - L));
                    cv[0] = lo.x; cv[1] = lo.y; cv[2] = lo.z; cv[3] = lo.w;
                    cv[4] = hi.x; cv[5] = hi.y; cv[6] = hi.z; cv[7] = hi.w;
                } else {
#pragma unroll
                    for (int i = 0; i < kRun; ++i) cv[i] = i < cnt ? cload(i) : 0.0f;
                }
            } else {
#pragma unroll
                for (int i = 0; i < kRun; ++i) cv[i] = i < cnt ? cload(i) : 0.0f;
            }
#pragma unroll
            for (int i = 0; i < kRun; ++i)
                if (t + i == 0 || t + i == L) a[i] = 0.0f;
        }
        // positions past the end act as the identity (a = 1, b = 0)
#pragma unroll
        for (int i = 0; i < kRun; ++i)
            if (i >= cnt) {
                a[i] = 1.0f;
                x[i] = 0.0f;
            }
        float P = 1.0f, H = 0.0f;
#pragma unroll
        for (int i = 0; i < kRun; ++i) {
            H = __builtin_fmaf(a[i], H, x[i]);
            P *= a[i];
        }
        wave_scan(P, H);
        // exclusive prefix: lane - 1's inclusive value, (1, 0) on lane 0
        const float Pex = dpp<0x138, 0xf>(1.0f, P);
        const float Hex = dpp<0x138, 0xf>(0.0f, H);
        // state leaving the chunk: lane 63's inclusive value applied to carry
        const float Pl = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, P), kWave - 1));
        const float Hl = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, H), kWave - 1));
        float h = __builtin_fmaf(Pex, carry, Hex);
        carry = __builtin_fmaf(Pl, carry, Hl);
        float out[kRun];
#pragma unroll
        for (int i = 0; i < kRun; ++i) {
            h = __builtin_fmaf(a[i], h, x[i]);
            out[i] = __builtin_fmaf(cv[i], h, kv[i]);
        }
        if (cnt > 0) store_run8<kVec>(yp + tl, cnt, out);
    }
}

// Few long sequences: one workgroup per sequence, wave w taking chunk w of
// each group of nw chunks. Each wave scans its chunk from a zero state, the
// chunk aggregates meet in LDS, and every wave folds the aggregates of the
// chunks before its own into the state entering the group, in chunk order:
// the same operations, in the same order, as one wave walking the chunks.
constexpr int kSplitMaxWaves = 16;

template <bool kVec>
__global__ __launch_bounds__(kWave* kSplitMaxWaves) void k_discrete_scan_split(
    const float* __restrict__ abar, const float* __restrict__ bu, const float* __restrict__ C,
    const float* __restrict__ skip, float* __restrict__ y, int channels, int L) {
    __shared__ float aggP[kSplitMaxWaves], aggH[kSplitMaxWaves];
    const int lane = threadIdx.x % kWave;
    const int w = threadIdx.x / kWave, nw = blockDim.x / kWave;
    const int64_t s = blockIdx.x;
    const size_t row = static_cast<size_t>(s) * L;
    const float* ap = abar + row;
    const float* bp = bu + row;
    const float* sp = skip ? skip + row : nullptr;
    const float* cp = C + static_cast<size_t>(s / channels) * L;
    float* yp = y + row;
    float carry = 0.0f;  // state entering the group (the same in every wave)
    for (int g0 = 0; g0 < L; g0 += nw * kChunk) {
        const int t0 = g0 + w * kChunk + lane * kRun;
        const int cnt = L - t0 < kRun ? (L - t0 > 0 ? L - t0 : 0) : kRun;
        const int tl = cnt > 0 ? t0 : 0;
        float a[kRun], x[kRun], cv[kRun], kv[kRun];
        load_run8<kVec>(ap + tl, cnt, a);
        load_run8<kVec>(bp + tl, cnt, x);
        load_run8<kVec>(cp + tl, cnt, cv);
        if (sp) {
            load_run8<kVec>(sp + tl, cnt, kv);
        } else {
#pragma unroll
            for (int i = 0; i < kRun; ++i) kv[i] = 0.0f;
        }
#pragma unroll
        for (int i = 0; i < kRun; ++i)
            if (i >= cnt) {
                a[i] = 1.0f;
                x[i] = 0.0f;
            }
        float P = 1.0f, H = 0.0f;
#pragma unroll
        for (int i = 0; i < kRun; ++i) {
            H = __builtin_fmaf(a[i], H, x[i]);
            P *= a[i];
        }
        wave_scan(P, H);
        const float Pex = dpp<0x138, 0xf>(1.0f, P);
        const float Hex = dpp<0x138, 0xf>(0.0f, H);
        if (lane == kWave - 1) {
            aggP[w] = P;
            aggH[w] = H;
        }
        __syncthreads();
        float hin = carry;  // state entering this wave's chunk
        for (int k = 0; k < w; ++k) hin = __builtin_fmaf(aggP[k], hin, aggH[k]);
        float next = hin;  // state leaving the group
        for (int k = w; k < nw; ++k) next = __builtin_fmaf(aggP[k], next, aggH[k]);
        __syncthreads();  // the aggregates are rewritten by the next group
        float h = __builtin_fmaf(Pex, hin, Hex);
        float out[kRun];
#pragma unroll
        for (int i = 0; i < kRun; ++i) {
            h = __builtin_fmaf(a[i], h, x[i]);
            out[i] = __builtin_fmaf(cv[i], h, kv[i]);
        }
        if (cnt > 0) store_run8<kVec>(yp + tl, cnt, out);
        carry = next;
    }
}

// Sequences shorter than 8 positions: four sequences per wave, one per
// 16-lane row, each lane a run of 4 positions; the scan stays inside the row
// (row_shr steps only), so rows never mix.
__global__ __launch_bounds__(kWave* kScanWaves) void k_discrete_scan_tiny(
    const float* __restrict__ abar, const float* __restrict__ bu, const float* __restrict__ C,
    const float* __restrict__ skip, float* __restrict__ y, int64_t nseq, int channels, int L) {
    constexpr int kRow = 16, T = 4;
    const int lane = threadIdx.x % kWave;
    const int r = lane / kRow, rl = lane % kRow;
    const int64_t s = (static_cast<int64_t>(blockIdx.x) * kScanWaves + threadIdx.x / kWave) * 4 + r;
    const bool live = s < nseq;
    const int64_t sc = live ? s : nseq - 1;  // clamped: addresses stay in range
    const size_t row = static_cast<size_t>(sc) * L;
    const int t0 = rl * T;
    const int cnt = !live ? 0 : (L - t0 < T ? (L - t0 > 0 ? L - t0 : 0) : T);
    const int tl = cnt > 0 ? t0 : 0;
    const float* cp = C + static_cast<size_t>(sc / channels) * L + tl;
    float a[T], x[T], cv[T], kv[T];
#pragma unroll
    for (int i = 0; i < T; ++i) {
        const bool on = i < cnt;
        a[i] = on ? abar[row + tl + i] : 1.0f;
        x[i] = on ? bu[row + tl + i] : 0.0f;
        cv[i] = on ? cp[i] : 0.0f;
        kv[i] = on && skip ? skip[row + tl + i] : 0.0f;
    }
    float P = 1.0f, H = 0.0f;
#pragma unroll
    for (int i = 0; i < T; ++i) {
        H = __builtin_fmaf(a[i], H, x[i]);
        P *= a[i];
    }
    asm("s_nop 1\n"
        "v_fmac_f32_dpp %0, %0, %1 row_shr:1 row_mask:0xf bank_mask:0xf\n"
        "v_mul_f32_dpp %1, %1, %1 row_shr:1 row_mask:0xf bank_mask:0xf\n"
        "s_nop 1\n"
        : "+v"(H), "+v"(P));
    // state entering the run: row lane - 1's inclusive H (0 on the row's lane 0)
    float h = dpp<0x111, 0xf>(0.0f, H);
#pragma unroll
    for (int i = 0; i < T; ++i) {
        h = __builtin_fmaf(a[i], h, x[i]);
        if (i < cnt) y[row + tl + i] = __builtin_fmaf(cv[i], h, kv[i]);
    }
}

constexpr int kMeanMaxWaves = 16;
constexpr int kMeanUnroll = 8;

// Channel mean over one batch element's [channels][L] slab, read as R rows of
// S contiguous elements, S a multiple of L: column e of every row is position
// e % L, so summing the rows column by column and then the S / L columns of
// each position gives the channel sum. A lane owns V consecutive columns of a
// 64 V-column tile; the block's waves take interleaved rows (eight loads in
// flight each), then add their partial column sums in wave order through LDS.
// Grid: (column tiles, batch); fold = S / L > 1 only when one tile holds the
// whole row (S <= 64 V).
template <int V, int U>
__global__ __launch_bounds__(kWave* kMeanMaxWaves) void k_channel_mean(
    const float* __restrict__ x, float* __restrict__ xm, int64_t slab, int L, int S, int R,
    float inv) {
    __shared__ float part[kMeanMaxWaves][kWave * V];
    __shared__ float col[kWave * V];
    const int lane = threadIdx.x % kWave, w = threadIdx.x / kWave;
    const int nw = blockDim.x / kWave;
    const int b = blockIdx.y;
    const int e0 = blockIdx.x * kWave * V;
    const int e = e0 + lane * V;
    // lanes past the row end read the row's first slot (a line the wave
    // reads anyway) and their sums are never used
    const float* xb = x + static_cast<size_t>(b) * slab + (e < S ? e : 0);
    float acc[V];
#pragma unroll
    for (int i = 0; i < V; ++i) acc[i] = 0.0f;
    auto load = [&](int r, float (&v)[V]) {
        const float* p = xb + static_cast<size_t>(r) * S;
        if constexpr (V == 4) {
            const float4 q = *reinterpret_cast<const float4*>(p);
            v[0] = q.x; v[1] = q.y; v[2] = q.z; v[3] = q.w;
        } else {
            v[0] = *p;
        }
    };
    // U rows in flight; rows past the end re-read the last row (a cached
    // line) and are not added
    for (int r = w; r < R; r += U * nw) {
        float v[U][V];
#pragma unroll
        for (int j = 0; j < U; ++j) load(r + j * nw < R ? r + j * nw : R - 1, v[j]);
#pragma unroll
        for (int j = 0; j < U; ++j)
            if (r + j * nw < R) {
#pragma unroll
                for (int i = 0; i < V; ++i) acc[i] += v[j][i];
            }
    }
#pragma unroll
    for (int i = 0; i < V; ++i) part[w][lane * V + i] = acc[i];
    __syncthreads();
    for (int c = threadIdx.x; c < kWave * V; c += blockDim.x) {
        float sum = 0.0f;
        for (int k = 0; k < nw; ++k) sum += part[k][c];
        col[c] = sum;
    }
    __syncthreads();
    float* ob = xm + static_cast<size_t>(b) * L;
    const int fold = S / L;
    if (fold == 1) {
        for (int c = threadIdx.x; c < kWave * V; c += blockDim.x)
            if (e0 + c < L) ob[e0 + c] = col[c] * inv;
    } else {
        for (int t = threadIdx.x; t < L; t += blockDim.x) {
            float sum = 0.0f;
            for (int k = 0; k < fold; ++k) sum += col[k * L + t];
            ob[t] = sum * inv;
        }
    }
}

}  // namespace

// Sequences per wave for the packed scan: Q L a multiple of 4 within one
// chunk, as full as possible (ties: larger Q), while keeping at least 2048
// waves when there are enough sequences. One chunk a wave: a wave's chunks
// run one after another (load, scan, store), so at these sizes many
// one-chunk waves keep more loads in flight than fewer longer ones.
// Below this many long sequences, one workgroup per sequence (chunks across
// its waves) instead of one wave walking the chunks.
constexpr int64_t kSplitBelow = 2048;

static int pick_group(int64_t nseq, int64_t L) {
    if (L > kChunk / 2) return 1;
    const int q0 = L % 4 == 0 ? 1 : (L % 2 == 0 ? 2 : 4);
    int64_t cap = nseq / 2048;
    cap = cap < q0 ? q0 : cap;
    int best = q0;
    double best_fill = -1.0;
    for (int64_t q = q0; q * L <= kChunk && q <= cap; q += q0) {
        const int64_t n = q * L;
        const double fill = static_cast<double>(n) / (((n + kChunk - 1) / kChunk) * kChunk);
        if (fill >= best_fill) {
            best_fill = fill;
            best = static_cast<int>(q);
        }
    }
    return best;
}

vmb_status launch_discrete_scan(const float* abar, const float* bu, const float* C,
                                const float* skip, float* y, int64_t batch, int64_t channels,
                                int64_t L, hipStream_t s) {
    const int64_t nseq = batch * channels;
    if (channels > 0x7fffffffLL) return VMB_ERR_UNSUPPORTED;
    const dim3 block(kWave * kScanWaves);
    if (L < kRun) {
        const int64_t blocks = (nseq + 4 * kScanWaves - 1) / (4 * kScanWaves);
        if (blocks > 0x7fffffffLL) return VMB_ERR_UNSUPPORTED;
        hipLaunchKernelGGL(k_discrete_scan_tiny, dim3(static_cast<unsigned>(blocks)), block, 0, s,
                           abar, bu, C, skip, y, nseq, int(channels), int(L));
        return check_launch();
    }
    const int Q = pick_group(nseq, L);
    if (Q == 1 && L > kChunk && nseq < kSplitBelow) {
        const int64_t chunks = (L + kChunk - 1) / kChunk;
        const int nw = chunks < kSplitMaxWaves ? static_cast<int>(chunks) : kSplitMaxWaves;
        const dim3 sgrid(static_cast<unsigned>(nseq)), sblock(kWave * nw);
        if (L % 4 == 0)
            hipLaunchKernelGGL(k_discrete_scan_split<true>, sgrid, sblock, 0, s, abar, bu, C, skip,
                               y, int(channels), int(L));
        else
            hipLaunchKernelGGL(k_discrete_scan_split<false>, sgrid, sblock, 0, s, abar, bu, C,
                               skip, y, int(channels), int(L));
        return check_launch();
    }
    const int64_t waves = (nseq + Q - 1) / Q;
    const int64_t blocks = (waves + kScanWaves - 1) / kScanWaves;
    if (blocks > 0x7fffffffLL) return VMB_ERR_UNSUPPORTED;
    const dim3 grid(static_cast<unsigned>(blocks));
    const bool cvec = L % 4 == 0;
#define VMB_SCAN(M, V)                                                                         \
    hipLaunchKernelGGL((k_discrete_scan<M, V>), grid, block, 0, s, abar, bu, C, skip, y, nseq, \
                       int(channels), int(L), Q)
    if (Q > 1) {
        if (cvec) VMB_SCAN(true, true);
        else VMB_SCAN(true, false);
    } else {
        if (cvec) VMB_SCAN(false, true);
        else VMB_SCAN(false, false);
    }
#undef VMB_SCAN
    return check_launch();
}

vmb_status launch_channel_mean(const float* x, float* xm, int64_t batch, int64_t channels,
                               int64_t L, hipStream_t s) {
    if (batch > 65535 || channels > 0x7fffffffLL || L > 0x7fffffffLL) return VMB_ERR_UNSUPPORTED;
    const float inv = 1.0f / static_cast<float>(channels);
    const int64_t slab = channels * L;
    // rows of lcm(L, 4) elements read 16 bytes a lane when every slab starts
    // 16-byte aligned and the row fits one tile or is a whole position row
    const int64_t S4 = L % 4 == 0 ? L : (L % 2 == 0 ? 2 * L : 4 * L);
    const bool vec = slab % 4 == 0 && (S4 == L || S4 <= kWave * 4);
    const int64_t S = vec ? S4 : L;
    const int64_t R = slab / S;
    if (R > 0x7fffffffLL) return VMB_ERR_UNSUPPORTED;
    // rows of at least 2048 positions: one element a lane (tiles of 64
    // positions, four times the blocks), which measures faster there
    const bool wide = vec && S < 2048;
    const int64_t tile = kWave * (wide ? 4 : 1);
    const int64_t nw = R / 16 < 1 ? 1 : (R / 16 > kMeanMaxWaves ? kMeanMaxWaves : R / 16);
    const dim3 grid(static_cast<unsigned>((S + tile - 1) / tile), static_cast<unsigned>(batch)),
        block(static_cast<unsigned>(kWave * nw));
    if (wide)
        hipLaunchKernelGGL((k_channel_mean<4, kMeanUnroll>), grid, block, 0, s, x, xm, slab,
                           int(L), int(S), int(R), inv);
    else
        hipLaunchKernelGGL((k_channel_mean<1, kMeanUnroll>), grid, block, 0, s, x, xm, slab,
                           int(L), int(S), int(R), inv);
    return check_launch();
}

}  // namespace vmb
