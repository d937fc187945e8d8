// scan_chunked.hip -- full selective scan, positions spread over lanes.
//
// Same recurrence as scan_full.hip (Appendix A: eq. 3, eq. 4 first line,
// eq. 6), organised for shapes with few channels and long sequences, where
// one lane per channel would leave most of the machine idle.
//
// Work decomposition. A workgroup owns G channels of one (batch, direction);
// each channel gets Wv waves, each lane a run of T consecutive positions, so
// one pass ("chunk") covers Wv*64*T positions and longer sequences loop over
// chunks. For every state n (outer loop) a lane
//   1. forms a_i = exp(Delta_i A_n) and b_i = Delta_i B_i u_i for its T
//      positions (kept in registers) and composes them into its run's
//      aggregate (prod a, state reached from zero),
//   2. joins the runs: an inclusive DPP scan of the aggregates across the 64
//      lanes, then, through LDS, across the Wv waves of the channel and with
//      the state carried in from the previous chunk,
//   3. re-walks its run from the state entering it, accumulating
//      y_i += C_i h_i.
// The aggregate's product is exp(A_n * sum_i Delta_i) (one exp per run, not
// per position). The pair combine is (a1, b1) then (a2, b2) ->
// (a1 a2, a2 b1 + b2), associative (Appendix A: the associative scan Mamba
// runs in its kernel). Per (position, state): mul, exp2, mul, 3 fma.
//
// States go in pairs, one workgroup barrier per pair: phase 1 (steps 1-2 up
// to the wave's aggregate) before it, the cross-wave join and phase 2 after;
// the two states' chains are interleaved, which gives each wave two
// independent dependency chains to issue from.
// B and C rows are shared by every channel of a direction. Four copy waves
// move each pair's slices of them once, straight from global memory into LDS
// (global_load_lds), double-buffered: before barrier p they issue C of pair p
// and B of pair p + 1. Lanes read their runs from LDS (stride-13 words:
// conflict-free).
//
// Delta and u: a sequence of one chunk has each wave's ranges (2-D layout:
// each channel's input plane, which every direction reads through its
// cross-scan map) copied into LDS the same way before the first barrier and
// the runs read from there; longer sequences load the runs from global
// memory (whole runs of rows with vector loads), the 2-D directions 1 and 3
// from column-major plane copies when the caller's workspace holds them.
// Sequences of one chunk have a kernel of their own (kOne), which carries
// no state out of the chunk and forms its timescales and per-position
// products before the first barrier: waves whose data arrived early work
// while the others' loads are still in flight.
//
// Workgroups are numbered so that the ones sharing a (batch, direction), and
// therefore B and C, land on the same XCD and its L2 (2-D sequences of one
// chunk: the four directions of a channel group, which share its planes).
#include "vmb_internal.h"

namespace vmb {
namespace {

constexpr int kWave = 64;

// DPP controls (GFX9 encoding)
constexpr int kWaveShr1 = 0x138;

template <int kCtrl, int kRowMask>
__device__ __forceinline__ float dpp(float old, float v) {
    return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(__builtin_bit_cast(int, old),
                                                                 __builtin_bit_cast(int, v), kCtrl,
                                                                 kRowMask, 0xf, false));
}

// T consecutive elements starting at p (element-aligned). full: all T are
// in range; otherwise only the first cnt are read, the rest become 0.
template <int T>
__device__ __forceinline__ void load_run(const float* p, float (&v)[T], bool full, int cnt) {
    if (full) {
#pragma unroll
        for (int i = 0; i + 4 <= T; i += 4) {
            float4 q;
            __builtin_memcpy(&q, p + i, 16);
            v[i] = q.x;
            v[i + 1] = q.y;
            v[i + 2] = q.z;
            v[i + 3] = q.w;
        }
#pragma unroll
        for (int i = T & ~3; i < T; ++i) v[i] = p[i];
    } else {
#pragma unroll
        for (int i = 0; i < T; ++i) v[i] = i < cnt ? p[i] : 0.0f;
    }
}

template <int T>
__device__ __forceinline__ void load_run(const bf16_t* p, float (&v)[T], bool full, int cnt) {
    if (full) {
#pragma unroll
        for (int i = 0; i + 2 <= T; i += 2) {
            uint32_t q;
            __builtin_memcpy(&q, p + i, 4);
            v[i] = __uint_as_float(q << 16);
            v[i + 1] = __uint_as_float(q & 0xffff0000u);
        }
        if (T & 1) v[T - 1] = to_f32(p[T - 1]);
    } else {
#pragma unroll
        for (int i = 0; i < T; ++i) v[i] = i < cnt ? to_f32(p[i]) : 0.0f;
    }
}

// Stores one wave's outputs: lane l holds the run of T values at positions
// seg0 + l*T .. seg0 + l*T + T - 1 (nval valid positions in all). Written
// straight from the runs, each store instruction would touch every lane's
// own cache lines; instead the wave passes the values through its own LDS
// slice (stride T words: no bank conflicts) and stores them lane-contiguous,
// 4 values per lane (aligned rows) or 1. Whole fp32 quads go out as
// non-temporal stores: nothing here reads them again, and streamed out they
// do not sit dirty in L2 until the end of the kernel, which writes them back
// after the last wave (the waves of a launch finish close together).
template <int T, typename Tout>
__device__ __forceinline__ void store_wave(Tout* dst, const float (&v)[T], float* slice, int lane,
                                           int nval, bool aligned4) {
#pragma unroll
    for (int i = 0; i < T; ++i) slice[lane * T + i] = v[i];
    if (aligned4) {
        constexpr int kQuads = (kWave * T) / 4;
#pragma unroll
        for (int j0 = 0; j0 < kQuads; j0 += kWave) {
            const int j = j0 + lane;
            if (j < kQuads && 4 * j < nval) {
                const float4 q = *reinterpret_cast<const float4*>(slice + 4 * j);
                if (4 * j + 4 <= nval) {
                    if constexpr (sizeof(Tout) == 4) {
                        typedef float f32x4 __attribute__((ext_vector_type(4)));
                        const f32x4 v = {q.x, q.y, q.z, q.w};
                        __builtin_nontemporal_store(v, reinterpret_cast<f32x4*>(dst + 4 * j));
                    } else {
                        Tout o[4] = {from_f32<Tout>(q.x), from_f32<Tout>(q.y), from_f32<Tout>(q.z),
                                     from_f32<Tout>(q.w)};
                        __builtin_memcpy(dst + 4 * j, o, sizeof(o));
                    }
                } else {
                    const float e[4] = {q.x, q.y, q.z, q.w};
                    for (int r = 0; r < nval - 4 * j; ++r) dst[4 * j + r] = from_f32<Tout>(e[r]);
                }
            }
        }
    } else {
#pragma unroll
        for (int i = 0; i < T; ++i) {
            const int j = i * kWave + lane;
            if (j < nval) dst[j] = from_f32<Tout>(slice[j]);
        }
    }
}

// u values of a run in the 2-D layout: position t of direction k reads pixel
// pixel_of(k, t); rows are walked incrementally for the column-major maps.
template <int T, typename Tin>
__device__ __forceinline__ void load_run_2d(const Tin* plane, int k, int t0, int H, int W, int L,
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

// load_run_2d from global memory: a whole run of a row-major direction
// (k = 0, or k = 2 reversed) is T consecutive elements of the plane, read
// with vector loads as in the sequence layout; other runs element by element.
template <int T, typename Tin>
__device__ __forceinline__ void load_run_2d_global(const Tin* plane, int k, int t0, int H, int W,
                                                   int L, float (&v)[T], int cnt) {
    if ((k & 1) == 0 && cnt == T) {
        if (k == 0) {
            load_run<T>(plane + t0, v, true, T);
        } else {
            float w[T];
            load_run<T>(plane + (L - t0 - T), w, true, T);
#pragma unroll
            for (int i = 0; i < T; ++i) v[i] = w[T - 1 - i];
        }
        return;
    }
    load_run_2d<T>(plane, k, t0, H, W, L, v, cnt);
}

// Phase 1 of a pair of states (an0, an1) for one lane: per state, a_i and
// b_i of its run (registers), the run aggregate, the inclusive scan over the
// wave (Pin, Hin, kept for phase 2), and this wave's aggregate published by
// the last lane to xg[slot] (the channel's row, see lane_entry). The two
// states' chains are interleaved (their aggregates and wave scans are
// independent). With kZoh, Bbar u takes the zero-order-hold form (zoh_q,
// from the run's u values uvr and inv = 1 / A_n) instead of Delta u.
template <int T, typename Tin, bool kZoh = false>
__device__ __forceinline__ void pair_phase1(float an0, float an1, const float (&dl2)[T],
                                            const float (&du)[T], float s2, const Tin* b0src,
                                            const Tin* b1src, float (&a0)[T], float (&bu0)[T],
                                            float (&a1)[T], float (&bu1)[T], float& Pin0,
                                            float& Hin0, float& Pin1, float& Hin1,
                                            float (*xg0)[2], float (*xg1)[2], int lane, int slot,
                                            const float (&uvr)[T], float inv0, float inv1) {
    float agg0 = 0.0f, agg1 = 0.0f;
#pragma unroll
    for (int i = 0; i < T; ++i) {
        const float x0 = dl2[i] * an0, x1 = dl2[i] * an1;
        a0[i] = fast_exp2(x0);
        a1[i] = fast_exp2(x1);
        const float q0 = kZoh ? zoh_q(x0, a0[i], du[i], uvr[i], inv0) : du[i];
        const float q1 = kZoh ? zoh_q(x1, a1[i], du[i], uvr[i], inv1) : du[i];
        bu0[i] = q0 * to_f32(b0src[i]);
        bu1[i] = q1 * to_f32(b1src[i]);
        agg0 = i == 0 ? bu0[0] : __builtin_fmaf(a0[i], agg0, bu0[i]);
        agg1 = i == 0 ? bu1[0] : __builtin_fmaf(a1[i], agg1, bu1[i]);
    }
    Pin0 = fast_exp2(s2 * an0);
    Pin1 = fast_exp2(s2 * an1);
    Hin0 = agg0;
    Hin1 = agg1;
    wave_scan2(Pin0, Hin0, Pin1, Hin1);
    if (lane == kWave - 1) {
        xg0[slot][0] = Pin0;
        xg0[slot][1] = Hin0;
        xg1[slot][0] = Pin1;
        xg1[slot][1] = Hin1;
    }
}

// Phase 2 (after the workgroup barrier), first part, for one state: the
// state entering this wave from the channel's earlier waves and the previous
// chunk (*hcar, this wave's own copy of the carry), then the state entering
// this lane (lane - 1's inclusive scan applied to it, read across lanes).
//
// xg is the channel's row of slots. With kCarryOut (chunks pass a carry on)
// it holds the aggregates of waves 0 .. kWv - 1; every wave composes all of
// them from the carry, which gives the state leaving the channel (the same
// in every wave's copy), and takes cin from the chain on the way. Without,
// the row starts with kWv - 1 identities (1, 0) and wave w composes the
// kWv - 1 slots from w on (identities, then waves 0 .. w - 1): the same
// count of steps for every wave, with no per-wave selection.
template <int kWv, bool kCarryOut>
__device__ __forceinline__ float lane_entry(float Pin, float Hin, const float (*xg)[2],
                                            float* hcar, int lane, int w) {
    const float hc = *hcar;
    float cin = hc;
    if constexpr (kCarryOut) {
        float cnext = hc;
#pragma unroll
        for (int j = 0; j < kWv; ++j) {
            const float2 x = *reinterpret_cast<const float2*>(xg[j]);
            cnext = __builtin_fmaf(x.x, cnext, x.y);
            if (j + 1 < kWv && j + 1 == w) cin = cnext;
        }
        if (lane == 0) *hcar = cnext;
    } else {
#pragma unroll
        for (int j = 0; j + 1 < kWv; ++j) {
            const float2 x = *reinterpret_cast<const float2*>(xg[w + j]);
            cin = __builtin_fmaf(x.x, cin, x.y);
        }
    }
    // lane 0 starts from cin itself (the shift leaves its old value)
    return dpp<kWaveShr1, 0xf>(cin, __builtin_fmaf(Pin, cin, Hin));
}

// Phase 2 of the pair: both re-walks from the lanes' entering states,
// interleaved, accumulating y_i += C0_i h0_i, then += C1_i h1_i. The end of
// the re-walk is pinned here: left to itself the compiler sinks it past the
// next step's phase 1, which then needs two steps' run arrays at once.
template <int T, int kWv, bool kCarryOut, typename Tin>
__device__ __forceinline__ void pair_phase2(const float (&a0)[T], const float (&bu0)[T],
                                            const float (&a1)[T], const float (&bu1)[T],
                                            float Pin0, float Hin0, float Pin1, float Hin1,
                                            const Tin* c0src, const Tin* c1src, float (&yv)[T],
                                            const float (*xg0)[2], const float (*xg1)[2],
                                            float* hcar0, float* hcar1, int lane, int w) {
    float h0 = lane_entry<kWv, kCarryOut>(Pin0, Hin0, xg0, hcar0, lane, w);
    float h1 = lane_entry<kWv, kCarryOut>(Pin1, Hin1, xg1, hcar1, lane, w);
#pragma unroll
    for (int i = 0; i < T; ++i) {
        h0 = __builtin_fmaf(a0[i], h0, bu0[i]);
        h1 = __builtin_fmaf(a1[i], h1, bu1[i]);
        yv[i] = __builtin_fmaf(to_f32(c0src[i]), h0, yv[i]);
        yv[i] = __builtin_fmaf(to_f32(c1src[i]), h1, yv[i]);
    }
#pragma unroll
    for (int i = 0; i < T; ++i) asm volatile("" : "+v"(yv[i]));
}

// Slice of the B or C row of one state copied into LDS: positions
// [cs, cs + len) of the row, len <= kStageMax. The copy goes straight from
// global memory to LDS (gfx950 global_load_lds: each lane of a wave moves 16
// or 4 bytes to LDS at base + lane * size), no registers involved. Rows of
// whole 16-byte pieces move 16-byte pieces, others 4-byte words (one fp32 or
// two bf16 elements: bf16 rows reach this kernel with even lengths only). The
// issuing wave must wait for vmcnt before the barrier that publishes them.
constexpr int kStageMax = 4 * kWave * 13;
constexpr int kComputeWaves = 12;  // G channels x Wv waves
constexpr int kCopyWaves = 4;      // one per SIMD, copies only
constexpr int kStageThreads = (kComputeWaves + kCopyWaves) * kWave;

// The loop over a row's pieces is unrolled (at most kIt per wave) with
// wave-uniform bounds, so issuing costs a few scalar instructions and one
// lane-offset add per copy. Lanes past the row's end copy nothing.
template <int kBytes, typename Tin>
__device__ __forceinline__ void stage_pieces(const Tin* src, Tin* dst, int len, int issuer,
                                             int lane) {
    constexpr int kPer = kBytes / static_cast<int>(sizeof(Tin));  // elements per lane-piece
    constexpr int kSpan = kWave * kPer;                            // per wave-instruction
    constexpr int kIt = (kStageMax + kCopyWaves * kSpan - 1) / (kCopyWaves * kSpan);
    const int jl = lane * kPer;
#pragma unroll
    for (int it = 0; it < kIt; ++it) {
        const int base = (issuer + it * kCopyWaves) * kSpan;
        if (base >= len) break;
        if (base + jl < len)
            __builtin_amdgcn_global_load_lds(src + base + jl, dst + base, kBytes, 0, 0);
    }
}

// One 16-byte piece per lane from global memory into LDS (gfx950
// global_load_lds: lane i's piece lands at dst + 16 i, dst wave-uniform).
typedef __attribute__((address_space(1))) void global_void;
typedef __attribute__((address_space(3))) void lds_void;
__device__ __forceinline__ void lds_dma16(const void* src, void* dst) {
    __builtin_amdgcn_global_load_lds((global_void*)src, (lds_void*)dst, 16, 0, 0);
}

// Copy of len elements from src into LDS at dst by one wave, in 16-byte
// pieces (len a multiple of the piece): pieces first, first + step, ... of
// 64 lanes each. The wave waits for vmcnt before it reads the copy.
template <typename Tin>
__device__ __forceinline__ void wave_copy(const Tin* src, Tin* dst, int len, int first, int step,
                                          int lane) {
    constexpr int kPer = 16 / static_cast<int>(sizeof(Tin));
    const int jl = lane * kPer;
    for (int base = first * kWave * kPer; base < len; base += step * kWave * kPer)
        if (base + jl < len) lds_dma16(src + base + jl, dst + base);
}

// Slot idx of size elements in the two C stage buffers viewed end to end
// (slots never straddle the two arrays).
template <typename Tin>
__device__ __forceinline__ Tin* stage_slot(Tin (*a)[kStageMax], Tin (*b)[kStageMax], int idx,
                                           int size) {
    const int per = (2 * kStageMax) / size;
    return idx < per ? &a[0][0] + idx * size : &b[0][0] + (idx - per) * size;
}

template <typename Tin>
__device__ __forceinline__ void stage_row(const Tin* row, Tin* dst, int cs, int len, bool vec4,
                                          int issuer, int lane) {
    if (vec4)
        stage_pieces<16>(row + cs, dst, len, issuer, lane);
    else
        stage_pieces<4>(row + cs, dst, len, issuer, lane);
}

// Row n0 + s of B or C for pair step p (chunk p / pairs, state
// 2 * (p % pairs) + s), positions of that chunk, into dst.
template <int kPairs, typename Tin>
__device__ __forceinline__ void stage_one(const Tin* base, int p, int s, Tin* dst, int L, int chunk,
                                          bool vec4, int issuer, int lane) {
    const int ci = p / kPairs, n0 = 2 * (p - ci * kPairs);
    const int cs = ci * chunk;
    const int len = L - cs < chunk ? L - cs : chunk;
    stage_row(base + static_cast<size_t>(n0 + s) * L, dst, cs, len, vec4, issuer, lane);
}

// Wait until this wave's outstanding vector-memory operations (including the
// LDS copies above) are done: vmcnt(0), other counters untouched.
__device__ __forceinline__ void wait_vmem() { __builtin_amdgcn_s_waitcnt(0x0f70); }

// kOne: the sequence fits one chunk (the launcher's choice), which then
// carries no state out; otherwise every chunk passes its carry on (the last
// one's is formed and not read).
template <int N, int T, int kWv, typename Tin, typename Tout, bool kTwoD, bool kZoh, bool kOne>
__global__ __launch_bounds__(kStageThreads) void k_full_scan_chunked(
    const Tin* __restrict__ u, const Tin* __restrict__ delta, const float* __restrict__ A,
    const Tin* __restrict__ Bm, const Tin* __restrict__ Cm, const float* __restrict__ D,
    const float* __restrict__ dt_bias, Tout* __restrict__ y, const Tin* __restrict__ xt, int K,
    int Dc, int L, int H, int W, int softplus, int n_groups, int n_wg) {
    static_assert(N % 4 == 0, "states go in pairs, and pairs alternate stage buffers");
    static_assert(kComputeWaves % kWv == 0, "whole channels per workgroup");
    constexpr int kPairs = N / 2;
    constexpr int G = kComputeWaves / kWv;  // channels per workgroup
    // per (parity, state of the pair, channel): aggregates exchanged across
    // waves, after kLead identity slots (see lane_entry)
    constexpr int kLead = kOne ? kWv - 1 : 0;  // identity slots before the waves'
    constexpr int kSlots = kLead + kWv;
    __shared__ __align__(16) float xagg[2][2][G][kSlots][2];
    __shared__ __align__(16) float arow[G][N];  // A rows of the workgroup's channels
    __shared__ float hcar[kComputeWaves][N];    // per wave: state carried into the next chunk
    // B and C slices of a pair of states, double-buffered (distinct arrays so
    // that copies into one buffer never order reads of the other)
    __shared__ __align__(16) Tin bst0[2][kStageMax], bst1[2][kStageMax];
    __shared__ __align__(16) Tin cst0[2][kStageMax], cst1[2][kStageMax];
    // per compute wave: its outputs on their way to a coalesced store
    __shared__ __align__(16) float ystage[kComputeWaves][kWave * T];

    // XCD-aware numbering: hardware places workgroup i on XCD i % 8, and
    // consecutive logical numbers share an XCD. Logical order: channel
    // groups of one (batch, direction) together (B and C are shared by them)
    // or, for a 2-D sequence of one chunk, the four directions of one
    // channel group together (they read the same input planes, which then
    // come from that XCD's L2 after the first read; 56x56: 26.2 -> 25.6 us
    // per SS2D step). Sequences of several chunks keep the first order,
    // where B and C are read once per chunk.
    const int bid = blockIdx.x;
    const int per = n_wg / 8, rem = n_wg % 8;
    const int xcd = bid % 8, slot = bid / 8;
    const int logical = xcd < rem ? xcd * (per + 1) + slot : rem * (per + 1) + (xcd - rem) * per + slot;
    int dg, bk;  // bk = b * K + k
    if constexpr (kTwoD && kOne) {
        const int rest = logical / K;
        dg = rest % n_groups;
        bk = (rest / n_groups) * K + logical % K;
    } else {
        dg = logical % n_groups;
        bk = logical / n_groups;
    }
    const int k = bk % K;
    const int b = bk / K;

    const int tid = threadIdx.x;
    const int lane = tid % kWave;
    const int wv = __builtin_amdgcn_readfirstlane(tid / kWave);
    constexpr int chunk = kWv * kWave * T;
    const int nchunks = kOne ? 1 : (L + chunk - 1) / chunk;
    const bool vec4 = (L % (16 / static_cast<int>(sizeof(Tin)))) == 0;
    // A sequence that fits one chunk, in rows of whole 16-byte pieces, has its
    // delta and u runs copied into LDS with coalesced pieces before the first
    // barrier and read from there (see the compute waves' prologue).
    const bool staged = nchunks == 1 && vec4;
    static_assert(kComputeWaves <= 2 * ((2 * kStageMax) / (kWave * T)), "u slots per wave");
    static_assert(G <= 2 * ((2 * kStageMax) / chunk), "plane slots per channel");
    const Tin* Bb = Bm + static_cast<size_t>(bk) * N * L;
    const Tin* Cb = Cm + static_cast<size_t>(bk) * N * L;

    if (wv >= kComputeWaves) {
        // Copy waves. Before barrier p they issue C of pair p and B of pair
        // p + 1, into buffers last read before barrier p - 1, then wait for
        // their completion; barrier p publishes them.
        const int npairs = nchunks * kPairs;  // step = (chunk, pair of states)
        const int issuer = wv - kComputeWaves;
        auto stage = [&](const Tin* base, int p, int st, Tin* dst) {
            stage_one<kPairs>(base, p, st, dst, L, chunk, vec4, issuer, lane);
        };
        stage(Bb, 0, 0, bst0[0]);
        stage(Bb, 0, 1, bst0[1]);
        wait_vmem();
        if (kTwoD && staged) __syncthreads();  // pairs with the plane barrier
        __syncthreads();
        for (int p = 0; p < npairs; ++p) {
            Tin (*cdst)[kStageMax] = (p & 1) ? cst1 : cst0;
            Tin (*bdst)[kStageMax] = (p & 1) ? bst0 : bst1;
            stage(Cb, p, 0, cdst[0]);
            stage(Cb, p, 1, cdst[1]);
            if (p + 1 < npairs) {
                stage(Bb, p + 1, 0, bdst[0]);
                stage(Bb, p + 1, 1, bdst[1]);
            }
            wait_vmem();
            __syncthreads();
        }
        return;
    }

    const int g = wv / kWv, w = wv - g * kWv;
    const int d_raw = dg * G + g;
    const bool d_ok = d_raw < Dc;
    const int d = d_ok ? d_raw : Dc - 1;
    const int c = k * Dc + d;
    const size_t row = (static_cast<size_t>(bk) * Dc + d) * static_cast<size_t>(L);
    const Tin* drow = delta + row;
    const Tin* urow = kTwoD ? u + (static_cast<size_t>(b) * Dc + d) * L : u + row;
    Tout* yrow = y + row;
    const float bias = dt_bias ? dt_bias[c] : 0.0f;
    const float dskip = D ? D[c] : 0.0f;
    const bool sp = softplus != 0;
    if (w == 0)
        for (int n = lane; n < N; n += kWave) arow[g][n] = A[static_cast<size_t>(c) * N + n];
    for (int n = lane; n < N; n += kWave) hcar[wv][n] = 0.0f;
    if constexpr (kLead > 0) {
        // the identity slots of the channel's rows (both parities, both states)
        constexpr int kId = kLead;
        if (w == 0 && lane < 4 * kId) {
            const int par = lane / (2 * kId), st = (lane / kId) % 2;
            xagg[par][st][g][lane % kId][0] = 1.0f;
            xagg[par][st][g][lane % kId][1] = 0.0f;
        }
    }
    const int run = (w * kWave + lane) * T;  // this lane's first position inside a chunk

    // This lane's run of delta and u for chunk ci; chunk 0's loads are issued
    // before the first barrier so that they overlap the first B copy.
    auto load_chunk = [&](int ci, float (&dv)[T], float (&uv)[T]) {
        const int t0 = ci * chunk + run;
        const int cnt = L - t0 < T ? (L - t0 > 0 ? L - t0 : 0) : T;
        const int tl = cnt > 0 ? t0 : 0;  // keep addresses in range for empty runs
        load_run<T>(drow + tl, dv, cnt == T, cnt);
        if constexpr (kTwoD) {
            // directions 1 and 3 from the column-major copy when given: its
            // rows are those directions' sequences, read like directions 0, 2
            if ((k & 1) && xt)
                load_run_2d_global<T>(xt + (static_cast<size_t>(b) * Dc + d) * L, k - 1, tl, H, W,
                                      L, uv, cnt);
            else
                load_run_2d_global<T>(urow, k, tl, H, W, L, uv, cnt);
        } else
            load_run<T>(urow + tl, uv, cnt == T, cnt);
    };
    const float* an = arow[g];
    // One chunk, from this lane's delta / u run (dv, uv) to the stored y run.
    // Per position of the lane's run: the timescale (delta through softplus),
    // its log2(e) multiple dl2, the products du = delta u and D u (yv, where
    // the outputs accumulate), and the run's sum of dl2.
    auto prep = [&](float (&dv)[T], const float (&uv)[T], float (&dl2)[T], float (&du)[T],
                    float (&yv)[T], float& s2) __attribute__((always_inline)) {
        s2 = 0.0f;
        {
            if (sp) {
#pragma unroll
                for (int i = 0; i < T; ++i) dv[i] = timescale(dv[i] + bias, true);
            } else {
#pragma unroll
                for (int i = 0; i < T; ++i) dv[i] += bias;
            }
            // Positions past the end of the sequence (in the last chunk only)
            // come after every valid position of it, in the lane's run, in
            // lane order and in wave order: whatever they hold reaches no
            // valid position's state and no stored output, so they need no
            // masking.
#pragma unroll
            for (int i = 0; i < T; ++i) {
                const float dl = dv[i];
                dl2[i] = dl * kLog2e;
                du[i] = dl * uv[i];
                yv[i] = dskip * uv[i];
                s2 += dl2[i];
            }
        }
    };
    // The state steps of chunk ci and the store of its outputs. With several
    // chunks, the delta / u runs of chunk ci + 1 are loaded into (dvn, uvn)
    // before the stores: vector-memory operations retire in order, so a wait
    // for loads issued after the stores would wait for the stores as well.
    auto chunk_steps = [&](int ci, const float (&dl2)[T], const float (&du)[T], float (&yv)[T],
                           float s2, const float (&uv)[T], float (&dvn)[T], float (&uvn)[T])
                           __attribute__((always_inline)) {
        // One pair step per barrier: phase 1 reads B of the pair (published
        // by the previous barrier), the barrier publishes the wave aggregates
        // and C of the pair, phase 2 reads them.
        auto pair_step = [&](int n0, Tin (*bcur)[kStageMax], Tin (*ccur)[kStageMax],
                             float (*xq)[G][kSlots][2]) {
            constexpr bool kOut = !kOne;  // chunks pass a carry on
            const float2 a01 = *reinterpret_cast<const float2*>(an + n0);
            const float inv0 = kZoh ? 1.0f / a01.x : 0.0f, inv1 = kZoh ? 1.0f / a01.y : 0.0f;
            float a0[T], bu0[T], a1[T], bu1[T];
            float Pin0, Hin0, Pin1, Hin1;
            pair_phase1<T, Tin, kZoh>(a01.x, a01.y, dl2, du, s2, &bcur[0][run], &bcur[1][run], a0,
                                      bu0, a1, bu1, Pin0, Hin0, Pin1, Hin1, xq[0][g], xq[1][g],
                                      lane, kLead + w, uv, inv0, inv1);
            __syncthreads();
            pair_phase2<T, kWv, kOut>(a0, bu0, a1, bu1, Pin0, Hin0, Pin1, Hin1, &ccur[0][run],
                                      &ccur[1][run], yv, xq[0][g], xq[1][g], &hcar[wv][n0],
                                      &hcar[wv][n0 + 1], lane, w);
        };
#pragma unroll 1
        for (int q = 0; q < kPairs; q += 2) {
            pair_step(2 * q, bst0, cst0, xagg[0]);
            pair_step(2 * q + 2, bst1, cst1, xagg[1]);
        }
        if constexpr (!kOne) {
            // unconditional (past the last chunk every run is empty and reads
            // nothing), so that dvn / uvn hold nothing across the steps
            __builtin_amdgcn_sched_barrier(0);
            load_chunk(ci + 1, dvn, uvn);
            __builtin_amdgcn_sched_barrier(0);
        }
        const int seg0 = ci * chunk + w * kWave * T;  // this wave's first position
        if (d_ok && seg0 < L)
            store_wave<T>(yrow + seg0, yv, ystage[wv], lane, min(kWave * T, L - seg0),
                          (L & 3) == 0);
    };

    float dv0[T], uv0[T];
    if (staged) {
        // Loaded straight from global memory, each instruction of a stride-T
        // run load touches a cache line per lane (and in the 2-D layout the
        // column-major directions gather across the whole plane). Instead the
        // wave copies its delta range into its output slice and its u range
        // (sequence layout) or a share of its channel's plane (2-D layout:
        // every direction's positions map into the one plane) into the C
        // stage buffers, which the copy waves first fill after the first
        // barrier, then reads its runs from LDS (stride-T words, T odd:
        // conflict-free).
        const int seg0 = w * kWave * T;
        const int n = L - seg0 < kWave * T ? (L - seg0 > 0 ? L - seg0 : 0) : kWave * T;
        Tin* dsl = reinterpret_cast<Tin*>(ystage[wv]);
        wave_copy(drow + seg0, dsl, n, 0, 1, lane);
        const Tin* usl;
        if constexpr (kTwoD) {
            Tin* pl = stage_slot(cst0, cst1, g, chunk);
            wave_copy(urow, pl, L, w, kWv, lane);
            wait_vmem();
            __syncthreads();  // the channel's plane is complete
            usl = pl;
        } else {
            Tin* ul = stage_slot(cst0, cst1, wv, kWave * T);
            wave_copy(urow + seg0, ul, n, 0, 1, lane);
            wait_vmem();
            usl = ul;
        }
        const int cnt = L - run < T ? (L - run > 0 ? L - run : 0) : T;
#pragma unroll
        for (int i = 0; i < T; ++i) dv0[i] = to_f32(dsl[lane * T + i]);  // past the end: any
        if constexpr (kTwoD) {
            load_run_2d<T>(usl, k, cnt > 0 ? run : 0, H, W, L, uv0, cnt);
        } else {
#pragma unroll
            for (int i = 0; i < T; ++i) uv0[i] = to_f32(usl[lane * T + i]);
        }
    } else {
        load_chunk(0, dv0, uv0);
    }

    float dl2[T], du[T], yv[T], s2;
    if constexpr (kOne) {
        // the per-position products before the first barrier: waves whose
        // loads arrived early work while the others' are still in flight
        prep(dv0, uv0, dl2, du, yv, s2);
        __syncthreads();  // pairs with the copy waves' first barrier (B of pair 0)
    } else {
        __syncthreads();  // pairs with the copy waves' first barrier (B of pair 0)
        // keep every use of the loaded values after the barrier (the compiler
        // would otherwise wait for the loads before it)
#pragma unroll
        for (int i = 0; i < T; ++i) asm volatile("" : "+v"(dv0[i]), "+v"(uv0[i]));
        prep(dv0, uv0, dl2, du, yv, s2);
    }
    float dvn[T], uvn[T];  // the next chunk's runs (several chunks only)
    chunk_steps(0, dl2, du, yv, s2, uv0, dvn, uvn);
    if constexpr (!kOne) {
        for (int ci = 1; ci < nchunks; ++ci) {
            prep(dvn, uvn, dl2, du, yv, s2);
            chunk_steps(ci, dl2, du, yv, s2, uvn, dvn, uvn);
        }
    }
}

}  // namespace

// Chunked full scan: picks the run length and waves per channel from L.
namespace {
template <int N, int kWv, typename Tin, typename Tout, bool kTwoD, bool kZoh, bool kOne>
vmb_status launch_chunked_wv(const ScanArgs& a, Tout* y, const void* xt) {
    constexpr int T = 13;  // positions per lane run
    constexpr int G = kComputeWaves / kWv;  // channels per workgroup
    const int n_groups = int((a.channels + G - 1) / G);
    const long long n_wg = static_cast<long long>(n_groups) * a.K * a.batch;
    if (n_wg > 0x7fffffffLL) return VMB_ERR_UNSUPPORTED;
    const dim3 grid(static_cast<unsigned>(n_wg)), block(kStageThreads);
    hipLaunchKernelGGL((k_full_scan_chunked<N, T, kWv, Tin, Tout, kTwoD, kZoh, kOne>), grid, block,
                       0, a.stream,
                       static_cast<const Tin*>(a.u), static_cast<const Tin*>(a.delta), a.A,
                       static_cast<const Tin*>(a.B), static_cast<const Tin*>(a.C), a.D, a.dt_bias,
                       y, static_cast<const Tin*>(xt), int(a.K), int(a.channels), int(a.L),
                       int(a.H), int(a.W), a.softplus, n_groups, int(n_wg));
    return check_launch();
}

// Waves per channel from L: cover the sequence in one chunk where possible
// (runs of 13 positions, 64 lanes per wave); longer sequences take chunks of
// the four-wave form.
template <int N, typename Tin, typename Tout, bool kTwoD, bool kZoh>
vmb_status launch_chunked_waves(const ScanArgs& a, Tout* y, const void* xt) {
    const int64_t L = a.L;
    if (L > kChunkedOneChunkMaxL)
        return launch_chunked_wv<N, 4, Tin, Tout, kTwoD, kZoh, false>(a, y, xt);
    if (L > 2 * kWave * 13) return launch_chunked_wv<N, 4, Tin, Tout, kTwoD, kZoh, true>(a, y, xt);
    if (L > kWave * 13) return launch_chunked_wv<N, 2, Tin, Tout, kTwoD, kZoh, true>(a, y, xt);
    return launch_chunked_wv<N, 1, Tin, Tout, kTwoD, kZoh, true>(a, y, xt);
}

template <int N, typename Tin, typename Tout, bool kTwoD>
vmb_status launch_chunked_impl(const ScanArgs& a, Tout* y, const void* xt) {
    return (a.options & VMB_SCAN_ZOH) ? launch_chunked_waves<N, Tin, Tout, kTwoD, true>(a, y, xt)
                                      : launch_chunked_waves<N, Tin, Tout, kTwoD, false>(a, y, xt);
}
}  // namespace

static_assert(4 * kWave * 13 == kChunkedOneChunkMaxL, "one pass of the four-wave form");

vmb_status launch_full_chunked(const ScanArgs& a, void* y_seq, const void* xt) {
    if (a.N != 16) return VMB_ERR_UNSUPPORTED;
    const bool two_d = a.layout == VMB_LAYOUT_2D;
    if (a.in_dt == VMB_F32)
        return two_d ? launch_chunked_impl<16, float, float, true>(a, static_cast<float*>(y_seq), xt)
                     : launch_chunked_impl<16, float, float, false>(a, static_cast<float*>(y_seq),
                                                                   nullptr);
    if (two_d) return launch_chunked_impl<16, bf16_t, float, true>(a, static_cast<float*>(y_seq), xt);
    if (a.out_dt == VMB_BF16)
        return launch_chunked_impl<16, bf16_t, bf16_t, false>(a, static_cast<bf16_t*>(y_seq), nullptr);
    return launch_chunked_impl<16, bf16_t, float, false>(a, static_cast<float*>(y_seq), nullptr);
}

}  // namespace vmb
