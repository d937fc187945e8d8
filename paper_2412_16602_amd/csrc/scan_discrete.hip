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
// Per element the kernel reads 8 bytes (12 with skip) and writes 4, with
// about six VALU slots of work: bound by HBM.
//
// Channel mean: a thread owns 4 consecutive positions of one batch row and
// sums the channels in index order, eight loads in flight.
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

// Inclusive scan of (P, H) over the 64 lanes in lane order; a lane without a
// partner keeps its value (the identity). DPP reads of a VALU result need two
// independent instructions or s_nop in between.
__device__ __forceinline__ void lane_scan(float& P, float& H) {
    asm("s_nop 1\n"
        "v_fmac_f32_dpp %0, %0, %1 row_shr:1 row_mask:0xf bank_mask:0xf\n"
        "v_mul_f32_dpp %1, %1, %1 row_shr:1 row_mask:0xf bank_mask:0xf\n"
        "s_nop 0\n"
        "v_fmac_f32_dpp %0, %0, %1 row_shr:2 row_mask:0xf bank_mask:0xf\n"
        "v_mul_f32_dpp %1, %1, %1 row_shr:2 row_mask:0xf bank_mask:0xf\n"
        "s_nop 0\n"
        "v_fmac_f32_dpp %0, %0, %1 row_shr:4 row_mask:0xf bank_mask:0xf\n"
        "v_mul_f32_dpp %1, %1, %1 row_shr:4 row_mask:0xf bank_mask:0xf\n"
        "s_nop 0\n"
        "v_fmac_f32_dpp %0, %0, %1 row_shr:8 row_mask:0xf bank_mask:0xf\n"
        "v_mul_f32_dpp %1, %1, %1 row_shr:8 row_mask:0xf bank_mask:0xf\n"
        "s_nop 0\n"
        "v_fmac_f32_dpp %0, %0, %1 row_bcast:15 row_mask:0xa bank_mask:0xf\n"
        "v_mul_f32_dpp %1, %1, %1 row_bcast:15 row_mask:0xa bank_mask:0xf\n"
        "s_nop 0\n"
        "v_fmac_f32_dpp %0, %0, %1 row_bcast:31 row_mask:0xc bank_mask:0xf\n"
        "v_mul_f32_dpp %1, %1, %1 row_bcast:31 row_mask:0xc bank_mask:0xf\n"
        "s_nop 1\n"
        : "+v"(H), "+v"(P));
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

// kVec: L % 4 == 0 (every run start is 16-byte aligned).
template <bool kVec>
__global__ __launch_bounds__(kWave* kScanWaves) void k_discrete_scan(
    const float* __restrict__ abar, const float* __restrict__ bu, const float* __restrict__ C,
    const float* __restrict__ skip, float* __restrict__ y, int64_t nseq, int channels, int L) {
    const int lane = threadIdx.x % kWave;
    const int64_t s = static_cast<int64_t>(blockIdx.x) * kScanWaves + threadIdx.x / kWave;
    if (s >= nseq) return;  // whole waves: s is wave-uniform
    const int64_t b = s / channels;
    const size_t row = static_cast<size_t>(s) * L;
    const float* ap = abar + row;
    const float* bp = bu + row;
    const float* sp = skip ? skip + row : nullptr;
    const float* cp = C + static_cast<size_t>(b) * L;
    float* yp = y + row;
    float carry = 0.0f;  // state entering the chunk
    for (int c0 = 0; c0 < L; c0 += kChunk) {
        const int t0 = c0 + lane * kRun;
        const int cnt = L - t0 < kRun ? (L - t0 > 0 ? L - t0 : 0) : kRun;
        const int tl = cnt > 0 ? t0 : 0;  // in range for empty runs
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
        lane_scan(P, H);
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

constexpr int kMeanThreads = 256;
constexpr int kMeanUnroll = 8;

// kVec: L % 4 == 0, a thread sums 4 consecutive positions; else 1.
template <bool kVec>
__global__ __launch_bounds__(kMeanThreads) void k_channel_mean(const float* __restrict__ x,
                                                               float* __restrict__ xm,
                                                               int channels, int L, float inv) {
    constexpr int kPer = kVec ? 4 : 1;
    const int b = blockIdx.y;
    const int t = (blockIdx.x * kMeanThreads + threadIdx.x) * kPer;
    if (t >= L) return;
    const float* xb = x + static_cast<size_t>(b) * channels * L + t;
    float acc[kPer];
#pragma unroll
    for (int i = 0; i < kPer; ++i) acc[i] = 0.0f;
    int d = 0;
    // channels in index order; the loads of eight channels in flight
    for (; d + kMeanUnroll <= channels; d += kMeanUnroll) {
        float v[kMeanUnroll][kPer];
#pragma unroll
        for (int j = 0; j < kMeanUnroll; ++j) {
            const float* p = xb + static_cast<size_t>(d + j) * L;
            if constexpr (kVec) {
                const float4 q = *reinterpret_cast<const float4*>(p);
                v[j][0] = q.x; v[j][1] = q.y; v[j][2] = q.z; v[j][3] = q.w;
            } else {
                v[j][0] = *p;
            }
        }
#pragma unroll
        for (int j = 0; j < kMeanUnroll; ++j)
#pragma unroll
            for (int i = 0; i < kPer; ++i) acc[i] += v[j][i];
    }
    for (; d < channels; ++d) {
        const float* p = xb + static_cast<size_t>(d) * L;
        if constexpr (kVec) {
            const float4 q = *reinterpret_cast<const float4*>(p);
            acc[0] += q.x; acc[1] += q.y; acc[2] += q.z; acc[3] += q.w;
        } else {
            acc[0] += *p;
        }
    }
    float* o = xm + static_cast<size_t>(b) * L + t;
    if constexpr (kVec) {
        *reinterpret_cast<float4*>(o) =
            make_float4(acc[0] * inv, acc[1] * inv, acc[2] * inv, acc[3] * inv);
    } else {
        o[0] = acc[0] * inv;
    }
}

}  // namespace

vmb_status launch_discrete_scan(const float* abar, const float* bu, const float* C,
                                const float* skip, float* y, int64_t batch, int64_t channels,
                                int64_t L, hipStream_t s) {
    const int64_t nseq = batch * channels;
    const int64_t blocks = (nseq + kScanWaves - 1) / kScanWaves;
    if (blocks > 0x7fffffffLL || channels > 0x7fffffffLL) return VMB_ERR_UNSUPPORTED;
    const dim3 grid(static_cast<unsigned>(blocks)), block(kWave * kScanWaves);
    if (L % 4 == 0)
        hipLaunchKernelGGL(k_discrete_scan<true>, grid, block, 0, s, abar, bu, C, skip, y, nseq,
                           int(channels), int(L));
    else
        hipLaunchKernelGGL(k_discrete_scan<false>, grid, block, 0, s, abar, bu, C, skip, y, nseq,
                           int(channels), int(L));
    return check_launch();
}

vmb_status launch_channel_mean(const float* x, float* xm, int64_t batch, int64_t channels,
                               int64_t L, hipStream_t s) {
    if (batch > 65535 || channels > 0x7fffffffLL) return VMB_ERR_UNSUPPORTED;
    const float inv = 1.0f / static_cast<float>(channels);
    const bool vec = L % 4 == 0;
    const int64_t per = vec ? 4 : 1;
    const int64_t blocks = (L + kMeanThreads * per - 1) / (kMeanThreads * per);
    const dim3 grid(static_cast<unsigned>(blocks), static_cast<unsigned>(batch)),
        block(kMeanThreads);
    if (vec)
        hipLaunchKernelGGL(k_channel_mean<true>, grid, block, 0, s, x, xm, int(channels), int(L),
                           inv);
    else
        hipLaunchKernelGGL(k_channel_mean<false>, grid, block, 0, s, x, xm, int(channels), int(L),
                           inv);
    return check_launch();
}

}  // namespace vmb
