// out_norm.hip -- the step after the cross-merge in VMamba's SS2D block: a
// layer normalisation over the channels of each pixel and the SiLU gate.
// (The paper's text stops at the merge; this follows the public VMamba
// block that the paper's models are built from.)
//
// Per pixel p of image b, over the channels d of y[b, d, p] (the 2-D layout):
//   mu    = mean_d y,   var = mean_d (y - mu)^2   (biased)
//   out   = (y - mu) / sqrt(var + eps) * gamma[d] + beta[d]
//   out  *= z / (1 + exp(-z))                     (when z is given)
//
// Pixels are flattened over (batch, p): a workgroup owns PX consecutive
// flattened pixels and its 1024 threads are PX pixels x 1024 / PX channel
// groups (channel d belongs to group d % groups), so every load covers PX
// consecutive pixels of 64 / PX channel rows: PX = 16 for fp32 and 32 for
// bf16 (64-byte row segments either way), halved down to a quarter while the
// grid has fewer than 512 workgroups and every thread keeps four channels
// (short maps: 7x7 at batch 32 has 1568 pixels of 1536 channels). A thread loads all of its
// channels' y and z at once into registers (up to J = 32 each), so the whole
// tensor is in flight and HBM is read once; the mean and the centred sum of
// squares (exact in fp32 for any offset of the mean) are then formed from
// the registers. Wider channel counts stream the channels three times (the
// second and third reads from cache). The group sums are added across each
// wave by shuffles, then the waves' sums in LDS in wave order
// (deterministic). As in the projections, the 1-D grid is dealt to the XCDs
// in contiguous ranges of tiles, so neighbouring tiles, which share the
// 128-byte lines of a channel row, read them through one L2.
#include "vmb_internal.h"

namespace vmb {
namespace {

constexpr int kThreads = 1024;

// Sum of v over the channel groups of this thread's pixel, in a fixed order:
// a wave holds 64 / PX groups of the same PX pixels (lane l: pixel l % PX),
// which are first added across the wave (xor shuffles over the lane bits
// above the pixel's), then the waves' sums in wave order.
template <int PX>
__device__ __forceinline__ float group_total(float (*red)[PX + 1], float* tot, float v, int px,
                                             int grp) {
    constexpr int kWave = 64, kWaves = kThreads / kWave;
#pragma unroll
    for (int m = PX; m < kWave; m *= 2) v += __shfl_xor(v, m, kWave);
    const int lane = threadIdx.x % kWave, wv = threadIdx.x / kWave;
    if (lane < PX) red[wv][px] = v;
    __syncthreads();
    if (grp == 0) {
        float t = 0.0f;
#pragma unroll
        for (int w = 0; w < kWaves; ++w) t += red[w][px];
        tot[px] = t;
    }
    __syncthreads();
    return tot[px];
}

// J > 0: a thread's channels grp + 64 j (j < J) held in registers; J == 0:
// streamed.
template <typename T, int J, int PX>
__global__ __launch_bounds__(kThreads) void k_out_norm(const T* __restrict__ y,
                                                       const T* __restrict__ z,
                                                       const float* __restrict__ gamma,
                                                       const float* __restrict__ beta, float eps,
                                                       T* __restrict__ out, int Dc, int P,
                                                       int64_t pixels) {
    constexpr int kPx = PX, kGroups = kThreads / PX;
    __shared__ float red[kGroups][kPx + 1];
    __shared__ float tot[kPx];
    const int nwg = static_cast<int>(gridDim.x), wg = static_cast<int>(blockIdx.x);
    const int q = nwg / 8, rem = nwg % 8, xcd = wg % 8;
    const int tile = xcd * q + (xcd < rem ? xcd : rem) + wg / 8;
    const int px = threadIdx.x % kPx, grp = threadIdx.x / kPx;
    const int64_t p = static_cast<int64_t>(tile) * kPx + px;
    const bool ok = p < pixels;
    const int64_t pc = ok ? p : 0;  // clamped: loads stay in bounds
    const int64_t b = pc / P;
    const size_t base = static_cast<size_t>(b) * Dc * P + static_cast<size_t>(pc - b * P);
    const size_t pstride = static_cast<size_t>(P);
    const float inv_dc = 1.0f / static_cast<float>(Dc);

    auto finish = [&](int d, float v, float zv, float mu, float rstd) {
        float o = (v - mu) * rstd;
        if (gamma) o *= gamma[d];
        if (beta) o += beta[d];
        if (z) o *= zv / (1.0f + __expf(-zv));
        out[base + d * pstride] = from_f32<T>(o);
    };

    if constexpr (J > 0) {
        // raw values, converted at use: a conversion next to its load (or a
        // test of z per element) would make each load wait for the last
        T yr[J], zr[J];
#pragma unroll
        for (int j = 0; j < J; ++j) {
            const int d = grp + kGroups * j;
            yr[j] = y[base + static_cast<size_t>(d < Dc ? d : 0) * pstride];
        }
        if (z) {
#pragma unroll
            for (int j = 0; j < J; ++j) {
                const int d = grp + kGroups * j;
                zr[j] = z[base + static_cast<size_t>(d < Dc ? d : 0) * pstride];
            }
        }
        float yv[J];
#pragma unroll
        for (int j = 0; j < J; ++j) yv[j] = to_f32(yr[j]);
        float s = 0.0f;
#pragma unroll
        for (int j = 0; j < J; ++j)
            if (grp + kGroups * j < Dc) s += yv[j];
        const float mu = group_total<PX>(red, tot, s, px, grp) * inv_dc;
        float s2 = 0.0f;
#pragma unroll
        for (int j = 0; j < J; ++j) {
            const float c = yv[j] - mu;
            if (grp + kGroups * j < Dc) s2 = __builtin_fmaf(c, c, s2);
        }
        const float rstd = 1.0f / sqrtf(group_total<PX>(red, tot, s2, px, grp) * inv_dc + eps);
        if (!ok) return;
#pragma unroll
        for (int j = 0; j < J; ++j) {
            const int d = grp + kGroups * j;
            if (d < Dc) finish(d, yv[j], z ? to_f32(zr[j]) : 0.0f, mu, rstd);
        }
    } else {
        float s = 0.0f;
#pragma unroll 8
        for (int d = grp; d < Dc; d += kGroups) s += to_f32(y[base + d * pstride]);
        const float mu = group_total<PX>(red, tot, s, px, grp) * inv_dc;
        float s2 = 0.0f;
#pragma unroll 8
        for (int d = grp; d < Dc; d += kGroups) {
            const float c = to_f32(y[base + d * pstride]) - mu;
            s2 = __builtin_fmaf(c, c, s2);
        }
        const float rstd = 1.0f / sqrtf(group_total<PX>(red, tot, s2, px, grp) * inv_dc + eps);
        if (!ok) return;
#pragma unroll 4
        for (int d = grp; d < Dc; d += kGroups) {
            const size_t off = base + d * pstride;
            finish(d, to_f32(y[off]), z ? to_f32(z[off]) : 0.0f, mu, rstd);
        }
    }
}

template <typename T, int PX>
void launch_t(int64_t channels, hipStream_t s, const void* y, const void* z, const float* gamma,
              const float* beta, float eps, void* out, int P, int64_t pixels) {
    constexpr int kGroups = kThreads / PX;
    const dim3 grid(static_cast<unsigned>((pixels + PX - 1) / PX));
    const T* yy = static_cast<const T*>(y);
    const T* zz = static_cast<const T*>(z);
    T* oo = static_cast<T*>(out);
    const int Dc = static_cast<int>(channels);
    const int64_t j = (channels + kGroups - 1) / kGroups;
    if (j <= 4)
        hipLaunchKernelGGL((k_out_norm<T, 4, PX>), grid, dim3(kThreads), 0, s, yy, zz, gamma, beta,
                           eps, oo, Dc, P, pixels);
    else if (j <= 8)
        hipLaunchKernelGGL((k_out_norm<T, 8, PX>), grid, dim3(kThreads), 0, s, yy, zz, gamma, beta,
                           eps, oo, Dc, P, pixels);
    else if (j <= 16)
        hipLaunchKernelGGL((k_out_norm<T, 16, PX>), grid, dim3(kThreads), 0, s, yy, zz, gamma, beta,
                           eps, oo, Dc, P, pixels);
    else if (j <= 32)
        hipLaunchKernelGGL((k_out_norm<T, 32, PX>), grid, dim3(kThreads), 0, s, yy, zz, gamma, beta,
                           eps, oo, Dc, P, pixels);
    else
        hipLaunchKernelGGL((k_out_norm<T, 0, PX>), grid, dim3(kThreads), 0, s, yy, zz, gamma, beta,
                           eps, oo, Dc, P, pixels);
}

}  // namespace

vmb_status launch_out_norm(const void* y, const void* z, const float* gamma, const float* beta,
                           float eps, void* out, int64_t batch, int64_t channels, int64_t P,
                           vmb_dtype dt, hipStream_t s) {
    const int64_t pixels = batch * P;
    if ((pixels + 3) / 4 > int64_t{0x7fffffff}) return VMB_ERR_UNSUPPORTED;
    // widest tile (64-byte row segments) whose grid has 512 workgroups, as
    // long as every thread keeps at least four channels (the group sums are
    // added serially, so idle groups cost)
    auto shrink = [&](int px) {
        int k = 0;
        while (k < 2 && (pixels + px - 1) / px < 512 && channels >= 4 * (kThreads / (px / 2)))
            px /= 2, ++k;
        return px;
    };
    if (dt == VMB_F32) {
        const int px = shrink(16);
        if (px == 16) launch_t<float, 16>(channels, s, y, z, gamma, beta, eps, out, int(P), pixels);
        else if (px == 8) launch_t<float, 8>(channels, s, y, z, gamma, beta, eps, out, int(P), pixels);
        else launch_t<float, 4>(channels, s, y, z, gamma, beta, eps, out, int(P), pixels);
    } else {
        const int px = shrink(32);
        if (px == 32) launch_t<bf16_t, 32>(channels, s, y, z, gamma, beta, eps, out, int(P), pixels);
        else if (px == 16) launch_t<bf16_t, 16>(channels, s, y, z, gamma, beta, eps, out, int(P), pixels);
        else launch_t<bf16_t, 8>(channels, s, y, z, gamma, beta, eps, out, int(P), pixels);
    }
    return check_launch();
}

}  // namespace vmb
