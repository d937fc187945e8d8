// cross.hip -- SS2D cross-scan (unfold) and cross-merge (fold) kernels.
//
// Appendix A (VMamba paragraph): the cross-scan unfolds an H x W map along
// four directions into four sequences of length L = H*W, and the cross-merge
// folds four sequences back into one map. Direction maps, pixel p = h*W + w:
//   pi_0 = p, pi_1 = w*H + h, pi_2 = L-1-pi_0, pi_3 = L-1-pi_1.
//
// Both kernels move a 32 x 32 pixel tile of one (batch, channel) plane per
// workgroup. The row-major directions are read / written along w; the
// column-major ones need the transposed tile, which goes through LDS so that
// every global access stays coalesced (consecutive lanes touch consecutive
// addresses, ascending for directions 0/1 and descending for 2/3).
#include "vmb_internal.h"

namespace vmb {
namespace {

constexpr int kTile = 32;
constexpr int kRows = 8;  // blockDim = (kTile, kRows)

template <typename T>
__global__ __launch_bounds__(kTile* kRows) void k_cross_scan(const T* __restrict__ x,
                                                             T* __restrict__ xs, int Dc, int H,
                                                             int W) {
    __shared__ T tile[kTile][kTile + 1];
    const int L = H * W;
    const int plane = blockIdx.x;  // b * Dc + d
    const int b = plane / Dc;
    const int d = plane - b * Dc;
    const int h0 = blockIdx.y * kTile, w0 = blockIdx.z * kTile;
    const T* src = x + static_cast<size_t>(plane) * L;
    const size_t seq = static_cast<size_t>(L);
    T* out0 = xs + (static_cast<size_t>(b) * 4 * Dc + d) * seq;  // direction 0
    T* out1 = out0 + static_cast<size_t>(Dc) * seq;              // direction 1
    T* out2 = out1 + static_cast<size_t>(Dc) * seq;              // direction 2
    T* out3 = out2 + static_cast<size_t>(Dc) * seq;              // direction 3

    const int tx = threadIdx.x, ty = threadIdx.y;
    // row-major directions straight from global, tile kept for the transpose
    for (int r = ty; r < kTile; r += kRows) {
        const int h = h0 + r, w = w0 + tx;
        if (h < H && w < W) {
            const int p = h * W + w;
            const T v = src[p];
            tile[r][tx] = v;
            out0[p] = v;
            out2[L - 1 - p] = v;
        }
    }
    __syncthreads();
    // column-major directions: lanes walk h (consecutive positions w*H + h)
    for (int r = ty; r < kTile; r += kRows) {
        const int w = w0 + r, h = h0 + tx;
        if (h < H && w < W) {
            const int q = w * H + h;
            const T v = tile[tx][r];
            out1[q] = v;
            out3[L - 1 - q] = v;
        }
    }
}

template <typename Tin, typename Tout>
__global__ __launch_bounds__(kTile* kRows) void k_cross_merge(const Tin* __restrict__ ys,
                                                              Tout* __restrict__ y, int Dc, int H,
                                                              int W) {
    __shared__ float t1[kTile][kTile + 1];
    __shared__ float t3[kTile][kTile + 1];
    const int L = H * W;
    const int plane = blockIdx.x;
    const int b = plane / Dc;
    const int d = plane - b * Dc;
    const int h0 = blockIdx.y * kTile, w0 = blockIdx.z * kTile;
    const size_t seq = static_cast<size_t>(L);
    const Tin* in0 = ys + (static_cast<size_t>(b) * 4 * Dc + d) * seq;
    const Tin* in1 = in0 + static_cast<size_t>(Dc) * seq;
    const Tin* in2 = in1 + static_cast<size_t>(Dc) * seq;
    const Tin* in3 = in2 + static_cast<size_t>(Dc) * seq;
    Tout* dst = y + static_cast<size_t>(plane) * L;

    const int tx = threadIdx.x, ty = threadIdx.y;
    // column-major directions: read along h (coalesced), park transposed
    for (int r = ty; r < kTile; r += kRows) {
        const int w = w0 + r, h = h0 + tx;
        if (h < H && w < W) {
            const int q = w * H + h;
            t1[tx][r] = to_f32(in1[q]);
            t3[tx][r] = to_f32(in3[L - 1 - q]);
        }
    }
    __syncthreads();
    for (int r = ty; r < kTile; r += kRows) {
        const int h = h0 + r, w = w0 + tx;
        if (h < H && w < W) {
            const int p = h * W + w;
            const float s02 = to_f32(in0[p]) + to_f32(in2[L - 1 - p]);
            const float s13 = t1[r][tx] + t3[r][tx];
            dst[p] = from_f32<Tout>(s02 + s13);
        }
    }
}

// grid: x = plane (b * channels + d), y = tile row, z = tile column
dim3 tile_grid(int64_t batch, int64_t channels, int64_t H, int64_t W) {
    return dim3(static_cast<unsigned>(batch * channels),
                static_cast<unsigned>((H + kTile - 1) / kTile),
                static_cast<unsigned>((W + kTile - 1) / kTile));
}

bool grid_fits(int64_t batch, int64_t channels, int64_t H, int64_t W) {
    return batch * channels <= (int64_t{1} << 24) && (H + kTile - 1) / kTile <= 65535 &&
           (W + kTile - 1) / kTile <= 65535;
}

}  // namespace

vmb_status launch_cross_scan(const void* x, void* xs, int64_t batch, int64_t channels,
                             int64_t H, int64_t W, vmb_dtype dt, hipStream_t s) {
    if (!grid_fits(batch, channels, H, W)) return VMB_ERR_UNSUPPORTED;
    const dim3 grid = tile_grid(batch, channels, H, W), block(kTile, kRows);
    if (dt == VMB_F32)
        hipLaunchKernelGGL(k_cross_scan<float>, grid, block, 0, s, static_cast<const float*>(x),
                           static_cast<float*>(xs), int(channels), int(H), int(W));
    else
        hipLaunchKernelGGL(k_cross_scan<bf16_t>, grid, block, 0, s,
                           static_cast<const bf16_t*>(x), static_cast<bf16_t*>(xs),
                           int(channels), int(H), int(W));
    return check_launch();
}

vmb_status launch_cross_merge(const void* ys, void* y, int64_t batch, int64_t channels,
                              int64_t H, int64_t W, vmb_dtype in_dt, vmb_dtype out_dt,
                              hipStream_t s) {
    if (!grid_fits(batch, channels, H, W)) return VMB_ERR_UNSUPPORTED;
    const dim3 grid = tile_grid(batch, channels, H, W), block(kTile, kRows);
    const int c = int(channels), h = int(H), w = int(W);
    if (in_dt == VMB_F32 && out_dt == VMB_F32)
        hipLaunchKernelGGL((k_cross_merge<float, float>), grid, block, 0, s,
                           static_cast<const float*>(ys), static_cast<float*>(y), c, h, w);
    else if (in_dt == VMB_F32 && out_dt == VMB_BF16)
        hipLaunchKernelGGL((k_cross_merge<float, bf16_t>), grid, block, 0, s,
                           static_cast<const float*>(ys), static_cast<bf16_t*>(y), c, h, w);
    else if (in_dt == VMB_BF16 && out_dt == VMB_BF16)
        hipLaunchKernelGGL((k_cross_merge<bf16_t, bf16_t>), grid, block, 0, s,
                           static_cast<const bf16_t*>(ys), static_cast<bf16_t*>(y), c, h, w);
    else
        return VMB_ERR_DTYPE;
    return check_launch();
}

}  // namespace vmb
