// cross.hip -- SS2D cross-scan (unfold) and cross-merge (fold) kernels.
//
// Appendix A (VMamba paragraph): the cross-scan unfolds an H x W map along
// four directions into four sequences of length L = H*W, and the cross-merge
// folds four sequences back into one map. Direction maps, pixel p = h*W + w:
//   pi_0 = p, pi_1 = w*H + h, pi_2 = L-1-pi_0, pi_3 = L-1-pi_1.
//
// Planes that fit in LDS (the feature maps of VMamba's stages) are moved by
// one workgroup each (small planes, and for the cross-scan mid-size planes
// when there are many, several to a workgroup), 16 bytes per lane: directions 0 and 2 (and the merge's
// own row order) straight between registers and memory, directions 1 and 3
// through a padded copy of the plane in LDS (row stride W + 1 words, so the
// column walk is free of bank conflicts). Every global access is a full
// 16-byte vector of consecutive elements. Larger planes use 32 x 32 pixel
// tiles (blockDim 32 x 8) with an LDS transpose for the column directions.
#include "vmb_internal.h"

namespace vmb {
namespace {

constexpr int kTile = 32;
constexpr int kRows = 8;  // blockDim = (kTile, kRows)

// kAll = false writes only the column-major copy of each plane (direction
// 1's sequence), to xs[plane][L].
template <typename T, bool kAll = true>
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
    T* out1 = kAll ? out0 + static_cast<size_t>(Dc) * seq         // direction 1
                   : xs + static_cast<size_t>(plane) * seq;
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
            if constexpr (kAll) {
                out0[p] = v;
                out2[L - 1 - p] = v;
            }
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
            if constexpr (kAll) out3[L - 1 - q] = v;
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

// ---- whole-plane kernels (one workgroup per (batch, channel) plane)

constexpr int kPlaneThreads = 768;
constexpr int kPlaneLdsWords = 12288;  // padded plane H * (W + 1) fp32 words (48 KB)

template <typename T, int V>
struct Vec {
    T v[V];
};

// Whole vectors at their natural alignment (callers guarantee it).
template <typename T, int V>
__device__ __forceinline__ Vec<T, V> load_vec(const T* p) {
    Vec<T, V> r;
    __builtin_memcpy(&r, __builtin_assume_aligned(p, sizeof(r)), sizeof(r));
    return r;
}

template <typename T, int V, bool kNt = false>
__device__ __forceinline__ void store_vec(T* p, const Vec<T, V>& r) {
    store_out<kNt>(reinterpret_cast<Vec<T, V>*>(p), r);
}

// V elements per lane; L % V == 0 and 16-byte aligned planes when V > 1.
// kAll = false writes only the column-major copy of each plane (direction 1's
// sequence), to xs[plane][L].
// TPP threads per plane, kPlaneThreads / TPP planes per workgroup, each with
// its share of the LDS (small planes are batched, one wave each).
template <typename T, int V, bool kAll, int TPP, bool kNt>
__global__ __launch_bounds__(kPlaneThreads) void k_cross_scan_plane(const T* __restrict__ x,
                                                                    T* __restrict__ xs, int Dc,
                                                                    int H, int W, int nplanes) {
    constexpr int kShare = kPlaneLdsWords / (kPlaneThreads / TPP);
    __shared__ T tiles[kPlaneLdsWords];
    const int L = H * W, Wp = W + 1;
    const int sub = threadIdx.x / TPP, tid = threadIdx.x % TPP;
    T* tile = tiles + sub * kShare;
    const int pl = blockIdx.x * (kPlaneThreads / TPP) + sub;  // b * Dc + d
    const bool active = pl < nplanes;
    const int plane = active ? pl : nplanes - 1;
    const int b = plane / Dc;
    const int d = plane - b * Dc;
    const T* src = x + static_cast<size_t>(plane) * L;
    const size_t seq = static_cast<size_t>(L);
    T* out0 = xs + (static_cast<size_t>(b) * 4 * Dc + d) * seq;
    T* out1 = kAll ? out0 + static_cast<size_t>(Dc) * seq : xs + static_cast<size_t>(plane) * seq;
    T* out2 = out1 + static_cast<size_t>(Dc) * seq;
    T* out3 = out2 + static_cast<size_t>(Dc) * seq;
    const int nv = L / V;
    // every load of this lane issued first (one memory round trip), then
    // directions 0 and 2 from registers and the plane parked (padded) for 1, 3
    constexpr int kPer = (kShare / V + TPP - 1) / TPP;
    Vec<T, V> v[kPer];
#pragma unroll
    for (int i = 0; i < kPer; ++i) {
        const int j = tid + i * TPP;
        if (active && j < nv) v[i] = load_vec<T, V>(src + j * V);
    }
#pragma unroll
    for (int i = 0; i < kPer; ++i) {
        const int j = tid + i * TPP;
        if (!active || j >= nv) break;
        const int p = j * V;
        if constexpr (kAll) {
            store_vec<T, V, kNt>(out0 + p, v[i]);
            Vec<T, V> r;
#pragma unroll
            for (int e = 0; e < V; ++e) r.v[e] = v[i].v[V - 1 - e];
            store_vec<T, V, kNt>(out2 + (L - V - p), r);
        }
#pragma unroll
        for (int e = 0; e < V; ++e) {
            const int pe = p + e, h = pe / W, w = pe - h * W;
            tile[h * Wp + w] = v[i].v[e];
        }
    }
    __syncthreads();
    // directions 1 and 3: position q = w * H + h reads pixel (h, w)
    for (int j = tid; active && j < nv; j += TPP) {
        const int q = j * V;
        Vec<T, V> v, r;
#pragma unroll
        for (int e = 0; e < V; ++e) {
            const int qe = q + e, w = qe / H, h = qe - w * H;
            v.v[e] = tile[h * Wp + w];
            r.v[V - 1 - e] = v.v[e];
        }
        store_vec<T, V, kNt>(out1 + q, v);
        if constexpr (kAll) store_vec<T, V, kNt>(out3 + (L - V - q), r);
    }
}

template <typename Tin, typename Tout, int V, int TPP, bool kNt>
__global__ __launch_bounds__(kPlaneThreads) void k_cross_merge_plane(const Tin* __restrict__ ys,
                                                                     Tout* __restrict__ y, int Dc,
                                                                     int H, int W, int nplanes) {
    constexpr int kShare = kPlaneLdsWords / (kPlaneThreads / TPP);
    __shared__ float s13s[kPlaneLdsWords];
    const int L = H * W, Wp = W + 1;
    const int sub = threadIdx.x / TPP, tid = threadIdx.x % TPP;
    float* s13 = s13s + sub * kShare;
    const int pl = blockIdx.x * (kPlaneThreads / TPP) + sub;
    const bool active = pl < nplanes;
    const int plane = active ? pl : nplanes - 1;
    const int b = plane / Dc;
    const int d = plane - b * Dc;
    const size_t seq = static_cast<size_t>(L);
    const Tin* in0 = ys + (static_cast<size_t>(b) * 4 * Dc + d) * seq;
    const Tin* in1 = in0 + static_cast<size_t>(Dc) * seq;
    const Tin* in2 = in1 + static_cast<size_t>(Dc) * seq;
    const Tin* in3 = in2 + static_cast<size_t>(Dc) * seq;
    Tout* dst = y + static_cast<size_t>(plane) * L;
    const int nv = L / V;
    // every load of this lane issued first (one memory round trip)
    constexpr int kPer = (kShare / V + TPP - 1) / TPP;
    Vec<Tin, V> a1[kPer], a3[kPer], a0[kPer], a2[kPer];
#pragma unroll
    for (int i = 0; i < kPer; ++i) {
        const int j = tid + i * TPP;
        if (active && j < nv) {
            const int o = j * V;
            a1[i] = load_vec<Tin, V>(in1 + o);
            a3[i] = load_vec<Tin, V>(in3 + (L - V - o));
            a0[i] = load_vec<Tin, V>(in0 + o);
            a2[i] = load_vec<Tin, V>(in2 + (L - V - o));
        }
    }
    // y1 + y3 of each pixel, in column order (q = w * H + h), parked by pixel
#pragma unroll
    for (int i = 0; i < kPer; ++i) {
        const int j = tid + i * TPP;
        if (!active || j >= nv) break;
        const int q = j * V;
#pragma unroll
        for (int e = 0; e < V; ++e) {
            const int qe = q + e, w = qe / H, h = qe - w * H;
            s13[h * Wp + w] = to_f32(a1[i].v[e]) + to_f32(a3[i].v[V - 1 - e]);
        }
    }
    __syncthreads();
#pragma unroll
    for (int i = 0; i < kPer; ++i) {
        const int j = tid + i * TPP;
        if (!active || j >= nv) break;
        const int p = j * V;
        Vec<Tout, V> o;
#pragma unroll
        for (int e = 0; e < V; ++e) {
            const int pe = p + e, h = pe / W, w = pe - h * W;
            const float s02 = to_f32(a0[i].v[e]) + to_f32(a2[i].v[V - 1 - e]);
            o.v[e] = from_f32<Tout>(s02 + s13[h * Wp + w]);
        }
        store_vec<Tout, V, kNt>(dst + p, o);
    }
}

bool plane_fits(int64_t batch, int64_t channels, int64_t H, int64_t W) {
    return H * (W + 1) <= kPlaneLdsWords && batch * channels <= 0x7fffffff;
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


// Threads per plane: one wave for planes of up to 1024 padded words (12 per
// workgroup), else the whole block (larger planes gain from the extra loads
// in flight per plane more than from batching).
inline int plane_tpp(int64_t H, int64_t W) {
    return H * (W + 1) <= kPlaneLdsWords / 12 ? 64 : kPlaneThreads;
}

// The cross-scan (and the column-major plane copies) also batch planes of up
// to 4096 padded words, three per workgroup of 256 threads each, when there
// are planes for at least four such workgroups per CU. A whole block on a
// 56x56 bf16 plane leaves half its lanes idle (392 vectors of 8) and holds
// two planes per CU, too few loads in flight: batch 128, 192 channels,
// 139 -> 114 us. With few planes (stage-1, 192) batching would leave most CUs
// idle. The merge keeps whole blocks: each of its planes already has four
// inputs in flight, and three per workgroup took 250 against 223 us there.
constexpr int64_t kBatchPlanesMin = 3 * 4 * 256;
inline int scan_plane_tpp(int64_t planes, int64_t H, int64_t W) {
    const int64_t words = H * (W + 1);
    if (words > kPlaneLdsWords / 12 && words <= kPlaneLdsWords / 3 && planes >= kBatchPlanesMin)
        return 256;
    return plane_tpp(H, W);
}

template <typename T, int V, bool kAll>
void launch_scan_tpp(const T* xi, T* xo, int64_t planes, int c, int h, int w, hipStream_t s) {
    const int tpp = scan_plane_tpp(planes, h, w);
    const int ppw = kPlaneThreads / tpp;
    const dim3 grid(static_cast<unsigned>((planes + ppw - 1) / ppw)), block(kPlaneThreads);
    const int np = static_cast<int>(planes);
    // non-temporal stores for planes of whole cache lines (V > 1 only: others
    // are not)
    const bool nt = V > 1 && whole_lines(int64_t(h) * w, sizeof(T));
    if (tpp == 256 && nt)
        hipLaunchKernelGGL((k_cross_scan_plane<T, V, kAll, 256, V != 1>), grid, block, 0, s, xi, xo,
                           c, h, w, np);
    else if (tpp == 256)
        hipLaunchKernelGGL((k_cross_scan_plane<T, V, kAll, 256, false>), grid, block, 0, s, xi, xo,
                           c, h, w, np);
    else if (tpp == 64 && nt)
        hipLaunchKernelGGL((k_cross_scan_plane<T, V, kAll, 64, V != 1>), grid, block, 0, s, xi, xo, c,
                           h, w, np);
    else if (tpp == 64)
        hipLaunchKernelGGL((k_cross_scan_plane<T, V, kAll, 64, false>), grid, block, 0, s, xi, xo, c,
                           h, w, np);
    else if (nt)
        hipLaunchKernelGGL((k_cross_scan_plane<T, V, kAll, kPlaneThreads, V != 1>), grid, block, 0, s,
                           xi, xo, c, h, w, np);
    else
        hipLaunchKernelGGL((k_cross_scan_plane<T, V, kAll, kPlaneThreads, false>), grid, block, 0, s,
                           xi, xo, c, h, w, np);
}

template <bool kAll>
vmb_status launch_scan_planes(const void* x, void* xs, int64_t batch, int64_t channels, int64_t H,
                              int64_t W, vmb_dtype dt, hipStream_t s) {
    const int c = int(channels), h = int(H), w = int(W);
    const int64_t L = H * W, planes = batch * channels;
    if (dt == VMB_F32) {
        const float* xi = static_cast<const float*>(x);
        float* xo = static_cast<float*>(xs);
        if (L % 4 == 0)
            launch_scan_tpp<float, 4, kAll>(xi, xo, planes, c, h, w, s);
        else
            launch_scan_tpp<float, 1, kAll>(xi, xo, planes, c, h, w, s);
    } else {
        const bf16_t* xi = static_cast<const bf16_t*>(x);
        bf16_t* xo = static_cast<bf16_t*>(xs);
        if (L % 8 == 0)
            launch_scan_tpp<bf16_t, 8, kAll>(xi, xo, planes, c, h, w, s);
        else
            launch_scan_tpp<bf16_t, 1, kAll>(xi, xo, planes, c, h, w, s);
    }
    return check_launch();
}

}  // namespace

bool cross_fits(int64_t batch, int64_t channels, int64_t H, int64_t W) {
    return plane_fits(batch, channels, H, W) || grid_fits(batch, channels, H, W);
}

vmb_status launch_transpose_planes(const void* x, void* xt, int64_t batch, int64_t channels,
                                   int64_t H, int64_t W, vmb_dtype dt, hipStream_t s) {
    if (plane_fits(batch, channels, H, W))
        return launch_scan_planes<false>(x, xt, batch, channels, H, W, dt, s);
    // planes beyond LDS: 32 x 32 tiles
    if (!grid_fits(batch, channels, H, W)) return VMB_ERR_UNSUPPORTED;
    const dim3 grid = tile_grid(batch, channels, H, W), block(kTile, kRows);
    if (dt == VMB_F32)
        hipLaunchKernelGGL((k_cross_scan<float, false>), grid, block, 0, s,
                           static_cast<const float*>(x), static_cast<float*>(xt), int(channels),
                           int(H), int(W));
    else
        hipLaunchKernelGGL((k_cross_scan<bf16_t, false>), grid, block, 0, s,
                           static_cast<const bf16_t*>(x), static_cast<bf16_t*>(xt), int(channels),
                           int(H), int(W));
    return check_launch();
}

vmb_status launch_cross_scan(const void* x, void* xs, int64_t batch, int64_t channels,
                             int64_t H, int64_t W, vmb_dtype dt, hipStream_t s) {
    if (plane_fits(batch, channels, H, W))
        return launch_scan_planes<true>(x, xs, batch, channels, H, W, dt, s);
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

template <typename Tin, typename Tout, int V>
void launch_merge_tpp(const Tin* in, Tout* out, int64_t planes, int c, int h, int w, hipStream_t s) {
    const int tpp = plane_tpp(h, w);
    const int ppw = kPlaneThreads / tpp;
    const dim3 grid(static_cast<unsigned>((planes + ppw - 1) / ppw)), block(kPlaneThreads);
    const int np = static_cast<int>(planes);
    const bool nt = V > 1 && whole_lines(int64_t(h) * w, sizeof(Tout));
    if (tpp == 64 && nt)
        hipLaunchKernelGGL((k_cross_merge_plane<Tin, Tout, V, 64, V != 1>), grid, block, 0, s, in, out,
                           c, h, w, np);
    else if (tpp == 64)
        hipLaunchKernelGGL((k_cross_merge_plane<Tin, Tout, V, 64, false>), grid, block, 0, s, in, out,
                           c, h, w, np);
    else if (nt)
        hipLaunchKernelGGL((k_cross_merge_plane<Tin, Tout, V, kPlaneThreads, V != 1>), grid, block, 0,
                           s, in, out, c, h, w, np);
    else
        hipLaunchKernelGGL((k_cross_merge_plane<Tin, Tout, V, kPlaneThreads, false>), grid, block, 0,
                           s, in, out, c, h, w, np);
}

namespace {

// Planes of fewer than 128 pixels (7x7 maps) span a couple of cache lines:
// one thread per output pixel gathers its four directions straight from
// them (same association as above), with no LDS pass and every lane busy
// (the plane kernel leaves part of its 64 lanes idle on 49 pixels and, with
// L % 4 != 0, loads element by element).
constexpr int kSmallPlane = 128;

template <typename Tin, typename Tout>
__global__ __launch_bounds__(256) void k_cross_merge_small(const Tin* __restrict__ ys,
                                                           Tout* __restrict__ y, int Dc, int H,
                                                           int W, int64_t total) {
    const int64_t f = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
    if (f >= total) return;
    const int L = H * W;
    const int64_t plane = f / L;
    const int p = static_cast<int>(f - plane * L);
    const int64_t b = plane / Dc, d = plane - b * Dc;
    const int h = p / W, w = p - h * W;
    const int q = w * H + h;  // the pixel's position in the column-major directions
    const size_t seq = static_cast<size_t>(L);
    const Tin* in0 = ys + (static_cast<size_t>(b) * 4 * Dc + d) * seq;
    const Tin* in1 = in0 + static_cast<size_t>(Dc) * seq;
    const Tin* in2 = in1 + static_cast<size_t>(Dc) * seq;
    const Tin* in3 = in2 + static_cast<size_t>(Dc) * seq;
    const float s02 = to_f32(in0[p]) + to_f32(in2[L - 1 - p]);
    const float s13 = to_f32(in1[q]) + to_f32(in3[L - 1 - q]);
    y[f] = from_f32<Tout>(s02 + s13);
}

template <typename Tin, typename Tout>
void launch_merge_small(const void* ys, void* y, int64_t batch, int64_t channels, int64_t H,
                        int64_t W, hipStream_t s) {
    const int64_t total = batch * channels * H * W;
    hipLaunchKernelGGL((k_cross_merge_small<Tin, Tout>),
                       dim3(static_cast<unsigned>((total + 255) / 256)), dim3(256), 0, s,
                       static_cast<const Tin*>(ys), static_cast<Tout*>(y), int(channels), int(H),
                       int(W), total);
}

}  // namespace

template <typename Tin, typename Tout>
void launch_merge_plane(const void* ys, void* y, int64_t batch, int64_t channels, int64_t H,
                        int64_t W, hipStream_t s) {
    const int c = int(channels), h = int(H), w = int(W);
    const Tin* in = static_cast<const Tin*>(ys);
    Tout* out = static_cast<Tout*>(y);
    // 16-byte vectors on both sides: 4 elements of the wider type
    constexpr int V = (sizeof(Tin) == 2 && sizeof(Tout) == 2) ? 8 : 4;
    if ((H * W) % V == 0)
        launch_merge_tpp<Tin, Tout, V>(in, out, batch * channels, c, h, w, s);
    else
        launch_merge_tpp<Tin, Tout, 1>(in, out, batch * channels, c, h, w, s);
}

vmb_status launch_cross_merge(const void* ys, void* y, int64_t batch, int64_t channels,
                              int64_t H, int64_t W, vmb_dtype in_dt, vmb_dtype out_dt,
                              hipStream_t s) {
    if (H * W < kSmallPlane && (batch * channels * H * W + 255) / 256 <= int64_t{0x7fffffff}) {
        if (in_dt == VMB_F32 && out_dt == VMB_F32)
            launch_merge_small<float, float>(ys, y, batch, channels, H, W, s);
        else if (in_dt == VMB_F32 && out_dt == VMB_BF16)
            launch_merge_small<float, bf16_t>(ys, y, batch, channels, H, W, s);
        else if (in_dt == VMB_BF16 && out_dt == VMB_BF16)
            launch_merge_small<bf16_t, bf16_t>(ys, y, batch, channels, H, W, s);
        else
            return VMB_ERR_DTYPE;
        return check_launch();
    }
    if (plane_fits(batch, channels, H, W)) {
        if (in_dt == VMB_F32 && out_dt == VMB_F32)
            launch_merge_plane<float, float>(ys, y, batch, channels, H, W, s);
        else if (in_dt == VMB_F32 && out_dt == VMB_BF16)
            launch_merge_plane<float, bf16_t>(ys, y, batch, channels, H, W, s);
        else if (in_dt == VMB_BF16 && out_dt == VMB_BF16)
            launch_merge_plane<bf16_t, bf16_t>(ys, y, batch, channels, H, W, s);
        else
            return VMB_ERR_DTYPE;
        return check_launch();
    }
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
