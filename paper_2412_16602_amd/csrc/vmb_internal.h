// vmb_internal.h -- shared declarations of libvmb (host argument records,
// launchers) and small device helpers for gfx950.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "vmb.h"

namespace vmb {

// ---------------------------------------------------------------- host side

struct ScanArgs {
    const void* u;
    const void* delta;
    const float* A;
    const void* B;
    const void* C;
    const float* D;
    const float* dt_bias;
    int softplus;
    void* y;
    int64_t batch, K, channels, L, N;
    vmb_dtype in_dt, out_dt;
    vmb_layout layout;
    int64_t H, W;
    void* ws;
    size_t ws_bytes;
    unsigned options;  // vmb_mean_option bits (mean scan only)
    hipStream_t stream;
};

// Pure host-side checks (no HIP calls); see vmb_validate.cpp.
// unfold = true for the cross-scan (in: map, out: sequences), false for the merge.
vmb_status validate_cross(const void* in, const void* out, int64_t batch, int64_t channels,
                          int64_t H, int64_t W, vmb_dtype dt, bool unfold);
vmb_status validate_scan(const ScanArgs& a, int mean_variant);
vmb_status validate_discrete(const float* abar, const float* bu, const float* C, const float* skip,
                             const float* y, int64_t batch, int64_t channels, int64_t L);
vmb_status validate_channel_mean(const float* x, const float* xm, int64_t batch, int64_t channels,
                                 int64_t L);
size_t scan_workspace_bytes(int mean_variant, int64_t batch, int64_t K, int64_t channels,
                            int64_t L, int64_t N, vmb_layout layout);
vmb_status validate_out_norm(const void* y, const void* z, const float* gamma, const float* beta,
                             float eps, const void* out, int64_t batch, int64_t channels,
                             int64_t P, vmb_dtype dt);
vmb_status validate_projections(const void* u, const float* W, const float* W_dt,
                                const void* delta, const void* B, const void* C, int64_t batch,
                                int64_t K, int64_t channels, int64_t L, int64_t N, int64_t R,
                                vmb_dtype dt);

// Chunk length (positions) of the mean variant's reduce / carry / finish passes.
constexpr int kMeanChunk = 64;

// Positions per chunk of the mean variant. Lanes are positions, so a
// workgroup's time does not depend on the chunk length; full 64-position
// chunks keep every row segment the reduce reads whole (fewer, aligned cache
// lines) at no cost in parallelism: the per-SIMD channel work is the same.
inline int mean_chunk(int64_t /*batch*/, int64_t /*K*/, int64_t /*L*/) { return kMeanChunk; }

// Channel groups of the mean's reduce pass. One 16-wave workgroup per chunk
// of a (batch, direction) sequence leaves most compute units idle when there
// are few chunks (7x7 maps: one per sequence); the channels of a chunk are
// then split over G workgroups, whose partial sums a combine pass adds in
// group order. G fills about two workgroups per compute unit and leaves each
// wave at least four channels.
constexpr int64_t kMeanSplitBelow = 160;  // chunk-sequence workgroups below which to split
// (at 196, the 56x56 map, the one-launch path is faster: 16.8 us against 28.2 split in three)
constexpr int kMeanMaxGroups = 16;
inline int mean_groups(int64_t batch, int64_t K, int64_t channels, int64_t L) {
    const int64_t wgs = (L + kMeanChunk - 1) / kMeanChunk * K * batch;
    if (wgs >= kMeanSplitBelow) return 1;
    int64_t g = (512 + wgs - 1) / wgs;
    if (g > kMeanMaxGroups) g = kMeanMaxGroups;
    if (g > channels / 64) g = channels / 64;
    return g > 1 ? static_cast<int>(g) : 1;
}

// Completion record at the start of every mean-scan workspace (both
// readings' layouts), 64-bit words: word 0 holds the tag (epoch, odd) of the
// last call that used the workspace and word 2 its complement, so that no fill
// pattern reads as a recorded call; word 1 holds the tag of the last call whose
// bounded wait gave up, XORed with kFailTag.
constexpr size_t kMeanStatusBytes = 256;
constexpr unsigned long long kFailTag = 0x9e3779b97f4a7c15ull;
struct MeanStatus {
    unsigned long long* words;  // workspace base
    unsigned long long epoch;   // this call's tag (odd)
};

// Byte offsets of the mean variant's workspace regions (each 256-byte
// aligned), for bk = batch * K direction sequences of L positions:
//   status                    : the completion record above
//   scan  [bk][N][L][2] float : chunk-local inclusive scan (P, H)
//   rmean [bk][L]       float : channel mean of D * u
//   agg   [bk][nch][N][2]     : chunk aggregates
//   carry [bk][nch][N]        : state entering each chunk
//   ytil  [bk][L]             : 2-D layout only, the reduced output
//   xt    [batch*channels][L] : 2-D layout with L >= kMeanTransposeMinL only,
//                               column-major copies of the input planes
//   flags [bk][nch]     u64   : one-launch path's chunk flags
//   gpart [bk][nch][G][2N+3][64] : with G = mean_groups(..) > 1 only, each
//                               channel group's partial sums of a chunk
struct MeanWsLayout {
    size_t scan, rmean, agg, carry, ytil, xt, flags, gpart, total;
};
// Short planes (a few cache lines) are gathered directly instead: the copy
// pass costs more than it saves there. Planes beyond LDS are copied in 32 x 32
// tiles (2 x 128 x 512: the copy takes 55 us, the column gathers it replaces
// about 200 us of the reduce).
constexpr int64_t kMeanTransposeMinL = 256;
inline bool mean_transposes(int64_t L, bool two_d) {
    return two_d && L >= kMeanTransposeMinL;
}
inline MeanWsLayout mean_ws_layout(int64_t batch, int64_t K, int64_t channels, int64_t L,
                                   int64_t N, bool two_d) {
    auto up = [](size_t v) { return (v + 255) & ~size_t{255}; };
    const size_t bk = static_cast<size_t>(batch) * static_cast<size_t>(K);
    const int chunk = mean_chunk(batch, K, L);
    const size_t nch = static_cast<size_t>((L + chunk - 1) / chunk);
    MeanWsLayout o;
    o.scan = kMeanStatusBytes;
    o.rmean = o.scan + up(bk * N * L * 2 * 4);
    o.agg = o.rmean + up(bk * L * 4);
    o.carry = o.agg + up(bk * nch * N * 2 * 4);
    o.ytil = o.carry + up(bk * nch * N * 4);
    o.xt = o.ytil + (two_d ? up(bk * L * 4) : 0);
    const size_t planes = static_cast<size_t>(batch) * static_cast<size_t>(channels);
    o.flags = o.xt + (mean_transposes(L, two_d) ? up(planes * L * 4) : 0);
    o.gpart = o.flags + up(bk * nch * 8);  // one 64-bit flag per chunk
    const size_t groups = static_cast<size_t>(mean_groups(batch, K, channels, L));
    o.total = o.gpart +
              (groups > 1 ? up(bk * nch * groups * static_cast<size_t>(2 * N + 3) * kMeanChunk * 4)
                          : 0);
    return o;
}

// Workspace of the pooled reading (VMB_MEAN_POOLED), 256-byte aligned regions:
//   psum  [bk][N+2][L] : per-direction channel sums (exp sums per state, Delta u, D u)
//   abar, bu, cbar, h [batch][N][L] : the pooled scan's inputs, C_mean and its states
//   ones  [batch][L]   : the scan's output coefficient (its states are wanted as they are)
//   rbar  [batch][L]   : pooled skip term
//   ytil  [batch][4][L]: ytilde written once per direction (2-D merge input)
//   xt    [batch*channels][L] : 2-D layout with L >= kMeanTransposeMinL, as in the main reading
// after the completion record (kMeanStatusBytes).
struct PooledWsLayout {
    size_t psum, abar, bu, cbar, h, ones, rbar, ytil, xt, total;
};
inline PooledWsLayout pooled_ws_layout(int64_t batch, int64_t K, int64_t channels, int64_t L,
                                       int64_t N, bool two_d) {
    auto up = [](size_t v) { return (v + 255) & ~size_t{255}; };
    const size_t bk = static_cast<size_t>(batch) * static_cast<size_t>(K);
    const size_t b = static_cast<size_t>(batch), l = static_cast<size_t>(L), n = static_cast<size_t>(N);
    PooledWsLayout o;
    o.psum = kMeanStatusBytes;
    o.abar = o.psum + up(bk * (n + 2) * l * 4);
    o.bu = o.abar + up(b * n * l * 4);
    o.cbar = o.bu + up(b * n * l * 4);
    o.h = o.cbar + up(b * n * l * 4);
    o.ones = o.h + up(b * n * l * 4);
    o.rbar = o.ones + up(b * l * 4);
    o.ytil = o.rbar + up(b * l * 4);
    o.xt = o.ytil + up(b * 4 * l * 4);
    o.total = o.xt + (mean_transposes(L, two_d) ? up(b * static_cast<size_t>(channels) * l * 4) : 0);
    return o;
}

// Launchers (enqueue only; arguments already validated).
vmb_status launch_cross_scan(const void* x, void* xs, int64_t batch, int64_t channels,
                             int64_t H, int64_t W, vmb_dtype dt, hipStream_t s);
// Whether the cross-scan / merge kernels take the map at all (a plane in LDS,
// or 32 x 32 tiles within the grid limits); checked before any launch.
bool cross_fits(int64_t batch, int64_t channels, int64_t H, int64_t W);
// Column-major copy of every (batch, channel) plane, xt[plane][w * H + h]
// (direction 1's sequence), for any plane cross_fits accepts.
vmb_status launch_transpose_planes(const void* x, void* xt, int64_t batch, int64_t channels,
                                   int64_t H, int64_t W, vmb_dtype dt, hipStream_t s);
// Merge with independent input / output element types (fp32 -> bf16 is used
// by the 2-D scan layouts).
vmb_status launch_cross_merge(const void* ys, void* y, int64_t batch, int64_t channels,
                              int64_t H, int64_t W, vmb_dtype in_dt, vmb_dtype out_dt,
                              hipStream_t s);
vmb_status launch_full_scan(const ScanArgs& a);
// Selection projections of eq. 6 (projections.hip).
vmb_status launch_out_norm(const void* y, const void* z, const float* gamma, const float* beta,
                           float eps, void* out, int64_t batch, int64_t channels, int64_t P,
                           vmb_dtype dt, hipStream_t s);
vmb_status launch_projections(const void* u, const float* W, const float* W_dt, void* delta,
                              void* B, void* C, int64_t batch, int64_t K, int64_t channels,
                              int64_t L, int64_t N, int64_t R, vmb_dtype dt, hipStream_t s);
// One-state scan on materialised inputs and the channel mean (scan_discrete.hip).
vmb_status launch_discrete_scan(const float* abar, const float* bu, const float* C,
                                const float* skip, float* y, int64_t batch, int64_t channels,
                                int64_t L, hipStream_t s);
vmb_status launch_channel_mean(const float* x, float* xm, int64_t batch, int64_t channels,
                               int64_t L, hipStream_t s);
// Positions-over-lanes full scan (N == 16); writes sequence-layout output to
// y_seq (a.y for the sequence layout, the fp32 workspace for the 2-D one).
// 2-D layout: xt, when given, holds the column-major copies of the input
// planes, which directions 1 and 3 then read as contiguous rows.
vmb_status launch_full_chunked(const ScanArgs& a, void* y_seq, const void* xt);
// Longest sequence that kernel covers in one pass (4 waves x 64 lanes x 13
// positions); longer ones walk several chunks.
constexpr int64_t kChunkedOneChunkMaxL = 3328;

// Rows of L elements of size bytes are whole 128-byte cache lines (kernels
// store such rows non-temporally).
inline bool whole_lines(int64_t L, int size) { return (L * size) % 128 == 0; }
// Short sequences (L <= kShortMaxL, N == 16): whole sequences in segments of
// 16 or 32 lanes of one wave; writes sequence-layout output to y_seq.
constexpr int64_t kShortMaxL = 416;
bool use_short_full(const ScanArgs& a);
vmb_status launch_full_short(const ScanArgs& a, void* y_seq);
// Whether the positions-over-lanes kernel is the better fit for this shape.
bool use_chunked_full(const ScanArgs& a);
// Channels over lanes, states over the four waves of a workgroup, positions
// in tiles (N == 16, at least kTilesMinRows batch * K * channels rows);
// writes sequence-layout output to y_seq.
constexpr int64_t kTilesMinRows = 16384;
bool use_tiles_full(const ScanArgs& a);
bool tiles_take(const ScanArgs& a);
// The 2-D layout of that path also reads column-major copies of the input
// planes (xt, written by launch_transpose_planes into the workspace after the
// per-direction outputs), so directions 1 and 3 load contiguous rows.
vmb_status launch_full_tiles(const ScanArgs& a, void* y_seq, const void* xt);
// Full scan, 2-D layout: whether the workspace holds xt (the tile path's
// shapes with planes of 128 to 6144 positions: below, a plane spans a few
// cache lines and the column-major reads gather it from L1 faster than a copy
// pass; and the positions-over-lanes path's sequences of more than one
// chunk, whose one-chunk form stages the plane in LDS instead), where it
// starts (after the per-direction fp32 outputs), and its size (4 bytes per
// element, either input type).
inline bool full_ws_has_xt(int64_t batch, int64_t K, int64_t channels, int64_t L, int64_t N) {
    if (N != 16) return false;
    const bool tiles = batch * K * channels >= kTilesMinRows;
    return tiles ? (L >= 128 && L <= 6144) : L > kChunkedOneChunkMaxL;
}
inline size_t full_ws_xt_offset(int64_t batch, int64_t K, int64_t channels, int64_t L) {
    const size_t seq = static_cast<size_t>(batch) * K * channels * L;
    return (seq * 4 + 255) & ~size_t{255};
}
inline size_t full_ws_xt_bytes(int64_t batch, int64_t channels, int64_t L) {
    return (static_cast<size_t>(batch) * channels * L * 4 + 255) & ~size_t{255};
}
vmb_status launch_mean_scan(const ScanArgs& a);
// Reads the completion record of a mean-scan workspace (synchronises the stream).
vmb_status mean_scan_status(const void* ws, hipStream_t s);

inline vmb_status check_launch() {
    return hipGetLastError() == hipSuccess ? VMB_OK : VMB_ERR_HIP;
}

}  // namespace vmb

#include "vmb_device.h"
