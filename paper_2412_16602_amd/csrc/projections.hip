// projections.hip -- the selection projections of eq. 6 ahead of the scan.
//
// Appendix A, Mamba paragraph, eq. 6: the selection functions make B, C and
// the timescale depend on the input through linear projections,
//   s_B(u) = Linear_N(u),  s_C(u) = Linear_N(u),
//   s_Delta(u) = Broadcast_D(Linear_1(u)),  Delta = softplus(Parameter + s_Delta(u)).
// Per (batch, direction k) sequence u[d, t] (d over the channels) and with
// the direction's weights W[k] = [R timescale rows; N rows for B; N for C]:
//   x_dbl[r, t]   = sum_d W[k, r, d] u[d, t]            (r < R + 2N)
//   B[n, t]       = x_dbl[R + n, t],  C[n, t] = x_dbl[R + N + n, t]
//   delta[d, t]   = sum_r W_dt[k, d, r] x_dbl[r, t]     (rank R; R = 1 and no W_dt:
//                                                        x_dbl[0, t], the broadcast)
// delta is s_Delta(u): the scan adds the Parameter (dt_bias) and applies softplus.
//
// Both products are dense contractions and run on the matrix cores
// (v_mfma_f32_16x16x4f32, fp32 inputs and accumulation). The weights of a
// direction are shared by every position of every batch entry, so positions
// are flattened over (batch, t): a workgroup owns P = 16 CB consecutive
// flattened positions of one direction (CB = 1, 2 or 4 column blocks of 16,
// chosen on the host so that the grid fills the chip), and short sequences
// still fill whole tiles. A tile of 16 or 32 positions reads only part of
// each 128-byte line of a channel row; its neighbours read the rest. The
// dispatcher deals workgroups to the eight XCDs (each with its own L2)
// round-robin, so the 1-D grid is remapped to give each XCD a contiguous
// range of tiles: neighbours then share one L2 instead of each XCD fetching
// the line again.
//   1. x_dbl: the channels are walked in chunks of 64; each chunk of u and of
//      W is staged in LDS (row strides padded by one word: the MFMA operand
//      reads are conflict-free) while the next chunk is already being loaded
//      into registers. The four waves split the work as CB column blocks x
//      KS = 4 / CB interleaved channel slices; each wave accumulates all
//      R + 2N rows (MB 16-row blocks) of its column block over its slice, and
//      the slices are summed through LDS. B and C rows leave from the
//      accumulators; the R timescale rows go to LDS.
//      bf16 inputs take the bf16 matrix cores (v_mfma_f32_16x16x16_bf16): u
//      is exact in bf16, W is split into bf16 hi + lo parts (hi the rounded
//      W, lo the rounded remainder), and the two products per row block
//      are exact in fp32, so W is carried to about 2^-17 of itself (far
//      below the bf16 rounding of the outputs) at eight times the fp32
//      matrix rate. u is staged transposed ([position][channel]) and W as
//      [row][channel], so each lane's four consecutive channels are one
//      8-byte LDS read.
//   2. delta: W_dt is staged in LDS 64 channels at a time (a contiguous
//      block); each wave takes one 16-channel row block of the chunk and all
//      column blocks, K = R in steps of 4.
// MFMA 16x16x4 operand layout: lane l holds A[l % 16][l / 16] and
// B[l / 16][l % 16]; result register v of lane l is D[4 (l / 16) + v][l % 16].
#include "vmb_internal.h"

namespace vmb {
namespace {

constexpr int kDC = 64;           // channels per staged chunk
constexpr int kPadD = kDC + 1;    // LDS row stride of the W chunk
constexpr int kMaxMB = 6;         // 16-row blocks of x_dbl at most (R <= 64, N <= 16)
constexpr int kMaxR = 64;         // timescale rank at most
constexpr int kPadR = kMaxR + 1;  // LDS row stride of the W_dt chunk

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef short s16x4 __attribute__((ext_vector_type(4)));
constexpr int kStrideB = kDC + 4;  // bf16 LDS row stride (elements): 8-byte aligned rows

__device__ __forceinline__ f32x4 mfma16x16x4(float a, float b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

// D += A B with A 16 x 16 (rows x K) and B 16 x 16 (K x columns) in bf16:
// lane l holds A[l % 16][4 (l / 16) .. + 3] and B[4 (l / 16) .. + 3][l % 16]
__device__ __forceinline__ f32x4 mfma16x16x16bf16(s16x4 a, s16x4 b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ unsigned short bf16_bits(float x) {
    const bf16_t h = from_f32<bf16_t>(x);
    return *reinterpret_cast<const unsigned short*>(&h);
}
__device__ __forceinline__ float bf16_value(unsigned short b) {
    return __uint_as_float(static_cast<unsigned>(b) << 16);
}

// an offset the compiler cannot see through: a load at a selected offset
// stays one unconditional load instead of a branch per arm of the select
__device__ __forceinline__ size_t opaque(size_t x) {
    asm("" : "+v"(x));
    return x;
}

template <typename T, int MB, int CB>
__global__ __launch_bounds__(256) void k_projections(
    const T* __restrict__ u, const float* __restrict__ W, const float* __restrict__ Wdt,
    T* __restrict__ delta, T* __restrict__ Bo, T* __restrict__ Co, int K, int Dc, int L, int N,
    int R, int64_t positions, int tiles) {
    constexpr int P = 16 * CB;   // positions per workgroup
    constexpr int PP = P + 1;    // LDS row stride of the u chunk and the timescale rows
    constexpr int KS = 4 / CB;   // channel slices
    constexpr bool kBf = sizeof(T) == 2;  // bf16 matrix-core path
    // staging sizes in floats: fp32 u [channel][position] and W [row][channel];
    // bf16 u [position][channel] and W hi, lo [row][channel] (2-byte elements)
    constexpr int kUsz = kBf ? (P * kStrideB) / 2 : kDC * PP;
    constexpr int kWsz = kBf ? 16 * MB * kStrideB : 16 * MB * kPadD;
    constexpr int kPool = (kUsz + kWsz) > kDC * kPadR ? (kUsz + kWsz) : kDC * kPadR;
    static_assert((KS - 1) * CB * MB * 256 <= kPool, "partials fit the staging pool");
    __shared__ __align__(16) float pool[kPool];  // phase 1: u chunk, W chunk, partials; phase 2: W_dt chunk
    __shared__ float ss[kMaxR * PP];  // timescale rows x_dbl[0 .. R)
    float* su = pool;
    float* sw = pool + kUsz;
    unsigned short* su16 = reinterpret_cast<unsigned short*>(pool);
    unsigned short* swh = reinterpret_cast<unsigned short*>(pool + kUsz);
    unsigned short* swl = swh + 16 * MB * kStrideB;

    // XCD-contiguous tile order: workgroup i runs on XCD i % 8; XCD x takes
    // tiles [x q + min(x, rem), ...) of the K * tiles in (k, tile) order
    const int nwg = static_cast<int>(gridDim.x), wg = static_cast<int>(blockIdx.x);
    const int q = nwg / 8, rem = nwg % 8, xcd = wg % 8, idx = wg / 8;
    const int logical = xcd * q + (xcd < rem ? xcd : rem) + idx;
    const int k = logical / tiles;
    const int64_t p0 = static_cast<int64_t>(logical - k * tiles) * P;
    const int tid = threadIdx.x, lane = tid & 63;
    const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int col = lane & 15, kq = lane >> 4;  // MFMA operand coordinates
    const int cb = wv % CB, ks = wv / CB;       // this wave's column block and channel slice
    const int M = R + 2 * N;                    // (M + 15) / 16 == MB
    const size_t l = static_cast<size_t>(L);
    const float* Wk = W + static_cast<size_t>(k) * M * Dc;

    // offset of flattened position p0 + c in a [batch, K, rows, L] tensor, row 0
    auto pos_base = [&](int c, int rows, bool& ok) -> size_t {
        const int64_t p = p0 + c;
        ok = p < positions;
        if (!ok) return 0;
        const int64_t b = p / L, t = p - b * L;
        return (static_cast<size_t>(b) * K + k) * rows * l + static_cast<size_t>(t);
    };

    // chunk loaders: u rows over threads with a fixed position per thread,
    // W rows with a fixed channel per thread
    constexpr int kURows = 256 / P;  // u rows per pass
    constexpr int kUL = kDC / kURows;
    constexpr int kWL = 16 * MB / 4;
    const int uc = tid % P, ur0 = tid / P;
    bool uok;
    const size_t ubase = pos_base(uc, Dc, uok);
    const int wc = tid & 63, wr0 = tid >> 6;
    // The loads are unconditional (an element out of range reads element 0
    // instead) and keep the raw values, so a chunk's loads stay in flight
    // until its LDS store. For 2-byte inputs the offset is made opaque: a
    // select between two addresses would otherwise become a branch per arm,
    // with the conversion (and so a wait) inside each.
    auto sel = [](size_t x) { return sizeof(T) == 2 ? opaque(x) : x; };
    T pu[kUL];
    float pw[kWL];
    auto u_ok = [&](int d0, int j) { return uok && d0 + ur0 + kURows * j < Dc; };
    auto w_ok = [&](int d0, int j) { return wr0 + 4 * j < M && d0 + wc < Dc; };
    auto load = [&](int d0) {
#pragma unroll
        for (int j = 0; j < kUL; ++j)
            pu[j] = u[sel(u_ok(d0, j) ? ubase + static_cast<size_t>(d0 + ur0 + kURows * j) * l
                                      : 0)];
#pragma unroll
        for (int j = 0; j < kWL; ++j)
            pw[j] = Wk[w_ok(d0, j) ? static_cast<size_t>(wr0 + 4 * j) * Dc + d0 + wc : 0];
    };

    // 1. x_dbl
    f32x4 acc[MB];
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) acc[mb] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
    load(0);
    for (int d0 = 0; d0 < Dc; d0 += kDC) {
        __syncthreads();  // the previous chunk has been read
        if constexpr (kBf) {
#pragma unroll
            for (int j = 0; j < kUL; ++j)
                su16[uc * kStrideB + ur0 + kURows * j] =
                    u_ok(d0, j) ? *reinterpret_cast<const unsigned short*>(&pu[j]) : 0;
#pragma unroll
            for (int j = 0; j < kWL; ++j) {
                const float w = w_ok(d0, j) ? pw[j] : 0.0f;
                const unsigned short hi = bf16_bits(w);
                swh[(wr0 + 4 * j) * kStrideB + wc] = hi;
                swl[(wr0 + 4 * j) * kStrideB + wc] = bf16_bits(w - bf16_value(hi));
            }
        } else {
#pragma unroll
            for (int j = 0; j < kUL; ++j)
                su[(ur0 + kURows * j) * PP + uc] = u_ok(d0, j) ? to_f32(pu[j]) : 0.0f;
#pragma unroll
            for (int j = 0; j < kWL; ++j)
                sw[(wr0 + 4 * j) * kPadD + wc] = w_ok(d0, j) ? pw[j] : 0.0f;
        }
        __syncthreads();
        if (d0 + kDC < Dc) load(d0 + kDC);  // in flight during this chunk's products
        if constexpr (kBf) {
#pragma unroll
            for (int j = 0; j < 4 / KS; ++j) {
                const int kk = 16 * (ks + KS * j) + 4 * kq;
                const s16x4 bv =
                    *reinterpret_cast<const s16x4*>(&su16[(16 * cb + col) * kStrideB + kk]);
#pragma unroll
                for (int mb = 0; mb < MB; ++mb) {
                    const int wo = (16 * mb + col) * kStrideB + kk;
                    acc[mb] = mfma16x16x16bf16(*reinterpret_cast<const s16x4*>(&swh[wo]), bv,
                                               acc[mb]);
                    acc[mb] = mfma16x16x16bf16(*reinterpret_cast<const s16x4*>(&swl[wo]), bv,
                                               acc[mb]);
                }
            }
        } else {
#pragma unroll
            for (int j = 0; j < 16 / KS; ++j) {
                const int kk = 4 * (ks + KS * j);
                const float bval = su[(kk + kq) * PP + 16 * cb + col];
#pragma unroll
                for (int mb = 0; mb < MB; ++mb)
                    acc[mb] = mfma16x16x4(sw[(16 * mb + col) * kPadD + kk + kq], bval, acc[mb]);
            }
        }
    }
    if constexpr (KS > 1) {  // sum the channel slices into slice 0
        __syncthreads();
        if (ks > 0) {
#pragma unroll
            for (int mb = 0; mb < MB; ++mb)
#pragma unroll
                for (int v = 0; v < 4; ++v)
                    pool[(((ks - 1) * CB + cb) * MB + mb) * 256 + v * 64 + lane] = acc[mb][v];
        }
        __syncthreads();
        if (ks == 0) {
#pragma unroll
            for (int s = 1; s < KS; ++s)
#pragma unroll
                for (int mb = 0; mb < MB; ++mb)
#pragma unroll
                    for (int v = 0; v < 4; ++v)
                        acc[mb][v] += pool[(((s - 1) * CB + cb) * MB + mb) * 256 + v * 64 + lane];
        }
    }
    // B and C rows from the accumulators; the timescale rows to LDS
    if (ks == 0) {
        bool ok;
        const size_t nb = pos_base(16 * cb + col, N, ok);
#pragma unroll
        for (int mb = 0; mb < MB; ++mb) {
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                const int m = 16 * mb + 4 * kq + v;
                const float x = acc[mb][v];
                if (m < R) {
                    ss[m * PP + 16 * cb + col] = x;
                } else if (ok && m < M) {
                    T* dst = m < R + N ? Bo + nb + static_cast<size_t>(m - R) * l
                                       : Co + nb + static_cast<size_t>(m - R - N) * l;
                    *dst = from_f32<T>(x);
                }
            }
        }
    }
    __syncthreads();  // timescale rows written; the staging pool is free

    // 2. delta
    if (Wdt == nullptr) {
        // R = 1, Broadcast_D: every channel takes the timescale row; a
        // thread keeps one position and walks the channels
        if (!uok) return;
        const T x = from_f32<T>(ss[uc]);
        for (int d = ur0; d < Dc; d += kURows) delta[ubase + static_cast<size_t>(d) * l] = x;
        return;
    }
    size_t dbase[CB];
    bool dok[CB];
#pragma unroll
    for (int c = 0; c < CB; ++c) dbase[c] = pos_base(16 * c + col, Dc, dok[c]);
    const float* Wd = Wdt + static_cast<size_t>(k) * Dc * R;
    constexpr int RS = kMaxR / 4;
    float* swd = pool;
    // With a wide x_dbl block (MB >= 4: rank 17 or more at N = 16) the next
    // chunk of W_dt is loaded into registers while the current one is in
    // use: at rank 48 (7x7 stage, 1536 channels) each chunk is 12 KB and the
    // product over it is short, so a load that waits before every chunk left
    // the matrix cores idle most of the time. At low ranks the chunk is a
    // few hundred bytes and the extra registers cost more than they hide.
    constexpr bool kPrefetch = MB >= 4;
    constexpr int kPf = kPrefetch ? (kDC * kMaxR) / 256 : 1;
    float pf[kPf];
    auto fetch = [&](int d0) {
        const int n = (Dc - d0 < kDC ? Dc - d0 : kDC) * R;
#pragma unroll
        for (int j = 0; j < kPf; ++j) {
            const int i = tid + 256 * j;
            pf[j] = i < n ? Wd[static_cast<size_t>(d0) * R + i] : 0.0f;
        }
    };
    if constexpr (kPrefetch) fetch(0);
    for (int d0 = 0; d0 < Dc; d0 += kDC) {
        // W_dt rows d0 .. d0 + 64 are one contiguous block
        const int rows = Dc - d0 < kDC ? Dc - d0 : kDC;
        if constexpr (kPrefetch) {
#pragma unroll
            for (int j = 0; j < kPf; ++j) {
                const int i = tid + 256 * j;
                if (i < rows * R) {
                    const int r = i / R, c = i - r * R;
                    swd[r * kPadR + c] = pf[j];
                }
            }
        } else {
            for (int i = tid; i < rows * R; i += 256) {
                const int r = i / R, c = i - r * R;
                swd[r * kPadR + c] = Wd[static_cast<size_t>(d0) * R + i];
            }
        }
        __syncthreads();
        if constexpr (kPrefetch) {
            if (d0 + kDC < Dc) fetch(d0 + kDC);  // in flight during this chunk's products
        }
        const int dl = 16 * wv + col;  // A-operand row (channel within the chunk)
        float a[RS];
#pragma unroll
        for (int rs = 0; rs < RS; ++rs) {
            const int r = 4 * rs + kq;
            a[rs] = (r < R && dl < rows) ? swd[dl * kPadR + r] : 0.0f;
        }
#pragma unroll
        for (int c = 0; c < CB; ++c) {
            f32x4 o = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
            for (int rs = 0; rs < RS; ++rs) {
                const int r = 4 * rs + kq;
                if (4 * rs < R) o = mfma16x16x4(a[rs], r < R ? ss[r * PP + 16 * c + col] : 0.0f, o);
            }
            if (dok[c]) {
#pragma unroll
                for (int v = 0; v < 4; ++v) {
                    const int d = d0 + 16 * wv + 4 * kq + v;
                    if (d < Dc) delta[dbase[c] + static_cast<size_t>(d) * l] = from_f32<T>(o[v]);
                }
            }
        }
        __syncthreads();  // the W_dt chunk has been read
    }
}

// widest tile whose grid still gives every compute unit two workgroups
int column_blocks(int64_t positions, int64_t K) {
    for (int cb : {4, 2}) {
        const int64_t tiles = (positions + 16 * cb - 1) / (16 * cb);
        if (tiles * K >= 2 * 256) return cb;
    }
    return 1;
}

template <typename T, int MB, int CB>
void launch_mb(int64_t positions, hipStream_t s, const void* u, const float* W, const float* W_dt,
               void* delta, void* B, void* C, int K, int Dc, int L, int N, int R) {
    const int64_t tiles = (positions + 16 * CB - 1) / (16 * CB);
    hipLaunchKernelGGL((k_projections<T, MB, CB>), dim3(static_cast<unsigned>(tiles * K)),
                       dim3(256), 0, s, static_cast<const T*>(u), W, W_dt, static_cast<T*>(delta),
                       static_cast<T*>(B), static_cast<T*>(C), K, Dc, L, N, R, positions,
                       static_cast<int>(tiles));
}

template <typename T, int CB>
void launch_cb(int mb, int64_t positions, hipStream_t s, const void* u, const float* W,
               const float* W_dt, void* delta, void* B, void* C, int K, int Dc, int L, int N,
               int R) {
    switch (mb) {
        case 1: return launch_mb<T, 1, CB>(positions, s, u, W, W_dt, delta, B, C, K, Dc, L, N, R);
        case 2: return launch_mb<T, 2, CB>(positions, s, u, W, W_dt, delta, B, C, K, Dc, L, N, R);
        case 3: return launch_mb<T, 3, CB>(positions, s, u, W, W_dt, delta, B, C, K, Dc, L, N, R);
        case 4: return launch_mb<T, 4, CB>(positions, s, u, W, W_dt, delta, B, C, K, Dc, L, N, R);
        case 5: return launch_mb<T, 5, CB>(positions, s, u, W, W_dt, delta, B, C, K, Dc, L, N, R);
        default: return launch_mb<T, 6, CB>(positions, s, u, W, W_dt, delta, B, C, K, Dc, L, N, R);
    }
}

template <typename T>
void launch_t(int mb, int64_t positions, hipStream_t s, const void* u, const float* W,
              const float* W_dt, void* delta, void* B, void* C, int K, int Dc, int L, int N,
              int R) {
    const int cb = column_blocks(positions, K);
    if (cb == 4) return launch_cb<T, 4>(mb, positions, s, u, W, W_dt, delta, B, C, K, Dc, L, N, R);
    if (cb == 2) return launch_cb<T, 2>(mb, positions, s, u, W, W_dt, delta, B, C, K, Dc, L, N, R);
    return launch_cb<T, 1>(mb, positions, s, u, W, W_dt, delta, B, C, K, Dc, L, N, R);
}

}  // namespace

vmb_status launch_projections(const void* u, const float* W, const float* W_dt, void* delta,
                              void* B, void* C, int64_t batch, int64_t K, int64_t channels,
                              int64_t L, int64_t N, int64_t R, vmb_dtype dt, hipStream_t s) {
    const int64_t positions = batch * L;
    if (R > kMaxR || R + 2 * N > 16 * kMaxMB || (positions + 15) / 16 * K > int64_t{0x7fffffff})
        return VMB_ERR_UNSUPPORTED;
    const int mb = static_cast<int>((R + 2 * N + 15) / 16);
    if (dt == VMB_F32)
        launch_t<float>(mb, positions, s, u, W, W_dt, delta, B, C, int(K), int(channels), int(L),
                        int(N), int(R));
    else
        launch_t<bf16_t>(mb, positions, s, u, W, W_dt, delta, B, C, int(K), int(channels), int(L),
                         int(N), int(R));
    return check_launch();
}

}  // namespace vmb
