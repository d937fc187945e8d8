// vmb_device.h -- device helpers of libvmb for gfx950: bf16 storage type and
// conversions, exp2 / reciprocal, the timescale of eq. 6 (softplus) and the
// cross-scan position maps.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace vmb {

constexpr float kLog2e = 1.4426950408889634f;

struct bf16_t {
    uint16_t bits;
};

__device__ __forceinline__ float to_f32(float v) { return v; }
__device__ __forceinline__ float to_f32(bf16_t v) {
    return __uint_as_float(static_cast<uint32_t>(v.bits) << 16);
}

template <typename T>
__device__ __forceinline__ T from_f32(float v);
template <>
__device__ __forceinline__ float from_f32<float>(float v) { return v; }
template <>
__device__ __forceinline__ bf16_t from_f32<bf16_t>(float v) {
    // gfx950 converts with round-to-nearest-even in hardware (v_cvt_pk_bf16_f32).
    __bf16 h = static_cast<__bf16>(v);
    bf16_t r;
    __builtin_memcpy(&r.bits, &h, 2);
    return r;
}

// Store of one value of 2, 4, 8 or 16 bytes at p (aligned to its size),
// non-temporal with kNt: outputs nothing in the kernel reads again then
// stream out instead of sitting dirty in L2 until the kernel ends. Launchers
// choose kNt only for rows of whole 128-byte lines (whole_lines): stores that
// cover parts of lines, streamed out one by one, cost more than merging them
// in L2.
template <bool kNt, typename T>
__device__ __forceinline__ void store_out(T* p, const T& v) {
    constexpr int kBytes = static_cast<int>(sizeof(T));
    if constexpr (!kNt) {
        __builtin_memcpy(__builtin_assume_aligned(p, kBytes), &v, kBytes);
    } else if constexpr (kBytes == 16) {
        typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
        u32x4 x;
        __builtin_memcpy(&x, &v, 16);
        __builtin_nontemporal_store(x, reinterpret_cast<u32x4*>(p));
    } else if constexpr (kBytes == 8) {
        typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));
        u32x2 x;
        __builtin_memcpy(&x, &v, 8);
        __builtin_nontemporal_store(x, reinterpret_cast<u32x2*>(p));
    } else if constexpr (kBytes == 4) {
        unsigned int x;
        __builtin_memcpy(&x, &v, 4);
        __builtin_nontemporal_store(x, reinterpret_cast<unsigned int*>(p));
    } else {
        static_assert(kBytes == 2, "2, 4, 8 or 16 bytes");
        unsigned short x;
        __builtin_memcpy(&x, &v, 2);
        __builtin_nontemporal_store(x, reinterpret_cast<unsigned short*>(p));
    }
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }
__device__ __forceinline__ float fast_rcp(float x) { return __builtin_amdgcn_rcpf(x); }

__device__ __forceinline__ float fast_log2(float x) { return __builtin_amdgcn_logf(x); }

// log(1 + e) for e in [0, 1]: w = 1 + e rounds, so log(w) alone would lose
// the low bits of a small e; c = e - (w - 1) is that rounding error exactly
// (w - 1 is exact for w in [1, 2]), and log(1 + e) = log(w) + c / w to first
// order in c (|c| <= 2^-24). 1 / w is taken as 2 - w, exact at w = 1 and
// within half of c's size elsewhere, far below the result's rounding.
// Checked on the GPU against fp64 log1p over 2^22 inputs: 1.6e-7 relative.
__device__ __forceinline__ float log1p_unit(float e) {
    const float w = 1.0f + e;
    const float c = e - (w - 1.0f);
    constexpr float kLn2 = 0.69314718055994531f;
    return __builtin_fmaf(fast_log2(w), kLn2, c * (2.0f - w));
}

// softplus(v) = max(v, 0) + log(1 + exp(-|v|)), the timescale map of eq. 6.
__device__ __forceinline__ float softplus(float v) {
    const float e = fast_exp2(-__builtin_fabsf(v) * kLog2e);
    return __builtin_fmaxf(v, 0.0f) + log1p_unit(e);
}

// Timescale of eq. 6: softplus(v), or v itself when the softplus flag is off.
__device__ __forceinline__ float timescale(float v, bool sp) { return sp ? softplus(v) : v; }

// Zero-order-hold coefficient of B (eq. 4, second line read as
// (Delta A)^-1 (exp(Delta A) - I) Delta B): Bbar u = q * B with
// q = phi(x) Delta u, phi(x) = (e^x - 1) / x, x = Delta A. The caller passes
// x2 = x log2(e) and a = exp2(x2), which it has for Abar, and inv_a = 1 / A.
// Near x = 0, e^x - 1 cancels in binary32, so |x| < 0.02 takes phi's cubic
// Taylor polynomial (truncation below 1.3e-9 relative) and larger |x| takes
// (a - 1) u / A (the rounding of a then costs below 3e-6 relative).
__device__ __forceinline__ float zoh_q(float x2, float a, float du, float u, float inv_a) {
    constexpr float kLn2 = 0.69314718055994531f;
    constexpr float c1 = kLn2 / 2.0f, c2 = kLn2 * kLn2 / 6.0f, c3 = kLn2 * kLn2 * kLn2 / 24.0f;
    const float p = __builtin_fmaf(__builtin_fmaf(__builtin_fmaf(c3, x2, c2), x2, c1), x2, 1.0f);
    const float near = p * du;
    const float far = (a - 1.0f) * (inv_a * u);
    return __builtin_fabsf(x2) < 0.02f * kLog2e ? near : far;
}

// Cross-scan position maps. Direction k reads pixel pix(k, t) at position t:
//   k = 0: t                         k = 2: L - 1 - t
//   k = 1: (t % H) * W + t / H       k = 3: same as 1 at L - 1 - t
__device__ __forceinline__ int pixel_of(int k, int t, int H, int W) {
    const int L = H * W;
    const int tt = (k >= 2) ? (L - 1 - t) : t;
    if ((k & 1) == 0) return tt;
    const int w = tt / H;
    const int h = tt - w * H;
    return h * W + w;
}

}  // namespace vmb

namespace vmb {

// ---------------------------------------------------------------- DPP scans
// Inclusive scans over the lanes of a wave of the pair combine of the
// linear recurrence (Appendix A: the associative scan of eq. 3),
//   (P1, H1) then (P2, H2) -> (P1 P2, P2 H1 + H2),
// in lane order. Each level reads the partner lane through DPP inside the
// arithmetic (v_fmac / v_mul with a DPP source operand); a lane whose partner
// does not exist is not written, which is the identity. Wait states: a VALU
// result read through DPP needs two independent instructions (or s_nop) in
// between. Plain asm (no side effects): the scheduler may move other work
// around it.

// One pair over all 64 lanes (row shifts 1, 2, 4, 8, then the row
// broadcasts of lanes 15 and 31).
__device__ __forceinline__ void wave_scan(float& P, float& Hs) {
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
        : "+v"(Hs), "+v"(P));
}

// Two independent pairs (P0, H0) and (P1, H1) over all 64 lanes, their
// levels interleaved: each DPP read then follows the write of its register
// by three other instructions, so no wait states are needed inside.
__device__ __forceinline__ void wave_scan2(float& P0, float& H0, float& P1, float& H1) {
    asm("s_nop 1\n"
        "v_fmac_f32_dpp %0, %0, %1 row_shr:1 row_mask:0xf bank_mask:0xf\n"
        "v_fmac_f32_dpp %2, %2, %3 row_shr:1 row_mask:0xf bank_mask:0xf\n"
        "v_mul_f32_dpp %1, %1, %1 row_shr:1 row_mask:0xf bank_mask:0xf\n"
        "v_mul_f32_dpp %3, %3, %3 row_shr:1 row_mask:0xf bank_mask:0xf\n"
        "v_fmac_f32_dpp %0, %0, %1 row_shr:2 row_mask:0xf bank_mask:0xf\n"
        "v_fmac_f32_dpp %2, %2, %3 row_shr:2 row_mask:0xf bank_mask:0xf\n"
        "v_mul_f32_dpp %1, %1, %1 row_shr:2 row_mask:0xf bank_mask:0xf\n"
        "v_mul_f32_dpp %3, %3, %3 row_shr:2 row_mask:0xf bank_mask:0xf\n"
        "v_fmac_f32_dpp %0, %0, %1 row_shr:4 row_mask:0xf bank_mask:0xf\n"
        "v_fmac_f32_dpp %2, %2, %3 row_shr:4 row_mask:0xf bank_mask:0xf\n"
        "v_mul_f32_dpp %1, %1, %1 row_shr:4 row_mask:0xf bank_mask:0xf\n"
        "v_mul_f32_dpp %3, %3, %3 row_shr:4 row_mask:0xf bank_mask:0xf\n"
        "v_fmac_f32_dpp %0, %0, %1 row_shr:8 row_mask:0xf bank_mask:0xf\n"
        "v_fmac_f32_dpp %2, %2, %3 row_shr:8 row_mask:0xf bank_mask:0xf\n"
        "v_mul_f32_dpp %1, %1, %1 row_shr:8 row_mask:0xf bank_mask:0xf\n"
        "v_mul_f32_dpp %3, %3, %3 row_shr:8 row_mask:0xf bank_mask:0xf\n"
        "v_fmac_f32_dpp %0, %0, %1 row_bcast:15 row_mask:0xa bank_mask:0xf\n"
        "v_fmac_f32_dpp %2, %2, %3 row_bcast:15 row_mask:0xa bank_mask:0xf\n"
        "v_mul_f32_dpp %1, %1, %1 row_bcast:15 row_mask:0xa bank_mask:0xf\n"
        "v_mul_f32_dpp %3, %3, %3 row_bcast:15 row_mask:0xa bank_mask:0xf\n"
        "v_fmac_f32_dpp %0, %0, %1 row_bcast:31 row_mask:0xc bank_mask:0xf\n"
        "v_fmac_f32_dpp %2, %2, %3 row_bcast:31 row_mask:0xc bank_mask:0xf\n"
        "v_mul_f32_dpp %1, %1, %1 row_bcast:31 row_mask:0xc bank_mask:0xf\n"
        "v_mul_f32_dpp %3, %3, %3 row_bcast:31 row_mask:0xc bank_mask:0xf\n"
        "s_nop 1\n"
        : "+v"(H0), "+v"(P0), "+v"(H1), "+v"(P1));
}

// One pair over segments of S lanes (S = 16 or 32): DPP row shifts stay
// inside a row of 16 lanes, so rows are natural segments; for S = 32 the
// broadcast of lane 15 joins rows 0-1 and 2-3 (row mask 0xa).
template <int S>
__device__ __forceinline__ void seg_scan(float& P, float& Hs) {
    static_assert(S == 16 || S == 32, "segments of 16 or 32 lanes");
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
        "s_nop 1\n"
        : "+v"(Hs), "+v"(P));
    if constexpr (S == 32) {
        asm("v_fmac_f32_dpp %0, %0, %1 row_bcast:15 row_mask:0xa bank_mask:0xf\n"
            "v_mul_f32_dpp %1, %1, %1 row_bcast:15 row_mask:0xa bank_mask:0xf\n"
            "s_nop 1\n"
            : "+v"(Hs), "+v"(P));
    }
}

}  // namespace vmb
