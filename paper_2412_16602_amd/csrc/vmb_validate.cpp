// vmb_validate.cpp -- host-side argument checks of the libvmb entry points.
// Pure C++: no HIP calls, so every error path can be exercised without a GPU.
#include <stdint.h>

#include <limits>

#include "vmb_internal.h"

namespace vmb {
namespace {

constexpr int64_t kMaxRow = (int64_t{1} << 31) - 1;   // elements per [.., L] row
constexpr int64_t kMaxTotal = int64_t{1} << 40;       // elements per tensor

bool aligned(const void* p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

size_t dsize(vmb_dtype t) { return t == VMB_BF16 ? 2 : 4; }

bool valid_dtype(vmb_dtype t) { return t == VMB_F32 || t == VMB_BF16; }

// overflow-checked product of positive sizes; returns -1 past kMaxTotal
int64_t prod(std::initializer_list<int64_t> v) {
    int64_t r = 1;
    for (int64_t x : v) {
        if (x <= 0) return -1;
        if (r > kMaxTotal / x) return -1;
        r *= x;
    }
    return r;
}

struct Range {
    uintptr_t lo, hi;  // [lo, hi)
};

Range range_of(const void* p, int64_t elems, size_t esz) {
    const uintptr_t lo = reinterpret_cast<uintptr_t>(p);
    return Range{lo, lo + static_cast<uintptr_t>(elems) * esz};
}

bool overlap(Range a, Range b) { return a.lo < b.hi && b.lo < a.hi; }

bool supported_n(int64_t N) { return N == 1 || N == 2 || N == 4 || N == 8 || N == 16; }

}  // namespace

vmb_status validate_cross(const void* in, const void* out, int64_t batch, int64_t channels,
                          int64_t H, int64_t W, vmb_dtype dt, bool unfold) {
    if (!in || !out) return VMB_ERR_NULL;
    if (!valid_dtype(dt)) return VMB_ERR_DTYPE;
    if (batch < 1 || channels < 1 || H < 1 || W < 1) return VMB_ERR_SHAPE;
    const int64_t L = prod({H, W});
    if (L < 0 || L > kMaxRow) return VMB_ERR_SHAPE;
    const int64_t n_map = prod({batch, channels, L});
    const int64_t n_seq = prod({batch, 4, channels, L});
    if (n_map < 0 || n_seq < 0) return VMB_ERR_SHAPE;
    if (!aligned(in, 16) || !aligned(out, 16)) return VMB_ERR_ALIGN;
    const size_t e = dsize(dt);
    const Range rin = range_of(in, unfold ? n_map : n_seq, e);
    const Range rout = range_of(out, unfold ? n_seq : n_map, e);
    if (overlap(rin, rout)) return VMB_ERR_ALIAS;
    return VMB_OK;
}

vmb_status validate_discrete(const float* abar, const float* bu, const float* C, const float* skip,
                             const float* y, int64_t batch, int64_t channels, int64_t L) {
    if (!abar || !bu || !C || !y) return VMB_ERR_NULL;
    if (batch < 1 || channels < 1 || L < 1 || L > kMaxRow) return VMB_ERR_SHAPE;
    const int64_t n = prod({batch, channels, L});
    const int64_t nc = prod({batch, L});
    if (n < 0 || nc < 0) return VMB_ERR_SHAPE;
    if (!aligned(abar, 16) || !aligned(bu, 16) || !aligned(C, 16) || !aligned(y, 16) ||
        (skip && !aligned(skip, 16)))
        return VMB_ERR_ALIGN;
    const Range ry = range_of(y, n, 4);
    if (overlap(ry, range_of(abar, n, 4)) || overlap(ry, range_of(bu, n, 4)) ||
        overlap(ry, range_of(C, nc, 4)) || (skip && overlap(ry, range_of(skip, n, 4))))
        return VMB_ERR_ALIAS;
    return VMB_OK;
}

vmb_status validate_channel_mean(const float* x, const float* xm, int64_t batch, int64_t channels,
                                 int64_t L) {
    if (!x || !xm) return VMB_ERR_NULL;
    if (batch < 1 || channels < 1 || L < 1 || L > kMaxRow) return VMB_ERR_SHAPE;
    const int64_t n = prod({batch, channels, L});
    const int64_t nm = prod({batch, L});
    if (n < 0 || nm < 0) return VMB_ERR_SHAPE;
    if (!aligned(x, 16) || !aligned(xm, 16)) return VMB_ERR_ALIGN;
    if (overlap(range_of(xm, nm, 4), range_of(x, n, 4))) return VMB_ERR_ALIAS;
    return VMB_OK;
}

vmb_status validate_projections(const void* u, const float* W, const float* W_dt,
                                const void* delta, const void* B, const void* C, int64_t batch,
                                int64_t K, int64_t channels, int64_t L, int64_t N, int64_t R,
                                vmb_dtype dt) {
    if (!u || !W || !delta || !B || !C) return VMB_ERR_NULL;
    if (!valid_dtype(dt)) return VMB_ERR_DTYPE;
    if (batch < 1 || K < 1 || channels < 1 || L < 1 || N < 1 || R < 1 || L > kMaxRow)
        return VMB_ERR_SHAPE;
    const int64_t seq = prod({batch, K, channels, L});
    const int64_t bc = prod({batch, K, N, L});
    const int64_t wn = prod({K, R + 2 * N, channels});
    const int64_t wd = prod({K, channels, R});
    if (seq < 0 || bc < 0 || wn < 0 || wd < 0 || prod({channels, L}) > kMaxRow) return VMB_ERR_SHAPE;
    if (!supported_n(N) || R > 64 || (!W_dt && R != 1)) return VMB_ERR_UNSUPPORTED;
    if (!aligned(u, 16) || !aligned(delta, 16) || !aligned(B, 16) || !aligned(C, 16) ||
        !aligned(W, 4) || (W_dt && !aligned(W_dt, 4)))
        return VMB_ERR_ALIGN;
    const size_t e = dsize(dt);
    const Range outs[] = {range_of(delta, seq, e), range_of(B, bc, e), range_of(C, bc, e)};
    const Range ins[] = {range_of(u, seq, e), range_of(W, wn, 4),
                         W_dt ? range_of(W_dt, wd, 4) : Range{0, 0}};
    for (const Range& o : outs)
        for (const Range& i : ins)
            if (overlap(o, i)) return VMB_ERR_ALIAS;
    if (overlap(outs[0], outs[1]) || overlap(outs[0], outs[2]) || overlap(outs[1], outs[2]))
        return VMB_ERR_ALIAS;
    return VMB_OK;
}

vmb_status validate_out_norm(const void* y, const void* z, const float* gamma, const float* beta,
                             float eps, const void* out, int64_t batch, int64_t channels,
                             int64_t P, vmb_dtype dt) {
    if (!y || !out) return VMB_ERR_NULL;
    if (!valid_dtype(dt)) return VMB_ERR_DTYPE;
    if (batch < 1 || channels < 1 || P < 1 || !(eps >= 0.0f) || eps > 3.0e38f)
        return VMB_ERR_SHAPE;
    const int64_t n = prod({batch, channels, P});
    if (n < 0 || prod({channels, P}) > kMaxRow) return VMB_ERR_SHAPE;
    const size_t e = dsize(dt);
    if (!aligned(y, e) || !aligned(out, e) || (z && !aligned(z, e)) ||
        (gamma && !aligned(gamma, 4)) || (beta && !aligned(beta, 4)))
        return VMB_ERR_ALIGN;
    const Range o = range_of(out, n, e);
    if (overlap(o, range_of(y, n, e)) || (z && overlap(o, range_of(z, n, e))) ||
        (gamma && overlap(o, range_of(gamma, channels, 4))) ||
        (beta && overlap(o, range_of(beta, channels, 4))))
        return VMB_ERR_ALIAS;
    return VMB_OK;
}

size_t scan_workspace_bytes(int mean_variant, int64_t batch, int64_t K, int64_t channels,
                            int64_t L, int64_t N, vmb_layout layout) {
    if (batch < 1 || K < 1 || channels < 1 || L < 1 || N < 1) return SIZE_MAX;
    const int64_t seq = prod({batch, K, channels, L});
    if (seq < 0) return SIZE_MAX;
    auto round_up = [](size_t v) { return (v + 255) & ~size_t{255}; };
    if (!mean_variant) {
        // 2-D layout: per-direction fp32 outputs, folded by the merge pass,
        // then (tile path) column-major copies of the input planes
        if (layout != VMB_LAYOUT_2D) return 0;
        size_t bytes = round_up(static_cast<size_t>(seq) * 4);
        if (full_ws_has_xt(batch, K, channels, L, N)) bytes += full_ws_xt_bytes(batch, channels, L);
        return bytes;
    }
    // room for the main reading and for the pooled one (VMB_MEAN_POOLED)
    const size_t main = mean_ws_layout(batch, K, channels, L, N, layout == VMB_LAYOUT_2D).total;
    const size_t pooled = pooled_ws_layout(batch, K, channels, L, N, layout == VMB_LAYOUT_2D).total;
    return main > pooled ? main : pooled;
}

vmb_status validate_scan(const ScanArgs& a, int mean_variant) {
    if (!a.u || !a.delta || !a.A || !a.B || !a.C || !a.y) return VMB_ERR_NULL;
    if (!valid_dtype(a.in_dt) || !valid_dtype(a.out_dt)) return VMB_ERR_DTYPE;
    if (a.in_dt == VMB_F32 && a.out_dt == VMB_BF16) return VMB_ERR_DTYPE;
    if (a.layout != VMB_LAYOUT_SEQ && a.layout != VMB_LAYOUT_2D) return VMB_ERR_SHAPE;
    if (a.batch < 1 || a.K < 1 || a.channels < 1 || a.L < 1 || a.N < 1) return VMB_ERR_SHAPE;
    if (a.L > kMaxRow) return VMB_ERR_SHAPE;
    const int64_t seq = prod({a.batch, a.K, a.channels, a.L});
    const int64_t bc = prod({a.batch, a.K, a.N, a.L});
    const int64_t kc = prod({a.K, a.channels});
    if (seq < 0 || bc < 0 || kc < 0 || kc > kMaxRow) return VMB_ERR_SHAPE;
    // B and C are indexed n*L + t inside one (batch, direction) block
    if (prod({a.N, a.L}) > kMaxRow) return VMB_ERR_SHAPE;
    if (a.layout == VMB_LAYOUT_2D) {
        if (a.K != 4 || a.H < 1 || a.W < 1 || prod({a.H, a.W}) != a.L) return VMB_ERR_SHAPE;
    }
    if (!supported_n(a.N)) return VMB_ERR_UNSUPPORTED;
    // the 2-D calls end with a merge pass: maps it cannot take fail here,
    // before anything is launched
    if (a.layout == VMB_LAYOUT_2D && !cross_fits(a.batch, a.channels, a.H, a.W))
        return VMB_ERR_UNSUPPORTED;
    const unsigned known = VMB_MEAN_SKIP_PER_CHANNEL | VMB_MEAN_RAW | VMB_MEAN_NO_BROADCAST |
                           VMB_MEAN_POOLED | VMB_SCAN_ZOH | VMB_MEAN_TEST_GIVE_UP;
    if (a.options & ~known) return VMB_ERR_UNSUPPORTED;
    if (!mean_variant && (a.options & ~static_cast<unsigned>(VMB_SCAN_ZOH))) return VMB_ERR_UNSUPPORTED;
    if ((a.options & VMB_MEAN_POOLED) && a.options != VMB_MEAN_POOLED) return VMB_ERR_UNSUPPORTED;
    if ((a.options & VMB_SCAN_ZOH) && (a.options & VMB_MEAN_RAW)) return VMB_ERR_UNSUPPORTED;
    const bool no_bcast = (a.options & VMB_MEAN_NO_BROADCAST) != 0;
    if (no_bcast && (a.layout != VMB_LAYOUT_SEQ || (a.options & VMB_MEAN_SKIP_PER_CHANNEL)))
        return VMB_ERR_UNSUPPORTED;
    // the chunk-local index math of the mean variant's passes is 32-bit
    if (mean_variant && prod({a.batch, a.K, a.N + 2, a.L}) > kMaxRow) return VMB_ERR_UNSUPPORTED;
    const void* streamed[] = {a.u, a.delta, a.B, a.C, a.y};
    for (const void* p : streamed)
        if (!aligned(p, 16)) return VMB_ERR_ALIGN;
    if (!aligned(a.A, 4) || (a.D && !aligned(a.D, 4)) || (a.dt_bias && !aligned(a.dt_bias, 4)))
        return VMB_ERR_ALIGN;
    const size_t need = scan_workspace_bytes(mean_variant, a.batch, a.K, a.channels, a.L, a.N,
                                             a.layout);
    if (need == SIZE_MAX) return VMB_ERR_SHAPE;
    if (need > 0) {
        if (!a.ws || a.ws_bytes < need) return VMB_ERR_WORKSPACE;
        if (!aligned(a.ws, 16)) return VMB_ERR_ALIGN;
    }
    // aliasing: the output must not overlap any input (or the workspace)
    const size_t ein = dsize(a.in_dt), eout = dsize(a.out_dt);
    const int64_t u_elems = a.layout == VMB_LAYOUT_2D ? seq / a.K : seq;
    const int64_t y_elems = a.layout == VMB_LAYOUT_2D ? seq / a.K : (no_bcast ? seq / a.channels : seq);
    const Range ry = range_of(a.y, y_elems, eout);
    const Range inputs[] = {range_of(a.u, u_elems, ein),
                            range_of(a.delta, seq, ein),
                            range_of(a.B, bc, ein),
                            range_of(a.C, bc, ein),
                            range_of(a.A, kc * a.N, 4),
                            a.D ? range_of(a.D, kc, 4) : Range{0, 0},
                            a.dt_bias ? range_of(a.dt_bias, kc, 4) : Range{0, 0}};
    for (const Range& r : inputs)
        if (r.hi > r.lo && overlap(ry, r)) return VMB_ERR_ALIAS;
    if (need > 0) {
        const Range rw = range_of(a.ws, static_cast<int64_t>(need), 1);
        if (overlap(ry, rw)) return VMB_ERR_ALIAS;
        for (const Range& r : inputs)
            if (r.hi > r.lo && overlap(rw, r)) return VMB_ERR_ALIAS;
    }
    return VMB_OK;
}

}  // namespace vmb
