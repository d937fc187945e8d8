/*
 * oracle.c -- plain fp64 reference for the SS2D selective-scan path.
 *
 * TEST INFRASTRUCTURE ONLY. Nothing in the product path may include, link,
 * load or call this file or the library built from it; only the test suite,
 * the smoke check and the benchmark's CPU-baseline leg use it. It shares no
 * code with the HIP kernels.
 *
 * What is computed (VMeanba, arXiv 2412.16602):
 *   - cross-scan / cross-merge of the SS2D module (Appendix A, VMamba
 *     paragraph): unfold an H x W map into K = 4 sequences of length L = H*W
 *     and fold four sequences back into one map;
 *   - the selective-scan recurrence of eq. 3 with the ZOH state matrix of
 *     eq. 4 (first line) and the softplus timescale of eq. 6;
 *   - the VMeanba variant of eq. 9: the transform T averages the discretised
 *     scan inputs over the inner channel axis, the scan runs on one channel,
 *     and T^-1 broadcasts its output back to every channel (Section 2.2).
 *
 * Readings where the paper is silent or garbled (all arithmetic in double on
 * the exact input values):
 *   - B-bar u is the first-order form delta * B * u (eq. 4's second line is
 *     garbled in the paper); C is used undiscretised. Option bit 16 of the
 *     *_opt functions takes eq. 4's second line as zero-order hold instead,
 *     (delta A)^-1 (exp(delta A) - I) delta B, i.e. B-bar u =
 *     phi(delta A) delta B u with phi(x) = (e^x - 1) / x (phi(0) = 1).
 *   - h starts at zero; no final state is returned.
 *   - T averages exp(delta*A) and delta*B*u over the channels of one
 *     direction; C carries no channel axis so T leaves it unchanged; the skip
 *     term D*u is averaged too and broadcast with the scan output.
 *   - Direction order of the cross-scan: 0 row-major, 1 column-major,
 *     2 reverse of 0, 3 reverse of 1. The merge sums the four directions as
 *     (y0 + y2) + (y1 + y3).
 *
 * Sequences are independent, so loops over them run under OpenMP; every sum
 * inside one sequence runs in index order.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

/* softplus(x) = log(1 + e^x), evaluated without overflow (eq. 6, tau_Delta). */
static double sp(double x) { return fmax(x, 0.0) + log1p(exp(-fabs(x))); }

/* Timescale of eq. 6: Delta = softplus(Parameter + s_Delta(u)); the
 * Parameter is the per-channel bias dt_bias, s_Delta(u) is the delta input.
 * With the softplus flag off the sum is used as is. */
static double timescale(double raw, const float* dt_bias, int64_t c, int softplus) {
    double v = raw + (dt_bias ? (double)dt_bias[c] : 0.0);
    return softplus ? sp(v) : v;
}

static void set_threads(int nthreads) {
#ifdef _OPENMP
    if (nthreads > 0) omp_set_num_threads(nthreads);
#else
    (void)nthreads;
#endif
}

int oracle_max_threads(void) {
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/*
 * Full selective scan (eq. 3 with eq. 4 first line and eq. 6), one channel
 * sequence at a time. Tensors (row-major):
 *   u, delta : [batch, K, Dc, L]     A : [K*Dc, N]     Bm, Cm : [batch, K, N, L]
 *   Ds, dt_bias : [K*Dc] (either may be NULL, meaning zero)
 * sel lists flat sequence indices s = (b*K + k)*Dc + d (NULL: all, in order);
 * y receives [nsel, L].
 *
 * For each selected (b, k, d), with c = k*Dc + d and every state n:
 *   h_{-1} = 0
 *   Abar   = exp(Delta_t * A[c, n])
 *   h_t    = Abar * h_{t-1} + Delta_t * B[n, t] * u_t
 *   y_t    = sum_n C[n, t] * h_t + D[c] * u_t
 */
/* The zero-order-hold gain of eq. 4, second line: (e^x - 1) / x at x = delta * A
 * (the limit 1 at x = 0), so that B-bar = gain * delta * B. */
static double zoh_gain(double x) { return x == 0.0 ? 1.0 : expm1(x) / x; }

/*
 * Full scan with option bits: 16 = zero-order-hold B-bar (see the header);
 * otherwise as oracle_full_scan.
 */
void oracle_full_scan_opt(const float* u, const float* delta, const float* A, const float* Bm,
                          const float* Cm, const float* Ds, const float* dt_bias, int softplus,
                          int64_t batch, int64_t K, int64_t Dc, int64_t L, int64_t N,
                          const int64_t* sel, int64_t nsel, int options, double* y,
                          int nthreads) {
    const int zoh = (options & 16) != 0;
    set_threads(nthreads);
    if (!sel) nsel = batch * K * Dc;
#pragma omp parallel
    {
        double* h = (double*)malloc(sizeof(double) * (size_t)(N > 0 ? N : 1));
#pragma omp for schedule(dynamic, 1)
        for (int64_t i = 0; i < nsel; ++i) {
            const int64_t s = sel ? sel[i] : i;
            const int64_t d = s % Dc;
            const int64_t bk = s / Dc;          /* b*K + k */
            const int64_t k = bk % K;
            const int64_t c = k * Dc + d;
            const float* us = u + s * L;
            const float* ds = delta + s * L;
            const float* Bs = Bm + bk * N * L;
            const float* Cs = Cm + bk * N * L;
            const double Dskip = Ds ? (double)Ds[c] : 0.0;
            for (int64_t n = 0; n < N; ++n) h[n] = 0.0;
            for (int64_t t = 0; t < L; ++t) {
                const double dl = timescale((double)ds[t], dt_bias, c, softplus);
                const double ut = (double)us[t];
                double acc = 0.0;
                for (int64_t n = 0; n < N; ++n) {
                    const double x = dl * (double)A[c * N + n];
                    const double abar = exp(x);
                    const double gain = zoh ? zoh_gain(x) : 1.0;
                    const double bu = gain * dl * (double)Bs[n * L + t] * ut;
                    h[n] = abar * h[n] + bu;
                    acc += (double)Cs[n * L + t] * h[n];
                }
                y[i * L + t] = acc + Dskip * ut;
            }
        }
        free(h);
    }
}

/*
 * Full selective scan, eq. 3 for every (b, k, d, n), c = k*Dc + d:
 *   Delta_t = softplus(delta_t + dt_bias[c])           (eq. 6)
 *   h_t[n]  = exp(Delta_t A[c,n]) h_{t-1}[n] + Delta_t B[b,k,n,t] u_t   (eq. 4, first line)
 *   y_t     = sum_n C[b,k,n,t] h_t[n] + D[c] u_t
 * sel lists flat sequence indices (b*K + k)*Dc + d (NULL: all); y is [nsel, L].
 */
void oracle_full_scan(const float* u, const float* delta, const float* A, const float* Bm,
                      const float* Cm, const float* Ds, const float* dt_bias, int softplus,
                      int64_t batch, int64_t K, int64_t Dc, int64_t L, int64_t N,
                      const int64_t* sel, int64_t nsel, double* y, int nthreads) {
    oracle_full_scan_opt(u, delta, A, Bm, Cm, Ds, dt_bias, softplus, batch, K, Dc, L, N, sel,
                         nsel, 0, y, nthreads);
}

/*
 * VMeanba scan (eq. 9 with T = channel mean, T^-1 = broadcast). Same tensors
 * as oracle_full_scan; sel lists flat direction indices s = b*K + k (NULL:
 * all); y receives [nsel, Dc, L], every channel row holding the same values.
 *
 * For each selected (b, k) and position t, over the Dc channels d of that
 * direction (c = k*Dc + d):
 *   Abar_mean[n, t] = (1/Dc) sum_d exp(Delta_{d,t} * A[c, n])      T(Abar)
 *   s_mean[t]       = (1/Dc) sum_d Delta_{d,t} * u_{d,t}           T(Bbar u) / B[n,t]
 *   r_mean[t]       = (1/Dc) sum_d D[c] * u_{d,t}                  T(D u)
 * then the one-channel scan
 *   h_t = Abar_mean[n, t] * h_{t-1} + B[n, t] * s_mean[t]
 *   ytilde_t = sum_n C[n, t] * h_t + r_mean[t]
 * and the broadcast y[d, t] = ytilde_t for every d.
 *
 * options (bit flags) select other readings of where T acts:
 *   1  skip per channel: D u stays outside T, as in eq. 3 for each channel:
 *        ytilde_t = sum_n C[n, t] h_t,  y[d, t] = ytilde_t + D[c] u_{d,t}
 *   2  mean before the discretisation of eq. 4: T averages the timescale,
 *      the input and the state matrix of the channels,
 *        Delta_mean[t] = (1/Dc) sum_d Delta_{d,t},  u_mean[t] = (1/Dc) sum_d u_{d,t},
 *        A_mean[n] = (1/Dc) sum_d A[c, n],
 *      and the one-channel scan discretises those:
 *        h_t = exp(Delta_mean[t] A_mean[n]) h_{t-1} + Delta_mean[t] B[n, t] u_mean[t]
 *      (the skip term as above, r_mean or per channel)
 *   4  no broadcast: T^-1 is left out and y receives [nsel, L], the reduced
 *      output ytilde of each (b, k) (not with option 1)
 *   16 zero-order-hold B-bar (see the header): T averages
 *        phi(Delta_{d,t} A[c,n]) Delta_{d,t} u_{d,t} per state n,
 *      h_t = Abar_mean[n,t] h_{t-1} + B[n,t] (1/Dc) sum_d phi(..) Delta u;
 *      with option 2 the means are discretised with it:
 *      phi(Delta_mean A_mean[n]) Delta_mean B[n,t] u_mean
 */
void oracle_mean_scan_opt(const float* u, const float* delta, const float* A, const float* Bm,
                          const float* Cm, const float* Ds, const float* dt_bias, int softplus,
                          int64_t batch, int64_t K, int64_t Dc, int64_t L, int64_t N,
                          const int64_t* sel, int64_t nsel, int options, double* y,
                          int nthreads) {
    const int skip_per_channel = (options & 1) != 0;
    const int raw_mean = (options & 2) != 0;
    const int broadcast = (options & 4) == 0;
    const int zoh = (options & 16) != 0;
    set_threads(nthreads);
    if (!sel) nsel = batch * K;
#pragma omp parallel
    {
        double* h = (double*)malloc(sizeof(double) * (size_t)(N > 0 ? N : 1));
        double* abar = (double*)malloc(sizeof(double) * (size_t)(N > 0 ? N : 1));
        double* amean = (double*)malloc(sizeof(double) * (size_t)(N > 0 ? N : 1));
        double* zsum = (double*)malloc(sizeof(double) * (size_t)(N > 0 ? N : 1));
#pragma omp for schedule(dynamic, 1)
        for (int64_t i = 0; i < nsel; ++i) {
            const int64_t bk = sel ? sel[i] : i;
            const int64_t k = bk % K;
            const float* Bs = Bm + bk * N * L;
            const float* Cs = Cm + bk * N * L;
            const double inv = 1.0 / (double)Dc;
            /* mean state matrix of the direction's channels (option 2) */
            for (int64_t n = 0; n < N; ++n) {
                double sum = 0.0;
                for (int64_t d = 0; d < Dc; ++d) sum += (double)A[(k * Dc + d) * N + n];
                amean[n] = sum * inv;
            }
            for (int64_t n = 0; n < N; ++n) h[n] = 0.0;
            for (int64_t t = 0; t < L; ++t) {
                /* T: mean over the inner channel axis */
                for (int64_t n = 0; n < N; ++n) abar[n] = zsum[n] = 0.0;
                double s_sum = 0.0, r_sum = 0.0, dl_sum = 0.0, u_sum = 0.0;
                for (int64_t d = 0; d < Dc; ++d) {
                    const int64_t c = k * Dc + d;
                    const int64_t off = (bk * Dc + d) * L + t;
                    const double dl = timescale((double)delta[off], dt_bias, c, softplus);
                    const double ut = (double)u[off];
                    for (int64_t n = 0; n < N; ++n) {
                        const double x = dl * (double)A[c * N + n];
                        abar[n] += exp(x);
                        zsum[n] += zoh_gain(x) * dl * ut;
                    }
                    s_sum += dl * ut;
                    r_sum += (Ds ? (double)Ds[c] : 0.0) * ut;
                    dl_sum += dl;
                    u_sum += ut;
                }
                const double r_mean = skip_per_channel ? 0.0 : r_sum * inv;
                /* Mamba on the reduced (one-channel) inputs */
                double acc = 0.0;
                for (int64_t n = 0; n < N; ++n) {
                    double a_n, bu_n;
                    if (raw_mean) {
                        /* eq. 4 applied to the means */
                        const double dm = dl_sum * inv, um = u_sum * inv;
                        a_n = exp(dm * amean[n]);
                        bu_n = (zoh ? zoh_gain(dm * amean[n]) : 1.0) * dm * (double)Bs[n * L + t] * um;
                    } else {
                        /* the means of the discretised terms */
                        a_n = abar[n] * inv;
                        bu_n = (double)Bs[n * L + t] * ((zoh ? zsum[n] : s_sum) * inv);
                    }
                    h[n] = a_n * h[n] + bu_n;
                    acc += (double)Cs[n * L + t] * h[n];
                }
                const double yt = acc + r_mean;
                if (!broadcast) {
                    y[i * L + t] = yt;
                    continue;
                }
                /* T^-1: broadcast to every channel */
                for (int64_t d = 0; d < Dc; ++d) {
                    const int64_t c = k * Dc + d;
                    const double own = skip_per_channel && Ds
                                           ? (double)Ds[c] * (double)u[(bk * Dc + d) * L + t]
                                           : 0.0;
                    y[(i * Dc + d) * L + t] = yt + own;
                }
            }
        }
        free(amean);
        free(zsum);
        free(abar);
        free(h);
    }
}

/* VMeanba with T taken over every channel of an image: the K directions'
 * channels pooled, K*Dc of them (Section 2.2, eq. 9, with the inner channel
 * axis read as all K*Dc sequences of the image). Channel c = k*Dc + d carries
 * its direction's B and C, so the channel means of the discretised terms are
 *   abar[n,t] = mean_c exp(Delta_c,t A[c,n])
 *   bu[n,t]   = mean_c Delta_c,t u_c,t B[b,k(c),n,t]
 *   cbar[n,t] = mean_c C[b,k(c),n,t]
 *   r[t]      = mean_c D[c] u_c,t
 * and Mamba (eq. 3) runs once per batch element on them:
 *   h[n] = abar h[n] + bu,   y[b,t] = sum_n cbar h[n] + r.
 * Output y: [batch][L] (T^-1 broadcasts it to every (k, d)). */
void oracle_mean_scan_pooled(const float* u, const float* delta, const float* A,
                             const float* Bm, const float* Cm, const float* Ds,
                             const float* dt_bias, int softplus, int64_t batch, int64_t K,
                             int64_t Dc, int64_t L, int64_t N, double* y, int nthreads) {
    set_threads(nthreads);
#pragma omp parallel
    {
        double* h = (double*)malloc(sizeof(double) * (size_t)(N > 0 ? N : 1));
        double* abar = (double*)malloc(sizeof(double) * (size_t)(N > 0 ? N : 1));
        double* bu = (double*)malloc(sizeof(double) * (size_t)(N > 0 ? N : 1));
        double* cbar = (double*)malloc(sizeof(double) * (size_t)(N > 0 ? N : 1));
#pragma omp for schedule(dynamic, 1)
        for (int64_t b = 0; b < batch; ++b) {
            const double inv = 1.0 / (double)(K * Dc);
            for (int64_t n = 0; n < N; ++n) h[n] = 0.0;
            for (int64_t t = 0; t < L; ++t) {
                for (int64_t n = 0; n < N; ++n) abar[n] = bu[n] = cbar[n] = 0.0;
                double r_sum = 0.0;
                for (int64_t k = 0; k < K; ++k) {
                    const int64_t bk = b * K + k;
                    for (int64_t d = 0; d < Dc; ++d) {
                        const int64_t c = k * Dc + d;
                        const int64_t off = (bk * Dc + d) * L + t;
                        const double dl = timescale((double)delta[off], dt_bias, c, softplus);
                        const double ut = (double)u[off];
                        for (int64_t n = 0; n < N; ++n) {
                            abar[n] += exp(dl * (double)A[c * N + n]);
                            bu[n] += dl * ut * (double)Bm[(bk * N + n) * L + t];
                            cbar[n] += (double)Cm[(bk * N + n) * L + t];
                        }
                        r_sum += (Ds ? (double)Ds[c] : 0.0) * ut;
                    }
                }
                double acc = 0.0;
                for (int64_t n = 0; n < N; ++n) {
                    h[n] = abar[n] * inv * h[n] + bu[n] * inv;
                    acc += cbar[n] * inv * h[n];
                }
                y[b * L + t] = acc + r_sum * inv;
            }
        }
        free(h);
        free(abar);
        free(bu);
        free(cbar);
    }
}

void oracle_mean_scan(const float* u, const float* delta, const float* A, const float* Bm,
                      const float* Cm, const float* Ds, const float* dt_bias, int softplus,
                      int64_t batch, int64_t K, int64_t Dc, int64_t L, int64_t N,
                      const int64_t* sel, int64_t nsel, double* y, int nthreads) {
    oracle_mean_scan_opt(u, delta, A, Bm, Cm, Ds, dt_bias, softplus, batch, K, Dc, L, N, sel, nsel,
                         0, y, nthreads);
}

/*
 * Scan on materialised, discretised inputs with one state (the decomposition
 * of the paper's kernel experiments, Appendix D and Table 1: discretisation
 * runs outside the kernel, which only walks the recurrence of eq. 3; the
 * computational-complexity appendix counts the scan per (d, t) with N = 1).
 * Tensors (row-major):
 *   abar, bu : [batch, Dc, L]     C : [batch, L]     skip : [batch, Dc, L] or NULL
 * For each (b, d):
 *   h_{-1} = 0
 *   h_t    = abar[b, d, t] * h_{t-1} + bu[b, d, t]
 *   y_t    = C[b, t] * h_t + skip[b, d, t]
 * y receives [batch, Dc, L].
 */
void oracle_discrete_scan(const float* abar, const float* bu, const float* C, const float* skip,
                          int64_t batch, int64_t Dc, int64_t L, double* y, int nthreads) {
    set_threads(nthreads);
#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t s = 0; s < batch * Dc; ++s) {
        const int64_t b = s / Dc;
        const float* as = abar + s * L;
        const float* bs = bu + s * L;
        const float* ks = skip ? skip + s * L : NULL;
        const float* cs = C + b * L;
        double h = 0.0;
        for (int64_t t = 0; t < L; ++t) {
            h = (double)as[t] * h + (double)bs[t];
            y[s * L + t] = (double)cs[t] * h + (ks ? (double)ks[t] : 0.0);
        }
    }
}

/*
 * The transform T of eq. 9 on a materialised input: the mean over the inner
 * channel axis (Section 2.2), summed in index order.
 *   x : [batch, Dc, L]  ->  xm : [batch, L],  xm[b, t] = (1/Dc) sum_d x[b, d, t]
 */
void oracle_channel_mean(const float* x, int64_t batch, int64_t Dc, int64_t L, double* xm,
                         int nthreads) {
    set_threads(nthreads);
#pragma omp parallel for schedule(static)
    for (int64_t b = 0; b < batch; ++b) {
        for (int64_t t = 0; t < L; ++t) {
            double acc = 0.0;
            for (int64_t d = 0; d < Dc; ++d) acc += (double)x[(b * Dc + d) * L + t];
            xm[b * L + t] = acc / (double)Dc;
        }
    }
}

/*
 * Cross-scan position maps for an H x W map, pixel p = h*W + w:
 *   pi_0(h, w) = h*W + w          (row-major)
 *   pi_1(h, w) = w*H + h          (column-major)
 *   pi_2(h, w) = L - 1 - pi_0     (row-major, reversed)
 *   pi_3(h, w) = L - 1 - pi_1     (column-major, reversed)
 */
static int64_t pos(int k, int64_t h, int64_t w, int64_t H, int64_t W) {
    const int64_t L = H * W;
    switch (k) {
        case 0: return h * W + w;
        case 1: return w * H + h;
        case 2: return L - 1 - (h * W + w);
        default: return L - 1 - (w * H + h);
    }
}

/* Cross-scan: xs[b, k, d, pi_k(h, w)] = x[b, d, h, w]. Element size esz
 * bytes (a pure copy, so any element type). */
void oracle_cross_scan(const void* x, void* xs, int64_t batch, int64_t Dc, int64_t H,
                       int64_t W, int64_t esz) {
    const int64_t L = H * W;
    const char* src = (const char*)x;
    char* dst = (char*)xs;
    for (int64_t b = 0; b < batch; ++b)
        for (int64_t k = 0; k < 4; ++k)
            for (int64_t d = 0; d < Dc; ++d)
                for (int64_t h = 0; h < H; ++h)
                    for (int64_t w = 0; w < W; ++w) {
                        const int64_t from = ((b * Dc + d) * L + h * W + w) * esz;
                        const int64_t to = (((b * 4 + k) * Dc + d) * L + pos((int)k, h, w, H, W)) * esz;
                        memcpy(dst + to, src + from, (size_t)esz);
                    }
}

/* Cross-merge in double: y[b, d, h, w] = (ys_0 + ys_2) + (ys_1 + ys_3), each
 * ys_k read at pi_k(h, w). */
void oracle_cross_merge_f64(const double* ys, double* y, int64_t batch, int64_t Dc,
                            int64_t H, int64_t W) {
    const int64_t L = H * W;
    for (int64_t b = 0; b < batch; ++b)
        for (int64_t d = 0; d < Dc; ++d)
            for (int64_t h = 0; h < H; ++h)
                for (int64_t w = 0; w < W; ++w) {
                    double v[4];
                    for (int k = 0; k < 4; ++k)
                        v[k] = ys[((b * 4 + k) * Dc + d) * L + pos(k, h, w, H, W)];
                    y[(b * Dc + d) * L + h * W + w] = (v[0] + v[2]) + (v[1] + v[3]);
                }
}

/* The same merge evaluated in binary32 with the same association: each add
 * is one IEEE single-precision rounding (built with -ffp-contract=off on an
 * SSE target, so no wider intermediates). */
void oracle_cross_merge_f32(const float* ys, float* y, int64_t batch, int64_t Dc,
                            int64_t H, int64_t W) {
    const int64_t L = H * W;
    for (int64_t b = 0; b < batch; ++b)
        for (int64_t d = 0; d < Dc; ++d)
            for (int64_t h = 0; h < H; ++h)
                for (int64_t w = 0; w < W; ++w) {
                    float v[4];
                    for (int k = 0; k < 4; ++k)
                        v[k] = ys[((b * 4 + k) * Dc + d) * L + pos(k, h, w, H, W)];
                    volatile float s02 = v[0] + v[2];
                    volatile float s13 = v[1] + v[3];
                    y[(b * Dc + d) * L + h * W + w] = s02 + s13;
                }
}

/* bfloat16 <-> binary32. A bfloat16 value is the top half of a binary32
 * pattern, so widening is exact; narrowing rounds to nearest, ties to even,
 * on the discarded 16 bits (NaNs stay NaN). */
static float bf16_to_f32(uint16_t v) {
    uint32_t bits = (uint32_t)v << 16;
    float f;
    memcpy(&f, &bits, 4);
    return f;
}
static uint16_t f32_to_bf16(float f) {
    uint32_t bits;
    memcpy(&bits, &f, 4);
    if ((bits & 0x7F800000u) == 0x7F800000u && (bits & 0x007FFFFFu))
        return (uint16_t)((bits >> 16) | 0x40u);
    const uint32_t half = 0x8000u;
    const uint32_t low = bits & 0xFFFFu;
    uint32_t hi = bits >> 16;
    if (low > half || (low == half && (hi & 1u))) hi += 1u;
    return (uint16_t)hi;
}

/* Merge of bfloat16 sequences: each value widened exactly, summed in
 * binary32 with the same association, one rounding to bfloat16 at the end. */
void oracle_cross_merge_bf16(const uint16_t* ys, uint16_t* y, int64_t batch, int64_t Dc,
                             int64_t H, int64_t W) {
    const int64_t L = H * W;
    for (int64_t b = 0; b < batch; ++b)
        for (int64_t d = 0; d < Dc; ++d)
            for (int64_t h = 0; h < H; ++h)
                for (int64_t w = 0; w < W; ++w) {
                    float v[4];
                    for (int k = 0; k < 4; ++k)
                        v[k] = bf16_to_f32(ys[((b * 4 + k) * Dc + d) * L + pos(k, h, w, H, W)]);
                    volatile float s02 = v[0] + v[2];
                    volatile float s13 = v[1] + v[3];
                    volatile float s = s02 + s13;
                    y[(b * Dc + d) * L + h * W + w] = f32_to_bf16(s);
                }
}

/* binary32 -> bfloat16 (nearest-even) for n values; exposed so tests can
 * round oracle outputs the way a bf16 store does. */
void oracle_f32_to_bf16(const float* in, uint16_t* out, int64_t n) {
    for (int64_t i = 0; i < n; ++i) out[i] = f32_to_bf16(in[i]);
}
