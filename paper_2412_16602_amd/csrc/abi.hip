// abi.hip -- extern "C" entry points of libvmb: validate on the host, then
// enqueue the kernels on the caller's stream. Nothing here allocates, prints
// or throws; only vmb_mean_scan_status synchronises (it reads a result back).
#include "vmb_internal.h"

using namespace vmb;

namespace {

ScanArgs pack(const void* u, const void* delta, const float* A, const void* B, const void* C,
              const float* D, const float* dt_bias, int delta_softplus, void* y, int64_t batch,
              int64_t K, int64_t channels, int64_t L, int64_t N, vmb_dtype in_dtype,
              vmb_dtype out_dtype, vmb_layout layout, int64_t H, int64_t W, void* workspace,
              size_t workspace_bytes, vmb_stream_t stream) {
    ScanArgs a;
    a.u = u;
    a.delta = delta;
    a.A = A;
    a.B = B;
    a.C = C;
    a.D = D;
    a.dt_bias = dt_bias;
    a.softplus = delta_softplus ? 1 : 0;
    a.y = y;
    a.batch = batch;
    a.K = K;
    a.channels = channels;
    a.L = L;
    a.N = N;
    a.in_dt = in_dtype;
    a.out_dt = out_dtype;
    a.layout = layout;
    a.H = layout == VMB_LAYOUT_2D ? H : 1;
    a.W = layout == VMB_LAYOUT_2D ? W : L;
    a.ws = workspace;
    a.ws_bytes = workspace_bytes;
    a.options = 0;
    a.stream = static_cast<hipStream_t>(stream);
    return a;
}

}  // namespace

extern "C" {

vmb_status vmb_cross_scan(const void* x, void* xs, int64_t batch, int64_t channels, int64_t H,
                          int64_t W, vmb_dtype dt, vmb_stream_t stream) {
    const vmb_status st = validate_cross(x, xs, batch, channels, H, W, dt, true);
    if (st != VMB_OK) return st;
    return launch_cross_scan(x, xs, batch, channels, H, W, dt, static_cast<hipStream_t>(stream));
}

vmb_status vmb_cross_merge(const void* ys, void* y, int64_t batch, int64_t channels, int64_t H,
                           int64_t W, vmb_dtype dt, vmb_stream_t stream) {
    const vmb_status st = validate_cross(ys, y, batch, channels, H, W, dt, false);
    if (st != VMB_OK) return st;
    return launch_cross_merge(ys, y, batch, channels, H, W, dt, dt,
                              static_cast<hipStream_t>(stream));
}

vmb_status vmb_selective_scan_fwd(const void* u, const void* delta, const float* A,
                                  const void* B, const void* C, const float* D,
                                  const float* dt_bias, int delta_softplus, void* y,
                                  int64_t batch, int64_t K, int64_t channels, int64_t L,
                                  int64_t N, vmb_dtype in_dtype, vmb_dtype out_dtype,
                                  vmb_layout layout, int64_t H, int64_t W, void* workspace,
                                  size_t workspace_bytes, vmb_stream_t stream) {
    const ScanArgs a = pack(u, delta, A, B, C, D, dt_bias, delta_softplus, y, batch, K, channels,
                            L, N, in_dtype, out_dtype, layout, H, W, workspace, workspace_bytes,
                            stream);
    const vmb_status st = validate_scan(a, 0);
    if (st != VMB_OK) return st;
    return launch_full_scan(a);
}

vmb_status vmb_selective_scan_fwd_ex(const void* u, const void* delta, const float* A,
                                     const void* B, const void* C, const float* D,
                                     const float* dt_bias, int delta_softplus, void* y,
                                     int64_t batch, int64_t K, int64_t channels, int64_t L,
                                     int64_t N, vmb_dtype in_dtype, vmb_dtype out_dtype,
                                     vmb_layout layout, int64_t H, int64_t W, void* workspace,
                                     size_t workspace_bytes, unsigned options,
                                     vmb_stream_t stream) {
    ScanArgs a = pack(u, delta, A, B, C, D, dt_bias, delta_softplus, y, batch, K, channels, L, N,
                      in_dtype, out_dtype, layout, H, W, workspace, workspace_bytes, stream);
    a.options = options;
    const vmb_status st = validate_scan(a, 0);
    if (st != VMB_OK) return st;
    return launch_full_scan(a);
}

vmb_status vmb_mean_scan_fwd(const void* u, const void* delta, const float* A, const void* B,
                             const void* C, const float* D, const float* dt_bias,
                             int delta_softplus, void* y, int64_t batch, int64_t K,
                             int64_t channels, int64_t L, int64_t N, vmb_dtype in_dtype,
                             vmb_dtype out_dtype, vmb_layout layout, int64_t H, int64_t W,
                             void* workspace, size_t workspace_bytes, vmb_stream_t stream) {
    const ScanArgs a = pack(u, delta, A, B, C, D, dt_bias, delta_softplus, y, batch, K, channels,
                            L, N, in_dtype, out_dtype, layout, H, W, workspace, workspace_bytes,
                            stream);
    const vmb_status st = validate_scan(a, 1);
    if (st != VMB_OK) return st;
    return launch_mean_scan(a);
}

vmb_status vmb_mean_scan_fwd_ex(const void* u, const void* delta, const float* A, const void* B,
                                const void* C, const float* D, const float* dt_bias,
                                int delta_softplus, void* y, int64_t batch, int64_t K,
                                int64_t channels, int64_t L, int64_t N, vmb_dtype in_dtype,
                                vmb_dtype out_dtype, vmb_layout layout, int64_t H, int64_t W,
                                void* workspace, size_t workspace_bytes, unsigned options,
                                vmb_stream_t stream) {
    ScanArgs a = pack(u, delta, A, B, C, D, dt_bias, delta_softplus, y, batch, K, channels, L, N,
                      in_dtype, out_dtype, layout, H, W, workspace, workspace_bytes, stream);
    a.options = options;
    const vmb_status st = validate_scan(a, 1);
    if (st != VMB_OK) return st;
    return launch_mean_scan(a);
}

vmb_status vmb_ss2d_projections(const void* u, const float* W, const float* W_dt, void* delta,
                                void* B, void* C, int64_t batch, int64_t K, int64_t channels,
                                int64_t L, int64_t N, int64_t R, vmb_dtype dtype,
                                vmb_stream_t stream) {
    const vmb_status st = validate_projections(u, W, W_dt, delta, B, C, batch, K, channels, L, N,
                                               R, dtype);
    if (st != VMB_OK) return st;
    return launch_projections(u, W, W_dt, delta, B, C, batch, K, channels, L, N, R, dtype,
                              static_cast<hipStream_t>(stream));
}

vmb_status vmb_ss2d_out_norm(const void* y, const void* z, const float* gamma, const float* beta,
                             float eps, void* out, int64_t batch, int64_t channels, int64_t P,
                             vmb_dtype dtype, vmb_stream_t stream) {
    const vmb_status st =
        validate_out_norm(y, z, gamma, beta, eps, out, batch, channels, P, dtype);
    if (st != VMB_OK) return st;
    return launch_out_norm(y, z, gamma, beta, eps, out, batch, channels, P, dtype,
                           static_cast<hipStream_t>(stream));
}

size_t vmb_scan_workspace_bytes(int mean_variant, int64_t batch, int64_t K, int64_t channels,
                                int64_t L, int64_t N, vmb_layout layout) {
    return scan_workspace_bytes(mean_variant, batch, K, channels, L, N, layout);
}

vmb_status vmb_discrete_scan(const float* abar, const float* bu, const float* C,
                             const float* skip, float* y, int64_t batch, int64_t channels,
                             int64_t L, vmb_stream_t stream) {
    const vmb_status st = validate_discrete(abar, bu, C, skip, y, batch, channels, L);
    if (st != VMB_OK) return st;
    return launch_discrete_scan(abar, bu, C, skip, y, batch, channels, L,
                                static_cast<hipStream_t>(stream));
}

vmb_status vmb_channel_mean(const float* x, float* xm, int64_t batch, int64_t channels,
                            int64_t L, vmb_stream_t stream) {
    const vmb_status st = validate_channel_mean(x, xm, batch, channels, L);
    if (st != VMB_OK) return st;
    return launch_channel_mean(x, xm, batch, channels, L, static_cast<hipStream_t>(stream));
}

vmb_status vmb_mean_scan_status(const void* workspace, vmb_stream_t stream) {
    if (!workspace) return VMB_ERR_NULL;
    if (reinterpret_cast<uintptr_t>(workspace) % 16 != 0) return VMB_ERR_ALIGN;
    return mean_scan_status(workspace, static_cast<hipStream_t>(stream));
}

const char* vmb_status_string(vmb_status s) {
    switch (s) {
        case VMB_OK: return "ok";
        case VMB_ERR_NULL: return "a required pointer is NULL";
        case VMB_ERR_SHAPE: return "invalid or inconsistent shape";
        case VMB_ERR_DTYPE: return "unsupported dtype or dtype combination";
        case VMB_ERR_ALIGN: return "misaligned pointer";
        case VMB_ERR_ALIAS: return "output overlaps an input";
        case VMB_ERR_UNSUPPORTED: return "valid but unsupported configuration";
        case VMB_ERR_WORKSPACE: return "workspace missing or too small";
        case VMB_ERR_HIP: return "HIP runtime error at launch";
        case VMB_ERR_INCOMPLETE: return "a bounded wait of the call gave up; its outputs are partly NaN";
        default: return "unknown status";
    }
}

int vmb_abi_version(void) { return VMB_ABI_VERSION; }

}  // extern "C"
