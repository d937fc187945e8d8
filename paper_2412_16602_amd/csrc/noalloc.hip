// noalloc.hip -- the VMeanba scan (Section 2.2, eq. 9) for callers that cannot
// allocate device memory: vmb_mean_scan_fwd_noalloc runs the kernels of
// vmb_mean_scan_fwd with their workspace taken from a fixed device array of
// this file instead of a caller-provided buffer.
//
// The array lives in every GPU the library runs on until the process ends.
// Its device address is read once per device (hipGetSymbolAddress, with that
// device current) and kept; the array's name itself is only a host-side
// stand-in and is never handed to a kernel or a copy.
#include <mutex>

#include "vmb_internal.h"

namespace vmb {
namespace {

constexpr size_t kScratchBytes = size_t{8} << 20;  // 8 MiB per device
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
std::once_flag g_once[kMaxDevices];
void* g_ptr[kMaxDevices];
hipError_t g_err[kMaxDevices];

// Device address of this device's copy of the array, or nullptr.
void* scratch_ptr() {
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
    std::call_once(g_once[dev], [dev] {
        void* p = nullptr;
        g_err[dev] = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        g_ptr[dev] = g_err[dev] == hipSuccess ? p : nullptr;
    });
    return g_ptr[dev];
}

}  // namespace
}  // namespace vmb

using namespace vmb;

extern "C" {

vmb_status vmb_mean_scan_fwd_noalloc(const void* u, const void* delta, const float* A,
                                     const void* B, const void* C, const float* D,
                                     const float* dt_bias, int delta_softplus, void* y,
                                     int64_t batch, int64_t K, int64_t channels, int64_t L,
                                     int64_t N, vmb_dtype in_dtype, vmb_dtype out_dtype,
                                     vmb_layout layout, int64_t H, int64_t W,
                                     vmb_stream_t stream) {
    const size_t need = scan_workspace_bytes(1, batch, K, channels, L, N, layout);
    if (need != SIZE_MAX && need > kScratchBytes) return VMB_ERR_WORKSPACE;
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
    a.options = 0;
    a.stream = static_cast<hipStream_t>(stream);
    // validate with a stand-in workspace first, so that a bad call touches no HIP state
    a.ws = reinterpret_cast<void*>(uintptr_t{256});
    a.ws_bytes = kScratchBytes;
    vmb_status st = validate_scan(a, 1);
    if (st != VMB_OK && st != VMB_ERR_ALIAS) return st;
    a.ws = scratch_ptr();
    if (!a.ws) return VMB_ERR_HIP;
    st = validate_scan(a, 1);
    if (st != VMB_OK) return st;
    return launch_mean_scan(a);
}

}  // extern "C"
