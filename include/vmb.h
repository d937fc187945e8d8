/*
 * vmb.h -- C ABI of the MI355X (gfx950) SS2D selective-scan library (libvmb.so).
 *
 * The library implements the hot path of one SS2D block as described by
 * VMeanba (arXiv 2412.16602), Appendix A (VMamba paragraph) and Section 2.2:
 *
 *   cross-scan  : unfold an H x W feature map into K = 4 sequences of length
 *                 L = H*W (row-major, column-major and their reverses);
 *   scan        : the Mamba selective scan of eq. 3 with Abar = exp(Delta*A)
 *                 (eq. 4, first line), Bbar*u = Delta*B*u, and
 *                 Delta = softplus(delta + dt_bias) (eq. 6) -- either per
 *                 channel (full) or on the channel mean of the discretised
 *                 inputs with the result broadcast back (VMeanba, eq. 9);
 *   cross-merge : fold the four sequences back into one H x W map.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  - All tensor arguments are DEVICE pointers to contiguous row-major
 *    buffers owned by the caller. The library keeps no pointer after a call
 *    returns and allocates no device memory; scratch space is passed in as
 *    `workspace` (size from vmb_scan_workspace_bytes).
 *  - Every call is asynchronous on `stream` (a hipStream_t; NULL means the
 *    null stream) and never synchronises. Calls on one stream run in order.
 *  - Every argument is validated on the host BEFORE any device work is
 *    enqueued; on a non-VMB_OK status nothing was launched and nothing was
 *    written. No call prints, aborts or throws.
 *  - Base pointers of streamed tensors (x, xs, ys, y, u, delta, B, C,
 *    workspace) must be 16-byte aligned; A, D and dt_bias 4-byte aligned.
 *  - Outputs must not overlap any input (VMB_ERR_ALIAS); in-place is not
 *    supported.
 *  - Non-finite inputs are not checked; they propagate.
 *  - The library keeps no per-call state and is thread-safe. Its only
 *    host-side state is a process-wide 64-bit counter (atomic) that gives
 *    each mean-scan call a distinct tag for the flags its workgroups
 *    exchange, and per-device occupancy figures read once. Results are
 *    deterministic: no floating-point atomics, fixed summation orders.
 *  - Sizes are int64_t; a tensor may hold up to 2^31 - 1 elements per
 *    [.., L] sequence row and 2^40 elements in total.
 */
#ifndef VMB_H
#define VMB_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define VMB_ABI_VERSION 2

typedef void* vmb_stream_t; /* a hipStream_t */

typedef enum {
    VMB_OK = 0,
    VMB_ERR_NULL = 1,        /* a required pointer is NULL                         */
    VMB_ERR_SHAPE = 2,       /* a size is < 1, inconsistent or too large           */
    VMB_ERR_DTYPE = 3,       /* dtype value or dtype combination not supported     */
    VMB_ERR_ALIGN = 4,       /* a base pointer violates the alignment rule         */
    VMB_ERR_ALIAS = 5,       /* an output overlaps an input                        */
    VMB_ERR_UNSUPPORTED = 6, /* valid but unsupported (e.g. N not in {1,2,4,8,16}) */
    VMB_ERR_WORKSPACE = 7,   /* workspace NULL or smaller than required            */
    VMB_ERR_HIP = 8,         /* the HIP runtime reported an error at launch        */
    VMB_ERR_INCOMPLETE = 9   /* vmb_mean_scan_status only: a bounded wait of the
                                call gave up; the outputs it covers are NaN      */
} vmb_status;

typedef enum {
    VMB_F32 = 0,  /* IEEE binary32                                      */
    VMB_BF16 = 1  /* bfloat16 (top half of binary32); stores round to nearest even */
} vmb_dtype;

typedef enum {
    /* u, delta, y are per-direction sequences [batch, K, channels, L]. */
    VMB_LAYOUT_SEQ = 0,
    /* u is the feature map x [batch, channels, H, W], read through the
     * cross-scan maps; y is the merged map [batch, channels, H, W].
     * delta stays [batch, K, channels, L]. Requires K == 4 and L == H*W. */
    VMB_LAYOUT_2D = 1
} vmb_layout;

/*
 * Cross-scan (Appendix A, VMamba: "unfold the input feature map along four
 * directions"). For pixel (h, w) of x[b, d] and L = H*W:
 *   xs[b, 0, d, h*W + w]          = x[b, d, h, w]   (row-major)
 *   xs[b, 1, d, w*H + h]          = x[b, d, h, w]   (column-major)
 *   xs[b, 2, d, L - 1 - (h*W+w)]  = x[b, d, h, w]   (row-major, reversed)
 *   xs[b, 3, d, L - 1 - (w*H+h)]  = x[b, d, h, w]   (column-major, reversed)
 *
 *   x  : [batch, channels, H, W] of dtype dt (input)
 *   xs : [batch, 4, channels, H*W] of dtype dt (output)
 * A pure copy: bit-exact for both dtypes.
 */
vmb_status vmb_cross_scan(const void* x, void* xs, int64_t batch, int64_t channels,
                          int64_t H, int64_t W, vmb_dtype dt, vmb_stream_t stream);

/*
 * Cross-merge (Appendix A, VMamba: "merges the 4 sets of 1D sequences back
 * to 2D feature map"), the sum over directions at each pixel:
 *   y[b, d, h, w] = (ys[b,0,d,pi_0] + ys[b,2,d,pi_2]) + (ys[b,1,d,pi_1] + ys[b,3,d,pi_3])
 * with pi_k the positions listed for vmb_cross_scan, evaluated in binary32
 * in exactly this association (bf16 inputs widened exactly, one
 * nearest-even rounding at the end for a bf16 output).
 *
 *   ys : [batch, 4, channels, H*W] of dtype dt (input)
 *   y  : [batch, channels, H, W] of dtype dt (output)
 */
vmb_status vmb_cross_merge(const void* ys, void* y, int64_t batch, int64_t channels,
                           int64_t H, int64_t W, vmb_dtype dt, vmb_stream_t stream);

/*
 * Full selective scan (Appendix A: eq. 3, eq. 4 first line, eq. 6), one
 * recurrence per (b, k, d, n), c = k*channels + d:
 *   Delta_t = softplus(delta[b,k,d,t] + dt_bias[c])   (delta_softplus != 0)
 *           = delta[b,k,d,t] + dt_bias[c]             (delta_softplus == 0)
 *   h_{-1}  = 0
 *   h_t[n]  = exp(Delta_t * A[c,n]) * h_{t-1}[n] + Delta_t * B[b,k,n,t] * u[b,k,d,t]
 *   y_t     = sum_n C[b,k,n,t] * h_t[n] + D[c] * u[b,k,d,t]
 * State and accumulation in binary32 for both input dtypes.
 *
 *   u        : in_dtype, [batch, K, channels, L] (SEQ) or x [batch, channels, H, W] (2D)
 *   delta    : in_dtype, [batch, K, channels, L]
 *   A        : float32,  [K*channels, N]  (negative for a decaying state)
 *   B, C     : in_dtype, [batch, K, N, L]
 *   D        : float32,  [K*channels] or NULL (treated as 0)
 *   dt_bias  : float32,  [K*channels] or NULL (treated as 0)
 *   y        : out_dtype, [batch, K, channels, L] (SEQ) or [batch, channels, H, W] (2D)
 *   N        : 1, 2, 4, 8 or 16
 *   (in_dtype, out_dtype) : (F32, F32), (BF16, BF16) or (BF16, F32)
 *   H, W     : used by the 2D layout only (ignored for SEQ)
 *   workspace: device scratch of at least vmb_scan_workspace_bytes(0, ...)
 *              bytes (may be NULL when that is 0); contents on entry are
 *              irrelevant and undefined on exit.
 * VMB_ERR_UNSUPPORTED also for 2D maps the merge pass cannot take: planes
 * larger than H * (W + 1) = 12288 fp32 words that need more than 65535 tiles
 * of 32 pixels along a side, or that come in more than 2^24 (batch, channel)
 * planes (the same rule holds for vmb_mean_scan_fwd).
 */
vmb_status vmb_selective_scan_fwd(const void* u, const void* delta, const float* A,
                                  const void* B, const void* C, const float* D,
                                  const float* dt_bias, int delta_softplus, void* y,
                                  int64_t batch, int64_t K, int64_t channels, int64_t L,
                                  int64_t N, vmb_dtype in_dtype, vmb_dtype out_dtype,
                                  vmb_layout layout, int64_t H, int64_t W, void* workspace,
                                  size_t workspace_bytes, vmb_stream_t stream);

/*
 * Options of vmb_selective_scan_fwd_ex (bit flags; vmb_mean_scan_fwd_ex
 * takes them too, next to its vmb_mean_option bits).
 */
typedef enum {
    /* Eq. 4's second line read as zero-order hold,
     *   Bbar = (Delta A)^-1 (exp(Delta A) - I) Delta B,
     * i.e. Bbar u = phi(Delta A[c,n]) Delta B[b,k,n,t] u with
     * phi(x) = (e^x - 1) / x (phi(0) = 1), in place of the first-order
     * Delta B u; Abar = exp(Delta A) as before. Under the mean (T of eq. 9)
     * the per-state means (1/channels) sum_d phi(Delta_d A[c,n]) Delta_d u_d
     * take the place of mean_d Delta_d u_d. */
    VMB_SCAN_ZOH = 16
} vmb_scan_option;

/*
 * vmb_selective_scan_fwd with options (a bitwise OR of vmb_scan_option
 * values; 0 is vmb_selective_scan_fwd). Arguments, workspace and errors as for
 * vmb_selective_scan_fwd, plus VMB_ERR_UNSUPPORTED for an unknown bit.
 */
vmb_status vmb_selective_scan_fwd_ex(const void* u, const void* delta, const float* A,
                                     const void* B, const void* C, const float* D,
                                     const float* dt_bias, int delta_softplus, void* y,
                                     int64_t batch, int64_t K, int64_t channels, int64_t L,
                                     int64_t N, vmb_dtype in_dtype, vmb_dtype out_dtype,
                                     vmb_layout layout, int64_t H, int64_t W, void* workspace,
                                     size_t workspace_bytes, unsigned options,
                                     vmb_stream_t stream);

/*
 * VMeanba scan (Section 2.2, eq. 9): T averages the discretised scan inputs
 * over the channels of each direction, the scan runs once per (b, k), and
 * T^-1 broadcasts its output to every channel. With Delta as above and the
 * sums over d = 0 .. channels-1 of direction k (c = k*channels + d):
 *   Abar_mean[n,t] = mean_d exp(Delta_{d,t} * A[c,n])
 *   s_mean[t]      = mean_d Delta_{d,t} * u[b,k,d,t]
 *   r_mean[t]      = mean_d D[c] * u[b,k,d,t]
 *   h_t[n]         = Abar_mean[n,t] * h_{t-1}[n] + B[b,k,n,t] * s_mean[t],  h_{-1} = 0
 *   ytilde_t       = sum_n C[b,k,n,t] * h_t[n] + r_mean[t]
 *   y[b,k,d,t]     = ytilde_t for every d              (SEQ)
 *   y[b,d,h,w]     = cross-merge of ytilde over k      (2D, same for every d)
 * Arguments, shapes, dtypes and workspace rules are those of
 * vmb_selective_scan_fwd (workspace sized by vmb_scan_workspace_bytes(1, ...)).
 * Channel sums are binary32 in a fixed order (deterministic).
 * HIP graphs: a call made while `stream` is capturing takes the separate
 * passes, ordered by kernel boundaries alone (the one-launch form, whose
 * workgroups wait on per-call flags, would carry one call's flag value into
 * every replay), so a captured call replayed on new inputs computes the
 * result for those inputs. The same holds for _ex and _noalloc.
 */
vmb_status vmb_mean_scan_fwd(const void* u, const void* delta, const float* A, const void* B,
                             const void* C, const float* D, const float* dt_bias,
                             int delta_softplus, void* y, int64_t batch, int64_t K,
                             int64_t channels, int64_t L, int64_t N, vmb_dtype in_dtype,
                             vmb_dtype out_dtype, vmb_layout layout, int64_t H, int64_t W,
                             void* workspace, size_t workspace_bytes, vmb_stream_t stream);

/*
 * Other readings of where T acts in eq. 9 (Section 2.2), as bit flags for
 * vmb_mean_scan_fwd_ex. The paper states T on (Abar, Bbar u, C) and leaves
 * the skip term and the output shape open; these select the alternatives.
 */
typedef enum {
    /* D u stays outside T, per channel as in eq. 3:
     *   ytilde_t = sum_n C[b,k,n,t] h_t[n]   (no r_mean)
     *   y[b,k,d,t] = ytilde_t + D[c] u[b,k,d,t]
     * 2D layout: each channel adds ((D[0,d] + D[2,d]) + (D[1,d] + D[3,d])) x[b,d,h,w]
     * to the merged reduced output. */
    VMB_MEAN_SKIP_PER_CHANNEL = 1,
    /* T averages the raw timescale, input and state matrix, and the scan
     * discretises the means (eq. 4 after T):
     *   Delta_mean[t] = mean_d Delta_{d,t}, u_mean[t] = mean_d u[b,k,d,t],
     *   A_mean[n] = mean_d A[c,n],
     *   h_t[n] = exp(Delta_mean[t] A_mean[n]) h_{t-1}[n] + Delta_mean[t] B[b,k,n,t] u_mean[t] */
    VMB_MEAN_RAW = 2,
    /* T^-1 left out: y is [batch, K, 1, L] and holds ytilde (SEQ layout only;
     * not with VMB_MEAN_SKIP_PER_CHANNEL) */
    VMB_MEAN_NO_BROADCAST = 4,
    /* T over every channel of an image: the K directions' channels pooled
     * (K*channels of them), each keeping its direction's B and C. With the
     * sums over k and d (c = k*channels + d) and M = K*channels:
     *   Abar_mean[n,t] = (1/M) sum_{k,d} exp(Delta_{k,d,t} A[c,n])
     *   Bu_mean[n,t]   = (1/M) sum_k B[b,k,n,t] sum_d Delta_{k,d,t} u[b,k,d,t]
     *   C_mean[n,t]    = (1/K) sum_k C[b,k,n,t]
     *   r_mean[t]      = (1/M) sum_{k,d} D[c] u[b,k,d,t]
     *   h_t[n] = Abar_mean[n,t] h_{t-1}[n] + Bu_mean[n,t],  ytilde_t = sum_n C_mean h_t[n] + r_mean
     * one scan per batch element, broadcast to every (k, d); in the 2D layout
     * the four directions' (identical) sequences are merged as usual. Only as
     * the sole option bit. */
    VMB_MEAN_POOLED = 8,
    /* Test hook of the error report (vmb_mean_scan_status), not a reading:
     * on the one-launch path (every sequence at most 64 chunks of 64
     * positions, and a small grid) the first chunk of each sequence does not
     * raise its flag and the other chunks poll at most 8 times, so each of
     * them gives up and leaves NaN outputs; every kernel still ends normally.
     * Calls that take the separate passes ignore it. */
    VMB_MEAN_TEST_GIVE_UP = 1 << 30
} vmb_mean_option;

/*
 * vmb_mean_scan_fwd with a reading of T chosen by `options` (a bitwise OR of
 * vmb_mean_option values; 0 is vmb_mean_scan_fwd). Arguments and workspace as
 * for vmb_mean_scan_fwd, except that y is [batch, K, 1, L] with
 * VMB_MEAN_NO_BROADCAST. Errors as for vmb_mean_scan_fwd, plus
 * VMB_ERR_UNSUPPORTED for an unknown bit, VMB_MEAN_NO_BROADCAST with the 2D
 * layout, VMB_MEAN_NO_BROADCAST with VMB_MEAN_SKIP_PER_CHANNEL, or
 * VMB_MEAN_POOLED with any other bit. VMB_SCAN_ZOH (vmb_scan_option) may be
 * added to 0, VMB_MEAN_SKIP_PER_CHANNEL or VMB_MEAN_NO_BROADCAST.
 */
vmb_status vmb_mean_scan_fwd_ex(const void* u, const void* delta, const float* A, const void* B,
                                const void* C, const float* D, const float* dt_bias,
                                int delta_softplus, void* y, int64_t batch, int64_t K,
                                int64_t channels, int64_t L, int64_t N, vmb_dtype in_dtype,
                                vmb_dtype out_dtype, vmb_layout layout, int64_t H, int64_t W,
                                void* workspace, size_t workspace_bytes, unsigned options,
                                vmb_stream_t stream);

/*
 * For callers that cannot allocate device memory (code under HIP graph
 * capture, serving loops and harnesses that forbid hipMalloc): the VMeanba
 * scan of vmb_mean_scan_fwd (same arguments, same kernels, same results)
 * without the workspace arguments. Its scratch space is a fixed 8 MiB device
 * array inside the library, one per GPU, held until the process ends; the
 * call allocates nothing. Shapes whose workspace
 * (vmb_scan_workspace_bytes(1, ...)) exceeds 8 MiB return VMB_ERR_WORKSPACE
 * (the 56x56 map with 192 channels at batch 1 needs about 1.7 MB in the SEQ
 * layout, 4.3 MB in the 2D layout). Every call on one GPU shares that GPU's
 * array: calls that overlap in time on one GPU (different streams, or several
 * host threads) race and must be serialised by the caller. Nothing in the
 * array needs clearing between calls. The completion record of the array is
 * not exposed (vmb_mean_scan_status needs a workspace pointer): a bounded
 * wait that gives up still leaves NaN outputs, never stale values.
 * Errors as for vmb_mean_scan_fwd, plus VMB_ERR_HIP if the array's device
 * address cannot be read.
 */
vmb_status vmb_mean_scan_fwd_noalloc(const void* u, const void* delta, const float* A,
                                     const void* B, const void* C, const float* D,
                                     const float* dt_bias, int delta_softplus, void* y,
                                     int64_t batch, int64_t K, int64_t channels, int64_t L,
                                     int64_t N, vmb_dtype in_dtype, vmb_dtype out_dtype,
                                     vmb_layout layout, int64_t H, int64_t W,
                                     vmb_stream_t stream);

/*
 * Completion report of the most recent vmb_mean_scan_fwd / _ex call that used
 * `workspace` (the same pointer that call received). With at most 64 chunks
 * of 64 positions per sequence and a small grid, the mean scan runs in one
 * launch in which each workgroup waits for the chunk aggregates of the
 * earlier chunks of its sequence (the carry of the chunked scan of eq. 3,
 * composed associatively as in Appendix A). Those waits are bounded
 * (65,536 polls); a workgroup that gives up does not use aggregates it has
 * not seen: it writes NaN to the outputs of its chunk (every channel, and in
 * the 2-D layout every pixel fed by them) and records the call's tag in the
 * workspace. This call waits for `stream` (hipStreamSynchronize), reads the
 * 24-byte record at the start of the workspace, and returns
 *   VMB_OK             the call completed, no wait gave up;
 *   VMB_ERR_INCOMPLETE a wait of that call gave up (outputs partly NaN);
 *   VMB_ERR_WORKSPACE  no mean-scan call is recorded in this workspace;
 *   VMB_ERR_NULL / VMB_ERR_ALIGN (workspace NULL / not 16-byte aligned);
 *   VMB_ERR_HIP        the stream or the copy reported an error.
 * The record is written by every path of the mean scan (one launch or
 * separate passes), so a later call on the same workspace replaces it.
 */
vmb_status vmb_mean_scan_status(const void* workspace, vmb_stream_t stream);

/*
 * One-state scan on materialised, discretised inputs: the decomposition of
 * the paper's kernel experiments (Appendix D: the kernel only walks the
 * recurrence of eq. 3, discretisation runs outside it; Table 1 shapes, one
 * state per (d, t) as in the computational-complexity appendix). For every
 * (b, d):
 *   h_{-1} = 0
 *   h_t    = abar[b,d,t] * h_{t-1} + bu[b,d,t]
 *   y_t    = C[b,t] * h_t + skip[b,d,t]
 * With channels = 1 and inputs reduced by vmb_channel_mean, the same call is
 * the VMeanba kernel of those experiments (the scan of T(Abar), T(Bbar u)).
 *
 *   abar, bu : float32, [batch, channels, L]
 *   C        : float32, [batch, L]
 *   skip     : float32, [batch, channels, L] or NULL (treated as 0)
 *   y        : float32, [batch, channels, L] (output)
 * Binary32 state. Errors: VMB_ERR_NULL (abar, bu, C or y), VMB_ERR_SHAPE
 * (a size < 1 or too large), VMB_ERR_ALIGN (a base not 16-byte aligned),
 * VMB_ERR_ALIAS (y overlaps an input).
 */
vmb_status vmb_discrete_scan(const float* abar, const float* bu, const float* C,
                             const float* skip, float* y, int64_t batch, int64_t channels,
                             int64_t L, vmb_stream_t stream);

/*
 * The transform T of eq. 9 on a materialised input (Section 2.2: the mean
 * over the inner channel axis):
 *   xm[b, t] = (1 / channels) * sum_{d = 0 .. channels-1} x[b, d, t]
 *   x  : float32, [batch, channels, L];  xm : float32, [batch, L] (output)
 * Binary32 sums in a fixed order (deterministic). Errors as for
 * vmb_discrete_scan.
 */
vmb_status vmb_channel_mean(const float* x, float* xm, int64_t batch, int64_t channels,
                            int64_t L, vmb_stream_t stream);

/*
 * Bytes of device workspace the scan of the given shape needs
 * (mean_variant = 0: vmb_selective_scan_fwd, 1: vmb_mean_scan_fwd).
 * Returns 0 when none is needed and SIZE_MAX for an invalid shape.
 */
size_t vmb_scan_workspace_bytes(int mean_variant, int64_t batch, int64_t K, int64_t channels,
                                int64_t L, int64_t N, vmb_layout layout);

/*
 * The selection projections of eq. 6 (Appendix A, Mamba paragraph), which
 * make the scan's B, C and timescale functions of its input: per (b, k)
 * sequence u[b,k,:,t] and with the direction's weights
 * W[k] = [R timescale rows; N rows for B; N rows for C] over the channels,
 *   x_dbl[r,t]       = sum_d W[k,r,d] u[b,k,d,t]          (r < R + 2N)
 *   B[b,k,n,t]       = x_dbl[R + n, t]                     (s_B = Linear_N)
 *   C[b,k,n,t]       = x_dbl[R + N + n, t]                 (s_C = Linear_N)
 *   delta[b,k,d,t]   = sum_r W_dt[k,d,r] x_dbl[r,t]        (s_Delta, rank R)
 * With W_dt NULL and R = 1, delta[b,k,d,t] = x_dbl[0,t] for every d: the
 * paper's Broadcast_D(Linear_1(u)). delta is s_Delta(u): the scan entry
 * points add the Parameter (dt_bias) and apply softplus. Products are
 * accumulated in binary32 on the matrix cores.
 *
 *   u      : [batch, K, channels, L] (SEQ layout), dtype
 *   W      : float32, [K, R + 2N, channels]
 *   W_dt   : float32, [K, channels, R], or NULL (then R must be 1)
 *   delta  : [batch, K, channels, L] (output), dtype
 *   B, C   : [batch, K, N, L] (outputs), dtype
 *   dtype  : VMB_F32 or VMB_BF16 (outputs rounded to nearest even)
 * Sizes: N in {1, 2, 4, 8, 16}; 1 <= R <= 64 (a rank of ceil(channels / 32)
 *   covers inner widths up to 2048).
 * Errors: VMB_ERR_NULL (u, W, delta, B or C NULL), VMB_ERR_SHAPE (sizes),
 * VMB_ERR_UNSUPPORTED (N, R, or W_dt NULL with R != 1), VMB_ERR_DTYPE,
 * VMB_ERR_ALIGN (a base pointer of u, delta, B, C not 16-byte aligned, of
 * W or W_dt not 4-byte aligned), VMB_ERR_ALIAS (an output overlaps an input
 * or another output).
 */
vmb_status vmb_ss2d_projections(const void* u, const float* W, const float* W_dt, void* delta,
                                void* B, void* C, int64_t batch, int64_t K, int64_t channels,
                                int64_t L, int64_t N, int64_t R, vmb_dtype dtype,
                                vmb_stream_t stream);

/*
 * The step after the cross-merge in VMamba's SS2D block, which the paper's
 * models are built from (the paper's text ends the SS2D computation at the
 * merge of Appendix A): a layer normalisation over the channels of each
 * pixel, then the SiLU gate by a second branch z. Per pixel p of image b:
 *   mu[b,p]    = mean_d y[b,d,p],  var[b,p] = mean_d (y[b,d,p] - mu[b,p])^2
 *   out[b,d,p] = (y[b,d,p] - mu[b,p]) / sqrt(var[b,p] + eps) * gamma[d] + beta[d]
 *   out[b,d,p] *= z[b,d,p] / (1 + exp(-z[b,d,p]))       (z not NULL)
 * Statistics in binary32 (a mean pass, then the centred sum of squares).
 *
 *   y, out : [batch, channels, P] (the 2-D layout, P = H * W), dtype
 *   z      : [batch, channels, P], dtype, or NULL (no gate)
 *   gamma, beta : float32 [channels], or NULL (1 and 0)
 *   eps    : >= 0, finite
 *   dtype  : VMB_F32 or VMB_BF16 (out rounded to nearest even)
 * Errors: VMB_ERR_NULL (y or out NULL), VMB_ERR_SHAPE (sizes, eps),
 * VMB_ERR_DTYPE, VMB_ERR_ALIGN (y, z, out not aligned to their element,
 * gamma, beta not 4-byte aligned), VMB_ERR_ALIAS (out overlaps y, z, gamma
 * or beta).
 */
vmb_status vmb_ss2d_out_norm(const void* y, const void* z, const float* gamma, const float* beta,
                             float eps, void* out, int64_t batch, int64_t channels, int64_t P,
                             vmb_dtype dtype, vmb_stream_t stream);

/* Static, NUL-terminated description of a status code. */
const char* vmb_status_string(vmb_status s);

/* VMB_ABI_VERSION of the loaded library. */
int vmb_abi_version(void);

#ifdef __cplusplus
}
#endif

#endif /* VMB_H */
