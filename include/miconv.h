/*
 * miconv: fp32 convolution-layer training passes for AMD Instinct MI355X
 * (gfx950), as a C ABI.
 *
 * The three passes are the ones a convolution layer runs in training
 * (swCaffe, Sec. II-C and Table II: "forward", "in_diff backward" and
 * "weight_diff backward"); Sec. IV-B defines the layer as im2col followed by
 * a GEMM with the filter bank seen as an (out-channel) x (in-channel x
 * filter rows x filter cols) matrix, zero padding, and col2im for the
 * backward data movement.
 *
 * Notation (all tensors fp32, contiguous, row-major):
 *   x  [N][C][H][W]      input          dx [N][C][H][W]   input gradient
 *   w  [K][C/G][R][S]    filters        dw [K][C/G][R][S] filter gradient
 *   b  [K]               bias           db [K]            bias gradient
 *   y  [N][K][P][Q]      output         dy [N][K][P][Q]   output gradient
 * with G = group, P = floor((H + 2 pad - R) / stride) + 1, Q likewise from
 * W and S.  Group g owns input channels [g C/G, (g+1) C/G) and filters
 * [g K/G, (g+1) K/G).  The forward pass is a cross-correlation:
 *   y[n,k,p,q] = b[k] + sum_{c,r,s} x[n, g C/G + c, p stride - pad + r,
 *                                     q stride - pad + s] * w[k,c,r,s]
 * where coordinates outside the image read zero.
 *
 * Ownership and execution:
 *   - every tensor pointer is a DEVICE pointer owned by the caller; inputs
 *     are read only; every element of every output is overwritten (input
 *     pixels that no window covers get an exact 0 in dx);
 *   - ws is a caller-allocated device workspace of at least
 *     conv_workspace_size(...) bytes; its contents are undefined afterwards;
 *   - kernels are enqueued on `stream` (NULL = the null stream) and the
 *     calls return without synchronising; the library keeps no pointer
 *     after returning and allocates no device memory;
 *   - results are bitwise reproducible for the same shape, inputs and
 *     device (every reduction runs in a fixed order, no float atomics);
 *   - the calls clear the calling thread's pending HIP error before
 *     launching; a fault inside a kernel surfaces at the caller's next
 *     synchronisation.
 *
 * Errors: every argument check runs before any launch, so a call that
 * returns an error has written nothing.
 */
#ifndef MICONV_H
#define MICONV_H

#include <stddef.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum miconv_status {
    MICONV_OK = 0,
    MICONV_ERR_SHAPE = -1,     /* a dim < 1, pad < 0, stride < 1, C or K not divisible by
                                  group, P or Q < 1, a tensor above 2^31 - 1 elements, one
                                  image (C*H*W or K*P*Q) or the filter bank above 2^29 - 1
                                  elements (also counted as K rows of (C/G)*R*S and as C
                                  rows of (K/G)*R*S, each rounded up to a multiple of 16),
                                  H, W, R, S or pad above 32767, or group above 65535 */
    MICONV_ERR_NULL = -2,      /* a required pointer is NULL */
    MICONV_ERR_WORKSPACE = -3, /* ws_bytes below conv_workspace_size(), or ws NULL when
                                  a workspace is needed */
    MICONV_ERR_ALIAS = -4,     /* an output range overlaps an input, another output or ws */
    MICONV_ERR_ALIGN = -5,     /* a tensor or workspace pointer is not 16-byte aligned */
    MICONV_ERR_DEVICE = -6,    /* no current HIP device, or it is not gfx950 */
    MICONV_ERR_LAUNCH = -7,    /* a kernel launch reported an error */
    MICONV_ERR_PASS = -8       /* conv_workspace_size: unknown pass id */
} miconv_status;

/* Pass ids for conv_workspace_size. */
#define MICONV_PASS_FWD 0
#define MICONV_PASS_BWD_DATA 1
#define MICONV_PASS_BWD_WEIGHT 2

/*
 * Output extent of the layer: P = floor((H + 2 pad - R) / stride) + 1 and
 * Q = floor((W + 2 pad - S) / stride) + 1 (zero padding on both sides, the
 * Caffe reading of the output-size formula of Sec. IV-B, which the paper
 * prints without padding or rounding).  Host-only; touches no device.
 * Returns MICONV_OK, MICONV_ERR_NULL if P or Q is NULL, or MICONV_ERR_SHAPE
 * if an argument is out of range or the window does not fit (P or Q < 1;
 * *P and *Q are then left unchanged).
 */
int conv_output_size(int H, int W, int R, int S, int stride, int pad, int *P, int *Q);

/*
 * Bytes of device workspace that pass `pass` (MICONV_PASS_*) needs for this
 * shape; 0 if it needs none or if the shape or pass id is invalid (the pass
 * itself then reports the error).  Host-only; touches no device.
 */
size_t conv_workspace_size(int pass, int N, int C, int H, int W, int K, int R, int S,
                           int stride, int pad, int group);

/*
 * Forward pass (Table II "forward"; Sec. IV-B im2col + GEMM):
 *   y = b + w (*) x   as defined above.
 * b may be NULL (no bias).  x, w, y required.
 */
int conv_fwd(int N, int C, int H, int W, int K, int R, int S, int stride, int pad, int group,
             const float *x, const float *w, const float *b, float *y,
             void *ws, size_t ws_bytes, hipStream_t stream);

/*
 * Backward-data pass (Table II "in_diff backward"; Sec. IV-B col2im): the
 * adjoint of the forward map in x,
 *   dx[n,c',h,w] = sum over filters k of c's group and taps (r,s) with
 *                  p = (h + pad - r) / stride, q = (w + pad - s) / stride
 *                  integers in [0,P) x [0,Q) of dy[n,k,p,q] * w[k,c,r,s],
 * where c' = g C/G + c.  dy, w, dx required.
 */
int conv_bwd_data(int N, int C, int H, int W, int K, int R, int S, int stride, int pad,
                  int group, const float *dy, const float *w, float *dx,
                  void *ws, size_t ws_bytes, hipStream_t stream);

/*
 * Backward-weight pass (Table II "weight_diff backward"): the adjoint of the
 * forward map in w, and the bias gradient,
 *   dw[k,c,r,s] = sum_{n,p,q} dy[n,k,p,q] * x[n, g C/G + c, p stride - pad + r,
 *                                             q stride - pad + s]
 *   db[k]       = sum_{n,p,q} dy[n,k,p,q].
 * db may be NULL (not computed).  x, dy, dw required.
 */
int conv_bwd_weight(int N, int C, int H, int W, int K, int R, int S, int stride, int pad,
                    int group, const float *x, const float *dy, float *dw, float *db,
                    void *ws, size_t ws_bytes, hipStream_t stream);

/*
 * Benchmark instrumentation; not needed to compute anything.  After this
 * call, every conv_fwd / conv_bwd_data / conv_bwd_weight made by the calling
 * thread records `before` on its stream immediately before the launch of the
 * pass's first implicit-GEMM kernel and `after` immediately after its last
 * one, so hipEventElapsedTime(before, after) is the GEMM kernels' device
 * time without the filter packing, split-K reduction and bias-gradient
 * kernels around them (for a conv_bwd_data computed phase by phase it spans
 * every stride phase, packing in between included; one with few input
 * channels per group runs a single blocked GEMM instead).  Pass two NULLs to stop.  The events
 * are created and owned by the caller.  Returns MICONV_OK, or
 * MICONV_ERR_NULL if exactly one of the two is NULL.
 */
int conv_set_timing_events(hipEvent_t before, hipEvent_t after);

/* Static, NUL-terminated description of a status code (never NULL). */
const char *conv_error_string(int status);

#ifdef __cplusplus
}
#endif

#endif /* MICONV_H */
