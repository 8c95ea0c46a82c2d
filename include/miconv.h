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
 *     after returning and allocates no device memory; as the passes only
 *     launch kernels (no memset, copy or synchronisation), they can be
 *     captured into a HIP graph and replayed (conv_tune, which times and
 *     synchronises, cannot);
 *   - results are bitwise reproducible for the same shape, inputs, device
 *     and plan (every reduction runs in a fixed order, no float atomics);
 *     the plan is the built-in rule unless one was set or tuned for the
 *     shape (conv_plan_set, conv_tune below);
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
    MICONV_ERR_WORKSPACE = -3, /* ws_bytes below the need of the plan the call runs (a size
                                  from conv_workspace_size() always suffices), or ws
                                  NULL when a workspace is needed */
    MICONV_ERR_ALIAS = -4,     /* an output range overlaps an input, another output or ws */
    MICONV_ERR_ALIGN = -5,     /* a tensor or workspace pointer is not 16-byte aligned */
    MICONV_ERR_DEVICE = -6,    /* no current HIP device, or it is not gfx950 */
    MICONV_ERR_LAUNCH = -7,    /* a kernel launch reported an error */
    MICONV_ERR_PASS = -8,      /* unknown pass id */
    MICONV_ERR_PLAN = -9,      /* plan index outside [0, conv_plan_count()) */
    MICONV_ERR_MODE = -10,     /* pooling mode other than MICONV_POOL_MAX / _AVG */
    MICONV_ERR_SCRATCH = -11   /* conv_bwd_weight_noalloc: the plan's workspace exceeds
                                  MICONV_NOALLOC_SCRATCH_BYTES */
} miconv_status;

/* Pass ids for conv_workspace_size and the plan calls. */
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
 * shape: the largest need over all of the shape's candidate plans (see
 * conv_plan_count below), so that a workspace of this size stays sufficient
 * whatever plan is stored for the shape later, by conv_plan_set or conv_tune,
 * from this or another thread.  conv_plan_workspace_size gives one plan's
 * (often smaller) need.  0 if no plan needs a workspace or if the shape or
 * pass id is invalid (the pass itself then reports the error).  Host-only
 * (the candidate plans depend on the current device's compute-unit count,
 * read once per device; 256 when no device can be queried).
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
 * conv_bwd_weight without a workspace argument, for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid allocation): the same pass, plan and kernels as
 * conv_bwd_weight (same results, bit for bit), with the workspace taken from
 * a fixed device array inside the library of MICONV_NOALLOC_SCRATCH_BYTES
 * (96 MiB), one per GPU, held from the library's first use on that GPU until
 * the process ends.  The call allocates nothing (no hipMalloc, no allocating
 * library routine); the first call on a device looks up that device's array.
 * Returns the statuses of conv_bwd_weight (but never MICONV_ERR_WORKSPACE),
 * or MICONV_ERR_SCRATCH, before any launch, when the plan the call would run
 * needs more than the array holds (conv_plan_workspace_size of the current
 * plan tells).  Every call on a GPU shares that GPU's array: calls that
 * overlap in time on one GPU (other threads, other streams without ordering)
 * race and must not be issued.  Nothing in the array needs to start at zero.
 */
#define MICONV_NOALLOC_SCRATCH_BYTES (96u << 20)
int conv_bwd_weight_noalloc(int N, int C, int H, int W, int K, int R, int S, int stride,
                            int pad, int group, const float *x, const float *dy, float *dw,
                            float *db, hipStream_t stream);

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

/*
 * Plan selection (Sec. IV-B: a mixed strategy of convolution plans, chosen
 * per layer; Sec. VI-A: the framework times its strategies over the first
 * training iterations and keeps the fastest).  Every pass of a shape has a
 * list of candidate plans (kernel tile, split of the reduction, and for
 * backward-data stride phases or pixel blocks); candidate 0 is the built-in
 * rule.  All candidates compute the same result up to fp32 rounding order.
 * The choice is kept per (device, pass, shape) in a process-wide table that
 * the conv_* calls consult; the table is thread-safe.  Arguments after
 * `pass` are those of the pass.
 *
 * conv_plan_count:  number of candidates (>= 1), or a negative status
 *                   (MICONV_ERR_SHAPE, MICONV_ERR_PASS).  Host-only.
 * conv_plan_get:    candidate the calls use now on the current device
 *                   (0 when none is stored).
 * conv_plan_set:    use candidate `index` from now on (0 restores the rule);
 *                   MICONV_ERR_PLAN if index is out of range.
 * conv_plan_clear:  forget every stored choice.
 * conv_plan_name:   NUL-terminated description of candidate `index` into
 *                   buf (truncated to len bytes); MICONV_ERR_NULL if buf is
 *                   NULL or len is 0.
 * conv_plan_workspace_size: workspace bytes of candidate `index` (0 if the
 *                   shape, pass or index is invalid, or it needs none).
 */
int conv_plan_count(int pass, int N, int C, int H, int W, int K, int R, int S, int stride,
                    int pad, int group);
int conv_plan_get(int pass, int N, int C, int H, int W, int K, int R, int S, int stride, int pad,
                  int group);
int conv_plan_set(int pass, int N, int C, int H, int W, int K, int R, int S, int stride, int pad,
                  int group, int index);
int conv_plan_clear(void);
int conv_plan_name(int pass, int N, int C, int H, int W, int K, int R, int S, int stride,
                   int pad, int group, int index, char *buf, size_t len);
size_t conv_plan_workspace_size(int pass, int N, int C, int H, int W, int K, int R, int S,
                                int stride, int pad, int group, int index);

/*
 * Times every candidate of `pass` whose workspace fits ws_bytes on the
 * caller's tensors (one untimed run, then `reps` timed runs back to back on
 * `stream`, HIP events around them; reps < 1 counts as 1), stores the
 * fastest for this shape as with conv_plan_set, writes its index to *chosen
 * (if not NULL), and runs it once more so the outputs hold its result.
 * Blocks the host until the timed runs finish.  Tensors:
 *   MICONV_PASS_FWD:         in0 = x, in1 = w, in2 = b (may be NULL), out0 = y
 *   MICONV_PASS_BWD_DATA:    in0 = dy, in1 = w, out0 = dx (in2, out1 ignored)
 *   MICONV_PASS_BWD_WEIGHT:  in0 = x, in1 = dy, out0 = dw, out1 = db (may be
 *                            NULL; in2 ignored)
 * Returns the statuses of the pass (checked on the first candidate run),
 * MICONV_ERR_WORKSPACE if no candidate fits ws_bytes, or MICONV_ERR_LAUNCH
 * if an event call fails; on an error nothing is stored.  The events of
 * conv_set_timing_events are not recorded by the runs inside.
 */
int conv_tune(int pass, int N, int C, int H, int W, int K, int R, int S, int stride, int pad,
              int group, const float *in0, const float *in1, const float *in2, float *out0,
              float *out1, void *ws, size_t ws_bytes, int reps, hipStream_t stream, int *chosen);

/*
 * Pooling layer (Sec. IV-D: each output is the maximum or the average of a
 * window of its input plane; the paper tiles the plane into non-overlapping
 * K x K windows, i.e. R = S = stride, pad = 0 below).  Caffe's general form:
 * window R x S, stride, zero padding pad < min(R, S), on x [N][C][H][W]
 * giving y [N][C][P][Q] with P = ceil((H + 2 pad - R) / stride) + 1, less one
 * when pad > 0 and the last window would start at or past H + pad (Q alike).
 *   MICONV_POOL_MAX: y = maximum over the window's elements inside the
 *     image; mask (may be NULL in pool_fwd) receives the first maximum's
 *     index h * W + w within its plane, in row-major order.
 *   MICONV_POOL_AVG: y = sum over the window's elements inside the image,
 *     divided by the window's area clipped to the padded image (padding
 *     counts, the overhang past it does not); mask is not used.
 * pool_bwd writes every element of dx: the sum, over the windows that cover
 * the element (in window order), of their dy (max: only windows whose mask
 * names the element; avg: dy / area).  mask is required for max.
 * Buffers are caller-owned device memory, 16-byte aligned, outputs not
 * overlapping inputs; no workspace.  Statuses as for the convolution calls,
 * plus MICONV_ERR_MODE; MICONV_ERR_SHAPE also when pad >= R or pad >= S,
 * when N*C*H*W or N*C*P*Q is above 2^31 - 1, or when the last window would
 * cover no element of the image (possible without padding when the stride
 * exceeds the window: the rounded-up count then puts that window past the
 * edge).  pool_output_size is host-only.
 */
#define MICONV_POOL_MAX 0
#define MICONV_POOL_AVG 1
int pool_output_size(int H, int W, int R, int S, int stride, int pad, int *P, int *Q);
int pool_fwd(int mode, int N, int C, int H, int W, int R, int S, int stride, int pad,
             const float *x, float *y, int *mask, hipStream_t stream);
int pool_bwd(int mode, int N, int C, int H, int W, int R, int S, int stride, int pad,
             const float *dy, const int *mask, float *dx, hipStream_t stream);

/* Static, NUL-terminated description of a status code (never NULL). */
const char *conv_error_string(int status);

#ifdef __cplusplus
}
#endif

#endif /* MICONV_H */
