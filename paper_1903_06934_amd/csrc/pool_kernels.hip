// Pooling layer (forward and backward), max with argmax mask or average.
// Memory-bound.  Planes that fit in LDS: one workgroup per (n, c) plane,
// staged once with consecutive loads.  Larger planes: one thread per written
// element, windows read through the caches.  Indices are decoded with
// constant-divisor division.
#include "internal.h"

namespace miconv {

namespace {

// Window of output index p along an axis: inside the image [lo, hi), and
// the extent of the window clipped to the padded image (the average's
// divisor counts padding but not the overhang past it).
struct Win {
    int lo, hi, ext;
};

__device__ __forceinline__ Win window(int p, int stride, int pad, int filt, int in)
{
    const int start = p * stride - pad;
    const int end = min(start + filt, in + pad);
    return Win{max(start, 0), min(end, in), end - start};
}

template <bool MAX>
__global__ __launch_bounds__(256) void pool_fwd_kernel(const float *__restrict__ x,
                                                       float *__restrict__ y,
                                                       int *__restrict__ mask, int H, int W,
                                                       int R, int S, int stride, int pad,
                                                       FastDiv pq, FastDiv q_, uint32_t total)
{
    for (uint32_t i = blockIdx.x * blockDim.x + threadIdx.x; i < total;
         i += gridDim.x * blockDim.x) {
        const uint32_t nc = fast_div(i, pq), pix = i - nc * pq.d;
        const uint32_t p = fast_div(pix, q_), q = pix - p * q_.d;
        const Win wh = window((int)p, stride, pad, R, H), ww = window((int)q, stride, pad, S, W);
        const float *xp = x + (size_t)nc * H * W;
        if constexpr (MAX) {
            // First maximum in row-major order; the window always holds an
            // image element (pad < window, and no window lies past the image),
            // so arg is set.
            float best = -__builtin_inff();
            int arg = -1;
            for (int h = wh.lo; h < wh.hi; h++)
                for (int w = ww.lo; w < ww.hi; w++) {
                    const float v = xp[h * W + w];
                    if (v > best) {
                        best = v;
                        arg = h * W + w;
                    }
                }
            y[i] = best;
            if (mask)
                mask[i] = arg;
        } else {
            float sum = 0.f;
            for (int h = wh.lo; h < wh.hi; h++)
                for (int w = ww.lo; w < ww.hi; w++)
                    sum += xp[h * W + w];
            y[i] = sum / (float)(wh.ext * ww.ext);
        }
    }
}

// dx[h][w] gathers, in the order of the windows (p, then q), the dy of every
// window that covers it: all of it for max when the window's argmax is this
// element, dy / area for the average.  No atomics: each thread writes one dx.
template <bool MAX>
__global__ __launch_bounds__(256) void pool_bwd_kernel(const float *__restrict__ dy,
                                                       const int *__restrict__ mask,
                                                       float *__restrict__ dx, int H, int W,
                                                       int P, int Q, int R, int S, int stride,
                                                       int pad, FastDiv hw, FastDiv w_,
                                                       FastDiv st_, uint32_t total)
{
    for (uint32_t i = blockIdx.x * blockDim.x + threadIdx.x; i < total;
         i += gridDim.x * blockDim.x) {
        const uint32_t nc = fast_div(i, hw), pix = i - nc * hw.d;
        const int h = (int)fast_div(pix, w_), w = (int)(pix - (uint32_t)h * w_.d);
        // windows p with p stride - pad <= h < p stride - pad + R
        const int hp = h + pad, wp = w + pad;  // >= 0
        const int p0 = hp < R ? 0 : (int)fast_div((uint32_t)(hp - R), st_) + 1;
        const int p1 = min((int)fast_div((uint32_t)hp, st_), P - 1);
        const int q0 = wp < S ? 0 : (int)fast_div((uint32_t)(wp - S), st_) + 1;
        const int q1 = min((int)fast_div((uint32_t)wp, st_), Q - 1);
        const size_t base = (size_t)nc * P * Q;
        float acc = 0.f;
        for (int p = p0; p <= p1; p++)
            for (int q = q0; q <= q1; q++) {
                const size_t o = base + (size_t)p * Q + q;
                if constexpr (MAX) {
                    // Both loads issued together; the select keeps the sum's order.
                    const float g = dy[o];
                    acc += mask[o] == (int)pix ? g : 0.f;
                } else {
                    const Win wh = window(p, stride, pad, R, H), ww = window(q, stride, pad, S, W);
                    acc += dy[o] / (float)(wh.ext * ww.ext);
                }
            }
        dx[i] = acc;
    }
}

// Whole-plane variants, for planes that fit in LDS: a workgroup stages one
// (n, c) plane with consecutive (coalesced) loads, then computes that
// plane's outputs from LDS, so every input byte is read from HBM once and in
// order.  Same arithmetic in the same order as the kernels above: the
// results are identical bit for bit.
template <bool MAX>
__global__ __launch_bounds__(256) void pool_fwd_plane_kernel(const float *__restrict__ x,
                                                             float *__restrict__ y,
                                                             int *__restrict__ mask, int H, int W,
                                                             int R, int S, int stride, int pad,
                                                             FastDiv q_, uint32_t P,
                                                             uint32_t planes)
{
    extern __shared__ float xs[];
    const uint32_t hw = (uint32_t)H * (uint32_t)W, pq = P * q_.d;
    for (uint32_t nc = blockIdx.x; nc < planes; nc += gridDim.x) {
        const float *xp = x + (size_t)nc * hw;
        for (uint32_t i = threadIdx.x; i < hw; i += blockDim.x)
            xs[i] = xp[i];
        __syncthreads();
        for (uint32_t o = threadIdx.x; o < pq; o += blockDim.x) {
            const uint32_t p = fast_div(o, q_), q = o - p * q_.d;
            const Win wh = window((int)p, stride, pad, R, H), ww = window((int)q, stride, pad, S, W);
            const size_t out = (size_t)nc * pq + o;
            if constexpr (MAX) {
                float best = -__builtin_inff();
                int arg = -1;
                for (int h = wh.lo; h < wh.hi; h++)
                    for (int w = ww.lo; w < ww.hi; w++) {
                        const float v = xs[h * W + w];
                        if (v > best) {
                            best = v;
                            arg = h * W + w;
                        }
                    }
                y[out] = best;
                if (mask)
                    mask[out] = arg;
            } else {
                float sum = 0.f;
                for (int h = wh.lo; h < wh.hi; h++)
                    for (int w = ww.lo; w < ww.hi; w++)
                        sum += xs[h * W + w];
                y[out] = sum / (float)(wh.ext * ww.ext);
            }
        }
        __syncthreads();  // the plane's reads are done before the next one lands
    }
}

template <bool MAX>
__global__ __launch_bounds__(256) void pool_bwd_plane_kernel(const float *__restrict__ dy,
                                                             const int *__restrict__ mask,
                                                             float *__restrict__ dx, int H, int W,
                                                             int P, int Q, int R, int S,
                                                             int stride, int pad, FastDiv w_,
                                                             FastDiv st_, uint32_t planes)
{
    extern __shared__ float gs[];  // dy plane, then (max) the mask plane
    int *ms = (int *)(gs + P * Q);
    const uint32_t hw = (uint32_t)H * (uint32_t)W, pq = (uint32_t)P * (uint32_t)Q;
    const uint32_t rows = blockDim.x / (uint32_t)W;
    for (uint32_t nc = blockIdx.x; nc < planes; nc += gridDim.x) {
        for (uint32_t i = threadIdx.x; i < pq; i += blockDim.x) {
            gs[i] = dy[(size_t)nc * pq + i];
            if constexpr (MAX)
                ms[i] = mask[(size_t)nc * pq + i];
        }
        __syncthreads();
        // Thread t keeps column w = t % W of rows t / W, t / W + rows, ...
        // (rows = blockDim.x / W rows at a time, W <= blockDim.x), so the
        // column's window range is decoded once and each row's once per row.
        if (threadIdx.x < rows * (uint32_t)W) {
            const int w = (int)(threadIdx.x - fast_div(threadIdx.x, w_) * w_.d);
            const int wp = w + pad;
            const int q0 = wp < S ? 0 : (int)fast_div((uint32_t)(wp - S), st_) + 1;
            const int q1 = min((int)fast_div((uint32_t)wp, st_), Q - 1);
            for (int h = (int)fast_div(threadIdx.x, w_); h < H; h += (int)rows) {
                const int pix = h * W + w;
                const int hp = h + pad;
                const int p0 = hp < R ? 0 : (int)fast_div((uint32_t)(hp - R), st_) + 1;
                const int p1 = min((int)fast_div((uint32_t)hp, st_), P - 1);
                float acc = 0.f;
                for (int p = p0; p <= p1; p++)
                    for (int q = q0; q <= q1; q++) {
                        const int o = p * Q + q;
                        if constexpr (MAX) {
                            acc += ms[o] == pix ? gs[o] : 0.f;
                        } else {
                            const Win wh = window(p, stride, pad, R, H),
                                      ww = window(q, stride, pad, S, W);
                            acc += gs[o] / (float)(wh.ext * ww.ext);
                        }
                    }
                dx[(size_t)nc * hw + pix] = acc;
            }
        }
        __syncthreads();
    }
}

// Planes of at least kPlaneMin elements whose staged data fits in kPlaneLds
// bytes take the whole-plane kernels (smaller planes leave most of a
// workgroup idle: AlexNet's 13 x 13 pool5 ran at half the speed that way).
constexpr size_t kPlaneLds = 48 * 1024;
constexpr long long kPlaneMin = 512;

unsigned pool_grid(uint32_t total)
{
    uint32_t b = (total + 255) / 256;
    return b < 65536u ? b : 65536u;
}

}  // namespace

hipError_t launch_pool_fwd(bool max_mode, const float *x, float *y, int *mask, int N, int C, int H,
                           int W, int R, int S, int stride, int pad, int P, int Q,
                           hipStream_t stream)
{
    const uint32_t total = (uint32_t)((long long)N * C * P * Q);
    const uint32_t planes = (uint32_t)((long long)N * C);
    const size_t lds = (size_t)H * W * sizeof(float);
    if (lds <= kPlaneLds && (long long)H * W >= kPlaneMin) {
        const dim3 grid(planes < 1048576u ? planes : 1048576u);
        if (max_mode)
            hipLaunchKernelGGL(pool_fwd_plane_kernel<true>, grid, dim3(256), lds, stream, x, y,
                               mask, H, W, R, S, stride, pad, make_fastdiv(Q), (uint32_t)P,
                               planes);
        else
            hipLaunchKernelGGL(pool_fwd_plane_kernel<false>, grid, dim3(256), lds, stream, x, y,
                               nullptr, H, W, R, S, stride, pad, make_fastdiv(Q), (uint32_t)P,
                               planes);
        return hipGetLastError();
    }
    if (max_mode)
        hipLaunchKernelGGL(pool_fwd_kernel<true>, dim3(pool_grid(total)), dim3(256), 0, stream, x,
                           y, mask, H, W, R, S, stride, pad, make_fastdiv(P * Q),
                           make_fastdiv(Q), total);
    else
        hipLaunchKernelGGL(pool_fwd_kernel<false>, dim3(pool_grid(total)), dim3(256), 0, stream,
                           x, y, nullptr, H, W, R, S, stride, pad, make_fastdiv(P * Q),
                           make_fastdiv(Q), total);
    return hipGetLastError();
}

hipError_t launch_pool_bwd(bool max_mode, const float *dy, const int *mask, float *dx, int N,
                           int C, int H, int W, int R, int S, int stride, int pad, int P, int Q,
                           hipStream_t stream)
{
    const uint32_t total = (uint32_t)((long long)N * C * H * W);
    const uint32_t planes = (uint32_t)((long long)N * C);
    const size_t lds = (size_t)P * Q * (max_mode ? 2 : 1) * sizeof(float);
    if (lds <= kPlaneLds && (long long)H * W >= kPlaneMin && W <= 256) {
        const dim3 grid(planes < 1048576u ? planes : 1048576u);
        if (max_mode)
            hipLaunchKernelGGL(pool_bwd_plane_kernel<true>, grid, dim3(256), lds, stream, dy, mask,
                               dx, H, W, P, Q, R, S, stride, pad, make_fastdiv(W),
                               make_fastdiv(stride), planes);
        else
            hipLaunchKernelGGL(pool_bwd_plane_kernel<false>, grid, dim3(256), lds, stream, dy,
                               nullptr, dx, H, W, P, Q, R, S, stride, pad, make_fastdiv(W),
                               make_fastdiv(stride), planes);
        return hipGetLastError();
    }
    if (max_mode)
        hipLaunchKernelGGL(pool_bwd_kernel<true>, dim3(pool_grid(total)), dim3(256), 0, stream,
                           dy, mask, dx, H, W, P, Q, R, S, stride, pad, make_fastdiv(H * W),
                           make_fastdiv(W), make_fastdiv(stride), total);
    else
        hipLaunchKernelGGL(pool_bwd_kernel<false>, dim3(pool_grid(total)), dim3(256), 0, stream,
                           dy, nullptr, dx, H, W, P, Q, R, S, stride, pad, make_fastdiv(H * W),
                           make_fastdiv(W), make_fastdiv(stride), total);
    return hipGetLastError();
}

}  // namespace miconv
