// Measured reference points of the GPU for the benchmark's roofline (the
// vendor peaks are datasheet figures): the fp32 matrix-core rate reachable by
// a register-only v_mfma_f32_16x16x4f32 loop, the HBM bandwidth of a plain
// device copy, and the shader clock the matrix loop ran at.  Declared in
// include/mipeak.h; a separate library from the convolution passes.
#include <stdint.h>
#include <hip/hip_runtime.h>

#include "mipeak.h"

namespace {

typedef float f32x4 __attribute__((ext_vector_type(4)));

// Each wave runs `iters` rounds of NCH independent accumulator chains (so
// that the matrix pipe never waits for a previous result), then folds its
// accumulators into sink[wave] so that nothing is optimised away.  Lane 0
// records the shader-clock counter (s_memtime) and the constant 100 MHz
// counter (s_memrealtime) around the loop.
template <int NCH>
__global__ void mfma_loop_kernel(int iters, float *sink, unsigned long long *clocks)
{
    const int lane = threadIdx.x & 63;
    const int wave = blockIdx.x * (blockDim.x >> 6) + (threadIdx.x >> 6);
    float a = 1.0f + 1e-7f * lane, b = 1.0f - 1e-7f * lane;
    f32x4 acc[NCH];
#pragma unroll
    for (int c = 0; c < NCH; c++)
        acc[c] = f32x4{0.f, 0.f, 0.f, 0.f};
    const unsigned long long t0 = clock64(), w0 = wall_clock64();
    for (int i = 0; i < iters; i++) {
#pragma unroll
        for (int c = 0; c < NCH; c++)
            acc[c] = __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, acc[c], 0, 0, 0);
    }
    const unsigned long long t1 = clock64(), w1 = wall_clock64();
    float s = 0.f;
#pragma unroll
    for (int c = 0; c < NCH; c++)
        s += acc[c][0] + acc[c][1] + acc[c][2] + acc[c][3];
    sink[(long long)wave * 64 + lane] = s;
    if (lane == 0 && clocks) {
        clocks[2 * wave] = t1 - t0;
        clocks[2 * wave + 1] = w1 - w0;
    }
}

// Grid-stride copy of 16-byte elements.
__global__ __launch_bounds__(256) void copy_kernel(const float4 *__restrict__ src,
                                                   float4 *__restrict__ dst, long long n)
{
    for (long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x; i < n;
         i += (long long)gridDim.x * blockDim.x)
        dst[i] = src[i];
}

}  // namespace

extern "C" {

int peak_mfma_f32(int blocks, int waves, int iters, int chains, float *sink,
                  unsigned long long *clocks, hipStream_t stream)
{
    if (blocks < 1 || waves < 1 || waves > 16 || iters < 1 || !sink)
        return -1;
    if (chains != 4 && chains != 8 && chains != 16)
        return -1;
    dim3 grid(blocks), block(64 * waves);
    switch (chains) {
    case 4: hipLaunchKernelGGL(mfma_loop_kernel<4>, grid, block, 0, stream, iters, sink, clocks); break;
    case 8: hipLaunchKernelGGL(mfma_loop_kernel<8>, grid, block, 0, stream, iters, sink, clocks); break;
    default: hipLaunchKernelGGL(mfma_loop_kernel<16>, grid, block, 0, stream, iters, sink, clocks); break;
    }
    return hipGetLastError() == hipSuccess ? 0 : -2;
}

int peak_copy(const void *src, void *dst, size_t bytes, int blocks, hipStream_t stream)
{
    if (!src || !dst || bytes % 16 || ((uintptr_t)src | (uintptr_t)dst) % 16 || blocks < 1)
        return -1;
    const long long n = (long long)(bytes / 16);
    hipLaunchKernelGGL(copy_kernel, dim3(blocks), dim3(256), 0, stream, (const float4 *)src,
                       (float4 *)dst, n);
    return hipGetLastError() == hipSuccess ? 0 : -2;
}

}  // extern "C"
