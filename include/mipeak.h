/*
 * mipeak: measured reference points for the convolution benchmark's
 * roofline on an AMD Instinct MI355X (gfx950).  The roofline of a pass
 * (flops over the fp32 matrix peak, or bytes over the HBM bandwidth) uses the
 * vendor's datasheet peaks; these two kernels measure what the chip sustains
 * next to them.  Not part of the convolution library (include/miconv.h).
 *
 * Both calls take caller-owned device buffers, enqueue one kernel on
 * `stream` (NULL = the null stream) and return without synchronising:
 * 0 on success, -1 for an invalid argument (nothing launched), -2 if the
 * launch reported an error.
 */
#ifndef MIPEAK_H
#define MIPEAK_H

#include <stddef.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

/*
 * fp32 matrix-core loop: `blocks` workgroups of `waves` waves (1..16), each
 * wave running `iters` rounds of `chains` (4, 8 or 16) independent
 * v_mfma_f32_16x16x4f32 accumulations, i.e.
 *   flops = blocks * waves * iters * chains * 2048.
 * sink receives blocks * waves * 64 floats (the folded accumulators, so that
 * nothing is optimised away).  clocks (may be NULL) receives, per wave w,
 * clocks[2w] = shader-clock cycles of the loop and clocks[2w + 1] = ticks of
 * the constant 100 MHz counter over the same loop (their ratio x 100 MHz is
 * the shader clock the loop ran at).
 */
int peak_mfma_f32(int blocks, int waves, int iters, int chains, float *sink,
                  unsigned long long *clocks, hipStream_t stream);

/*
 * Device copy of `bytes` (a multiple of 16; both pointers 16-byte aligned)
 * from src to dst by `blocks` workgroups of 256 threads, 16 bytes per thread
 * and step; the HBM traffic is 2 * bytes.
 */
int peak_copy(const void *src, void *dst, size_t bytes, int blocks, hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* MIPEAK_H */
