"""ctypes binding of libmipeak.so (include/mipeak.h): the measured reference
points of the benchmark's roofline.  Argument marshalling and event timing
only; both measurements run in the library's HIP kernels."""
from __future__ import annotations

import ctypes
import os

PKG = os.path.dirname(os.path.abspath(__file__))
LIBRARY = os.path.join(PKG, "libmipeak.so")

_lib = None


def lib():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIBRARY):
        raise RuntimeError(f"{LIBRARY} is not built; run paper_1903_06934_amd.build.build()")
    import torch  # noqa: F401  (its HIP runtime serves the library too)
    L = ctypes.CDLL(LIBRARY)
    I, P = ctypes.c_int, ctypes.c_void_p
    L.peak_mfma_f32.argtypes = [I, I, I, I, P, P, P]
    L.peak_mfma_f32.restype = I
    L.peak_copy.argtypes = [P, P, ctypes.c_size_t, I, P]
    L.peak_copy.restype = I
    _lib = L
    return L


def _timed(launch, reps):
    """Median device ms of launch() over reps, torch events on the current stream."""
    import statistics
    import torch
    ts = []
    for _ in range(reps):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        launch()
        b.record()
        b.synchronize()
        ts.append(a.elapsed_time(b))
    return statistics.median(ts)


def mfma_f32(waves_per_simd, cus, chains=8, iters=20000, reps=5):
    """fp32 matrix-core rate of a register-only v_mfma_f32_16x16x4f32 loop with
    `waves_per_simd` waves on each of the 4 SIMDs of `cus` CUs (one workgroup
    of 4 * waves_per_simd waves per CU, at most 16 waves a workgroup): returns
    (TFLOP/s, shader GHz measured over the loop)."""
    import torch
    waves = 4 * waves_per_simd
    per_block = min(waves, 16)
    blocks = cus * (waves // per_block)
    nw = blocks * per_block
    sink = torch.empty(nw * 64, dtype=torch.float32, device="cuda")
    clocks = torch.zeros(2 * nw, dtype=torch.int64, device="cuda")
    stream = torch.cuda.current_stream().cuda_stream
    L = lib()

    def launch():
        st = L.peak_mfma_f32(blocks, per_block, iters, chains, sink.data_ptr(),
                             clocks.data_ptr(), stream)
        if st != 0:
            raise RuntimeError(f"peak_mfma_f32 failed ({st})")

    launch()  # warm-up (clocks ramp up)
    ms = _timed(launch, reps)
    c = clocks.view(-1, 2).double()
    ghz = float((c[:, 0] / c[:, 1].clamp(min=1)).median()) * 0.1
    flops = float(nw) * iters * chains * 2048
    return flops / ms / 1e9, ghz


def copy_gbs(nbytes=1 << 30, blocks=None, reps=5):
    """HBM bandwidth of a device copy of nbytes (read + write bytes / time)."""
    import torch
    src = torch.ones(nbytes // 4, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    props = torch.cuda.get_device_properties(0)
    nblk = blocks or 8 * props.multi_processor_count
    stream = torch.cuda.current_stream().cuda_stream
    L = lib()

    def launch():
        st = L.peak_copy(src.data_ptr(), dst.data_ptr(), nbytes, nblk, stream)
        if st != 0:
            raise RuntimeError(f"peak_copy failed ({st})")

    launch()
    ms = _timed(launch, reps)
    ok = bool(torch.equal(src[:1024], dst[:1024]) and torch.equal(src[-1024:], dst[-1024:]))
    del src, dst
    return 2.0 * nbytes / ms / 1e6, ok
