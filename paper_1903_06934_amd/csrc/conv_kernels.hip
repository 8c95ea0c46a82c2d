// HIP kernels for gfx950 (CDNA4): implicit-GEMM convolution passes on fp32
// MFMA, filter packing, split-K reduction and the bias gradient.
//
// GEMM core: a workgroup of WM x WN waves computes a BM x BN tile of C with
// v_mfma_f32_32x32x2f32 (each wave owns a (BM/WM) x (BN/WN) sub-tile made of
// 32x32 accumulator blocks).  The reduction dimension is walked in BK-deep
// slices that are staged through LDS in a double buffer: while the MFMAs
// consume slice t from LDS, the global loads of slice t+1 are in flight in
// registers; one barrier per slice.  LDS holds both operands k-major
// (As[k][m], Bs[k][n]) so that the 32 lanes of an MFMA operand read 32
// consecutive words.
#include "internal.h"

namespace miconv {

typedef float f32x16 __attribute__((ext_vector_type(16)));

// v_mfma_f32_32x32x2f32 operand layout (64 lanes):
//   A (32 x 2): lane l holds A[l % 32][l / 32];  B (2 x 32): B[l / 32][l % 32]
//   D (32 x 32): lane l, register v holds D[8 (v / 4) + 4 (l / 32) + v % 4][l % 32]
__device__ __forceinline__ int acc_row(int v, int lane)
{
    return 8 * (v >> 2) + 4 * (lane >> 5) + (v & 3);
}

template <int BM, int BN, int BK, int WM, int WN, int LDA, int LDB>
__device__ __forceinline__ void mfma_slice(const float (*As)[LDA], const float (*Bs)[LDB],
                                           f32x16 (&acc)[BM / WM / 32][BN / WN / 32],
                                           int lane, int wm, int wn)
{
    constexpr int FM = BM / WM / 32, FN = BN / WN / 32;
    const int kr = lane >> 5, lc = lane & 31;
#pragma unroll
    for (int kk = 0; kk < BK; kk += 2) {
        float af[FM], bf[FN];
#pragma unroll
        for (int i = 0; i < FM; i++)
            af[i] = As[kk + kr][wm * (BM / WM) + i * 32 + lc];
#pragma unroll
        for (int j = 0; j < FN; j++)
            bf[j] = Bs[kk + kr][wn * (BN / WN) + j * 32 + lc];
#pragma unroll
        for (int i = 0; i < FM; i++)
#pragma unroll
            for (int j = 0; j < FN; j++)
                acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(af[i], bf[j], acc[i][j], 0, 0, 0);
    }
}

// ---------------------------------------------------------------------------
// Forward / backward-data implicit GEMM (see ImgGemmArgs).
// FAST: cin % BK == 0, so every BK slice of the reduction lies inside one
// filter tap and the tap's (tr, ts) and the spatial bounds test are uniform
// over the slice; otherwise each element decodes its own (tap, channel).
// ---------------------------------------------------------------------------
template <int BM, int BN, int BK, int WM, int WN, bool FAST>
__global__ __launch_bounds__(64 * WM * WN) void img_gemm_kernel(const ImgGemmArgs a)
{
    constexpr int NT = 64 * WM * WN;
    constexpr int FM = BM / WM / 32, FN = BN / WN / 32;
    constexpr int APT = BM * BK / NT, BPT = BN * BK / NT;
    constexpr int AKS = NT / BM, BKS = NT / BN;
    constexpr int LDA = BM, LDB = BN;
    static_assert(NT % BM == 0 && NT % BN == 0, "loader mapping");
    static_assert(APT * AKS == BK && BPT * BKS == BK, "loader mapping");

    __shared__ float As[2][BK][LDA];
    __shared__ float Bs[2][BK][LDB];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave % WM, wn = wave / WM;
    const int g = blockIdx.z;
    const int mtiles = (a.M + BM - 1) / BM;
    const int mt = blockIdx.x % mtiles, nt = blockIdx.x / mtiles;
    const int m0 = mt * BM, n0 = nt * BN;

    // A loader: thread -> (m = tid % BM, k = tid / BM + AKS * i); coalesced along m.
    const int a_m = tid % BM, a_k = tid / BM;
    const bool a_mok = m0 + a_m < a.M;
    const float *Ag = a.A + (long long)g * a.a_gstride + m0 + a_m;

    // B loader: thread -> (n = tid % BN, k = tid / BN + BKS * i); coalesced along n.
    const int b_n = tid % BN, b_k = tid / BN;
    const int col = n0 + b_n;
    const bool colok = col < a.Ncol;
    int hb = 0, wb = 0;
    const float *sb = a.src;
    {
        uint32_t c = colok ? (uint32_t)col : 0u;
        uint32_t img = fast_div(c, a.col_hw);
        uint32_t rem = c - img * a.col_hw.d;
        uint32_t ci = fast_div(rem, a.col_w);
        uint32_t cj = rem - ci * a.col_w.d;
        hb = (int)ci * a.cstep + a.coff_h;
        wb = (int)cj * a.cstep + a.coff_w;
        sb = a.src + (long long)img * a.src_img_stride + (long long)g * a.cin * a.src_hw;
    }

    float ra[APT], rb[BPT];

    auto load_slice = [&](int k0) {
#pragma unroll
        for (int i = 0; i < APT; i++) {
            int k = k0 + a_k + AKS * i;
            ra[i] = (a_mok && k < a.Kred) ? Ag[(long long)k * a.M] : 0.f;
        }
        if constexpr (FAST) {
            uint32_t tap = fast_div((uint32_t)k0, a.k_cin);
            int ch0 = k0 - (int)(tap * a.k_cin.d);
            uint32_t tr = fast_div(tap, a.k_tw);
            int ts = (int)(tap - tr * a.k_tw.d);
            int hy = hb + a.tsign * (int)tr, wx = wb + a.tsign * ts;
            bool ok = colok && (unsigned)hy < (unsigned)a.src_h && (unsigned)wx < (unsigned)a.src_w;
            long long off = (long long)(ch0 + b_k) * a.src_hw + (long long)hy * a.src_w + wx;
#pragma unroll
            for (int i = 0; i < BPT; i++)
                rb[i] = ok ? sb[off + (long long)(BKS * i) * a.src_hw] : 0.f;
        } else {
#pragma unroll
            for (int i = 0; i < BPT; i++) {
                int k = k0 + b_k + BKS * i;
                uint32_t kc = k < a.Kred ? (uint32_t)k : 0u;
                uint32_t tap = fast_div(kc, a.k_cin);
                int ch = (int)(kc - tap * a.k_cin.d);
                uint32_t tr = fast_div(tap, a.k_tw);
                int ts = (int)(tap - tr * a.k_tw.d);
                int hy = hb + a.tsign * (int)tr, wx = wb + a.tsign * ts;
                bool ok = colok && k < a.Kred && (unsigned)hy < (unsigned)a.src_h &&
                          (unsigned)wx < (unsigned)a.src_w;
                rb[i] = ok ? sb[(long long)ch * a.src_hw + (long long)hy * a.src_w + wx] : 0.f;
            }
        }
    };
    auto store_slice = [&](int buf) {
#pragma unroll
        for (int i = 0; i < APT; i++)
            As[buf][a_k + AKS * i][a_m] = ra[i];
#pragma unroll
        for (int i = 0; i < BPT; i++)
            Bs[buf][b_k + BKS * i][b_n] = rb[i];
    };

    f32x16 acc[FM][FN];
#pragma unroll
    for (int i = 0; i < FM; i++)
#pragma unroll
        for (int j = 0; j < FN; j++)
#pragma unroll
            for (int v = 0; v < 16; v++)
                acc[i][j][v] = 0.f;

    const int nslices = (a.Kred + BK - 1) / BK;
    if (nslices > 0) {
        load_slice(0);
        store_slice(0);
    }
    __syncthreads();
    for (int t = 0; t < nslices; t++) {
        const int buf = t & 1;
        if (t + 1 < nslices)
            load_slice((t + 1) * BK);
        mfma_slice<BM, BN, BK, WM, WN, LDA, LDB>(As[buf], Bs[buf], acc, lane, wm, wn);
        if (t + 1 < nslices)
            store_slice(buf ^ 1);
        __syncthreads();
    }

    // Epilogue: + bias, scatter columns back to image coordinates.
    long long obase[FN];
    bool nok[FN];
#pragma unroll
    for (int j = 0; j < FN; j++) {
        int n = n0 + wn * (BN / WN) + j * 32 + (lane & 31);
        nok[j] = n < a.Ncol;
        uint32_t c = nok[j] ? (uint32_t)n : 0u;
        uint32_t img = fast_div(c, a.col_hw);
        uint32_t rem = c - img * a.col_hw.d;
        uint32_t ci = fast_div(rem, a.col_w);
        uint32_t cj = rem - ci * a.col_w.d;
        obase[j] = (long long)img * a.out_img_stride +
                   (long long)((int)ci * a.ostep + a.ooff_h) * a.out_w + ((int)cj * a.ostep + a.ooff_w);
    }
#pragma unroll
    for (int i = 0; i < FM; i++)
#pragma unroll
        for (int v = 0; v < 16; v++) {
            int m = m0 + wm * (BM / WM) + i * 32 + acc_row(v, lane);
            if (m >= a.M)
                continue;
            int oc = g * a.M + m;
            float bv = a.bias ? a.bias[oc] : 0.f;
            long long choff = (long long)oc * a.out_hw;
#pragma unroll
            for (int j = 0; j < FN; j++)
                if (nok[j])
                    a.out[obase[j] + choff] = acc[i][j][v] + bv;
        }
}

// ---------------------------------------------------------------------------
// Backward-weight GEMM (see WgradArgs).  The reduction runs over pixels, so
// both operands are loaded with lanes along the pixel index (coalesced along
// q) and transposed into the k-major LDS tiles; the per-column filter tap
// decode (c, r, s) is computed once per workgroup into an LDS table.
// ---------------------------------------------------------------------------
template <int BM, int BN, int BK, int WM, int WN>
__global__ __launch_bounds__(64 * WM * WN) void wgrad_gemm_kernel(const WgradArgs a)
{
    constexpr int NT = 64 * WM * WN;
    constexpr int FM = BM / WM / 32, FN = BN / WN / 32;
    constexpr int RS = NT / BK;  // rows covered per loader pass
    constexpr int APT = BM / RS, BPT = BN / RS;
    constexpr int LDA = BM + 4, LDB = BN + 4;
    static_assert(NT % BK == 0 && BM % RS == 0 && BN % RS == 0, "loader mapping");

    __shared__ float As[2][BK][LDA];
    __shared__ float Bs[2][BK][LDB];
    __shared__ int2 ctab[BN];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave % WM, wn = wave / WM;
    const int g = blockIdx.z, split = blockIdx.y;
    const int mtiles = (a.M + BM - 1) / BM;
    const int mt = blockIdx.x % mtiles, nt = blockIdx.x / mtiles;
    const int m0 = mt * BM, n0 = nt * BN;
    const int kbeg = split * a.chunk;
    const int kend = min(a.Kred, kbeg + a.chunk);

    for (int n = tid; n < BN; n += NT) {
        int col = n0 + n;
        int2 e = make_int2(-1, 0);
        if (col < a.Ncol) {
            uint32_t c = fast_div((uint32_t)col, a.n_rs);
            uint32_t rs = col - c * a.n_rs.d;
            uint32_t r = fast_div(rs, a.n_s);
            uint32_t s = rs - r * a.n_s.d;
            e = make_int2((int)(c * a.HW + r * a.W + s), (int)((r << 16) | s));
        }
        ctab[n] = e;
    }
    __syncthreads();

    // Loader: thread -> (pixel kk = tid % BK, row = tid / BK + RS * i).
    const int kk = tid % BK, rrow = tid / BK;
    const float *dyg = a.dy + (long long)g * a.Kg * a.PQ;
    const float *xg = a.x + (long long)g * a.Cg * a.HW;
    int2 ce[BPT];
#pragma unroll
    for (int i = 0; i < BPT; i++)
        ce[i] = ctab[rrow + RS * i];

    float ra[APT], rb[BPT];
    auto load_slice = [&](int k0) {
        int pix = k0 + kk;
        bool ok = pix < kend;
        uint32_t pc = ok ? (uint32_t)pix : 0u;
        uint32_t img = fast_div(pc, a.pix_pq);
        uint32_t pq = pc - img * a.pix_pq.d;
        uint32_t p = fast_div(pq, a.pix_q);
        uint32_t q = pq - p * a.pix_q.d;
        long long abase = (long long)img * a.K * a.PQ + pq;
#pragma unroll
        for (int i = 0; i < APT; i++) {
            int m = m0 + rrow + RS * i;
            ra[i] = (ok && m < a.M) ? dyg[abase + (long long)m * a.PQ] : 0.f;
        }
        int h0 = (int)p * a.stride - a.pad, w0 = (int)q * a.stride - a.pad;
        long long xbase = (long long)img * a.C * a.HW + (long long)h0 * a.W + w0;
#pragma unroll
        for (int i = 0; i < BPT; i++) {
            int r = ce[i].y >> 16, s = ce[i].y & 0xffff;
            bool okb = ok && ce[i].x >= 0 && (unsigned)(h0 + r) < (unsigned)a.H &&
                       (unsigned)(w0 + s) < (unsigned)a.W;
            rb[i] = okb ? xg[xbase + ce[i].x] : 0.f;
        }
    };
    auto store_slice = [&](int buf) {
#pragma unroll
        for (int i = 0; i < APT; i++)
            As[buf][kk][rrow + RS * i] = ra[i];
#pragma unroll
        for (int i = 0; i < BPT; i++)
            Bs[buf][kk][rrow + RS * i] = rb[i];
    };

    f32x16 acc[FM][FN];
#pragma unroll
    for (int i = 0; i < FM; i++)
#pragma unroll
        for (int j = 0; j < FN; j++)
#pragma unroll
            for (int v = 0; v < 16; v++)
                acc[i][j][v] = 0.f;

    const int nslices = kend > kbeg ? (kend - kbeg + BK - 1) / BK : 0;
    if (nslices > 0) {
        load_slice(kbeg);
        store_slice(0);
    }
    __syncthreads();
    for (int t = 0; t < nslices; t++) {
        const int buf = t & 1;
        if (t + 1 < nslices)
            load_slice(kbeg + (t + 1) * BK);
        mfma_slice<BM, BN, BK, WM, WN, LDA, LDB>(As[buf], Bs[buf], acc, lane, wm, wn);
        if (t + 1 < nslices)
            store_slice(buf ^ 1);
        __syncthreads();
    }

    float *outg = a.out + (long long)split * a.split_stride + (long long)g * a.M * a.Ncol;
#pragma unroll
    for (int i = 0; i < FM; i++)
#pragma unroll
        for (int v = 0; v < 16; v++) {
            int m = m0 + wm * (BM / WM) + i * 32 + acc_row(v, lane);
            if (m >= a.M)
                continue;
#pragma unroll
            for (int j = 0; j < FN; j++) {
                int n = n0 + wn * (BN / WN) + j * 32 + (lane & 31);
                if (n < a.Ncol)
                    outg[(long long)m * a.Ncol + n] = acc[i][j][v];
            }
        }
}

// ---------------------------------------------------------------------------
// Filter packing.
// ---------------------------------------------------------------------------
__global__ void pack_fwd_kernel(const float *__restrict__ w, float *__restrict__ wp, int Kg,
                                int Cg, int R, int S, long long total)
{
    long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= total)
        return;
    // i = ((g * R*S*Cg) + (r*S + s)*Cg + c) * Kg + k
    int k = (int)(i % Kg);
    long long t = i / Kg;
    int c = (int)(t % Cg);
    t /= Cg;
    int rs = (int)(t % (R * S));
    int g = (int)(t / (R * S));
    int r = rs / S, s = rs % S;
    wp[i] = w[(((long long)(g * Kg + k) * Cg + c) * R + r) * S + s];
}

__global__ void pack_bwd_phase_kernel(const float *__restrict__ w, float *__restrict__ wr,
                                      int Kg, int Cg, int R, int S, int r0, int s0, int nr,
                                      int ns, int stride, long long total)
{
    long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= total)
        return;
    // i = ((g * nr*ns + rr*ns + ss) * Kg + k) * Cg + c
    int c = (int)(i % Cg);
    long long t = i / Cg;
    int k = (int)(t % Kg);
    t /= Kg;
    int tap = (int)(t % (nr * ns));
    int g = (int)(t / (nr * ns));
    int r = r0 + stride * (tap / ns), s = s0 + stride * (tap % ns);
    wr[i] = w[(((long long)(g * Kg + k) * Cg + c) * R + r) * S + s];
}

// ---------------------------------------------------------------------------
// Deterministic split-K reduction: fixed order over splits.
// ---------------------------------------------------------------------------
__global__ void splitk_reduce_kernel(const float *__restrict__ part, int nsplit,
                                     long long stride, long long count, float *__restrict__ out)
{
    for (long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x; i < count;
         i += (long long)gridDim.x * blockDim.x) {
        float s = part[i];
        for (int k = 1; k < nsplit; k++)
            s += part[(long long)k * stride + i];
        out[i] = s;
    }
}

// ---------------------------------------------------------------------------
// Bias gradient, stage 1: workgroup (k = blockIdx.x, chunk j = blockIdx.y)
// sums dy[img][k][pq] over flat positions e = img*PQ + pq in its chunk.
// Each thread sums a strided sequence, then a fixed butterfly over the
// wavefront and a fixed-order sum over the waves: deterministic.
// ---------------------------------------------------------------------------
constexpr int BIAS_NT = 256;

__device__ __forceinline__ float wave_sum(float v)
{
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1)
        v += __shfl_xor(v, off, 64);
    return v;
}

__global__ __launch_bounds__(BIAS_NT) void bias_grad_partial_kernel(
    const float *__restrict__ dy, int N, int K, int PQ, int nchunk, float *__restrict__ part)
{
    __shared__ float wsum[BIAS_NT / 64];
    const int k = blockIdx.x, j = blockIdx.y;
    const long long total = (long long)N * PQ;
    const long long per = (total + nchunk - 1) / nchunk;
    const long long e0 = (long long)j * per;
    const long long e1 = min(total, e0 + per);
    float s = 0.f;
    for (long long e = e0 + threadIdx.x; e < e1; e += BIAS_NT) {
        long long img = e / PQ, pq = e - img * PQ;
        s += dy[(img * K + k) * PQ + pq];
    }
    s = wave_sum(s);
    if ((threadIdx.x & 63) == 0)
        wsum[threadIdx.x >> 6] = s;
    __syncthreads();
    if (threadIdx.x == 0) {
        float t = wsum[0];
        for (int i = 1; i < BIAS_NT / 64; i++)
            t += wsum[i];
        part[(long long)k * nchunk + j] = t;
    }
}

__global__ void bias_grad_final_kernel(const float *__restrict__ part, int K, int nchunk,
                                       float *__restrict__ db)
{
    int k = blockIdx.x * blockDim.x + threadIdx.x;
    if (k >= K)
        return;
    float s = part[(long long)k * nchunk];
    for (int j = 1; j < nchunk; j++)
        s += part[(long long)k * nchunk + j];
    db[k] = s;
}

// ---------------------------------------------------------------------------
// Launchers.
// ---------------------------------------------------------------------------
template <int BM, int BN, int BK, int WM, int WN, bool FAST>
static hipError_t img_launch(const ImgGemmArgs &a, int groups, hipStream_t stream)
{
    int tiles = ((a.M + BM - 1) / BM) * ((a.Ncol + BN - 1) / BN);
    dim3 grid(tiles, 1, groups);
    hipLaunchKernelGGL((img_gemm_kernel<BM, BN, BK, WM, WN, FAST>), grid, dim3(64 * WM * WN), 0,
                       stream, a);
    return hipGetLastError();
}

hipError_t launch_img_gemm(const ImgGemmArgs &a, int groups, int tile, bool fast,
                           hipStream_t stream)
{
    if (tile == TILE_128x128)
        return fast ? img_launch<128, 128, 16, 2, 2, true>(a, groups, stream)
                    : img_launch<128, 128, 16, 2, 2, false>(a, groups, stream);
    return fast ? img_launch<64, 64, 16, 2, 2, true>(a, groups, stream)
                : img_launch<64, 64, 16, 2, 2, false>(a, groups, stream);
}

template <int BM, int BN, int BK, int WM, int WN>
static hipError_t wgrad_launch(const WgradArgs &a, int groups, int nsplit, hipStream_t stream)
{
    int tiles = ((a.M + BM - 1) / BM) * ((a.Ncol + BN - 1) / BN);
    dim3 grid(tiles, nsplit, groups);
    hipLaunchKernelGGL((wgrad_gemm_kernel<BM, BN, BK, WM, WN>), grid, dim3(64 * WM * WN), 0,
                       stream, a);
    return hipGetLastError();
}

hipError_t launch_wgrad_gemm(const WgradArgs &a, int groups, int nsplit, int tile,
                             hipStream_t stream)
{
    if (tile == TILE_128x128)
        return wgrad_launch<128, 128, 16, 2, 2>(a, groups, nsplit, stream);
    return wgrad_launch<64, 64, 16, 2, 2>(a, groups, nsplit, stream);
}

static unsigned blocks_for(long long total, int nt)
{
    return (unsigned)((total + nt - 1) / nt);
}

hipError_t launch_pack_fwd(const float *w, float *wp, int K, int Cg, int R, int S, int G,
                           hipStream_t stream)
{
    long long total = (long long)K * Cg * R * S;
    hipLaunchKernelGGL(pack_fwd_kernel, dim3(blocks_for(total, 256)), dim3(256), 0, stream, w,
                       wp, K / G, Cg, R, S, total);
    return hipGetLastError();
}

hipError_t launch_pack_bwd_phase(const float *w, float *wr, int K, int Cg, int R, int S,
                                 int G, int r0, int s0, int nr, int ns, int stride,
                                 hipStream_t stream)
{
    long long total = (long long)K * Cg * nr * ns;
    if (total == 0)
        return hipSuccess;
    hipLaunchKernelGGL(pack_bwd_phase_kernel, dim3(blocks_for(total, 256)), dim3(256), 0,
                       stream, w, wr, K / G, Cg, R, S, r0, s0, nr, ns, stride, total);
    return hipGetLastError();
}

hipError_t launch_splitk_reduce(const float *part, int nsplit, long long stride,
                                long long count, float *out, hipStream_t stream)
{
    long long blocks = (count + 255) / 256;
    if (blocks > 65536)
        blocks = 65536;
    hipLaunchKernelGGL(splitk_reduce_kernel, dim3((unsigned)blocks), dim3(256), 0, stream, part,
                       nsplit, stride, count, out);
    return hipGetLastError();
}

hipError_t launch_bias_grad(const float *dy, int N, int K, int PQ, int nchunk, float *part,
                            float *db, hipStream_t stream)
{
    hipLaunchKernelGGL(bias_grad_partial_kernel, dim3(K, nchunk), dim3(BIAS_NT), 0, stream, dy,
                       N, K, PQ, nchunk, part);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess)
        return e;
    hipLaunchKernelGGL(bias_grad_final_kernel, dim3((K + 255) / 256), dim3(256), 0, stream, part,
                       K, nchunk, db);
    return hipGetLastError();
}

}  // namespace miconv
