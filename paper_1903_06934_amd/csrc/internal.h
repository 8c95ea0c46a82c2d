// Internal declarations shared by the C-ABI layer (api.hip) and the kernels
// (conv_kernels.hip).  Not installed; the public interface is miconv.h.
#pragma once

#include <stdint.h>
#include <hip/hip_runtime.h>

namespace miconv {

// Division by a run-time constant d (1 <= d < 2^31) for dividends n < 2^31:
// q = (mulhi(n, mul) + n) >> shift, with shift = ceil(log2 d) and
// mul = floor(2^32 (2^shift - d) / d) + 1 (Granlund & Montgomery, 1994).
struct FastDiv {
    uint32_t mul;
    uint32_t shift;
    uint32_t d;
};

__host__ __device__ inline uint32_t fast_div(uint32_t n, FastDiv f)
{
    uint32_t hi = (uint32_t)(((uint64_t)n * f.mul) >> 32);
    return (hi + n) >> f.shift;
}

FastDiv make_fastdiv(uint32_t d);

// ---------------------------------------------------------------------------
// Implicit GEMM whose columns are pixels of an image-like output and whose
// B operand gathers from an image-like source.  Used for the forward pass
// (source x, columns = output pixels, taps = filter taps) and for each stride
// phase of the backward-data pass (source dy, columns = the input pixels of
// one phase, taps = the filter taps of that phase).
//
// Per group g (folded with the tile and split index into the 1-D grid):
//   out[g] (M x Ncol) = A[g] (M x Kred) * B[g] (Kred x Ncol)
//   A[g][m][k]  = Ap[(g * M + m) * a_ld + k]            (packed m-major), or, for
//                 the tiles of one wave row (img_tile_shares_a), Ap[(g * a_ld + k) * M + m]
//                 (k-major); a_ld = Kred rounded up to a multiple of 16, rows past
//                 Kred zero
//   k           = tap * cin + ch (general), or, when cin % 16 == 0 (FAST),
//                 (cb * taps + tap) * 16 + ci with ch = 16 cb + ci: the taps of a
//                 16-channel block are consecutive, so the source rows a
//                 workgroup re-reads tap after tap stay in cache;
//   tap         = tr * taps_w + ts
//   column n    = (img, ci, cj) over  N x col_h x col_w
//   B[g][k][n]  = src[img][g * cin + ch][hy][wx] or 0 outside the source, with
//                 hy = ci * cstep + coff_h + tsign * tr,
//                 wx = cj * cstep + coff_w + tsign * ts
//   out[img][g * M + m][ci * ostep + ooff_h][cj * ostep + ooff_w] = C + bias
// ---------------------------------------------------------------------------
struct ImgGemmArgs {
    int M, Ncol, Kred, groups;
    const float *A;
    int a_ld;             // packed row length: Kred rounded up to a multiple of 16
    uint32_t a_bytes;     // groups * M * a_ld * 4 (< 2^31)
    const float *src;
    uint32_t src_bytes;   // bytes of the source images this launch reads (< 2^31)
    int cin;              // source channels per group
    int src_h, src_w, src_hw;
    uint32_t src_img_words;  // words per source image
    FastDiv col_hw, col_w;  // d = col_h * col_w, col_w
    int cstep, coff_h, coff_w, tsign;
    FastDiv k_cin, k_tw;    // d = cin, taps_w
    FastDiv k_taps;         // d = taps (FAST order)
    float *out;
    const float *bias;      // may be null
    long long out_img_stride;
    int out_hw, out_w;
    int ostep, ooff_h, ooff_w;
    // Blocked backward-data (mblock = b > 1): row m = (c * b + ph) * b + pw is
    // input channel g * (M / b^2) + c at offset (ph, pw) of column (ci, cj)'s
    // b x b block: out[img][.][ci * ostep + ooff_h + ph][cj * ostep + ooff_w + pw],
    // stored only inside out_h x out_w.  mblock = 0: the row is channel g * M + m.
    int mblock, out_h;
    // Split-K: split s covers reduction rows [s * kchunk, min((s+1) * kchunk, Kred))
    // and, when nsplit > 1, writes its partial sums (no bias) to out + s * split_stride.
    int nsplit, kchunk;
    long long split_stride;
};

// ---------------------------------------------------------------------------
// Halo-staged implicit GEMM for stride-1 R x R layers (R = 3 or 5) with
// channel-aligned slices (the forward pass, or the single stride phase of a
// stride-1 backward-data pass).  Same GEMM as ImgGemmArgs with cstep = 1, but
// the columns of a tile are a TR x TW block of output pixels of one image
// (rows p0 .. p0 + TR - 1, columns q0 .. q0 + TW - 1; column n of the tile is
// (n / TW, n % TW)), TW one of 112, 56, 28, 14 (R = 3) or 28, 14 (R = 5) and
// TR = 112 / TW, and for each 16-channel block the source region all R R taps
// of the block need (the halo) is staged in LDS once:
//   halo[c][i][j] = src[img][g * cin + 16 cb + c][p0 + row0 + i][q0 + col0 + j]
//                   (0 outside the source),
// loaded 4 words per lane (R = 3, TW >= 28: needs col0 and the source width
// to be multiples of 4) or 1 (R = 3, TW = 14, and R = 5).  Tap (r, s) of
// pixel (dr, dq) reads halo[c][dr + rr][dq + slack + ss] with (rr, ss) =
// (r, s), or (R - 1 - r, R - 1 - s) for the backward-data phase (flip; its
// source rows are p + coff_h - r).  The reduction order is the
// channel-block-major one of the packed filter: k = (cb * R R + tap) * 16 + ci.
// ---------------------------------------------------------------------------
struct HaloGemmArgs {
    int M, Kred, groups;
    int R;                     // filter rows = columns: 3 or 5
    const float *A;
    int a_ld;
    uint32_t a_bytes;
    const float *src;
    uint32_t src_bytes;
    int cin;                   // source channels per group (multiple of 16)
    int src_h, src_w, src_hw;
    uint32_t src_img_words;
    int P, Q;                  // output extents (the pixel grid of the columns)
    int TR, TW;                // pixel block of a tile
    int row_blocks, col_segs;  // blocks per image: ceil(P / TR) x ceil(Q / TW)
    int nimg;                  // images of this launch
    int row0, col0, slack;     // halo origin relative to (p0, q0); slack = first tap column
    float *out;
    const float *bias;         // may be null
    long long out_img_stride;
    int out_hw, out_w;
    // Split-K over channel blocks: split s covers blocks [s * cbchunk, ...)
    // and, when nsplit > 1, writes its partial sums (no bias) to
    // out + s * split_stride.
    int nsplit, cbchunk;
    long long split_stride;
    // Wave groups of a workgroup (halo_gemm_kernel KS): 1, or 2 (eight waves,
    // each group of four over half the channel blocks; unsplit plans only).
    int ks;
};

// ---------------------------------------------------------------------------
// Backward-weight GEMM, per split s and group g (both folded into the 1-D grid):
//   out[s][g][m][n] = sum over pixels pix in split s of
//                     dy[img][g*Kg + m][p][q] * x[img][g*Cg + c][p*st - pad + r][q*st - pad + s']
//   m in [0, Kg),  n = c * R * S + r * S + s'  in [0, Cg R S),
//   pix = img * P * Q + p * Q + q in [s * chunk, min((s+1) * chunk, Kred)),
// where img counts from the launch's first image (dy and x point there).
// ---------------------------------------------------------------------------
struct WgradArgs {
    int M, Ncol, Kred, groups, nsplit;
    const float *dy;
    const float *x;
    uint32_t dy_bytes, x_bytes;      // bytes of this launch's images (< 2^31)
    uint32_t dy_img_words, x_img_words;
    int Cg;                          // input channels per group
    int H, W, HW, PQ, stride, pad;
    FastDiv pix_pq, pix_q;  // d = P * Q, Q
    FastDiv n_rs, n_s;      // d = R * S, S
    int chunk;
    float *out;
    long long split_stride;  // G * M * Ncol
    int K;                   // all filters (G * M): the stride of db_part
    float *db_part;          // [split][K] partial bias gradients, or null
};

// ---------------------------------------------------------------------------
// Halo backward-weight for stride-1 3 x 3 layers (channels per group a
// multiple of 16, dy rows a multiple of 4 wide): a workgroup computes all nine
// taps of 64 filters x 16 CT input channels, its reduction running over TR x TW
// pixel blocks of the images (TW = 112, 56, 28 or 14, TR = 112 / TW; the same
// blocks as HaloGemmArgs).  Per block it stages the 64 dy rows of the block
// (dy[img][g Kg + k][p0 .. p0 + TR - 1][q0 .. q0 + TW - 1]) and the x halo of
// its 16 CT channels (rows p0 - pad .., columns q0 - pad ..) in LDS once, then
// runs the nine taps from them.  Split s covers pixel blocks
// [s chunk, (s + 1) chunk) of the nimg x row_blocks x col_segs blocks and
// writes partial sums out[s][g Kg + k][tap][c] (and, for the first channel
// tile, db_part[s][g Kg + k]).
// ---------------------------------------------------------------------------
struct WgradHaloArgs {
    int Kg, Cg, groups, K;
    const float *dy, *x;
    uint32_t dy_bytes, x_bytes;
    uint32_t dy_img_words, x_img_words;
    int H, W, P, Q;
    int TW, CT, row_blocks, col_segs, nimg;  // CT: 16-channel sub-tiles per workgroup (1, 2)
    int db;                   // CT = 2 only: 1 eight waves, two LDS stages; 2 eight waves, one stage
    int row0, col0, slack;    // x halo origin relative to (p0, q0); slack: first tap column
    int chunk, nsplit;        // pixel blocks per split
    float *out;               // [split][K][9][Cg]
    long long split_stride;   // K * Cg * 9
    float *db_part;           // [split][K], or null
};
bool wgrad_halo_supported(int TW, int P, int Q, int W);
hipError_t launch_wgrad_halo(const WgradHaloArgs &a, hipStream_t stream);

// Image-GEMM tile shapes (BM x BN; 4 waves, 3 for 48x64).
enum ImgTile {
    IMG_64x64 = 0, IMG_128x64, IMG_16x128, IMG_32x64, IMG_48x64, IMG_96x64, IMG_96x128,
    IMG_128x128, IMG_64x128
};
// Tiles with one wave row (WM == 1 in launch_img_gemm): every wave needs the
// same filter rows, which the kernel then shares through LDS, packed k-major.
inline bool img_tile_shares_a(int tile) { return tile == IMG_16x128; }
// Backward-weight tiles of the one-pixel-per-lane kernel: tap-uniform
// (BM rows of K/G x BN channels of one tap) or packed (BM rows x BN
// consecutive (c, r, s) columns).
enum WgradTile {
    WG_TAP_64x32 = 0, WG_TAP_64x48, WG_TAP_64x16, WG_PIX_96x64, WG_PIX_64x64, WG_PIX_64x32,
    WG_TAP_128x32, WG_TAP_64x64, WG_TAP_128x64
};
inline bool wgrad_tile_is_tap(int tile) { return tile <= WG_TAP_64x16 || tile >= WG_TAP_128x32; }

hipError_t launch_img_gemm(const ImgGemmArgs &a, int tile, bool fast, hipStream_t stream);
// Halo tiles: BM rows (64 or 128) x 112 columns (TR x TW = 112 pixels), or
// 64 x 176 for a whole 13 x 13 map (3 x 3); flip for the backward-data
// phase.  halo_block_supported: whether TR x TW pixel blocks (112, 56, 28, 14
// wide for R = 3; 28, 14 for R = 5; a whole 13 x 13 map for R = 3) can stage
// this source (16-byte loads need the width and col0 to be multiples of 4);
// halo_load_words: the words per lane and load (4 or 1).
enum HaloTile { HALO_64x112 = 0, HALO_128x112 };
constexpr int kHaloCols = 112;
bool halo_whole_image(int TW, int TR, int R);
bool halo_block_supported(int TW, int TR, int R, int src_w, int col0);
int halo_load_words(int TW, int TR, int R);
hipError_t launch_halo_gemm(const HaloGemmArgs &a, int tile, bool flip, hipStream_t stream);
hipError_t launch_wgrad_gemm(const WgradArgs &a, int tile, hipStream_t stream);

// wp[(g*Kg + k) * a_ld + kk] (or, if kmajor, wp[(g*a_ld + kk) * Kg + k]) =
// w[g*Kg + k][c][r][s] with kk = (r*S + s)*Cg + c, or, if cblock (Cg % 16 == 0),
// kk = ((c / 16) * R*S + r*S + s) * 16 + c % 16; zero for kk >= Cg*R*S.
hipError_t launch_pack_fwd(const float *w, float *wp, int K, int Cg, int R, int S, int G,
                           bool cblock, int a_ld, bool kmajor, hipStream_t stream);
// One stride phase of the backward-data filter: wr[(g*Cg + c) * a_ld + kk] (or, if
// kmajor, wr[(g*a_ld + kk) * Cg + c]) = w[g*Kg + k][c][r0 + st*rr][s0 + st*ss] with
// tap = rr*ns + ss and kk = tap*Kg + k, or, if cblock (Kg % 16 == 0),
// kk = ((k / 16) * nr*ns + tap) * 16 + k % 16; zero for kk >= nr*ns*Kg.
hipError_t launch_pack_bwd_phase(const float *w, float *wr, int K, int Cg, int R, int S,
                                 int G, int r0, int s0, int nr, int ns, int stride,
                                 bool cblock, int a_ld, bool kmajor, hipStream_t stream);
// Blocked backward-data filter (b = stride * f, taps ntr x nts per block):
// wp[(g*M + m) * a_ld + kk] (or, if kmajor, wp[(g*a_ld + kk) * M + m]) with
// M = Cg b^2, m = (c*b + ph)*b + pw, tap = tu*nts + tv and kk = tap*Kg + k, or,
// if cblock (Kg % 16 == 0), kk = ((k / 16) * ntr*nts + tap) * 16 + k % 16:
// w[g*Kg + k][c][ph - stride*(f-1-tu)][pw - stride*(f-1-tv)], zero where that
// tap lies outside the filter and for kk >= ntr*nts*Kg.
hipError_t launch_pack_bwd_block(const float *w, float *wp, int K, int Cg, int R, int S, int G,
                                 int stride, int f, int ntr, int nts, bool cblock, int a_ld,
                                 bool kmajor, hipStream_t stream);
// Explicit plan (im2col / col2im around a 1x1 GEMM).  The column tensor of n
// images is col[n][c'][p][q], c' = (c_all * R + r) * S + s over all C channels
// (group g owns c' in [g (C/G) R S, (g+1) (C/G) R S)), p < P, q < Q:
//   im2col:  col[n][c'][p][q] = x[n][c_all][p st - pad + r][q st - pad + s] (0 outside)
//   col2im:  dx[n][c_all][h][w] = sum over (r, s) in order of col[n][c'][p][q] with
//            h + pad - r = p st, w + pad - s = q st, 0 <= p < P, 0 <= q < Q (0 if none)
// Both need fewer than 2^31 written elements.
hipError_t launch_im2col(const float *x, float *col, int n, int C, int H, int W, int R, int S,
                         int stride, int pad, int P, int Q, hipStream_t stream);
hipError_t launch_col2im(const float *col, float *dx, int n, int C, int H, int W, int R, int S,
                         int stride, int pad, int P, int Q, hipStream_t stream);
// Pooling (max with argmax mask h * W + w within the plane, or average over
// the window clipped to the padded image), forward over N*C*P*Q outputs and
// backward over N*C*H*W inputs (both < 2^31); pad < window.
hipError_t launch_pool_fwd(bool max_mode, const float *x, float *y, int *mask, int N, int C, int H,
                           int W, int R, int S, int stride, int pad, int P, int Q,
                           hipStream_t stream);
hipError_t launch_pool_bwd(bool max_mode, const float *dy, const int *mask, float *dx, int N,
                           int C, int H, int W, int R, int S, int stride, int pad, int P, int Q,
                           hipStream_t stream);
// out[c][r] = in[r][c] for a rows x cols row-major matrix; rows < 65536 * 32.
hipError_t launch_transpose(const float *in, float *out, int rows, int cols, hipStream_t stream);
// Packed reduction-row length of the image GEMM's filter operand.
inline int pad16(int k) { return (k + 15) & ~15; }
// out[dst(i)] = sum over s < nsplit of part[s * stride + i] for i < count, in a
// fixed order; dst = identity, or (tap_cg > 0) [k][tap][c] -> [k][c][tap].
hipError_t launch_splitk_reduce(const float *part, int nsplit, long long stride, int count,
                                float *out, int taps, int tap_cg, hipStream_t stream);
// out[i] = sum over s < nsplit of part[s * stride + i] in a fixed order,
// + bias[(i / hw) % K] if bias is given, for i < count.
hipError_t launch_splitk_bias_reduce(const float *part, int nsplit, long long stride, int count,
                                     const float *bias, int hw, int K, float *out,
                                     hipStream_t stream);

}  // namespace miconv
