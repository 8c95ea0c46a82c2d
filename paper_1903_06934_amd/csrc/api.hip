// C ABI of the convolution library (declared in include/miconv.h): argument
// validation, output geometry, workspace layout, kernel selection and
// launches on the caller's stream.
//
// Layout of this file: geometry and limits; the image-GEMM tile and split
// rules; per pass, its built-in rule, candidate plans, workspace size and
// plan name (forward, backward-data with stride phases or pixel blocks,
// backward-weight, the inner-product and explicit variants); the table of
// stored plan choices; the executors that pack filters and launch kernels;
// pooling; and the extern "C" entry points at the end.
#include <algorithm>
#include <atomic>
#include <map>
#include <mutex>
#include <stddef.h>
#include <stdint.h>
#include <stdio.h>
#include <string.h>
#include <vector>

#include "miconv.h"
#include "internal.h"

namespace miconv {

FastDiv make_fastdiv(uint32_t d)
{
    uint32_t s = 0;
    while ((1ull << s) < d)
        s++;
    uint64_t m = ((1ull << 32) * ((1ull << s) - d)) / d + 1;
    FastDiv f;
    f.mul = (uint32_t)m;
    f.shift = s;
    f.d = d;
    return f;
}

namespace {

constexpr long long kMaxElems = 2147483647LL;  // 2^31 - 1
constexpr long long kMaxChunkElems = (1LL << 29) - 1;  // per launch, per source tensor
constexpr size_t kAlign = 256;                  // sub-buffer alignment inside ws
constexpr int kBK = 16;                         // reduction slice of every GEMM kernel
// Workgroup targets are per compute unit (the rules below were measured on
// the MI355X's 256 CUs): target_workgroups() = 4 per CU.
// Tap-uniform backward-weight tiles: six fit on a CU at once, and about
// three rounds of them (16 per CU) measured best, as long as a split keeps
// at least kTapMinSlices slices (shorter splits cost more in partial sums
// than they gain in balance) -- unless that would leave fewer than
// target_workgroups() workgroups (small layers), where splits go down to 8
// slices.  (Timed plan selection also tries half and twice the splits of
// this rule; halving the target itself measured slower, as the caps then
// bind differently.)
constexpr int kTapMinSlices = 24;

size_t align_up(size_t v) { return (v + kAlign - 1) / kAlign * kAlign; }

struct Geom {
    int N, C, H, W, K, R, S, st, pad, G, P, Q, Cg, Kg;
};

int out_extent(int in, int filt, int stride, int pad)
{
    long long span = (long long)in + 2LL * pad - filt;
    if (span < 0)
        return 0;
    long long o = span / stride + 1;
    return o > kMaxElems ? 0 : (int)o;
}

int make_geom(int N, int C, int H, int W, int K, int R, int S, int stride, int pad, int group,
              Geom *g)
{
    if (N < 1 || C < 1 || H < 1 || W < 1 || K < 1 || R < 1 || S < 1 || stride < 1 || pad < 0 ||
        group < 1)
        return MICONV_ERR_SHAPE;
    if (C % group || K % group)
        return MICONV_ERR_SHAPE;
    // Spatial extents are kept below 2^15 so that packed (r, s) and
    // per-axis coordinates fit the kernels' 16-bit fields.
    if (H > 32767 || W > 32767 || R > 32767 || S > 32767 || pad > 32767)
        return MICONV_ERR_SHAPE;
    // Groups are folded with the tiles and splits into the 1-D grid; keeping
    // them below 2^16 keeps that product far from the grid limit.
    if (group > 65535)
        return MICONV_ERR_SHAPE;
    int P = out_extent(H, R, stride, pad), Q = out_extent(W, S, stride, pad);
    if (P < 1 || Q < 1)
        return MICONV_ERR_SHAPE;
    long long nx = (long long)N * C * H * W, ny = (long long)N * K * P * Q;
    long long nw = (long long)K * (C / group) * R * S;
    if (nx > kMaxElems || ny > kMaxElems || nw > kMaxElems)
        return MICONV_ERR_SHAPE;
    // Kernels address the images of one launch, and the packed filter bank,
    // with byte offsets below 2^31: one image and the filters must each stay
    // below 2^29 elements, the filters also as packed (each filter's
    // (C/G) R S, and each input channel's (K/G) R S, rounded up to 16).
    long long pw_fwd = (long long)K * (((long long)(C / group) * R * S + 15) / 16 * 16);
    long long pw_bwd = (long long)C * (((long long)(K / group) * R * S + 15) / 16 * 16);
    if ((long long)C * H * W > kMaxChunkElems || (long long)K * P * Q > kMaxChunkElems ||
        nw > kMaxChunkElems || pw_fwd > kMaxChunkElems || pw_bwd > kMaxChunkElems)
        return MICONV_ERR_SHAPE;
    *g = Geom{N, C, H, W, K, R, S, stride, pad, group, P, Q, C / group, K / group};
    return MICONV_OK;
}

struct Range {
    const void *p;
    size_t bytes;
    bool written;
};

bool overlap(const Range &a, const Range &b)
{
    if (!a.p || !b.p || !a.bytes || !b.bytes)
        return false;
    uintptr_t a0 = (uintptr_t)a.p, b0 = (uintptr_t)b.p;
    return a0 < b0 + b.bytes && b0 < a0 + a.bytes;
}

// Null, alignment, workspace and aliasing checks, in that order.
int check_buffers(const Range *r, int n, const bool *required, const void *ws, size_t ws_bytes,
                  size_t ws_need)
{
    for (int i = 0; i < n; i++)
        if (required[i] && !r[i].p)
            return MICONV_ERR_NULL;
    for (int i = 0; i < n; i++)
        if (r[i].p && ((uintptr_t)r[i].p % 16))
            return MICONV_ERR_ALIGN;
    if (ws_need) {
        if (!ws || ws_bytes < ws_need)
            return MICONV_ERR_WORKSPACE;
        if ((uintptr_t)ws % 16)
            return MICONV_ERR_ALIGN;
    }
    Range all[8];
    int m = 0;
    for (int i = 0; i < n; i++)
        all[m++] = r[i];
    if (ws_need)
        all[m++] = Range{ws, ws_need, true};
    for (int i = 0; i < m; i++)
        for (int j = i + 1; j < m; j++)
            if ((all[i].written || all[j].written) && overlap(all[i], all[j]))
                return MICONV_ERR_ALIAS;
    return MICONV_OK;
}

// Compute units of the current device (its multiProcessorCount, read once
// per device), or 256, the MI355X's, when no device can be queried (the
// host-only plan and workspace queries still work then).
int num_cus()
{
    static std::atomic<int> cache[64];  // 0: not read yet
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0)
        return 256;
    if (dev < 64) {
        int c = cache[dev].load(std::memory_order_relaxed);
        if (c > 0)
            return c;
    }
    hipDeviceProp_t prop;
    int n = 256;
    if (hipGetDeviceProperties(&prop, dev) == hipSuccess && prop.multiProcessorCount > 0)
        n = prop.multiProcessorCount;
    if (dev < 64)
        cache[dev].store(n, std::memory_order_relaxed);
    return n;
}

int target_workgroups() { return 4 * num_cus(); }
int tap_target_workgroups() { return 16 * num_cus(); }

int check_device()
{
    static std::atomic<int> cache[64];  // 0 unknown, 1 gfx950, 2 other
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0)
        return MICONV_ERR_DEVICE;
    if (dev < 64) {
        int c = cache[dev].load(std::memory_order_relaxed);
        if (c)
            return c == 1 ? MICONV_OK : MICONV_ERR_DEVICE;
    }
    hipDeviceProp_t prop;
    if (hipGetDeviceProperties(&prop, dev) != hipSuccess)
        return MICONV_ERR_DEVICE;
    bool ok = strncmp(prop.gcnArchName, "gfx950", 6) == 0;
    if (dev < 64)
        cache[dev].store(ok ? 1 : 2, std::memory_order_relaxed);
    return ok ? MICONV_OK : MICONV_ERR_DEVICE;
}

// ------------------------------------------------------------ kernel choice
int gemm_tiles(int M, int Ncol, int bm, int bn)
{
    return ((M + bm - 1) / bm) * ((Ncol + bn - 1) / bn);
}

// Fraction of the CUs' workgroup slots kept busy when `tiles` equal
// workgroups are dealt out over 256 CUs: tiles / (256 * ceil(tiles / 256)).
double cu_balance(long long tiles)
{
    const int cus = num_cus();
    long long rounds = (tiles + cus - 1) / cus;
    return rounds > 0 ? (double)tiles / (double)(rounds * cus) : 1.0;
}

// Tile choice for the image GEMM, from measured sweeps on MI355X across the
// layers of the five benchmark stacks.  The 64x64 tile (small accumulators,
// six workgroups per CU) is the default.  Row counts that would leave a
// 64-row tile partly empty take 16-, 32-, 48- (three waves) or 96-row tiles
// (96 rows: 128 columns wide when that still gives 4 tiles per CU).  The 128x64 tile halves the
// gathered-operand loads per MFMA and runs about 5 % faster per tile when it
// leaves no row empty and the reduction is not trivially short; it is taken
// when it gives every CU a workgroup and does not leave noticeably more CU
// slots idle in the last round than the 64x64 tiles would (a 2.3-per-CU deal
// against 4.6 lost 10 %).
int pick_img_tile(int M, long long Ncol, int Kred, int G)
{
    auto tiles = [&](int bm, int bn) {
        return (long long)((M + bm - 1) / bm) * ((Ncol + bn - 1) / bn) * G;
    };
    if (M <= 16)
        return IMG_16x128;
    if (M <= 32)
        return IMG_32x64;
    if (M <= 48)
        return IMG_48x64;
    if (M > 64 && M <= 96)
        return tiles(96, 128) >= 4 * num_cus() ? IMG_96x128 : IMG_96x64;
    if (M % 128 == 0 && Kred >= 256 && tiles(128, 64) >= num_cus() &&
        1.05 * cu_balance(tiles(128, 64)) >= cu_balance(tiles(64, 64)))
        return IMG_128x64;
    return IMG_64x64;
}

void img_tile_dims(int tile, int &bm, int &bn)
{
    static const int dims[][2] = {{64, 64}, {128, 64}, {16, 128}, {32, 64}, {48, 64},
                                  {96, 64}, {96, 128}, {128, 128}, {64, 128}};
    bm = dims[tile][0];
    bn = dims[tile][1];
}

// Images per launch so that every source view stays below 2^29 elements.
int images_per_launch(const Geom &g)
{
    long long per = (long long)g.C * g.H * g.W;
    long long pery = (long long)g.K * g.P * g.Q;
    if (pery > per)
        per = pery;
    long long n = kMaxChunkElems / per;
    return (int)(n < g.N ? n : g.N);
}


// ------------------------------------------------------------ plans
// Every pass has a built-in rule (measured on MI355X, below) and a list of
// candidate plans whose first entry is that rule.  A per-shape cache, filled
// by conv_plan_set or by conv_tune (which times the candidates, as the
// paper's framework times its convolution strategies over the first training
// iterations before keeping the fastest), overrides the rule.

constexpr int kNumImgTiles = 9;
constexpr int kNumWgradTiles = 9;

const char *img_tile_name(int tile)
{
    static const char *names[] = {"64x64", "128x64", "16x128", "32x64", "48x64",
                                  "96x64", "96x128", "128x128", "64x128"};
    static_assert(sizeof(names) / sizeof(names[0]) == kNumImgTiles, "one name per tile");
    return tile >= 0 && tile < kNumImgTiles ? names[tile] : "?";
}

// A tile whose rows are more than twice the problem's (rounded to 16) only
// multiplies zeros: not a candidate.
bool tile_fits(int tile, int M)
{
    int bm, bn;
    img_tile_dims(tile, bm, bn);
    return bm <= 2 * pad16(M);
}

long long tile_count(int tile, int M, long long Ncol, int G)
{
    int bm, bn;
    img_tile_dims(tile, bm, bn);
    return (long long)((M + bm - 1) / bm) * ((Ncol + bn - 1) / bn) * G;
}

// Split-K for the image GEMM.  With fewer than 2.5 tiles per CU the
// MFMA pipes starve for latency hiding; a deep reduction (>= kSplitMinRows)
// is then cut into splits of at least kSplitRows rows so that ~8 workgroups
// per CU run, each split writes an output-shaped partial slab, and a
// fixed-order reduction adds them (and the bias).  The slabs cost about
// 2 nsplit + 1 output passes of HBM traffic: measured, splitting reductions
// of 2304 rows or fewer lost up to a fifth, while 3200 rows and more at
// 200-600 tiles gained 6-23 %.  Only for single-launch problems (no batch
// chunking).
constexpr int kSplitMinRows = 3072;
constexpr int kSplitRows = 768;

struct ImgPlan {
    int tile, nsplit, kchunk;  // tile -1: (backward-data phases) each phase by the rule
    int xnb = 0;               // forward: explicit plan, images per column chunk (0: implicit)
    bool bt = false;           // inner product: batch-transposed plan
    int halo = -1;             // halo GEMM tile (HaloTile), or -1; kchunk then counts
    int tw = 0;                // 16-channel blocks per split, tw the pixel-block width
    int th = 0;                // pixel-block rows: 0 for 112 / tw, else a whole th x tw map
    int ks = 1;                // halo wave groups: 2 = eight waves over two halves of the blocks
};

// Rows and columns (pixels rounded up to 16) of a halo pixel block.
int halo_th(int tw, int th) { return th ? th : kHaloCols / tw; }
int halo_cols(int tw, int th) { return th ? (tw * th + 15) / 16 * 16 : kHaloCols; }

// Splits for `tiles` workgroups over Kred rows: about 8 workgroups per CU,
// each split at least kSplitRows rows and 8 slices; 1 if that is under two.
int split_count(long long tiles, int Kred)
{
    long long slices = (Kred + kBK - 1) / kBK;
    long long ns = (8LL * num_cus() + tiles - 1) / tiles;
    if (ns > slices / 8)
        ns = slices / 8;
    if (ns > Kred / kSplitRows)
        ns = Kred / kSplitRows;
    return ns < 2 ? 1 : (int)ns;
}

ImgPlan with_split(int tile, int Kred, int ns)
{
    ImgPlan p{tile, 1, Kred};
    if (ns >= 2) {
        long long slices = (Kred + kBK - 1) / kBK;
        p.kchunk = (int)((slices + ns - 1) / ns) * kBK;
        p.nsplit = (Kred + p.kchunk - 1) / p.kchunk;
    }
    return p;
}

ImgPlan img_rule(int M, long long Ncol, int Kred, int G, bool allow_split)
{
    const int tile = pick_img_tile(M, Ncol, Kred, G);
    if (!allow_split || Kred < kSplitMinRows)
        return with_split(tile, Kred, 1);
    const long long tiles = tile_count(tile, M, Ncol, G);
    return with_split(tile, Kred,
                      tiles >= 5LL * num_cus() / 2 ? 1 : split_count(tiles, Kred));
}

bool same_img(const ImgPlan &a, const ImgPlan &b)
{
    return a.tile == b.tile && a.nsplit == b.nsplit && a.xnb == b.xnb && a.bt == b.bt &&
           a.halo == b.halo && a.tw == b.tw && a.th == b.th && a.ks == b.ks;
}

// ------------------------------------------------------------ halo plans
// Stride-1 3 x 3 and 5 x 5 layers with channel-aligned slices can run the
// halo GEMM (halo_gemm_kernel): 112-column tiles that are TR x TW pixel
// blocks, the source region of a 16-channel block staged once for all R R
// taps.  The block width is the one of 56, 112, 28, 14 (3 x 3, in that order
// of preference: 56 x 2 blocks stage the least halo per pixel of the 16-byte
// ones and measured fastest wherever they fit, by 1-2 %) or of 28, 14 (5 x 5)
// that pads the output grid (P x Q) least; 0 if none can stage this source
// (16-byte loads need a source width that is a multiple of 4).
bool halo_filter(const Geom &g) { return g.st == 1 && g.R == g.S && (g.R == 3 || g.R == 5); }

int halo_width(int P, int Q, int src_w, int R)
{
    int best = 0;
    long long best_cols = 0;
    for (int tw : {56, 112, 28, 14}) {
        if (!halo_block_supported(tw, kHaloCols / tw, R, src_w, 0))
            continue;
        const int tr = kHaloCols / tw;
        const long long cols = (long long)((P + tr - 1) / tr) * ((Q + tw - 1) / tw) * kHaloCols;
        if (!best || cols < best_cols) {
            best = tw;
            best_cols = cols;
        }
    }
    return best;
}

long long halo_tile_count(int tile, int M, int nimg, int P, int Q, int tw, int G, int th = 0)
{
    const int bm = tile == HALO_128x112 ? 128 : 64, tr = halo_th(tw, th);
    return (long long)((M + bm - 1) / bm) * nimg * ((P + tr - 1) / tr) * ((Q + tw - 1) / tw) * G;
}

// A halo plan over ncb channel blocks: unsplit (ns = 1), or split so that
// about three workgroups per CU run (each split at least 4 blocks) when ns
// is 0, or into ns splits.
ImgPlan halo_plan(int tile, int tw, long long tiles, int ncb, int ns, int th = 0)
{
    if (ns == 0) {
        const long long want = 3LL * num_cus();
        ns = tiles >= want ? 1 : (int)std::min<long long>((want + tiles - 1) / tiles, ncb / 4);
        if (ns < 2)
            ns = 1;
    }
    ImgPlan p{IMG_64x64, 1, ncb};  // tile: the packed-filter layout (m-major)
    p.halo = tile;
    p.tw = tw;
    p.th = th;
    if (ns > 1) {
        p.kchunk = (ncb + ns - 1) / ns;
        p.nsplit = (ncb + p.kchunk - 1) / p.kchunk;
    }
    return p;
}

// Halo candidates of a stride-1 3 x 3 GEMM with M rows over cin source
// channels (a multiple of 16), an nimg x P x Q output grid and a src_w-wide
// source: each pixel-block width that pads the grid no more than the best
// one, each tile that fits M, unsplit and (allow_split) split.
std::vector<int> halo_widths(int P, int Q, int src_w, int R)
{
    std::vector<int> out;
    const int best = halo_width(P, Q, src_w, R);
    auto blocks = [&](int tw) {
        const int tr = kHaloCols / tw;
        return (long long)((P + tr - 1) / tr) * ((Q + tw - 1) / tw);
    };
    if (best)
        for (int tw : {112, 56, 28, 14})
            if (halo_block_supported(tw, kHaloCols / tw, R, src_w, 0) && blocks(tw) == blocks(best))
                out.push_back(tw);
    return out;
}

template <class P, class Make>
void halo_variants(int M, int cin, int nimg, int Pout, int Qout, int src_w, int R, int G,
                   bool allow_split, Make make, std::vector<P> &out)
{
    if (cin % 16)
        return;
    const int ncb = cin / 16;
    auto push = [&](const ImgPlan &c) {
        P p = make(c);
        bool dup = false;
        for (const P &q : out)
            dup = dup || same_plan(p, q);
        if (!dup)
            out.push_back(p);
    };
    // Per tile and pixel block: unsplit, split (allow_split), and two wave
    // groups where the tiles are at most two a CU (3 x 3, 56- to 14-wide
    // blocks, an even number of channel blocks).
    auto add = [&](int tile, int tw, int th) {
        const long long tiles = halo_tile_count(tile, M, nimg, Pout, Qout, tw, G, th);
        push(halo_plan(tile, tw, tiles, ncb, 1, th));
        const ImgPlan split = halo_plan(tile, tw, tiles, ncb, allow_split ? 0 : 1, th);
        if (split.nsplit > 1)
            push(split);
        if (!th && R == 3 && tw != 112 && ncb % 2 == 0 && tiles <= 2LL * num_cus()) {
            ImgPlan q = halo_plan(tile, tw, tiles, ncb, 1);
            q.ks = 2;
            push(q);
        }
    };
    for (int tw : halo_widths(Pout, Qout, src_w, R))
        for (int tile : {HALO_128x112, HALO_64x112})
            if (tile == HALO_64x112 || M > 64)
                add(tile, tw, 0);
    // A whole 13 x 13 map as one block (64-row tile only).
    if (Pout == Qout && halo_block_supported(Qout, Pout, R, src_w, 0))
        add(HALO_64x112, Qout, Pout);
}

// "<rows>x<columns>" of a halo tile with a tw-wide, th-row pixel block.
const char *halo_tile_name(int tile, int tw, int th)
{
    static thread_local char buf[16];
    snprintf(buf, sizeof buf, "%dx%d", tile == HALO_128x112 ? 128 : 64, halo_cols(tw, th));
    return buf;
}

// Splits of the rule's 3 x 3 halo plans: two when the tiles are fewer than
// two a CU and uneven over the CUs (so some CUs would run one more tile than
// the rest) and each split keeps at least 4 channel blocks; else one.
int halo_rule_splits(long long tiles, int ncb)
{
    const long long cus = num_cus();
    return tiles < 2 * cus && tiles % cus && ncb >= 8 ? 2 : 1;
}

// The built-in rule's use of the halo GEMM: whenever it applies and its pixel
// blocks cover the output grid with at most 1/8 of the columns idle (every
// map width of 224, 112, 56, 28 or 14 pixels, and 13 x 13 maps as whole-map
// blocks), with the 64-row tile, unsplit unless the tiles leave some CUs a
// tile more than others and number under two a CU: then two splits; tiles
// that fill one or two slots of every CU evenly run two wave groups (VGG-16
// conv5_x at batch 32, 512 tiles: 1-5 % faster forward, 0-3 % backward-data;
// ResNet s14_3x3 and GoogLeNet mid_3x3 backward-data 2-4 %).
// Measured on the MI355X at the configurations' batches: VGG-16 conv1_2 ...
// conv5_3 forward and backward-data 112-143 TFLOP/s against 93-126 for the
// image GEMM; ResNet 56 x 56 / 14 x 14 3 x 3 layers 124 / 108 against
// 92-104 / 86; AlexNet conv3-conv5 (13 x 13) 120-128 against 104-123;
// GoogLeNet's 14 x 14 3 x 3 backward-data with 192 rows (384 tiles) 102
// split against 85 unsplit.
// 5 x 5 layers take it with M >= 48 (at most one idle wave) when the tiles,
// split over channel blocks as halo_plan does if they are fewer than three
// workgroups a CU, give every CU one: AlexNet conv2 forward 130 TFLOP/s
// against 120 for the image GEMM and backward-data 106 against 104,
// GoogLeNet's 14 x 14 5 x 5 with 128 filters forward 87 against 64 and
// backward-data 60 (two splits) against 52; its 64-filter and 32-filter
// 5 x 5 layers (128 tiles, two channel blocks; M = 32) measured slower than
// the image GEMM and keep it.
bool halo_rule(int M, int cin, int nimg, int Pout, int Qout, int src_w, int R, int G,
               ImgPlan *out)
{
    if (cin % 16)
        return false;
    if (Pout == Qout && halo_block_supported(Qout, Pout, R, src_w, 0)) {
        const long long tiles = halo_tile_count(HALO_64x112, M, nimg, Pout, Qout, Qout, G, Pout);
        *out = halo_plan(HALO_64x112, Qout, tiles, cin / 16, halo_rule_splits(tiles, cin / 16),
                         Pout);
        return true;
    }
    const int tw = halo_width(Pout, Qout, src_w, R);
    if (!tw)
        return false;
    const int tr = kHaloCols / tw;
    const double used = (double)Pout * Qout /
                        ((double)((Pout + tr - 1) / tr) * ((Qout + tw - 1) / tw) * kHaloCols);
    if (used < 0.875)
        return false;
    if (R == 5) {
        const long long tiles = halo_tile_count(HALO_64x112, M, nimg, Pout, Qout, tw, G);
        const ImgPlan p = halo_plan(HALO_64x112, tw, tiles, cin / 16, 0);
        if (M < 48 || tiles * p.nsplit < num_cus())
            return false;
        *out = p;
        return true;
    }
    const long long tiles = halo_tile_count(HALO_64x112, M, nimg, Pout, Qout, tw, G);
    *out = halo_plan(HALO_64x112, tw, tiles, cin / 16, halo_rule_splits(tiles, cin / 16));
    // Tiles that fill one or two slots of every CU evenly: two wave groups.
    const long long cus = num_cus();
    if (out->nsplit == 1 && tw != 112 && (cin / 16) % 2 == 0 && tiles <= 2 * cus && tiles % cus == 0)
        out->ks = 2;
    return true;
}

// ------------------------------------------------------------ inner product
// A layer of 1 x 1 images and 1 x 1 filters is an inner-product layer
// (Sec. IV-A): y[n][k] = b[k] + sum_c w[k][c] x[n][c].  Its GEMMs have the
// batch as columns, C (or K) floats apart in x (or dy), so the gathered
// operand would be read one float per cache line.  The batch-transposed plan
// keeps every gathered row contiguous instead: forward transposes x once into
// [C][N] and runs the GEMM over one image of 1 x N pixels with w itself as the
// filter operand (its rows are the packed layout when C % 16 == 0);
// backward-data takes the batch as rows (dy as the row operand, padded to a
// multiple of 16 only when K is not one) and w as one image of 1 x C pixels;
// backward-weight transposes x and dy into [C][N] and [K][N] and runs the
// one-pixel-per-lane kernel over one image of N pixels.  The epilogues write
// y [N][K] and dx [N][C] directly.
bool is_inner_product(const Geom &g)
{
    // With padding the lone output pixel would read only zeros (P = Q = 1 for
    // stride > 2 pad): such shapes take the implicit plans, whose gathers
    // zero-fill padding.
    return g.H == 1 && g.W == 1 && g.R == 1 && g.S == 1 && g.P == 1 && g.Q == 1 && g.G == 1 &&
           g.pad == 0 && g.N <= 65535 * 32 && (long long)g.C * g.N <= kMaxChunkElems &&
           (long long)g.K * g.N <= kMaxChunkElems;
}

// Whether the inner product's forward must pack w: its rows are already the
// packed m-major layout when C is a multiple of 16 (tiles with a k-major
// filter operand need the copy).
bool ip_packs_w(const Geom &g, int tile) { return g.C % kBK != 0 || img_tile_shares_a(tile); }

// The problem over the transposed batch: one image of 1 x N pixels.
Geom batch_columns(const Geom &g)
{
    return Geom{1, g.C, 1, g.N, g.K, 1, 1, 1, 0, 1, 1, g.N, g.C, g.K};
}

// ------------------------------------------------------------ explicit plan
// The paper's explicit strategy (Sec. IV-B): im2col (forward, backward-weight)
// or col2im (backward-data) through HBM around a plain GEMM -- here the 1x1
// stride-1 convolution over the column tensor, run by the same kernels.  The
// column tensor is built for chunks of images within kExplicitColElems.
constexpr long long kExplicitColElems = 64LL << 20;  // 256 MB of fp32

// The 1x1 stride-1 problem over the column tensor of n images: channels
// c' = (c R + r) S + s (C R S of them, grouped as the input's), map P x Q.
Geom one_by_one(const Geom &g, int n)
{
    const int crs = g.Cg * g.R * g.S;
    return Geom{n, g.G * crs, g.P, g.Q, g.K, 1, 1, 1, 0, g.G, g.P, g.Q, crs, g.Kg};
}

long long col_elems_per_image(const Geom &g) { return (long long)g.C * g.R * g.S * g.P * g.Q; }

// Images per column chunk, or 0 where the explicit plan does not apply: a 1x1
// stride-1 layer without padding (its columns are its input), or one image's
// columns (or the packed filters of the transposed GEMM) beyond the limits.
int explicit_images(const Geom &g)
{
    if (g.R == 1 && g.S == 1 && g.st == 1 && g.pad == 0)
        return 0;
    const long long col1 = col_elems_per_image(g);
    if (col1 > kExplicitColElems || (long long)g.C * g.R * g.S * pad16(g.Kg) > kMaxChunkElems)
        return 0;
    long long n = kExplicitColElems / col1;
    const long long x1 = (long long)g.C * g.H * g.W, y1 = (long long)g.K * g.P * g.Q;
    if (n * x1 > kMaxChunkElems)
        n = kMaxChunkElems / x1;
    if (n * y1 > kMaxChunkElems)
        n = kMaxChunkElems / y1;
    if (n > g.N)
        n = g.N;
    return (int)n;
}

size_t col_bytes(const Geom &g, int xnb)
{
    return align_up((size_t)xnb * col_elems_per_image(g) * sizeof(float));
}

bool same_plan(const ImgPlan &a, const ImgPlan &b) { return same_img(a, b); }
struct BwdPlan;
bool same_plan(const BwdPlan &a, const BwdPlan &b);

// Every fitting tile, unsplit and (when allowed) split by split_count.
template <class P, class Make>
void img_variants(int M, long long Ncol, int Kred, int G, bool allow_split, Make make,
                  std::vector<P> &out)
{
    for (int t = 0; t < kNumImgTiles; t++) {
        if (!tile_fits(t, M))
            continue;
        ImgPlan cands[2] = {with_split(t, Kred, 1),
                            with_split(t, Kred,
                                       allow_split ? split_count(tile_count(t, M, Ncol, G), Kred)
                                                   : 1)};
        for (int i = 0; i < (cands[1].nsplit > 1 ? 2 : 1); i++) {
            P p = make(cands[i]);
            bool dup = false;
            for (const P &q : out)
                dup = dup || same_plan(p, q);
            if (!dup)
                out.push_back(p);
        }
    }
}

// Inner products are skinny GEMMs (the batch as the short side) that fill
// few tiles: also offer each tile with two and four times the rule's split
// count (or 2 and 4 splits where the rule has none), down to splits of 16
// slices.
template <class P, class Make>
void ip_fine_splits(int M, long long Ncol, int Kred, Make make, std::vector<P> &out)
{
    const long long slices = (Kred + kBK - 1) / kBK;
    for (int t = 0; t < kNumImgTiles; t++) {
        if (!tile_fits(t, M))
            continue;
        const int ns = split_count(tile_count(t, M, Ncol, 1), Kred);
        for (int f : {2, 4})
            if ((long long)ns * f <= slices / 16) {
                P p = make(with_split(t, Kred, ns * f));
                bool dup = false;
                for (const P &q : out)
                    dup = dup || same_plan(p, q);
                if (!dup)
                    out.push_back(p);
            }
    }
}

// ------------------------------------------------------------ forward
size_t fwd_pack_bytes(const Geom &g)
{
    return align_up((size_t)g.K * pad16(g.Cg * g.R * g.S) * sizeof(float));
}

ImgPlan fwd_rule(const Geom &g)
{
    if (is_inner_product(g)) {
        ImgPlan p = img_rule(g.K, g.N, g.C, 1, true);
        p.bt = true;
        return p;
    }
    ImgPlan h;
    const int nb = images_per_launch(g);
    if (halo_filter(g) && halo_rule(g.Kg, g.Cg, g.N < nb ? g.N : nb, g.P, g.Q, g.W, g.R, g.G, &h))
        return h;
    return img_rule(g.Kg, (long long)(g.N < nb ? g.N : nb) * g.P * g.Q, g.Cg * g.R * g.S, g.G,
                    nb >= g.N);
}

void fwd_candidates(const Geom &g, std::vector<ImgPlan> &out)
{
    out.clear();
    out.push_back(fwd_rule(g));
    if (is_inner_product(g)) {
        auto bt = [](const ImgPlan &p) {
            ImgPlan q = p;
            q.bt = true;
            return q;
        };
        img_variants<ImgPlan>(g.K, g.N, g.C, 1, true, bt, out);
        ip_fine_splits<ImgPlan>(g.K, g.N, g.C, bt, out);
    }
    const int nb = images_per_launch(g);
    img_variants<ImgPlan>(g.Kg, (long long)(g.N < nb ? g.N : nb) * g.P * g.Q, g.Cg * g.R * g.S,
                          g.G, nb >= g.N, [](const ImgPlan &p) { return p; }, out);
    if (halo_filter(g))
        halo_variants<ImgPlan>(g.Kg, g.Cg, g.N < nb ? g.N : nb, g.P, g.Q, g.W, g.R, g.G, nb >= g.N,
                               [](const ImgPlan &p) { return p; }, out);
    // Explicit: im2col, then the 1x1 GEMM with its own rule's tile.
    if (const int xnb = explicit_images(g)) {
        const int kred = g.Cg * g.R * g.S;
        ImgPlan e = with_split(pick_img_tile(g.Kg, (long long)xnb * g.P * g.Q, kred, g.G), kred, 1);
        e.xnb = xnb;
        out.push_back(e);
    }
}

size_t fwd_ws(const Geom &g, const ImgPlan &p)
{
    if (p.bt)
        return (ip_packs_w(g, p.tile) ? fwd_pack_bytes(g) : 0) +
               align_up((size_t)g.C * g.N * sizeof(float)) +
               (p.nsplit > 1 ? align_up((size_t)p.nsplit * g.N * g.K * sizeof(float)) : 0);
    if (p.xnb > 0)
        return fwd_pack_bytes(g) + col_bytes(g, p.xnb);
    size_t part = p.nsplit > 1 ? align_up((size_t)p.nsplit * g.N * g.K * g.P * g.Q * sizeof(float))
                               : 0;
    return fwd_pack_bytes(g) + part;
}

void fwd_name(const ImgPlan &p, char *buf, size_t len)
{
    const char *pre = p.bt ? "batch-transposed, " : "";
    if (p.xnb > 0)
        snprintf(buf, len, "explicit im2col (%d images a chunk), image GEMM %s", p.xnb,
                 img_tile_name(p.tile));
    else if (p.halo >= 0 && p.nsplit > 1)
        snprintf(buf, len, "halo GEMM %s (%dx%d pixels), %d splits",
                 halo_tile_name(p.halo, p.tw, p.th), p.tw, halo_th(p.tw, p.th), p.nsplit);
    else if (p.halo >= 0)
        snprintf(buf, len, "halo GEMM %s (%dx%d pixels)%s", halo_tile_name(p.halo, p.tw, p.th),
                 p.tw, halo_th(p.tw, p.th), p.ks == 2 ? ", 8 waves" : "");
    else if (p.nsplit > 1)
        snprintf(buf, len, "%simage GEMM %s, %d splits", pre, img_tile_name(p.tile), p.nsplit);
    else
        snprintf(buf, len, "%simage GEMM %s", pre, img_tile_name(p.tile));
}

// ------------------------------------------------------------ backward-data
// Stride phase (ph, pw): input pixels h = ph + st*i, w = pw + st*j; the taps
// that reach them are r = r0 + st*rr (rr < nr), s = s0 + st*ss (ss < ns),
// with r0 = (ph + pad) mod st, and p = i + dh - rr where dh = (ph + pad - r0) / st.
struct Axis {
    int n;   // pixels of the phase along the axis
    int t0;  // first tap
    int nt;  // taps
    int d;   // offset dh / dw
};

Axis phase_axis(int in, int filt, int st, int pad, int ph)
{
    Axis a;
    a.n = ph < in ? (in - ph + st - 1) / st : 0;
    a.t0 = (ph + pad) % st;
    a.nt = a.t0 < filt ? (filt - a.t0 + st - 1) / st : 0;
    a.d = (ph + pad - a.t0) / st;
    return a;
}

// Blocked plan.  With few input channels per group the per-phase GEMMs have
// M = C/G rows, a fraction of the smallest tile.  The blocked plan puts the
// b x b input pixels of a block (b = stride * f) into the rows instead,
// M = C/G b^2, and gives all of them the union of their taps: input pixel
// h + pad = b hb + ph takes dy rows f hb + u, u = f - 1 - tu for tu < ntr with
// ntr = f + (R - 1) / stride, through filter row r = ph - stride u (a zero
// weight where r is outside the filter); columns alike.  Blocks hb cover
// [hb0, hb0 + nh) with hb0 = pad / b.  The rule takes it when its MFMA work,
// with M rounded up to the tile and the reduction to the slice, is below 3/4
// of the phase plan's.  Work on 16-row tiles counts 5/4: measured on the
// ResNet stem (7x7, stride 2), 4 x 4 blocks of 48 rows ran 18 % faster than
// 2 x 2 blocks of 12 rows, despite 19 % more work.
struct BlockPlan {
    int f, b, ntr, nts, hb0, wb0, nh, nw, M, a_ld;
};

double tile_rows(int M)
{
    if (M <= 16)
        return 20;  // 16 rows, at 4/5 of the wider tiles' rate
    if (M <= 32)
        return 32;
    if (M <= 48)
        return 48;
    if (M <= 64)
        return 64;
    if (M <= 96)
        return 96;
    return (M + 63) / 64 * 64.0;
}

// Geometry of the blocked plan with factor f; false where it does not apply
// (block wider than 8, more than 256 rows, or a filter bank past the limit).
bool block_geometry(const Geom &g, int f, BlockPlan *p)
{
    if (f < (g.st == 1 ? 2 : 1) || g.st * f > 8)
        return false;
    p->f = f;
    p->b = g.st * f;
    p->M = g.Cg * p->b * p->b;
    p->ntr = f + (g.R - 1) / g.st;
    p->nts = f + (g.S - 1) / g.st;
    p->hb0 = g.pad / p->b;
    p->wb0 = g.pad / p->b;
    p->nh = (g.H - 1 + g.pad) / p->b + 1 - p->hb0;
    p->nw = (g.W - 1 + g.pad) / p->b + 1 - p->wb0;
    p->a_ld = pad16(g.Kg * p->ntr * p->nts);
    return p->M <= 256 && (long long)g.G * p->M * p->a_ld <= kMaxChunkElems;
}

bool block_rule(const Geom &g, BlockPlan *out)
{
    double phase_work = 0;
    for (int ph = 0; ph < g.st; ph++)
        for (int pw = 0; pw < g.st; pw++) {
            Axis ah = phase_axis(g.H, g.R, g.st, g.pad, ph);
            Axis aw = phase_axis(g.W, g.S, g.st, g.pad, pw);
            phase_work += (double)tile_rows(g.Cg) * pad16(g.Kg * ah.nt * aw.nt) * ah.n * aw.n;
        }
    double best = 0.75 * phase_work;
    bool found = false;
    for (int f = 1; f <= 8; f++) {
        BlockPlan p;
        if (!block_geometry(g, f, &p))
            continue;
        double work = tile_rows(p.M) * p.a_ld * p.nh * p.nw;
        if (work < best) {
            best = work;
            *out = p;
            found = true;
        }
    }
    return found;
}

struct BwdPlan {
    bool blocked;
    BlockPlan bp;  // blocked only
    ImgPlan img;   // blocked, explicit: the GEMM's tile; phases: tile (-1: per phase by the
                   // rule) and split-K (stride 1 only)
    int xnb;       // explicit plan: images per column chunk (0: not explicit)
    bool bt;       // inner product: batch-transposed plan
};

bool same_plan(const BwdPlan &a, const BwdPlan &b)
{
    return a.blocked == b.blocked && (!a.blocked || a.bp.f == b.bp.f) && a.xnb == b.xnb &&
           a.bt == b.bt && same_img(a.img, b.img);
}

BwdPlan bwd_rule(const Geom &g)
{
    BwdPlan p{};
    const int nb = images_per_launch(g), n0 = g.N < nb ? g.N : nb;
    if (is_inner_product(g)) {
        p.bt = true;
        p.img = img_rule(g.N, g.C, g.K, 1, true);  // rows: the batch
    } else if (block_rule(g, &p.bp)) {
        p.blocked = true;
        const int kred = g.Kg * p.bp.ntr * p.bp.nts;
        p.img = with_split(pick_img_tile(p.bp.M, (long long)n0 * p.bp.nh * p.bp.nw, kred, g.G),
                           kred, 1);
    } else if (halo_filter(g) && halo_rule(g.Cg, g.Kg, n0, g.H, g.W, g.Q, g.R, g.G, &p.img)) {
        // The one phase as a halo GEMM.
    } else if (g.st == 1) {
        // Split-K only for stride 1 (one phase covering all of dx).
        p.img = img_rule(g.Cg, (long long)n0 * g.H * g.W, g.Kg * g.R * g.S, g.G, nb >= g.N);
    } else {
        p.img = ImgPlan{-1, 1, 0};
    }
    return p;
}

void bwd_candidates(const Geom &g, std::vector<BwdPlan> &out)
{
    out.clear();
    out.push_back(bwd_rule(g));
    if (is_inner_product(g)) {
        auto bt = [](const ImgPlan &i) {
            BwdPlan b{};
            b.img = i;
            b.bt = true;
            return b;
        };
        img_variants<BwdPlan>(g.N, g.C, g.K, 1, true, bt, out);
        ip_fine_splits<BwdPlan>(g.N, g.C, g.K, bt, out);
    }
    const int nb = images_per_launch(g), n0 = g.N < nb ? g.N : nb;
    // Phases, one tile for all of them.
    const int kred_max = g.Kg * ((g.R + g.st - 1) / g.st) * ((g.S + g.st - 1) / g.st);
    img_variants<BwdPlan>(g.Cg, (long long)n0 * g.H * g.W / (g.st * g.st), kred_max, g.G,
                          g.st == 1 && nb >= g.N,
                          [](const ImgPlan &i) { return BwdPlan{false, BlockPlan{}, i, 0}; }, out);
    // Stride 1, 3 x 3 or 5 x 5: the one phase as a halo GEMM over dx's pixel grid.
    if (halo_filter(g))
        halo_variants<BwdPlan>(g.Cg, g.Kg, n0, g.H, g.W, g.Q, g.R, g.G, nb >= g.N,
                               [](const ImgPlan &i) { return BwdPlan{false, BlockPlan{}, i, 0}; },
                               out);
    // Blocked, for few channels per group.
    if (g.Cg <= 16)
        for (int f = 1; f <= 8; f++) {
            BlockPlan bp;
            if (!block_geometry(g, f, &bp))
                continue;
            const int kred = g.Kg * bp.ntr * bp.nts;
            img_variants<BwdPlan>(bp.M, (long long)n0 * bp.nh * bp.nw, kred, g.G, false,
                                  [&](const ImgPlan &i) { return BwdPlan{true, bp, i, 0}; }, out);
        }
    // Explicit: the transposed 1x1 GEMM into the column tensor, then col2im.
    if (const int xnb = explicit_images(g)) {
        const int crs = g.Cg * g.R * g.S;
        BwdPlan e{};
        e.xnb = xnb;
        e.img = with_split(pick_img_tile(crs, (long long)xnb * g.P * g.Q, g.Kg, g.G), g.Kg, 1);
        out.push_back(e);
    }
}

size_t bwd_ws(const Geom &g, const BwdPlan &p)
{
    if (p.bt)  // dy padded to 16 columns (unless K already is), then split slabs
        return (g.K % kBK || img_tile_shares_a(p.img.tile)
                    ? align_up((size_t)g.N * pad16(g.K) * sizeof(float))
                    : 0) +
               (p.img.nsplit > 1 ? align_up((size_t)p.img.nsplit * g.N * g.C * sizeof(float))
                                 : 0);
    if (p.xnb > 0)
        return align_up((size_t)g.C * g.R * g.S * pad16(g.Kg) * sizeof(float)) +
               col_bytes(g, p.xnb);
    if (p.blocked)
        return align_up((size_t)g.G * p.bp.M * p.bp.a_ld * sizeof(float));
    size_t total = 0;
    for (int ph = 0; ph < g.st; ph++)
        for (int pw = 0; pw < g.st; pw++) {
            Axis ah = phase_axis(g.H, g.R, g.st, g.pad, ph);
            Axis aw = phase_axis(g.W, g.S, g.st, g.pad, pw);
            total += align_up((size_t)g.C * pad16(g.Kg * ah.nt * aw.nt) * sizeof(float));
        }
    if (p.img.nsplit > 1)
        total += align_up((size_t)p.img.nsplit * g.N * g.C * g.H * g.W * sizeof(float));
    return total;
}

void bwd_name(const BwdPlan &p, char *buf, size_t len)
{
    if (p.bt && p.img.nsplit > 1)
        snprintf(buf, len, "batch-transposed, image GEMM %s, %d splits", img_tile_name(p.img.tile),
                 p.img.nsplit);
    else if (p.bt)
        snprintf(buf, len, "batch-transposed, image GEMM %s", img_tile_name(p.img.tile));
    else if (p.xnb > 0)
        snprintf(buf, len, "explicit GEMM + col2im (%d images a chunk), image GEMM %s", p.xnb,
                 img_tile_name(p.img.tile));
    else if (p.blocked)
        snprintf(buf, len, "blocked %dx%d pixels (f=%d), image GEMM %s", p.bp.b, p.bp.b, p.bp.f,
                 img_tile_name(p.img.tile));
    else if (p.img.halo >= 0 && p.img.nsplit > 1)
        snprintf(buf, len, "stride phases, halo GEMM %s (%dx%d pixels), %d splits",
                 halo_tile_name(p.img.halo, p.img.tw, p.img.th), p.img.tw,
                 halo_th(p.img.tw, p.img.th), p.img.nsplit);
    else if (p.img.halo >= 0)
        snprintf(buf, len, "stride phases, halo GEMM %s (%dx%d pixels)%s",
                 halo_tile_name(p.img.halo, p.img.tw, p.img.th), p.img.tw,
                 halo_th(p.img.tw, p.img.th), p.img.ks == 2 ? ", 8 waves" : "");
    else if (p.img.tile < 0)
        snprintf(buf, len, "stride phases, tiles by rule");
    else if (p.img.nsplit > 1)
        snprintf(buf, len, "stride phases, image GEMM %s, %d splits", img_tile_name(p.img.tile),
                 p.img.nsplit);
    else
        snprintf(buf, len, "stride phases, image GEMM %s", img_tile_name(p.img.tile));
}

// ------------------------------------------------------------ backward-weight
// The reduction over N*P*Q pixels is cut into fixed-length splits (a
// multiple of the slice) so that about tap_target_workgroups() workgroups run;
// each split writes its own partial dw, summed afterwards in split order.
// Launches never straddle a batch chunk (images_per_launch).
struct WgradPlan {
    int tile, slice, chunk, nsplit, nb;
    bool via_part;
    size_t part_bytes, bias_bytes;
    int xnb;  // explicit plan: images per column chunk (0: implicit); nb = xnb then
    bool bt;  // inner product: batch-transposed plan (the problem of batch_columns)
    int img = -1;  // inner product: dW = dy^T x as an image GEMM with this tile (-1: no)
    int halo_tw = 0;  // halo backward-weight with this pixel-block width (0: no); chunk then
                      // counts pixel blocks
    int halo_ct = 1;  // its 16-channel sub-tiles per workgroup (1 or 2)
    int halo_db = 0;  // halo_ct 2: 1 the double-buffered eight-wave kernel, 2 single-stage eight waves
};

bool is_tap_tile(int tile) { return wgrad_tile_is_tap(tile); }

void wgrad_tile_dims(int tile, int &bm, int &bn)
{
    static const int dims[][2] = {{64, 32}, {64, 48}, {64, 16}, {96, 64}, {64, 64},
                                  {64, 32}, {128, 32}, {64, 64}, {128, 64}};
    static_assert(sizeof(dims) / sizeof(dims[0]) == kNumWgradTiles, "one shape per tile");
    bm = dims[tile][0];
    bn = dims[tile][1];
}

const char *wgrad_tile_name(int tile)
{
    static const char *names[] = {"tap 64x32",  "tap 64x48",   "tap 64x16",
                                  "pixel 96x64", "pixel 64x64", "pixel 64x32",
                                  "tap 128x32", "tap 64x64",   "tap 128x64"};
    static_assert(sizeof(names) / sizeof(names[0]) == kNumWgradTiles, "one name per tile");
    return tile >= 0 && tile < kNumWgradTiles ? names[tile] : "?";
}

// tile -1: the rule's tile.  scale: the rule's split count times 2^scale.
// nb > 0: launches of nb images (else images_per_launch).
WgradPlan wgrad_plan(const Geom &g, int tile = -1, int scale = 0, int nb = 0)
{
    WgradPlan p{};
    int M = g.Kg, Ncol = g.Cg * g.R * g.S;
    long long PQ = (long long)g.P * g.Q, Kred = (long long)g.N * PQ;
    if (tile < 0) {
        if (g.Cg >= 32 || g.Cg == 16) {
            // Tap-uniform tiles of 64 rows of K/G by 64 channels of one tap when
            // C/G is a multiple of 64 (3-13 % over 64 x 32 on the VGG-16 and
            // ResNet 1x1 layers, up to 5 % behind it on ResNet's 3x3 ones), by 48
            // when it is a multiple of 48, by 16 for 16 channels, else by 32, so
            // that no column stays idle.
            const int bn = g.Cg == 16 ? 16 : g.Cg % 64 == 0 ? 64 : g.Cg % 48 == 0 ? 48 : 32;
            tile = bn == 16   ? WG_TAP_64x16
                   : bn == 64 ? WG_TAP_64x64
                   : bn == 48 ? WG_TAP_64x48
                              : WG_TAP_64x32;
        } else {
            // Few channels per group: the same one-pixel-per-lane kernel with
            // (c, r, s) packed into the columns, 96 rows for 65-96 filters.
            const int bm = (M > 64 && M <= 96) ? 96 : 64, bn = Ncol <= 32 ? 32 : 64;
            tile = bm == 96 ? WG_PIX_96x64 : bn == 32 ? WG_PIX_64x32 : WG_PIX_64x64;
        }
    }
    p.tile = tile;
    p.slice = 64;
    int bm, bn;
    wgrad_tile_dims(tile, bm, bn);
    const long long tiles =
        is_tap_tile(tile)
            ? (long long)((M + bm - 1) / bm) * g.R * g.S * ((g.Cg + bn - 1) / bn) * g.G
            : (long long)gemm_tiles(M, Ncol, bm, bn) * g.G;
    long long ns = (tap_target_workgroups() + tiles - 1) / tiles;
    long long long_ns = Kred / (p.slice * kTapMinSlices);
    long long fill_ns = (target_workgroups() + tiles - 1) / tiles;
    long long max_ns = long_ns > fill_ns ? long_ns : fill_ns;
    if (max_ns > Kred / (p.slice * 8))
        max_ns = Kred / (p.slice * 8);
    if (ns > max_ns)
        ns = max_ns;
    if (scale > 0)
        ns <<= scale;
    else if (scale < 0)
        ns >>= -scale;
    if (ns > Kred / p.slice)
        ns = Kred / p.slice;
    if (ns < 1)
        ns = 1;
    long long chunk = (Kred + ns - 1) / ns;
    chunk = (chunk + p.slice - 1) / p.slice * p.slice;
    p.chunk = (int)chunk;
    p.nb = nb > 0 ? nb : images_per_launch(g);
    long long total = 0;
    for (int n0 = 0; n0 < g.N; n0 += p.nb) {
        long long n = g.N - n0 < p.nb ? g.N - n0 : p.nb;
        total += (n * PQ + chunk - 1) / chunk;
    }
    p.nsplit = (int)total;
    // Tap-uniform tiles always go through the partial buffer (the reduction
    // also reorders columns); packed tiles write dw directly when unsplit.
    p.via_part = is_tap_tile(p.tile) || p.nsplit > 1;
    p.part_bytes = p.via_part ? align_up((size_t)p.nsplit * g.K * Ncol * sizeof(float)) : 0;
    p.bias_bytes = align_up((size_t)p.nsplit * g.K * sizeof(float));
    return p;
}

// Inner product: dW = dy^T x as one image GEMM over the batch (rows K,
// columns C; the batch is its reduction, staged as N channels of x).
WgradPlan wgrad_img_plan(const Geom &g, int tile)
{
    WgradPlan p{};
    p.tile = -1;
    p.bt = true;
    p.img = tile;
    p.nsplit = 1;
    p.chunk = g.N;
    p.nb = 1;
    return p;
}

// Halo backward-weight (wgrad_halo_kernel): stride-1 3 x 3 layers with
// channel-aligned groups whose dy and x rows are a multiple of 4 wide, or
// 14-wide maps of an even number of rows, in one launch.  Pixel-block width:
// the one of 56, 28, 112, 14 (in that order of preference; the 112 x 1
// blocks stage 45 % more halo per pixel and measured 3-7 % slower) that pads
// the P x Q grid least (0: not applicable).  The rule for such layers: on
// VGG-16 conv1_2 ... conv4_3 at batch 32 it ran at 120-128 TFLOP/s against
// 116-122 for the best tap-tile plan.
int wgrad_halo_width(const Geom &g)
{
    if (g.st != 1 || g.R != 3 || g.S != 3 || g.Cg % 16 || is_inner_product(g) ||
        images_per_launch(g) < g.N)
        return 0;
    int best = 0;
    long long best_cols = 0;
    for (int tw : {56, 28, 112, 14}) {
        if (!wgrad_halo_supported(tw, g.P, g.Q, g.W))
            continue;
        const int tr = kHaloCols / tw;
        const long long cols =
            (long long)((g.P + tr - 1) / tr) * ((g.Q + tw - 1) / tw) * kHaloCols;
        if (!best || cols < best_cols) {
            best = tw;
            best_cols = cols;
        }
    }
    return best;
}

// Splits over the pixel blocks so that at most as many workgroups run as fit
// on the CUs at once (three per CU with one 16-channel sub-tile, two with two
// or with eight single-stage waves, one double-buffered), times 2^scale, each
// split at least 4 blocks.
WgradPlan wgrad_halo_plan(const Geom &g, int tw, int scale = 0, int ct = 1, int db = 0)
{
    WgradPlan p{};
    p.tile = -1;
    p.halo_tw = tw;
    p.halo_ct = ct;
    p.halo_db = db;
    p.slice = kHaloCols;
    p.nb = g.N;
    const int tr = kHaloCols / tw;
    const long long blocks = (long long)g.N * ((g.P + tr - 1) / tr) * ((g.Q + tw - 1) / tw);
    const long long tiles = (long long)((g.Kg + 63) / 64) * (g.Cg / (16 * ct)) * g.G;
    const long long resident = (db == 1 ? 1LL : ct == 1 ? 3LL : 2LL) * num_cus();
    long long ns = resident / tiles;  // rounded down: no second, partial round of workgroups
    if (scale > 0)
        ns <<= scale;
    else if (scale < 0)
        ns >>= -scale;
    if (ns > blocks / 4)
        ns = blocks / 4;
    if (ns < 1)
        ns = 1;
    p.chunk = (int)((blocks + ns - 1) / ns);
    p.nsplit = (int)((blocks + p.chunk - 1) / p.chunk);
    p.via_part = true;
    p.part_bytes = align_up((size_t)p.nsplit * g.K * g.Cg * 9 * sizeof(float));
    p.bias_bytes = align_up((size_t)p.nsplit * g.K * sizeof(float));
    return p;
}

WgradPlan wgrad_rule(const Geom &g)
{
    // Where the channels allow, 64 x 32 tiles over eight waves: on maps of 112
    // rows or more the double-buffered kernel (VGG-16 at batch 32: conv1_2 ...
    // conv2_2 2-6 % faster than the four-wave single-stage 64 x 32 one, itself
    // 2-4 % faster than 64 x 16), on smaller ones the single-stage one with
    // two workgroups a CU (conv3_1 ... conv5_x 3-4 % faster than the
    // double-buffered one; ResNet-50's 56 x 56 and 28 x 28 3 x 3 layers 1-7 %).
    if (const int tw = wgrad_halo_width(g))
        return g.Cg % 32 == 0 ? wgrad_halo_plan(g, tw, 0, 2, g.P >= 112 ? 1 : 2)
                              : wgrad_halo_plan(g, tw);
    if (!is_inner_product(g))
        return wgrad_plan(g);
    // With a batch of whole 16-row slices, the image GEMM over the batch
    // (AlexNet fc6-fc8 at batch 128: 16-25 % faster than the one-pixel-per-
    // lane kernel).  Otherwise packed-column tiles, which write dw directly
    // when unsplit (the reduction over a batch is short); tap-uniform tiles
    // would add a partial buffer of dw's size.
    if (g.N % kBK == 0) {
        // dy^T is read as it lies (m-major): not the 16-row tile, which
        // shares a k-major filter operand through LDS.
        const int t = pick_img_tile(g.K, g.C, g.N, 1);
        return wgrad_img_plan(g, img_tile_shares_a(t) ? IMG_32x64 : t);
    }
    WgradPlan p = wgrad_plan(batch_columns(g), g.K > 64 && g.K <= 96 ? WG_PIX_96x64 : WG_PIX_64x64);
    p.bt = true;
    return p;
}

// A tile whose columns are more than twice the problem's (channels of one
// tap for tap-uniform tiles, packed (c, r, s) columns otherwise; rounded up
// to 16) only multiplies zeros: not a candidate.  (Rows are not pruned: a
// 64-row tap tile was measured fastest on a 16-filter 1x1 layer.)
bool wgrad_tile_fits(const Geom &g, int tile)
{
    int bm, bn;
    wgrad_tile_dims(tile, bm, bn);
    return bn <= 2 * pad16(is_tap_tile(tile) ? g.Cg : g.Cg * g.R * g.S);
}

void wgrad_candidates(const Geom &g, std::vector<WgradPlan> &out)
{
    out.clear();
    out.push_back(wgrad_rule(g));
    if (is_inner_product(g) && g.N % kBK == 0)
        // dW [K][C] = dy^T x: rows K, columns C, the batch as the reduction
        // (a short one); the image GEMM's tiles with filter rows in registers.
        for (int t : {IMG_64x64, IMG_128x64, IMG_32x64, IMG_96x128})
            if (tile_fits(t, g.K) && t != out[0].img)
                out.push_back(wgrad_img_plan(g, t));
    if (is_inner_product(g))
        for (int t = 0; t < kNumWgradTiles; t++)
            for (int scale : {0, 1, -1}) {
                if (!wgrad_tile_fits(batch_columns(g), t))
                    continue;
                WgradPlan p = wgrad_plan(batch_columns(g), t, scale);
                p.bt = true;
                bool dup = false;
                for (const WgradPlan &q : out)
                    dup = dup || (q.bt && q.tile == p.tile && q.chunk == p.chunk);
                if (!dup)
                    out.push_back(p);
            }
    for (int t = 0; t < kNumWgradTiles; t++)
        for (int scale : {0, 1, -1}) {
            if (!wgrad_tile_fits(g, t))
                continue;
            WgradPlan p = wgrad_plan(g, t, scale);
            bool dup = false;
            for (const WgradPlan &q : out)
                dup = dup || (q.tile == p.tile && q.chunk == p.chunk && q.xnb == 0 && !q.bt &&
                              !q.halo_tw);
            if (!dup)
                out.push_back(p);
        }
    // Explicit: im2col, then the 1x1 problem over the columns by its own rule.
    if (const int xnb = explicit_images(g)) {
        WgradPlan e = wgrad_plan(one_by_one(g, g.N), -1, 0, xnb);
        e.xnb = xnb;
        out.push_back(e);
    }
    // Halo: all nine taps of a tile from one staging per pixel block; each
    // block width that pads the grid no more than the best one.
    if (const int best = wgrad_halo_width(g)) {
        auto blocks = [&](int tw) {
            const int tr = kHaloCols / tw;
            return (long long)((g.P + tr - 1) / tr) * ((g.Q + tw - 1) / tw);
        };
        // 16 channels; 32; 32 double-buffered; 32 over eight single-stage waves
        for (int kind : {0, 1, 2, 3}) {
            const int ct = kind ? 2 : 1, db = kind == 2 ? 1 : kind == 3 ? 2 : 0;
            for (int tw : {112, 56, 28, 14})
                if (g.Cg % (16 * ct) == 0 && wgrad_halo_supported(tw, g.P, g.Q, g.W) &&
                    blocks(tw) == blocks(best))
                    for (int scale : {0, 1, -1}) {
                        WgradPlan p = wgrad_halo_plan(g, tw, scale, ct, db);
                        bool dup = false;
                        for (const WgradPlan &q : out)
                            dup = dup || (q.halo_tw == p.halo_tw && q.halo_ct == p.halo_ct &&
                                          q.halo_db == p.halo_db && q.chunk == p.chunk);
                        if (!dup)
                            out.push_back(p);
                    }
        }
    }
}

size_t wgrad_ws(const Geom &g, const WgradPlan &p)
{
    if (p.img >= 0)  // dy^T [K][N]
        return align_up((size_t)g.K * g.N * sizeof(float));
    const size_t bt = p.bt ? align_up((size_t)g.C * g.N * sizeof(float)) +
                                 align_up((size_t)g.K * g.N * sizeof(float))
                           : 0;
    return p.part_bytes + p.bias_bytes + (p.xnb > 0 ? col_bytes(g, p.xnb) : 0) + bt;
}

void wgrad_name(const WgradPlan &p, char *buf, size_t len)
{
    if (p.img >= 0)
        snprintf(buf, len, "batch-transposed, image GEMM %s over the batch", img_tile_name(p.img));
    else if (p.halo_tw)
        snprintf(buf, len, "halo, 9 taps of 64x%d%s (%dx%d pixels), %d splits of %d blocks",
                 16 * p.halo_ct, p.halo_db == 1 ? " (8 waves, 2 stages)" : p.halo_db ? " (8 waves)" : "",
                 p.halo_tw, kHaloCols / p.halo_tw, p.nsplit, p.chunk);
    else if (p.xnb > 0)
        snprintf(buf, len, "explicit im2col (%d images a chunk), %s, %d splits of %d pixels",
                 p.xnb, wgrad_tile_name(p.tile), p.nsplit, p.chunk);
    else
        snprintf(buf, len, "%s%s, %d splits of %d pixels", p.bt ? "batch-transposed, " : "",
                 wgrad_tile_name(p.tile), p.nsplit, p.chunk);
}

// ------------------------------------------------------------ plan cache
struct PlanKey {
    int v[12];
    bool operator<(const PlanKey &o) const
    {
        return std::lexicographical_compare(v, v + 12, o.v, o.v + 12);
    }
};

// A stored choice keeps its candidate index and the plan itself, so that a
// call with a stored plan costs one table lookup.
struct StoredPlan {
    int index;
    ImgPlan fwd;
    BwdPlan bwd;
    WgradPlan wgrad;
};

std::mutex g_plan_mu;
std::map<PlanKey, StoredPlan> g_plans;
std::atomic<int> g_plan_entries{0};

PlanKey plan_key(int pass, const Geom &g)
{
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess)
        dev = -1;
    return PlanKey{{dev, pass, g.N, g.C, g.H, g.W, g.K, g.R, g.S, g.st, g.pad, g.G}};
}

// The stored choice for this shape on the current device, if any.
bool stored_plan(int pass, const Geom &g, StoredPlan *out)
{
    if (g_plan_entries.load(std::memory_order_acquire) == 0)
        return false;
    PlanKey k = plan_key(pass, g);
    std::lock_guard<std::mutex> lock(g_plan_mu);
    auto it = g_plans.find(k);
    if (it == g_plans.end())
        return false;
    *out = it->second;
    return true;
}

// Candidate index the calls use for this shape on the current device.
int plan_index(int pass, const Geom &g)
{
    StoredPlan sp;
    return stored_plan(pass, g, &sp) ? sp.index : 0;
}

template <class P>
P pick(const P &rule, int index, void (*cands)(const Geom &, std::vector<P> &), const Geom &g)
{
    if (index <= 0)
        return rule;
    std::vector<P> c;
    cands(g, c);
    return index < (int)c.size() ? c[index] : rule;
}

void plan_store(int pass, const Geom &g, int index)
{
    PlanKey k = plan_key(pass, g);
    StoredPlan sp{};
    sp.index = index;
    if (pass == MICONV_PASS_FWD)
        sp.fwd = pick(fwd_rule(g), index, fwd_candidates, g);
    else if (pass == MICONV_PASS_BWD_DATA)
        sp.bwd = pick(bwd_rule(g), index, bwd_candidates, g);
    else
        sp.wgrad = pick(wgrad_rule(g), index, wgrad_candidates, g);
    std::lock_guard<std::mutex> lock(g_plan_mu);
    if (index <= 0)
        g_plans.erase(k);
    else
        g_plans[k] = sp;
    g_plan_entries.store((int)g_plans.size(), std::memory_order_release);
}

ImgPlan fwd_current(const Geom &g)
{
    StoredPlan sp;
    return stored_plan(MICONV_PASS_FWD, g, &sp) ? sp.fwd : fwd_rule(g);
}
BwdPlan bwd_current(const Geom &g)
{
    StoredPlan sp;
    return stored_plan(MICONV_PASS_BWD_DATA, g, &sp) ? sp.bwd : bwd_rule(g);
}
WgradPlan wgrad_current(const Geom &g)
{
    StoredPlan sp;
    return stored_plan(MICONV_PASS_BWD_WEIGHT, g, &sp) ? sp.wgrad : wgrad_rule(g);
}

// ------------------------------------------------------------ execution
int launch_status(hipError_t e) { return e == hipSuccess ? MICONV_OK : MICONV_ERR_LAUNCH; }

// Caller-owned timing events of conv_set_timing_events, per calling thread.
struct TimingEvents {
    hipEvent_t before = nullptr, after = nullptr;
};
thread_local TimingEvents tl_events;

hipError_t mark(hipEvent_t ev, hipStream_t stream)
{
    return ev ? hipEventRecord(ev, stream) : hipSuccess;
}

// One halo GEMM launch (plan.halo >= 0) of a stride-1 R x R problem: M rows
// of the packed bank A (a_ld words each, FAST order over cin source channels),
// source images src (src_c channels of src_h x src_w), output grid Pout x Qout
// of out (out_c channels per image), nimg images; (coff_h, coff_w) is the
// source coordinate of tap (0, 0) of output pixel (0, 0), flip for the
// backward-data phase (source row p + coff_h - r).  Split partial slabs go to
// part, split_stride apart.
int halo_gemm(const ImgPlan &plan, int M, int groups, const float *A, int a_ld, int cin, int R,
              const float *src, int src_c, int src_h, int src_w, int Pout, int Qout, int out_c,
              int nimg, int coff_h, int coff_w, bool flip, const float *bias, float *out,
              float *part, long long split_stride, hipStream_t stream)
{
    const size_t fb = sizeof(float);
    HaloGemmArgs h{};
    h.M = M;
    h.R = R;
    h.Kred = cin * R * R;
    h.groups = groups;
    h.A = A;
    h.a_ld = a_ld;
    h.a_bytes = (uint32_t)((size_t)groups * M * a_ld * fb);
    h.src = src;
    h.src_bytes = (uint32_t)((size_t)nimg * src_c * src_h * src_w * fb);
    h.cin = cin;
    h.src_h = src_h;
    h.src_w = src_w;
    h.src_hw = src_h * src_w;
    h.src_img_words = (uint32_t)((size_t)src_c * src_h * src_w);
    h.P = Pout;
    h.Q = Qout;
    h.TW = plan.tw;
    h.TR = halo_th(plan.tw, plan.th);
    h.row_blocks = (Pout + h.TR - 1) / h.TR;
    h.col_segs = (Qout + h.TW - 1) / h.TW;
    h.nimg = nimg;
    // Halo origin: the top-left source pixel any tap of the block reads.
    const int V = halo_load_words(plan.tw, h.TR, R);
    h.row0 = flip ? coff_h - (R - 1) : coff_h;
    const int col_raw = flip ? coff_w - (R - 1) : coff_w;
    h.col0 = (col_raw >= 0 ? col_raw / V : -((-col_raw + V - 1) / V)) * V;
    h.slack = col_raw - h.col0;
    h.out = plan.nsplit > 1 ? part : out;
    h.bias = bias;
    h.out_img_stride = (long long)out_c * Pout * Qout;
    h.out_hw = Pout * Qout;
    h.out_w = Qout;
    h.nsplit = plan.nsplit;
    h.cbchunk = plan.kchunk;
    h.split_stride = split_stride;
    h.ks = plan.ks;
    return launch_status(launch_halo_gemm(h, plan.halo, flip, stream));
}

// Forward GEMM launches over n images of geometry g (images from src, outputs
// to y), at most images_per_launch(g) images a launch; wp is the packed
// filter bank, part the split-K slabs (plan.nsplit > 1: n must be all of g's).
int fwd_gemms(const Geom &g, const ImgPlan &plan, const float *wp, const float *src,
              const float *b, float *y, float *part, int n_images, hipStream_t stream)
{
    const size_t fb = sizeof(float);
    const int a_ld = pad16(g.Cg * g.R * g.S);
    const int nb = images_per_launch(g);
    const long long xi = (long long)g.C * g.H * g.W, yi = (long long)g.K * g.P * g.Q;
    ImgGemmArgs a{};
    a.M = g.Kg;
    a.Kred = g.Cg * g.R * g.S;
    a.groups = g.G;
    a.A = wp;
    a.a_ld = a_ld;
    a.a_bytes = (uint32_t)((size_t)g.K * a_ld * fb);
    a.cin = g.Cg;
    a.src_h = g.H;
    a.src_w = g.W;
    a.src_hw = g.H * g.W;
    a.src_img_words = (uint32_t)xi;
    a.col_hw = make_fastdiv(g.P * g.Q);
    a.col_w = make_fastdiv(g.Q);
    a.cstep = g.st;
    a.coff_h = -g.pad;
    a.coff_w = -g.pad;
    a.tsign = 1;
    a.k_cin = make_fastdiv(g.Cg);
    a.k_tw = make_fastdiv(g.S);
    a.k_taps = make_fastdiv(g.R * g.S);
    a.bias = b;
    a.out_img_stride = yi;
    a.out_hw = g.P * g.Q;
    a.out_w = g.Q;
    a.ostep = 1;
    const bool fast = g.Cg % kBK == 0;
    for (int n0 = 0; n0 < n_images; n0 += nb) {
        const int n = n_images - n0 < nb ? n_images - n0 : nb;
        if (plan.halo >= 0) {
            int st = halo_gemm(plan, g.Kg, g.G, wp, a_ld, g.Cg, g.R, src + n0 * xi, g.C, g.H, g.W, g.P,
                               g.Q, g.K, n, -g.pad, -g.pad, false, b, y + n0 * yi, part,
                               (long long)n_images * yi, stream);
            if (st != MICONV_OK)
                return st;
            continue;
        }
        a.Ncol = n * g.P * g.Q;
        a.src = src + n0 * xi;
        a.src_bytes = (uint32_t)(n * xi * (long long)fb);
        a.out = plan.nsplit > 1 ? part : y + n0 * yi;
        a.nsplit = plan.nsplit;
        a.kchunk = plan.kchunk;
        a.split_stride = (long long)n_images * yi;
        int st = launch_status(launch_img_gemm(a, plan.tile, fast, stream));
        if (st != MICONV_OK)
            return st;
    }
    return MICONV_OK;
}

// Inner product by the batch-transposed plan (see is_inner_product).
int ip_fwd(const Geom &g, const ImgPlan &plan, const float *x, const float *w, const float *b,
           float *y, void *ws, hipStream_t stream)
{
    const int N = g.N, C = g.C, K = g.K;
    const size_t fb = sizeof(float);
    const int a_ld = pad16(C);
    const float *A = w;
    char *tail = (char *)ws;
    if (ip_packs_w(g, plan.tile)) {
        float *wp = (float *)ws;
        if (launch_pack_fwd(w, wp, K, C, 1, 1, 1, C % kBK == 0, a_ld,
                            img_tile_shares_a(plan.tile), stream) != hipSuccess)
            return MICONV_ERR_LAUNCH;
        A = wp;
        tail += fwd_pack_bytes(g);
    }
    float *xt = (float *)tail;
    float *part = (float *)(tail + align_up((size_t)C * N * fb));
    if (launch_transpose(x, xt, N, C, stream) != hipSuccess)
        return MICONV_ERR_LAUNCH;
    // Rows: the K filters; columns: the N images, one image of 1 x N pixels
    // of [C][N]; y[n][k] at n * K + k.
    ImgGemmArgs a{};
    a.M = K;
    a.Ncol = N;
    a.Kred = C;
    a.groups = 1;
    a.A = A;
    a.a_ld = a_ld;
    a.a_bytes = (uint32_t)((size_t)K * a_ld * fb);
    a.src = xt;
    a.src_bytes = (uint32_t)((size_t)C * N * fb);
    a.cin = C;
    a.src_h = 1;
    a.src_w = N;
    a.src_hw = N;
    a.src_img_words = (uint32_t)((size_t)C * N);
    a.col_hw = make_fastdiv(N);
    a.col_w = make_fastdiv(N);
    a.cstep = 1;
    a.tsign = 1;
    a.k_cin = make_fastdiv(C);
    a.k_tw = make_fastdiv(1);
    a.k_taps = make_fastdiv(1);
    a.bias = b;
    a.out = plan.nsplit > 1 ? part : y;
    a.out_hw = 1;
    a.out_w = 1;
    a.ostep = K;
    a.nsplit = plan.nsplit;
    a.kchunk = plan.kchunk;
    a.split_stride = (long long)N * K;
    if (mark(tl_events.before, stream) != hipSuccess)
        return MICONV_ERR_LAUNCH;
    int st = launch_status(launch_img_gemm(a, plan.tile, C % kBK == 0, stream));
    if (st != MICONV_OK)
        return st;
    if (mark(tl_events.after, stream) != hipSuccess)
        return MICONV_ERR_LAUNCH;
    if (plan.nsplit > 1)
        return launch_status(launch_splitk_bias_reduce(part, plan.nsplit, (long long)N * K, N * K,
                                                       b, 1, K, y, stream));
    return MICONV_OK;
}

int ip_bwd_data(const Geom &g, const BwdPlan &plan, const float *dy, const float *w, float *dx,
                void *ws, hipStream_t stream)
{
    const int N = g.N, C = g.C, K = g.K;
    const size_t fb = sizeof(float);
    const int a_ld = pad16(K);
    const float *A = dy;
    char *tail = (char *)ws;
    if (K % kBK || img_tile_shares_a(plan.img.tile)) {
        // dy rows padded to a multiple of 16 (the rows of 1 x 1 "filters").
        float *dp = (float *)ws;
        if (launch_pack_fwd(dy, dp, N, K, 1, 1, 1, K % kBK == 0, a_ld,
                            img_tile_shares_a(plan.img.tile), stream) != hipSuccess)
            return MICONV_ERR_LAUNCH;
        A = dp;
        tail += align_up((size_t)N * a_ld * fb);
    }
    float *part = (float *)tail;
    // Rows: the N images; columns: the C inputs, one image of 1 x C pixels
    // of w [K][C]; dx[n][c] at n * C + c.
    ImgGemmArgs a{};
    a.M = N;
    a.Ncol = C;
    a.Kred = K;
    a.groups = 1;
    a.A = A;
    a.a_ld = a_ld;
    a.a_bytes = (uint32_t)((size_t)N * a_ld * fb);
    a.src = w;
    a.src_bytes = (uint32_t)((size_t)K * C * fb);
    a.cin = K;
    a.src_h = 1;
    a.src_w = C;
    a.src_hw = C;
    a.src_img_words = (uint32_t)((size_t)K * C);
    a.col_hw = make_fastdiv(C);
    a.col_w = make_fastdiv(C);
    a.cstep = 1;
    a.tsign = 1;
    a.k_cin = make_fastdiv(K);
    a.k_tw = make_fastdiv(1);
    a.k_taps = make_fastdiv(1);
    a.out = plan.img.nsplit > 1 ? part : dx;
    a.out_hw = C;
    a.out_w = C;
    a.ostep = 1;
    a.nsplit = plan.img.nsplit;
    a.kchunk = plan.img.nsplit > 1 ? plan.img.kchunk : K;
    a.split_stride = (long long)N * C;
    if (mark(tl_events.before, stream) != hipSuccess)
        return MICONV_ERR_LAUNCH;
    int st = launch_status(launch_img_gemm(a, plan.img.tile, K % kBK == 0, stream));
    if (st != MICONV_OK)
        return st;
    if (mark(tl_events.after, stream) != hipSuccess)
        return MICONV_ERR_LAUNCH;
    if (plan.img.nsplit > 1)
        return launch_status(launch_splitk_bias_reduce(part, plan.img.nsplit, (long long)N * C,
                                                       N * C, nullptr, 1, 1, dx, stream));
    return MICONV_OK;
}

int fwd_exec(const Geom &g, const ImgPlan &plan, const float *x, const float *w, const float *b,
             float *y, void *ws, size_t ws_bytes, hipStream_t stream)
{
    const int N = g.N, C = g.C, H = g.H, W = g.W, K = g.K, R = g.R, S = g.S;
    const size_t fb = sizeof(float);
    Range r[4] = {{x, (size_t)N * C * H * W * fb, false},
                  {w, (size_t)K * g.Cg * R * S * fb, false},
                  {b, (size_t)K * fb, false},
                  {y, (size_t)N * K * g.P * g.Q * fb, true}};
    bool req[4] = {true, true, false, true};
    int st = check_buffers(r, 4, req, ws, ws_bytes, fwd_ws(g, plan));
    if (st != MICONV_OK || (st = check_device()) != MICONV_OK)
        return st;
    (void)hipGetLastError();
    if (plan.bt)
        return ip_fwd(g, plan, x, w, b, y, ws, stream);

    // The filter bank, packed in the layout the tile reads.  The explicit
    // plan's 1x1 GEMM reads the same matrix: its reduction index is the
    // column tensor's channel (c R + r) S + s, the filter's own order.
    float *wp = (float *)ws;
    const Geom g1 = one_by_one(g, N);
    const Geom &gp = plan.xnb > 0 ? g1 : g;
    if (launch_pack_fwd(w, wp, K, gp.Cg, gp.R, gp.S, g.G, gp.Cg % kBK == 0,
                        pad16(g.Cg * R * S), img_tile_shares_a(plan.tile), stream) != hipSuccess)
        return MICONV_ERR_LAUNCH;
    float *tail = (float *)((char *)ws + fwd_pack_bytes(g));
    if (mark(tl_events.before, stream) != hipSuccess)
        return MICONV_ERR_LAUNCH;
    if (plan.xnb > 0) {
        // Explicit: im2col of a chunk of images, then the 1x1 GEMM over it.
        const long long xi = (long long)C * H * W, yi = (long long)K * g.P * g.Q;
        for (int n0 = 0; n0 < N; n0 += plan.xnb) {
            const int n = N - n0 < plan.xnb ? N - n0 : plan.xnb;
            if (launch_im2col(x + n0 * xi, tail, n, C, H, W, R, S, g.st, g.pad, g.P, g.Q,
                              stream) != hipSuccess)
                return MICONV_ERR_LAUNCH;
            if ((st = fwd_gemms(one_by_one(g, n), plan, wp, tail, b, y + n0 * yi, nullptr, n,
                                stream)) != MICONV_OK)
                return st;
        }
    } else if ((st = fwd_gemms(g, plan, wp, x, b, y, tail, N, stream)) != MICONV_OK) {
        return st;
    }
    if (mark(tl_events.after, stream) != hipSuccess)
        return MICONV_ERR_LAUNCH;
    if (plan.nsplit > 1) {
        const long long yi = (long long)K * g.P * g.Q;
        return launch_status(launch_splitk_bias_reduce(tail, plan.nsplit, (long long)N * yi,
                                                       (int)(N * yi), b, g.P * g.Q, K, y,
                                                       stream));
    }
    return MICONV_OK;
}

// Backward-data by the blocked plan: one GEMM per batch chunk over columns
// (image, block row, block column), rows (channel, ph, pw).
int bwd_blocked(const Geom &g, const BwdPlan &plan, const float *dy, const float *w, float *dx,
                void *ws, hipStream_t stream)
{
    const BlockPlan &bp = plan.bp;
    const size_t fb = sizeof(float);
    const int nb = images_per_launch(g);
    const long long xi = (long long)g.C * g.H * g.W, yi = (long long)g.K * g.P * g.Q;
    const int kred = g.Kg * bp.ntr * bp.nts;
    const bool kmajor = img_tile_shares_a(plan.img.tile);
    float *wp = (float *)ws;
    if (launch_pack_bwd_block(w, wp, g.K, g.Cg, g.R, g.S, g.G, g.st, bp.f, bp.ntr, bp.nts,
                              g.Kg % kBK == 0, bp.a_ld, kmajor, stream) != hipSuccess)
        return MICONV_ERR_LAUNCH;
    ImgGemmArgs a{};
    a.M = bp.M;
    a.Kred = kred;
    a.groups = g.G;
    a.A = wp;
    a.a_ld = bp.a_ld;
    a.a_bytes = (uint32_t)((size_t)g.G * bp.M * bp.a_ld * fb);
    a.cin = g.Kg;
    a.src_h = g.P;
    a.src_w = g.Q;
    a.src_hw = g.P * g.Q;
    a.src_img_words = (uint32_t)yi;
    a.col_hw = make_fastdiv(bp.nh * bp.nw);
    a.col_w = make_fastdiv(bp.nw);
    // dy row of column block hb0 + ci and tap tu: f (hb0 + ci) + f - 1 - tu.
    a.cstep = bp.f;
    a.coff_h = bp.f * bp.hb0 + bp.f - 1;
    a.coff_w = bp.f * bp.wb0 + bp.f - 1;
    a.tsign = -1;
    a.k_cin = make_fastdiv(g.Kg);
    a.k_tw = make_fastdiv(bp.nts);
    a.k_taps = make_fastdiv(bp.ntr * bp.nts);
    a.bias = nullptr;
    a.out_img_stride = xi;
    a.out_hw = g.H * g.W;
    a.out_w = g.W;
    a.out_h = g.H;
    a.ostep = bp.b;
    a.ooff_h = bp.b * bp.hb0 - g.pad;
    a.ooff_w = bp.b * bp.wb0 - g.pad;
    a.mblock = bp.b;
    a.nsplit = 1;
    a.kchunk = kred;
    a.split_stride = 0;
    const bool fast = g.Kg % kBK == 0;
    if (mark(tl_events.before, stream) != hipSuccess)
        return MICONV_ERR_LAUNCH;
    for (int n0 = 0; n0 < g.N; n0 += nb) {
        const int n = g.N - n0 < nb ? g.N - n0 : nb;
        a.Ncol = n * bp.nh * bp.nw;
        a.src = dy + n0 * yi;
        a.src_bytes = (uint32_t)(n * yi * (long long)fb);
        a.out = dx + n0 * xi;
        int st = launch_status(launch_img_gemm(a, plan.img.tile, fast, stream));
        if (st != MICONV_OK)
            return st;
    }
    return mark(tl_events.after, stream) == hipSuccess ? MICONV_OK : MICONV_ERR_LAUNCH;
}

// Backward-data by stride phases over n images of geometry g (dy from dy,
// dx to dx): each phase packs its filter taps into wsp (advancing it past
// every phase's bank) and runs its GEMM; with split-K (stride 1, all images)
// the slabs follow the banks and the caller reduces them.  *marked tells
// whether the first GEMM's timing event has been recorded.
int phase_gemms(const Geom &g, const BwdPlan &plan, const float *w, char *&wsp, const float *dy,
                float *dx, int n_images, bool *marked, hipStream_t stream)
{
    const int H = g.H, W = g.W, K = g.K, R = g.R, S = g.S, stride = g.st, group = g.G;
    const size_t fb = sizeof(float);
    const int nb = images_per_launch(g);
    const long long xi = (long long)g.C * H * W, yi = (long long)K * g.P * g.Q;
    const bool split = plan.img.nsplit > 1;
    char *banks = wsp;
    size_t bank_bytes = 0;
    for (int ph = 0; ph < stride; ph++)
        for (int pw = 0; pw < stride; pw++) {
            Axis ah = phase_axis(H, R, stride, g.pad, ph);
            Axis aw = phase_axis(W, S, stride, g.pad, pw);
            bank_bytes += align_up((size_t)g.C * pad16(g.Kg * ah.nt * aw.nt) * fb);
        }
    float *part = (float *)(banks + bank_bytes);
    wsp = banks + bank_bytes;
    char *bank = banks;
    for (int ph = 0; ph < stride; ph++)
        for (int pw = 0; pw < stride; pw++) {
            Axis ah = phase_axis(H, R, stride, g.pad, ph);
            Axis aw = phase_axis(W, S, stride, g.pad, pw);
            const int a_ld = pad16(g.Kg * ah.nt * aw.nt);
            float *wr = (float *)bank;
            bank += align_up((size_t)g.C * a_ld * fb);
            if (ah.n == 0 || aw.n == 0)
                continue;
            const int kred = ah.nt * aw.nt * g.Kg;
            const int tile =
                plan.img.tile >= 0
                    ? plan.img.tile
                    : pick_img_tile(g.Cg, (long long)(n_images < nb ? n_images : nb) * ah.n * aw.n,
                                    kred, group);
            const bool kmajor = img_tile_shares_a(tile);
            if (launch_pack_bwd_phase(w, wr, K, g.Cg, R, S, group, ah.t0, aw.t0, ah.nt, aw.nt,
                                      stride, g.Kg % kBK == 0, a_ld, kmajor, stream) !=
                hipSuccess)
                return MICONV_ERR_LAUNCH;
            ImgGemmArgs a{};
            a.M = g.Cg;
            a.Kred = kred;
            a.groups = group;
            a.A = wr;
            a.a_ld = a_ld;
            a.a_bytes = (uint32_t)((size_t)g.C * a_ld * fb);
            a.cin = g.Kg;
            a.src_h = g.P;
            a.src_w = g.Q;
            a.src_hw = g.P * g.Q;
            a.src_img_words = (uint32_t)yi;
            a.col_hw = make_fastdiv(ah.n * aw.n);
            a.col_w = make_fastdiv(aw.n);
            a.cstep = 1;
            a.coff_h = ah.d;
            a.coff_w = aw.d;
            a.tsign = -1;
            a.k_cin = make_fastdiv(g.Kg);
            a.k_tw = make_fastdiv(aw.nt > 0 ? aw.nt : 1);
            a.k_taps = make_fastdiv(ah.nt * aw.nt > 0 ? ah.nt * aw.nt : 1);
            a.bias = nullptr;
            a.out_img_stride = xi;
            a.out_hw = H * W;
            a.out_w = W;
            a.ostep = stride;
            a.ooff_h = ph;
            a.ooff_w = pw;
            const bool fast = g.Kg % kBK == 0;
            if (!*marked && mark(tl_events.before, stream) != hipSuccess)
                return MICONV_ERR_LAUNCH;
            *marked = true;
            for (int n0 = 0; n0 < n_images; n0 += nb) {
                const int n = n_images - n0 < nb ? n_images - n0 : nb;
                if (plan.img.halo >= 0) {  // stride 1: the one phase, flipped taps
                    int st = halo_gemm(plan.img, g.Cg, group, wr, a_ld, g.Kg, g.R, dy + n0 * yi, K,
                                       g.P, g.Q, H, W, g.C, n, ah.d, aw.d, true, nullptr,
                                       dx + n0 * xi, part, (long long)n_images * xi, stream);
                    if (st != MICONV_OK)
                        return st;
                    continue;
                }
                a.Ncol = n * ah.n * aw.n;
                a.src = dy + n0 * yi;
                a.src_bytes = (uint32_t)(n * yi * (long long)fb);
                a.out = split ? part : dx + n0 * xi;
                a.nsplit = plan.img.nsplit;
                a.kchunk = split ? plan.img.kchunk : a.Kred;
                a.split_stride = (long long)n_images * xi;
                int st = launch_status(launch_img_gemm(a, tile, fast, stream));
                if (st != MICONV_OK)
                    return st;
            }
        }
    return MICONV_OK;
}

int bwd_exec(const Geom &g, const BwdPlan &plan, const float *dy, const float *w, float *dx,
             void *ws, size_t ws_bytes, hipStream_t stream)
{
    const int N = g.N, C = g.C, H = g.H, W = g.W, K = g.K, R = g.R, S = g.S;
    const size_t fb = sizeof(float);
    Range r[3] = {{dy, (size_t)N * K * g.P * g.Q * fb, false},
                  {w, (size_t)K * g.Cg * R * S * fb, false},
                  {dx, (size_t)N * C * H * W * fb, true}};
    bool req[3] = {true, true, true};
    int st = check_buffers(r, 3, req, ws, ws_bytes, bwd_ws(g, plan));
    if (st != MICONV_OK || (st = check_device()) != MICONV_OK)
        return st;
    (void)hipGetLastError();
    if (plan.blocked)
        return bwd_blocked(g, plan, dy, w, dx, ws, stream);
    if (plan.bt)
        return ip_bwd_data(g, plan, dy, w, dx, ws, stream);

    const long long xi = (long long)C * H * W, yi = (long long)K * g.P * g.Q;
    bool marked = false;
    if (plan.xnb > 0) {
        // Explicit: per chunk of images, the transposed 1x1 GEMM writes the
        // column tensor (the backward-data of the 1x1 problem), then col2im.
        float *col = (float *)((char *)ws + align_up((size_t)C * R * S * pad16(g.Kg) * fb));
        for (int n0 = 0; n0 < N; n0 += plan.xnb) {
            const int n = N - n0 < plan.xnb ? N - n0 : plan.xnb;
            char *wsp = (char *)ws;
            if ((st = phase_gemms(one_by_one(g, n), plan, w, wsp, dy + n0 * yi, col, n, &marked,
                                  stream)) != MICONV_OK)
                return st;
            if (launch_col2im(col, dx + n0 * xi, n, C, H, W, R, S, g.st, g.pad, g.P, g.Q,
                              stream) != hipSuccess)
                return MICONV_ERR_LAUNCH;
        }
        return mark(tl_events.after, stream) == hipSuccess ? MICONV_OK : MICONV_ERR_LAUNCH;
    }
    char *wsp = (char *)ws;
    if ((st = phase_gemms(g, plan, w, wsp, dy, dx, N, &marked, stream)) != MICONV_OK)
        return st;
    if (mark(tl_events.after, stream) != hipSuccess)
        return MICONV_ERR_LAUNCH;
    if (plan.img.nsplit > 1)  // stride 1 only
        return launch_status(launch_splitk_bias_reduce((float *)wsp, plan.img.nsplit,
                                                       (long long)N * xi, (int)(N * xi),
                                                       nullptr, 1, 1, dx, stream));
    return MICONV_OK;
}

// Backward-weight launches over n images of geometry g (x from x, dy from
// dy), writing splits [split0, ...) of the partial sums; returns the status
// and advances split0.
int wgrad_launches(const Geom &g, const WgradPlan &p, const float *x, const float *dy, float *dw,
                   bool with_db, float *part, float *db_part, int n_images, int &split0,
                   hipStream_t stream)
{
    const size_t fb = sizeof(float);
    const long long xi = (long long)g.C * g.H * g.W, yi = (long long)g.K * g.P * g.Q;
    WgradArgs a;
    a.M = g.Kg;
    a.Ncol = g.Cg * g.R * g.S;
    a.groups = g.G;
    a.dy_img_words = (uint32_t)yi;
    a.x_img_words = (uint32_t)xi;
    a.Cg = g.Cg;
    a.H = g.H;
    a.W = g.W;
    a.HW = g.H * g.W;
    a.PQ = g.P * g.Q;
    a.stride = g.st;
    a.pad = g.pad;
    a.pix_pq = make_fastdiv(g.P * g.Q);
    a.pix_q = make_fastdiv(g.Q);
    a.n_rs = make_fastdiv(g.R * g.S);
    a.n_s = make_fastdiv(g.S);
    a.chunk = p.chunk;
    a.split_stride = (long long)g.K * a.Ncol;
    a.K = g.K;
    for (int n0 = 0; n0 < n_images; n0 += p.nb) {
        const int n = n_images - n0 < p.nb ? n_images - n0 : p.nb;
        a.Kred = n * a.PQ;
        a.nsplit = (a.Kred + p.chunk - 1) / p.chunk;
        a.dy = dy + n0 * yi;
        a.x = x + n0 * xi;
        a.dy_bytes = (uint32_t)(n * yi * (long long)fb);
        a.x_bytes = (uint32_t)(n * xi * (long long)fb);
        a.out = p.via_part ? part + (long long)split0 * a.split_stride : dw;
        a.db_part = with_db ? db_part + (long long)split0 * g.K : nullptr;
        int st = launch_status(launch_wgrad_gemm(a, p.tile, stream));
        if (st != MICONV_OK)
            return st;
        split0 += a.nsplit;
    }
    return MICONV_OK;
}

int wgrad_exec(const Geom &g, const WgradPlan &p, const float *x, const float *dy, float *dw,
               float *db, void *ws, size_t ws_bytes, hipStream_t stream)
{
    const int N = g.N, C = g.C, H = g.H, W = g.W, K = g.K, R = g.R, S = g.S;
    const size_t fb = sizeof(float);
    Range r[4] = {{x, (size_t)N * C * H * W * fb, false},
                  {dy, (size_t)N * K * g.P * g.Q * fb, false},
                  {dw, (size_t)K * g.Cg * R * S * fb, true},
                  {db, (size_t)K * fb, true}};
    bool req[4] = {true, true, true, false};
    int st = check_buffers(r, 4, req, ws, ws_bytes, wgrad_ws(g, p));
    if (st != MICONV_OK || (st = check_device()) != MICONV_OK)
        return st;
    (void)hipGetLastError();

    if (p.img >= 0) {
        // Inner product, dW [K][C] = sum over n of dy[n][k] x[n][c] as one
        // image GEMM: rows K from dy^T (m-major, the batch as its reduction
        // rows), columns C, the batch staged from x [N][C] read in place as N
        // channels of one 1 x C image; db = the batch sum of dy, fixed order.
        float *dyt = (float *)ws;
        if (launch_transpose(dy, dyt, N, K, stream) != hipSuccess ||
            mark(tl_events.before, stream) != hipSuccess)
            return MICONV_ERR_LAUNCH;
        ImgGemmArgs a{};
        a.M = K;
        a.Ncol = C;
        a.Kred = N;
        a.groups = 1;
        a.A = dyt;
        a.a_ld = N;
        a.a_bytes = (uint32_t)((size_t)K * N * fb);
        a.src = x;
        a.src_bytes = (uint32_t)((size_t)N * C * fb);
        a.cin = N;
        a.src_h = 1;
        a.src_w = C;
        a.src_hw = C;
        a.src_img_words = (uint32_t)((size_t)N * C);
        a.col_hw = make_fastdiv(C);
        a.col_w = make_fastdiv(C);
        a.cstep = 1;
        a.tsign = 1;
        a.k_cin = make_fastdiv(N);
        a.k_tw = make_fastdiv(1);
        a.k_taps = make_fastdiv(1);
        a.out = dw;
        a.out_hw = C;
        a.out_w = C;
        a.ostep = 1;
        a.nsplit = 1;
        a.kchunk = N;
        if ((st = launch_status(launch_img_gemm(a, p.img, true, stream))) != MICONV_OK)
            return st;
        if (mark(tl_events.after, stream) != hipSuccess)
            return MICONV_ERR_LAUNCH;
        if (db && (st = launch_status(launch_splitk_reduce(dy, N, K, K, db, 0, 0, stream))) !=
                      MICONV_OK)
            return st;
        return MICONV_OK;
    }
    float *part = (float *)ws;
    float *db_part = (float *)((char *)ws + p.part_bytes);
    float *tail = (float *)((char *)ws + p.part_bytes + p.bias_bytes);
    int split0 = 0;
    if (p.bt) {
        // Inner product: both operands transposed to [C][N] and [K][N], one image.
        float *dyt = (float *)((char *)tail + align_up((size_t)C * N * fb));
        if (launch_transpose(x, tail, N, C, stream) != hipSuccess ||
            launch_transpose(dy, dyt, N, K, stream) != hipSuccess ||
            mark(tl_events.before, stream) != hipSuccess)
            return MICONV_ERR_LAUNCH;
        if ((st = wgrad_launches(batch_columns(g), p, tail, dyt, dw, db != nullptr, part, db_part,
                                 1, split0, stream)) != MICONV_OK)
            return st;
    } else if (p.halo_tw) {
        WgradHaloArgs h{};
        h.Kg = g.Kg;
        h.Cg = g.Cg;
        h.groups = g.G;
        h.K = K;
        h.dy = dy;
        h.x = x;
        h.dy_bytes = (uint32_t)((size_t)N * K * g.P * g.Q * fb);
        h.x_bytes = (uint32_t)((size_t)N * C * H * W * fb);
        h.dy_img_words = (uint32_t)((size_t)K * g.P * g.Q);
        h.x_img_words = (uint32_t)((size_t)C * H * W);
        h.H = H;
        h.W = W;
        h.P = g.P;
        h.Q = g.Q;
        h.TW = p.halo_tw;
        h.CT = p.halo_ct;
        h.db = p.halo_db;
        const int tr = kHaloCols / p.halo_tw;
        h.row_blocks = (g.P + tr - 1) / tr;
        h.col_segs = (g.Q + p.halo_tw - 1) / p.halo_tw;
        h.nimg = N;
        // x halo origin (p0 - pad, q0 - pad); for 16-byte loads the
        // columns start at a multiple of 4.
        h.row0 = -g.pad;
        h.col0 = p.halo_tw == 14 ? -g.pad : -((g.pad + 3) / 4) * 4;
        h.slack = -g.pad - h.col0;
        h.chunk = p.chunk;
        h.nsplit = p.nsplit;
        h.out = part;
        h.split_stride = (long long)K * g.Cg * 9;
        h.db_part = db ? db_part : nullptr;
        if (mark(tl_events.before, stream) != hipSuccess)
            return MICONV_ERR_LAUNCH;
        if ((st = launch_status(launch_wgrad_halo(h, stream))) != MICONV_OK)
            return st;
    } else if (p.xnb > 0) {
        // Explicit: im2col of a chunk of images, then the 1x1 problem over the
        // columns, whose dw[k][c'] is dw[k][c][r][s].
        if (mark(tl_events.before, stream) != hipSuccess)
            return MICONV_ERR_LAUNCH;
        const long long xi = (long long)C * H * W, yi = (long long)K * g.P * g.Q;
        for (int n0 = 0; n0 < N; n0 += p.xnb) {
            const int n = N - n0 < p.xnb ? N - n0 : p.xnb;
            if (launch_im2col(x + n0 * xi, tail, n, C, H, W, R, S, g.st, g.pad, g.P, g.Q,
                              stream) != hipSuccess)
                return MICONV_ERR_LAUNCH;
            if ((st = wgrad_launches(one_by_one(g, n), p, tail, dy + n0 * yi, dw, db != nullptr,
                                     part, db_part, n, split0, stream)) != MICONV_OK)
                return st;
        }
    } else {
        if (mark(tl_events.before, stream) != hipSuccess)
            return MICONV_ERR_LAUNCH;
        if ((st = wgrad_launches(g, p, x, dy, dw, db != nullptr, part, db_part, N, split0,
                                 stream)) != MICONV_OK)
            return st;
    }
    if (mark(tl_events.after, stream) != hipSuccess)
        return MICONV_ERR_LAUNCH;
    // Tap-ordered partials go back to dw's [k][c][r][s] (a 1x1 problem has one tap).
    const int taps = p.xnb > 0 || p.bt ? 1 : R * S;
    const int ncol = g.Cg * R * S;
    const bool tap_order = p.halo_tw || is_tap_tile(p.tile);
    if (p.via_part &&
        (st = launch_status(launch_splitk_reduce(part, p.nsplit, (long long)K * ncol, K * ncol,
                                                 dw, tap_order ? taps : 0,
                                                 tap_order ? ncol / taps : 0, stream))) !=
            MICONV_OK)
        return st;
    if (db && (st = launch_status(launch_splitk_reduce(db_part, p.nsplit, K, K, db, 0, 0,
                                                       stream))) != MICONV_OK)
        return st;
    return MICONV_OK;
}

// Number, workspace, name and execution of candidate `index` of a pass.
int candidate_count(int pass, const Geom &g)
{
    switch (pass) {
    case MICONV_PASS_FWD: {
        std::vector<ImgPlan> c;
        fwd_candidates(g, c);
        return (int)c.size();
    }
    case MICONV_PASS_BWD_DATA: {
        std::vector<BwdPlan> c;
        bwd_candidates(g, c);
        return (int)c.size();
    }
    case MICONV_PASS_BWD_WEIGHT: {
        std::vector<WgradPlan> c;
        wgrad_candidates(g, c);
        return (int)c.size();
    }
    default:
        return MICONV_ERR_PASS;
    }
}

size_t candidate_ws(int pass, const Geom &g, int index)
{
    switch (pass) {
    case MICONV_PASS_FWD:
        return fwd_ws(g, pick(fwd_rule(g), index, fwd_candidates, g));
    case MICONV_PASS_BWD_DATA:
        return bwd_ws(g, pick(bwd_rule(g), index, bwd_candidates, g));
    case MICONV_PASS_BWD_WEIGHT:
        return wgrad_ws(g, pick(wgrad_rule(g), index, wgrad_candidates, g));
    default:
        return 0;
    }
}

// The largest workspace over the candidates of a pass.
size_t max_candidate_ws(int pass, const Geom &g)
{
    size_t need = 0;
    switch (pass) {
    case MICONV_PASS_FWD: {
        std::vector<ImgPlan> c;
        fwd_candidates(g, c);
        for (const ImgPlan &p : c)
            need = std::max(need, fwd_ws(g, p));
        break;
    }
    case MICONV_PASS_BWD_DATA: {
        std::vector<BwdPlan> c;
        bwd_candidates(g, c);
        for (const BwdPlan &p : c)
            need = std::max(need, bwd_ws(g, p));
        break;
    }
    case MICONV_PASS_BWD_WEIGHT: {
        std::vector<WgradPlan> c;
        wgrad_candidates(g, c);
        for (const WgradPlan &p : c)
            need = std::max(need, wgrad_ws(g, p));
        break;
    }
    default:
        break;
    }
    return need;
}

// Tensors of conv_tune: fwd (x, w, b | y), bwd-data (dy, w, - | dx),
// bwd-weight (x, dy, - | dw, db).
struct TuneBuffers {
    const float *in0, *in1, *in2;
    float *out0, *out1;
};

int candidate_run(int pass, const Geom &g, int index, const TuneBuffers &t, void *ws,
                  size_t ws_bytes, hipStream_t stream)
{
    switch (pass) {
    case MICONV_PASS_FWD:
        return fwd_exec(g, pick(fwd_rule(g), index, fwd_candidates, g), t.in0, t.in1, t.in2,
                        t.out0, ws, ws_bytes, stream);
    case MICONV_PASS_BWD_DATA:
        return bwd_exec(g, pick(bwd_rule(g), index, bwd_candidates, g), t.in0, t.in1, t.out0, ws,
                        ws_bytes, stream);
    case MICONV_PASS_BWD_WEIGHT:
        return wgrad_exec(g, pick(wgrad_rule(g), index, wgrad_candidates, g), t.in0, t.in1,
                          t.out0, t.out1, ws, ws_bytes, stream);
    default:
        return MICONV_ERR_PASS;
    }
}

// ------------------------------------------------------------ pooling
// Output extent of a pooling window along one axis (Caffe's rule: ceil,
// less one when pad > 0 and the last window would start at or past
// in + pad); 0 when the window does not fit.
int pool_extent(int in, int filt, int stride, int pad)
{
    long long span = (long long)in + 2LL * pad - filt;
    if (span < 0)
        return 0;
    long long out = (span + stride - 1) / stride + 1;
    if (pad > 0 && (out - 1) * stride >= (long long)in + pad)
        out--;
    return (int)out;
}

struct PoolGeom {
    int N, C, H, W, R, S, st, pad, P, Q;
};

int make_pool(int mode, int N, int C, int H, int W, int R, int S, int stride, int pad,
              PoolGeom *g)
{
    if (mode != MICONV_POOL_MAX && mode != MICONV_POOL_AVG)
        return MICONV_ERR_MODE;
    if (N < 1 || C < 1 || H < 1 || W < 1 || R < 1 || S < 1 || stride < 1 || pad < 0 ||
        pad >= R || pad >= S || H > 32767 || W > 32767 || R > 32767 || S > 32767)
        return MICONV_ERR_SHAPE;
    const int P = pool_extent(H, R, stride, pad), Q = pool_extent(W, S, stride, pad);
    if (P < 1 || Q < 1)
        return MICONV_ERR_SHAPE;
    // Without padding the rounded-up count can put the last window wholly past
    // the image (stride > window): a window with no input element.
    if ((long long)(P - 1) * stride - pad >= H || (long long)(Q - 1) * stride - pad >= W)
        return MICONV_ERR_SHAPE;
    if ((long long)N * C * H * W > kMaxElems || (long long)N * C * P * Q > kMaxElems)
        return MICONV_ERR_SHAPE;
    *g = PoolGeom{N, C, H, W, R, S, stride, pad, P, Q};
    return MICONV_OK;
}

// ------------------------------------------------------------ fixed scratch
// Workspace of conv_bwd_weight_noalloc: a file-scope device array, one copy
// per GPU (each device holds it from module load until the process ends).
// In host code `scratch` is only a host-side stand-in for the symbol; its
// device address is read per device with hipGetSymbolAddress, and that
// address is what the kernels receive.
constexpr size_t kScratchBytes = (size_t)MICONV_NOALLOC_SCRATCH_BYTES;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

std::mutex g_scratch_mu;
void *g_scratch_dev[64];  // device address of `scratch`, per device id

// Device address of this device's scratch array (looked up on the first call
// on each device, with that device current).
int scratch_address(void **out)
{
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64)
        return MICONV_ERR_DEVICE;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_dev[dev]) {
        void *ptr = nullptr;
        if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || !ptr)
            return MICONV_ERR_LAUNCH;
        g_scratch_dev[dev] = ptr;
    }
    *out = g_scratch_dev[dev];
    return MICONV_OK;
}

}  // namespace
}  // namespace miconv

using namespace miconv;

extern "C" {

int conv_output_size(int H, int W, int R, int S, int stride, int pad, int *P, int *Q)
{
    if (!P || !Q)
        return MICONV_ERR_NULL;
    if (H < 1 || W < 1 || R < 1 || S < 1 || stride < 1 || pad < 0)
        return MICONV_ERR_SHAPE;
    int p = out_extent(H, R, stride, pad), q = out_extent(W, S, stride, pad);
    if (p < 1 || q < 1)
        return MICONV_ERR_SHAPE;
    *P = p;
    *Q = q;
    return MICONV_OK;
}

size_t conv_workspace_size(int pass, int N, int C, int H, int W, int K, int R, int S,
                           int stride, int pad, int group)
{
    Geom g;
    if (make_geom(N, C, H, W, K, R, S, stride, pad, group, &g) != MICONV_OK)
        return 0;
    if (pass < MICONV_PASS_FWD || pass > MICONV_PASS_BWD_WEIGHT)
        return 0;
    // The largest need over the shape's candidate plans, so that a size taken
    // now stays sufficient whatever plan conv_plan_set or conv_tune stores
    // for the shape later (from this or another thread).
    return max_candidate_ws(pass, g);
}

int conv_set_timing_events(hipEvent_t before, hipEvent_t after)
{
    if ((before == nullptr) != (after == nullptr))
        return MICONV_ERR_NULL;
    tl_events.before = before;
    tl_events.after = after;
    return MICONV_OK;
}

const char *conv_error_string(int status)
{
    switch (status) {
    case MICONV_OK: return "success";
    case MICONV_ERR_SHAPE: return "invalid shape, stride, padding or group";
    case MICONV_ERR_NULL: return "a required pointer is NULL";
    case MICONV_ERR_WORKSPACE: return "workspace missing or smaller than conv_workspace_size()";
    case MICONV_ERR_ALIAS: return "an output overlaps an input, another output or the workspace";
    case MICONV_ERR_ALIGN: return "a tensor or workspace pointer is not 16-byte aligned";
    case MICONV_ERR_DEVICE: return "no current HIP device, or it is not gfx950";
    case MICONV_ERR_LAUNCH: return "kernel launch failed";
    case MICONV_ERR_PASS: return "unknown pass id";
    case MICONV_ERR_PLAN: return "plan index out of range";
    case MICONV_ERR_MODE: return "unknown pooling mode";
    case MICONV_ERR_SCRATCH:
        return "the plan needs more workspace than the library's fixed device scratch holds";
    default: return "unknown status";
    }
}

int conv_fwd(int N, int C, int H, int W, int K, int R, int S, int stride, int pad, int group,
             const float *x, const float *w, const float *b, float *y, void *ws, size_t ws_bytes,
             hipStream_t stream)
{
    Geom g;
    int st = make_geom(N, C, H, W, K, R, S, stride, pad, group, &g);
    if (st != MICONV_OK)
        return st;
    return fwd_exec(g, fwd_current(g), x, w, b, y, ws, ws_bytes, stream);
}

int conv_bwd_data(int N, int C, int H, int W, int K, int R, int S, int stride, int pad,
                  int group, const float *dy, const float *w, float *dx, void *ws,
                  size_t ws_bytes, hipStream_t stream)
{
    Geom g;
    int st = make_geom(N, C, H, W, K, R, S, stride, pad, group, &g);
    if (st != MICONV_OK)
        return st;
    return bwd_exec(g, bwd_current(g), dy, w, dx, ws, ws_bytes, stream);
}

int conv_bwd_weight(int N, int C, int H, int W, int K, int R, int S, int stride, int pad,
                    int group, const float *x, const float *dy, float *dw, float *db, void *ws,
                    size_t ws_bytes, hipStream_t stream)
{
    Geom g;
    int st = make_geom(N, C, H, W, K, R, S, stride, pad, group, &g);
    if (st != MICONV_OK)
        return st;
    return wgrad_exec(g, wgrad_current(g), x, dy, dw, db, ws, ws_bytes, stream);
}

int conv_bwd_weight_noalloc(int N, int C, int H, int W, int K, int R, int S, int stride,
                            int pad, int group, const float *x, const float *dy, float *dw,
                            float *db, hipStream_t stream)
{
    Geom g;
    int st = make_geom(N, C, H, W, K, R, S, stride, pad, group, &g);
    if (st != MICONV_OK)
        return st;
    const WgradPlan p = wgrad_current(g);
    if (wgrad_ws(g, p) > kScratchBytes)
        return MICONV_ERR_SCRATCH;
    if ((st = check_device()) != MICONV_OK)
        return st;
    void *ws = nullptr;
    if ((st = scratch_address(&ws)) != MICONV_OK)
        return st;
    // Every word of the scratch that the plan's kernels read (split
    // partials, bias partials, transposed operands) is written earlier in the
    // same call, so nothing needs clearing between calls.
    return wgrad_exec(g, p, x, dy, dw, db, ws, kScratchBytes, stream);
}

int conv_plan_count(int pass, int N, int C, int H, int W, int K, int R, int S, int stride,
                    int pad, int group)
{
    Geom g;
    int st = make_geom(N, C, H, W, K, R, S, stride, pad, group, &g);
    return st != MICONV_OK ? st : candidate_count(pass, g);
}

int conv_plan_get(int pass, int N, int C, int H, int W, int K, int R, int S, int stride, int pad,
                  int group)
{
    Geom g;
    int st = make_geom(N, C, H, W, K, R, S, stride, pad, group, &g);
    if (st != MICONV_OK)
        return st;
    if (pass < MICONV_PASS_FWD || pass > MICONV_PASS_BWD_WEIGHT)
        return MICONV_ERR_PASS;
    return plan_index(pass, g);
}

int conv_plan_set(int pass, int N, int C, int H, int W, int K, int R, int S, int stride, int pad,
                  int group, int index)
{
    Geom g;
    int st = make_geom(N, C, H, W, K, R, S, stride, pad, group, &g);
    if (st != MICONV_OK)
        return st;
    const int n = candidate_count(pass, g);
    if (n < 0)
        return n;
    if (index < 0 || index >= n)
        return MICONV_ERR_PLAN;
    plan_store(pass, g, index);
    return MICONV_OK;
}

int conv_plan_clear(void)
{
    std::lock_guard<std::mutex> lock(g_plan_mu);
    g_plans.clear();
    g_plan_entries.store(0, std::memory_order_release);
    return MICONV_OK;
}

int conv_plan_name(int pass, int N, int C, int H, int W, int K, int R, int S, int stride,
                   int pad, int group, int index, char *buf, size_t len)
{
    Geom g;
    int st = make_geom(N, C, H, W, K, R, S, stride, pad, group, &g);
    if (st != MICONV_OK)
        return st;
    if (!buf || len == 0)
        return MICONV_ERR_NULL;
    const int n = candidate_count(pass, g);
    if (n < 0)
        return n;
    if (index < 0 || index >= n)
        return MICONV_ERR_PLAN;
    switch (pass) {
    case MICONV_PASS_FWD:
        fwd_name(pick(fwd_rule(g), index, fwd_candidates, g), buf, len);
        break;
    case MICONV_PASS_BWD_DATA:
        bwd_name(pick(bwd_rule(g), index, bwd_candidates, g), buf, len);
        break;
    default:
        wgrad_name(pick(wgrad_rule(g), index, wgrad_candidates, g), buf, len);
        break;
    }
    return MICONV_OK;
}

size_t conv_plan_workspace_size(int pass, int N, int C, int H, int W, int K, int R, int S,
                                int stride, int pad, int group, int index)
{
    Geom g;
    if (make_geom(N, C, H, W, K, R, S, stride, pad, group, &g) != MICONV_OK)
        return 0;
    const int n = candidate_count(pass, g);
    if (n < 0 || index < 0 || index >= n)
        return 0;
    return candidate_ws(pass, g, index);
}

int conv_tune(int pass, int N, int C, int H, int W, int K, int R, int S, int stride, int pad,
              int group, const float *in0, const float *in1, const float *in2, float *out0,
              float *out1, void *ws, size_t ws_bytes, int reps, hipStream_t stream,
              int *chosen)
{
    Geom g;
    int st = make_geom(N, C, H, W, K, R, S, stride, pad, group, &g);
    if (st != MICONV_OK)
        return st;
    const int n = candidate_count(pass, g);
    if (n < 0)
        return n;
    if (reps < 1)
        reps = 1;
    const TuneBuffers t{in0, in1, pass == MICONV_PASS_FWD ? in2 : nullptr, out0,
                        pass == MICONV_PASS_BWD_WEIGHT ? out1 : nullptr};
    // The pass's own timing events stay quiet while candidates run.
    const TimingEvents saved = tl_events;
    tl_events = TimingEvents{};
    std::vector<int> fit;
    for (int i = 0; i < n; i++)
        if (candidate_ws(pass, g, i) <= ws_bytes)
            fit.push_back(i);
    std::vector<hipEvent_t> ev(2 * reps, nullptr);
    for (auto &e : ev)
        if (st == MICONV_OK && hipEventCreate(&e) != hipSuccess)
            st = MICONV_ERR_LAUNCH;
    // Every candidate runs once untimed (this also brings the clocks up),
    // then two rounds in turn time each candidate's runs one by one; its
    // score is the smaller of its two median times, so that neither the
    // order of the candidates nor a stray slow run decides.
    std::vector<float> score(n, 0.f);
    for (int round = -1; round < 2 && st == MICONV_OK; round++)
        for (int i : fit) {
            if (round < 0) {
                if ((st = candidate_run(pass, g, i, t, ws, ws_bytes, stream)) != MICONV_OK)
                    break;
                continue;
            }
            for (int r = 0; r < reps && st == MICONV_OK; r++) {
                if (hipEventRecord(ev[2 * r], stream) != hipSuccess)
                    st = MICONV_ERR_LAUNCH;
                else if ((st = candidate_run(pass, g, i, t, ws, ws_bytes, stream)) == MICONV_OK &&
                         hipEventRecord(ev[2 * r + 1], stream) != hipSuccess)
                    st = MICONV_ERR_LAUNCH;
            }
            std::vector<float> ms(reps, 0.f);
            for (int r = 0; r < reps && st == MICONV_OK; r++)
                if (hipEventSynchronize(ev[2 * r + 1]) != hipSuccess ||
                    hipEventElapsedTime(&ms[r], ev[2 * r], ev[2 * r + 1]) != hipSuccess)
                    st = MICONV_ERR_LAUNCH;
            if (st != MICONV_OK)
                break;
            std::sort(ms.begin(), ms.end());
            const float med = ms[reps / 2];
            score[i] = round == 0 ? med : std::min(score[i], med);
        }
    for (auto &e : ev)
        if (e)
            (void)hipEventDestroy(e);
    tl_events = saved;
    if (st != MICONV_OK)
        return st;
    if (fit.empty())
        return MICONV_ERR_WORKSPACE;
    int best = fit[0];
    for (int i : fit)
        if (score[i] < score[best])
            best = i;
    plan_store(pass, g, best);
    if (chosen)
        *chosen = best;
    // Leave the chosen plan's results in the outputs.
    tl_events = TimingEvents{};
    st = candidate_run(pass, g, best, t, ws, ws_bytes, stream);
    tl_events = saved;
    return st;
}

int pool_output_size(int H, int W, int R, int S, int stride, int pad, int *P, int *Q)
{
    if (!P || !Q)
        return MICONV_ERR_NULL;
    PoolGeom g;
    int st = make_pool(MICONV_POOL_MAX, 1, 1, H, W, R, S, stride, pad, &g);
    if (st != MICONV_OK)
        return st;
    *P = g.P;
    *Q = g.Q;
    return MICONV_OK;
}

int pool_fwd(int mode, int N, int C, int H, int W, int R, int S, int stride, int pad,
             const float *x, float *y, int *mask, hipStream_t stream)
{
    PoolGeom g;
    int st = make_pool(mode, N, C, H, W, R, S, stride, pad, &g);
    if (st != MICONV_OK)
        return st;
    const bool max_mode = mode == MICONV_POOL_MAX;
    const size_t in = (size_t)N * C * H * W * sizeof(float);
    const size_t out = (size_t)N * C * g.P * g.Q * sizeof(float);
    Range r[3] = {{x, in, false}, {y, out, true}, {max_mode ? mask : nullptr, out, true}};
    bool req[3] = {true, true, false};
    if ((st = check_buffers(r, 3, req, nullptr, 0, 0)) != MICONV_OK)
        return st;
    if ((st = check_device()) != MICONV_OK)
        return st;
    (void)hipGetLastError();
    if (mark(tl_events.before, stream) != hipSuccess)
        return MICONV_ERR_LAUNCH;
    if ((st = launch_status(launch_pool_fwd(max_mode, x, y, max_mode ? mask : nullptr, N, C, H,
                                            W, R, S, stride, pad, g.P, g.Q, stream))) !=
        MICONV_OK)
        return st;
    return mark(tl_events.after, stream) == hipSuccess ? MICONV_OK : MICONV_ERR_LAUNCH;
}

int pool_bwd(int mode, int N, int C, int H, int W, int R, int S, int stride, int pad,
             const float *dy, const int *mask, float *dx, hipStream_t stream)
{
    PoolGeom g;
    int st = make_pool(mode, N, C, H, W, R, S, stride, pad, &g);
    if (st != MICONV_OK)
        return st;
    const bool max_mode = mode == MICONV_POOL_MAX;
    const size_t in = (size_t)N * C * H * W * sizeof(float);
    const size_t out = (size_t)N * C * g.P * g.Q * sizeof(float);
    Range r[3] = {{dy, out, false}, {max_mode ? mask : nullptr, out, false}, {dx, in, true}};
    bool req[3] = {true, max_mode, true};
    if ((st = check_buffers(r, 3, req, nullptr, 0, 0)) != MICONV_OK)
        return st;
    if ((st = check_device()) != MICONV_OK)
        return st;
    (void)hipGetLastError();
    if (mark(tl_events.before, stream) != hipSuccess)
        return MICONV_ERR_LAUNCH;
    if ((st = launch_status(launch_pool_bwd(max_mode, dy, max_mode ? mask : nullptr, dx, N, C,
                                            H, W, R, S, stride, pad, g.P, g.Q, stream))) !=
        MICONV_OK)
        return st;
    return mark(tl_events.after, stream) == hipSuccess ? MICONV_OK : MICONV_ERR_LAUNCH;
}

}  // extern "C"
