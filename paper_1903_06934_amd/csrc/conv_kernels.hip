// HIP kernels for gfx950 (CDNA4): implicit-GEMM convolution passes on fp32
// MFMA, filter packing, split-K reduction and the bias gradient.
//
// GEMM core: a workgroup of WM x WN waves computes a BM x BN tile of C with
// v_mfma_f32_16x16x4f32 (each wave owns a (BM/WM) x (BN/WN) sub-tile made of
// 16x16 accumulator blocks).
// Operands go from HBM straight into LDS with buffer_load_dword ... lds (no
// register staging); out-of-range elements read zero through the buffer
// range check, so padding and ragged tiles need no branches.
#include "internal.h"

namespace miconv {

// v_mfma_f32_16x16x4f32 operand layout (64 lanes): A (16 x 4): lane l holds
// A[l % 16][l / 16]; B (4 x 16): B[l / 16][l % 16]; D (16 x 16): lane l,
// register v holds D[4 (l / 16) + v][l % 16].
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
#define LDS_AS __attribute__((address_space(3)))
constexpr int MF = 16;  // accumulator block edge

__device__ __forceinline__ int acc_row(int v, int lane) { return 4 * (lane >> 4) + v; }

// Two aligned words of LDS as one ds_read_b64 (word: even index into base).
// The read is volatile so that the compiler does not fuse two of them into
// one ds_read2_b64: on gfx950 a two-address LDS read (ds_read2_b32,
// ds_read2_b64) at the operand patterns used here (16 rows a fixed stride
// apart, two words per lane) costs 4-8 bank-conflict cycles where the
// single ds_read_b64 costs none.
typedef LDS_AS const volatile f32x2 lds_f32x2;
__device__ __forceinline__ f32x2 lds_b64(const float *base, int word)
{
    return *(lds_f32x2 *)(base + word);
}
// A per-lane word offset hidden from the optimizer, so that the reads off
// base + offset (which keep base's provenance: the compiler still knows
// which LDS array they read) share one address register with their
// constants in the instruction's offset field instead of each read's full
// address being precomputed, loop-invariant, into a register of its own.
__device__ __forceinline__ int opaque(int v)
{
    __asm__ volatile("" : "+v"(v));
    return v;
}

__device__ __forceinline__ f32x4 mfma16(float a, float b, f32x4 c)
{
    return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}


// ---------------------------------------------------------------------------
// Operand staging: buffer loads that write straight into LDS.
//
// `buffer_load_dword ... lds` moves one dword per lane from a buffer into LDS
// at (M0 + 4 * lane): a wave fills 64 consecutive words of an LDS row, with no
// register staging and no ds_write.  A lane whose byte offset lies outside the
// buffer's range reads 0 (hardware range checking), which is how padding,
// ragged tiles and the reduction tail are zero-filled without branches.
// Every buffer a launch reads is below 2^31 bytes, so a valid offset never
// has bit 31 set and OR-ing bit 31 into an offset makes it out of range
// (for every dword of a multi-dword load too).
// ---------------------------------------------------------------------------

constexpr uint32_t kOob = 0x80000000u;  // beyond any buffer of < 2^31 bytes

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void *p, uint32_t bytes)
{
    // Raw buffer (stride 0), dword 3 = 0x00020000 for the gfx9 family.
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(p), (short)0, (int)bytes,
                                             0x00020000);
}

__device__ __forceinline__ void lds_load(__amdgpu_buffer_rsrc_t r, float *lds_row, uint32_t voff)
{
    __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (LDS_AS void *)lds_row, 4, voff, 0, 0, 0);
}

// The same raw buffer descriptor as four dwords, for inline assembly.
typedef int i32x4 __attribute__((ext_vector_type(4)));
__device__ __forceinline__ i32x4 rsrc_words(const void *p, uint32_t bytes)
{
    const uint64_t a = (uint64_t)p;
    i32x4 r;
    r[0] = __builtin_amdgcn_readfirstlane((int)(uint32_t)a);
    r[1] = __builtin_amdgcn_readfirstlane((int)(uint32_t)(a >> 32));
    r[2] = __builtin_amdgcn_readfirstlane((int)bytes);
    r[3] = 0x00020000;
    return r;
}

// buffer_load_dwordx4 into registers, issued as inline assembly so that the
// compiler does not track it as a pending memory operation: its own waits
// (which it places conservatively across the rotating register stages,
// draining the pipeline) are then not generated.  The caller owns the wait
// (s_waitcnt vmcnt) before the result is read, and the result must reach its
// only consumers (MFMAs after that wait) without compiler-made copies:
// paper_1903_06934_amd/isa_check.py verifies both on the built code.
__device__ __forceinline__ f32x4 load4_untracked(i32x4 rsrc, uint32_t voff)
{
    f32x4 v;
    // Early-clobber output: the destination never doubles as the address
    // register, so only these loads write the destination registers.
    asm volatile("buffer_load_dwordx4 %0, %1, %2, 0 offen" : "=&v"(v) : "v"(voff), "s"(rsrc));
    return v;
}

// Out-of-range bit for a lane whose element is absent.
__device__ __forceinline__ uint32_t oob_mask(bool ok) { return ok ? 0u : kOob; }

// Workgroup id -> tile id, so that the workgroups the dispatcher sends to
// one XCD (hardware ids congruent mod 8) own a contiguous range of tiles:
// neighbouring tiles share operand rows in that XCD's L2.
__device__ __forceinline__ int xcd_tile(int hw, int total)
{
    int xcd = hw & 7, idx = hw >> 3;
    int per = total >> 3, rem = total & 7;
    return xcd * per + min(xcd, rem) + idx;
}

// ---------------------------------------------------------------------------
// Forward / backward-data implicit GEMM (see ImgGemmArgs).
//
// Workgroup = WM x WN waves computing a BM x BN tile on the 16x16x4 MFMA; each
// wave owns a (BM/WM) x (BN/WN) block of 16x16 accumulators.  The reduction is
// walked in 16-row slices; MFMA lane group kr (lanes 16 kr .. 16 kr + 15) takes
// reduction rows 4 kr .. 4 kr + 3 of a slice, one per MFMA step.
//
// A (the packed filter) goes straight into registers when the waves split
// the tile's rows (WM > 1): packed m-major with each filter's reduction rows
// contiguous, a lane's A[m][4 kr .. 4 kr + 3] is one aligned
// buffer_load_dwordx4.  With one wave row (WM == 1, the 16-row tile)
// every wave needs the same A rows, so A is packed k-major and shared through
// LDS like B (one wave-load = 64 consecutive rows m of one reduction row).  B (the
// gathered image) is shared by the waves of the workgroup through LDS: a
// wave-load (buffer_load_dword ... lds) fills one LDS row of 64 pixels of one
// reduction row, coalesced along the pixel row; rows are padded to BN + 4
// words so that the four lane groups of a ds_read_b32, which read rows 4
// apart, hit distinct banks.  k is the same for the whole wave, so the
// (tap, channel) decode of k is scalar work.
// FAST: cin % 16 == 0, so a slice lies inside one filter tap; the spatial
// bounds test and offset are then computed once per slice and column.
// ONE (with FAST, 64-column tiles): the 1x1 direct GEMM -- one tap, stride 1,
// no offset, the source pixel index equal to the column's pixel index and
// pixels per image a multiple of 4 -- so each source row of a slice is 64
// consecutive pixels in 16 aligned groups of 4 that never straddle an image.
// B is then staged with 16-byte direct-to-LDS loads (buffer_load_dwordx4 ...
// lds): one wave-load fills 4 rows x 64 columns, a quarter of the load
// instructions of the one-dword gather.  LDS layout of a stage: 4-row
// groups of 256 words plus 16 words of padding, so that the four lane groups
// of a ds_read_b32 (rows 4 apart, i.e. one row in each group) hit distinct
// banks.
//
// Pipeline: three stages (LDS buffers for B, and for A or register sets for
// A); slices t + 1 and t + 2 are in flight while slice t computes.
// ---------------------------------------------------------------------------
template <int BM, int BN, int BK, int WM, int WN, int PAD, bool FAST, int NST, bool ONE = false>
__global__ __launch_bounds__(64 * WM * WN) void img_gemm_kernel(const ImgGemmArgs a)
{
    constexpr int NW = WM * WN;
    constexpr int TM = BM / WM, TN = BN / WN;
    constexpr int FM = TM / 16, FN = TN / 16;
    constexpr bool ASH = WM == 1;          // A shared through LDS
    constexpr int HA = ASH ? (BM + 63) / 64 : 1, HB = BN / 64;  // 64-wide row segments
    constexpr int LA = ASH ? BK * HA / NW : FM;  // A loads per wave and slice
    // B wave-loads per slice and wave; when the waves do not divide the BK
    // rows (3-wave tiles, one 64-wide segment), the waves with a row fewer
    // issue one more load into a spare LDS row (out-of-range offset: it
    // reads zero and touches no memory), so every wave issues LB loads.
    // ONE: BK / 4 wave-loads of 4 rows x 64 columns per slice; waves with a
    // load fewer issue one into a spare group (out of range: reads zero).
    constexpr int NG = BK / 4;
    constexpr int LB = ONE ? (NG + NW - 1) / NW : (BK * HB + NW - 1) / NW;
    constexpr int BROWS = ONE ? NG + (NG % NW ? 1 : 0) : BK + ((BK * HB) % NW ? 1 : 0);
    constexpr int LDA = 64 * HA + PAD, LDB = ONE ? 4 * 64 + 16 : BN + PAD;
    static_assert(BK == 16 && NST == 3, "16-row slices, 3 stages");
    static_assert(BN % 64 == 0 && TM % 16 == 0 && TN % 16 == 0, "tile");
    static_assert(BK % NW == 0 || HB == 1, "uneven B rows need one segment per row");
    static_assert(!ASH || (BK * HA) % NW == 0, "A rows per wave");
    static_assert(!ONE || (FAST && HB == 1 && !ASH), "1x1 direct GEMM: 64-column tiles");

    // One distinct array per pipeline stage, so that the compiler's alias
    // analysis can tell an in-flight direct-to-LDS load from a read of
    // another stage's buffer (it would otherwise wait for every load).
    // B element (row k, column n) lies at [k][n], or for ONE at
    // [k / 4][(k % 4) * 64 + n].
    __shared__ float As0[ASH ? BK : 1][LDA], As1[ASH ? BK : 1][LDA], As2[ASH ? BK : 1][LDA];
    __shared__ __attribute__((aligned(16))) float Bs0[BROWS][LDB], Bs1[BROWS][LDB],
        Bs2[BROWS][LDB];

    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int wm = wave % WM, wn = wave / WM;
    const int mtiles = (a.M + BM - 1) / BM;
    const int ntiles = (a.Ncol + BN - 1) / BN;
    const int tiles = mtiles * ntiles;
    const int lin = xcd_tile(blockIdx.x, tiles * a.groups * a.nsplit);
    const int split = lin / (tiles * a.groups);
    const int rest = lin - split * tiles * a.groups;
    const int g = rest / tiles, tile = rest - g * tiles;
    const int mt = tile % mtiles, nt = tile / mtiles;
    const int m0 = mt * BM, n0 = nt * BN;
    const int kbeg = split * a.kchunk;
    const int kend = min(a.Kred, kbeg + a.kchunk);
    const int kr = lane >> 4, lc = lane & 15;

    const i32x4 rAw = rsrc_words(a.A, a.a_bytes);
    const __amdgpu_buffer_rsrc_t rA = make_rsrc(a.A, a.a_bytes);
    const __amdgpu_buffer_rsrc_t rB = make_rsrc(a.src, a.src_bytes);

    // Per-lane A byte offsets; rows past M read zero (and are not stored).
    // Registers (m-major): row m of the packed filter, reduction rows 4 kr ..;
    // the reduction rows of a filter are zero-padded to a multiple of 16
    // (a.a_ld), so a slice never reads another filter's rows.  LDS (k-major):
    // row m within a packed reduction row of M floats.
    constexpr int NAO = ASH ? HA : FM;
    uint32_t a_off[NAO], a_msk[NAO];
#pragma unroll
    for (int i = 0; i < NAO; i++) {
        if constexpr (ASH) {
            const int m = m0 + 64 * i + lane;
            a_off[i] = (uint32_t)(m * 4);
            a_msk[i] = oob_mask(m < a.M);
        } else {
            const int m = m0 + wm * TM + i * 16 + lc;
            a_off[i] = ((uint32_t)(g * a.M + (m < a.M ? m : 0)) * (uint32_t)a.a_ld + 4u * kr) * 4u;
            a_msk[i] = oob_mask(m < a.M);
        }
    }
    const uint32_t a_gbase = (uint32_t)g * (uint32_t)a.a_ld * (uint32_t)a.M * 4u;

    // ONE: lane l stages row l / 16 of a 4-row group at columns
    // n0 + 4 (l % 16) .. + 3; byte offset of that source row segment for
    // channel 0 of the group (or out of range past the last column).
    uint32_t b4_base = 0;
    if constexpr (ONE) {
        const int n = n0 + 4 * (lane & 15);
        const uint32_t c = n < a.Ncol ? (uint32_t)n : 0u;
        const uint32_t img = fast_div(c, a.col_hw);
        const uint32_t pix = c - img * a.col_hw.d;
        b4_base = ((img * a.src_img_words + ((uint32_t)g * a.cin + (uint32_t)(lane >> 4)) *
                                                (uint32_t)a.src_hw + pix) * 4u) |
                  oob_mask(n < a.Ncol);
    }

    // Per-lane B column data: image base offset, base coordinates, validity.
    uint32_t b_base[HB];
    int b_hb[HB], b_wb[HB];
    bool b_ok[HB];
#pragma unroll
    for (int h = 0; h < HB; h++) {
        int n = n0 + 64 * h + lane;
        b_ok[h] = n < a.Ncol;
        uint32_t c = b_ok[h] ? (uint32_t)n : 0u;
        uint32_t img = fast_div(c, a.col_hw);
        uint32_t rem = c - img * a.col_hw.d;
        uint32_t ci = fast_div(rem, a.col_w);
        uint32_t cj = rem - ci * a.col_w.d;
        b_hb[h] = (int)ci * a.cstep + a.coff_h;
        b_wb[h] = (int)cj * a.cstep + a.coff_w;
        b_base[h] = (img * a.src_img_words + (uint32_t)g * a.cin * a.src_hw) * 4u;
    }

    // Loads of the slice starting at reduction row k0: A into registers ar
    // or into the LDS buffer Ad, B into the LDS buffer Bd (wave-load j fills
    // LDS row kk = wave + NW * (j / H), 64-wide segment h = j % H).
    auto issue = [&](int k0, float (*Ad)[LDA], float (*Bd)[LDB], f32x4 (&ar)[FM]) {
        if constexpr (ASH) {
#pragma unroll
            for (int j = 0; j < LA; j++) {
                const int kk = wave + NW * (j / HA), h = j % HA;
                const uint32_t row = a_gbase + (uint32_t)(k0 + kk) * (uint32_t)a.M * 4u;
                lds_load(rA, &Ad[kk][64 * h], (row + a_off[h]) | a_msk[h]);
            }
        } else {
#pragma unroll
            for (int i = 0; i < FM; i++)
                ar[i] = load4_untracked(rAw, (a_off[i] + (uint32_t)k0 * 4u) | a_msk[i]);
        }
        if constexpr (ONE) {
            // Slice k0 covers channels k0 .. k0 + 15 (one tap); group j its
            // rows 4 j .. 4 j + 3.
#pragma unroll
            for (int j = 0; j < LB; j++) {
                const int grp = wave + NW * j;
                const bool live = grp < NG;
                const uint32_t off =
                    (b4_base + (uint32_t)(k0 + 4 * grp) * (uint32_t)a.src_hw * 4u) | oob_mask(live);
                __builtin_amdgcn_raw_ptr_buffer_load_lds(rB, (LDS_AS void *)&Bd[live ? grp : NG][0],
                                                         16, off, 0, 0, 0);
            }
        } else if constexpr (FAST) {
            // Slice k0 / 16 = cb * taps + tap covers channels 16 cb .. 16 cb + 15.
            const uint32_t sl = (uint32_t)k0 / 16u;
            const uint32_t cb = fast_div(sl, a.k_taps);
            const uint32_t tap = sl - cb * a.k_taps.d;
            const int ch0 = (int)cb * 16;
            const uint32_t tr = fast_div(tap, a.k_tw);
            const int ts = (int)(tap - tr * a.k_tw.d);
            uint32_t sp[HB], msk[HB];
#pragma unroll
            for (int h = 0; h < HB; h++) {
                int hy = b_hb[h] + a.tsign * (int)tr, wx = b_wb[h] + a.tsign * ts;
                bool ok = b_ok[h] && (unsigned)hy < (unsigned)a.src_h &&
                          (unsigned)wx < (unsigned)a.src_w;
                sp[h] = b_base[h] + ((uint32_t)ch0 * (uint32_t)a.src_hw +
                                     (uint32_t)(hy * a.src_w + wx)) * 4u;
                msk[h] = oob_mask(ok);
            }
#pragma unroll
            for (int j = 0; j < LB; j++) {
                const int kk = wave + NW * (j / HB), h = j % HB;
                const bool live = kk < BK;
                lds_load(rB, &Bd[live ? kk : BK][64 * h],
                         (sp[h] + (uint32_t)kk * (uint32_t)a.src_hw * 4u) | msk[h] |
                             oob_mask(live));
            }
        } else {
#pragma unroll
            for (int j = 0; j < LB; j++) {
                const int kk = wave + NW * (j / HB), h = j % HB;
                const bool live = kk < BK;
                const int k = k0 + kk;
                const bool kok = live && k < kend;
                const uint32_t kc = kok ? (uint32_t)k : 0u;
                const uint32_t tap = fast_div(kc, a.k_cin);
                const int ch = (int)(kc - tap * a.k_cin.d);
                const uint32_t tr = fast_div(tap, a.k_tw);
                const int ts = (int)(tap - tr * a.k_tw.d);
                int hy = b_hb[h] + a.tsign * (int)tr, wx = b_wb[h] + a.tsign * ts;
                bool ok = kok && b_ok[h] && (unsigned)hy < (unsigned)a.src_h &&
                          (unsigned)wx < (unsigned)a.src_w;
                uint32_t off = b_base[h] + ((uint32_t)ch * (uint32_t)a.src_hw +
                                            (uint32_t)(hy * a.src_w + wx)) * 4u;
                lds_load(rB, &Bd[live ? kk : BK][64 * h], off | oob_mask(ok));
            }
        }
    };

    f32x4 acc[FM][FN];
#pragma unroll
    for (int i = 0; i < FM; i++)
#pragma unroll
        for (int j = 0; j < FN; j++)
#pragma unroll
            for (int v = 0; v < 4; v++)
                acc[i][j][v] = 0.f;

    const int nslices = kend > kbeg ? (kend - kbeg + BK - 1) / BK : 0;

    // Operands of one slice -> registers, then MFMAs.
    auto compute = [&](float (*Ac)[LDA], float (*Bc)[LDB], const f32x4 (&ar)[FM],
                       auto &&between) {
        float bf[4][FN];
#pragma unroll
        for (int s = 0; s < 4; s++)
#pragma unroll
            for (int j = 0; j < FN; j++) {
                if constexpr (ONE)
                    bf[s][j] = Bc[kr][s * 64 + wn * TN + j * 16 + lc];
                else
                    bf[s][j] = Bc[4 * kr + s][wn * TN + j * 16 + lc];
            }
        f32x4 af[FM];
#pragma unroll
        for (int i = 0; i < FM; i++) {
            if constexpr (ASH) {
#pragma unroll
                for (int s = 0; s < 4; s++)
                    af[i][s] = Ac[4 * kr + s][i * 16 + lc];
            } else {
                // The untracked load's value is only valid after the stage's
                // wait (s_waitcnt before the barrier).  Nothing here orders
                // this copy after that wait: the build-time check in
                // isa_check.py verifies on the generated code that the
                // registers are read by MFMAs only, after the second barrier.
                af[i] = ar[i];
            }
        }
        between();  // issue later slices' loads once this slice's reads are out
#pragma unroll
        for (int s = 0; s < 4; s++)
#pragma unroll
            for (int i = 0; i < FM; i++)
#pragma unroll
                for (int j = 0; j < FN; j++)
                    acc[i][j] = mfma16(af[i][s], bf[s][j], acc[i][j]);
    };

    // Before the barrier of slice t a wave waits only until its own loads of
    // slice t are done (vmcnt counts down in issue order, and the FM + LB
    // loads of slice t + 1 may stay outstanding).  This wait is also the one
    // that makes the A registers of slice t valid: their loads are untracked
    // by the compiler.  A raw s_barrier (no fence, which would wait for every
    // load) then publishes the B slice, and the compiler barriers keep LDS
    // accesses on their side.
    constexpr int LPS = LA + LB;
    constexpr int WAIT_NEXT = (LPS & 15) | (((LPS >> 4) & 3) << 14) | (7 << 4) | (15 << 8);
    static_assert(LPS < 64, "vmcnt range");
    f32x4 ar0[FM], ar1[FM], ar2[FM];
    auto stage = [&](int t, float (*Ac)[LDA], float (*Bc)[LDB], const f32x4 (&ac)[FM],
                     float (*An)[LDA], float (*Bn)[LDB], f32x4 (&an)[FM]) {
        if (t + 1 < nslices)
            __builtin_amdgcn_s_waitcnt(WAIT_NEXT);
        else
            __builtin_amdgcn_s_waitcnt(0);
        __asm__ volatile("" ::: "memory");
        __builtin_amdgcn_s_barrier();
        __asm__ volatile("" ::: "memory");
        compute(Ac, Bc, ac, [&] {
            if (t + 2 < nslices)
                issue(kbeg + (t + 2) * BK, An, Bn, an);
        });
    };
    if (nslices > 0)
        issue(kbeg, As0, Bs0, ar0);
    if (nslices > 1)
        issue(kbeg + BK, As1, Bs1, ar1);
    for (int t = 0; t < nslices; t += 3) {
        stage(t, As0, Bs0, ar0, As2, Bs2, ar2);
        if (t + 1 < nslices)
            stage(t + 1, As1, Bs1, ar1, As0, Bs0, ar0);
        if (t + 2 < nslices)
            stage(t + 2, As2, Bs2, ar2, As1, Bs1, ar1);
    }

    // Epilogue: + bias, scatter columns back to image coordinates (a split
    // writes its partial sums, without bias, to its own output-shaped slab).
    float *const out = a.nsplit > 1 ? a.out + (long long)split * a.split_stride : a.out;
    if (a.mblock > 1) {
        // Blocked backward-data: row m is channel c, block offset (ph, pw).
        const int b = a.mblock, bb = b * b, cg = a.M / bb;
        int oh[FN], ow[FN];
        long long cbase[FN];
#pragma unroll
        for (int j = 0; j < FN; j++) {
            int n = n0 + wn * TN + j * MF + lc;
            bool ok = n < a.Ncol;
            uint32_t c = ok ? (uint32_t)n : 0u;
            uint32_t img = fast_div(c, a.col_hw);
            uint32_t rem = c - img * a.col_hw.d;
            uint32_t ci = fast_div(rem, a.col_w);
            uint32_t cj = rem - ci * a.col_w.d;
            oh[j] = ok ? (int)ci * a.ostep + a.ooff_h : -b;  // -b: no row is inside
            ow[j] = (int)cj * a.ostep + a.ooff_w;
            cbase[j] = (long long)img * a.out_img_stride + (long long)oh[j] * a.out_w + ow[j];
        }
#pragma unroll
        for (int i = 0; i < FM; i++)
#pragma unroll
            for (int v = 0; v < 4; v++) {
                int m = m0 + wm * TM + i * MF + acc_row(v, lane);
                if (m >= a.M)
                    continue;
                const int c = m / bb, rem = m - c * bb, ph = rem / b, pw = rem - ph * b;
                const long long roff = (long long)(g * cg + c) * a.out_hw + ph * a.out_w + pw;
#pragma unroll
                for (int j = 0; j < FN; j++)
                    if ((unsigned)(oh[j] + ph) < (unsigned)a.out_h &&
                        (unsigned)(ow[j] + pw) < (unsigned)a.out_w)
                        out[cbase[j] + roff] = acc[i][j][v];
            }
        return;
    }
    const float *const bias = a.nsplit > 1 ? nullptr : a.bias;
    long long obase[FN];
    bool nok[FN];
#pragma unroll
    for (int j = 0; j < FN; j++) {
        int n = n0 + wn * TN + j * MF + lc;
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
        for (int v = 0; v < 4; v++) {
            int m = m0 + wm * TM + i * MF + acc_row(v, lane);
            if (m >= a.M)
                continue;
            int oc = g * a.M + m;
            float bv = bias ? bias[oc] : 0.f;
            long long choff = (long long)oc * a.out_hw;
#pragma unroll
            for (int j = 0; j < FN; j++)
                if (nok[j])
                    out[obase[j] + choff] = acc[i][j][v] + bv;
        }
}

// ---------------------------------------------------------------------------
// Halo-staged implicit GEMM for stride-1 R x R layers, R = 3 or 5 (see
// HaloGemmArgs).
//
// A tile is BM filter rows x 112 columns, the columns being a TR x TW block of
// output pixels of one image.  The gathered operand of a 16-channel block is
// the same image region for all R R taps, shifted: it is staged once per
// block (the halo, V words per lane and load, direct to LDS) and the R R
// slices of the block read their B operands from it at per-tap offsets.  For
// 3 x 3 that divides the staging-load lanes per MFMA by 5 to 6 (by 20 with
// 16-byte loads) against the per-slice gather of img_gemm_kernel, whose
// load-issue rate (one dword per lane) is what bounds it; for 5 x 5 by 15 or
// more, even with one-word loads.
//
// The pixel block is fixed per instantiation (HaloCfg): TW = 112, 56, 28 or 14
// columns (the map widths of the 3 x 3 layers at 224 ... 14 pixels; 28 or 14
// for 5 x 5, whose maps of 27 or 28 and 14 pixels fit them) by TR = 112 / TW
// rows, so every LDS offset of a tap is a compile-time constant and the B
// reads need no address arithmetic.  LDS layout of a block: halo[c][i][j] at
// c CS + i HWW + j, either dense (the wave-loads fill consecutive words,
// CS = HR HWW) or LPC whole wave-loads per channel in a padded slot of CS
// words; CS is chosen so that the four MFMA lane groups, which read channels 4
// apart, fall on different LDS banks.  5 x 5 blocks use one-word loads, so any
// map width can be staged (AlexNet's 27-wide maps included).
//
// Four waves split the rows (BM / 4 each, FM = BM / 64 accumulator blocks
// high) and each covers all 112 columns (7 blocks of 16; 11 for a whole
// 13 x 13 map); in 5 x 5 tiles a
// wave whose rows all lie past M (M = 48 on the 64-row tile) stages its share
// of the halo and skips the MFMAs.  The filter
// operand of a slice is one 16-byte load per lane and row block, straight
// into registers, issued two slices ahead into a ring of NR register sets
// (NR = 3, or 5 for 5 x 5: NR divides R R, so slice t always sits in set
// t mod NR).  The halo has two LDS stages: the next block's loads are issued
// at the start of a block and complete under its R R slices; one barrier per
// block.
// ---------------------------------------------------------------------------
template <int TW, int TR, int R>
struct HaloCfg;
template <>
struct HaloCfg<112, 1, 3> {
    static constexpr int V = 4, HWW = 124, LPC = 0, CS = 3 * 124;
};
template <>
struct HaloCfg<56, 2, 3> {
    static constexpr int V = 4, HWW = 64, LPC = 1, CS = 260;
};
template <>
struct HaloCfg<28, 4, 3> {
    static constexpr int V = 4, HWW = 36, LPC = 1, CS = 260;
};
template <>
struct HaloCfg<14, 8, 3> {
    static constexpr int V = 1, HWW = 18, LPC = 0, CS = 10 * 18;
};
template <>
struct HaloCfg<28, 4, 5> {  // 8 x 32 words a channel: four wave-loads
    static constexpr int V = 1, HWW = 32, LPC = 4, CS = 260;
};
template <>
struct HaloCfg<14, 8, 5> {  // 12 x 18 words a channel in four wave-loads
    static constexpr int V = 1, HWW = 18, LPC = 4, CS = 260;
};
// Whole-image blocks of 13 x 13 maps (3 x 3): 176 columns, 169 used, against
// 169 of 224 for two 14 x 8 blocks; 15 halo rows of 16 words, four
// wave-loads a channel.  (A 14 x 14 map as one 208-column block measured
// slower than two 14 x 8 blocks, which already use 7/8 of their columns.)
template <>
struct HaloCfg<13, 13, 3> {
    static constexpr int V = 1, HWW = 16, LPC = 4, CS = 260;
};

constexpr int kHaloStageWords = 6400;  // largest stage (25 KiB, 112-wide blocks): three workgroups a CU

// Waves per SIMD the register allocation must allow: four for 64-row tiles
// (four workgroups a CU) whose LDS stages allow it (all but 112-wide 3 x 3
// blocks), three for the rest of 3 x 3 (whole 13 x 13 maps, 176 columns of
// accumulators, included); 128-row 5 x 5 tiles fit three
// without the bound.  The waves are latency-bound (each issues an MFMA only
// every few slots), so a SIMD's throughput grows with its waves: four
// workgroups instead of three measured 1-3 % faster on VGG-16's 224- to
// 28-pixel layers.
//
// KS = 2 (small grids): eight waves, two groups of four over the two halves of
// the channel blocks, each group with its own two halo stages; the second
// group's partial sums are added to the first's through LDS before the
// epilogue.  This doubles the waves a SIMD holds where the tiles are too few to
// fill the CU slots, without the partial-sum round trip through memory of a
// split plan.
template <int BM, int TW, int TR, int R, int KS = 1>
constexpr int halo_min_waves()
{
    return KS == 2 ? (BM == 64 ? 4 : 2)
           : TR * TW != kHaloCols ? 3 : BM == 64 && (TW != 112 || R != 3) ? 4 : R == 3 ? 3 : 1;
}

template <int BM, int TW, int TR, int R, bool FLIP, int KS = 1>
__global__ __launch_bounds__(256 * KS) __attribute__((amdgpu_waves_per_eu(halo_min_waves<BM, TW, TR, R, KS>())))
void halo_gemm_kernel(const HaloGemmArgs a)
{
    typedef HaloCfg<TW, TR, R> C;
    constexpr int S = R, RS = R * S, NR = RS % 3 == 0 ? 3 : 5, DIST = 2;
    constexpr int PIX = TR * TW;  // pixels of a block; columns past it are padding
    constexpr int NW = 4, BN = (PIX + 15) / 16 * 16, TM = BM / NW, FM = TM / 16, FN = BN / 16;
    constexpr int V = C::V, HWW = C::HWW, CS = C::CS, LPC = C::LPC;
    constexpr int HR = TR + R - 1;
    constexpr int GPR = HWW / V;                  // load groups per halo row
    constexpr int EPC = HR * GPR;                 // load groups per channel
    // Dense: wave-loads over 16 EPC groups; per channel: LPC each.
    constexpr int NWL = LPC ? 16 * LPC : (16 * EPC + 63) / 64;
    constexpr int LPW = (NWL + NW - 1) / NW;      // wave-loads per wave and block
    constexpr int SPARE = LPC ? 16 * CS : NWL * 64 * V;  // slot of padding loads
    // Words per LDS stage: what the block uses (25 KiB for 112-wide blocks,
    // 17 KiB for 56- and 28-wide ones and 5 x 5, 11.5 KiB for 14-wide 3 x 3),
    // so that four 64-row workgroups fit a CU where the registers allow.
    constexpr int STG = SPARE + 64 * V;
    static_assert(RS % NR == 0, "filter ring");
    static_assert(BM == 64 || BM == 128, "tile rows");
    static_assert(PIX == kHaloCols || (TR == TW && BN > kHaloCols), "pixel block: 112 pixels or a whole small map");
    static_assert(HWW % V == 0 && HWW >= TW + S - 1, "halo row");
    // A wave-load writes all 64 lanes (masked lanes write zeros), so a
    // channel's slot must hold LPC 64 V words.
    static_assert(LPC ? (EPC <= 64 * LPC && CS >= 64 * V * LPC && (CS * 4) % 16 == 0)
                      : CS == HR * HWW, "channel stride");
    static_assert(SPARE + 64 * V <= STG && STG <= kHaloStageWords && STG % 4 == 0, "halo stage");
    static_assert(KS == 1 || (KS == 2 && R == 3 && PIX == kHaloCols && TW != 112), "wave groups");

    // Stages of wave group kh: H0[kh], H1[kh].
    __shared__ __attribute__((aligned(16))) float H0[KS][STG], H1[KS][STG];
    static_assert(KS == 1 || NW * 4 * 64 * 4 <= KS * STG, "partial sums of four column blocks fit H0");

    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6) & (NW - 1);
    const int kh = KS == 2 ? __builtin_amdgcn_readfirstlane(threadIdx.x >> 8) : 0;
    const int mtiles = (a.M + BM - 1) / BM;
    const int per_img = a.row_blocks * a.col_segs;
    const int tiles = mtiles * a.nimg * per_img;
    const int lin = xcd_tile(blockIdx.x, tiles * a.groups * a.nsplit);
    const int split = lin / (tiles * a.groups);
    const int rest = lin - split * tiles * a.groups;
    const int g = rest / tiles, tile = rest - g * tiles;
    // Pixel blocks fastest: an XCD's range of tiles is then one or two
    // filter-row tiles over many pixel blocks, so the filter rows it re-reads
    // stay in its L2 (filter-row tiles fastest made every XCD stream the
    // whole bank, 9.4 MB for VGG-16's 512-channel layers, past its 4 MB L2:
    // 0.3-2.8 % slower).
    const int ptiles = a.nimg * per_img;
    const int pt = tile % ptiles, mt = tile / ptiles;
    const int img = pt / per_img;
    const int prem = pt - img * per_img;
    const int rb = prem / a.col_segs, csg = prem - rb * a.col_segs;
    const int p0 = rb * TR, q0 = csg * TW;
    const int m0 = mt * BM;
    const int ncb = a.Kred / (16 * RS);
    // The split's channel blocks; with KS = 2 the group's half of them (the
    // host makes their count even).
    const int cb_lo = split * a.cbchunk;
    const int cb_n = (min(ncb, cb_lo + a.cbchunk) - cb_lo) / KS;
    const int cb_beg = cb_lo + kh * cb_n;
    const int cb_end = cb_beg + cb_n;
    const int kr = lane >> 4, lc = lane & 15;
    // Wave-uniform: some row of this wave is real (checked for 5 x 5 only,
    // whose M = 48 backward-data phases leave a 64-row tile's last wave idle).
    const int wrow = wave;  // the wave's row block of the tile
    const bool live = R == 3 || m0 + wrow * TM < a.M;

    // Filter operand: row m = m0 + wrow * TM + 16 i + lc, reduction words
    // 16 t + 4 kr .. + 3 of slice t; rows past M read zero.
    const __amdgpu_buffer_rsrc_t rA = make_rsrc(a.A, a.a_bytes);
    uint32_t a_off[FM];
#pragma unroll
    for (int i = 0; i < FM; i++) {
        const int m = m0 + wrow * TM + i * 16 + lc;
        a_off[i] = (((uint32_t)(g * a.M + (m < a.M ? m : 0)) * (uint32_t)a.a_ld + 4u * kr) * 4u) |
                   oob_mask(m < a.M);
    }
    const int t_last = cb_end * RS - 1;  // last slice of this split
    auto loadA = [&](int t, f32x4 (&dst)[FM]) {
        const int tc = t < t_last ? t : t_last;  // past the end: a harmless repeat
#pragma unroll
        for (int i = 0; i < FM; i++)
            dst[i] = __builtin_bit_cast(
                f32x4, __builtin_amdgcn_raw_buffer_load_b128(
                           rA, (int)(a_off[i] + (uint32_t)tc * 64u), 0, 0));
    };

    // Halo staging.  Wave-load i = wave + 4 j carries, per lane, load group
    // e of channel c (dense: e + EPC c = 64 i + lane; per channel: c = i / LPC,
    // e = 64 (i mod LPC) + lane) into LDS word c CS + V e (dense: 64 V i +
    // V lane) of a stage.
    // Group e = row * GPR + grp is source pixel (p0 + row0 + row,
    // q0 + col0 + V grp) .. + V - 1 of channel 16 cb + c, zero outside the
    // source (with V = 4 the source width and col0, q0 are multiples of 4, so
    // a group lies inside or outside a row).  Loads past the last wave-load
    // go to a spare slot and read zero.
    // With as many wave-loads per channel as waves (LPC = NW), wave w loads
    // part w of every channel, wave-load j being channel j: one lane offset
    // then serves all of them, plus j channel strides.
    constexpr bool PARTS = LPC == NW;
    const __amdgpu_buffer_rsrc_t rB = make_rsrc(a.src, a.src_bytes);
    uint32_t h_off[PARTS ? 1 : LPW];
#pragma unroll
    for (int j = 0; j < (PARTS ? 1 : LPW); j++) {
        const int i = wave + NW * j;
        int c, e;
        if constexpr (LPC) {
            c = i / LPC;
            e = (i % LPC) * 64 + lane;
        } else {
            const int ge = i * 64 + lane;
            c = ge / EPC;
            e = ge - c * EPC;
        }
        const int row = e / GPR, grp = e - row * GPR;
        const int h = p0 + a.row0 + row, w = q0 + a.col0 + grp * V;
        const bool ok = i < NWL && c < 16 && e < EPC && (unsigned)h < (unsigned)a.src_h &&
                        w >= 0 && w + V <= a.src_w;
        h_off[j] = ok ? ((uint32_t)img * a.src_img_words +
                         (uint32_t)(g * a.cin + c) * (uint32_t)a.src_hw +
                         (uint32_t)(h * a.src_w + w)) * 4u
                      : kOob;
    }
    const uint32_t ch_bytes = (uint32_t)a.src_hw * 4u, cb_bytes = 16u * ch_bytes;
    auto issue_halo = [&](int cb, float *Hd) {
#pragma unroll
        for (int j = 0; j < LPW; j++) {
            const int i = wave + NW * j;
            float *dst = Hd + (i >= NWL ? SPARE
                               : LPC ? (i / LPC) * CS + (i % LPC) * 64 * V
                                     : i * 64 * V);
            const uint32_t h = h_off[PARTS ? 0 : j];
            const uint32_t off =
                h == kOob ? kOob : h + (uint32_t)cb * cb_bytes + (PARTS ? (uint32_t)j * ch_bytes : 0u);
            if constexpr (V == 4)
                __builtin_amdgcn_raw_ptr_buffer_load_lds(rB, (LDS_AS void *)dst, 16, off, 0, 0, 0);
            else
                __builtin_amdgcn_raw_ptr_buffer_load_lds(rB, (LDS_AS void *)dst, 4, off, 0, 0, 0);
        }
    };

    // B operand: column n = 16 j + lc is pixel (dr, dq) = (n / TW, n % TW) of
    // the block; for channel 4 kr + s4 and tap (rr, ss) its halo word is
    // bofs[j] + s4 CS + rr HWW + ss, with bofs[j] = 4 kr CS + dr HWW + dq + slack
    // (a compile-time offset from a per-lane base).  Columns outside the
    // output read word 0 and are not stored (reading their own halo words
    // instead measured 8 % slower on AlexNet conv2's backward-data phase).
    int bofs[FN];
    bool nok[FN];
#pragma unroll
    for (int j = 0; j < FN; j++) {
        const int n = j * 16 + lc;
        const int dr = n / TW, dq = n - (n / TW) * TW;
        nok[j] = n < PIX && p0 + dr < a.P && q0 + dq < a.Q;
        bofs[j] = nok[j] ? kr * 4 * CS + dr * HWW + dq + a.slack : 0;
    }

    f32x4 acc[FM][FN];
#pragma unroll
    for (int i = 0; i < FM; i++)
#pragma unroll
        for (int j = 0; j < FN; j++)
            acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

    f32x4 ring[NR][FM];
    auto block = [&](int cb, const float *Hc, float *Hn, bool stage_next) __attribute__((always_inline)) {
        // The other stage is free (every wave passed the barrier after
        // reading it): stage the next block into it.
        if (stage_next)
            issue_halo(cb + 1, Hn);
        __asm__ volatile("" ::: "memory");
        if (!live) {
            // Only this wave's halo loads are outstanding.
            __builtin_amdgcn_s_waitcnt(0);
            __asm__ volatile("" ::: "memory");
            __builtin_amdgcn_s_barrier();
            __asm__ volatile("" ::: "memory");
            return;
        }
        // MFMA step u = 4 tap + s4 takes channels 4 kr + s4 of the tap.  Its
        // FN B values are read one step ahead, into bq[u & 1] while the MFMAs
        // of step u - 1 run, so a step's MFMAs wait only for reads issued a
        // whole step earlier (at most 2 FN reads in flight); the scheduling
        // barriers keep the compiler from sinking each read onto its MFMA.
        constexpr int NSTEP = 4 * RS;
        float bq[2][FN];
        auto readB = [&](int u, float (&dst)[FN]) __attribute__((always_inline)) {
            const int tap = u >> 2, s4 = u & 3;
            const int r = tap / S, sx = tap % S;
            const int toff = (FLIP ? R - 1 - r : r) * HWW + (FLIP ? S - 1 - sx : sx) + s4 * CS;
#pragma unroll
            for (int j = 0; j < FN; j++)
                dst[j] = Hc[bofs[j] + toff];
        };
        readB(0, bq[0]);
#pragma unroll
        for (int u = 0; u < NSTEP; u++) {
            const int tap = u >> 2, s4 = u & 3;
            if (s4 == 0)
                loadA(cb * RS + tap + DIST, ring[(tap + DIST) % NR]);
            if (u + 1 < NSTEP)
                readB(u + 1, bq[(u + 1) & 1]);
            __builtin_amdgcn_sched_barrier(0);
#pragma unroll
            for (int i = 0; i < FM; i++)
#pragma unroll
                for (int j = 0; j < FN; j++)
                    acc[i][j] = mfma16(ring[tap % NR][i][s4], bq[u & 1][j], acc[i][j]);
            __builtin_amdgcn_sched_barrier(0);
        }
        // The next block's halo has landed once at most the DIST filter loads
        // issued last (the next block's first DIST slices) are outstanding.
        __asm__ volatile("" ::: "memory");
        __builtin_amdgcn_s_waitcnt((DIST * FM & 15) | (((DIST * FM) >> 4) << 14) | (7 << 4) |
                                   (15 << 8));
        __asm__ volatile("" ::: "memory");
        __builtin_amdgcn_s_barrier();
        __asm__ volatile("" ::: "memory");
    };

    float *const G0 = H0[kh], *const G1 = H1[kh];
    if (cb_beg < cb_end) {
        issue_halo(cb_beg, G0);
#pragma unroll
        for (int d = 0; d < DIST; d++)
            loadA(cb_beg * RS + d, ring[d]);
        __builtin_amdgcn_s_waitcnt(0);
        __asm__ volatile("" ::: "memory");
        __builtin_amdgcn_s_barrier();
        __asm__ volatile("" ::: "memory");
    }
    int cb = cb_beg;
    for (; cb + 1 < cb_end; cb += 2) {
        block(cb, G0, G1, true);
        block(cb + 1, G1, G0, cb + 2 < cb_end);
    }
    if (cb < cb_end)
        block(cb, G0, G1, false);

    if constexpr (KS == 2) {
        // Group 1's sums into group 0's, four column blocks of one row block
        // at a time through H0 (free: the last block ended with a barrier and
        // staged nothing), in a fixed order (each group summed its own half
        // of the channel blocks first).
        f32x4 *const red = reinterpret_cast<f32x4 *>(&H0[0][0]);
#pragma unroll
        for (int i = 0; i < FM; i++)
#pragma unroll
            for (int j0 = 0; j0 < FN; j0 += 4) {
                if (kh == 1) {
#pragma unroll
                    for (int j = j0; j < min(FN, j0 + 4); j++)
                        red[(wrow * 4 + j - j0) * 64 + lane] = acc[i][j];
                }
                __asm__ volatile("" ::: "memory");
                __builtin_amdgcn_s_barrier();
                __asm__ volatile("" ::: "memory");
                if (kh == 0) {
#pragma unroll
                    for (int j = j0; j < min(FN, j0 + 4); j++) {
                        const f32x4 o = red[(wrow * 4 + j - j0) * 64 + lane];
                        acc[i][j] = f32x4{acc[i][j][0] + o[0], acc[i][j][1] + o[1],
                                          acc[i][j][2] + o[2], acc[i][j][3] + o[3]};
                    }
                }
                __asm__ volatile("" ::: "memory");
                __builtin_amdgcn_s_barrier();
                __asm__ volatile("" ::: "memory");
            }
        if (kh == 1)
            return;
    }

    // Epilogue: + bias (unsplit), pixel (p0 + dr, q0 + dq) of the tile's image.
    float *const out = a.nsplit > 1 ? a.out + (long long)split * a.split_stride : a.out;
    const float *const bias = a.nsplit > 1 ? nullptr : a.bias;
#pragma unroll
    for (int i = 0; i < FM; i++)
#pragma unroll
        for (int v = 0; v < 4; v++) {
            const int m = m0 + wrow * TM + i * 16 + acc_row(v, lane);
            if (m >= a.M)
                continue;
            const int oc = g * a.M + m;
            const float bv = bias ? bias[oc] : 0.f;
            const long long base = (long long)img * a.out_img_stride + (long long)oc * a.out_hw;
#pragma unroll
            for (int j = 0; j < FN; j++) {
                const int n = j * 16 + lc;
                const int dr = n / TW, dq = n - (n / TW) * TW;
                if (nok[j])
                    out[base + (long long)(p0 + dr) * a.out_w + (q0 + dq)] = acc[i][j][v] + bv;
            }
        }
}

// ---------------------------------------------------------------------------
// Backward-weight GEMM with one pixel per lane (same WgradArgs).
//
// Tap-uniform tiles (PACKED = false) take dw columns in (tap, channel) order:
// a workgroup tile owns one tap
// t = r S + s and BN consecutive channels, so its B operand is x shifted by
// (r, s) — for a given pixel, the BN rows of B are BN channels at one
// spatial position.  A slice of the reduction is 64 consecutive pixels; lane
// l owns pixel k0 + l of the slice and computes, once per slice, the byte
// offset of its dy element (row m0) and of its x element (channel c0, shifted
// by the tap), or an out-of-range offset when the pixel is outside the split
// or the image.  Every row of the A (dy) and B (x) tiles is then one
// direct-to-LDS wave-load whose offset is that base plus a row stride: one
// VALU add.  Rows past K/G or C/G read neighbouring data (or zeros) and are
// simply not stored.
//
// Packed tiles (PACKED = true, for few channels per group, e.g. the 3 colour
// channels of a first layer) own BN consecutive columns n = (c R + r) S + s
// of dw instead.  The byte offset of x for (pixel, column) splits into a
// per-lane part, (h0 W + w0) with h0 = p stride - pad and w0 = q stride - pad,
// and a per-column part, c H W + r W + s, which is wave-uniform (scalar
// registers); a row-load adds the two and checks h0 + r and w0 + s against
// the image (skipped when pad = 0, where every tap of a valid output pixel
// lies inside the image).
//
// LDS holds each row pixel-contiguous (64 words + 4 of padding, so the
// ds_read_b128 of 16 consecutive rows hit distinct banks).  The four 16-lane
// groups of the 16x16x4 MFMA take the four quarters of the slice, 16
// contiguous operands each: 4 ds_read_b128.  The tile is single-buffered: after a barrier
// every wave copies its operands of the slice into registers, a second
// barrier frees the LDS, the next slice's loads are issued, and the slice's
// MFMAs run while they land.
// ---------------------------------------------------------------------------
template <int BM, int BN, int WM, int WN, bool PACKED>
__global__ __launch_bounds__(64 * WM * WN) void wgrad_kernel(const WgradArgs a)
{
    constexpr int BK = 64, LDR = BK + 4;
    constexpr int NW = WM * WN, TM = BM / WM, TN = BN / WN, FM = TM / MF, FN = TN / MF;
    constexpr int PB = BK * MF / 64;  // pixels of the slice per lane group
    static_assert(BM % NW == 0 && BN % NW == 0, "rows per wave");
    static_assert(TM % MF == 0 && TN % MF == 0, "tile");

    __shared__ __attribute__((aligned(16))) float L[(BM + BN) * LDR];

    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int wm = wave % WM, wn = wave / WM;
    const int RS = (int)a.n_rs.d;
    const int cblocks = (a.Cg + BN - 1) / BN;
    const int mtiles = (a.M + BM - 1) / BM;
    const int ntiles = PACKED ? (a.Ncol + BN - 1) / BN : RS * cblocks;
    const int tiles = mtiles * ntiles;
    const int lin = xcd_tile(blockIdx.x, tiles * a.groups * a.nsplit);
    const int split = lin / (tiles * a.groups);
    const int rest = lin - split * tiles * a.groups;
    const int g = rest / tiles, tile = rest - g * tiles;
    const int mt = tile % mtiles, nt = tile / mtiles;
    // Tap-uniform: tap and first channel of the tile.  Packed: first column.
    const int tap = PACKED ? 0 : nt / cblocks;
    const int c0 = PACKED ? 0 : (nt - tap * cblocks) * BN;
    const int n0 = PACKED ? nt * BN : 0;
    const int r = (int)fast_div((uint32_t)tap, a.n_s), s_ = tap - r * (int)a.n_s.d;
    const int m0 = mt * BM;
    const int kbeg = split * a.chunk;
    const int kend = min(a.Kred, kbeg + a.chunk);

    const __amdgpu_buffer_rsrc_t rdy = make_rsrc(a.dy, a.dy_bytes);
    const __amdgpu_buffer_rsrc_t rx = make_rsrc(a.x, a.x_bytes);
    const uint32_t a_rowstep = (uint32_t)a.PQ * 4u, b_rowstep = (uint32_t)a.HW * 4u;
    const uint32_t a_row0 = (uint32_t)(g * a.M + m0) * a_rowstep;
    const uint32_t b_row0 = (uint32_t)(g * a.Cg + c0) * b_rowstep;

    auto issue = [&](int k0) {
        const int pix = k0 + lane;
        const bool pok = pix < kend;
        const uint32_t pc = pok ? (uint32_t)pix : 0u;
        const uint32_t img = fast_div(pc, a.pix_pq);
        const uint32_t pq = pc - img * a.pix_pq.d;
        const uint32_t p = fast_div(pq, a.pix_q);
        const int q = (int)(pq - p * a.pix_q.d);
        const uint32_t abase = pok ? (img * a.dy_img_words + pq) * 4u + a_row0 : kOob;
#pragma unroll
        for (int i = 0; i < BM / NW; i++) {
            const int j = wave + NW * i;
            lds_load(rdy, &L[j * LDR], abase + (uint32_t)j * a_rowstep);
        }
        if constexpr (PACKED) {
            const int h0 = (int)p * a.stride - a.pad, w0 = q * a.stride - a.pad;
            const uint32_t pbase = (img * a.x_img_words + (uint32_t)(h0 * a.W + w0)) * 4u + b_row0;
#pragma unroll
            for (int i = 0; i < BN / NW; i++) {
                const int n = n0 + wave + NW * i;  // wave-uniform column
                const uint32_t c = fast_div((uint32_t)n, a.n_rs);
                const uint32_t rs = (uint32_t)n - c * a.n_rs.d;
                const uint32_t rr = fast_div(rs, a.n_s);
                const int ss = (int)(rs - rr * a.n_s.d);
                bool ok = pok && n < a.Ncol;
                if (a.pad != 0)
                    ok = ok && (unsigned)(h0 + (int)rr) < (unsigned)a.H &&
                         (unsigned)(w0 + ss) < (unsigned)a.W;
                const uint32_t cofs = (c * (uint32_t)a.HW + rr * (uint32_t)a.W + (uint32_t)ss) * 4u;
                lds_load(rx, &L[(BM + wave + NW * i) * LDR], ok ? pbase + cofs : kOob);
            }
        } else {
            const int h = (int)p * a.stride - a.pad + r, w = q * a.stride - a.pad + s_;
            const bool xok = pok && (unsigned)h < (unsigned)a.H && (unsigned)w < (unsigned)a.W;
            const uint32_t bbase =
                xok ? (img * a.x_img_words + (uint32_t)(h * a.W + w)) * 4u + b_row0 : kOob;
#pragma unroll
            for (int i = 0; i < BN / NW; i++) {
                const int j = wave + NW * i;
                lds_load(rx, &L[(BM + j) * LDR], bbase + (uint32_t)j * b_rowstep);
            }
        }
    };

    f32x4 acc[FM][FN];
#pragma unroll
    for (int i = 0; i < FM; i++)
#pragma unroll
        for (int j = 0; j < FN; j++)
#pragma unroll
            for (int v = 0; v < 4; v++)
                acc[i][j][v] = 0.f;

    // Bias gradient: the workgroups of the first column tile also sum the dy
    // rows they stage (thread -> row tid / TPR, 64 / TPR pixels; TPR is the
    // largest power of two with BM * TPR threads at most).
    constexpr int TPR = 64 * NW / BM >= 8 ? 8 : 64 * NW / BM >= 4 ? 4 : 64 * NW / BM >= 2 ? 2 : 1;
    static_assert(BM <= 64 * NW, "one thread per bias row at least");
    const bool do_bias = a.db_part != nullptr && nt == 0;
    const int brow = threadIdx.x / TPR, bpart = threadIdx.x % TPR;
    float bsum = 0.f;

    const int kr = lane / MF, lc = lane % MF;
    const int nslices = kend > kbeg ? (kend - kbeg + BK - 1) / BK : 0;
    if (nslices > 0)
        issue(kbeg);
    for (int t = 0; t < nslices; t++) {
        __builtin_amdgcn_s_waitcnt(0);
        __syncthreads();  // slice t is in LDS
        if (do_bias && brow < BM) {
            const float *rowp = &L[brow * LDR + bpart * (BK / TPR)];
#pragma unroll
            for (int u = 0; u < BK / TPR; u += 4) {
                float4 v = *(const float4 *)&rowp[u];
                bsum += v.x;
                bsum += v.y;
                bsum += v.z;
                bsum += v.w;
            }
        }
        // MFMA step (u, e) of lane group kr takes pixel 8 u + 2 kr + e of the
        // slice: a lane's operands of steps (u, 0), (u, 1) are one aligned
        // ds_read_b64, and with 68-word rows the 32 lanes of a pass (16 rows
        // x lane groups 0, 1) hit all 64 banks.  (Sixteen consecutive pixels
        // a lane group read as ds_read_b128 cost bank conflicts.)
        static_assert(PB == 16 && LDR % 64 == 4, "pixel pairs over 68-word rows");
        f32x2 af[FM][PB / 2], bf[FN][PB / 2];
#pragma unroll
        for (int i = 0; i < FM; i++) {
            const float *rowp = &L[(wm * TM + i * MF + lc) * LDR + 2 * kr];
#pragma unroll
            for (int u = 0; u < PB / 2; u++)
                af[i][u] = lds_b64(rowp, 8 * u);
        }
#pragma unroll
        for (int j = 0; j < FN; j++) {
            const float *rowp = &L[(BM + wn * TN + j * MF + lc) * LDR + 2 * kr];
#pragma unroll
            for (int u = 0; u < PB / 2; u++)
                bf[j][u] = lds_b64(rowp, 8 * u);
        }
        __syncthreads();  // every wave holds its operands: the tile is free
        if (t + 1 < nslices)
            issue(kbeg + (t + 1) * BK);
#pragma unroll
        for (int u = 0; u < PB / 2; u++)
#pragma unroll
            for (int e = 0; e < 2; e++)
#pragma unroll
                for (int i = 0; i < FM; i++)
#pragma unroll
                    for (int j = 0; j < FN; j++)
                        acc[i][j] = mfma16(af[i][u][e], bf[j][u][e], acc[i][j]);
    }

    if (do_bias) {
        // Fixed butterfly over the TPR threads of a row.
#pragma unroll
        for (int off = 1; off < TPR; off <<= 1)
            bsum += __shfl_xor(bsum, off, 64);
        const int m = m0 + brow;
        if (bpart == 0 && brow < BM && m < a.M)
            a.db_part[(long long)split * a.K + g * a.M + m] = bsum;
    }

    // Tap-uniform: partial dw in tile order [split][g*Kg + m][tap][c]
    // (coalesced along c); the reduction kernel moves it to dw[k][c][r][s].
    // Packed: dw[k][n] itself, or its partial [split][k][n].
    float *outg = a.out + (long long)split * a.split_stride + (long long)g * a.M * a.Ncol +
                  (PACKED ? (long long)n0 : (long long)tap * a.Cg);
    const int ncols = PACKED ? a.Ncol - n0 : a.Cg - c0;
#pragma unroll
    for (int i = 0; i < FM; i++)
#pragma unroll
        for (int v = 0; v < 4; v++) {
            int m = m0 + wm * TM + i * MF + acc_row(v, lane);
            if (m >= a.M)
                continue;
#pragma unroll
            for (int j = 0; j < FN; j++) {
                int c = wn * TN + j * MF + lc;
                if (c < ncols)
                    outg[(long long)m * a.Ncol + (PACKED ? 0 : c0) + c] = acc[i][j][v];
            }
        }
}

// ---------------------------------------------------------------------------
// Halo backward-weight for stride-1 3 x 3 layers (see WgradHaloArgs).
//
// The one-pixel-per-lane kernel above stages, per 64-pixel slice and tap
// tile, one dword per lane and operand row: about one staging load per two
// MFMAs.  Here a workgroup owns all nine taps of a 64-filter x 16 CT-channel
// tile, so each 112-pixel block's dy rows and x halo are staged once and used
// by nine taps: about one load per twenty MFMAs.
//
// Pixel blocks (WgHaloCfg): TW = 112, 56, 28 or 14 columns by TR = 112 / TW
// rows.  dy rows are staged as 16-byte groups of 4 pixels (29 groups a row,
// the last padding); for TW = 14 a block is 8 whole rows of a 14-wide map,
// which lie contiguously in dy.  x halo of a channel: HR = TR + 2 rows of HWW
// columns from (p0 - pad, q0 + col0), 16-byte loads (V = 4; col0 rounded down
// to a multiple of 4, the tap columns then start slack words in) or one-word
// loads (V = 1; col0 = -pad, slack 0).  Layout: channel c at c CS, either
// dense (consecutive wave-loads, CS = the channel's words) or WPC wave-loads
// per channel with CS padded.  CS and HWW are chosen so that the operand
// reads below hit all 64 banks.
// ---------------------------------------------------------------------------
constexpr int kWhDyLd = 116;  // dy row: 112 pixels + one 4-word group of padding

template <int TW>
struct WgHaloCfg;
template <>
struct WgHaloCfg<112> {
    static constexpr int TR = 1, V = 4, HWW = 124, CS = 3 * 124, WPC = 0;
};
template <>
struct WgHaloCfg<56> {
    static constexpr int TR = 2, V = 4, HWW = 64, CS = 260, WPC = 1;
};
template <>
struct WgHaloCfg<28> {
    static constexpr int TR = 4, V = 4, HWW = 36, CS = 260, WPC = 1;
};
template <>
struct WgHaloCfg<14> {
    static constexpr int TR = 8, V = 1, HWW = 16, CS = 194, WPC = 3;
};

// Staging of one pixel block (dy rows of 64 filters, x halo of NCH channels)
// by NWV waves into LDS.  dy: wave-load i is issued by wave i % NWV.  x, WPC
// wave-loads per channel: wave w loads channels w, w + NWV, ..., so a lane's
// element of part p (p < WPC) of a channel is the same for every channel;
// dense layout: wave-load i by wave i % NWV.
template <int TW, int NCH, int NWV>
struct WgHaloStage {
    typedef WgHaloCfg<TW> C;
    static constexpr int TR = C::TR, V = C::V, HWW = C::HWW, CS = C::CS, WPC = C::WPC;
    static constexpr int HR = TR + 2, GPR = HWW / V, EPC = HR * GPR;  // elements of V words
    static constexpr int XNWL = WPC ? NCH * WPC : (NCH * EPC * V + 255) / 256;
    static constexpr int YNWL = 64 * (kWhDyLd / 4) / 64;  // 29
    static constexpr int XW = WPC ? NCH * CS : XNWL * 256;
    static constexpr int YW = 64 * kWhDyLd;
    static constexpr int YL = (YNWL + NWV - 1) / NWV;
    static constexpr int XL = WPC ? WPC : (XNWL + NWV - 1) / NWV;  // per-lane x slots
    static constexpr int NCC = (NCH + NWV - 1) / NWV;              // channels per wave (WPC > 0)
    static_assert(TR * TW == kHaloCols && HWW % V == 0, "112-pixel blocks");
    static_assert(WPC ? CS >= WPC * 64 * V && WPC * 64 >= EPC : CS == EPC * V,
                  "channel c's halo at c CS, regions disjoint");
    static_assert(V == 4 || V == 1, "16-byte or one-word halo loads");

    int y_row[YL], y_px[YL];
    int x_c[XL], x_row[XL], x_col[XL];  // x_c: dense layout's channel, or 0 / NCH (masked)

    __device__ void init(int wave, int lane)
    {
#pragma unroll
        for (int j = 0; j < YL; j++) {
            const int L = (wave + NWV * j) * 64 + lane;
            y_row[j] = L / (kWhDyLd / 4);
            y_px[j] = 4 * (L - y_row[j] * (kWhDyLd / 4));
        }
#pragma unroll
        for (int j = 0; j < XL; j++) {
            int c, e;
            if constexpr (WPC > 0) {
                c = 0;
                e = j * 64 + lane;
            } else {
                const int ge = (wave + NWV * j) * 64 + lane;
                c = ge / EPC;
                e = ge - c * EPC;
            }
            x_c[j] = (c < NCH && e < EPC) ? c : NCH;  // NCH: masked
            x_row[j] = e / GPR;
            x_col[j] = V * (e - x_row[j] * GPR);
        }
    }

    __device__ void load_x(__amdgpu_buffer_rsrc_t rx, uint32_t off, float *dst) const
    {
        if constexpr (V == 4)
            __builtin_amdgcn_raw_ptr_buffer_load_lds(rx, (LDS_AS void *)dst, 16, off, 0, 0, 0);
        else
            __builtin_amdgcn_raw_ptr_buffer_load_lds(rx, (LDS_AS void *)dst, 4, off, 0, 0, 0);
    }

    // DMA of pixel block b into Yd, Xd.
    __device__ void issue(const WgradHaloArgs &a, __amdgpu_buffer_rsrc_t rdy, __amdgpu_buffer_rsrc_t rx,
                          int wave, int b, int g, int m0, int c0, float *Yd, float *Xd) const
    {
        const int per_img = a.row_blocks * a.col_segs;
        const int img = b / per_img, prem = b - img * per_img;
        const int rb = prem / a.col_segs, csg = prem - rb * a.col_segs;
        const int p0 = rb * TR, q0 = csg * TW;
#pragma unroll
        for (int j = 0; j < YL; j++) {
            const int i = wave + NWV * j;
            if (i < YNWL) {
                const int px = y_px[j], dr = px / TW, dq = px - (px / TW) * TW;
                const int k = m0 + y_row[j];
                const bool ok = px < kHaloCols && k < a.Kg && p0 + dr < a.P && q0 + dq < a.Q;
                const uint32_t off =
                    ok ? ((uint32_t)img * a.dy_img_words + (uint32_t)(g * a.Kg + k) * (uint32_t)(a.P * a.Q) +
                          (uint32_t)((p0 + dr) * a.Q + q0 + dq)) * 4u
                       : kOob;
                __builtin_amdgcn_raw_ptr_buffer_load_lds(rdy, (LDS_AS void *)&Yd[i * 256], 16, off, 0, 0, 0);
            }
        }
        const uint32_t xim = (uint32_t)img * a.x_img_words, hw = (uint32_t)(a.H * a.W);
        if constexpr (WPC > 0) {
            // The lane's pixel offset and validity of each part, then one
            // wave-load per channel and part.
            uint32_t poff[WPC];
            bool pok[WPC];
#pragma unroll
            for (int j = 0; j < WPC; j++) {
                const int h = p0 + a.row0 + x_row[j], w = q0 + a.col0 + x_col[j];
                pok[j] = x_c[j] < NCH && (unsigned)h < (unsigned)a.H && w >= 0 && w + V <= a.W;
                poff[j] = (uint32_t)(h * a.W + w);
            }
#pragma unroll
            for (int cc = 0; cc < NCC; cc++) {
                const int c = wave + NWV * cc;
                if (c < NCH) {
                    const uint32_t cb = xim + (uint32_t)(g * a.Cg + c0 + c) * hw;
#pragma unroll
                    for (int j = 0; j < WPC; j++)
                        load_x(rx, pok[j] ? (cb + poff[j]) * 4u : kOob, &Xd[c * CS + j * 64 * V]);
                }
            }
        } else {
#pragma unroll
            for (int j = 0; j < XL; j++) {
                const int i = wave + NWV * j;
                if (i < XNWL) {
                    const int h = p0 + a.row0 + x_row[j], w = q0 + a.col0 + x_col[j];
                    const bool ok = x_c[j] < NCH && (unsigned)h < (unsigned)a.H && w >= 0 && w + V <= a.W;
                    const uint32_t off =
                        ok ? (xim + (uint32_t)(g * a.Cg + c0 + x_c[j]) * hw + (uint32_t)(h * a.W + w)) * 4u
                           : kOob;
                    load_x(rx, off, &Xd[i * 64 * V]);
                }
            }
        }
    }
};

// MFMA mapping (16x16x4, reduction over pixels): 28 steps s = 2 t + e (t <
// 14, e < 2) of 4 pixels, lane group kr taking one of them; pairs of steps
// cover 8 pixels, lane group kr an adjacent pair of columns, so that a lane's
// A operands of steps 2 t and 2 t + 1 (dy, filter lc of its wave's 16) are one
// aligned two-word LDS read, and its B operands (x of channel lc, shifted by
// the tap) for the three columns sx of filter row r are the four words
// x0 .. x0 + 3, x0 = lc CS + slack + (lane part) + (dr + r) HWW + (the pair's
// column), read as two aligned two-word reads when slack is even and three
// from x0 - 1 when it is odd (SODD).  Pixel of step pair t, lane group kr:
//   TW % 8 == 0: row-major pixel 8 t + 2 kr + e;
//   TW == 28:    row 2 (t / 7) + kr / 2, column 4 (t % 7) + 2 (kr % 2) + e;
//   TW == 14:    row 2 kr + t / 7, column 2 (t % 7) + e
// (pairs never straddle a row).  The lane part goes into the bases, the (t,
// e) part is a compile-time offset.
template <int TW>
struct WgHaloMap {
    static constexpr int kdr(int kr) { return TW == 28 ? kr >> 1 : TW == 14 ? 2 * kr : 0; }
    static constexpr int kdq(int kr) { return TW == 28 ? 2 * (kr & 1) : TW == 14 ? 0 : 2 * kr; }
    static constexpr int dr(int t) { return TW == 28 ? 2 * (t / 7) : TW == 14 ? t / 7 : (8 * t) / TW; }
    static constexpr int dq(int t) { return TW == 28 ? 4 * (t % 7) : TW == 14 ? 2 * (t % 7) : (8 * t) % TW; }
    static_assert(TW % 8 == 0 || TW == 28 || TW == 14, "pixel pairs");
};

// Nine taps of 16 filters x 16 channels from one staged block: A from Yc at
// lane offset ya, B from Xc at lane offset xw (both even), into acc[tap];
// the A values are summed into bsum when do_bias.  mid() runs after the
// MFMAs of step pair MIDT (a place for the next block's DMA that does not
// compete with the first LDS reads of the block).
struct WgNoMid {
    __device__ void operator()() const {}
};
template <int TW, bool SODD, int MIDT = -1, class Mid = WgNoMid>
__device__ __forceinline__ void wg_halo_block_mfma(const float *Yc, const float *Xc, int ya, int xw,
                                                   f32x4 (&acc)[9], bool do_bias, float &bsum,
                                                   const Mid &mid = Mid())
{
    typedef WgHaloCfg<TW> C;
    typedef WgHaloMap<TW> M;
    const float *yp = Yc + opaque(ya), *xp = Xc + opaque(xw);
    float av[28];
#pragma unroll
    for (int t = 0; t < 14; t++) {
        const f32x2 v = lds_b64(yp, M::dr(t) * TW + M::dq(t));
        av[2 * t] = v.x;
        av[2 * t + 1] = v.y;
    }
    if (do_bias) {
#pragma unroll
        for (int st = 0; st < 28; st++)
            bsum += av[st];
    }
    // B words of step pair t, read one pair ahead of their MFMAs.
    constexpr int NRD = SODD ? 3 : 2;
    f32x2 wb[2][3][NRD];
    auto load_b = [&](f32x2 (&dst)[3][NRD], int t) {
#pragma unroll
        for (int r = 0; r < 3; r++)
#pragma unroll
            for (int k = 0; k < NRD; k++)
                dst[r][k] = lds_b64(xp, (M::dr(t) + r) * C::HWW + M::dq(t) + 2 * k);
    };
    load_b(wb[0], 0);
    // Taps innermost: the nine accumulators are independent, so consecutive
    // MFMAs never wait for each other's result.
#pragma unroll
    for (int t = 0; t < 14; t++) {
        if (t + 1 < 14)
            load_b(wb[(t + 1) & 1], t + 1);
        const f32x2(&wc)[3][NRD] = wb[t & 1];
#pragma unroll
        for (int e = 0; e < 2; e++)
#pragma unroll
            for (int tap = 0; tap < 9; tap++) {
                const int r = tap / 3, i = e + tap % 3 + (SODD ? 1 : 0);  // word of the row
                acc[tap] = mfma16(av[2 * t + e], wc[r][i >> 1][i & 1], acc[tap]);
            }
        __builtin_amdgcn_sched_barrier(0);
        if (t == MIDT) {
            mid();
            __builtin_amdgcn_sched_barrier(0);
        }
    }
}

// Work item of a workgroup: split, group, filter tile m0, channel tile c0
// (NCH channels) and the split's pixel blocks [b_beg, b_end).
struct WgHaloTile {
    int split, g, m0, c0, b_beg, b_end;
    __device__ WgHaloTile(const WgradHaloArgs &a, int nch)
    {
        const int mtiles = (a.Kg + 63) / 64, ctiles = a.Cg / nch;
        const int tiles = mtiles * ctiles;
        const int lin = xcd_tile(blockIdx.x, tiles * a.groups * a.nsplit);
        split = lin / (tiles * a.groups);
        const int rest = lin - split * tiles * a.groups;
        g = rest / tiles;
        const int tile = rest - g * tiles;
        m0 = (tile % mtiles) * 64;
        c0 = (tile / mtiles) * nch;
        const int nblocks = a.nimg * a.row_blocks * a.col_segs;
        b_beg = split * a.chunk;
        b_end = min(nblocks, b_beg + a.chunk);
    }
};

// Partial sums of a wave's nine 16 x 16 tiles (filters m0 + fk .., channels
// c0 + fc ..) and, when do_bias, of its 16 filters' bias gradient.
__device__ __forceinline__ void wg_halo_store(const WgradHaloArgs &a, const WgHaloTile &w, int fk, int fc,
                                              const f32x4 (&acc)[9], bool do_bias, float bsum)
{
    const int lane = threadIdx.x & 63, kr = lane >> 4, lc = lane & 15;
    if (do_bias) {
        // The four lane groups of a filter row summed disjoint pixels;
        // combine them in a fixed order.
        bsum += __shfl_xor(bsum, 16, 64);
        bsum += __shfl_xor(bsum, 32, 64);
        const int k = w.m0 + fk + lc;
        if (kr == 0 && k < a.Kg)
            a.db_part[(long long)w.split * a.K + w.g * a.Kg + k] = bsum;
    }
    float *outs = a.out + (long long)w.split * a.split_stride;
#pragma unroll
    for (int tap = 0; tap < 9; tap++)
#pragma unroll
        for (int v = 0; v < 4; v++) {
            const int k = w.m0 + fk + 4 * kr + v;
            if (k < a.Kg)
                outs[((long long)(w.g * a.Kg + k) * 9 + tap) * a.Cg + w.c0 + fc + lc] = acc[tap][v];
        }
}

// Single-stage kernel: NW = 4 waves, each the nine taps of 16 filters x the
// CT 16-channel sub-tiles of the workgroup's 64 x 16 CT tile, or NW = 8 waves
// (CT = 2), each one sub-tile.  Per block: barrier, DMA, wait, barrier, MFMAs.
// Three four-wave workgroups fit a CU with one sub-tile, two with two (which
// stage each block's dy once for twice the MFMAs, and read dy from memory
// half as often over the channel tiles); two eight-wave ones, four waves a
// SIMD, each workgroup's DMA wait covered by the other's MFMAs.
template <int TW, int CT, bool SODD, int NW = 4>
__global__ __launch_bounds__(NW * 64) void wgrad_halo_kernel(const WgradHaloArgs a)
{
    typedef WgHaloStage<TW, 16 * CT, NW> St;
    typedef WgHaloMap<TW> M;
    constexpr int CTW = CT * 4 / NW;  // sub-tiles of a wave
    static_assert(NW == 4 || (NW == 8 && CT == 2), "four waves, or eight over two sub-tiles");
    __shared__ __attribute__((aligned(16))) float Y[St::YW];
    __shared__ __attribute__((aligned(16))) float X[St::XW];

    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int wm = wave & 3, wj = wave >> 2;  // filters 16 wm .., sub-tiles wj CTW ..
    const int kr = lane >> 4, lc = lane & 15;
    const WgHaloTile w(a, 16 * CT);
    const __amdgpu_buffer_rsrc_t rdy = make_rsrc(a.dy, a.dy_bytes);
    const __amdgpu_buffer_rsrc_t rx = make_rsrc(a.x, a.x_bytes);
    St st;
    st.init(wave, lane);

    const int ya = (16 * wm + lc) * kWhDyLd + M::kdr(kr) * TW + M::kdq(kr);
    const int xw = (16 * wj * CTW + lc) * St::CS + a.slack - (SODD ? 1 : 0) + M::kdr(kr) * St::HWW +
                   M::kdq(kr);  // even

    f32x4 acc[CTW][9];
#pragma unroll
    for (int j = 0; j < CTW; j++)
#pragma unroll
        for (int t = 0; t < 9; t++)
            acc[j][t] = f32x4{0.f, 0.f, 0.f, 0.f};
    float bsum = 0.f;
    const bool do_bias = a.db_part != nullptr && w.c0 == 0 && wj == 0;

    for (int b = w.b_beg; b < w.b_end; b++) {
        // Every wave is done reading the previous block.
        __builtin_amdgcn_s_barrier();
        __asm__ volatile("" ::: "memory");
        st.issue(a, rdy, rx, wave, b, w.g, w.m0, w.c0, Y, X);
        __builtin_amdgcn_s_waitcnt(0);
        __asm__ volatile("" ::: "memory");
        __builtin_amdgcn_s_barrier();
        __asm__ volatile("" ::: "memory");
#pragma unroll
        for (int j = 0; j < CTW; j++)
            wg_halo_block_mfma<TW, SODD>(Y, X + j * 16 * St::CS, ya, xw, acc[j], do_bias && j == 0, bsum);
    }
#pragma unroll
    for (int j = 0; j < CTW; j++)
        wg_halo_store(a, w, 16 * wm, 16 * (wj * CTW + j), acc[j], do_bias && j == 0, bsum);
}

// Double-buffered kernel: eight waves (two per SIMD), 64 filters x 32
// channels, pixel blocks staged one ahead.  Wave w computes the nine taps of
// filters 16 (w % 4) .. + 15 and channels 16 (w / 4) .. + 15 of the tile.
// While the waves run the MFMAs of block b from one LDS stage, the DMA of
// block b + 1 fills the other, so a block costs one barrier and no exposed
// load latency.  Two stages take 99-152 KiB of LDS: one workgroup a CU.  The
// two stages are distinct arrays (blocks are taken in pairs), so the
// compiler's wait for in-flight DMA before an LDS read only ever covers the
// stage being read.
template <int TW, bool SODD>
__global__ __launch_bounds__(512) void wgrad_halo_db_kernel(const WgradHaloArgs a)
{
    typedef WgHaloStage<TW, 32, 8> St;
    typedef WgHaloMap<TW> M;
    static_assert(2 * (St::YW + St::XW) * 4 <= 160 * 1024, "two stages in LDS");
    __shared__ __attribute__((aligned(16))) float Y0[St::YW];
    __shared__ __attribute__((aligned(16))) float X0[St::XW];
    __shared__ __attribute__((aligned(16))) float Y1[St::YW];
    __shared__ __attribute__((aligned(16))) float X1[St::XW];

    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int wm = wave & 3, wj = wave >> 2;
    const int kr = lane >> 4, lc = lane & 15;
    const WgHaloTile w(a, 32);
    const __amdgpu_buffer_rsrc_t rdy = make_rsrc(a.dy, a.dy_bytes);
    const __amdgpu_buffer_rsrc_t rx = make_rsrc(a.x, a.x_bytes);
    St st;
    st.init(wave, lane);

    const int ya = (16 * wm + lc) * kWhDyLd + M::kdr(kr) * TW + M::kdq(kr);
    const int xw = (16 * wj + lc) * St::CS + a.slack - (SODD ? 1 : 0) + M::kdr(kr) * St::HWW +
                   M::kdq(kr);  // even

    f32x4 acc[9];
#pragma unroll
    for (int t = 0; t < 9; t++)
        acc[t] = f32x4{0.f, 0.f, 0.f, 0.f};
    float bsum = 0.f;
    const bool do_bias = a.db_part != nullptr && w.c0 == 0 && wj == 0;

    // One block: wait for this wave's DMA of it, barrier (every wave's DMA
    // has landed and every wave is done with the other stage), start the DMA
    // of the next block into the other stage, compute.
    auto block = [&](int b, const float *Yc, const float *Xc, float *Yn, float *Xn) {
        __builtin_amdgcn_s_waitcnt(0);
        __asm__ volatile("" ::: "memory");
        __builtin_amdgcn_s_barrier();
        __asm__ volatile("" ::: "memory");
        auto next = [&]() {
            if (b + 1 < w.b_end)
                st.issue(a, rdy, rx, wave, b + 1, w.g, w.m0, w.c0, Yn, Xn);
        };
        wg_halo_block_mfma<TW, SODD, 3>(Yc, Xc, ya, xw, acc, do_bias, bsum, next);
    };

    if (w.b_beg < w.b_end)
        st.issue(a, rdy, rx, wave, w.b_beg, w.g, w.m0, w.c0, Y0, X0);
    int b = w.b_beg;
    for (; b + 1 < w.b_end; b += 2) {
        block(b, Y0, X0, Y1, X1);
        block(b + 1, Y1, X1, Y0, X0);
    }
    if (b < w.b_end)
        block(b, Y0, X0, Y1, X1);
    wg_halo_store(a, w, 16 * wm, 16 * wj, acc, do_bias, bsum);
}

// ---------------------------------------------------------------------------
// Filter packing.
// ---------------------------------------------------------------------------
__global__ void pack_fwd_kernel(const float *__restrict__ w, float *__restrict__ wp, int Kg,
                                int Cg, int R, int S, int cblock, int a_ld, int kmajor,
                                long long total)
{
    long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= total)
        return;
    // m-major: i = (g * Kg + k) * a_ld + kk; k-major: i = (g * a_ld + kk) * Kg + k;
    // zero for kk >= R*S*Cg
    int kk, k, g;
    if (kmajor) {
        k = (int)(i % Kg);
        long long t = i / Kg;
        kk = (int)(t % a_ld);
        g = (int)(t / a_ld);
    } else {
        kk = (int)(i % a_ld);
        long long t = i / a_ld;
        k = (int)(t % Kg);
        g = (int)(t / Kg);
    }
    if (kk >= R * S * Cg) {
        wp[i] = 0.f;
        return;
    }
    int c, rs;
    if (cblock) {  // kk = (cb * RS + rs) * 16 + ci
        int ci = kk % 16, sl = kk / 16;
        rs = sl % (R * S);
        c = (sl / (R * S)) * 16 + ci;
    } else {       // kk = rs * Cg + c
        c = kk % Cg;
        rs = kk / Cg;
    }
    int r = rs / S, s = rs % S;
    wp[i] = w[(((long long)(g * Kg + k) * Cg + c) * R + r) * S + s];
}

__global__ void pack_bwd_phase_kernel(const float *__restrict__ w, float *__restrict__ wr,
                                      int Kg, int Cg, int R, int S, int r0, int s0, int nr,
                                      int ns, int stride, int cblock, int a_ld, int kmajor,
                                      long long total)
{
    long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= total)
        return;
    // m-major: i = (g * Cg + c) * a_ld + kk; k-major: i = (g * a_ld + kk) * Cg + c;
    // zero for kk >= nr*ns*Kg
    int kk, c, g;
    if (kmajor) {
        c = (int)(i % Cg);
        long long t = i / Cg;
        kk = (int)(t % a_ld);
        g = (int)(t / a_ld);
    } else {
        kk = (int)(i % a_ld);
        long long t = i / a_ld;
        c = (int)(t % Cg);
        g = (int)(t / Cg);
    }
    int ntap = nr * ns;
    if (kk >= ntap * Kg) {
        wr[i] = 0.f;
        return;
    }
    int k, tap;
    if (cblock) {  // kk = (kb * ntap + tap) * 16 + ki
        int ki = kk % 16, sl = kk / 16;
        tap = sl % ntap;
        k = (sl / ntap) * 16 + ki;
    } else {       // kk = tap * Kg + k
        k = kk % Kg;
        tap = kk / Kg;
    }
    int r = r0 + stride * (tap / ns), s = s0 + stride * (tap % ns);
    wr[i] = w[(((long long)(g * Kg + k) * Cg + c) * R + r) * S + s];
}

// Blocked backward-data filter.  Input pixel h with h + pad = b hb + ph
// (b = stride * f) receives dy rows p = f hb + u through filter row
// r = ph - stride u, for u = f - 1 - tu, tu < ntr; the taps of all b phases
// share these ntr dy rows, and a (phase, tap) pair whose r falls outside the
// filter gets a zero weight.  Likewise for columns.
__global__ void pack_bwd_block_kernel(const float *__restrict__ w, float *__restrict__ wp, int Kg,
                                      int Cg, int R, int S, int st, int f, int ntr, int nts,
                                      int cblock, int a_ld, int kmajor, long long total)
{
    long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= total)
        return;
    const int b = st * f, M = Cg * b * b;
    int kk, m, g;
    if (kmajor) {
        m = (int)(i % M);
        long long t = i / M;
        kk = (int)(t % a_ld);
        g = (int)(t / a_ld);
    } else {
        kk = (int)(i % a_ld);
        long long t = i / a_ld;
        m = (int)(t % M);
        g = (int)(t / M);
    }
    const int ntap = ntr * nts;
    if (kk >= ntap * Kg) {
        wp[i] = 0.f;
        return;
    }
    int k, tap;
    if (cblock) {  // kk = (kb * ntap + tap) * 16 + ki
        int ki = kk % 16, sl = kk / 16;
        tap = sl % ntap;
        k = (sl / ntap) * 16 + ki;
    } else {       // kk = tap * Kg + k
        k = kk % Kg;
        tap = kk / Kg;
    }
    const int c = m / (b * b), ph = (m / b) % b, pw = m % b;
    const int r = ph - st * (f - 1 - tap / nts), s = pw - st * (f - 1 - tap % nts);
    wp[i] = (r >= 0 && r < R && s >= 0 && s < S)
                ? w[(((long long)(g * Kg + k) * Cg + c) * R + r) * S + s]
                : 0.f;
}

// ---------------------------------------------------------------------------
// Explicit plan: im2col and col2im (memory-bound; one thread per written
// element, the index decoded with constant-divisor division).
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void im2col_kernel(const float *__restrict__ x,
                                                     float *__restrict__ col, FastDiv pq,
                                                     FastDiv q_, FastDiv rs, FastDiv s_,
                                                     int H, int W, int stride, int pad,
                                                     long long total)
{
    for (long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x; i < total;
         i += (long long)gridDim.x * blockDim.x) {
        // i = row * PQ + pix, row = (n * C + c) * RS + tap; total < 2^31
        const uint32_t row = fast_div((uint32_t)i, pq);
        const uint32_t pix = (uint32_t)i - row * pq.d;
        const uint32_t p = fast_div(pix, q_), q = pix - p * q_.d;
        const uint32_t nc = fast_div(row, rs), tap = row - nc * rs.d;
        const uint32_t r = fast_div(tap, s_), sx = tap - r * s_.d;
        const int h = (int)(p * stride + r) - pad, w = (int)(q * stride + sx) - pad;
        float v = 0.f;
        if ((unsigned)h < (unsigned)H && (unsigned)w < (unsigned)W)
            v = x[((long long)nc * H + h) * W + w];
        col[i] = v;
    }
}

__global__ __launch_bounds__(256) void col2im_kernel(const float *__restrict__ col,
                                                     float *__restrict__ dx, FastDiv hw,
                                                     FastDiv w_, int R, int S, int stride,
                                                     int pad, int P, int Q, long long total)
{
    for (long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x; i < total;
         i += (long long)gridDim.x * blockDim.x) {
        // i = nc * HW + h * W + w; total < 2^31
        const uint32_t nc = fast_div((uint32_t)i, hw);
        const uint32_t pix = (uint32_t)i - nc * hw.d;
        const uint32_t h = fast_div(pix, w_), w = pix - h * w_.d;
        const long long base = (long long)nc * R * S * P * Q;
        float acc = 0.f;
        for (int r = 0; r < R; r++) {
            const int hp = (int)h + pad - r;
            if (hp < 0 || hp % stride)
                continue;
            const int p = hp / stride;
            if (p >= P)
                continue;
            for (int s = 0; s < S; s++) {
                const int wp = (int)w + pad - s;
                if (wp < 0 || wp % stride)
                    continue;
                const int q = wp / stride;
                if (q >= Q)
                    continue;
                acc += col[base + ((long long)(r * S + s) * P + p) * Q + q];
            }
        }
        dx[i] = acc;
    }
}

// out[c][r] = in[r][c] for a rows x cols row-major matrix: 32 x 32 tiles
// through LDS (rows padded to 33 words), coalesced on both sides.
__global__ __launch_bounds__(256) void transpose_kernel(const float *__restrict__ in,
                                                        float *__restrict__ out, int rows,
                                                        int cols)
{
    __shared__ float t[32][33];
    const int c0 = blockIdx.x * 32, r0 = blockIdx.y * 32;
    const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;
    for (int j = ty; j < 32; j += 8) {
        const int r = r0 + j, c = c0 + tx;
        if (r < rows && c < cols)
            t[j][tx] = in[(size_t)r * cols + c];
    }
    __syncthreads();
    for (int j = ty; j < 32; j += 8) {
        const int c = c0 + j, r = r0 + tx;
        if (c < cols && r < rows)
            out[(size_t)c * rows + r] = t[tx][j];
    }
}

// ---------------------------------------------------------------------------
// Deterministic split-K reduction.  out[dst(i)] = sum over s < nsplit of
// part[s * stride + i].  A block handles 32 V consecutive elements with 8
// threads each (a thread V consecutive ones, V = 4 with 16-byte loads where
// the count, the split stride and the buffer allow): thread j sums splits j,
// j + 8, j + 16, ... in order, and the 8 partial sums are then added in the
// order j = 0..7, so the result depends only on nsplit (and not on V).  dst
// is the identity, or (tap_cg > 0) the move from the tap-uniform kernel's
// [k][tap][c] order to dw's [k][c][tap] order.
// ---------------------------------------------------------------------------
constexpr int RED_E = 32, RED_J = 8;

template <int V>
__global__ __launch_bounds__(RED_E * RED_J) void splitk_reduce_kernel(
    const float *__restrict__ part, int nsplit, long long stride, int count,
    float *__restrict__ out, int taps, int tap_cg)
{
    __shared__ float sh[RED_J][RED_E * V];
    const int e = threadIdx.x % RED_E, j = threadIdx.x / RED_E;
    for (int base = blockIdx.x * RED_E * V; base < count; base += gridDim.x * RED_E * V) {
        const int i0 = base + V * e;  // V = 4: count % 4 = 0, so i0 + 3 < count with i0
        float sv[V];
#pragma unroll
        for (int v = 0; v < V; v++)
            sv[v] = 0.f;
        if (i0 < count)
            for (int k = j; k < nsplit; k += RED_J) {
                if constexpr (V == 4) {
                    const f32x4 x = *(const f32x4 *)&part[(long long)k * stride + i0];
#pragma unroll
                    for (int v = 0; v < 4; v++)
                        sv[v] += x[v];
                } else {
                    sv[0] += part[(long long)k * stride + i0];
                }
            }
#pragma unroll
        for (int v = 0; v < V; v++)
            sh[j][V * e + v] = sv[v];
        __syncthreads();
        if (j == 0 && i0 < count) {
#pragma unroll
            for (int v = 0; v < V; v++) {
                float t = sh[0][V * e + v];
#pragma unroll
                for (int jj = 1; jj < RED_J; jj++)
                    t += sh[jj][V * e + v];
                const int i = i0 + v;
                int d = i;
                if (tap_cg > 0) {
                    const int per = taps * tap_cg;
                    const int k = i / per, rem = i - k * per;
                    const int tap = rem / tap_cg, c = rem - tap * tap_cg;
                    d = k * per + c * taps + tap;
                }
                out[d] = t;
            }
        }
        __syncthreads();
    }
}

// ---------------------------------------------------------------------------
// Launchers.
// ---------------------------------------------------------------------------

// Whether a launch is a 1x1 direct GEMM the ONE variant can stage with
// 16-byte loads: one tap, stride 1, no offset, the source pixel index equal
// to the column's, channel-aligned slices, pixels per image a multiple of 4.
static bool one_by_one_direct(const ImgGemmArgs &a, bool fast)
{
    return fast && a.k_taps.d == 1 && a.k_tw.d == 1 && a.cstep == 1 && a.coff_h == 0 &&
           a.coff_w == 0 && a.mblock <= 1 && a.src_hw == (int)a.col_hw.d &&
           a.src_w == (int)a.col_w.d && a.col_hw.d % 4 == 0;
}

template <int BM, int BN, int BK, int WM, int WN, int PAD>
static hipError_t img_launch(const ImgGemmArgs &a, bool fast, hipStream_t stream)
{
    constexpr int NST = 3;
    int tiles = ((a.M + BM - 1) / BM) * ((a.Ncol + BN - 1) / BN);
    dim3 grid(tiles * a.groups * a.nsplit);
    if constexpr (BN == 64 && WM > 1) {
        if (one_by_one_direct(a, fast)) {
            hipLaunchKernelGGL((img_gemm_kernel<BM, BN, BK, WM, WN, PAD, true, NST, true>), grid,
                               dim3(64 * WM * WN), 0, stream, a);
            return hipGetLastError();
        }
    }
    if (fast)
        hipLaunchKernelGGL((img_gemm_kernel<BM, BN, BK, WM, WN, PAD, true, NST>), grid,
                           dim3(64 * WM * WN), 0, stream, a);
    else
        hipLaunchKernelGGL((img_gemm_kernel<BM, BN, BK, WM, WN, PAD, false, NST>), grid,
                           dim3(64 * WM * WN), 0, stream, a);
    return hipGetLastError();
}

#ifndef MICONV_IMG_BK
#define MICONV_IMG_BK 16
#endif

hipError_t launch_img_gemm(const ImgGemmArgs &a, int tile, bool fast, hipStream_t stream)
{
    constexpr int K = MICONV_IMG_BK;
    switch (tile) {
    // Every shape runs on the 16x16x4 MFMA with LDS rows padded by 4 words,
    // so that its four 16-lane groups, which read rows 4 apart, hit distinct
    // banks.  Waves: 4 x 1 or 3 x 1 (each wave a 16- or 32-row band across
    // the tile), 2 x 2, or 1 x 4 (each wave a column band, 16 rows).
    case IMG_128x64: return img_launch<128, 64, K, 4, 1, 4>(a, fast, stream);
    case IMG_16x128: return img_launch<16, 128, K, 1, 4, 4>(a, fast, stream);
    case IMG_32x64: return img_launch<32, 64, K, 2, 2, 4>(a, fast, stream);
    case IMG_48x64: return img_launch<48, 64, K, 3, 1, 4>(a, fast, stream);
    case IMG_96x64: return img_launch<96, 64, K, 2, 2, 4>(a, fast, stream);
    case IMG_96x128: return img_launch<96, 128, K, 2, 2, 4>(a, fast, stream);
    case IMG_128x128: return img_launch<128, 128, K, 2, 2, 4>(a, fast, stream);
    case IMG_64x128: return img_launch<64, 128, K, 2, 2, 4>(a, fast, stream);
    default: return img_launch<64, 64, K, 4, 1, 4>(a, fast, stream);
    }
}

template <int BM, int TW, int TR, int R>
static hipError_t halo_launch(const HaloGemmArgs &a, bool flip, hipStream_t stream)
{
    const int tiles = ((a.M + BM - 1) / BM) * a.nimg * a.row_blocks * a.col_segs;
    const dim3 grid(tiles * a.groups * a.nsplit), block(256);
    if constexpr (R == 3 && TR * TW == kHaloCols && TW != 112) {
        if (a.ks == 2) {
            if (flip)
                hipLaunchKernelGGL((halo_gemm_kernel<BM, TW, TR, R, true, 2>), grid, dim3(512), 0, stream, a);
            else
                hipLaunchKernelGGL((halo_gemm_kernel<BM, TW, TR, R, false, 2>), grid, dim3(512), 0, stream, a);
            return hipGetLastError();
        }
    }
    if (a.ks != 1)
        return hipErrorInvalidValue;
    if (flip)
        hipLaunchKernelGGL((halo_gemm_kernel<BM, TW, TR, R, true>), grid, block, 0, stream, a);
    else
        hipLaunchKernelGGL((halo_gemm_kernel<BM, TW, TR, R, false>), grid, block, 0, stream, a);
    return hipGetLastError();
}

template <int BM>
static hipError_t halo_launch_tw(const HaloGemmArgs &a, bool flip, hipStream_t stream)
{
    if (a.TR * a.TW != kHaloCols) {  // whole-image blocks: 64-row tiles
        if constexpr (BM == 64) {
            if (a.R == 3 && a.TW == 13 && a.TR == 13)
                return halo_launch<BM, 13, 13, 3>(a, flip, stream);
        }
        return hipErrorInvalidValue;
    }
    if (a.R == 5)
        switch (a.TW) {
        case 28: return halo_launch<BM, 28, 4, 5>(a, flip, stream);
        case 14: return halo_launch<BM, 14, 8, 5>(a, flip, stream);
        default: return hipErrorInvalidValue;
        }
    switch (a.TW) {
    case 112: return halo_launch<BM, 112, 1, 3>(a, flip, stream);
    case 56: return halo_launch<BM, 56, 2, 3>(a, flip, stream);
    case 28: return halo_launch<BM, 28, 4, 3>(a, flip, stream);
    case 14: return halo_launch<BM, 14, 8, 3>(a, flip, stream);
    default: return hipErrorInvalidValue;
    }
}

bool wgrad_halo_supported(int TW, int P, int Q, int W)
{
    if (TW == 14)  // whole rows of a 14-wide map (contiguous in dy), one-word x loads
        return Q == 14 && P % 2 == 0;
    return (TW == 112 || TW == 56 || TW == 28) && Q % 4 == 0 && W % 4 == 0;
}

template <bool SODD>
static hipError_t wgrad_halo_launch_par(const WgradHaloArgs &a, int tiles, hipStream_t stream)
{
    const dim3 grid(tiles), block(256), block8(512);
    if (a.db == 2) {
        switch (a.TW) {
        case 112: hipLaunchKernelGGL((wgrad_halo_kernel<112, 2, SODD, 8>), grid, block8, 0, stream, a); break;
        case 56: hipLaunchKernelGGL((wgrad_halo_kernel<56, 2, SODD, 8>), grid, block8, 0, stream, a); break;
        case 28: hipLaunchKernelGGL((wgrad_halo_kernel<28, 2, SODD, 8>), grid, block8, 0, stream, a); break;
        default: hipLaunchKernelGGL((wgrad_halo_kernel<14, 2, false, 8>), grid, block8, 0, stream, a); break;
        }
    } else if (a.db) {
        switch (a.TW) {
        case 112: hipLaunchKernelGGL((wgrad_halo_db_kernel<112, SODD>), grid, block8, 0, stream, a); break;
        case 56: hipLaunchKernelGGL((wgrad_halo_db_kernel<56, SODD>), grid, block8, 0, stream, a); break;
        case 28: hipLaunchKernelGGL((wgrad_halo_db_kernel<28, SODD>), grid, block8, 0, stream, a); break;
        default: hipLaunchKernelGGL((wgrad_halo_db_kernel<14, false>), grid, block8, 0, stream, a); break;
        }
    } else if (a.CT == 2) {
        switch (a.TW) {
        case 112: hipLaunchKernelGGL((wgrad_halo_kernel<112, 2, SODD>), grid, block, 0, stream, a); break;
        case 56: hipLaunchKernelGGL((wgrad_halo_kernel<56, 2, SODD>), grid, block, 0, stream, a); break;
        case 28: hipLaunchKernelGGL((wgrad_halo_kernel<28, 2, SODD>), grid, block, 0, stream, a); break;
        default: hipLaunchKernelGGL((wgrad_halo_kernel<14, 2, false>), grid, block, 0, stream, a); break;
        }
    } else {
        switch (a.TW) {
        case 112: hipLaunchKernelGGL((wgrad_halo_kernel<112, 1, SODD>), grid, block, 0, stream, a); break;
        case 56: hipLaunchKernelGGL((wgrad_halo_kernel<56, 1, SODD>), grid, block, 0, stream, a); break;
        case 28: hipLaunchKernelGGL((wgrad_halo_kernel<28, 1, SODD>), grid, block, 0, stream, a); break;
        default: hipLaunchKernelGGL((wgrad_halo_kernel<14, 1, false>), grid, block, 0, stream, a); break;
        }
    }
    return hipGetLastError();
}

hipError_t launch_wgrad_halo(const WgradHaloArgs &a, hipStream_t stream)
{
    // col0: the x halo's first column relative to q0, -pad for one-word
    // loads, rounded down to a multiple of 4 for 16-byte ones.
    if (!wgrad_halo_supported(a.TW, a.P, a.Q, a.W) || (a.TW == 14 ? a.slack != 0 : a.col0 % 4 != 0))
        return hipErrorInvalidValue;
    if ((a.CT != 1 && a.CT != 2) || a.Cg % (16 * a.CT) || a.slack < 0 || a.slack > 3 ||
        a.db < 0 || a.db > 2 || (a.db && a.CT != 2))
        return hipErrorInvalidValue;
    const int tiles = ((a.Kg + 63) / 64) * (a.Cg / (16 * a.CT)) * a.groups * a.nsplit;
    return (a.slack & 1) ? wgrad_halo_launch_par<true>(a, tiles, stream)
                         : wgrad_halo_launch_par<false>(a, tiles, stream);
}

bool halo_whole_image(int TW, int TR, int R)
{
    return R == 3 && TW == 13 && TR == 13;
}

int halo_load_words(int TW, int TR, int R)
{
    return R == 3 && TW != 14 && !halo_whole_image(TW, TR, R) ? 4 : 1;
}

bool halo_block_supported(int TW, int TR, int R, int src_w, int col0)
{
    if (TR * TW != kHaloCols)
        return halo_whole_image(TW, TR, R);  // one-word loads
    if (R == 5)
        return TW == 28 || TW == 14;  // one-word loads
    if (R != 3)
        return false;
    if (TW == 14)
        return true;  // one-word loads
    return (TW == 112 || TW == 56 || TW == 28) && src_w % 4 == 0 && col0 % 4 == 0;
}

hipError_t launch_halo_gemm(const HaloGemmArgs &a, int tile, bool flip, hipStream_t stream)
{
    // slack (the first tap's column in the halo row) must lie within one
    // load group: the halo rows hold slack + TW + R - 1 words.
    if (!halo_block_supported(a.TW, a.TR, a.R, a.src_w, a.col0) ||
        a.Kred != a.cin * a.R * a.R || a.slack < 0 || a.slack >= halo_load_words(a.TW, a.TR, a.R))
        return hipErrorInvalidValue;
    // Two wave groups: 3 x 3 blocks 56, 28 or 14 wide, unsplit, an even number
    // of channel blocks (one half per group).
    if (a.ks == 2 && (a.R != 3 || a.TR * a.TW != kHaloCols || a.TW == 112 || a.nsplit != 1 ||
                      (a.cin / 16) % 2 != 0 || a.cbchunk != a.cin / 16))
        return hipErrorInvalidValue;
    return tile == HALO_128x112 ? halo_launch_tw<128>(a, flip, stream)
                                : halo_launch_tw<64>(a, flip, stream);
}

template <int BM, int BN, int WM, int WN, bool PACKED = false>
static hipError_t wgrad_launch(const WgradArgs &a, hipStream_t stream)
{
    int RS = (int)a.n_rs.d;
    int ntiles = PACKED ? (a.Ncol + BN - 1) / BN : RS * ((a.Cg + BN - 1) / BN);
    int tiles = ((a.M + BM - 1) / BM) * ntiles;
    hipLaunchKernelGGL((wgrad_kernel<BM, BN, WM, WN, PACKED>),
                       dim3(tiles * a.groups * a.nsplit), dim3(64 * WM * WN), 0, stream, a);
    return hipGetLastError();
}

hipError_t launch_wgrad_gemm(const WgradArgs &a, int tile, hipStream_t stream)
{
    switch (tile) {
    case WG_TAP_64x32: return wgrad_launch<64, 32, 2, 2>(a, stream);
    case WG_TAP_64x48: return wgrad_launch<64, 48, 4, 1>(a, stream);
    case WG_TAP_64x16: return wgrad_launch<64, 16, 4, 1>(a, stream);
    case WG_TAP_128x32: return wgrad_launch<128, 32, 4, 1>(a, stream);
    case WG_TAP_64x64: return wgrad_launch<64, 64, 2, 2>(a, stream);
    case WG_TAP_128x64: return wgrad_launch<128, 64, 2, 2>(a, stream);
    case WG_PIX_96x64: return wgrad_launch<96, 64, 2, 2, true>(a, stream);
    case WG_PIX_64x64: return wgrad_launch<64, 64, 4, 1, true>(a, stream);
    case WG_PIX_64x32: return wgrad_launch<64, 32, 2, 2, true>(a, stream);
    default: return hipErrorInvalidValue;
    }
}

static unsigned blocks_for(long long total, int nt)
{
    return (unsigned)((total + nt - 1) / nt);
}

hipError_t launch_pack_fwd(const float *w, float *wp, int K, int Cg, int R, int S, int G,
                           bool cblock, int a_ld, bool kmajor, hipStream_t stream)
{
    long long total = (long long)K * a_ld;
    hipLaunchKernelGGL(pack_fwd_kernel, dim3(blocks_for(total, 256)), dim3(256), 0, stream, w,
                       wp, K / G, Cg, R, S, cblock ? 1 : 0, a_ld, kmajor ? 1 : 0, total);
    return hipGetLastError();
}

hipError_t launch_pack_bwd_phase(const float *w, float *wr, int K, int Cg, int R, int S,
                                 int G, int r0, int s0, int nr, int ns, int stride, bool cblock,
                                 int a_ld, bool kmajor, hipStream_t stream)
{
    long long total = (long long)G * Cg * a_ld;
    if (total == 0)
        return hipSuccess;
    hipLaunchKernelGGL(pack_bwd_phase_kernel, dim3(blocks_for(total, 256)), dim3(256), 0,
                       stream, w, wr, K / G, Cg, R, S, r0, s0, nr, ns, stride, cblock ? 1 : 0,
                       a_ld, kmajor ? 1 : 0, total);
    return hipGetLastError();
}

hipError_t launch_pack_bwd_block(const float *w, float *wp, int K, int Cg, int R, int S, int G,
                                 int stride, int f, int ntr, int nts, bool cblock, int a_ld,
                                 bool kmajor, hipStream_t stream)
{
    const int b = stride * f;
    long long total = (long long)G * Cg * b * b * a_ld;
    hipLaunchKernelGGL(pack_bwd_block_kernel, dim3(blocks_for(total, 256)), dim3(256), 0, stream,
                       w, wp, K / G, Cg, R, S, stride, f, ntr, nts, cblock ? 1 : 0, a_ld,
                       kmajor ? 1 : 0, total);
    return hipGetLastError();
}

static unsigned grid_for(long long total)
{
    long long b = (total + 255) / 256;
    return (unsigned)(b < 65536 ? b : 65536);
}

hipError_t launch_im2col(const float *x, float *col, int n, int C, int H, int W, int R, int S,
                         int stride, int pad, int P, int Q, hipStream_t stream)
{
    const long long total = (long long)n * C * R * S * P * Q;
    hipLaunchKernelGGL(im2col_kernel, dim3(grid_for(total)), dim3(256), 0, stream, x, col,
                       make_fastdiv(P * Q), make_fastdiv(Q), make_fastdiv(R * S),
                       make_fastdiv(S), H, W, stride, pad, total);
    return hipGetLastError();
}

hipError_t launch_col2im(const float *col, float *dx, int n, int C, int H, int W, int R, int S,
                         int stride, int pad, int P, int Q, hipStream_t stream)
{
    const long long total = (long long)n * C * H * W;
    hipLaunchKernelGGL(col2im_kernel, dim3(grid_for(total)), dim3(256), 0, stream, col, dx,
                       make_fastdiv(H * W), make_fastdiv(W), R, S, stride, pad, P, Q, total);
    return hipGetLastError();
}

hipError_t launch_transpose(const float *in, float *out, int rows, int cols, hipStream_t stream)
{
    dim3 grid((cols + 31) / 32, (rows + 31) / 32);
    hipLaunchKernelGGL(transpose_kernel, grid, dim3(256), 0, stream, in, out, rows, cols);
    return hipGetLastError();
}

// Split-K reduction of the image GEMM: same fixed order as splitk_reduce_kernel
// (8 threads per element, strided over splits, combined in thread order; V
// consecutive elements a thread), then + bias of the element's channel.
template <int V>
__global__ __launch_bounds__(RED_E * RED_J) void splitk_bias_reduce_kernel(
    const float *__restrict__ part, int nsplit, long long stride, int count,
    const float *__restrict__ bias, FastDiv hw, FastDiv K, float *__restrict__ out)
{
    __shared__ float sh[RED_J][RED_E * V];
    const int e = threadIdx.x % RED_E, j = threadIdx.x / RED_E;
    for (int base = blockIdx.x * RED_E * V; base < count; base += gridDim.x * RED_E * V) {
        const int i0 = base + V * e;  // V = 4: count % 4 = 0, so i0 + 3 < count with i0
        float sv[V];
#pragma unroll
        for (int v = 0; v < V; v++)
            sv[v] = 0.f;
        if (i0 < count)
            for (int k = j; k < nsplit; k += RED_J) {
                if constexpr (V == 4) {
                    const f32x4 x = *(const f32x4 *)&part[(long long)k * stride + i0];
#pragma unroll
                    for (int v = 0; v < 4; v++)
                        sv[v] += x[v];
                } else {
                    sv[0] += part[(long long)k * stride + i0];
                }
            }
#pragma unroll
        for (int v = 0; v < V; v++)
            sh[j][V * e + v] = sv[v];
        __syncthreads();
        if (j == 0 && i0 < count) {
#pragma unroll
            for (int v = 0; v < V; v++) {
                float t = sh[0][V * e + v];
#pragma unroll
                for (int jj = 1; jj < RED_J; jj++)
                    t += sh[jj][V * e + v];
                const int i = i0 + v;
                if (bias) {
                    const uint32_t q = fast_div((uint32_t)i, hw);
                    t += bias[q - fast_div(q, K) * K.d];
                }
                out[i] = t;
            }
        }
        __syncthreads();
    }
}

// The 16-byte form of the split reductions where the count, the split stride
// and the buffer allow it and the count gives at least 2048 blocks of 128
// elements: 10-15 us faster per reduction of 2-10 M elements (VGG-16 conv4_x,
// conv5_x backward-weight, image-GEMM split-K partials); on smaller counts
// with many splits (conv1_2: 37 K elements, 128 splits) the one-word form's
// four times as many blocks measured 2-6 us faster.
static bool reduce_vec(const float *part, long long stride, int count)
{
    return count % 4 == 0 && stride % 4 == 0 && (uintptr_t)part % 16 == 0 && count >= 2048 * 128;
}

hipError_t launch_splitk_bias_reduce(const float *part, int nsplit, long long stride, int count,
                                     const float *bias, int hw, int K, float *out,
                                     hipStream_t stream)
{
    const bool vec = reduce_vec(part, stride, count);
    const int per_block = RED_E * (vec ? 4 : 1);
    long long blocks = (count + per_block - 1) / per_block;
    if (blocks > 65536)
        blocks = 65536;
    if (vec)
        hipLaunchKernelGGL(splitk_bias_reduce_kernel<4>, dim3((unsigned)blocks), dim3(RED_E * RED_J),
                           0, stream, part, nsplit, stride, count, bias, make_fastdiv(hw),
                           make_fastdiv(K), out);
    else
        hipLaunchKernelGGL(splitk_bias_reduce_kernel<1>, dim3((unsigned)blocks), dim3(RED_E * RED_J),
                           0, stream, part, nsplit, stride, count, bias, make_fastdiv(hw),
                           make_fastdiv(K), out);
    return hipGetLastError();
}

hipError_t launch_splitk_reduce(const float *part, int nsplit, long long stride, int count,
                                float *out, int taps, int tap_cg, hipStream_t stream)
{
    const bool vec = reduce_vec(part, stride, count);
    const int per_block = RED_E * (vec ? 4 : 1);
    long long blocks = (count + per_block - 1) / per_block;
    if (blocks > 65536)
        blocks = 65536;
    if (vec)
        hipLaunchKernelGGL(splitk_reduce_kernel<4>, dim3((unsigned)blocks), dim3(RED_E * RED_J), 0,
                           stream, part, nsplit, stride, count, out, taps, tap_cg);
    else
        hipLaunchKernelGGL(splitk_reduce_kernel<1>, dim3((unsigned)blocks), dim3(RED_E * RED_J), 0,
                           stream, part, nsplit, stride, count, out, taps, tap_cg);
    return hipGetLastError();
}

}  // namespace miconv
