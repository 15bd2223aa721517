// smol_rows_yuv.h -- the I420 row-streaming kernel (yuv_rows_kernel) and the
// choice of its instance for a plan. The smol_rows_yuv_*.hip files instantiate
// its parts.
#pragma once

#include "smol_rows.h"

namespace smol {
namespace {

// ---------------------------------------------------------------------------
// I420, row streaming: one wave per workgroup, the scheme of the RGB kernel.
//
// For each output row the wave loads eight row segments into registers and
// then into its LDS slot (1 KiB each): luma rows y0 and y1 over the crop's
// luma column span and, for each chroma plane, the chroma rows that the
// vertical chroma taps of y0 and y1 read over the matching chroma span. Those
// are at most three rows, staged so that y0 reads chroma rows (r0, r1) and y1
// reads (r1, r2): the taps of consecutive luma rows (y1 = y0 + 1 or the
// clamped y0) either move on by one chroma row (y1's first row is y0's
// second; r2 is y1's second) or stay on y0's pair (y1's second row is y0's
// second; r2 is then y1's first row and y1's weights are swapped, which gives
// the same exact integer sums).
//
// Every luma tap is converted as defined: chroma bilinear at centred siting,
// BT.601 full range, clamp; then the four converted taps are interpolated
// and normalised. The chroma weights are 0, 1/4 and 3/4, so the chroma value
// at a luma tap is S / 16 with S = the sum of its four chroma samples times
// integer weights (4 - fy or fy) * (4 - fx or fx), fx, fy in {0, 1, 3}: every
// interpolation step of the definition is exact, and so is S. One v_dot4
// forms S - 2048 = 16 * (chroma - 128) from the four sample bytes and the four
// weight bytes; the BT.601 products then use the coefficients divided by 16,
// which gives the same real products and so the same rounded values.
//
// Lane l computes output columns c = 2l + 128j and c + 1 (j < J). Per column
// it keeps: the luma tap (offset of x0 in the staged luma span, weight), and
// for its two luma columns x0, x1 the offset of the first chroma column they
// read, per luma column a v_perm selector that picks its two chroma samples
// from each of two chroma rows, and its horizontal weight bytes
// (4 - fx, fx).
// ---------------------------------------------------------------------------
// A frame's plane offsets and the processed region: W x H luma pixels at
// (rx, ry) in a frame of fw x fh (chroma taps use frame coordinates).
struct YuvImg {
    long long off[3];
    int W, H, Wr, Hr, left, top, xf, span;
    int rx, ry, fw, fh;
};

__device__ __forceinline__ YuvImg yuv_img(const BatchArgs &a, int img)
{
    YuvImg g;
    if (a.table) {
        const ConstDesc *t = (const ConstDesc *)a.table + img;
        g.off[0] = t->off[0];
        g.off[1] = t->off[1];
        g.off[2] = t->off[2];
        g.W = t->W;
        g.H = t->H;
        g.Wr = t->Wr;
        g.Hr = t->Hr;
        g.left = t->left;
        g.top = t->top;
        g.xf = t->xf;
        g.span = t->span;
        g.rx = t->rx;
        g.ry = t->ry;
        g.fw = t->pitch;
        g.fh = t->fh;
    } else {
        g.off[0] = a.uni.off[0] + (long long)img * a.stride;
        g.off[1] = a.uni.off[1] + (long long)img * a.stride;
        g.off[2] = a.uni.off[2] + (long long)img * a.stride;
        g.rx = a.uni.rx;
        g.ry = a.uni.ry;
        g.fw = a.uni.pitch;
        g.fh = a.uni.fh;
        g.W = a.uni.W;
        g.H = a.uni.H;
        g.Wr = a.uni.Wr;
        g.Hr = a.uni.Hr;
        g.left = a.uni.left;
        g.top = a.uni.top;
        g.xf = a.uni.xf;
        g.span = a.uni.span;
    }
    return g;
}

// One output row's eight segments in registers: Y y0, Y y1, Cb r0, Cb r1,
// Cb r2, Cr r0, Cr r1, Cr r2 (y0 reads chroma rows r0, r1 and y1 reads r1,
// r2), with each segment's offset in its first chunk, the luma vertical
// weight and the chroma weights of rows r1 (for y0) and r2 (for y1), in
// quarters. A lane holds one 16-byte chunk of each segment, and with GL = 2 a
// second chunk of each luma segment (luma rows of up to 2 KiB).
template <int GL>
struct YuvStaged {
    u32x4 c[8];
    u32x4 c2[2];  // second luma chunks (GL = 2)
    int sh[8];
    float wy;
    int fy0, fy1;  // weights of chroma rows r1 (in y0's pair) and r2 (in y1's), in quarters
};

// Load cursor over the output rows of I420 frames (the walk of the RGB
// cursor, with the three plane bases).
struct YuvCursor {
    int img, rr;
    VCursor v;          // luma vertical map over the region's rows
    double rcp;         // 1 / v.den, rounded to nearest
    uintptr_t base[3];  // first staged byte of the region's row 0 (Y), of chroma row 0 (Cb, Cr)
    int W, Wc, Hc, yspan, cspan;  // frame luma pitch, chroma pitch and rows
    int ry;             // the region's first frame row
};

template <int STRIDE>
__device__ __forceinline__ void yuv_cursor_image(YuvCursor &c, const BatchArgs &a, int img, int rr,
                                                 const RowStep &s)
{
    const YuvImg g = yuv_img(a, img);
    c.img = img;
    c.rr = rr;
    RowImg lg{};
    lg.H = g.H;
    lg.Hr = g.Hr;
    lg.top = g.top;
    vcursor_init<STRIDE>(c.v, a, lg, rr, s);
    c.rcp = 1.0 / (double)c.v.den;
    c.W = g.fw;
    c.Wc = (g.fw + 1) >> 1;
    c.Hc = (g.fh + 1) >> 1;
    c.ry = g.ry;
    const int cxf = chroma_tap(g.rx + g.xf, c.Wc, a.siting).x0;
    const int cxl = chroma_tap(g.rx + g.xf + g.span - 1, c.Wc, a.siting).x1;
    c.yspan = g.span;
    c.cspan = cxl - cxf + 1;
    c.base[0] = (uintptr_t)(a.src + g.off[0]) + (uintptr_t)g.ry * (uintptr_t)g.fw +
                (uintptr_t)(g.rx + g.xf);
    c.base[1] = (uintptr_t)(a.src + g.off[1]) + (uintptr_t)cxf;
    c.base[2] = (uintptr_t)(a.src + g.off[2]) + (uintptr_t)cxf;
}

template <int STRIDE>
__device__ __forceinline__ void yuv_cursor_next(YuvCursor &c, const BatchArgs &a, const RowStep &s)
{
    if (!STRIDE) {
        vcursor_add(c.v, c.v.qs, c.v.rs);
        if (++c.rr == s.Ch && c.img + 1 < a.n)
            yuv_cursor_image<0>(c, a, c.img + 1, 0, s);
        return;
    }
    const int img0 = c.img;
    c.img += s.di;
    c.rr += s.dr;
    const bool wrapped = c.rr >= s.Ch;
    if (wrapped) {
        c.rr -= s.Ch;
        ++c.img;
    }
    if (!a.table) {
        const uintptr_t d = (uintptr_t)(c.img - img0) * (uintptr_t)a.stride;
        c.base[0] += d;
        c.base[1] += d;
        c.base[2] += d;
        vcursor_add(c.v, wrapped ? c.v.qw : c.v.qs, wrapped ? c.v.rw : c.v.rs);
    } else if (c.img != img0) {
        yuv_cursor_image<1>(c, a, c.img, c.rr, s);
    } else {
        vcursor_add(c.v, c.v.qs, c.v.rs);
    }
}

// LDS layout of a wave's slot: luma segments of 1 KiB * GL, then the six
// chroma segments of 1 KiB.
template <int GL>
__device__ __forceinline__ constexpr uint32_t yuv_seg(int s)
{
    return s < 2 ? 1024u * GL * (uint32_t)s : 2048u * GL + 1024u * (uint32_t)(s - 2);
}

// The vertical chroma taps of frame luma row y (centred siting; the rows
// and weight of chroma_tap) with the weight of the second row in quarters.
__device__ __forceinline__ void chroma_rows(int y, int n, int &r0, int &r1, int &f)
{
    const int num = 2 * y - 1;
    const int q = num >> 2;
    if (num <= 0) {
        r0 = r1 = 0;
        f = 0;
    } else if (q >= n - 1) {
        r0 = r1 = n - 1;
        f = 0;
    } else {
        r0 = q;
        r1 = q + 1;
        f = num & 3;
    }
}

template <int GL>
__device__ __forceinline__ void yuv_load(YuvStaged<GL> &st, const YuvCursor &c, int lane,
                                         bool repeat)
{
    int y0, y1;
    if (c.v.q < 0 || (c.v.q == 0 && c.v.rem == 0)) {
        y0 = y1 = 0;
        st.wy = 0.0f;
    } else if (c.v.q >= c.v.H - 1) {
        y0 = y1 = c.v.H - 1;
        st.wy = 0.0f;
    } else {
        y0 = c.v.q;
        y1 = y0 + 1;
        // rem / den rounded to nearest fp32 (0 < rem < den <= 2^24): the
        // fp64 product rem * RN(1 / den) is within 2^-52 (relative) of the
        // quotient, and no such quotient lies within 2^-49 (relative) of a
        // midpoint between fp32 values (that would need 2^25 | den), so
        // both round to the same fp32 value
        st.wy = (float)((double)c.v.rem * c.rcp);
    }
    int a0, a1, f0, b0, b1, f1;
    chroma_rows(c.ry + y0, c.Hc, a0, a1, f0);
    chroma_rows(c.ry + y1, c.Hc, b0, b1, f1);
    // y1's taps move on by one chroma row (b0 == a1) or keep y0's second row
    // (b1 == a1); y1 reads (r1 = a1, r2) either way
    const bool next = b0 == a1;
    const int r2 = next ? b1 : b0;
    st.fy0 = f0;
    st.fy1 = next ? f1 : 4 - f1;
    const uintptr_t row[8] = {
        c.base[0] + (uintptr_t)y0 * (uintptr_t)c.W,  c.base[0] + (uintptr_t)y1 * (uintptr_t)c.W,
        c.base[1] + (uintptr_t)a0 * (uintptr_t)c.Wc, c.base[1] + (uintptr_t)a1 * (uintptr_t)c.Wc,
        c.base[1] + (uintptr_t)r2 * (uintptr_t)c.Wc, c.base[2] + (uintptr_t)a0 * (uintptr_t)c.Wc,
        c.base[2] + (uintptr_t)a1 * (uintptr_t)c.Wc, c.base[2] + (uintptr_t)r2 * (uintptr_t)c.Wc};
    typedef __attribute__((address_space(1))) const uint8_t GlobalByte;
    typedef const __attribute__((address_space(1))) u32x4 GlobalChunk;
    const uint32_t lane16 = 16u * (uint32_t)lane;
#pragma unroll
    for (int s = 0; s < 8; ++s) {
        st.sh[s] = (int)(row[s] & 15);
        // byte offset of the lane's chunk: lanes past the segment's last
        // chunk load that chunk again
        const uint32_t last16 =
            repeat ? 0u : (uint32_t)(st.sh[s] + (s < 2 ? c.yspan : c.cspan) - 1) & ~15u;
        GlobalByte *p = (GlobalByte *)(row[s] - (uintptr_t)st.sh[s]);
        // chroma rows are shared by consecutive output rows (a chroma row
        // covers two luma rows): ordinary loads, so the next row's loads of
        // the same rows hit in the caches; luma rows are streamed once
        if (s < 2)
            st.c[s] = __builtin_nontemporal_load((GlobalChunk *)(p + min(lane16, last16)));
        else
            st.c[s] = *(GlobalChunk *)(p + min(lane16, last16));
        if (GL == 2 && s < 2)
            st.c2[s] = __builtin_nontemporal_load((GlobalChunk *)(p + min(1024u + lane16, last16)));
    }
}

template <int GL>
__device__ __forceinline__ void yuv_write(uint8_t *slot, const YuvStaged<GL> &st, int lane)
{
#pragma unroll
    for (int s = 0; s < 8; ++s) {
        ((u32x4 *)(slot + yuv_seg<GL>(s)))[lane] = st.c[s];
        if (GL == 2 && s < 2)
            ((u32x4 *)(slot + yuv_seg<GL>(s)))[64 + lane] = st.c2[s];
    }
}

// Per-lane column taps of the I420 kernel.
template <int J>
struct YuvCols {
    int ox[J][2];        // luma x0 - xf
    float wx[J][2];      // luma weight
    int oc[J][2];            // first chroma column read - cxf
    uint32_t sel[J][2][2];   // per luma column: v_perm selector of its 2 x 2 chroma samples
    uint32_t hw[J][2][2];    // per luma column: horizontal weight bytes (4 - fx, fx)
};

// The column data of pixel px of column iteration j (one column of the lane)
// as 8 words: ox, wx (bits), oc, sel[0], sel[1], hw[0], hw[1], 0.
__device__ __forceinline__ void yuv_col(uint32_t (&w)[8], const YuvImg &g, int Cw, int lane,
                                        int siting, int j, int px)
{
    const int Wc = (g.fw + 1) >> 1;
    const int cxf = chroma_tap(g.rx + g.xf, Wc, siting).x0;
    const int c = min(pair_col(lane, j, Cw) + px, Cw - 1);
    const Tap t = axis_tap(g.left + c, g.W, g.Wr);
    const Tap a0 = chroma_tap(g.rx + t.x0, Wc, siting), a1 = chroma_tap(g.rx + t.x1, Wc, siting);
    w[0] = (uint32_t)(t.x0 - g.xf);
    w[1] = __builtin_bit_cast(uint32_t, t.w);
    w[2] = (uint32_t)(a0.x0 - cxf);
    // the samples of luma column xi are bytes d0, d1 of the 4 read from each
    // chroma row; perm(row b, row a) yields a[d0], a[d1], b[d0], b[d1]
    const Tap ax[2] = {a0, a1};
#pragma unroll
    for (int xi = 0; xi < 2; ++xi) {
        const uint32_t d0 = (uint32_t)(ax[xi].x0 - a0.x0);
        const uint32_t d1 = (uint32_t)(ax[xi].x1 - a0.x0);
        w[3 + xi] = d0 | d1 << 8 | (4 + d0) << 16 | (4 + d1) << 24;
        const uint32_t fx = (uint32_t)(4.0f * ax[xi].w);  // exact: 0 .. 3
        w[5 + xi] = (4 - fx) | fx << 8;
    }
    w[7] = 0;
}

template <int J>
__device__ __forceinline__ void yuv_col_set(YuvCols<J> &k, int j, int px, const uint32_t (&w)[8])
{
    k.ox[j][px] = (int)w[0];
    k.wx[j][px] = __builtin_bit_cast(float, w[1]);
    k.oc[j][px] = (int)w[2];
    k.sel[j][px][0] = w[3];
    k.sel[j][px][1] = w[4];
    k.hw[j][px][0] = w[5];
    k.hw[j][px][1] = w[6];
}

template <int J>
__device__ __forceinline__ void yuv_cols(YuvCols<J> &k, const YuvImg &g, int Cw, int lane,
                                         int siting)
{
#pragma unroll
    for (int j = 0; j < J; ++j)
#pragma unroll
        for (int px = 0; px < 2; ++px) {
            uint32_t w[8];
            yuv_col(w, g, Cw, lane, siting, j, px);
            yuv_col_set<J>(k, j, px, w);
        }
}

// LDS bytes of the column table that the waves of a workgroup share when a
// uniform batch gives them all one geometry: 32 bytes per lane and pixel.
template <int J>
__device__ __host__ constexpr uint32_t yuv_col_table_bytes()
{
    return 2u * J * 64u * 32u;  // the host adds the same to a uniform launch's LDS
}

// yuv_cols for the waves of a workgroup that share one geometry: wave wid
// computes the pixels (j, px) with (2 j + px) % wpg == wid into the table,
// then every wave reads all of them (each pixel's data is the same for every
// wave's lane). The barrier waits for this wave's LDS writes only, not for
// the row loads already in flight.
template <int J>
__device__ __forceinline__ void yuv_cols_shared(YuvCols<J> &k, uint8_t *table, const YuvImg &g,
                                                int Cw, int lane, int siting, int wid, int wpg)
{
#pragma unroll
    for (int t = 0; t < 2 * J; ++t)
        if (t % wpg == wid) {
            uint32_t w[8];
            yuv_col(w, g, Cw, lane, siting, t / 2, t & 1);
            u32x4 *e = (u32x4 *)(table + 32u * (64u * (uint32_t)t + (uint32_t)lane));
            e[0] = u32x4{w[0], w[1], w[2], w[3]};
            e[1] = u32x4{w[4], w[5], w[6], w[7]};
        }
    asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
#pragma unroll
    for (int t = 0; t < 2 * J; ++t) {
        const u32x4 *e = (const u32x4 *)(table + 32u * (64u * (uint32_t)t + (uint32_t)lane));
        const u32x4 lo = e[0], hi = e[1];
        const uint32_t w[8] = {lo.x, lo.y, lo.z, lo.w, hi.x, hi.y, hi.z, hi.w};
        yuv_col_set<J>(k, t / 2, t & 1, w);
    }
}

// Dword-aligned reads of N byte groups (at LDS byte addresses A), realigned:
// bytes A .. A + 3 of each group.
template <int N>
__device__ __forceinline__ void lds_read_quads(const uint32_t (&A)[N], uint32_t (&q)[N]);

#define SMOL_RD2(D, A) "ds_read2_b32 " D ", " A " offset1:1\n\t"
template <>
__device__ __forceinline__ void lds_read_quads<8>(const uint32_t (&A)[8], uint32_t (&q)[8])
{
    uint32_t ad[8];
    u32x2 d[8];
#pragma unroll
    for (int t = 0; t < 8; ++t)
        ad[t] = A[t] & ~3u;
    asm volatile(SMOL_RD2("%0", "%8") SMOL_RD2("%1", "%9") SMOL_RD2("%2", "%10")
                 SMOL_RD2("%3", "%11") SMOL_RD2("%4", "%12") SMOL_RD2("%5", "%13")
                 SMOL_RD2("%6", "%14") SMOL_RD2("%7", "%15") "s_waitcnt lgkmcnt(0)"
                 : "=&v"(d[0]), "=&v"(d[1]), "=&v"(d[2]), "=&v"(d[3]), "=&v"(d[4]),
                   "=&v"(d[5]), "=&v"(d[6]), "=&v"(d[7])
                 : "v"(ad[0]), "v"(ad[1]), "v"(ad[2]), "v"(ad[3]), "v"(ad[4]), "v"(ad[5]),
                   "v"(ad[6]), "v"(ad[7])
                 : "memory");
#pragma unroll
    for (int t = 0; t < 8; ++t)
        q[t] = __builtin_amdgcn_alignbyte(d[t].y, d[t].x, A[t]);
}
#undef SMOL_RD2

// The reads of one output pixel when both luma segments start at one offset
// in their first chunk and all six chroma segments at another (planes whose
// pitches and offsets are multiples of 16 give that on every row). aY: LDS
// byte address of luma column x0 in segment Y y0; aC: of the pixel's first
// chroma column in segment Cb r0. The other segments lie whole KiB further
// (yuv_seg). lum: luma bytes x0, x0 + 1 of row y0, then of row y1 (byte reads,
// zero-extended); q[2 .. 7]: bytes aC .. aC + 3 of Cb r0 .. r2, Cr r0 .. r2,
// from dword reads of two segments at a time (offsets in units of 256 bytes)
// at the aligned address and the next dword, realigned. (Byte reads into
// register halves would save registers, but with ECC-protected registers the
// hardware clears the other half, so each byte gets a register of its own.)
template <int GL>
__device__ __forceinline__ void yuv_read_px(uint32_t aY, uint32_t aC, uint32_t (&lum)[4],
                                            uint32_t (&q)[8])
{
    constexpr int kY1 = (int)(yuv_seg<GL>(1) - yuv_seg<GL>(0));
    static_assert(yuv_seg<GL>(7) - yuv_seg<GL>(2) == 5 * 1024, "chroma segments 1 KiB apart");
    const uint32_t m = aC & ~3u, m4 = m + 4;
    u32x2 d[3], e[3];
    asm volatile("ds_read_u8 %0, %10\n\t"
                 "ds_read_u8 %1, %10 offset:1\n\t"
                 "ds_read_u8 %2, %10 offset:%13\n\t"
                 "ds_read_u8 %3, %10 offset:%14\n\t"
                 "ds_read2st64_b32 %4, %11 offset1:4\n\t"
                 "ds_read2st64_b32 %5, %11 offset0:8 offset1:12\n\t"
                 "ds_read2st64_b32 %6, %11 offset0:16 offset1:20\n\t"
                 "ds_read2st64_b32 %7, %12 offset1:4\n\t"
                 "ds_read2st64_b32 %8, %12 offset0:8 offset1:12\n\t"
                 "ds_read2st64_b32 %9, %12 offset0:16 offset1:20\n\t"
                 "s_waitcnt lgkmcnt(0)"
                 : "=&v"(lum[0]), "=&v"(lum[1]), "=&v"(lum[2]), "=&v"(lum[3]), "=&v"(d[0]),
                   "=&v"(d[1]), "=&v"(d[2]), "=&v"(e[0]), "=&v"(e[1]), "=&v"(e[2])
                 : "v"(aY), "v"(m), "v"(m4), "i"(kY1), "i"(kY1 + 1)
                 : "memory");
#pragma unroll
    for (int t = 0; t < 3; ++t) {
        q[2 + 2 * t] = __builtin_amdgcn_alignbyte(e[t].x, d[t].x, aC);
        q[3 + 2 * t] = __builtin_amdgcn_alignbyte(e[t].y, d[t].y, aC);
    }
}

// s * v for factors below 2^24 as one v_mul_u32_u24 with s in a scalar
// register. (__umul24 of a factor computed in another basic block reaches
// instruction selection as a plain 32-bit multiply, v_mul_lo_u32.) s must be
// the same in every lane.
__device__ __forceinline__ uint32_t mul_u24_sv(uint32_t s, uint32_t v)
{
    uint32_t r;
    asm("v_mul_u32_u24 %0, %1, %2" : "=v"(r) : "s"(s), "v"(v));
    return r;
}

// 16 * (chroma - 128) at one luma tap: the tap's four chroma samples
// (selected from chroma rows ra and rb) dotted with its weight bytes, minus
// 2048, exact in integers. The sum, in [-2048, 2032], is accumulated onto the
// bit pattern of 1.5 * 2^23, where consecutive floats are 1 apart, so the
// result reads as the float 1.5 * 2^23 + (S - 2048); subtracting 1.5 * 2^23
// is exact. (One fp32 subtraction instead of an integer conversion, which
// issues at half the rate.)
__device__ __forceinline__ float chroma16(uint32_t ra, uint32_t rb, uint32_t sel, uint32_t wts)
{
    const uint32_t smp = __builtin_amdgcn_perm(rb, ra, sel);
    return __uint_as_float(__builtin_amdgcn_udot4(smp, wts, 0x4B400000u - 2048u, false)) -
           12582912.0f;
}

// One output row from the staged segments. SAME: every luma segment of the
// row starts at offset sh[0] in its first chunk and every chroma segment at
// sh[2] (the reads of yuv_read_px); otherwise each segment is addressed on
// its own.
template <int F16, int J, int EXACT, int GL, int SAME>
__device__ __forceinline__ void yuv_compute(const NormK &nk, uint32_t slot, const int (&sh)[8],
                                            float wy, int fy0, int fy1, const YuvCols<J> &k,
                                            RowOut<F16, J> &out)
{
    // weight bytes of luma row yi and column xi: hw(xi) * (4 + 65535 fy(yi))
    // = (4 - fy) * [4 - fx, fx, 0, 0] + fy * [0, 0, 4 - fx, fx] (no carries)
    const uint32_t vm[2] = {
        (uint32_t)__builtin_amdgcn_readfirstlane((int)(4u + 65535u * (uint32_t)fy0)),
        (uint32_t)__builtin_amdgcn_readfirstlane((int)(4u + 65535u * (uint32_t)fy1))};
    const uint32_t baseY = slot + yuv_seg<GL>(0) + (uint32_t)sh[0];
    const uint32_t baseC = slot + yuv_seg<GL>(2) + (uint32_t)sh[2];
#pragma unroll
    for (int j = 0; j < J; ++j) {
        float o[3][2];
#pragma unroll
        for (int px = 0; px < 2; ++px) {
            // reads: Y y0, Y y1, Cb r0..r2, Cr r0..r2
            uint32_t q[8], lum[4];
            if (SAME) {
                yuv_read_px<GL>(baseY + (uint32_t)k.ox[j][px], baseC + (uint32_t)k.oc[j][px], lum,
                                q);
            } else {
                uint32_t A[8];
#pragma unroll
                for (int s = 0; s < 8; ++s)
                    A[s] = slot + yuv_seg<GL>(s) + (uint32_t)sh[s] +
                           (uint32_t)(s < 2 ? k.ox[j][px] : k.oc[j][px]);
                lds_read_quads<8>(A, q);
            }
            // 16 * (chroma - 128) at (y0, y1) x (x0, x1) for both planes:
            // luma row y0 reads chroma rows r0, r1 and y1 reads r1, r2
            float cc[2][2][2];  // [plane][luma row][luma col]
#pragma unroll
            for (int pl = 0; pl < 2; ++pl) {
                const uint32_t r0 = q[2 + 3 * pl], r1 = q[3 + 3 * pl], r2 = q[4 + 3 * pl];
#pragma unroll
                for (int xi = 0; xi < 2; ++xi) {
                    cc[pl][0][xi] = chroma16(r0, r1, k.sel[j][px][xi], mul_u24_sv(vm[0], k.hw[j][px][xi]));
                    cc[pl][1][xi] = chroma16(r1, r2, k.sel[j][px][xi], mul_u24_sv(vm[1], k.hw[j][px][xi]));
                }
            }
            float rgb[2][2][3];  // [luma row][luma col][channel]
#pragma unroll
            for (int yi = 0; yi < 2; ++yi)
#pragma unroll
                for (int xi = 0; xi < 2; ++xi) {
                    const float Y = SAME ? cvt_ubyte0(lum[2 * yi + xi])
                                         : xi ? cvt_ubyte1(q[yi]) : cvt_ubyte0(q[yi]);
                    ycbcr16_to_rgb(Y, cc[0][yi][xi], cc[1][yi][xi], rgb[yi][xi][0],
                                   rgb[yi][xi][1], rgb[yi][xi][2]);
                }
#pragma unroll
            for (int ch = 0; ch < 3; ++ch)
                o[ch][px] = normalize_k<EXACT>(
                    nk, ch,
                    lerp(lerp(rgb[0][0][ch], rgb[0][1][ch], k.wx[j][px]),
                         lerp(rgb[1][0][ch], rgb[1][1][ch], k.wx[j][px]), wy));
        }
        pack_pair<F16, EXACT, J>(out, j, o);
    }
}

// Whether every luma segment of a row starts at one offset in its first
// chunk and every chroma segment at another.
__device__ __forceinline__ bool yuv_same_offsets(const int (&sh)[8])
{
    return sh[1] == sh[0] && sh[3] == sh[2] && sh[4] == sh[2] && sh[5] == sh[2] &&
           sh[6] == sh[2] && sh[7] == sh[2];
}

template <int F16, int J, int EXACT, int GL>
__device__ __forceinline__ void yuv_compute_row(const NormK &nk, uint32_t slot, const int (&sh)[8],
                                                float wy, int fy0, int fy1, const YuvCols<J> &k,
                                                RowOut<F16, J> &out)
{
    if (yuv_same_offsets(sh))
        yuv_compute<F16, J, EXACT, GL, 1>(nk, slot, sh, wy, fy0, fy1, k, out);
    else
        yuv_compute<F16, J, EXACT, GL, 0>(nk, slot, sh, wy, fy0, fy1, k, out);
}

// FORM as for rgb_rows_kernel; GL: chunks per lane of a luma segment (staged
// luma rows of up to 1 or 2 KiB).
template <int F16, int J, int EXACT, int STRIDE, int FORM, int GL>
__global__ void __launch_bounds__(64 * kRowsMaxWavesPerGroup) __attribute__((amdgpu_waves_per_eu(J <= 2 ? 3 : 1)))
yuv_rows_kernel(BatchArgs a)
{
    constexpr int NHWC = FORM & kFormNhwc, ODD = (FORM & kFormOdd) ? 1 : 0;
    extern __shared__ __attribute__((aligned(16))) uint8_t lds_all[];
    int lane;
    long long r0;
    int n_rows;
    const int Ch = a.Ch;
    uint8_t *const lds = rows_wave<STRIDE>(lds_all, yuv_seg<GL>(8), a, lane, r0, n_rows);
    // The host launches at most one wave per row, so every wave has rows (an
    // early exit here would hold the remaining argument loads behind it).
    __builtin_assume(n_rows > 0);
    const RowStep step = row_step_of<STRIDE>(a);
    constexpr int kEsz = F16 == 2 ? 1 : F16 ? 2 : 4;
    int c_img, c_rr;  // row to interpolate
    split_row<STRIDE>(r0, Ch, c_img, c_rr);
    YuvCursor lc;  // next row to load
    yuv_cursor_image<STRIDE>(lc, a, c_img, c_rr, step);

    // One register set: row k + 1 is loaded before row k is interpolated.
    // The loop runs the n_rows - 1 steps that stage a next row and leaves
    // only at its end; the last row is interpolated after it. The first row
    // is requested before the column taps and the rest of the set-up are
    // computed.
    int lrow = 0;
    auto advance = [&]() {
        if (lrow + 1 < n_rows) {
            yuv_cursor_next<STRIDE>(lc, a, step);
            ++lrow;
        }
    };
    YuvStaged<GL> R;
    yuv_load<GL>(R, lc, lane, false);
    advance();
    // bytes between an image's output rows: Cw elements per plane (NCHW) or
    // 3 Cw (NHWC); a wrap to the next image skips the rest of the image.
    const long long rb = (long long)a.Cw * kEsz, rowb = NHWC ? 3 * rb : rb;
    const long long imgb = 3LL * Ch * rb;
    uint8_t *orow = (uint8_t *)a.out + (long long)(a.img_base + c_img) * imgb + c_rr * rowb;
    const long long ostep = step.di * imgb + step.dr * rowb, owrap = imgb - Ch * rowb;

    YuvCols<J> cols;
    int cW, cWr, cleft;
    {
        const YuvImg g = yuv_img(a, c_img);
        if (!a.table && a.wpg > 1)
            yuv_cols_shared<J>(cols, lds_all + a.wpg * yuv_seg<GL>(8), g, a.Cw, lane, a.siting,
                               __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6)), a.wpg);
        else
            yuv_cols<J>(cols, g, a.Cw, lane, a.siting);
        cW = g.W;
        cWr = g.Wr;
        cleft = g.left;
    }
    const NormK nk = norm_consts(a);
    const uint32_t lds0 = lds_addr(lds);

    const long long plane = (long long)Ch * a.Cw * kEsz;
    RowOut<F16, J> out;
    yuv_write<GL>(lds, R, lane);
    int csh[8];
#pragma unroll
    for (int s = 0; s < 8; ++s)
        csh[s] = R.sh[s];
    float cwy = R.wy;
    int cfy0 = R.fy0, cfy1 = R.fy1;
    for (int left = n_rows - 1; left > 0; --left) {
        yuv_load<GL>(R, lc, lane, false);
        advance();
        yuv_compute_row<F16, J, EXACT, GL>(nk, lds0, csh, cwy, cfy0, cfy1, cols, out);
        yuv_write<GL>(lds, R, lane);
        store_row<F16, J, ODD>(orow, plane, a.Cw, lane, out, NHWC);
#pragma unroll
        for (int s = 0; s < 8; ++s)
            csh[s] = R.sh[s];
        cwy = R.wy;
        cfy0 = R.fy0;
        cfy1 = R.fy1;
        const int pimg = c_img;
        c_img += step.di;
        c_rr += step.dr;
        orow += ostep;
        if (c_rr >= Ch) {
            c_rr -= Ch;
            ++c_img;
            orow += owrap;
        }
        if (c_img != pimg) {
            const YuvImg g = yuv_img(a, c_img);
            if (g.W != cW || g.Wr != cWr || g.left != cleft) {
                cW = g.W;
                cWr = g.Wr;
                cleft = g.left;
                yuv_cols<J>(cols, g, a.Cw, lane, a.siting);
            }
        }
    }
    yuv_compute_row<F16, J, EXACT, GL>(nk, lds0, csh, cwy, cfy0, cfy1, cols, out);
    store_row<F16, J, ODD>(orow, plane, a.Cw, lane, out, NHWC);
}


template <int F16, int EXACT, int STRIDE, int FORM, int GL>
const void *yuv_rows_g(int col_iters)
{
    return col_iters <= 1   ? (const void *)yuv_rows_kernel<F16, 1, EXACT, STRIDE, FORM, GL>
           : col_iters <= 2 ? (const void *)yuv_rows_kernel<F16, 2, EXACT, STRIDE, FORM, GL>
                            : (const void *)yuv_rows_kernel<F16, 4, EXACT, STRIDE, FORM, GL>;
}

// a.row_groups: KiB per staged luma row, 1 or 2
template <int F16, int EXACT, int STRIDE, int FORM>
const void *yuv_rows_e(const BatchArgs &a)
{
    return a.row_groups >= 2 ? yuv_rows_g<F16, EXACT, STRIDE, FORM, 2>(a.col_iters)
                             : yuv_rows_g<F16, EXACT, STRIDE, FORM, 1>(a.col_iters);
}

template <int F16, int EXACT, int STRIDE, int NHWC>
const void *yuv_rows_f(const BatchArgs &a)
{
    return (a.Cw & 1) ? yuv_rows_e<F16, EXACT, STRIDE, NHWC | kFormOdd>(a)
                      : yuv_rows_e<F16, EXACT, STRIDE, NHWC>(a);
}

template <int STRIDE, int NHWC>
const void *yuv_rows_table(const BatchArgs &a, int f16)
{
    return f16 ? (a.exact ? yuv_rows_f<1, 1, STRIDE, NHWC>(a) : yuv_rows_f<1, 0, STRIDE, NHWC>(a))
               : (a.exact ? yuv_rows_f<0, 1, STRIDE, NHWC>(a) : yuv_rows_f<0, 0, STRIDE, NHWC>(a));
}

}  // namespace
}  // namespace smol
