// smol_rows.h -- the pieces the row-streaming kernels (RGB in smol_rows_rgb.h,
// I420 in smol_rows_yuv.h) share: the row walk over waves, the vertical tap
// cursor, row staging and tap reads for RGB rows, normalisation, output
// packing and stores. Each smol_rows_*.hip file instantiates one part of the
// kernels (input, output type, row walk, output layout), so the parts build
// in parallel.
#pragma once

#include <limits.h>

#include "smol_device.h"

namespace smol {
namespace {

// ---------------------------------------------------------------------------
// RGB, row streaming: one wave per workgroup, no barriers.
//
// Work items are output rows (image, row), image-major. With STRIDE = 0 wave
// g takes the contiguous range [g*T/G, (g+1)*T/G) of the T rows; with
// STRIDE = 1 it takes rows q, q + G, q + 2G, ... (q: g remapped so the waves
// of one XCD take neighbouring rows), so the rows in flight on the chip at
// any moment form one band of the output. For each output row the
// wave loads the two source rows its vertical taps read -- only the crop's
// source column span, as the 16-byte chunks that hold it, aligned in the
// global address space, one coalesced 16-byte load per lane and 64 chunks --
// into registers, two rows ahead of the row it interpolates (three register
// sets in rotation), and writes a row's chunks into its LDS slot right after
// interpolating the previous row. The bytes in flight live in registers, so a
// compute unit keeps more loads outstanding than its LDS could stage, and
// the compiler orders each LDS write after exactly the loads it needs.
//
// Only images whose chunks all lie inside src come here; the host sends the
// others to the direct kernel. Lanes past a row's last chunk load that chunk
// again (their copy lands past the row in the slot and is never read).
//
// A cursor steps the vertical half-pixel map incrementally with exact integer
// arithmetic (the numerator grows by 2*H per output row, or by a precomputed
// constant per strided step): no division per row but the one for the
// weight.
//
// Lane l computes output columns c = 2l + 128j and c + 1 (j < J); their taps
// (byte offset in the staged span, weight) stay in registers while the
// horizontal geometry is unchanged. Each pixel's two horizontal taps are 6
// bytes of a staged row, read as three aligned dwords and realigned.
//
// The three lerps are always evaluated as defined, every product and sum
// rounded on its own. EXACT selects the rest: 1 forms the normalisation as
// the correctly rounded quotient and rounds to fp16 from that fp32 value,
// bit-identical to a scalar fp32 evaluation of the definition; 0 multiplies
// the same difference v - mean by RN(1/std), at most one fp32 ulp from the
// quotient, and lets the fp16 conversion fuse with that product (fp16 output
// within one fp16 ulp of the definition's).
// ---------------------------------------------------------------------------
struct RowImg {
    long long off;
    int W, H, pitch, Wr, Hr, left, top, xf, span;
};

// The descriptor table is read-only for the whole launch: read it through the
// constant address space so the wave uses scalar loads, which do not count
// against (or wait for) the vector-memory counter.
typedef __attribute__((address_space(4))) const Desc ConstDesc;

__device__ __forceinline__ RowImg row_img(const BatchArgs &a, int img)
{
    RowImg g;
    if (a.table) {
        const ConstDesc *t = (const ConstDesc *)a.table + img;
        g.off = t->off[0];
        g.W = t->W;
        g.H = t->H;
        g.pitch = t->pitch;
        g.Wr = t->Wr;
        g.Hr = t->Hr;
        g.left = t->left;
        g.top = t->top;
        g.xf = t->xf;
        g.span = t->span;
    } else {
        g.off = a.uni.off[0] + (long long)img * a.stride;
        g.W = a.uni.W;
        g.H = a.uni.H;
        g.pitch = a.uni.pitch;
        g.Wr = a.uni.Wr;
        g.Hr = a.uni.Hr;
        g.left = a.uni.left;
        g.top = a.uni.top;
        g.xf = a.uni.xf;
        g.span = a.uni.span;
            }
    return g;
}

// First output column of the pair lane `lane` computes in column iteration
// j: 2 * lane + 128 * j, clamped to the last pair (Cw - 2 for even Cw, the
// last column for odd Cw). Lanes past the crop thus compute and store a
// copy of the last pair, the same values to the same addresses: every lane
// runs the same stores, with no branch around them, and the compiler can
// count the memory operations in flight exactly (a branch that might skip
// the stores would make it wait for them before every write to LDS).
__device__ __forceinline__ int pair_col(int lane, int j, int Cw)
{
    return min(2 * lane + 128 * j, Cw - 2 + (Cw & 1));
}

template <int J>
__device__ __forceinline__ void row_taps(const RowImg &g, const int Cw, int (&cx)[J][2],
                                         float (&cw)[J][2], int lane)
{
#pragma unroll
    for (int j = 0; j < J; ++j)
#pragma unroll
        for (int px = 0; px < 2; ++px) {
            const int col = min(pair_col(lane, j, Cw) + px, Cw - 1);
            const Tap t = axis_tap(g.left + col, g.W, g.Wr);
            cx[j][px] = 3 * (t.x0 - g.xf);
            cw[j][px] = t.w;
        }
}

// Pixels x0 (bytes 0..2) and x0 + 1 (bytes 3..5) of an 8-byte window, as
// a = value at x0 and d = (value at x0 + 1) - a per channel; d is an exact
// small integer, so a + w * d is the definition's a + w * (b - a).
#define SMOL_CVT_UBYTE(N)                                                                     \
    __device__ __forceinline__ float cvt_ubyte##N(uint32_t x)                                 \
    {                                                                                         \
        float f;                                                                              \
        asm("v_cvt_f32_ubyte" #N " %0, %1" : "=v"(f) : "v"(x));                               \
        return f;                                                                             \
    }
SMOL_CVT_UBYTE(0)
SMOL_CVT_UBYTE(1)
SMOL_CVT_UBYTE(2)
SMOL_CVT_UBYTE(3)
#undef SMOL_CVT_UBYTE

__device__ __forceinline__ void unpack_ad(uint64_t v, float (&a)[3], float (&d)[3])
{
    // One conversion per byte (the compiler's own selection extracts some
    // bytes with extra shifts first).
    const uint32_t lo = (uint32_t)v, hi = (uint32_t)(v >> 32);
    a[0] = cvt_ubyte0(lo);
    a[1] = cvt_ubyte1(lo);
    a[2] = cvt_ubyte2(lo);
    d[0] = cvt_ubyte3(lo) - a[0];  // exact: small integers
    d[1] = cvt_ubyte0(hi) - a[1];
    d[2] = cvt_ubyte1(hi) - a[2];
}

// a + w * d with the product and the sum rounded on their own.
__device__ __forceinline__ float lerp_ad(float a, float d, float w) { return a + w * d; }

// Normalisation constants of the three channels.
struct NormK {
    float mean[3], stdv[3], rcp[3];
};

__device__ __forceinline__ NormK norm_consts(const BatchArgs &a)
{
    NormK k;
#pragma unroll
    for (int ch = 0; ch < 3; ++ch) {
        k.mean[ch] = a.mean[ch];
        k.stdv[ch] = a.stdv[ch];
        k.rcp[ch] = a.rcp[ch];
    }
    return k;
}

// (v - mean) / std: the correctly rounded quotient (EXACT), or the product
// of the same difference with RN(1/std), which is within one fp32 ulp of it.
template <int EXACT>
__device__ __forceinline__ float normalize_k(const NormK &k, int ch, float v)
{
    return EXACT ? normalize(v, k.mean[ch], k.stdv[ch], k.rcp[ch]) : (v - k.mean[ch]) * k.rcp[ch];
}

// The value an output element holds: normalised (fp32 / fp16 output, OUT 0 /
// 1), or the resized value itself (uint8 output, OUT 2; rounded when packed).
template <int OUT, int EXACT>
__device__ __forceinline__ float out_value(const NormK &k, int ch, float v)
{
    return OUT == 2 ? v : normalize_k<EXACT>(k, ch, v);
}


typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// One output row's two source rows in registers (G chunk loads each), with
// the offset of each row's first byte in its first chunk and the vertical
// weight.
template <int G>
struct StagedRows {
    u32x4 c0[G], c1[G];
    int sh0, sh1;
    float wy;
    int y0, y1;  // the source rows
};

// The rows a wave walks: batch rows r0, r0 + d, r0 + 2d, ... as (image, crop
// row) pairs, which advance by (d / Ch, d % Ch) per step. STRIDE = 0: d = 1,
// a wave takes a contiguous range of rows. STRIDE = 1: d = the number of
// waves G, wave q takes rows q, q + G, ..., so at any moment the waves work
// on a band of consecutive output rows, close together in memory.
struct RowStep {
    int di, dr, Ch;
};

template <int STRIDE>
__device__ __forceinline__ RowStep row_step_of(const BatchArgs &a)
{
    return STRIDE ? RowStep{a.step_di, a.step_dr, a.Ch} : RowStep{0, 1, a.Ch};
}

// First row and row count of wave `w`: the host splits the n * Ch rows as
// rows_q * grid + rows_r, so every wave walks rows_q rows and waves
// w < rows_r one more. STRIDE = 1: wave w starts at row w; STRIDE = 0: at the
// end of the ranges of waves 0 .. w - 1.
template <int STRIDE>
__device__ __forceinline__ void wave_rows(const BatchArgs &a, int w, long long &r0, int &n_rows)
{
    n_rows = a.rows_q + (w < a.rows_r ? 1 : 0);
    r0 = STRIDE ? (long long)w : (long long)w * a.rows_q + min(w, a.rows_r);
}

// Image and crop row of batch row r (r < 2^31 in a strided walk, where it is
// a wave index).
template <int STRIDE>
__device__ __forceinline__ void split_row(long long r, int Ch, int &img, int &rr)
{
    if (STRIDE) {
        img = (int)((unsigned)r / (unsigned)Ch);
        rr = (int)r - img * Ch;
    } else {
        img = (int)(r / Ch);
        rr = (int)(r - (long long)img * Ch);
    }
}

// Workgroups are dealt to the 8 XCDs round-robin; remap so the waves of one
// XCD take consecutive rows (neighbouring output rows share source rows when
// the vertical scale is below 2, and share the XCD's L2).
__device__ __forceinline__ int xcd_position(int g, int G)
{
    return G % 8 == 0 ? (g % 8) * (G / 8) + g / 8 : g;
}

// A workgroup holds a.wpg independent waves (no barriers), each with its own
// LDS slot of `slot_bytes`; several waves per workgroup cut the cost of
// dispatching the grid. Returns the wave's slot and sets its lane and rows.
// (The wave count comes from the arguments: blockDim would be a memory read
// that every wave waits for before its first address is known.)
template <int STRIDE>
__device__ __forceinline__ uint8_t *rows_wave(uint8_t *lds_all, int slot_bytes, const BatchArgs &a,
                                              int &lane, long long &r0, int &n_rows)
{
    const int wpg = a.wpg;
    const int wid = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
    lane = (int)(threadIdx.x & 63);
    const int g = STRIDE ? xcd_position((int)blockIdx.x, (int)gridDim.x) : (int)blockIdx.x;
    wave_rows<STRIDE>(a, g * wpg + wid, r0, n_rows);
    return lds_all + wid * slot_bytes;
}

// floor(n / d) and n - d floor(n / d) for d > 0: one truncating division (a
// 32-bit one when n fits), then the correction for negative n.
__device__ __forceinline__ void floor_divmod(long long n, int d, int &q, int &r)
{
    long long qq = (n >= INT_MIN && n <= INT_MAX) ? (long long)((int)n / d) : n / d;
    long long rr = n - qq * d;
    if (rr < 0) {
        --qq;
        rr += d;
    }
    q = (int)qq;
    r = (int)rr;
}

// Vertical half-pixel taps along a walk over rows of one geometry:
// num(rr) = (2 * (top + rr) + 1) * H - Hr, den = 2 * Hr, q = floor(num / den),
// rem = num - q * den. A step moves rr by dr, or by dr - Ch when it wraps to
// the next image of the same geometry, so num by one of two constants whose
// floor quotients and remainders are precomputed: exact integer arithmetic,
// no division per row. (num <= 0 exactly when q < 0 or q == rem == 0.)
struct VCursor {
    int q, rem, den, H;
    int qs, rs;    // step within an image
    int qw, rw;    // step that wraps (strided walks of a uniform batch)
};

template <int STRIDE>
__device__ __forceinline__ void vcursor_init(VCursor &v, const BatchArgs &a, const RowImg &g, int rr,
                                             const RowStep &s)
{
    const int den = 2 * g.Hr;
    int q, rem, qs, rs, qw = 0, rw = 0;
    floor_divmod((long long)(2 * (g.top + rr) + 1) * g.H - g.Hr, den, q, rem);
    if (STRIDE && !a.table) {
        // one geometry for the whole launch: the host computed the steps
        qs = a.vq_s;
        rs = a.vr_s;
        qw = a.vq_w;
        rw = a.vr_w;
    } else if (STRIDE) {
        // a walk over a table reads the next image's descriptor on a wrap
        floor_divmod(2LL * g.H * s.dr, den, qs, rs);
    } else {
        qs = (2 * g.H) / den;
        rs = 2 * g.H - qs * den;
    }
    // (every field stored on every path: stores that differ by branch can be
    // merged into one store to a chosen field, which keeps the cursor in
    // memory)
    v = VCursor{q, rem, den, g.H, qs, rs, qw, rw};
}

__device__ __forceinline__ void vcursor_add(VCursor &v, int dq, int dr)
{
    v.q += dq;
    v.rem += dr;
    if (v.rem >= v.den) {
        v.rem -= v.den;
        ++v.q;
    }
}

__device__ __forceinline__ void vcursor_tap(const VCursor &v, int &y0, int &y1, float &w)
{
    if (v.q < 0 || (v.q == 0 && v.rem == 0)) {
        y0 = y1 = 0;
        w = 0.0f;
    } else if (v.q >= v.H - 1) {
        y0 = y1 = v.H - 1;
        w = 0.0f;
    } else {
        y0 = v.q;
        y1 = y0 + 1;
        w = (float)v.rem / (float)v.den;  // IEEE division, both operands exact
    }
}

// Load cursor: image, crop row, vertical map and the image's row addressing.
struct RowCursor {
    int img, rr;
    VCursor v;
    uintptr_t base;  // first staged byte of source row 0
    int pitch, span;
};

template <int STRIDE>
__device__ __forceinline__ void cursor_image(RowCursor &c, const BatchArgs &a, int img, int rr,
                                             const RowStep &s)
{
    const RowImg g = row_img(a, img);
    c.img = img;
    c.rr = rr;
    vcursor_init<STRIDE>(c.v, a, g, rr, s);
    c.base = (uintptr_t)(a.src + g.off) + 3 * (uintptr_t)g.xf;
    c.pitch = g.pitch;
    c.span = g.span;
}

// Next row of the walk. A strided walk over a uniform batch (one geometry,
// images `stride` bytes apart) moves the base address and steps the vertical
// map; over a table it reads the new image's descriptor when the image
// changes.
template <int STRIDE>
__device__ __forceinline__ void cursor_next(RowCursor &c, const BatchArgs &a, const RowStep &s)
{
    if (!STRIDE) {
        vcursor_add(c.v, c.v.qs, c.v.rs);
        if (++c.rr == s.Ch && c.img + 1 < a.n)
            cursor_image<0>(c, a, c.img + 1, 0, s);
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
        c.base += (uintptr_t)(c.img - img0) * (uintptr_t)a.stride;
        vcursor_add(c.v, wrapped ? c.v.qw : c.v.qs, wrapped ? c.v.rw : c.v.rs);
    } else if (c.img != img0) {
        cursor_image<1>(c, a, c.img, c.rr, s);
    } else {
        vcursor_add(c.v, c.v.qs, c.v.rs);
    }
}

// `repeat`: the row was loaded already (past the end of the wave's range);
// every lane then loads the rows' first chunk, so the instruction stream is
// unchanged but almost nothing is fetched.
// NT: nontemporal loads, for walks that read each source row once (the
// strided walk of large frames); a contiguous walk meets a source row again
// when consecutive output rows share it (upscales, downscales by less than
// 2, and the rows of an image's neighbours in the walk), and ordinary loads
// let those reads hit in the caches.
template <int G, int NT = 1>
__device__ __forceinline__ void load_rows(StagedRows<G> &st, const RowCursor &c, int lane,
                                          bool repeat)
{
    int y0, y1;
    vcursor_tap(c.v, y0, y1, st.wy);
    st.y0 = y0;
    st.y1 = y1;
    const uintptr_t r0 = c.base + (uintptr_t)y0 * (uintptr_t)c.pitch;
    const uintptr_t r1 = c.base + (uintptr_t)y1 * (uintptr_t)c.pitch;
    st.sh0 = (int)(r0 & 15);
    st.sh1 = (int)(r1 & 15);
    const int last0 = repeat ? 0 : (st.sh0 + c.span - 1) >> 4;
    const int last1 = repeat ? 0 : (st.sh1 + c.span - 1) >> 4;
    // global address space: a generic (flat) load would also count against
    // the LDS counter and make every LDS access wait for it
    // (a uniform base and a 32-bit lane offset: the loads take the base from
    // scalar registers)
    typedef __attribute__((address_space(1))) const uint8_t GlobalByte;
    GlobalByte *p0 = (GlobalByte *)(r0 - (uintptr_t)st.sh0);
    GlobalByte *p1 = (GlobalByte *)(r1 - (uintptr_t)st.sh1);
#pragma unroll
    for (int g = 0; g < G; ++g) {
        const uint32_t o0 = 16u * (uint32_t)min(64 * g + lane, last0);
        const uint32_t o1 = 16u * (uint32_t)min(64 * g + lane, last1);
        typedef const __attribute__((address_space(1))) u32x4 GlobalChunk;
        if (NT) {
            st.c0[g] = __builtin_nontemporal_load((GlobalChunk *)(p0 + o0));
            st.c1[g] = __builtin_nontemporal_load((GlobalChunk *)(p1 + o1));
        } else {
            st.c0[g] = *(GlobalChunk *)(p0 + o0);
            st.c1[g] = *(GlobalChunk *)(p1 + o1);
        }
    }
}

template <int G>
__device__ __forceinline__ void write_rows(uint8_t *slot, const StagedRows<G> &st, int lane)
{
#pragma unroll
    for (int g = 0; g < G; ++g) {
        ((u32x4 *)slot)[64 * g + lane] = st.c0[g];
        ((u32x4 *)(slot + 1024 * G))[64 * g + lane] = st.c1[g];
    }
}

// LDS byte address of a pointer into the dynamic LDS array.
__device__ __forceinline__ uint32_t lds_addr(const uint8_t *p)
{
    return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) uint8_t *)p;
}

// Tap pairs (6 bytes at LDS byte address A) are read as the three dwords at
// A & ~3 and realigned with v_alignbyte, which takes its shift from the low
// bits of A (an unaligned LDS access is split lane by lane). The reads of a
// row's tap pairs are issued together from inline assembly, then waited for
// once: the compiler would wait after every pixel.
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

#define SMOL_RD3(D2, D1, A) "ds_read2_b32 " D2 ", " A " offset1:1\n\tds_read_b32 " D1 ", " A " offset:8\n\t"
__device__ __forceinline__ void lds_read_taps4(const uint32_t (&ad)[4], u32x2 (&lo)[4],
                                               uint32_t (&hi)[4])
{
    asm volatile(SMOL_RD3("%0", "%4", "%8") SMOL_RD3("%1", "%5", "%9") SMOL_RD3("%2", "%6", "%10")
                 SMOL_RD3("%3", "%7", "%11") "s_waitcnt lgkmcnt(0)"
                 : "=&v"(lo[0]), "=&v"(lo[1]), "=&v"(lo[2]), "=&v"(lo[3]), "=&v"(hi[0]),
                   "=&v"(hi[1]), "=&v"(hi[2]), "=&v"(hi[3])
                 : "v"(ad[0]), "v"(ad[1]), "v"(ad[2]), "v"(ad[3])
                 : "memory");
}
__device__ __forceinline__ void lds_read_taps8(const uint32_t (&ad)[8], u32x2 (&lo)[8],
                                               uint32_t (&hi)[8])
{
    asm volatile(SMOL_RD3("%0", "%8", "%16") SMOL_RD3("%1", "%9", "%17")
                 SMOL_RD3("%2", "%10", "%18") SMOL_RD3("%3", "%11", "%19")
                 SMOL_RD3("%4", "%12", "%20") SMOL_RD3("%5", "%13", "%21")
                 SMOL_RD3("%6", "%14", "%22") SMOL_RD3("%7", "%15", "%23")
                 "s_waitcnt lgkmcnt(0)"
                 : "=&v"(lo[0]), "=&v"(lo[1]), "=&v"(lo[2]), "=&v"(lo[3]), "=&v"(lo[4]),
                   "=&v"(lo[5]), "=&v"(lo[6]), "=&v"(lo[7]), "=&v"(hi[0]), "=&v"(hi[1]),
                   "=&v"(hi[2]), "=&v"(hi[3]), "=&v"(hi[4]), "=&v"(hi[5]), "=&v"(hi[6]),
                   "=&v"(hi[7])
                 : "v"(ad[0]), "v"(ad[1]), "v"(ad[2]), "v"(ad[3]), "v"(ad[4]), "v"(ad[5]),
                   "v"(ad[6]), "v"(ad[7])
                 : "memory");
}
__device__ __forceinline__ void lds_read_taps2(const uint32_t (&ad)[2], u32x2 (&lo)[2],
                                               uint32_t (&hi)[2])
{
    asm volatile(SMOL_RD3("%0", "%2", "%4") SMOL_RD3("%1", "%3", "%5") "s_waitcnt lgkmcnt(0)"
                 : "=&v"(lo[0]), "=&v"(lo[1]), "=&v"(hi[0]), "=&v"(hi[1])
                 : "v"(ad[0]), "v"(ad[1])
                 : "memory");
}
#undef SMOL_RD3

// The 2J tap pairs of one staged row (pixel c and c + 1 of every column
// iteration), realigned to 8-byte values: tap 2j + px.
template <int J>
__device__ __forceinline__ void read_row_taps(uint32_t row, const int (&cx)[J][2],
                                              uint64_t (&v)[2 * J])
{
    constexpr int N = 2 * J;
    uint32_t A[N], ad[N], hi[N];
    u32x2 lo[N];
#pragma unroll
    for (int t = 0; t < N; ++t) {
        A[t] = row + (uint32_t)cx[t / 2][t & 1];
        ad[t] = A[t] & ~3u;
    }
    if constexpr (N == 8)
        lds_read_taps8(ad, lo, hi);
    else if constexpr (N == 4)
        lds_read_taps4(ad, lo, hi);
    else
        lds_read_taps2(ad, lo, hi);
#pragma unroll
    for (int t = 0; t < N; ++t)
        v[t] = (uint64_t)__builtin_amdgcn_alignbyte(lo[t].y, lo[t].x, A[t]) |
               ((uint64_t)__builtin_amdgcn_alignbyte(hi[t], lo[t].y, A[t]) << 32);
}

// The tap pairs of column iterations j0 .. j0 + N/4 - 1 (pixel c, c + 1 of
// rows 0 and 1 each), realigned to 8-byte values.
template <int J, int N>
__device__ __forceinline__ void read_taps(uint32_t row0, uint32_t row1, const int (&cx)[J][2],
                                          int j0, uint64_t (&v)[N])
{
    uint32_t A[N], ad[N], hi[N];
    u32x2 lo[N];
#pragma unroll
    for (int t = 0; t < N; ++t) {
        const int j = j0 + t / 4, px = t & 1;
        A[t] = ((t & 2) ? row1 : row0) + (uint32_t)cx[j][px];
        ad[t] = A[t] & ~3u;
    }
    if constexpr (N == 8)
        lds_read_taps8(ad, lo, hi);
    else
        lds_read_taps4(*(const uint32_t(*)[4])ad, *(u32x2(*)[4])lo, *(uint32_t(*)[4])hi);
#pragma unroll
    for (int t = 0; t < N; ++t)
        v[t] = (uint64_t)__builtin_amdgcn_alignbyte(lo[t].y, lo[t].x, A[t]) |
               ((uint64_t)__builtin_amdgcn_alignbyte(hi[t], lo[t].y, A[t]) << 32);
}

// One output row's values of a lane, ready to store: per column iteration
// and channel the pair (c, c + 1) as one dword (fp16) or two (fp32).
//
// A row's stores are issued after the next row's chunks are written to LDS,
// not before: the wait for those chunks' loads then never includes the
// completion of this row's stores (the compiler cannot count stores among
// the loads they may overtake, so a wait for a load issued before a store
// lasts until the store is done as well).
// Output form of a row-streaming kernel instance (its FORM template
// parameter): NHWC layout, odd crop width.
constexpr int kFormNhwc = 1;
constexpr int kFormOdd = 2;

// A lane's output pairs of one row: per column pair and channel two fp32
// words (F16 0), one word of two fp16 (F16 1) or the low half-word of one
// word holding two uint8 (F16 2, uint8 output).
template <int F16, int J>
struct RowOut {
    uint32_t w[J][3][F16 ? 1 : 2];
};

template <int F16, int EXACT, int J>
__device__ __forceinline__ void pack_pair(RowOut<F16, J> &out, int j, const float (&o)[3][2])
{
#pragma unroll
    for (int ch = 0; ch < 3; ++ch) {
        if (F16 == 2) {
            // clamped to [0, 255] and rounded to nearest even, into bytes 0
            // and 1 (v_cvt_pk_u8_f32 does clamp, round, convert and insert)
            out.w[j][ch][0] = __builtin_amdgcn_cvt_pk_u8_f32(
                o[ch][1], 1u, __builtin_amdgcn_cvt_pk_u8_f32(o[ch][0], 0u, 0u));
        } else if (F16 && !EXACT) {
            // The conversion may fuse with the last product (one rounding
            // to fp16 instead of two).
            typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));
            const f16x2 h = {(_Float16)o[ch][0], (_Float16)o[ch][1]};
            out.w[j][ch][0] = __builtin_bit_cast(uint32_t, h);
        } else if (F16) {
            out.w[j][ch][0] = f16_bits(o[ch][0]) | (f16_bits(o[ch][1]) << 16);
        } else {
            out.w[j][ch][0] = __builtin_bit_cast(uint32_t, o[ch][0]);
            out.w[j][ch][F16 ? 0 : 1] = __builtin_bit_cast(uint32_t, o[ch][1]);
        }
    }
}

// Store a lane's pairs of one output row: three planes (NCHW), or the six
// interleaved elements of the two pixels (NHWC). ODD is Cw & 1, a template
// parameter so that the stores are straight-line code: the compiler then
// counts them exactly in the vmcnt waits of the row loop (with a branch here
// it waits for them as well when it waits for the next rows' loads).
template <int F16, int J, int ODD>
__device__ __forceinline__ void store_row(uint8_t *orow, long long plane, int Cw, int lane,
                                          const RowOut<F16, J> &out, int nhwc)
{
    if constexpr (F16 == 2) {
        // uint8: a pair is 6 bytes (NHWC) or 2 per plane (NCHW); with Cw even
        // every pair starts on an even byte, so it goes out as 16-bit stores
#pragma unroll
        for (int j = 0; j < J; ++j) {
            const int c = pair_col(lane, j, Cw);
            const uint32_t r = out.w[j][0][0], g = out.w[j][1][0], b = out.w[j][2][0];
            if (nhwc && !ODD) {
                uint16_t *dst = (uint16_t *)(orow + 3LL * c);
                __builtin_nontemporal_store((uint16_t)((r & 0xffu) | ((g & 0xffu) << 8)), dst);
                __builtin_nontemporal_store((uint16_t)((b & 0xffu) | (r & 0xff00u)), dst + 1);
                __builtin_nontemporal_store((uint16_t)(((g >> 8) & 0xffu) | (b & 0xff00u)),
                                            dst + 2);
            } else if (nhwc) {
                // odd Cw: pixel c + 1 is the last column again past the end
                uint8_t *d0 = orow + 3LL * c, *d1 = orow + 3LL * min(c + 1, Cw - 1);
                d0[0] = (uint8_t)r;
                d0[1] = (uint8_t)g;
                d0[2] = (uint8_t)b;
                d1[0] = (uint8_t)(r >> 8);
                d1[1] = (uint8_t)(g >> 8);
                d1[2] = (uint8_t)(b >> 8);
            } else if (!ODD) {
#pragma unroll
                for (int ch = 0; ch < 3; ++ch)
                    __builtin_nontemporal_store((uint16_t)out.w[j][ch][0],
                                                (uint16_t *)(orow + ch * plane + c));
            } else {
                const int c1 = min(c + 1, Cw - 1);
#pragma unroll
                for (int ch = 0; ch < 3; ++ch) {
                    orow[ch * plane + c] = (uint8_t)out.w[j][ch][0];
                    orow[ch * plane + c1] = (uint8_t)(out.w[j][ch][0] >> 8);
                }
            }
        }
        return;
    }
    constexpr int kEsz = F16 ? 2 : 4;
    if (nhwc) {
#pragma unroll
        for (int j = 0; j < J; ++j) {
            const int c = pair_col(lane, j, Cw);
            uint8_t *dst = orow + (long long)3 * c * kEsz;
            if constexpr (!ODD) {
                // c even: 6 c bytes (fp16) is a multiple of 4, 12 c (fp32) of 8
                if (F16) {
                    const uint32_t w0 = out.w[j][0][0], w1 = out.w[j][1][0], w2 = out.w[j][2][0];
                    __builtin_nontemporal_store((w0 & 0xffffu) | (w1 << 16), (uint32_t *)dst);
                    __builtin_nontemporal_store((w2 & 0xffffu) | (w0 & 0xffff0000u),
                                                (uint32_t *)dst + 1);
                    __builtin_nontemporal_store((w1 >> 16) | (w2 & 0xffff0000u),
                                                (uint32_t *)dst + 2);
                } else {
                    // pixel c: r g b, pixel c + 1: r g b, as three 8-byte
                    // words (built from scalars: a vector gathered from the
                    // array's elements would keep the array in memory)
                    const uint64_t r0 = out.w[j][0][0], g0 = out.w[j][1][0], b0 = out.w[j][2][0];
                    const uint64_t r1 = out.w[j][0][F16 ? 0 : 1], g1 = out.w[j][1][F16 ? 0 : 1],
                                   b1 = out.w[j][2][F16 ? 0 : 1];
                    __builtin_nontemporal_store(r0 | (g0 << 32), (uint64_t *)dst);
                    __builtin_nontemporal_store(b0 | (r1 << 32), (uint64_t *)dst + 1);
                    __builtin_nontemporal_store(g1 | (b1 << 32), (uint64_t *)dst + 2);
                }
            } else {
                // odd Cw: element by element, pixel c + 1 is the last
                // column again past the end
                uint8_t *dst1 = orow + (long long)3 * min(c + 1, Cw - 1) * kEsz;
#pragma unroll
                for (int ch = 0; ch < 3; ++ch) {
                    if (F16) {
                        ((uint16_t *)dst)[ch] = (uint16_t)out.w[j][ch][0];
                        ((uint16_t *)dst1)[ch] = (uint16_t)(out.w[j][ch][0] >> 16);
                    } else {
                        ((uint32_t *)dst)[ch] = out.w[j][ch][0];
                        ((uint32_t *)dst1)[ch] = out.w[j][ch][F16 ? 0 : 1];
                    }
                }
            }
        }
        return;
    }
#pragma unroll
    for (int j = 0; j < J; ++j) {
        const int c = pair_col(lane, j, Cw);
        const uint32_t lo = (uint32_t)c * kEsz;
        if constexpr (!ODD) {  // every pair is whole and 2-element aligned
#pragma unroll
            for (int ch = 0; ch < 3; ++ch) {
                uint8_t *dst = orow + ch * plane + lo;
                if (F16) {
                    __builtin_nontemporal_store(out.w[j][ch][0], (uint32_t *)dst);
                } else {
                    typedef uint32_t u32x2v __attribute__((ext_vector_type(2)));
                    const u32x2v w = {out.w[j][ch][0], out.w[j][ch][F16 ? 0 : 1]};
                    __builtin_nontemporal_store(w, (u32x2v *)dst);
                }
            }
        } else {
            // odd Cw: element c + 1 is the last column again past the end
            // (its value is that column's too)
            const uint32_t lo1 = (uint32_t)min(c + 1, Cw - 1) * kEsz;
#pragma unroll
            for (int ch = 0; ch < 3; ++ch) {
                uint8_t *dst = orow + ch * plane;
                if (F16) {
                    *(uint16_t *)(dst + lo) = (uint16_t)out.w[j][ch][0];
                    *(uint16_t *)(dst + lo1) = (uint16_t)(out.w[j][ch][0] >> 16);
                } else {
                    *(uint32_t *)(dst + lo) = out.w[j][ch][0];
                    *(uint32_t *)(dst + lo1) = out.w[j][ch][F16 ? 0 : 1];
                }
            }
        }
    }
}

// Interpolate, normalise and store one output row from its staged rows
// (row 0 at byte `row0` of lds, row 1 at `row1`, both including the offset
// of the first byte in its chunk).
template <int F16, int J, int EXACT>
__device__ __forceinline__ void rows_compute(const NormK &nk, uint32_t row0, uint32_t row1,
                                             float wy, const int (&cx)[J][2],
                                             const float (&cw)[J][2], RowOut<F16, J> &out)
{
    // tap pairs, 4 per column iteration: pixel c and c + 1 of row 0, then row 1
    constexpr int kN = J == 1 ? 4 : 8;
    uint64_t v[J * 4];
#pragma unroll
    for (int j0 = 0; j0 < J; j0 += kN / 4)
        read_taps<J, kN>(row0, row1, cx, j0, *(uint64_t(*)[kN]) & v[4 * j0]);
#pragma unroll
    for (int j = 0; j < J; ++j) {
        float o[3][2];
#pragma unroll
        for (int px = 0; px < 2; ++px) {
            float pa[3], pd[3], qa[3], qd[3];
            unpack_ad(v[4 * j + px], pa, pd);
            unpack_ad(v[4 * j + 2 + px], qa, qd);
#pragma unroll
            for (int ch = 0; ch < 3; ++ch) {
                const float top = lerp_ad(pa[ch], pd[ch], cw[j][px]);
                const float bot = lerp_ad(qa[ch], qd[ch], cw[j][px]);
                o[ch][px] = out_value<F16, EXACT>(nk, ch, lerp(top, bot, wy));
            }
        }
        pack_pair<F16, EXACT, J>(out, j, o);
    }
}

// Horizontal lerps of one staged row at the lane's columns: h[j][px][ch].
template <int J>
__device__ __forceinline__ void rows_horizontal(uint32_t row, const int (&cx)[J][2],
                                                const float (&cw)[J][2], float (&h)[J][2][3])
{
    uint64_t v[2 * J];
    read_row_taps<J>(row, cx, v);
#pragma unroll
    for (int j = 0; j < J; ++j)
#pragma unroll
        for (int px = 0; px < 2; ++px) {
            float pa[3], pd[3];
            unpack_ad(v[2 * j + px], pa, pd);
#pragma unroll
            for (int ch = 0; ch < 3; ++ch)
                h[j][px][ch] = lerp_ad(pa[ch], pd[ch], cw[j][px]);
        }
}

// Vertical lerp of two rows of horizontal lerps, normalise, store.
template <int F16, int J, int EXACT>
__device__ __forceinline__ void rows_vertical(const NormK &nk, const float (&h0)[J][2][3],
                                              const float (&h1)[J][2][3], float wy,
                                              RowOut<F16, J> &out)
{
#pragma unroll
    for (int j = 0; j < J; ++j) {
        float o[3][2];
#pragma unroll
        for (int px = 0; px < 2; ++px)
#pragma unroll
            for (int ch = 0; ch < 3; ++ch)
                o[ch][px] = out_value<F16, EXACT>(nk, ch,
                                                  lerp(h0[j][px][ch], h1[j][px][ch], wy));
        pack_pair<F16, EXACT, J>(out, j, o);
    }
}

// One output row with horizontal lerps kept across rows (contiguous row
// ranges): a wave walking consecutive output rows of an upscale, or of a
// downscale by less than 2, meets the same source row again, and its
// horizontal lerps at the same columns are the same numbers. (py0, py1) are
// the source rows whose lerps h0, h1 hold, -1 when none (a new image or new
// column taps).
template <int F16, int J, int EXACT>
__device__ __forceinline__ void rows_compute_reuse(const NormK &nk, uint32_t row0, uint32_t row1,
                                                   float wy, int y0, int y1, int &py0, int &py1,
                                                   float (&h0)[J][2][3], float (&h1)[J][2][3],
                                                   const int (&cx)[J][2],
                                                   const float (&cw)[J][2], RowOut<F16, J> &out)
{
    const bool same = y0 == py0 && y1 == py1;
    if (!same && y0 == py1) {
#pragma unroll
        for (int j = 0; j < J; ++j)
#pragma unroll
            for (int px = 0; px < 2; ++px)
#pragma unroll
                for (int ch = 0; ch < 3; ++ch)
                    h0[j][px][ch] = h1[j][px][ch];
    } else if (!same) {
        rows_horizontal<J>(row0, cx, cw, h0);
    }
    if (!same)
        rows_horizontal<J>(row1, cx, cw, h1);
    py0 = y0;
    py1 = y1;
    rows_vertical<F16, J, EXACT>(nk, h0, h1, wy, out);
}

}  // namespace
}  // namespace smol
