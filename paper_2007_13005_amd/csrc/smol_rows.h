// smol_rows.h -- the row-streaming kernels (RGB and I420) as templates. Each
// smol_rows_*.hip file instantiates one part of them (input, output type, row
// walk, output layout), so the parts build in parallel.
#pragma once

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
__device__ __forceinline__ RowStep row_step_of(int waves, int Ch)
{
    return STRIDE ? RowStep{waves / Ch, waves % Ch, Ch} : RowStep{0, 1, Ch};
}

// First row and row count of wave `w` (of `waves`) over T rows.
template <int STRIDE>
__device__ __forceinline__ void wave_rows(long long T, int w, int waves, long long &r0,
                                          int &n_rows)
{
    if (STRIDE) {
        r0 = w;
        n_rows = w < T ? (int)((T - w + waves - 1) / waves) : 0;
    } else {
        r0 = T * w / waves;
        n_rows = (int)(T * (w + 1) / waves - r0);
    }
}

// Workgroups are dealt to the 8 XCDs round-robin; remap so the waves of one
// XCD take consecutive rows (neighbouring output rows share source rows when
// the vertical scale is below 2, and share the XCD's L2).
__device__ __forceinline__ int xcd_position(int g, int G)
{
    return G % 8 == 0 ? (g % 8) * (G / 8) + g / 8 : g;
}

// A workgroup holds blockDim.x / 64 independent waves (no barriers), each
// with its own LDS slot of `slot_bytes`; several waves per workgroup cut the
// cost of dispatching the grid. Returns the wave's slot and sets its lane,
// the number of waves and the wave's rows.
template <int STRIDE>
__device__ __forceinline__ uint8_t *rows_wave(uint8_t *lds_all, int slot_bytes, long long T,
                                              int &lane, int &nw, long long &r0, int &n_rows)
{
    const int wpg = (int)(blockDim.x >> 6);
    const int wid = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
    lane = (int)(threadIdx.x & 63);
    const int ng = (int)gridDim.x;
    nw = ng * wpg;
    const int g = STRIDE ? xcd_position((int)blockIdx.x, ng) : (int)blockIdx.x;
    wave_rows<STRIDE>(T, g * wpg + wid, nw, r0, n_rows);
    return lds_all + wid * slot_bytes;
}

__device__ __forceinline__ void floor_divmod(long long n, int d, int &q, int &r)
{
    const long long qq = n >= 0 ? n / d : -((-n + d - 1) / d);
    q = (int)qq;
    r = (int)(n - qq * d);
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
__device__ __forceinline__ void vcursor_init(VCursor &v, const RowImg &g, int rr, const RowStep &s)
{
    v.H = g.H;
    v.den = 2 * g.Hr;
    floor_divmod((long long)(2 * (g.top + rr) + 1) * g.H - g.Hr, v.den, v.q, v.rem);
    if (STRIDE) {
        floor_divmod(2LL * g.H * s.dr, v.den, v.qs, v.rs);
        floor_divmod(2LL * g.H * (s.dr - s.Ch), v.den, v.qw, v.rw);
    } else {
        v.qs = (2 * g.H) / v.den;
        v.rs = 2 * g.H - v.qs * v.den;
    }
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
    vcursor_init<STRIDE>(c.v, g, rr, s);
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
template <int G>
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
        st.c0[g] = __builtin_nontemporal_load(
            (const __attribute__((address_space(1))) u32x4 *)(p0 + o0));
        st.c1[g] = __builtin_nontemporal_load(
            (const __attribute__((address_space(1))) u32x4 *)(p1 + o1));
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
            // nearest, ties to even (v_rndne_f32), of a value in [0, 255]
            const uint32_t b0 = (uint32_t)__builtin_rintf(clamp255(o[ch][0]));
            const uint32_t b1 = (uint32_t)__builtin_rintf(clamp255(o[ch][1]));
            out.w[j][ch][0] = b0 | (b1 << 8);
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
                    typedef uint32_t u32x2v __attribute__((ext_vector_type(2)));
                    const u32x2v q0 = {out.w[j][0][0], out.w[j][1][0]};
                    const u32x2v q1 = {out.w[j][2][0], out.w[j][0][F16 ? 0 : 1]};
                    const u32x2v q2 = {out.w[j][1][F16 ? 0 : 1], out.w[j][2][F16 ? 0 : 1]};
                    __builtin_nontemporal_store(q0, (u32x2v *)dst);
                    __builtin_nontemporal_store(q1, (u32x2v *)dst + 1);
                    __builtin_nontemporal_store(q2, (u32x2v *)dst + 2);
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

// FORM: bit 0 NHWC output, bit 1 odd crop width (kFormNhwc, kFormOdd).
template <int F16, int J, int EXACT, int G, int P, int STRIDE, int FORM>
__global__ void __launch_bounds__(64 * kRowsMaxWavesPerGroup) rgb_rows_kernel(BatchArgs a)
{
    constexpr int NHWC = FORM & kFormNhwc, ODD = (FORM & kFormOdd) ? 1 : 0;
    extern __shared__ __attribute__((aligned(16))) uint8_t lds_all[];
    int lane, nw;
    long long r0;
    int n_rows;
    const int Ch = a.Ch;
    uint8_t *const lds = rows_wave<STRIDE>(lds_all, 2048 * G, (long long)a.n * Ch, lane, nw, r0,
                                           n_rows);
    if (n_rows <= 0)
        return;
    const RowStep step = row_step_of<STRIDE>(nw, Ch);
    constexpr int kEsz = F16 == 2 ? 1 : F16 ? 2 : 4;
    int c_img = (int)(r0 / Ch), c_rr = (int)(r0 - (long long)c_img * Ch);  // row to interpolate
    RowCursor lc;                                                          // next row to load
    cursor_image<STRIDE>(lc, a, c_img, c_rr, step);

    // Output row pointer of the row to interpolate: a step adds 3 Ch di + dr
    // rows, plus 2 Ch (planes 1 and 2 of the image left) when it wraps.
    // bytes between an image's output rows: Cw elements per plane (NCHW) or
    // 3 Cw (NHWC); a wrap to the next image skips the rest of the image.
    const long long rb = (long long)a.Cw * kEsz, rowb = NHWC ? 3 * rb : rb;
    const long long imgb = 3LL * Ch * rb;
    uint8_t *orow = (uint8_t *)a.out + (long long)(a.img_base + c_img) * imgb + c_rr * rowb;
    const long long ostep = step.di * imgb + step.dr * rowb, owrap = imgb - Ch * rowb;
    int cx[J][2];
    float cw[J][2];
    int cW, cWr, cleft;
    {
        const RowImg g = row_img(a, c_img);
        row_taps<J>(g, a.Cw, cx, cw, lane);
        cW = g.W;
        cWr = g.Wr;
        cleft = g.left;
    }
    const NormK nk = norm_consts(a);
    const uint32_t lds0 = lds_addr(lds);

    // The load cursor stops at the wave's last row: past the end the loads
    // repeat that row (fetching one chunk), so every step issues the same
    // loads and the compiler can count exactly what is outstanding when a
    // row is written to LDS.
    int lrow = 0;
    bool at_end = false;  // the cursor sits on the wave's last row, already loaded
    auto advance = [&]() {
        if (lrow + 1 < n_rows) {
            cursor_next<STRIDE>(lc, a, step);
            ++lrow;
        } else {
            at_end = true;
        }
    };
    // P = 2: a step loads row k + 2 into FUT, interpolates row k (staged in
    // LDS), writes row k + 1 (in NXT) into the slot; the three register sets
    // rotate over three steps without copies. P = 1: one register set, loaded
    // with row k + 1 before row k is interpolated. The loop runs the n_rows - 1
    // steps that stage a next row and leaves only at its end, with nothing
    // outstanding but the prefetched row; the last row is interpolated after
    // it.
    StagedRows<G> A, B, C;
    load_rows<G>(A, lc, lane, false);
    advance();
    if (P == 2) {
        load_rows<G>(B, lc, lane, at_end);
        advance();
    }
    write_rows<G>(lds, A, lane);
    int csh0 = A.sh0, csh1 = A.sh1, cy0 = A.y0, cy1 = A.y1;
    float cwy = A.wy;
    // Contiguous ranges keep the horizontal lerps of the last two source
    // rows (see rows_compute_reuse); J = 4 would need 48 more registers.
    constexpr bool kReuse = STRIDE == 0 && J <= 2;
    float h0[J][2][3], h1[J][2][3];
    int py0 = -1, py1 = -1;
    const long long plane = (long long)Ch * a.Cw * kEsz;
    RowOut<F16, J> out;
    auto compute = [&]() {
        if constexpr (kReuse)
            rows_compute_reuse<F16, J, EXACT>(nk, lds0 + (uint32_t)csh0,
                                              lds0 + (uint32_t)(1024 * G + csh1), cwy, cy0, cy1,
                                              py0, py1, h0, h1, cx, cw, out);
        else
            rows_compute<F16, J, EXACT>(nk, lds0 + (uint32_t)csh0,
                                        lds0 + (uint32_t)(1024 * G + csh1), cwy, cx, cw, out);
    };
#define SMOL_ROWS_STEP(NXT, FUT)                                                              \
    {                                                                                         \
        load_rows<G>(FUT, lc, lane, at_end);                                                  \
        advance();                                                                            \
        compute();                                                                            \
        write_rows<G>(lds, NXT, lane);                                                        \
        store_row<F16, J, ODD>(orow, plane, a.Cw, lane, out, NHWC);                         \
        csh0 = NXT.sh0;                                                                       \
        csh1 = NXT.sh1;                                                                       \
        cy0 = NXT.y0;                                                                         \
        cy1 = NXT.y1;                                                                         \
        cwy = NXT.wy;                                                                         \
        const int pimg = c_img;                                                               \
        c_img += step.di;                                                                     \
        c_rr += step.dr;                                                                      \
        orow += ostep;                                                                        \
        if (c_rr >= Ch) {                                                                     \
            c_rr -= Ch;                                                                       \
            ++c_img;                                                                          \
            orow += owrap;                                                                    \
        }                                                                                     \
        if (c_img != pimg) {                                                                  \
            py0 = py1 = -1; /* another image's rows */                                        \
            const RowImg g = row_img(a, c_img);                                               \
            if (g.W != cW || g.Wr != cWr || g.left != cleft) {                                \
                cW = g.W;                                                                     \
                cWr = g.Wr;                                                                   \
                cleft = g.left;                                                               \
                row_taps<J>(g, a.Cw, cx, cw, lane);                                           \
            }                                                                                 \
        }                                                                                     \
    }
    int left = n_rows - 1;
    if (P == 2) {
        for (; left >= 3; left -= 3) {
            SMOL_ROWS_STEP(B, C)
            SMOL_ROWS_STEP(C, A)
            SMOL_ROWS_STEP(A, B)
        }
        if (left >= 1)
            SMOL_ROWS_STEP(B, C)
        if (left >= 2)
            SMOL_ROWS_STEP(C, A)
    } else {
        for (; left > 0; --left)
            SMOL_ROWS_STEP(A, A)
    }
#undef SMOL_ROWS_STEP
    compute();
    store_row<F16, J, ODD>(orow, plane, a.Cw, lane, out, NHWC);
}

// ---------------------------------------------------------------------------
// I420, row streaming: one wave per workgroup, the scheme of the RGB kernel.
//
// For each output row the wave loads eight row segments into registers and
// then into its LDS slot (1 KiB each): luma rows y0 and y1 over the crop's
// luma column span and, for each chroma plane, the chroma rows that the
// vertical chroma taps of y0 and y1 read over the matching chroma span. Those
// are at most three rows: the first chroma row of y1 is always one of the two
// of y0 (y1 = y0 + 1 or the clamped y0).
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
// Cb r2, Cr r0, Cr r1, Cr r2 (r0, r1: the chroma rows of y0; r2: the second
// chroma row of y1), with each segment's offset in its first chunk, the luma
// vertical weight, the chroma vertical weights of y0 and y1, and which of r0,
// r1 is y1's first chroma row. A lane holds one 16-byte chunk of each
// segment, and with GL = 2 a second chunk of each luma segment (luma rows of
// up to 2 KiB).
template <int GL>
struct YuvStaged {
    u32x4 c[8];
    u32x4 c2[2];  // second luma chunks (GL = 2)
    int sh[8];
    float wy;
    int fy0, fy1;  // vertical chroma weights of luma rows y0, y1, in quarters
    int b0;
};

// Load cursor over the output rows of I420 frames (the walk of the RGB
// cursor, with the three plane bases).
struct YuvCursor {
    int img, rr;
    VCursor v;          // luma vertical map over the region's rows
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
    vcursor_init<STRIDE>(c.v, lg, rr, s);
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

template <int GL>
__device__ __forceinline__ void yuv_load(YuvStaged<GL> &st, const YuvCursor &c, int lane,
                                         bool repeat)
{
    int y0, y1;
    vcursor_tap(c.v, y0, y1, st.wy);
    const Tap t0 = chroma_tap(c.ry + y0, c.Hc), t1 = chroma_tap(c.ry + y1, c.Hc);
    st.fy0 = (int)(4.0f * t0.w);  // exact: 0, 1 or 3
    st.fy1 = (int)(4.0f * t1.w);
    st.b0 = t1.x0 == t0.x0 ? 0 : 1;
    const uintptr_t row[8] = {
        c.base[0] + (uintptr_t)y0 * (uintptr_t)c.W,     c.base[0] + (uintptr_t)y1 * (uintptr_t)c.W,
        c.base[1] + (uintptr_t)t0.x0 * (uintptr_t)c.Wc, c.base[1] + (uintptr_t)t0.x1 * (uintptr_t)c.Wc,
        c.base[1] + (uintptr_t)t1.x1 * (uintptr_t)c.Wc, c.base[2] + (uintptr_t)t0.x0 * (uintptr_t)c.Wc,
        c.base[2] + (uintptr_t)t0.x1 * (uintptr_t)c.Wc, c.base[2] + (uintptr_t)t1.x1 * (uintptr_t)c.Wc};
    typedef __attribute__((address_space(1))) const uint8_t GlobalByte;
#pragma unroll
    for (int s = 0; s < 8; ++s) {
        st.sh[s] = (int)(row[s] & 15);
        const int last = repeat ? 0 : (st.sh[s] + (s < 2 ? c.yspan : c.cspan) - 1) >> 4;
        GlobalByte *p = (GlobalByte *)(row[s] - (uintptr_t)st.sh[s]);
        st.c[s] = __builtin_nontemporal_load(
            (const __attribute__((address_space(1))) u32x4 *)(p + 16u * (uint32_t)min(lane, last)));
        if (GL == 2 && s < 2)
            st.c2[s] = __builtin_nontemporal_load(
                (const __attribute__((address_space(1))) u32x4 *)(p + 16u * (uint32_t)min(64 + lane,
                                                                                           last)));
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

template <int J>
__device__ __forceinline__ void yuv_cols(YuvCols<J> &k, const YuvImg &g, int Cw, int lane,
                                         int siting)
{
    const int Wc = (g.fw + 1) >> 1;
    const int cxf = chroma_tap(g.rx + g.xf, Wc, siting).x0;
#pragma unroll
    for (int j = 0; j < J; ++j)
#pragma unroll
        for (int px = 0; px < 2; ++px) {
            const int c = min(pair_col(lane, j, Cw) + px, Cw - 1);
            const Tap t = axis_tap(g.left + c, g.W, g.Wr);
            const Tap a0 = chroma_tap(g.rx + t.x0, Wc, siting),
                      a1 = chroma_tap(g.rx + t.x1, Wc, siting);
            k.ox[j][px] = t.x0 - g.xf;
            k.wx[j][px] = t.w;
            k.oc[j][px] = a0.x0 - cxf;
            // the samples of luma column xi are bytes d0, d1 of the 4 read
            // from each chroma row; perm(row b, row a) yields a[d0], a[d1],
            // b[d0], b[d1]
            const Tap ax[2] = {a0, a1};
#pragma unroll
            for (int xi = 0; xi < 2; ++xi) {
                const uint32_t d0 = (uint32_t)(ax[xi].x0 - a0.x0);
                const uint32_t d1 = (uint32_t)(ax[xi].x1 - a0.x0);
                k.sel[j][px][xi] = d0 | d1 << 8 | (4 + d0) << 16 | (4 + d1) << 24;
                const uint32_t fx = (uint32_t)(4.0f * ax[xi].w);  // exact: 0 .. 3
                k.hw[j][px][xi] = (4 - fx) | fx << 8;
            }
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

// 16 * (chroma - 128) at one luma tap: the tap's four chroma samples
// (selected from chroma rows ra and rb) dotted with its weight bytes, minus
// 2048, exact in integers.
__device__ __forceinline__ float chroma16(uint32_t ra, uint32_t rb, uint32_t sel, uint32_t wts)
{
    const uint32_t smp = __builtin_amdgcn_perm(rb, ra, sel);
    return (float)(int)__builtin_amdgcn_udot4(smp, wts, (uint32_t)-2048, false);
}

template <int F16, int J, int EXACT, int GL>
__device__ __forceinline__ void yuv_compute(const NormK &nk, uint32_t slot, const int (&sh)[8],
                                            float wy, int fy0, int fy1, int b0,
                                            const YuvCols<J> &k, RowOut<F16, J> &out)
{
    // weight bytes of luma row yi and column xi: hw(xi) * (4 + 65535 fy(yi))
    // = (4 - fy) * [4 - fx, fx, 0, 0] + fy * [0, 0, 4 - fx, fx] (no carries)
    const uint32_t vm[2] = {4u + 65535u * (uint32_t)fy0, 4u + 65535u * (uint32_t)fy1};
#pragma unroll
    for (int j = 0; j < J; ++j) {
        float o[3][2];
#pragma unroll
        for (int px = 0; px < 2; ++px) {
            // reads: Y y0, Y y1, Cb r0..r2, Cr r0..r2
            uint32_t A[8], q[8];
#pragma unroll
            for (int s = 0; s < 8; ++s)
                A[s] = slot + yuv_seg<GL>(s) + (uint32_t)sh[s] +
                       (uint32_t)(s < 2 ? k.ox[j][px] : k.oc[j][px]);
            lds_read_quads<8>(A, q);
            // 16 * (chroma - 128) at (y0, y1) x (x0, x1) for both planes:
            // luma row y0 reads chroma rows r0, r1; y1 reads r0 or r1 (b0),
            // and r2
            float cc[2][2][2];  // [plane][luma row][luma col]
#pragma unroll
            for (int pl = 0; pl < 2; ++pl) {
                const uint32_t r0 = q[2 + 3 * pl], r1 = q[3 + 3 * pl], r2 = q[4 + 3 * pl];
                const uint32_t ra1 = b0 ? r1 : r0;
#pragma unroll
                for (int xi = 0; xi < 2; ++xi) {
                    cc[pl][0][xi] = chroma16(r0, r1, k.sel[j][px][xi], __umul24(k.hw[j][px][xi], vm[0]));
                    cc[pl][1][xi] = chroma16(ra1, r2, k.sel[j][px][xi], __umul24(k.hw[j][px][xi], vm[1]));
                }
            }
            float rgb[2][2][3];  // [luma row][luma col][channel]
#pragma unroll
            for (int yi = 0; yi < 2; ++yi)
#pragma unroll
                for (int xi = 0; xi < 2; ++xi) {
                    const float Y = xi ? cvt_ubyte1(q[yi]) : cvt_ubyte0(q[yi]);
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

// FORM as for rgb_rows_kernel; GL: chunks per lane of a luma segment (staged
// luma rows of up to 1 or 2 KiB).
template <int F16, int J, int EXACT, int STRIDE, int FORM, int GL>
__global__ void __launch_bounds__(64 * kRowsMaxWavesPerGroup) __attribute__((amdgpu_waves_per_eu(J <= 2 ? 3 : 1)))
yuv_rows_kernel(BatchArgs a)
{
    constexpr int NHWC = FORM & kFormNhwc, ODD = (FORM & kFormOdd) ? 1 : 0;
    extern __shared__ __attribute__((aligned(16))) uint8_t lds_all[];
    int lane, nw;
    long long r0;
    int n_rows;
    const int Ch = a.Ch;
    uint8_t *const lds = rows_wave<STRIDE>(lds_all, yuv_seg<GL>(8), (long long)a.n * Ch, lane,
                                           nw, r0, n_rows);
    if (n_rows <= 0)
        return;
    const RowStep step = row_step_of<STRIDE>(nw, Ch);
    constexpr int kEsz = F16 == 2 ? 1 : F16 ? 2 : 4;
    int c_img = (int)(r0 / Ch), c_rr = (int)(r0 - (long long)c_img * Ch);  // row to interpolate
    YuvCursor lc;                                                          // next row to load
    yuv_cursor_image<STRIDE>(lc, a, c_img, c_rr, step);
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
        yuv_cols<J>(cols, g, a.Cw, lane, a.siting);
        cW = g.W;
        cWr = g.Wr;
        cleft = g.left;
    }
    const NormK nk = norm_consts(a);
    const uint32_t lds0 = lds_addr(lds);

    // One register set: row k + 1 is loaded before row k is interpolated.
    // The loop runs the n_rows - 1 steps that stage a next row and leaves
    // only at its end; the last row is interpolated after it.
    int lrow = 0;
    auto advance = [&]() {
        if (lrow + 1 < n_rows) {
            yuv_cursor_next<STRIDE>(lc, a, step);
            ++lrow;
        }
    };
    const long long plane = (long long)Ch * a.Cw * kEsz;
    RowOut<F16, J> out;
    YuvStaged<GL> R;
    yuv_load<GL>(R, lc, lane, false);
    advance();
    yuv_write<GL>(lds, R, lane);
    int csh[8];
#pragma unroll
    for (int s = 0; s < 8; ++s)
        csh[s] = R.sh[s];
    float cwy = R.wy;
    int cfy0 = R.fy0, cfy1 = R.fy1;
    int cb0 = R.b0;
    for (int left = n_rows - 1; left > 0; --left) {
        yuv_load<GL>(R, lc, lane, false);
        advance();
        yuv_compute<F16, J, EXACT, GL>(nk, lds0, csh, cwy, cfy0, cfy1, cb0, cols, out);
        yuv_write<GL>(lds, R, lane);
        store_row<F16, J, ODD>(orow, plane, a.Cw, lane, out, NHWC);
#pragma unroll
        for (int s = 0; s < 8; ++s)
            csh[s] = R.sh[s];
        cwy = R.wy;
        cfy0 = R.fy0;
        cfy1 = R.fy1;
        cb0 = R.b0;
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
    yuv_compute<F16, J, EXACT, GL>(nk, lds0, csh, cwy, cfy0, cfy1, cb0, cols, out);
    store_row<F16, J, ODD>(orow, plane, a.Cw, lane, out, NHWC);
}


// Kernel for a plan: output type, arithmetic mode, chunk groups, column
// pairs per lane and prefetch depth from the launch arguments.
template <int F16, int EXACT, int G, int STRIDE, int FORM>
const void *rgb_rows_g(int col_iters, int prefetch)
{
    if (prefetch == 1)
        return col_iters <= 1   ? (const void *)rgb_rows_kernel<F16, 1, EXACT, G, 1, STRIDE, FORM>
               : col_iters <= 2 ? (const void *)rgb_rows_kernel<F16, 2, EXACT, G, 1, STRIDE, FORM>
                                : (const void *)rgb_rows_kernel<F16, 4, EXACT, G, 1, STRIDE, FORM>;
    return col_iters <= 1   ? (const void *)rgb_rows_kernel<F16, 1, EXACT, G, 2, STRIDE, FORM>
           : col_iters <= 2 ? (const void *)rgb_rows_kernel<F16, 2, EXACT, G, 2, STRIDE, FORM>
                            : (const void *)rgb_rows_kernel<F16, 4, EXACT, G, 2, STRIDE, FORM>;
}

template <int F16, int EXACT, int STRIDE, int FORM>
const void *rgb_rows_e(int col_iters, int groups, int prefetch)
{
    return groups <= 1   ? rgb_rows_g<F16, EXACT, 1, STRIDE, FORM>(col_iters, prefetch)
           : groups <= 2 ? rgb_rows_g<F16, EXACT, 2, STRIDE, FORM>(col_iters, prefetch)
                         : rgb_rows_g<F16, EXACT, 4, STRIDE, FORM>(col_iters, prefetch);
}

// The crop width's parity picks the FORM of a layout.
template <int F16, int EXACT, int STRIDE, int NHWC>
const void *rgb_rows_f(const BatchArgs &a)
{
    return (a.Cw & 1) ? rgb_rows_e<F16, EXACT, STRIDE, NHWC | kFormOdd>(a.col_iters, a.row_groups,
                                                                       a.prefetch)
                      : rgb_rows_e<F16, EXACT, STRIDE, NHWC>(a.col_iters, a.row_groups, a.prefetch);
}

template <int F16, int STRIDE, int NHWC>
const void *rgb_rows_table(const BatchArgs &a)
{
    return a.exact ? rgb_rows_f<F16, 1, STRIDE, NHWC>(a) : rgb_rows_f<F16, 0, STRIDE, NHWC>(a);
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
