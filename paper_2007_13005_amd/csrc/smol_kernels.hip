// smol_kernels.hip -- fused preprocessing kernels for gfx950 (MI355X).
//
// One pass per output element does the whole standard ResNet preprocessing of
// the paper's section 2 (steps 2-4): short-side bilinear resize, centre crop,
// float conversion + per-channel normalisation, channels-first store; for I420
// input the BT.601 conversion of App. A ("Components") runs first at every luma
// tap. Section 6.2's rules license the fusion: normalisation, conversion and
// channel reordering fuse, and the crop is applied in output space (resize and
// crop swap), so only source pixels that feed a cropped output are read.
//
// The work is an HBM-bound gather/stencil, not a contraction: no MFMA. The
// LDS kernels stage exactly the source rows the vertical taps use, over the
// crop's column span, with wavefront-wide 16-byte direct-to-LDS loads; the
// bilinear taps then read those rows from LDS as aligned dwords.
//
// Arithmetic follows the definition operation for operation: each lerp is
// a + w * (b - a) with every operation rounded on its own (this file is built
// with -ffp-contract=off), horizontal before vertical, and the normalisation
// is the correctly rounded quotient (v - mean) / std. The quotient is formed
// from the host-rounded reciprocal y = RN(1/std) as q0 = a*y, corrected once
// with the exact FMA residual: q = q0 + (a - std*q0) * y. With y correctly
// rounded this gives RN(a / std) whenever the quotient is a normal number
// (Markstein's correction step), which covers every value a = v - mean can
// take here. fp16 outputs are the round-to-nearest-even of those fp32 values.
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <algorithm>
#include <map>
#include <mutex>
#include <tuple>

#include "smol_device.h"

namespace smol {
namespace {

constexpr int kThreads = 256;


// Two horizontally adjacent RGB pixels (6 bytes) at LDS byte address `addr`,
// read as three aligned dwords and realigned with v_alignbyte.
__device__ __forceinline__ void lds_pixel_pair(const uint8_t *lds, int addr, float (&p)[6])
{
    const uint32_t *w = (const uint32_t *)(lds + (addr & ~3));
    const uint32_t d0 = w[0], d1 = w[1], d2 = w[2];
    const uint32_t sh = (uint32_t)addr & 3u;
    const uint32_t lo = __builtin_amdgcn_alignbyte(d1, d0, sh);
    const uint32_t hi = __builtin_amdgcn_alignbyte(d2, d1, sh);
    p[0] = (float)(lo & 0xffu);
    p[1] = (float)((lo >> 8) & 0xffu);
    p[2] = (float)((lo >> 16) & 0xffu);
    p[3] = (float)(lo >> 24);
    p[4] = (float)(hi & 0xffu);
    p[5] = (float)((hi >> 8) & 0xffu);
}

typedef __attribute__((address_space(3))) void lds_void_t;

// Copy `nbytes` source bytes starting at absolute address `row` into an LDS
// slot, as 16-byte chunks aligned in the global address space, so the slot
// holds the bytes from (row & ~15) on. Called by one whole wave with
// wave-uniform arguments. When every chunk lies inside [gbase, gend) the
// wave issues one direct-to-LDS load per 64 chunks (1 KiB per instruction)
// with no per-lane checks; otherwise (a row touching either end of the
// buffer) the chunks that straddle an end are copied byte by byte.
__device__ __forceinline__ void stage_row(uint8_t *slot, uintptr_t row, int nbytes,
                                          uintptr_t gbase, uintptr_t gend, int lane)
{
    const uintptr_t al = row & ~(uintptr_t)15;
    const int nch = (int)((row - al + (uintptr_t)nbytes + 15) >> 4);
    if (al >= gbase && al + 16 * (uintptr_t)nch <= gend) {
        for (int j0 = 0; j0 < nch; j0 += 64) {
            if (j0 + lane < nch)
                __builtin_amdgcn_global_load_lds(
                    (const void *)(al + 16 * (uintptr_t)(j0 + lane)),
                    (lds_void_t *)(slot + 16 * j0), 16, 0, 0);
        }
        return;
    }
    // Every 64-chunk group below issues at least one vector-memory
    // instruction (its first chunk holds bytes of the row), as the fast path
    // does; the row-streaming kernel's wait counts rely on that.
    for (int j0 = 0; j0 < nch; j0 += 64) {
        const int j = j0 + lane;
        const uintptr_t ga = al + 16 * (uintptr_t)j;
        if (j < nch && ga >= gbase && ga + 16 <= gend) {
            __builtin_amdgcn_global_load_lds((const void *)ga, (lds_void_t *)(slot + 16 * j0), 16,
                                             0, 0);
        } else if (j < nch) {
            for (int k = 0; k < 16; ++k)
                if (ga + k >= gbase && ga + k < gend)
                    slot[16 * j + k] = *(const uint8_t *)(ga + k);
        }
    }
}

// ---------------------------------------------------------------------------
// RGB, LDS-staged, persistent, double-buffered.
//
// Work items are (image, band of R output rows), image-major; workgroup g
// takes the contiguous range [g*T/G, (g+1)*T/G) of the T items, so it walks
// consecutive bands of the same image and recomputes column taps only when
// the image geometry changes. LDS holds two buffers; item k uses buffer k&1.
//
// Iteration k: (1) wait until this wave's gathers for item k have landed,
// (2) barrier -- now every wave's gathers for item k are in LDS and every
// wave has finished reading buffer (k+1)&1 for item k-1, (3) prepare item
// k+1 in buffer (k+1)&1 and issue its gathers (each wave stages every fourth
// distinct source row), (4) interpolate item k and store it while those
// gathers are in flight. Vector-memory operations complete in issue order,
// so step (1) waits with vmcnt(n), n = a lower bound on the stores this
// wave issued after item k's gathers: it never waits for item k+1's
// gathers, and exposes no store latency.
//
// Buffer layout: colx/colw [Cw] | rowa0/rowa1/twy [R] | 2R source-row slots.
// ---------------------------------------------------------------------------
constexpr int kWavesPerGroup = kThreads / 64;

// s_waitcnt vmcnt(n) for a wave-uniform n in 0..63 (the count is an
// immediate, so dispatch on it).
__device__ __forceinline__ void wait_vmcnt(int n)
{
#define SMOL_W(N)                                                                             \
    case N:                                                                                   \
        asm volatile("s_waitcnt vmcnt(" #N ")" ::: "memory");                                 \
        break;
    switch (n) {
        SMOL_W(0) SMOL_W(1) SMOL_W(2) SMOL_W(3) SMOL_W(4) SMOL_W(5) SMOL_W(6) SMOL_W(7)
        SMOL_W(8) SMOL_W(9) SMOL_W(10) SMOL_W(11) SMOL_W(12) SMOL_W(13) SMOL_W(14) SMOL_W(15)
        SMOL_W(16) SMOL_W(17) SMOL_W(18) SMOL_W(19) SMOL_W(20) SMOL_W(21) SMOL_W(22) SMOL_W(23)
        SMOL_W(24) SMOL_W(25) SMOL_W(26) SMOL_W(27) SMOL_W(28) SMOL_W(29) SMOL_W(30) SMOL_W(31)
        SMOL_W(32) SMOL_W(33) SMOL_W(34) SMOL_W(35) SMOL_W(36) SMOL_W(37) SMOL_W(38) SMOL_W(39)
        SMOL_W(40) SMOL_W(41) SMOL_W(42) SMOL_W(43) SMOL_W(44) SMOL_W(45) SMOL_W(46) SMOL_W(47)
        SMOL_W(48) SMOL_W(49) SMOL_W(50) SMOL_W(51) SMOL_W(52) SMOL_W(53) SMOL_W(54) SMOL_W(55)
        SMOL_W(56) SMOL_W(57) SMOL_W(58) SMOL_W(59) SMOL_W(60) SMOL_W(61) SMOL_W(62)
    default:
        asm volatile("s_waitcnt vmcnt(63)" ::: "memory");
        break;
    }
#undef SMOL_W
}

__device__ __forceinline__ void barrier_lds()
{
    asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

struct BufView {
    int *colx;
    float *colw;
    int *rowa0, *rowa1;
    float *twy;
};

__device__ __forceinline__ BufView buf_view(uint8_t *base, int Cw, int R)
{
    BufView v;
    v.colx = (int *)base;
    v.colw = (float *)(v.colx + Cw);
    v.rowa0 = (int *)(v.colw + Cw);
    v.rowa1 = v.rowa0 + R;
    v.twy = (float *)(v.rowa1 + R);
    return v;
}

// Number of set bits of the 64-bit mask in lanes below the calling lane.
__device__ __forceinline__ int bits_below(unsigned long long m)
{
    return __builtin_amdgcn_mbcnt_hi((unsigned)(m >> 32),
                                     __builtin_amdgcn_mbcnt_lo((unsigned)m, 0u));
}

struct Geo {
    int W, Wr, left;
};

// Fill buffer `bi` for item w and issue this wave's share of its gathers.
// Returns the number of vector-memory instructions issued, or -1 if a row
// touched an end of the source buffer (byte copies: count unknown).
__device__ __forceinline__ int prepare(const BatchArgs &a, long long w, int bi, uint8_t *lds,
                                       Geo &held, int tid)
{
    const int lane = tid & 63, wave = tid >> 6;
    const int Cw = a.Cw, R = a.R;
    const int img = (int)(w / a.bands);
    const int band = (int)(w - (long long)img * a.bands);
    const int boff = bi * a.stage_bytes;
    const BufView v = buf_view(lds + boff, Cw, R);
    const int slot0 = boff + a.slots_off;  // LDS address of slot 0
    Desc d;
    image_desc(a, img, d);
    const int r_begin = band * R;
    const int r_cnt = min(R, a.Ch - r_begin);
    const int xs = axis_tap(d.left, d.W, d.Wr).x0;
    const int span_bytes = 3 * (axis_tap(d.left + Cw - 1, d.W, d.Wr).x1 - xs + 1);
    if (d.W != held.W || d.Wr != held.Wr || d.left != held.left) {
        held.W = d.W;
        held.Wr = d.Wr;
        held.left = d.left;
        for (int c = tid; c < Cw; c += kThreads) {
            const Tap t = axis_tap(d.left + c, d.W, d.Wr);
            v.colx[c] = 3 * (t.x0 - xs);
            v.colw[c] = t.w;
        }
    }

    // Row taps of band row `lane` (every wave computes them). Both tap
    // sequences are non-decreasing and y1 is y0 or y0 + 1, so among the
    // candidates y0[0], y1[0], y0[1], ... y0[r] is new iff it exceeds
    // y1[r-1], and y1[r] is new iff it differs from y0[r] and from y1[r-1].
    // The k-th new candidate goes to slot k. The distinct rows seen before
    // row r end with y1[r-1] (slot before-1), preceded by y0[r-1] when
    // y1[r-1] = y0[r-1] + 1 (slot before-2): a repeated y0[r] is one of
    // those two, a repeated y1[r] is y0[r] (clamped) or y1[r-1].
    const bool live = lane < r_cnt;
    const Tap t = axis_tap(d.top + r_begin + min(lane, r_cnt - 1), d.H, d.Hr);
    const int prev_y1 = __shfl_up(t.x1, 1, 64);
    const bool new0 = live && (lane == 0 || t.x0 > prev_y1);
    const bool new1 = live && t.x1 != t.x0 && (lane == 0 || t.x1 != prev_y1);
    const unsigned long long m0 = __ballot(new0);
    const unsigned long long m1 = __ballot(new1);
    const int before = bits_below(m0) + bits_below(m1);  // new candidates in rows < lane
    const int s0 = new0 ? before : (t.x0 == prev_y1 ? before - 1 : before - 2);
    const int s1 = new1 ? before + (new0 ? 1 : 0) : (t.x1 == t.x0 ? s0 : before - 1);
    const uintptr_t gbase = (uintptr_t)a.src, gend = gbase + (uintptr_t)a.src_bytes;
    const uintptr_t img_base = gbase + (uintptr_t)d.off[0] + 3 * (uintptr_t)xs;
    if (wave == 0 && live) {
        const uintptr_t r0 = img_base + (uintptr_t)t.x0 * (uintptr_t)d.pitch;
        const uintptr_t r1 = img_base + (uintptr_t)t.x1 * (uintptr_t)d.pitch;
        v.rowa0[lane] = slot0 + s0 * a.slot_bytes + (int)(r0 & 15);
        v.rowa1[lane] = slot0 + s1 * a.slot_bytes + (int)(r1 & 15);
        v.twy[lane] = t.w;
    }

    // Gathers: slot k is staged by wave k % 4.
    int issued = 0;
    int slot = 0;
    for (int r = 0; r < r_cnt; ++r) {
        for (int h = 0; h < 2; ++h) {
            const unsigned long long m = h ? m1 : m0;
            if (!((m >> r) & 1ull))
                continue;
            if (slot % kWavesPerGroup == wave) {
                const int y = __builtin_amdgcn_readlane(h ? t.x1 : t.x0, r);
                const uintptr_t row = img_base + (uintptr_t)y * (uintptr_t)d.pitch;
                const uintptr_t al = row & ~(uintptr_t)15;
                const int nch = (int)((row - al + (uintptr_t)span_bytes + 15) >> 4);
                if (issued >= 0 && al >= gbase && al + 16 * (uintptr_t)nch <= gend)
                    issued += (nch + 63) >> 6;
                else
                    issued = -1;
                stage_row(lds + slot0 + slot * a.slot_bytes, row, span_bytes, gbase, gend,
                          lane);
            }
            ++slot;
        }
    }
    return issued;
}

// Interpolate item w out of buffer `bi` and store it. Threads take pairs of
// adjacent pixels of the band; the band's output rows are contiguous in every
// plane (pixel p of the band lands at element r_begin * Cw + p), so each pair
// is one 32-bit (fp16) or 64-bit (fp32) store per plane. Returns the number
// of pair iterations this wave ran (each issues at least three stores).
template <int F16>
__device__ __forceinline__ int interpolate(const BatchArgs &a, long long w, int bi, uint8_t *lds,
                                           int tid)
{
    const int Cw = a.Cw, R = a.R;
    const int img = (int)(w / a.bands);
    const int band = (int)(w - (long long)img * a.bands);
    const BufView v = buf_view(lds + bi * a.stage_bytes, Cw, R);
    const int r_begin = band * R;
    const int npx = min(R, a.Ch - r_begin) * Cw;
    const long long plane = (long long)a.Ch * Cw;
    const long long out_band = (long long)(a.img_base + img) * 3 * plane + (long long)r_begin * Cw;
    const int step = 2 * kThreads;
    const int step_r = step / Cw, step_c = step - step_r * Cw;
    const int first = 2 * (tid & ~63);  // first pixel of this wave
    const int iters = npx > first ? (npx - first + step - 1) / step : 0;
    int r = (2 * tid) / Cw;
    int c = 2 * tid - r * Cw;
    for (int p0 = 2 * tid; p0 < npx; p0 += step) {
        float o[3][2];
        int rr = r, cc = c;
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            if (j == 1) {
                if (p0 + 1 >= npx) {
                    o[0][1] = o[1][1] = o[2][1] = 0.0f;
                    break;
                }
                if (++cc == Cw) {
                    cc = 0;
                    ++rr;
                }
            }
            const int xo = v.colx[cc];
            const float wx = v.colw[cc];
            const float wy = v.twy[rr];
            float p[6], q[6];
            lds_pixel_pair(lds, v.rowa0[rr] + xo, p);
            lds_pixel_pair(lds, v.rowa1[rr] + xo, q);
#pragma unroll
            for (int ch = 0; ch < 3; ++ch) {
                const float t = lerp(p[ch], p[ch + 3], wx);
                const float b = lerp(q[ch], q[ch + 3], wx);
                o[ch][j] = normalize(lerp(t, b, wy), a.mean[ch], a.stdv[ch], a.rcp[ch]);
            }
        }
        const int valid = min(2, npx - p0);
#pragma unroll
        for (int ch = 0; ch < 3; ++ch)
            store2<F16>(a.out, out_band + ch * plane + p0, o[ch], valid);
        c += step_c;
        r += step_r;
        if (c >= Cw) {
            c -= Cw;
            ++r;
        }
    }
    return iters;
}

template <int F16>
__global__ void __launch_bounds__(kThreads) rgb_lds_kernel(BatchArgs a)
{
    extern __shared__ __attribute__((aligned(16))) uint8_t lds[];
    const int tid = threadIdx.x;
    const long long total = (long long)a.n * a.bands;
    const long long w_begin = total * blockIdx.x / gridDim.x;
    const long long w_end = total * (blockIdx.x + 1) / gridDim.x;
    const int items = (int)(w_end - w_begin);
    Geo held0 = {-1, -1, -1}, held1 = {-1, -1, -1};  // geometry of each buffer's column taps
    if (items > 0)
        prepare(a, w_begin, 0, lds, held0, tid);
    int stores_after = 0;  // lower bound on vector-memory ops issued after item k's gathers
    for (int k = 0; k < items; ++k) {
        wait_vmcnt(min(stores_after, 63));
        barrier_lds();
        int after = 0;
        if (k + 1 < items) {
            if ((k + 1) & 1)
                after = prepare(a, w_begin + k + 1, 1, lds, held1, tid);
            else
                after = prepare(a, w_begin + k + 1, 0, lds, held0, tid);
        }
        const int iters = interpolate<F16>(a, w_begin + k, k & 1, lds, tid);
        // Item k+1's gathers are followed by at least 3 * iters stores; if a
        // row needed byte copies, wait for everything.
        stores_after = after < 0 ? 0 : 3 * iters;
    }
}

// ---------------------------------------------------------------------------
// RGB, register gather, persistent and software-pipelined.
//
// The output of one image is Ch x Cw pixels per plane; a "pass" is the next
// kPassPx of them in row-major order (pixel p is element p of every plane).
// Work items are (image, pass), image-major; workgroup g takes the
// contiguous range [g*T/G, (g+1)*T/G) of the T items.
//
// LDS holds the taps of the current image geometry: per output column the
// byte offset 3*x0 and weight, per output row the byte offsets of rows y0,
// y1 and the weight. They are rebuilt only when the geometry changes (never,
// in a batch of equal images).
//
// Per pass each thread takes kPairs pairs of adjacent output pixels. For each
// pixel it loads the 8 source bytes at pixel x0 of rows y0 and y1 (one
// unaligned load each; x0 and x0 + 1 sit at fixed byte positions). The loads
// of pass j+1 go into the other of two register sets before pass j is
// interpolated, so a pass's source bytes are in flight while the previous
// one computes; vector-memory operations complete in issue order, so the
// waits before using a set do not wait for the newer one. Overlapping
// windows of neighbouring lanes share cache lines, so HBM sees each touched
// line once. The host routes any image whose windows could reach past the
// end of the source buffer to the direct-gather kernel instead.
// ---------------------------------------------------------------------------
constexpr int kPairs = 4;                       // pixel pairs per thread per pass
constexpr int kPassPx = 2 * kPairs * kThreads;  // output pixels per pass

// Pixel x0 (bytes 0..2) and x0 + 1 (bytes 3..5) of an 8-byte window.
__device__ __forceinline__ void unpack_pair(uint64_t v, float (&p)[6])
{
    const uint32_t lo = (uint32_t)v, hi = (uint32_t)(v >> 32);
    p[0] = (float)(lo & 0xffu);
    p[1] = (float)((lo >> 8) & 0xffu);
    p[2] = (float)((lo >> 16) & 0xffu);
    p[3] = (float)(lo >> 24);
    p[4] = (float)(hi & 0xffu);
    p[5] = (float)((hi >> 8) & 0xffu);
}

struct GatherTabs {
    const int *colx;               // 3 * x0 per output column
    const float *colw;             // weight per output column
    const long long *row0, *row1;  // byte offsets of rows y0, y1 per output row
    const float *twy;              // weight per output row
};

typedef uint64_t PassRegs[kPairs][4];  // per pair: px0 row0, px0 row1, px1 row0, px1 row1

// Output pixel (row, column) of pair k's first pixel in a pass, and of its
// second pixel (which may wrap to the next row). Pixels beyond the image map
// to pixel 0 (loaded but never stored).
struct PairPos {
    int r0, c0, r1, c1;
};

__device__ __forceinline__ void pass_positions(PairPos (&pos)[kPairs], int Cw, int npx,
                                               int pass_px, int tid)
{
    const int p_first = pass_px + 2 * tid;
    int r = p_first / Cw;
    int c = p_first - r * Cw;
    const int step = 2 * kThreads;
    const int step_r = step / Cw, step_c = step - step_r * Cw;
#pragma unroll
    for (int k = 0; k < kPairs; ++k) {
        const int p0 = p_first + k * step;
        const bool in0 = p0 < npx, in1 = p0 + 1 < npx;
        const bool wrap = c + 1 == Cw;
        pos[k].r0 = in0 ? r : 0;
        pos[k].c0 = in0 ? c : 0;
        pos[k].r1 = in1 ? (wrap ? r + 1 : r) : 0;
        pos[k].c1 = in1 ? (wrap ? 0 : c + 1) : 0;
        c += step_c;
        r += step_r;
        if (c >= Cw) {
            c -= Cw;
            ++r;
        }
    }
}

__device__ __forceinline__ uint64_t load8(const uint8_t *p)
{
    uint64_t v;
    __builtin_memcpy(&v, p, 8);  // one unaligned global_load_dwordx2
    return v;
}

__device__ __forceinline__ void load_pass(PassRegs &v, const GatherTabs &T, const uint8_t *base,
                                          int Cw, int npx, int pass_px, int tid)
{
    PairPos pos[kPairs];
    pass_positions(pos, Cw, npx, pass_px, tid);
#pragma unroll
    for (int k = 0; k < kPairs; ++k) {
        const uint8_t *q0 = base + T.colx[pos[k].c0];
        const uint8_t *q1 = base + T.colx[pos[k].c1];
        v[k][0] = load8(q0 + T.row0[pos[k].r0]);
        v[k][1] = load8(q0 + T.row1[pos[k].r0]);
        v[k][2] = load8(q1 + T.row0[pos[k].r1]);
        v[k][3] = load8(q1 + T.row1[pos[k].r1]);
    }
}

template <int F16>
__device__ __forceinline__ void compute_pass(const PassRegs &v, const GatherTabs &T,
                                             const BatchArgs &a, long long out_img, int npx,
                                             int pass_px, int tid)
{
    PairPos pos[kPairs];
    pass_positions(pos, a.Cw, npx, pass_px, tid);
    const int p_first = pass_px + 2 * tid;
#pragma unroll
    for (int k = 0; k < kPairs; ++k) {
        const int p0 = p_first + k * 2 * kThreads;
        if (p0 >= npx)
            break;
        const int valid = min(2, npx - p0);
        float o[3][2];
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            const float wx = T.colw[j ? pos[k].c1 : pos[k].c0];
            const float wy = T.twy[j ? pos[k].r1 : pos[k].r0];
            float p[6], q[6];
            unpack_pair(v[k][2 * j], p);
            unpack_pair(v[k][2 * j + 1], q);
#pragma unroll
            for (int ch = 0; ch < 3; ++ch) {
                const float t = lerp(p[ch], p[ch + 3], wx);
                const float b = lerp(q[ch], q[ch + 3], wx);
                o[ch][j] = normalize(lerp(t, b, wy), a.mean[ch], a.stdv[ch], a.rcp[ch]);
            }
        }
#pragma unroll
        for (int ch = 0; ch < 3; ++ch)
            store2<F16>(a.out, out_img + ch * (long long)npx + p0, o[ch], valid);
    }
}

// The fields of an image the gather kernel uses, as plain scalars (a copy of
// the 80-byte descriptor would not stay in registers across the loop).
struct ImgGeo {
    long long off;
    int W, H, pitch, Wr, Hr, left, top;
};

__device__ __forceinline__ ImgGeo image_geo(const BatchArgs &a, int img)
{
    ImgGeo g;
    if (a.table) {
        const Desc *t = a.table + img;
        g.off = t->off[0];
        g.W = t->W;
        g.H = t->H;
        g.pitch = t->pitch;
        g.Wr = t->Wr;
        g.Hr = t->Hr;
        g.left = t->left;
        g.top = t->top;
    } else {
        g.off = a.uni.off[0] + (long long)img * a.stride;
        g.W = a.uni.W;
        g.H = a.uni.H;
        g.pitch = a.uni.pitch;
        g.Wr = a.uni.Wr;
        g.Hr = a.uni.Hr;
        g.left = a.uni.left;
        g.top = a.uni.top;
    }
    return g;
}

// Fill the tap tables for the geometry of image d (all threads; caller syncs).
__device__ __forceinline__ void build_tabs(uint8_t *lds, const BatchArgs &a, const ImgGeo &d,
                                           int tid)
{
    const int Cw = a.Cw, Ch = a.Ch;
    int *colx = (int *)lds;
    float *colw = (float *)(colx + Cw);
    long long *row0 = (long long *)(lds + a.slots_off);
    long long *row1 = row0 + Ch;
    float *twy = (float *)(row1 + Ch);
    for (int c = tid; c < Cw; c += kThreads) {
        const Tap t = axis_tap(d.left + c, d.W, d.Wr);
        colx[c] = 3 * t.x0;
        colw[c] = t.w;
    }
    for (int r = tid; r < Ch; r += kThreads) {
        const Tap t = axis_tap(d.top + r, d.H, d.Hr);
        row0[r] = (long long)t.x0 * d.pitch;
        row1[r] = (long long)t.x1 * d.pitch;
        twy[r] = t.w;
    }
}

__device__ __forceinline__ bool same_geometry(const ImgGeo &x, const ImgGeo &y)
{
    return x.W == y.W && x.H == y.H && x.pitch == y.pitch && x.Wr == y.Wr && x.Hr == y.Hr &&
           x.left == y.left && x.top == y.top;
}

template <int F16>
__global__ void __launch_bounds__(kThreads) rgb_gather_kernel(BatchArgs a)
{
    extern __shared__ __attribute__((aligned(16))) uint8_t lds[];
    const int tid = threadIdx.x;
    const int Cw = a.Cw;
    const int npx = a.Ch * Cw;
    const int passes = (npx + kPassPx - 1) / kPassPx;  // per image
    const long long total = (long long)a.n * passes;
    const long long w_begin = total * blockIdx.x / gridDim.x;
    const long long w_end = total * (blockIdx.x + 1) / gridDim.x;
    if (w_begin >= w_end)
        return;

    GatherTabs T;
    T.colx = (const int *)lds;
    T.colw = (const float *)(T.colx + Cw);
    T.row0 = (const long long *)(lds + a.slots_off);
    T.row1 = T.row0 + a.Ch;
    T.twy = (const float *)(T.row1 + a.Ch);

    PassRegs A, B;
    long long w = w_begin;
    int img = (int)(w / passes);
    ImgGeo d = image_geo(a, img);
    build_tabs(lds, a, d, tid);
    __syncthreads();
    int pass_px = (int)(w - (long long)img * passes) * kPassPx;
    load_pass(A, T, a.src + d.off, Cw, npx, pass_px, tid);

    // One step computes the current set and prefetches the next item into
    // the other; two steps per trip so the sets alternate without copies.
#define SMOL_GATHER_STEP(CUR, NXT)                                                            \
    {                                                                                         \
        const long long wn = w + 1;                                                           \
        const bool more = wn < w_end;                                                         \
        int nimg = img, npass = 0;                                                            \
        ImgGeo dn = d;                                                                        \
        bool pre = false;                                                                     \
        if (more) {                                                                           \
            nimg = (int)(wn / passes);                                                        \
            npass = (int)(wn - (long long)nimg * passes) * kPassPx;                           \
            if (nimg != img)                                                                  \
                dn = image_geo(a, nimg);                                                      \
            pre = same_geometry(dn, d);                                                       \
            if (pre)                                                                          \
                load_pass(NXT, T, a.src + dn.off, Cw, npx, npass, tid);                       \
        }                                                                                     \
        compute_pass<F16>(CUR, T, a, (long long)(a.img_base + img) * 3 * npx, npx, pass_px,   \
                          tid);                                                               \
        if (!more)                                                                            \
            break;                                                                            \
        if (!pre) { /* new geometry: rebuild the tables, then load */                         \
            __syncthreads();                                                                  \
            build_tabs(lds, a, dn, tid);                                                      \
            __syncthreads();                                                                  \
            load_pass(NXT, T, a.src + dn.off, Cw, npx, npass, tid);                           \
        }                                                                                     \
        w = wn;                                                                               \
        img = nimg;                                                                           \
        d = dn;                                                                               \
        pass_px = npass;                                                                      \
    }
    while (true) {
        SMOL_GATHER_STEP(A, B)
        SMOL_GATHER_STEP(B, A)
    }
#undef SMOL_GATHER_STEP
}


// ---------------------------------------------------------------------------
// RGB, direct gather: a workgroup per output row (the image's descriptor and
// the row's vertical taps once per row), a thread per output pixel, taps
// read from global memory. Used for images whose staged rows would cross an
// end of src, NHWC and uint8 outputs, and spans beyond the LDS budgets.
// ---------------------------------------------------------------------------
template <int OUT>
__global__ void __launch_bounds__(kThreads) rgb_direct_kernel(BatchArgs a)
{
    const long long plane = (long long)a.Ch * a.Cw;
    const long long rows = (long long)a.Ch * a.n;
    for (long long row = blockIdx.x; row < rows; row += gridDim.x) {
        const int img = (int)(row / a.Ch);
        const int yc = (int)(row - (long long)img * a.Ch);
        Desc d;
        image_desc(a, img, d);
        const Tap ty = axis_tap(d.top + yc, d.H, d.Hr);
        const uint8_t *r0 = a.src + d.off[0] + (long long)ty.x0 * d.pitch;
        const uint8_t *r1 = a.src + d.off[0] + (long long)ty.x1 * d.pitch;
        const long long ibase = (long long)(a.img_base + img) * 3 * plane;
        const long long pix0 = (long long)yc * a.Cw;  // first pixel of the row in the crop
        for (int xc = threadIdx.x; xc < a.Cw; xc += blockDim.x) {
            const Tap tx = axis_tap(d.left + xc, d.W, d.Wr);
            // element of channel ch: NCHW base + ch * plane, NHWC base + ch
            const long long base = ibase + (a.nhwc ? 3 * (pix0 + xc) : pix0 + xc);
            const long long cstep = a.nhwc ? 1 : plane;
#pragma unroll
            for (int ch = 0; ch < 3; ++ch) {
                const float p00 = r0[3 * tx.x0 + ch], p01 = r0[3 * tx.x1 + ch];
                const float p10 = r1[3 * tx.x0 + ch], p11 = r1[3 * tx.x1 + ch];
                const float v = lerp(lerp(p00, p01, tx.w), lerp(p10, p11, tx.w), ty.w);
                emit1<OUT>(a, base + ch * cstep, ch, v);
            }
        }
    }
}

// ---------------------------------------------------------------------------
// I420, direct gather: converts at each of the four luma taps, then resizes.
// ---------------------------------------------------------------------------
__device__ __forceinline__ float chroma_at(const uint8_t *pl, int Wc, const Tap &cx, const Tap &cy)
{
    const uint8_t *r0 = pl + (long long)cy.x0 * Wc;
    const uint8_t *r1 = pl + (long long)cy.x1 * Wc;
    const float t = lerp((float)r0[cx.x0], (float)r0[cx.x1], cx.w);
    const float b = lerp((float)r1[cx.x0], (float)r1[cx.x1], cx.w);
    return lerp(t, b, cy.w);
}

template <int OUT>
__global__ void __launch_bounds__(kThreads) yuv_direct_kernel(BatchArgs a)
{
    const long long plane = (long long)a.Ch * a.Cw;
    const long long rows = (long long)a.Ch * a.n;
    for (long long row = blockIdx.x; row < rows; row += gridDim.x) {
        const int img = (int)(row / a.Ch);
        const int yc = (int)(row - (long long)img * a.Ch);
        Desc d;
        image_desc(a, img, d);
        // the region (d.W x d.H at (rx, ry)) inside a frame of pitch x fh;
        // chroma taps in frame coordinates
        const int Wc = (d.pitch + 1) >> 1, Hc = (d.fh + 1) >> 1;
        const uint8_t *yp = a.src + d.off[0] + (long long)d.ry * d.pitch + d.rx;
        const uint8_t *cbp = a.src + d.off[1];
        const uint8_t *crp = a.src + d.off[2];
        const Tap ty = axis_tap(d.top + yc, d.H, d.Hr);
        const int yy[2] = {ty.x0, ty.x1};
        const Tap cy[2] = {chroma_tap(d.ry + yy[0], Hc), chroma_tap(d.ry + yy[1], Hc)};
        const long long ibase = (long long)(a.img_base + img) * 3 * plane;
        const long long pix0 = (long long)yc * a.Cw;  // first pixel of the row in the crop
        for (int xc = threadIdx.x; xc < a.Cw; xc += blockDim.x) {
            const Tap tx = axis_tap(d.left + xc, d.W, d.Wr);
            const int xx[2] = {tx.x0, tx.x1};
            float rgb[2][2][3];
#pragma unroll
            for (int i = 0; i < 2; ++i) {
#pragma unroll
                for (int k = 0; k < 2; ++k) {
                    const Tap cx = chroma_tap(d.rx + xx[k], Wc, a.siting);
                    const float Y = (float)yp[(long long)yy[i] * d.pitch + xx[k]];
                    ycbcr_to_rgb(Y, chroma_at(cbp, Wc, cx, cy[i]), chroma_at(crp, Wc, cx, cy[i]),
                                 rgb[i][k][0], rgb[i][k][1], rgb[i][k][2]);
                }
            }
            const long long base = ibase + (a.nhwc ? 3 * (pix0 + xc) : pix0 + xc);
            const long long cstep = a.nhwc ? 1 : plane;
#pragma unroll
            for (int ch = 0; ch < 3; ++ch) {
                const float v = lerp(lerp(rgb[0][0][ch], rgb[0][1][ch], tx.w),
                                     lerp(rgb[1][0][ch], rgb[1][1][ch], tx.w), ty.w);
                emit1<OUT>(a, base + ch * cstep, ch, v);
            }
        }
    }
}

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// A ragged batch's descriptor table, 16 bytes per thread, from the pinned
// staging slot (read over the bus) to device memory.
__global__ void __launch_bounds__(kThreads) table_copy_kernel(const u32x4 *src, u32x4 *dst, int n)
{
    for (int i = blockIdx.x * kThreads + threadIdx.x; i < n; i += gridDim.x * kThreads)
        dst[i] = src[i];
}

// Direct kernels: a workgroup per output row, 64 to 256 threads (whole
// waves covering the crop's width where it is narrower than 256), at most
// 2^20 workgroups looping over the rows.
dim3 direct_grid(const BatchArgs &a)
{
    const long long rows = (long long)a.Ch * a.n;
    const long long cap = 1 << 20;
    return dim3((unsigned)(rows < cap ? rows : cap));
}

dim3 direct_block(const BatchArgs &a)
{
    const int waves = (a.Cw + 63) / 64;
    return dim3(64 * (waves < kThreads / 64 ? waves : kThreads / 64));
}

// Launches `kernel` with its one argument `a`. `done`, when not null, is an
// event that the launch signals at the kernel's completion: it rides on the
// dispatch itself, with no event packet of its own behind the kernel (such a
// packet holds the queue about 5 us before the next dispatch).
int launch_one(const void *kernel, dim3 grid, dim3 block, size_t lds, const BatchArgs &a,
               void *stream, void *done)
{
    void *args[] = {(void *)&a};
    return (int)hipExtLaunchKernel(kernel, grid, block, args, lds, (hipStream_t)stream, nullptr,
                                   (hipEvent_t)done, 0);
}

}  // namespace

int launch_table_copy(const void *src, void *dst, size_t bytes, void *stream)
{
    const int n = (int)(bytes / 16);
    const dim3 grid((unsigned)std::min(64, (n + kThreads - 1) / kThreads)), block(kThreads);
    hipLaunchKernelGGL(table_copy_kernel, grid, block, 0, (hipStream_t)stream,
                       (const u32x4 *)src, (u32x4 *)dst, n);
    return (int)hipGetLastError();
}

int launch_rgb_direct(const BatchArgs &a, int out_type, void *stream, void *done)
{
    const void *k = out_type == 2   ? (const void *)rgb_direct_kernel<2>
                    : out_type == 1 ? (const void *)rgb_direct_kernel<1>
                                    : (const void *)rgb_direct_kernel<0>;
    return launch_one(k, direct_grid(a), direct_block(a), 0, a, stream, done);
}

int launch_rgb_lds(const BatchArgs &a, int out_f16, size_t lds_bytes, void *stream, void *done)
{
    const void *k = out_f16 ? (const void *)rgb_lds_kernel<1> : (const void *)rgb_lds_kernel<0>;
    return launch_one(k, dim3((unsigned)a.grid), dim3(kThreads), lds_bytes, a, stream, done);
}

int launch_rgb_gather(const BatchArgs &a, int out_f16, size_t lds_bytes, void *stream, void *done)
{
    const void *k =
        out_f16 ? (const void *)rgb_gather_kernel<1> : (const void *)rgb_gather_kernel<0>;
    return launch_one(k, dim3((unsigned)a.grid), dim3(kThreads), lds_bytes, a, stream, done);
}

// f16: the output type, 0 fp32, 1 fp16, 2 uint8 (contiguous ranges only)
const void *rows_kernel(const BatchArgs &a, int f16)
{
    if (f16 == 2)
        return a.nhwc ? rows_rgb_u8_range_nhwc(a) : rows_rgb_u8_range(a);
    if (a.nhwc)
        return f16 ? (a.interleave ? rows_rgb_f16_stride_nhwc(a) : rows_rgb_f16_range_nhwc(a))
                   : (a.interleave ? rows_rgb_f32_stride_nhwc(a) : rows_rgb_f32_range_nhwc(a));
    return f16 ? (a.interleave ? rows_rgb_f16_stride(a) : rows_rgb_f16_range(a))
               : (a.interleave ? rows_rgb_f32_stride(a) : rows_rgb_f32_range(a));
}

int launch_rgb_rows(const BatchArgs &a, int out_f16, size_t lds_bytes, void *stream, void *done)
{
    return launch_one(rows_kernel(a, out_f16), dim3((unsigned)(a.grid / a.wpg)), dim3(64 * a.wpg),
                      lds_bytes * a.wpg, a, stream, done);
}

// Resident workgroups per compute unit of a kernel at a block size and LDS
// size, queried once per device and remembered (the query costs more than
// the rest of a call's host work).
static int occupancy(const void *fn, int block, size_t lds, int *blocks_per_cu)
{
    static std::mutex mu;
    static std::map<std::tuple<int, const void *, int, size_t>, int> cache;
    int device = 0;
    hipError_t e = hipGetDevice(&device);
    if (e != hipSuccess)
        return (int)e;
    const auto key = std::make_tuple(device, fn, block, lds);
    {
        std::lock_guard<std::mutex> lk(mu);
        const auto it = cache.find(key);
        if (it != cache.end()) {
            *blocks_per_cu = it->second;
            return (int)hipSuccess;
        }
    }
    e = hipOccupancyMaxActiveBlocksPerMultiprocessor(blocks_per_cu, fn, block, lds);
    if (e == hipSuccess) {
        std::lock_guard<std::mutex> lk(mu);
        cache[key] = *blocks_per_cu;
    }
    return (int)e;
}

int occupancy_rgb_rows(const BatchArgs &a, int out_f16, size_t lds_bytes, int *blocks_per_cu)
{
    return occupancy(rows_kernel(a, out_f16), 64 * a.wpg, lds_bytes * a.wpg, blocks_per_cu);
}

int occupancy_rgb_gather(int out_f16, size_t lds_bytes, int *blocks_per_cu)
{
    return occupancy(out_f16 ? (const void *)rgb_gather_kernel<1> : (const void *)rgb_gather_kernel<0>,
                     kThreads, lds_bytes, blocks_per_cu);
}

int occupancy_rgb_lds(int out_f16, size_t lds_bytes, int *blocks_per_cu)
{
    return occupancy(out_f16 ? (const void *)rgb_lds_kernel<1> : (const void *)rgb_lds_kernel<0>,
                     kThreads, lds_bytes, blocks_per_cu);
}

int launch_yuv_direct(const BatchArgs &a, int out_type, void *stream, void *done)
{
    const void *k = out_type == 2   ? (const void *)yuv_direct_kernel<2>
                    : out_type == 1 ? (const void *)yuv_direct_kernel<1>
                                    : (const void *)yuv_direct_kernel<0>;
    return launch_one(k, direct_grid(a), direct_block(a), 0, a, stream, done);
}

const void *yuv_rows_kernel_for(const BatchArgs &a, int f16)
{
    if (a.nhwc)
        return a.interleave ? rows_yuv_stride_nhwc(a, f16) : rows_yuv_range_nhwc(a, f16);
    return a.interleave ? rows_yuv_stride(a, f16) : rows_yuv_range(a, f16);
}

// LDS bytes of the column table that the waves of an I420 row-streaming
// workgroup share when the batch is uniform (no descriptor table) and the
// group has more than one wave: 32 bytes per lane and pixel of the lane's
// 2 J columns (the kernel's yuv_col_table_bytes).
static size_t yuv_rows_table_lds(const BatchArgs &a, bool uniform)
{
    const size_t J = a.col_iters <= 1 ? 1 : a.col_iters <= 2 ? 2 : 4;
    return uniform && a.wpg > 1 ? 2 * J * 64 * 32 : 0;
}

int launch_yuv_rows(const BatchArgs &a, int out_f16, size_t lds_bytes, void *stream, void *done)
{
    return launch_one(yuv_rows_kernel_for(a, out_f16), dim3((unsigned)(a.grid / a.wpg)),
                      dim3(64 * a.wpg), lds_bytes * a.wpg + yuv_rows_table_lds(a, !a.table), a,
                      stream, done);
}

int occupancy_yuv_rows(const BatchArgs &a, int out_f16, size_t lds_bytes, int *blocks_per_cu)
{
    // queried before the batch's table is known: counts the shared table
    return occupancy(yuv_rows_kernel_for(a, out_f16), 64 * a.wpg,
                     lds_bytes * a.wpg + yuv_rows_table_lds(a, true), blocks_per_cu);
}

}  // namespace smol
