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
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "smol_internal.h"

namespace smol {
namespace {

constexpr int kThreads = 256;


struct Tap {
    int x0, x1;
    float w;
};

// Half-pixel map of output index x (resized length `out`) onto the source
// (length `in`): u = ((2x + 1) * in - out) / (2 * out), clamped to
// [0, in - 1]; taps floor(u), floor(u) + 1 and weight u - floor(u).
// num < 2^39 and den < 2^23 are exact doubles and a non-integer quotient is at
// least 1/den from the next integer, far above the quotient's rounding error,
// so truncating the double quotient gives the exact floor.
__device__ __forceinline__ Tap axis_tap(int x, int in, int out)
{
    const long long num = (long long)(2 * x + 1) * in - out;
    const int den = 2 * out;
    Tap t;
    if (num <= 0) {
        t.x0 = 0;
        t.x1 = 0;
        t.w = 0.0f;
        return t;
    }
    const long long q = num < 0x7fffffffLL ? (long long)((unsigned)num / (unsigned)den)
                                           : (long long)((double)num / (double)den);
    if (q >= in - 1) {
        t.x0 = in - 1;
        t.x1 = in - 1;
        t.w = 0.0f;
        return t;
    }
    const int rem = (int)(num - q * den);
    t.x0 = (int)q;
    t.x1 = (int)q + 1;
    t.w = (float)rem / (float)den;  // IEEE division, both operands exact
    return t;
}

// Centred 4:2:0 chroma siting: luma index x samples chroma at
// u = x/2 - 1/4 = (2x - 1)/4, clamped like the luma map; the weight is 1/4 or
// 3/4 in the interior.
__device__ __forceinline__ Tap chroma_tap(int x, int n)
{
    const int num = 2 * x - 1;
    Tap t;
    if (num <= 0) {
        t.x0 = 0;
        t.x1 = 0;
        t.w = 0.0f;
        return t;
    }
    const int q = num >> 2;
    if (q >= n - 1) {
        t.x0 = n - 1;
        t.x1 = n - 1;
        t.w = 0.0f;
        return t;
    }
    t.x0 = q;
    t.x1 = q + 1;
    t.w = (float)(num & 3) * 0.25f;
    return t;
}

// BT.601 full range: Kr = 0.299, Kb = 0.114, Kg = 1 - Kr - Kb; coefficients
// formed in double, rounded once to fp32.
constexpr double kKr = 0.299, kKb = 0.114, kKg = 1.0 - kKr - kKb;
constexpr float kRCr = (float)(2.0 * (1.0 - kKr));
constexpr float kGCb = (float)(2.0 * kKb * (1.0 - kKb) / kKg);
constexpr float kGCr = (float)(2.0 * kKr * (1.0 - kKr) / kKg);
constexpr float kBCb = (float)(2.0 * (1.0 - kKb));

__device__ __forceinline__ float clamp255(float v) { return fminf(fmaxf(v, 0.0f), 255.0f); }

__device__ __forceinline__ void ycbcr_to_rgb(float y, float cb, float cr, float &r, float &g,
                                             float &b)
{
    cb -= 128.0f;
    cr -= 128.0f;
    r = clamp255(y + kRCr * cr);
    g = clamp255((y - kGCb * cb) - kGCr * cr);
    b = clamp255(y + kBCb * cb);
}

__device__ __forceinline__ float lerp(float a, float b, float w) { return a + w * (b - a); }

__device__ __forceinline__ float normalize(float v, float mean, float stdv, float rcp)
{
    const float a = v - mean;
    const float q0 = a * rcp;
    return fmaf(fmaf(-stdv, q0, a), rcp, q0);
}

__device__ __forceinline__ uint32_t f16_bits(float v)
{
    // The output is RNE-to-fp16 of the *fp32* result. Without this barrier
    // the compiler folds the final FMA of the normalisation into the
    // narrowing (v_fma_mix*_f16), rounding once from the exact value instead.
    asm volatile("" : "+v"(v));
    _Float16 h = (_Float16)v;  // round to nearest even (MODE default)
    return (uint32_t)__builtin_bit_cast(uint16_t, h);
}

// Store 2 consecutive outputs starting at element index idx of one plane.
template <int F16>
__device__ __forceinline__ void store2(void *out, long long idx, const float (&v)[2], int valid)
{
    if (F16) {
        uint16_t *o = (uint16_t *)out + idx;
        if (valid == 2 && (idx & 1) == 0) {
            __builtin_nontemporal_store(f16_bits(v[0]) | (f16_bits(v[1]) << 16), (uint32_t *)o);
        } else {
            o[0] = (uint16_t)f16_bits(v[0]);
            if (valid == 2)
                o[1] = (uint16_t)f16_bits(v[1]);
        }
    } else {
        float *o = (float *)out + idx;
        if (valid == 2 && (idx & 1) == 0) {
            typedef float f32x2 __attribute__((ext_vector_type(2)));
            const f32x2 w = {v[0], v[1]};
            __builtin_nontemporal_store(w, (f32x2 *)o);
        } else {
            o[0] = v[0];
            if (valid == 2)
                o[1] = v[1];
        }
    }
}

template <int F16>
__device__ __forceinline__ void store1(void *out, long long idx, float v)
{
    if (F16)
        ((uint16_t *)out)[idx] = (uint16_t)f16_bits(v);
    else
        ((float *)out)[idx] = v;
}

__device__ __forceinline__ void image_desc(const BatchArgs &a, int img, Desc &d)
{
    if (a.table) {
        d = a.table[img];
    } else {
        d = a.uni;
        d.off[0] += (long long)img * a.stride;
        d.off[1] += (long long)img * a.stride;
        d.off[2] += (long long)img * a.stride;
    }
}

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
// the 64-byte descriptor would not stay in registers across the loop).
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
// RGB, row streaming: one wave per workgroup, no barriers.
//
// Work items are output rows (image, row), image-major; wave g takes the
// contiguous range [g*T/G, (g+1)*T/G) of the T rows. For each output row the
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
// arithmetic (the numerator grows by 2*H per output row): no division per
// row but the one for the weight.
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

// Vertical half-pixel map of output rows rr, rr + 1, ... of one image:
// num = (2 * (top + rr) + 1) * H - Hr, den = 2 * Hr, q = floor(num / den),
// rem = num - q * den; num <= 0 exactly when q < 0 or q == rem == 0.
struct VCursor {
    int q, rem, den, qs, rs, H;
};

__device__ __forceinline__ void vcursor_init(VCursor &v, const RowImg &g, int rr)
{
    v.H = g.H;
    v.den = 2 * g.Hr;
    const long long n = (long long)(2 * (g.top + rr) + 1) * g.H - g.Hr;
    // floor division (num may be negative near the top edge, down to -Hr)
    const long long q = n >= 0 ? n / v.den : -((-n + v.den - 1) / v.den);
    v.q = (int)q;
    v.rem = (int)(n - q * v.den);
    v.qs = (2 * g.H) / v.den;
    v.rs = 2 * g.H - v.qs * v.den;
}

__device__ __forceinline__ void vcursor_next(VCursor &v)
{
    v.q += v.qs;
    v.rem += v.rs;
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

template <int J>
__device__ __forceinline__ void row_taps(const RowImg &g, const int Cw, int (&cx)[J][2],
                                         float (&cw)[J][2], int lane)
{
#pragma unroll
    for (int j = 0; j < J; ++j)
#pragma unroll
        for (int px = 0; px < 2; ++px) {
            const int c = 2 * lane + 128 * j + px;
            cx[j][px] = 0;
            cw[j][px] = 0.0f;
            if (c < Cw) {
                const Tap t = axis_tap(g.left + c, g.W, g.Wr);
                cx[j][px] = 3 * (t.x0 - g.xf);
                cw[j][px] = t.w;
            }
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


typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// One output row's two source rows in registers (G chunk loads each), with
// the offset of each row's first byte in its first chunk and the vertical
// weight.
template <int G>
struct StagedRows {
    u32x4 c0[G], c1[G];
    int sh0, sh1;
    float wy;
};

// Row cursor: image, crop row, vertical map and the image's row addressing.
struct RowCursor {
    int img, rr;
    VCursor v;
    uintptr_t base;  // first staged byte of source row 0
    int pitch, span;
};

__device__ __forceinline__ void cursor_image(RowCursor &c, const BatchArgs &a, int img, int rr)
{
    const RowImg g = row_img(a, img);
    c.img = img;
    c.rr = rr;
    vcursor_init(c.v, g, rr);
    c.base = (uintptr_t)(a.src + g.off) + 3 * (uintptr_t)g.xf;
    c.pitch = g.pitch;
    c.span = g.span;
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

__device__ __forceinline__ void cursor_next(RowCursor &c, const BatchArgs &a)
{
    vcursor_next(c.v);
    if (++c.rr == a.Ch && c.img + 1 < a.n)
        cursor_image(c, a, c.img + 1, 0);
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
#undef SMOL_RD3

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

// Interpolate, normalise and store one output row from its staged rows
// (row 0 at byte `row0` of lds, row 1 at `row1`, both including the offset
// of the first byte in its chunk).
template <int F16, int J, int EXACT>
__device__ __forceinline__ void rows_compute(const BatchArgs &a, const NormK &nk, uint8_t *orow,
                                             uint32_t row0, uint32_t row1, float wy,
                                             const int (&cx)[J][2], const float (&cw)[J][2],
                                             int lane)
{
    const int Cw = a.Cw;
    constexpr int kEsz = F16 ? 2 : 4;
    const long long plane = (long long)a.Ch * Cw * kEsz;
    const bool pairs = (Cw & 1) == 0;  // every pair is whole and 2-element aligned
    // tap pairs, 4 per column iteration: pixel c and c + 1 of row 0, then row 1
    // (lanes past the crop read column 0 and store nothing)
    constexpr int kN = J == 1 ? 4 : 8;
    uint64_t v[J * 4];
#pragma unroll
    for (int j0 = 0; j0 < J; j0 += kN / 4)
        read_taps<J, kN>(row0, row1, cx, j0, *(uint64_t(*)[kN]) & v[4 * j0]);
#pragma unroll
    for (int j = 0; j < J; ++j) {
        const int c = 2 * lane + 128 * j;
        if (c < Cw) {
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
                    o[ch][px] = normalize_k<EXACT>(nk, ch, lerp(top, bot, wy));
                }
            }
            const uint32_t lo = (uint32_t)c * kEsz;
            if (pairs) {
#pragma unroll
                for (int ch = 0; ch < 3; ++ch) {
                    uint8_t *dst = orow + ch * plane + lo;
                    if (F16 && !EXACT) {
                        // The conversion may fuse with the last product (one
                        // rounding to fp16 instead of two).
                        typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));
                        const f16x2 h = {(_Float16)o[ch][0], (_Float16)o[ch][1]};
                        __builtin_nontemporal_store(__builtin_bit_cast(uint32_t, h),
                                                    (uint32_t *)dst);
                    } else if (F16) {
                        __builtin_nontemporal_store(f16_bits(o[ch][0]) | (f16_bits(o[ch][1]) << 16),
                                                    (uint32_t *)dst);
                    } else {
                        typedef float f32x2 __attribute__((ext_vector_type(2)));
                        const f32x2 w = {o[ch][0], o[ch][1]};
                        __builtin_nontemporal_store(w, (f32x2 *)dst);
                    }
                }
            } else {
                const bool second = c + 1 < Cw;
#pragma unroll
                for (int ch = 0; ch < 3; ++ch) {
                    uint8_t *dst = orow + ch * plane + lo;
                    if (F16) {
                        ((uint16_t *)dst)[0] = (uint16_t)f16_bits(o[ch][0]);
                        if (second)
                            ((uint16_t *)dst)[1] = (uint16_t)f16_bits(o[ch][1]);
                    } else {
                        ((float *)dst)[0] = o[ch][0];
                        if (second)
                            ((float *)dst)[1] = o[ch][1];
                    }
                }
            }
        }
    }
}

template <int F16, int J, int EXACT, int G, int P>
__global__ void __launch_bounds__(64) rgb_rows_kernel(BatchArgs a)
{
    extern __shared__ __attribute__((aligned(16))) uint8_t lds[];
    const int lane = threadIdx.x;
    const int Ch = a.Ch;
    const long long T = (long long)a.n * Ch;
    const long long r_begin = T * blockIdx.x / gridDim.x;
    const long long r_end = T * (blockIdx.x + 1) / gridDim.x;
    if (r_begin >= r_end)
        return;
    constexpr int kEsz = F16 ? 2 : 4;
    const int n_rows = (int)(r_end - r_begin);
    const int img0 = (int)(r_begin / Ch);
    const int rr0 = (int)(r_begin - (long long)img0 * Ch);

    // Load cursor (the next row to load) and compute state.
    RowCursor lc;
    cursor_image(lc, a, img0, rr0);
    int c_img = img0, c_rr = rr0;
    uint8_t *orow = (uint8_t *)a.out +
                    ((long long)(a.img_base + c_img) * 3 * Ch + c_rr) * (long long)a.Cw * kEsz;
    int cx[J][2];
    float cw[J][2];
    {
        const RowImg g = row_img(a, img0);
        row_taps<J>(g, a.Cw, cx, cw, lane);
    }
    int cW = 0, cWr = 0, cleft = 0;
    {
        const RowImg g = row_img(a, img0);
        cW = g.W;
        cWr = g.Wr;
        cleft = g.left;
    }
    const NormK nk = norm_consts(a);
    const uint32_t lds0 = lds_addr(lds);

    // The load cursor stops at the wave's last row: past the end the loads
    // repeat that row, so every step issues the same loads and the compiler
    // can count exactly what is outstanding when a row is written to LDS.
    int lrow = 0;
    bool at_end = false;  // the cursor sits on the wave's last row, already loaded
    auto advance = [&]() {
        if (lrow + 1 < n_rows) {
            cursor_next(lc, a);
            ++lrow;
        } else {
            at_end = true;
        }
    };
    int k = 0;
    // P = 2: one step loads row k + 2 into FUT, interpolates row k (staged
    // from CUR), writes row k + 1 (in NXT) into the slot; three steps per
    // trip so the register sets rotate without copies. P = 1: one register
    // set, loaded with row k + 1 before row k is interpolated.
    StagedRows<G> A, B, C;
    load_rows<G>(A, lc, lane, false);
    advance();
    if (P == 2) {
        load_rows<G>(B, lc, lane, at_end);
        advance();
    }
    write_rows<G>(lds, A, lane);
    int csh0 = A.sh0, csh1 = A.sh1;
    float cwy = A.wy;
#define SMOL_ROWS_STEP(CUR, NXT, FUT)                                                         \
    {                                                                                         \
        load_rows<G>(FUT, lc, lane, at_end);                                                  \
        advance();                                                                            \
        rows_compute<F16, J, EXACT>(a, nk, orow, lds0 + (uint32_t)csh0,                       \
                                    lds0 + (uint32_t)(1024 * G + csh1), cwy, cx, cw, lane);   \
        if (++k == n_rows)                                                                    \
            break;                                                                            \
        write_rows<G>(lds, NXT, lane);                                                        \
        csh0 = NXT.sh0;                                                                       \
        csh1 = NXT.sh1;                                                                       \
        cwy = NXT.wy;                                                                         \
        orow += (long long)a.Cw * kEsz;                                                       \
        if (++c_rr == Ch) {                                                                   \
            c_rr = 0;                                                                         \
            ++c_img;                                                                          \
            orow += 2 * (long long)Ch * a.Cw * kEsz; /* skip planes 1 and 2 */                \
            const RowImg g = row_img(a, c_img);                                               \
            if (g.W != cW || g.Wr != cWr || g.left != cleft) {                                \
                cW = g.W;                                                                     \
                cWr = g.Wr;                                                                   \
                cleft = g.left;                                                               \
                row_taps<J>(g, a.Cw, cx, cw, lane);                                           \
            }                                                                                 \
        }                                                                                     \
    }
    if (P == 2) {
        while (true) {
            SMOL_ROWS_STEP(A, B, C)
            SMOL_ROWS_STEP(B, C, A)
            SMOL_ROWS_STEP(C, A, B)
        }
    } else {
        while (true)
            SMOL_ROWS_STEP(A, A, A)
    }
#undef SMOL_ROWS_STEP
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
// and normalised. The chroma weights are 0, 1/4 and 3/4, so each chroma
// interpolation step is exact in fp32 (multiples of 1/16 below 256) and a
// fused multiply-add gives the value the separately rounded form gives.
//
// Lane l computes output columns c = 2l + 128j and c + 1 (j < J). Per column
// it keeps: the luma tap (offset of x0 in the staged luma span, weight), and
// for its two luma columns x0, x1 the chroma taps as the offset of the first
// chroma column they read and a byte selector that picks the chroma samples
// (x0's pair, x1's pair) out of the four bytes read there.
// ---------------------------------------------------------------------------
struct YuvImg {
    long long off[3];
    int W, H, Wr, Hr, left, top, xf, span;
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
    } else {
        g.off[0] = a.uni.off[0] + (long long)img * a.stride;
        g.off[1] = a.uni.off[1] + (long long)img * a.stride;
        g.off[2] = a.uni.off[2] + (long long)img * a.stride;
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

// Load cursor over the output rows of I420 frames.
struct YuvCursor {
    int img, rr;
    VCursor v;               // luma vertical map
    uintptr_t base[3];       // first staged byte of row 0 of Y, Cb, Cr
    int W, Wc, Hc, yspan, cspan;
};

__device__ __forceinline__ void yuv_cursor_image(YuvCursor &c, const BatchArgs &a, int img, int rr)
{
    const YuvImg g = yuv_img(a, img);
    c.img = img;
    c.rr = rr;
    VCursor v;
    v.H = g.H;
    v.den = 2 * g.Hr;
    const long long n = (long long)(2 * (g.top + rr) + 1) * g.H - g.Hr;
    const long long q = n >= 0 ? n / v.den : -((-n + v.den - 1) / v.den);
    v.q = (int)q;
    v.rem = (int)(n - q * v.den);
    v.qs = (2 * g.H) / v.den;
    v.rs = 2 * g.H - v.qs * v.den;
    c.v = v;
    c.W = g.W;
    c.Wc = (g.W + 1) >> 1;
    c.Hc = (g.H + 1) >> 1;
    const int xl = g.xf + g.span - 1;
    const int cxf = chroma_tap(g.xf, c.Wc).x0;
    const int cxl = chroma_tap(xl, c.Wc).x1;
    c.yspan = g.span;
    c.cspan = cxl - cxf + 1;
    c.base[0] = (uintptr_t)(a.src + g.off[0]) + (uintptr_t)g.xf;
    c.base[1] = (uintptr_t)(a.src + g.off[1]) + (uintptr_t)cxf;
    c.base[2] = (uintptr_t)(a.src + g.off[2]) + (uintptr_t)cxf;
}

__device__ __forceinline__ void yuv_cursor_next(YuvCursor &c, const BatchArgs &a)
{
    vcursor_next(c.v);
    if (++c.rr == a.Ch && c.img + 1 < a.n)
        yuv_cursor_image(c, a, c.img + 1, 0);
}

// One output row's eight segments in registers: Y y0, Y y1, Cb r0, Cb r1,
// Cb r2, Cr r0, Cr r1, Cr r2 (r0, r1: the chroma rows of y0; r2: the second
// chroma row of y1), with each segment's offset in its first chunk, the luma
// vertical weight, the chroma vertical weights of y0 and y1, and which of r0,
// r1 is y1's first chroma row.
struct YuvStaged {
    u32x4 c[8];
    int sh[8];
    float wy, wc0, wc1;
    int b0;
};

__device__ __forceinline__ void yuv_load(YuvStaged &st, const YuvCursor &c, int lane, bool repeat)
{
    int y0, y1;
    vcursor_tap(c.v, y0, y1, st.wy);
    const Tap t0 = chroma_tap(y0, c.Hc), t1 = chroma_tap(y1, c.Hc);
    st.wc0 = t0.w;
    st.wc1 = t1.w;
    st.b0 = t1.x0 == t0.x0 ? 0 : 1;
    const uintptr_t row[8] = {
        c.base[0] + (uintptr_t)y0 * (uintptr_t)c.W,   c.base[0] + (uintptr_t)y1 * (uintptr_t)c.W,
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
    }
}

__device__ __forceinline__ void yuv_write(uint8_t *slot, const YuvStaged &st, int lane)
{
#pragma unroll
    for (int s = 0; s < 8; ++s)
        ((u32x4 *)(slot + 1024 * s))[lane] = st.c[s];
}

// Per-lane column taps of the I420 kernel.
template <int J>
struct YuvCols {
    int ox[J][2];        // luma x0 - xf
    float wx[J][2];      // luma weight
    int oc[J][2];        // first chroma column read - cxf
    uint32_t sel[J][2];  // v_perm selector: bytes (x0 pair, x1 pair) of the 4 read
    float wc0[J][2], wc1[J][2];  // chroma weights of luma columns x0 and x1
};

template <int J>
__device__ __forceinline__ void yuv_cols(YuvCols<J> &k, const YuvImg &g, int Cw, int lane)
{
    const int Wc = (g.W + 1) >> 1;
    const int cxf = chroma_tap(g.xf, Wc).x0;
#pragma unroll
    for (int j = 0; j < J; ++j)
#pragma unroll
        for (int px = 0; px < 2; ++px) {
            const int c = min(2 * lane + 128 * j + px, Cw - 1);
            const Tap t = axis_tap(g.left + c, g.W, g.Wr);
            const Tap a0 = chroma_tap(t.x0, Wc), a1 = chroma_tap(t.x1, Wc);
            k.ox[j][px] = t.x0 - g.xf;
            k.wx[j][px] = t.w;
            k.oc[j][px] = a0.x0 - cxf;
            k.sel[j][px] = (uint32_t)(a0.x1 - a0.x0) << 8 | (uint32_t)(a1.x0 - a0.x0) << 16 |
                           (uint32_t)(a1.x1 - a0.x0) << 24;
            k.wc0[j][px] = a0.w;
            k.wc1[j][px] = a1.w;
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

// Chroma of luma columns x0, x1 at one chroma row: (horizontal lerps).
__device__ __forceinline__ void chroma_h(uint32_t quad, uint32_t sel, float w0, float w1, float &h0,
                                         float &h1)
{
    const uint32_t b = __builtin_amdgcn_perm(0u, quad, sel);  // x0 pair, x1 pair
    const float a0 = cvt_ubyte0(b), a1 = cvt_ubyte2(b);
    h0 = fmaf(w0, cvt_ubyte1(b) - a0, a0);  // exact (see above)
    h1 = fmaf(w1, cvt_ubyte3(b) - a1, a1);
}

template <int F16, int J, int EXACT>
__device__ __forceinline__ void yuv_compute(const BatchArgs &a, const NormK &nk, uint8_t *orow,
                                            uint32_t slot, const int (&sh)[8], float wy,
                                            float wc0, float wc1, int b0, const YuvCols<J> &k,
                                            int lane)
{
    const int Cw = a.Cw;
    constexpr int kEsz = F16 ? 2 : 4;
    const long long plane = (long long)a.Ch * Cw * kEsz;
    const bool pairs = (Cw & 1) == 0;
#pragma unroll
    for (int j = 0; j < J; ++j) {
        float o[3][2];
#pragma unroll
        for (int px = 0; px < 2; ++px) {
            // reads: Y y0, Y y1, Cb r0..r2, Cr r0..r2
            uint32_t A[8], q[8];
#pragma unroll
            for (int s = 0; s < 8; ++s)
                A[s] = slot + 1024u * s + (uint32_t)sh[s] +
                       (uint32_t)(s < 2 ? k.ox[j][px] : k.oc[j][px]);
            lds_read_quads<8>(A, q);
            // chroma at (x0, x1) x (y0, y1) for both planes
            float cc[2][2][2];  // [plane][luma row][luma col]
#pragma unroll
            for (int pl = 0; pl < 2; ++pl) {
                float h[3][2];
#pragma unroll
                for (int r = 0; r < 3; ++r)
                    chroma_h(q[2 + 3 * pl + r], k.sel[j][px], k.wc0[j][px], k.wc1[j][px], h[r][0],
                             h[r][1]);
#pragma unroll
                for (int xi = 0; xi < 2; ++xi) {
                    cc[pl][0][xi] = fmaf(wc0, h[1][xi] - h[0][xi], h[0][xi]);
                    const float hb = b0 ? h[1][xi] : h[0][xi];
                    cc[pl][1][xi] = fmaf(wc1, h[2][xi] - hb, hb);
                }
            }
            float rgb[2][2][3];  // [luma row][luma col][channel]
#pragma unroll
            for (int yi = 0; yi < 2; ++yi)
#pragma unroll
                for (int xi = 0; xi < 2; ++xi) {
                    const float Y = xi ? cvt_ubyte1(q[yi]) : cvt_ubyte0(q[yi]);
                    ycbcr_to_rgb(Y, cc[0][yi][xi], cc[1][yi][xi], rgb[yi][xi][0], rgb[yi][xi][1],
                                 rgb[yi][xi][2]);
                }
#pragma unroll
            for (int ch = 0; ch < 3; ++ch)
                o[ch][px] = normalize_k<EXACT>(
                    nk, ch,
                    lerp(lerp(rgb[0][0][ch], rgb[0][1][ch], k.wx[j][px]),
                         lerp(rgb[1][0][ch], rgb[1][1][ch], k.wx[j][px]), wy));
        }
        const int c = 2 * lane + 128 * j;
        if (c < Cw) {
            const uint32_t lo = (uint32_t)c * kEsz;
            if (pairs) {
#pragma unroll
                for (int ch = 0; ch < 3; ++ch) {
                    uint8_t *dst = orow + ch * plane + lo;
                    if (F16 && !EXACT) {
                        typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));
                        const f16x2 h = {(_Float16)o[ch][0], (_Float16)o[ch][1]};
                        __builtin_nontemporal_store(__builtin_bit_cast(uint32_t, h),
                                                    (uint32_t *)dst);
                    } else if (F16) {
                        __builtin_nontemporal_store(f16_bits(o[ch][0]) | (f16_bits(o[ch][1]) << 16),
                                                    (uint32_t *)dst);
                    } else {
                        typedef float f32x2 __attribute__((ext_vector_type(2)));
                        const f32x2 w = {o[ch][0], o[ch][1]};
                        __builtin_nontemporal_store(w, (f32x2 *)dst);
                    }
                }
            } else {
                const bool second = c + 1 < Cw;
#pragma unroll
                for (int ch = 0; ch < 3; ++ch) {
                    uint8_t *dst = orow + ch * plane + lo;
                    if (F16) {
                        ((uint16_t *)dst)[0] = (uint16_t)f16_bits(o[ch][0]);
                        if (second)
                            ((uint16_t *)dst)[1] = (uint16_t)f16_bits(o[ch][1]);
                    } else {
                        ((float *)dst)[0] = o[ch][0];
                        if (second)
                            ((float *)dst)[1] = o[ch][1];
                    }
                }
            }
        }
    }
}

template <int F16, int J, int EXACT>
__global__ void __launch_bounds__(64) yuv_rows_kernel(BatchArgs a)
{
    extern __shared__ __attribute__((aligned(16))) uint8_t lds[];
    const int lane = threadIdx.x;
    const int Ch = a.Ch;
    const long long T = (long long)a.n * Ch;
    const long long r_begin = T * blockIdx.x / gridDim.x;
    const long long r_end = T * (blockIdx.x + 1) / gridDim.x;
    if (r_begin >= r_end)
        return;
    constexpr int kEsz = F16 ? 2 : 4;
    const int n_rows = (int)(r_end - r_begin);
    const int img0 = (int)(r_begin / Ch);
    const int rr0 = (int)(r_begin - (long long)img0 * Ch);

    YuvCursor lc;
    yuv_cursor_image(lc, a, img0, rr0);
    int c_img = img0, c_rr = rr0;
    uint8_t *orow = (uint8_t *)a.out +
                    ((long long)(a.img_base + c_img) * 3 * Ch + c_rr) * (long long)a.Cw * kEsz;
    YuvCols<J> cols;
    int cW, cWr, cleft;
    {
        const YuvImg g = yuv_img(a, img0);
        yuv_cols<J>(cols, g, a.Cw, lane);
        cW = g.W;
        cWr = g.Wr;
        cleft = g.left;
    }
    const NormK nk = norm_consts(a);
    const uint32_t lds0 = lds_addr(lds);

    // One register set: row k + 1 is loaded before row k is interpolated
    // (the loads past the wave's last row repeat that row).
    int lrow = 0;
    bool at_end = false;  // the cursor sits on the wave's last row, already loaded
    auto advance = [&]() {
        if (lrow + 1 < n_rows) {
            yuv_cursor_next(lc, a);
            ++lrow;
        } else {
            at_end = true;
        }
    };
    YuvStaged R;
    yuv_load(R, lc, lane, false);
    advance();
    yuv_write(lds, R, lane);
    int csh[8];
#pragma unroll
    for (int s = 0; s < 8; ++s)
        csh[s] = R.sh[s];
    float cwy = R.wy, cwc0 = R.wc0, cwc1 = R.wc1;
    int cb0 = R.b0;
    for (int k = 0;;) {
        yuv_load(R, lc, lane, at_end);
        advance();
        yuv_compute<F16, J, EXACT>(a, nk, orow, lds0, csh, cwy, cwc0, cwc1, cb0, cols, lane);
        if (++k == n_rows)
            break;
        yuv_write(lds, R, lane);
#pragma unroll
        for (int s = 0; s < 8; ++s)
            csh[s] = R.sh[s];
        cwy = R.wy;
        cwc0 = R.wc0;
        cwc1 = R.wc1;
        cb0 = R.b0;
        orow += (long long)a.Cw * kEsz;
        if (++c_rr == Ch) {
            c_rr = 0;
            ++c_img;
            orow += 2 * (long long)Ch * a.Cw * kEsz;  // skip planes 1 and 2
            const YuvImg g = yuv_img(a, c_img);
            if (g.W != cW || g.Wr != cWr || g.left != cleft) {
                cW = g.W;
                cWr = g.Wr;
                cleft = g.left;
                yuv_cols<J>(cols, g, a.Cw, lane);
            }
        }
    }
}

// ---------------------------------------------------------------------------
// RGB, direct gather: one thread per output pixel, taps read from global
// memory. Used when the crop's source span does not fit the LDS budget.
// ---------------------------------------------------------------------------
template <int F16>
__global__ void __launch_bounds__(kThreads) rgb_direct_kernel(BatchArgs a)
{
    const long long plane = (long long)a.Ch * a.Cw;
    const long long total = plane * a.n;
    for (long long gid = (long long)blockIdx.x * kThreads + threadIdx.x; gid < total;
         gid += (long long)gridDim.x * kThreads) {
        const int img = (int)(gid / plane);
        const long long pix = gid - (long long)img * plane;
        const int yc = (int)(pix / a.Cw);
        const int xc = (int)(pix - (long long)yc * a.Cw);
        Desc d;
        image_desc(a, img, d);
        const Tap tx = axis_tap(d.left + xc, d.W, d.Wr);
        const Tap ty = axis_tap(d.top + yc, d.H, d.Hr);
        const uint8_t *r0 = a.src + d.off[0] + (long long)ty.x0 * d.pitch;
        const uint8_t *r1 = a.src + d.off[0] + (long long)ty.x1 * d.pitch;
        const long long base = (long long)(a.img_base + img) * 3 * plane + pix;
#pragma unroll
        for (int ch = 0; ch < 3; ++ch) {
            const float p00 = r0[3 * tx.x0 + ch], p01 = r0[3 * tx.x1 + ch];
            const float p10 = r1[3 * tx.x0 + ch], p11 = r1[3 * tx.x1 + ch];
            const float v = lerp(lerp(p00, p01, tx.w), lerp(p10, p11, tx.w), ty.w);
            store1<F16>(a.out, base + ch * plane, normalize(v, a.mean[ch], a.stdv[ch], a.rcp[ch]));
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

template <int F16>
__global__ void __launch_bounds__(kThreads) yuv_direct_kernel(BatchArgs a)
{
    const long long plane = (long long)a.Ch * a.Cw;
    const long long total = plane * a.n;
    for (long long gid = (long long)blockIdx.x * kThreads + threadIdx.x; gid < total;
         gid += (long long)gridDim.x * kThreads) {
        const int img = (int)(gid / plane);
        const long long pix = gid - (long long)img * plane;
        const int yc = (int)(pix / a.Cw);
        const int xc = (int)(pix - (long long)yc * a.Cw);
        Desc d;
        image_desc(a, img, d);
        const int Wc = (d.W + 1) >> 1, Hc = (d.H + 1) >> 1;
        const uint8_t *yp = a.src + d.off[0];
        const uint8_t *cbp = a.src + d.off[1];
        const uint8_t *crp = a.src + d.off[2];
        const Tap tx = axis_tap(d.left + xc, d.W, d.Wr);
        const Tap ty = axis_tap(d.top + yc, d.H, d.Hr);
        const int xx[2] = {tx.x0, tx.x1};
        const int yy[2] = {ty.x0, ty.x1};
        float rgb[2][2][3];
#pragma unroll
        for (int i = 0; i < 2; ++i) {
            const Tap cy = chroma_tap(yy[i], Hc);
#pragma unroll
            for (int k = 0; k < 2; ++k) {
                const Tap cx = chroma_tap(xx[k], Wc);
                const float Y = (float)yp[(long long)yy[i] * d.W + xx[k]];
                ycbcr_to_rgb(Y, chroma_at(cbp, Wc, cx, cy), chroma_at(crp, Wc, cx, cy),
                             rgb[i][k][0], rgb[i][k][1], rgb[i][k][2]);
            }
        }
        const long long base = (long long)(a.img_base + img) * 3 * plane + pix;
#pragma unroll
        for (int ch = 0; ch < 3; ++ch) {
            const float v = lerp(lerp(rgb[0][0][ch], rgb[0][1][ch], tx.w),
                                 lerp(rgb[1][0][ch], rgb[1][1][ch], tx.w), ty.w);
            store1<F16>(a.out, base + ch * plane, normalize(v, a.mean[ch], a.stdv[ch], a.rcp[ch]));
        }
    }
}

unsigned direct_grid(const BatchArgs &a)
{
    const long long total = (long long)a.Ch * a.Cw * a.n;
    long long blocks = (total + kThreads - 1) / kThreads;
    const long long cap = 1 << 20;
    return (unsigned)(blocks < cap ? blocks : cap);
}

}  // namespace

int launch_rgb_direct(const BatchArgs &a, int out_f16, void *stream)
{
    hipStream_t s = (hipStream_t)stream;
    const dim3 grid(direct_grid(a)), block(kThreads);
    if (out_f16)
        hipLaunchKernelGGL(rgb_direct_kernel<1>, grid, block, 0, s, a);
    else
        hipLaunchKernelGGL(rgb_direct_kernel<0>, grid, block, 0, s, a);
    return (int)hipGetLastError();
}

int launch_rgb_lds(const BatchArgs &a, int out_f16, size_t lds_bytes, void *stream)
{
    hipStream_t s = (hipStream_t)stream;
    const dim3 grid((unsigned)a.grid), block(kThreads);
    if (out_f16)
        hipLaunchKernelGGL(rgb_lds_kernel<1>, grid, block, lds_bytes, s, a);
    else
        hipLaunchKernelGGL(rgb_lds_kernel<0>, grid, block, lds_bytes, s, a);
    return (int)hipGetLastError();
}

int launch_rgb_gather(const BatchArgs &a, int out_f16, size_t lds_bytes, void *stream)
{
    hipStream_t s = (hipStream_t)stream;
    const dim3 grid((unsigned)a.grid), block(kThreads);
    if (out_f16)
        hipLaunchKernelGGL(rgb_gather_kernel<1>, grid, block, lds_bytes, s, a);
    else
        hipLaunchKernelGGL(rgb_gather_kernel<0>, grid, block, lds_bytes, s, a);
    return (int)hipGetLastError();
}

template <int F16, int EXACT, int G>
const void *rows_kernel_g(int col_iters, int prefetch)
{
    if (prefetch == 1)
        return col_iters <= 1   ? (const void *)rgb_rows_kernel<F16, 1, EXACT, G, 1>
               : col_iters <= 2 ? (const void *)rgb_rows_kernel<F16, 2, EXACT, G, 1>
                                : (const void *)rgb_rows_kernel<F16, 4, EXACT, G, 1>;
    return col_iters <= 1   ? (const void *)rgb_rows_kernel<F16, 1, EXACT, G, 2>
           : col_iters <= 2 ? (const void *)rgb_rows_kernel<F16, 2, EXACT, G, 2>
                            : (const void *)rgb_rows_kernel<F16, 4, EXACT, G, 2>;
}

template <int F16, int EXACT>
const void *rows_kernel_e(int col_iters, int groups, int prefetch)
{
    return groups <= 1   ? rows_kernel_g<F16, EXACT, 1>(col_iters, prefetch)
           : groups <= 2 ? rows_kernel_g<F16, EXACT, 2>(col_iters, prefetch)
                         : rows_kernel_g<F16, EXACT, 4>(col_iters, prefetch);
}

const void *rows_kernel(const BatchArgs &a, int f16)
{
    const int e = a.exact, c = a.col_iters, g = a.row_groups, p = a.prefetch;
    return f16 ? (e ? rows_kernel_e<1, 1>(c, g, p) : rows_kernel_e<1, 0>(c, g, p))
               : (e ? rows_kernel_e<0, 1>(c, g, p) : rows_kernel_e<0, 0>(c, g, p));
}

int launch_rgb_rows(const BatchArgs &a, int out_f16, size_t lds_bytes, void *stream)
{
    hipStream_t s = (hipStream_t)stream;
    const dim3 grid((unsigned)a.grid), block(64);
    void *args[] = {(void *)&a};
    return (int)hipLaunchKernel(rows_kernel(a, out_f16), grid, block, args, lds_bytes, s);
}

int occupancy_rgb_rows(const BatchArgs &a, int out_f16, size_t lds_bytes, int *blocks_per_cu)
{
    return (int)hipOccupancyMaxActiveBlocksPerMultiprocessor(
        blocks_per_cu, rows_kernel(a, out_f16), 64, lds_bytes);
}

int occupancy_rgb_gather(int out_f16, size_t lds_bytes, int *blocks_per_cu)
{
    hipError_t e = out_f16 ? hipOccupancyMaxActiveBlocksPerMultiprocessor(
                                 blocks_per_cu, rgb_gather_kernel<1>, kThreads, lds_bytes)
                           : hipOccupancyMaxActiveBlocksPerMultiprocessor(
                                 blocks_per_cu, rgb_gather_kernel<0>, kThreads, lds_bytes);
    return (int)e;
}

int occupancy_rgb_lds(int out_f16, size_t lds_bytes, int *blocks_per_cu)
{
    hipError_t e = out_f16 ? hipOccupancyMaxActiveBlocksPerMultiprocessor(
                                 blocks_per_cu, rgb_lds_kernel<1>, kThreads, lds_bytes)
                           : hipOccupancyMaxActiveBlocksPerMultiprocessor(
                                 blocks_per_cu, rgb_lds_kernel<0>, kThreads, lds_bytes);
    return (int)e;
}

int launch_yuv_direct(const BatchArgs &a, int out_f16, void *stream)
{
    hipStream_t s = (hipStream_t)stream;
    const dim3 grid(direct_grid(a)), block(kThreads);
    if (out_f16)
        hipLaunchKernelGGL(yuv_direct_kernel<1>, grid, block, 0, s, a);
    else
        hipLaunchKernelGGL(yuv_direct_kernel<0>, grid, block, 0, s, a);
    return (int)hipGetLastError();
}

template <int F16, int EXACT>
const void *yuv_rows_kernel_e(int col_iters)
{
    return col_iters <= 1   ? (const void *)yuv_rows_kernel<F16, 1, EXACT>
           : col_iters <= 2 ? (const void *)yuv_rows_kernel<F16, 2, EXACT>
                            : (const void *)yuv_rows_kernel<F16, 4, EXACT>;
}

const void *yuv_rows_kernel_for(const BatchArgs &a, int f16)
{
    return f16 ? (a.exact ? yuv_rows_kernel_e<1, 1>(a.col_iters) : yuv_rows_kernel_e<1, 0>(a.col_iters))
               : (a.exact ? yuv_rows_kernel_e<0, 1>(a.col_iters) : yuv_rows_kernel_e<0, 0>(a.col_iters));
}

int launch_yuv_rows(const BatchArgs &a, int out_f16, size_t lds_bytes, void *stream)
{
    hipStream_t s = (hipStream_t)stream;
    const dim3 grid((unsigned)a.grid), block(64);
    void *args[] = {(void *)&a};
    return (int)hipLaunchKernel(yuv_rows_kernel_for(a, out_f16), grid, block, args, lds_bytes, s);
}

int occupancy_yuv_rows(const BatchArgs &a, int out_f16, size_t lds_bytes, int *blocks_per_cu)
{
    return (int)hipOccupancyMaxActiveBlocksPerMultiprocessor(
        blocks_per_cu, yuv_rows_kernel_for(a, out_f16), 64, lds_bytes);
}

}  // namespace smol
