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
// is (v - mean) / std with an IEEE division. The fp32 results are therefore
// the correctly rounded values of that sequence, and fp16 outputs are their
// round-to-nearest-even.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "smol_internal.h"

namespace smol {
namespace {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / 64;

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

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
    const long long q = (long long)((double)num / (double)den);
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

__device__ __forceinline__ float normalize(float v, float mean, float stdv) { return (v - mean) / stdv; }

__device__ __forceinline__ uint32_t f16_bits(float v)
{
    _Float16 h = (_Float16)v;  // v_cvt_f16_f32: round to nearest even
    return (uint32_t)__builtin_bit_cast(uint16_t, h);
}

// Store 8 consecutive outputs starting at element index idx of one plane.
template <int F16>
__device__ __forceinline__ void store8(void *out, long long idx, const float (&v)[8], int valid)
{
    if (F16) {
        uint16_t *o = (uint16_t *)out + idx;
        if (valid == 8 && (idx & 7) == 0) {
            u32x4 q;
            q.x = f16_bits(v[0]) | (f16_bits(v[1]) << 16);
            q.y = f16_bits(v[2]) | (f16_bits(v[3]) << 16);
            q.z = f16_bits(v[4]) | (f16_bits(v[5]) << 16);
            q.w = f16_bits(v[6]) | (f16_bits(v[7]) << 16);
            __builtin_nontemporal_store(q, (u32x4 *)o);
        } else {
#pragma unroll
            for (int j = 0; j < 8; ++j)
                if (j < valid)
                    o[j] = (uint16_t)f16_bits(v[j]);
        }
    } else {
        float *o = (float *)out + idx;
        if (valid == 8 && (idx & 3) == 0) {
            const f32x4 lo = {v[0], v[1], v[2], v[3]};
            const f32x4 hi = {v[4], v[5], v[6], v[7]};
            __builtin_nontemporal_store(lo, (f32x4 *)o);
            __builtin_nontemporal_store(hi, (f32x4 *)(o + 4));
        } else {
#pragma unroll
            for (int j = 0; j < 8; ++j)
                if (j < valid)
                    o[j] = v[j];
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

// First index i in [0, n) with a[i] >= v (a non-decreasing).
__device__ __forceinline__ int lower_bound(const int *a, int n, int v)
{
    int lo = 0, hi = n;
    while (lo < hi) {
        const int mid = (lo + hi) >> 1;
        if (a[mid] < v)
            lo = mid + 1;
        else
            hi = mid;
    }
    return lo;
}

typedef __attribute__((address_space(3))) void lds_void_t;

// Copy `nbytes` source bytes starting at absolute address `row` into the LDS
// slot, as 16-byte chunks aligned in the global address space; the slot then
// holds the bytes from (row & ~15) on. One wave per call; chunks entirely
// inside [gbase, gend) use direct-to-LDS loads, the (at most two) chunks that
// straddle the buffer ends are copied byte by byte within the buffer.
__device__ __forceinline__ void stage_row(uint8_t *slot, uintptr_t row, int nbytes,
                                          uintptr_t gbase, uintptr_t gend, int lane)
{
    const uintptr_t al = row & ~(uintptr_t)15;
    const int nch = (int)((row - al + (uintptr_t)nbytes + 15) >> 4);
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
// RGB, LDS-staged. Workgroup = (image, band of R output rows), full crop width.
// ---------------------------------------------------------------------------
template <int F16>
__global__ void __launch_bounds__(kThreads) rgb_lds_kernel(BatchArgs a)
{
    extern __shared__ __attribute__((aligned(16))) uint8_t lds[];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int img = (int)(blockIdx.x / (unsigned)a.bands);
    const int band = (int)blockIdx.x - img * a.bands;
    Desc d;
    image_desc(a, img, d);
    const int Cw = a.Cw, Ch = a.Ch, R = a.R;
    const int r_begin = band * R;
    const int r_cnt = min(R, Ch - r_begin);

    int *colx = (int *)lds;
    float *colw = (float *)(colx + Cw);
    int *ty0 = (int *)(colw + Cw);
    int *ty1 = ty0 + R;
    float *twy = (float *)(ty1 + R);
    int *smap = (int *)(twy + R);
    int *rowa = smap + 2 * R;
    uint8_t *slots = lds + a.slots_off;

    const int xs = axis_tap(d.left, d.W, d.Wr).x0;
    const int xe = axis_tap(d.left + Cw - 1, d.W, d.Wr).x1;
    const int span_bytes = 3 * (xe - xs + 1);

    for (int c = tid; c < Cw; c += kThreads) {
        const Tap t = axis_tap(d.left + c, d.W, d.Wr);
        colx[c] = 3 * (t.x0 - xs);
        colw[c] = t.w;
    }
    for (int r = tid; r < r_cnt; r += kThreads) {
        const Tap t = axis_tap(d.top + r_begin + r, d.H, d.Hr);
        ty0[r] = t.x0;
        ty1[r] = t.x1;
        twy[r] = t.w;
    }
    __syncthreads();

    // Candidate 2r is row ty0[r], 2r+1 is ty1[r]; each maps to the first
    // candidate holding the same source row, so every row is staged once.
    for (int s = tid; s < 2 * r_cnt; s += kThreads) {
        const int v = (s & 1) ? ty1[s >> 1] : ty0[s >> 1];
        const int i0 = lower_bound(ty0, r_cnt, v);
        const int i1 = lower_bound(ty1, r_cnt, v);
        int first = 2 * r_cnt;
        if (i0 < r_cnt && ty0[i0] == v)
            first = 2 * i0;
        if (i1 < r_cnt && ty1[i1] == v)
            first = min(first, 2 * i1 + 1);
        smap[s] = first;
    }
    __syncthreads();

    const uintptr_t gbase = (uintptr_t)a.src, gend = gbase + (uintptr_t)a.src_bytes;
    const uintptr_t img_base = gbase + (uintptr_t)d.off[0] + 3 * (uintptr_t)xs;
    for (int s = wave; s < 2 * r_cnt; s += kWaves) {
        if (smap[s] != s)
            continue;
        const int y = (s & 1) ? ty1[s >> 1] : ty0[s >> 1];
        stage_row(slots + s * a.slot_bytes, img_base + (uintptr_t)y * (uintptr_t)d.pitch,
                  span_bytes, gbase, gend, lane);
    }
    for (int s = tid; s < 2 * r_cnt; s += kThreads) {
        const int y = (s & 1) ? ty1[s >> 1] : ty0[s >> 1];
        const uintptr_t row = img_base + (uintptr_t)y * (uintptr_t)d.pitch;
        rowa[s] = a.slots_off + smap[s] * a.slot_bytes + (int)(row & 15);
    }
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();

    const int gpr = (Cw + 7) >> 3;
    const int items = r_cnt * gpr;
    const long long plane = (long long)Ch * Cw;
    const long long out_img = (long long)(a.img_base + img) * 3 * plane;
    for (int it = tid; it < items; it += kThreads) {
        const int r = it / gpr;
        const int c0 = (it - r * gpr) * 8;
        const int a0 = rowa[2 * r], a1 = rowa[2 * r + 1];
        const float wy = twy[r];
        float o[3][8];
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            const int c = min(c0 + j, Cw - 1);
            const int xo = colx[c];
            const float wx = colw[c];
            float p[6], q[6];
            lds_pixel_pair(lds, a0 + xo, p);
            lds_pixel_pair(lds, a1 + xo, q);
#pragma unroll
            for (int ch = 0; ch < 3; ++ch) {
                const float t = lerp(p[ch], p[ch + 3], wx);
                const float b = lerp(q[ch], q[ch + 3], wx);
                o[ch][j] = normalize(lerp(t, b, wy), a.mean[ch], a.stdv[ch]);
            }
        }
        const int valid = min(8, Cw - c0);
        const long long idx = out_img + (long long)(r_begin + r) * Cw + c0;
#pragma unroll
        for (int ch = 0; ch < 3; ++ch)
            store8<F16>(a.out, idx + ch * plane, o[ch], valid);
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
            store1<F16>(a.out, base + ch * plane, normalize(v, a.mean[ch], a.stdv[ch]));
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
            store1<F16>(a.out, base + ch * plane, normalize(v, a.mean[ch], a.stdv[ch]));
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
    const dim3 grid((unsigned)a.n * (unsigned)a.bands), block(kThreads);
    if (out_f16)
        hipLaunchKernelGGL(rgb_lds_kernel<1>, grid, block, lds_bytes, s, a);
    else
        hipLaunchKernelGGL(rgb_lds_kernel<0>, grid, block, lds_bytes, s, a);
    return (int)hipGetLastError();
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

int launch_yuv_lds(const BatchArgs &, int, size_t, void *)
{
    return (int)hipErrorNotSupported;
}

}  // namespace smol
