// smol_device.h -- device helpers shared by the kernel files of libsmol:
// the half-pixel tap map, chroma siting, BT.601 conversion, the separately
// rounded lerp, normalisation, fp16 rounding and output stores.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "smol_internal.h"

namespace smol {
namespace {
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

// Chroma tap of luma index x over n chroma samples, in quarters of a
// sample: centred 4:2:0 siting puts luma x at chroma u = x/2 - 1/4
// (4u = 2x - 1), co-sited (left) siting at u = x/2 (4u = 2x). Taps floor(u)
// and floor(u) + 1 with weight frac(u) (a multiple of 1/4, exact), clamped at
// both ends like the luma map.
__device__ __forceinline__ Tap chroma_tap(int x, int n, int left = 0)
{
    const int num = 2 * x - 1 + left;
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

// The same conversion from cb16 = 16 * (cb - 128) and cr16 = 16 * (cr - 128):
// with the coefficients divided by 16 (exact) each product is the same real
// number as above, so every rounded value is identical.
__device__ __forceinline__ void ycbcr16_to_rgb(float y, float cb16, float cr16, float &r,
                                               float &g, float &b)
{
    constexpr float s = 0.0625f;
    r = clamp255(y + (kRCr * s) * cr16);
    g = clamp255((y - (kGCb * s) * cb16) - (kGCr * s) * cr16);
    b = clamp255(y + (kBCb * s) * cb16);
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

// Output element for channel ch of resized value v: OUT 0 / 1 the normalised
// value as fp32 / fp16; OUT 2 (uint8 output) v itself rounded to the nearest
// integer, ties to even (v_rndne_f32), clamped to 0..255, not normalised.
template <int OUT>
__device__ __forceinline__ void emit1(const BatchArgs &a, long long idx, int ch, float v)
{
    if (OUT == 2)
        ((uint8_t *)a.out)[idx] = (uint8_t)__builtin_rintf(clamp255(v));
    else
        store1<OUT>(a.out, idx, normalize(v, a.mean[ch], a.stdv[ch], a.rcp[ch]));
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

}  // namespace
}  // namespace smol
