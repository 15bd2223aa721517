// smol_jpeg_kernels.hip -- the GPU part of partial JPEG decoding (section 6.4, "ROI
// decoding"): dequantisation and the 8 x 8 inverse DCT of the blocks of a
// 4:2:0 frame that meet a rectangle, written to I420 planes. The entropy
// decoding that produces the coefficients is the CPU decoder's.
//
// A wave decodes up to eight horizontally adjacent blocks of one block row
// at a time. Each 1-D transform x(n) = sum_k c(k, n) D(k) is evaluated
// through the parity of the cosine basis, c(k, 7 - n) = (-1)^k c(k, n): for
// n < 4 the even-frequency sum E and the odd-frequency sum O (each in
// increasing frequency), then x(n) = E + O and x(7 - n) = E - O (T.81 A.3.3
// evaluated separably), each product and sum rounded on its own (no
// contraction). Pass 1: lane l loads coefficient row v = l % 8 of block
// b = l / 8 (16 contiguous bytes) and forms G(v, x) for all x in registers.
// After an exchange through LDS, pass 2: lane l forms output rows y and 7 - y
// (y = l % 4) of block b at columns 4 h .. 4 h + 3 (h = (l % 8) / 4). Then
// + 128, clamped to [0, 255] and rounded to nearest even.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "smol_internal.h"

namespace smol {
namespace {

constexpr int kBlocksPerWave = 8;
constexpr int kBlockWords = 68;

// The 32-bit word at a 4-byte aligned field, and its two 16-bit halves.
__device__ __forceinline__ uint32_t word_of(const int16_t *p)
{
    uint32_t w;
    __builtin_memcpy(&w, p, 4);
    return w;
}
__device__ __forceinline__ int lo16(uint32_t w) { return (int)(int16_t)(w & 0xffffu); }
__device__ __forceinline__ int hi16(uint32_t w) { return (int)(int16_t)(w >> 16); }

// floor(n / d) from the run's m = ceil(2^s / d) (exact for n < 2^31)
__device__ __forceinline__ uint32_t magic_div(uint32_t n, uint32_t m, uint32_t s)
{
    return (uint32_t)(((uint64_t)n * m) >> s);
}

__global__ void __launch_bounds__(64) jpeg_idct_kernel(JpegArgs a)
{
    // G(v, x) of block b at word b * kBlockWords + 8 v + x: the 4-word pad
    // per block spreads the eight blocks' rows over the LDS banks (with 64
    // words per block every block's row v sits in the same banks)
    __shared__ __attribute__((aligned(16))) float g[kBlocksPerWave * kBlockWords];
    const int l = threadIdx.x;
    const int b = l >> 3, row = l & 7;  // block of the group; coefficient row v of pass 1
    const int y = row & 3, h = row >> 2;  // pass 2: output rows y, 7 - y; columns 4h .. 4h + 3
    float cy[8];                          // c(k, y) for pass 2
#pragma unroll
    for (int k = 0; k < 8; ++k)
        cy[k] = a.c[k * 8 + y];
    // job indices stay below 2^31 (the host splits launches), so the job
    // mapping runs in 32-bit unsigned arithmetic, its divisions by the run's
    // divisors as multiplications (JpegRun)
    const uint32_t jobs = a.run[a.runs - 1].jobs_end;
    int ri = 0;  // run of the current job (jobs ascend within a workgroup)
    for (uint32_t job = blockIdx.x; job < jobs; job += gridDim.x) {
        while (a.run[ri].jobs_end <= job)
            ++ri;
        const JpegRun &r = a.run[ri];
        // groups of up to eight blocks along each block row of the rectangle
        const uint32_t lg = r.groups & 0x7ffu, cg = (r.groups >> 11) & 0x7ffu;
        const uint32_t lum = r.lum, chr = r.chr, per_frame = lum + 2 * chr;
        const uint32_t local = job - (ri ? a.run[ri - 1].jobs_end : 0);
        const uint32_t f = magic_div(local, r.m_pf, r.shifts & 0xffu);
        uint32_t k = local - f * per_frame;
        // the 16-bit fields in pairs, as the words that hold them (a 16-bit
        // field read alone becomes a vector load that the wave waits for)
        const uint32_t wxy = word_of(&r.wx0), wm = word_of(&r.wmx);
        int comp, by, bx0, nb, gw, ox, oy, pw, ph;  // (ox, oy): the stored grid's first block
        long long cbase, pbase;
        if (k < lum) {
            comp = 0;
            const uint32_t kr = magic_div(k, r.m_lg, (r.shifts >> 8) & 0xffu);
            const uint32_t lb = word_of(&r.lbx0);
            by = hi16(lb) + (int)kr;
            const uint32_t gi = k - kr * lg;
            bx0 = lo16(lb) + (int)gi * kBlocksPerWave;
            nb = gi + 1 == lg ? (int)((r.groups >> 22) & 0xfu) : kBlocksPerWave;
            gw = 2 * lo16(wm);
            ox = 2 * lo16(wxy);
            oy = 2 * hi16(wxy);
            cbase = 0;
            pbase = 0;
            pw = r.W;
            ph = r.H;
        } else {
            k -= lum;
            comp = k < chr ? 1 : 2;
            k -= comp == 1 ? 0 : chr;
            const uint32_t kr = magic_div(k, r.m_cg, (r.shifts >> 16) & 0xffu);
            const uint32_t cb = word_of(&r.cbx0);
            by = hi16(cb) + (int)kr;
            const uint32_t gi = k - kr * cg;
            bx0 = lo16(cb) + (int)gi * kBlocksPerWave;
            nb = gi + 1 == cg ? (int)(r.groups >> 26) : kBlocksPerWave;
            gw = lo16(wm);
            ox = lo16(wxy);
            oy = hi16(wxy);
            cbase = 64LL * lo16(wm) * hi16(wm) * (comp == 1 ? 4 : 5);
            pbase = comp == 1 ? r.cboff : r.croff;
            pw = (r.W + 1) >> 1;
            ph = (r.H + 1) >> 1;
        }
        // lanes of blocks past the group's end repeat its last block
        const int bb = min(b, nb - 1);
        const int16_t *blk = a.coef + r.coef + f * r.coef_stride + cbase +
                             64LL * ((long long)(by - oy) * gw + bx0 + bb - ox);
        typedef short short8 __attribute__((ext_vector_type(8)));
        const short8 raw = *(const short8 *)(blk + 8 * row);
        const uint8_t *q = a.q[r.shifts >> 24][comp == 0 ? 0 : 1];
        float d[8];
#pragma unroll
        for (int u = 0; u < 8; ++u)
            d[u] = (float)((int)raw[u] * (int)q[8 * row + u]);  // exact: |.| < 2^24
        // horizontal pass for row v = row of block bb: x = 0..3 and 7..4,
        // written as two 16-byte stores
        typedef float f32x4 __attribute__((ext_vector_type(4)));
        f32x4 lo, hi;
#pragma unroll
        for (int n = 0; n < 4; ++n) {
            float e = a.c[0 * 8 + n] * d[0];
            e = e + a.c[2 * 8 + n] * d[2];
            e = e + a.c[4 * 8 + n] * d[4];
            e = e + a.c[6 * 8 + n] * d[6];
            float o = a.c[1 * 8 + n] * d[1];
            o = o + a.c[3 * 8 + n] * d[3];
            o = o + a.c[5 * 8 + n] * d[5];
            o = o + a.c[7 * 8 + n] * d[7];
            lo[n] = e + o;
            hi[3 - n] = e - o;
        }
        f32x4 *grow = (f32x4 *)&g[b * kBlockWords + 8 * row];
        grow[0] = lo;
        grow[1] = hi;
        __syncthreads();
        // vertical pass: rows y and 7 - y of block bb at columns 4h .. 4h + 3
        f32x4 gv[8];
#pragma unroll
        for (int v = 0; v < 8; ++v)
            gv[v] = *(const f32x4 *)&g[b * kBlockWords + 8 * v + 4 * h];
        uint32_t top = 0, bot = 0;  // four pixels of row y, four of row 7 - y
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            float e = cy[0] * gv[0][i];
            e = e + cy[2] * gv[2][i];
            e = e + cy[4] * gv[4][i];
            e = e + cy[6] * gv[6][i];
            float o = cy[1] * gv[1][i];
            o = o + cy[3] * gv[3][i];
            o = o + cy[5] * gv[5][i];
            o = o + cy[7] * gv[7][i];
            // v_cvt_pk_u8_f32: byte i = the value clamped to [0, 255] and
            // rounded to nearest even (one instruction for clamp, round,
            // convert and insert)
            top = __builtin_amdgcn_cvt_pk_u8_f32((e + o) + 128.0f, (uint32_t)i, top);
            bot = __builtin_amdgcn_cvt_pk_u8_f32((e - o) + 128.0f, (uint32_t)i, bot);
        }
        const int gx = 8 * (bx0 + b) + 4 * h;
        if (b < nb && gx < pw) {
            uint8_t *base = a.out + r.out + f * r.out_stride + pbase;
            const int gy[2] = {8 * by + y, 8 * by + 7 - y};
            const uint32_t pix[2] = {top, bot};
#pragma unroll
            for (int k = 0; k < 2; ++k) {
                if (gy[k] >= ph)
                    continue;
                uint8_t *dst = base + (long long)gy[k] * pw + gx;
                if (gx + 4 <= pw && ((uintptr_t)dst & 3) == 0) {
                    *(uint32_t *)dst = pix[k];
                } else {
#pragma unroll
                    for (int x = 0; x < 4; ++x)
                        if (gx + x < pw)
                            dst[x] = (uint8_t)(pix[k] >> (8 * x));
                }
            }
        }
        __syncthreads();
    }
}

}  // namespace

int launch_jpeg_idct(const JpegArgs &a, int grid, void *stream)
{
    hipLaunchKernelGGL(jpeg_idct_kernel, dim3((unsigned)grid), dim3(64), 0, (hipStream_t)stream,
                       a);
    return (int)hipGetLastError();
}

}  // namespace smol
