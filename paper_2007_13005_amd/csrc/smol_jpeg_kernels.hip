// smol_jpeg_kernels.hip -- the GPU part of partial JPEG decoding (section 6.4, "ROI
// decoding"): dequantisation and the 8 x 8 inverse DCT of the blocks of a
// 4:2:0 frame that meet a rectangle, written to I420 planes. The entropy
// decoding that produces the coefficients is the CPU decoder's.
//
// A wave decodes up to eight horizontally adjacent blocks of one block row
// at a time: lane l loads coefficient row v = l % 8 of block b = l / 8 (16
// contiguous bytes), forms the horizontal pass G(v, x) = sum_u c(u, x) D(v, u)
// for all x in registers, and, after an exchange through LDS, output row
// y = l % 8 of block b: f(y, x) = sum_v c(v, y) G(v, x). Both sums run in
// increasing frequency (T.81 A.3.3 evaluated separably), each product and
// sum rounded on its own (no contraction); then + 128, rounded to nearest
// even, clamped.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "smol_internal.h"

namespace smol {
namespace {

constexpr int kBlocksPerWave = 8;

__global__ void __launch_bounds__(64) jpeg_idct_kernel(JpegArgs a)
{
    __shared__ float g[kBlocksPerWave][8][8];  // [block][v][x]
    const int l = threadIdx.x;
    const int b = l >> 3, row = l & 7;  // block of the group; v (pass 1) or y (pass 2)
    float cr[8];                        // c(k, row) for pass 2
#pragma unroll
    for (int k = 0; k < 8; ++k)
        cr[k] = a.c[k * 8 + row];
    // job indices stay below 2^31 (the host splits launches), so the job
    // mapping runs in 32-bit unsigned arithmetic
    const uint32_t jobs = a.run[a.runs - 1].jobs_end;
    int ri = 0;  // run of the current job (jobs ascend within a workgroup)
    for (uint32_t job = blockIdx.x; job < jobs; job += gridDim.x) {
        while (a.run[ri].jobs_end <= job)
            ++ri;
        const JpegRun &r = a.run[ri];
        // groups of up to eight blocks along each block row of the rectangle
        const uint32_t lg = ((uint32_t)r.lnbx + kBlocksPerWave - 1) / kBlocksPerWave;
        const uint32_t cg = ((uint32_t)r.cnbx + kBlocksPerWave - 1) / kBlocksPerWave;
        const uint32_t lum = lg * (uint32_t)r.lnby, chr = cg * (uint32_t)r.cnby;
        const uint32_t per_frame = lum + 2 * chr;
        const uint32_t local = job - (ri ? a.run[ri - 1].jobs_end : 0);
        const uint32_t f = local / per_frame;
        uint32_t k = local - f * per_frame;
        int comp, by, bx0, nb, gw, ox, oy, pw, ph;  // (ox, oy): the stored grid's first block
        long long cbase, pbase;
        if (k < lum) {
            comp = 0;
            by = r.lby0 + (int)(k / lg);
            const int gi = (int)(k - (k / lg) * lg);
            bx0 = r.lbx0 + gi * kBlocksPerWave;
            nb = min(kBlocksPerWave, r.lnbx - gi * kBlocksPerWave);
            gw = 2 * r.wmx;
            ox = 2 * r.wx0;
            oy = 2 * r.wy0;
            cbase = 0;
            pbase = 0;
            pw = r.W;
            ph = r.H;
        } else {
            k -= lum;
            comp = k < chr ? 1 : 2;
            k -= comp == 1 ? 0 : chr;
            by = r.cby0 + (int)(k / cg);
            const int gi = (int)(k - (k / cg) * cg);
            bx0 = r.cbx0 + gi * kBlocksPerWave;
            nb = min(kBlocksPerWave, r.cnbx - gi * kBlocksPerWave);
            gw = r.wmx;
            ox = r.wx0;
            oy = r.wy0;
            cbase = 64LL * r.wmx * r.wmy * (comp == 1 ? 4 : 5);
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
        const uint8_t *q = a.q[r.qt][comp == 0 ? 0 : 1];
        float d[8];
#pragma unroll
        for (int u = 0; u < 8; ++u)
            d[u] = (float)((int)raw[u] * (int)q[8 * row + u]);  // exact: |.| < 2^24
        // horizontal pass for row v = row of block bb
#pragma unroll
        for (int x = 0; x < 8; ++x) {
            float s = 0.0f;
#pragma unroll
            for (int u = 0; u < 8; ++u)
                s = s + a.c[u * 8 + x] * d[u];
            g[b][row][x] = s;
        }
        __syncthreads();
        // vertical pass for row y = row of block bb
        uint32_t px4[2] = {0, 0};
        uint8_t px[8];
#pragma unroll
        for (int x = 0; x < 8; ++x) {
            float t = 0.0f;
#pragma unroll
            for (int v = 0; v < 8; ++v)
                t = t + cr[v] * g[b][v][x];
            px[x] = (uint8_t)__builtin_rintf(fminf(fmaxf(t + 128.0f, 0.0f), 255.0f));
            px4[x >> 2] |= (uint32_t)px[x] << (8 * (x & 3));
        }
        const int gx = 8 * (bx0 + b), gy = 8 * by + row;
        if (b < nb && gy < ph) {
            uint8_t *dst = a.out + r.out + f * r.out_stride + pbase + (long long)gy * pw + gx;
            if (gx + 8 <= pw && ((uintptr_t)dst & 7) == 0) {
                typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
                *(u32x2 *)dst = u32x2{px4[0], px4[1]};
            } else {
#pragma unroll
                for (int x = 0; x < 8; ++x)
                    if (gx + x < pw)
                        dst[x] = px[x];
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
