// smol_stream.hip -- the streaming-bandwidth probe (smol_stream_probe): one
// launch that reads one buffer and writes another with coalesced 16-byte
// accesses, every wave interleaving its reads and writes in the ratio of the
// two sizes. It measures the memory ceiling that the preprocessing kernels'
// byte mix can reach on the device.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "smol.h"
#include "smol_internal.h"
#include "smol_stream.h"

namespace smol {
namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(1))) const u32x4 GlobalIn;
typedef __attribute__((address_space(1))) u32x4 GlobalOut;

constexpr int kWavesPerGroup = 4;

struct StreamArgs {
    const u32x4 *src;
    u32x4 *dst;
    uint64_t nr, nw;  // 16-byte granules read and written
    uint32_t waves;
};

template <int NTL>
__device__ __forceinline__ u32x4 ld(const u32x4 *p, uint64_t i)
{
    GlobalIn *g = (GlobalIn *)p + i;
    return NTL ? __builtin_nontemporal_load(g) : *g;
}

template <int NTS>
__device__ __forceinline__ void st(u32x4 *p, uint64_t i, u32x4 v)
{
    GlobalOut *g = (GlobalOut *)p + i;
    if (NTS)
        __builtin_nontemporal_store(v, g);
    else
        *g = v;
}

// Wave w owns granules [n w / W, n (w + 1) / W) of each buffer. A read step
// loads kUnroll * 64 granules (kUnroll 16-byte loads per lane in flight);
// after each step the wave writes, 64 granules per store, until its writes
// have kept pace with its reads (writes done = floor(reads done * its writes
// / its reads)).
template <int NTL, int NTS, int kUnroll>
__global__ void __launch_bounds__(64 * kWavesPerGroup) stream_kernel(StreamArgs a)
{
    const uint32_t w = __builtin_amdgcn_readfirstlane(blockIdx.x * kWavesPerGroup +
                                                      (threadIdx.x >> 6));
    if (w >= a.waves)
        return;
    const uint32_t lane = threadIdx.x & 63;
    const uint64_t r0 = a.nr * w / a.waves, r1 = a.nr * (w + 1) / a.waves;
    const uint64_t w0 = a.nw * w / a.waves, w1 = a.nw * (w + 1) / a.waves;
    const uint64_t nr = r1 - r0, nw = w1 - w0;
    u32x4 acc = {0x9e3779b9u, 0x7f4a7c15u, 0x85ebca6bu, 0xc2b2ae35u};
    // credit counts reads times the wave's writes; each 64-granule store
    // spends 64 times its reads, so stores keep pace without a division
    uint64_t written = 0, credit = 0;
    const uint64_t unit = 64 * nr;
    for (uint64_t done = 0; done < nr;) {
        const uint64_t step = nr - done < (uint64_t)(64 * kUnroll) ? nr - done : 64 * kUnroll;
        u32x4 v[kUnroll];
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
            const uint64_t k = done + 64 * u + lane;
            // past the wave's range a lane reloads its last granule
            v[u] = ld<NTL>(a.src, r0 + (k < nr ? k : nr - 1));
        }
#pragma unroll
        for (int u = 0; u < kUnroll; ++u)
            acc ^= v[u];
        done += step;
        credit += step * nw;
        while (written < nw && (credit >= unit || done == nr)) {
            const uint64_t k = written + lane;
            if (k < nw)
                st<NTS>(a.dst, w0 + k, acc);
            written += 64;
            credit = credit >= unit ? credit - unit : 0;
        }
    }
    if (nr == 0) {
        for (; written < nw; written += 64 * kUnroll) {
#pragma unroll
            for (int u = 0; u < kUnroll; ++u) {
                const uint64_t k = written + 64 * u + lane;
                if (k < nw)
                    st<NTS>(a.dst, w0 + k, acc + (uint32_t)k);
            }
        }
    }
    // keep the loads of a pure read stream
    asm volatile("" ::"v"(acc.x), "v"(acc.y), "v"(acc.z), "v"(acc.w));
}

// Eight independent chains of one instruction (operands %0 .. %7 the chains,
// %8 and %9 shared sources, %10 a lane mask).
#define SMOL_V8(I) I("%0") I("%1") I("%2") I("%3") I("%4") I("%5") I("%6") I("%7")
#define SMOL_MUL(R) "v_mul_f32 " R ", " R ", %8\n\t"
#define SMOL_ADD(R) "v_add_f32 " R ", " R ", %8\n\t"
#define SMOL_FMA(R) "v_fma_f32 " R ", " R ", %8, %9\n\t"
#define SMOL_PERM(R) "v_perm_b32 " R ", " R ", %8, %9\n\t"
#define SMOL_ALIGN(R) "v_alignbyte_b32 " R ", " R ", %8, %9\n\t"
#define SMOL_DOT4(R) "v_dot4_u32_u8 " R ", %8, %9, " R "\n\t"
#define SMOL_MED3(R) "v_med3_f32 " R ", " R ", %8, %9\n\t"
#define SMOL_CVT(R) "v_cvt_f32_i32 " R ", " R "\n\t"
#define SMOL_MULU24(R) "v_mul_u32_u24 " R ", " R ", %8\n\t"
#define SMOL_MULLO(R) "v_mul_lo_u32 " R ", " R ", %8\n\t"
#define SMOL_MAX(R) "v_max_f32 " R ", " R ", %8\n\t"
#define SMOL_ADDU(R) "v_add_u32 " R ", " R ", %8\n\t"
#define SMOL_CND(R) "v_cndmask_b32_e64 " R ", " R ", %8, %10\n\t"
#define SMOL_UBYTE(R) "v_cvt_f32_ubyte0 " R ", " R "\n\t"
#define SMOL_AND(R) "v_and_b32 " R ", " R ", %8\n\t"
#define SMOL_VALU_STEP(BODY)                                                                     \
    asm volatile(SMOL_V8(BODY)                                                                   \
                 : "+v"(r[0]), "+v"(r[1]), "+v"(r[2]), "+v"(r[3]), "+v"(r[4]), "+v"(r[5]),     \
                   "+v"(r[6]), "+v"(r[7])                                                       \
                 : "v"(x), "v"(y), "s"(m))

// v_add_f32 on the eight chains, each followed by an s_add_u32 on one scalar
// chain (%8): whether scalar instructions take a wave's VALU issue slots.
#define SMOL_ADD_SALU(R) "v_add_f32 " R ", " R ", %9\n\ts_add_u32 %8, %8, 1\n\t"
#define SMOL_VALU_SALU_STEP                                                                      \
    asm volatile(SMOL_V8(SMOL_ADD_SALU)                                                          \
                 : "+v"(r[0]), "+v"(r[1]), "+v"(r[2]), "+v"(r[3]), "+v"(r[4]), "+v"(r[5]),     \
                   "+v"(r[6]), "+v"(r[7]), "+s"(sc)                                             \
                 : "v"(x)                                                                       \
                 : "scc")

template <int K>
__global__ void __launch_bounds__(64) valu_kernel(uint64_t *ticks, int32_t iters)
{
    uint32_t r[8];
#pragma unroll
    for (int k = 0; k < 8; ++k)
        r[k] = 0x3f800000u + 977u * (uint32_t)k + (uint32_t)threadIdx.x;
    const uint32_t x = 0x3f7ffff0u + (uint32_t)threadIdx.x, y = 0x3f800010u;
    const uint64_t m = 0x5555555555555555ull;
    uint32_t sc = 0;
    const uint64_t t0 = __builtin_amdgcn_s_memrealtime();
#pragma unroll 4
    for (int32_t it = 0; it < iters; ++it) {
        if constexpr (K == 0) SMOL_VALU_STEP(SMOL_MUL);
        else if constexpr (K == 1) SMOL_VALU_STEP(SMOL_ADD);
        else if constexpr (K == 2) SMOL_VALU_STEP(SMOL_FMA);
        else if constexpr (K == 3) SMOL_VALU_STEP(SMOL_PERM);
        else if constexpr (K == 4) SMOL_VALU_STEP(SMOL_ALIGN);
        else if constexpr (K == 5) SMOL_VALU_STEP(SMOL_DOT4);
        else if constexpr (K == 6) SMOL_VALU_STEP(SMOL_MED3);
        else if constexpr (K == 7) SMOL_VALU_STEP(SMOL_CVT);
        else if constexpr (K == 8) SMOL_VALU_STEP(SMOL_MULU24);
        else if constexpr (K == 9) SMOL_VALU_STEP(SMOL_MULLO);
        else if constexpr (K == 10) SMOL_VALU_STEP(SMOL_MAX);
        else if constexpr (K == 11) SMOL_VALU_STEP(SMOL_ADDU);
        else if constexpr (K == 12) SMOL_VALU_STEP(SMOL_CND);
        else if constexpr (K == 13) SMOL_VALU_STEP(SMOL_UBYTE);
        else if constexpr (K == 14) SMOL_VALU_STEP(SMOL_AND);
        else SMOL_VALU_SALU_STEP;
    }
    const uint64_t t1 = __builtin_amdgcn_s_memrealtime();
    // keep the chains
    asm volatile("" ::"v"(r[0]), "v"(r[1]), "v"(r[2]), "v"(r[3]), "v"(r[4]), "v"(r[5]),
                 "v"(r[6]), "v"(r[7]), "s"(sc));
    if (threadIdx.x == 0)
        ticks[blockIdx.x] = t1 - t0;
}
#undef SMOL_VALU_STEP
#undef SMOL_VALU_SALU_STEP

}  // namespace
}  // namespace smol

extern "C" int smol_valu_probe(int32_t kind, int32_t waves, int32_t iters, uint64_t *ticks,
                               void *stream)
{
    using namespace smol;
    clear_error();
    if (kind < 0 || kind >= SMOL_VALU_KINDS)
        return set_error(SMOL_ERR_INVALID_ARG, "kind %d unknown", kind);
    if (waves < 1 || waves > (1 << 20) || iters < 1 || iters > (1 << 20))
        return set_error(SMOL_ERR_INVALID_ARG, "waves and iters must be in 1 .. 2^20");
    if (!ticks)
        return set_error(SMOL_ERR_INVALID_ARG, "ticks is NULL");
    static const void *const kernels[SMOL_VALU_KINDS] = {
        (const void *)valu_kernel<0>, (const void *)valu_kernel<1>, (const void *)valu_kernel<2>,
        (const void *)valu_kernel<3>, (const void *)valu_kernel<4>, (const void *)valu_kernel<5>,
        (const void *)valu_kernel<6>, (const void *)valu_kernel<7>, (const void *)valu_kernel<8>,
        (const void *)valu_kernel<9>, (const void *)valu_kernel<10>, (const void *)valu_kernel<11>,
        (const void *)valu_kernel<12>, (const void *)valu_kernel<13>, (const void *)valu_kernel<14>,
        (const void *)valu_kernel<15>};
    void *args[] = {(void *)&ticks, (void *)&iters};
    const hipError_t e = hipLaunchKernel(kernels[kind], dim3((unsigned)waves), dim3(64), args, 0,
                                         (hipStream_t)stream);
    if (e != hipSuccess)
        return set_error(SMOL_ERR_HIP, "VALU probe launch: %s", hipGetErrorString(e));
    return SMOL_OK;
}

extern "C" int smol_stream_probe(const void *src, uint64_t read_bytes, void *dst,
                                 uint64_t write_bytes, int32_t waves, int32_t flags, void *stream)
{
    using namespace smol;
    clear_error();
    if (read_bytes % 16 || write_bytes % 16)
        return set_error(SMOL_ERR_INVALID_ARG, "sizes must be multiples of 16 bytes");
    if (read_bytes == 0 && write_bytes == 0)
        return set_error(SMOL_ERR_INVALID_ARG, "nothing to read or write");
    if ((read_bytes && (!src || (uintptr_t)src % 16)) ||
        (write_bytes && (!dst || (uintptr_t)dst % 16)))
        return set_error(SMOL_ERR_INVALID_ARG, "buffers must be non-null and 16-byte aligned");
    if (waves < 1 || waves > (1 << 20))
        return set_error(SMOL_ERR_INVALID_ARG, "waves must be in 1 .. 2^20");
    if (flags & ~(SMOL_STREAM_NT_LOADS | SMOL_STREAM_NT_STORES | SMOL_STREAM_DEEP))
        return set_error(SMOL_ERR_INVALID_ARG, "unknown flags");
    StreamArgs a;
    a.src = (const u32x4 *)src;
    a.dst = (u32x4 *)dst;
    a.nr = read_bytes / 16;
    a.nw = write_bytes / 16;
    a.waves = (uint32_t)waves;
    const dim3 grid((unsigned)((waves + kWavesPerGroup - 1) / kWavesPerGroup)),
        block(64 * kWavesPerGroup);
    hipStream_t s = (hipStream_t)stream;
    switch (flags) {
    case 0: hipLaunchKernelGGL((stream_kernel<0, 0, 4>), grid, block, 0, s, a); break;
    case 1: hipLaunchKernelGGL((stream_kernel<1, 0, 4>), grid, block, 0, s, a); break;
    case 2: hipLaunchKernelGGL((stream_kernel<0, 1, 4>), grid, block, 0, s, a); break;
    case 3: hipLaunchKernelGGL((stream_kernel<1, 1, 4>), grid, block, 0, s, a); break;
    case 4: hipLaunchKernelGGL((stream_kernel<0, 0, 8>), grid, block, 0, s, a); break;
    case 5: hipLaunchKernelGGL((stream_kernel<1, 0, 8>), grid, block, 0, s, a); break;
    case 6: hipLaunchKernelGGL((stream_kernel<0, 1, 8>), grid, block, 0, s, a); break;
    default: hipLaunchKernelGGL((stream_kernel<1, 1, 8>), grid, block, 0, s, a); break;
    }
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess)
        return set_error(SMOL_ERR_HIP, "stream probe launch: %s", hipGetErrorString(e));
    return SMOL_OK;
}
