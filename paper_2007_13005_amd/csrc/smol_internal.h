// smol_internal.h -- types shared by the host side and the kernels of libsmol.
#pragma once

#include <stddef.h>
#include <stdint.h>

#include "smol.h"

namespace smol {

// Per-image descriptor, 80 bytes. For RGB input off[0] is the byte offset of
// the first pixel of the processed region (the image, or its ROI) and W x H
// its size; for I420 input off[0..2] are the Y, Cb and Cr plane offsets of
// the frame, W x H the size of the processed region, (rx, ry) its origin in
// the frame, pitch the frame's luma width and fh its luma height. Wr/Hr are
// the resized sizes and left/top the crop offsets (host-computed per image;
// per-element taps are computed by the kernels). xf is the first column of
// the region any output pixel reads and span the bytes from that column's
// first byte to the end of the last column read (luma bytes for I420); safe
// is 1 when every 16-byte aligned chunk that holds a byte of a staged row
// lies inside src.
struct alignas(16) Desc {
    int64_t off[3];
    int32_t W, H, pitch, Wr, Hr, left, top, xf;
    int32_t span, safe;
    int32_t rx, ry, fh, pad;
};
static_assert(sizeof(Desc) == 80, "descriptor must be 80 bytes");

// Kernel arguments (passed by value). When `table` is null every image shares
// `uni` and image i's offsets are uni.off[k] + i * stride.
struct BatchArgs {
    const uint8_t *src;
    int64_t src_bytes;
    const Desc *table;
    Desc uni;
    int64_t stride;
    void *out;
    int32_t n;
    int32_t Ch, Cw;
    int32_t R;       // output rows per workgroup band (LDS kernels)
    int32_t bands;   // ceil(Ch / R)
    int32_t slot_bytes;  // bytes per staged source-row slot (LDS kernels)
    int32_t slots_off;   // byte offset of the first slot in dynamic LDS
    int32_t cslot_bytes; // bytes per staged chroma-row slot (I420 LDS kernel)
    int32_t cslots_off;
    int32_t img_base;    // index of this launch's first image in the output
    int32_t grid;        // workgroups of a persistent launch (LDS kernels)
    int32_t stage_bytes; // bytes of one of the two LDS buffers of a wave
    int32_t row_groups;  // 1 KiB chunk groups per staged source row (row-streaming kernel)
    int32_t col_iters;   // column pairs per lane: 1, 2 or 4 (row-streaming kernel)
    int32_t prefetch;    // rows loaded ahead of the one interpolated: 1 or 2 (row streaming)
    int32_t interleave;  // row streaming: wave q takes rows q, q + G, ... (else a range)
    int32_t exact;       // 1: operation-by-operation fp32 arithmetic (row-streaming kernel)
    int32_t wpg;         // row streaming: waves per workgroup (grid = waves / wpg)
    // Row streaming, from the host: the n * Ch rows are rows_q * grid + rows_r
    // (wave w walks rows_q rows, one more when w < rows_r), and a strided walk
    // steps by grid rows = step_di images and step_dr rows.
    int32_t rows_q, rows_r;
    int32_t step_di, step_dr;
    // Strided walk of a uniform batch: floor quotient and remainder of
    // 2 H step_dr and of 2 H (step_dr - Ch) by 2 Hr (the vertical map's
    // steps within an image and across a wrap), from the host.
    int32_t vq_s, vr_s, vq_w, vr_w;
    int32_t nhwc;        // 1: output n x Ch x Cw x 3 (row-streaming and direct kernels)
    int32_t siting;      // I420 chroma columns: 0 centred (x/2 - 1/4), 1 co-sited (x/2)
    float mean[3];   // per channel, 0..255 units
    float stdv[3];
    float rcp[3];    // RN(1 / stdv), fp32
    float bias[3];   // RN(-mean / stdv), fp32
};

enum Path { PATH_AUTO = 0, PATH_DIRECT = 1, PATH_LDS = 2, PATH_GATHER = 3, PATH_ROWS = 4 };

// Pseudo path of the I420 row-streaming kernel in run_batch (reported as PATH_ROWS).
constexpr int PATH_YUV_ROWS = 5;

// Row-streaming kernel limits: crops up to 2 * 64 * kRowsMaxColIters columns,
// staged source rows (span + 32 bytes) up to kRowsMaxGroups KiB.
constexpr int kRowsMaxColIters = 4;
constexpr int kRowsMaxGroups = 4;
// Waves per workgroup of the row-streaming kernels (each wave independent).
constexpr int kRowsMaxWavesPerGroup = 4;

// Block decoding (smol_jpeg_kernels.hip). A launch decodes up to
// kJpegMaxRuns runs; a run is `frames` frames of one geometry and one pair of
// dequantisation tables (q[qt]) whose coefficients start at element coef
// (from JpegArgs::coef) and step by coef_stride, and whose Y planes start at
// byte out (from JpegArgs::out) and step by out_stride, the Cb and Cr planes
// cboff / croff bytes after the Y plane (W x H and ceil(W/2) x ceil(H/2),
// tightly pitched). The coefficients hold the blocks of MCU columns wx0 ..
// wx0 + wmx - 1 and rows wy0 .. wy0 + wmy - 1 (the whole frame, or a
// rectangle's MCU window): luma blocks 2 wmx x 2 wmy, then Cb and Cr
// wmx x wmy, 64 each in natural order. Luma blocks lbx0 .. lbx0 + lnbx - 1
// (rows likewise) and chroma blocks cbx0 .. are decoded; jobs_end counts the
// kernel's jobs (groups of up to eight blocks along a block row) of this and
// the earlier runs.
constexpr int kJpegMaxRuns = 24;
constexpr int kJpegMaxTables = 8;
struct JpegRun {
    long long coef, coef_stride, out, out_stride, cboff, croff;
    int32_t W, H;
    int16_t wx0, wy0, wmx, wmy;
    int16_t lbx0, lby0, lnbx, lnby, cbx0, cby0, cnbx, cnby;
    // Jobs of a frame: lum = lg * lnby luma groups (lg groups of up to eight
    // blocks per block row), then chr = cg * cnby groups of each chroma
    // plane; a row's last group holds lrem (cg: crem) blocks.
    uint32_t lum, chr;
    uint32_t jobs_end;  // < 2^31
    // Division by a divisor d of the run (jobs per frame, lg, cg) as
    // floor(n m / 2^s) with m = ceil(2^s / d), s = 31 + ceil(log2 d): exact
    // for every n < 2^31.
    uint32_t m_pf, m_lg, m_cg;
    uint32_t groups;  // lg | cg << 11 | lrem << 22 | crem << 26
    uint32_t shifts;  // s of the frame's jobs | s of lg << 8 | s of cg << 16 | qt << 24
};
struct JpegArgs {
    const int16_t *coef;
    uint8_t *out;
    int32_t runs, pad;
    uint8_t q[kJpegMaxTables][2][64];  // luma, chroma dequantisation (entries 1..255)
    float c[64];                       // c[k * 8 + n] = fp32(C(k)/2 cos((2n + 1) k pi / 16))
    JpegRun run[kJpegMaxRuns];
};
static_assert(sizeof(JpegRun) == 112, "run table entry of block decoding");
static_assert(sizeof(JpegArgs) <= 4096, "kernel arguments of block decoding");
int launch_jpeg_idct(const JpegArgs &a, int grid, void *stream);

// The MCU-aligned rectangle (x, y, w, h) holding every luma and chroma sample
// the preprocessing of a W x H 4:2:0 frame reads (smol_host.cpp). Returns a
// status; fails as the batch calls would on these parameters.
int mcu_rect(int64_t W, int64_t H, const smol_params *p, int resize_mode, int32_t rect[4]);

// smol_preprocess_batch_noalloc keeps a ragged batch's descriptor table in a
// fixed device array of kNoallocTableBytes (smol_scratch.hip) instead of
// memory the library allocates. scratch_table() returns that array's device
// address on `device` (the current device), looked up once per device.
constexpr int kNoallocMaxImages = SMOL_NOALLOC_MAX_IMAGES;
constexpr size_t kNoallocTableBytes = (size_t)kNoallocMaxImages * sizeof(Desc);
int scratch_table(int device, void **table);

// Adds k launches to the calling thread's last plan (smol_last_plan), for
// calls made of several library calls (partial JPEG decoding).
void add_plan_launches(int k);

// Device compute units (0 when unknown).
int device_cus();

// The calling thread's smol_last_error() message (smol_host.cpp): set_error
// formats it and returns `code`; clear_error empties it.
int set_error(int code, const char *fmt, ...);
void clear_error();

// Launchers (smol_kernels.hip). Return a hipError_t as int. `done`, where
// given, is an event (or null) that the launch itself signals when the kernel
// completes.
// Copies `bytes` (a multiple of 16) from src to dst with a small kernel on
// `stream` (src may be pinned host memory as the device addresses it).
int launch_table_copy(const void *src, void *dst, size_t bytes, void *stream);
// Direct kernels: out_type 0 fp32, 1 fp16, 2 uint8 (rounded, not normalised).
int launch_rgb_direct(const BatchArgs &a, int out_type, void *stream, void *done);
int launch_rgb_lds(const BatchArgs &a, int out_f16, size_t lds_bytes, void *stream, void *done);
int launch_rgb_gather(const BatchArgs &a, int out_f16, size_t lds_bytes, void *stream, void *done);
// Row-streaming launches: `lds_bytes` is one wave's slot; a workgroup holds
// a.wpg waves and a.grid is the number of waves (a multiple of a.wpg).
int launch_rgb_rows(const BatchArgs &a, int out_f16, size_t lds_bytes, void *stream, void *done);
// Resident workgroups of a.wpg waves per compute unit.
int occupancy_rgb_rows(const BatchArgs &a, int out_f16, size_t lds_bytes, int *blocks_per_cu);
// Resident workgroups per compute unit for the persistent kernels.
int occupancy_rgb_gather(int out_f16, size_t lds_bytes, int *blocks_per_cu);
int occupancy_rgb_lds(int out_f16, size_t lds_bytes, int *blocks_per_cu);
int launch_yuv_direct(const BatchArgs &a, int out_type, void *stream, void *done);
int launch_yuv_rows(const BatchArgs &a, int out_f16, size_t lds_bytes, void *stream, void *done);
int occupancy_yuv_rows(const BatchArgs &a, int out_f16, size_t lds_bytes, int *blocks_per_cu);

// Row-streaming kernels for the plan in the arguments (the file of each part:
// smol_rows_<input>_<walk>[_nhwc].hip); `interleave` picks the walk, `nhwc`
// the output layout.
const void *rows_rgb_f16_range(const BatchArgs &a);
const void *rows_rgb_f16_range_nhwc(const BatchArgs &a);
const void *rows_rgb_f16_stride(const BatchArgs &a);
const void *rows_rgb_f16_stride_nhwc(const BatchArgs &a);
const void *rows_rgb_f32_range(const BatchArgs &a);
const void *rows_rgb_f32_range_nhwc(const BatchArgs &a);
const void *rows_rgb_f32_stride(const BatchArgs &a);
const void *rows_rgb_f32_stride_nhwc(const BatchArgs &a);
const void *rows_rgb_u8_range(const BatchArgs &a);  // uint8: contiguous ranges only
const void *rows_rgb_u8_range_nhwc(const BatchArgs &a);
const void *rows_yuv_range(const BatchArgs &a, int f16);
const void *rows_yuv_range_nhwc(const BatchArgs &a, int f16);
const void *rows_yuv_stride(const BatchArgs &a, int f16);
const void *rows_yuv_stride_nhwc(const BatchArgs &a, int f16);

}  // namespace smol
