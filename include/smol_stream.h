/*
 * smol_stream.h -- streaming-bandwidth probe of libsmol.
 *
 * The preprocessing path moves bytes and does little arithmetic per byte
 * (section 2's steps 2-4 on decoded pixels), so its roofline is the device's
 * memory bandwidth. This call measures what plain streams reach on the same
 * device: a kernel that reads `read_bytes` from `src` and writes
 * `write_bytes` to `dst` in one launch, both as coalesced 16-byte accesses,
 * every wave interleaving its reads and writes in the ratio of the two
 * sizes. With write_bytes = 0 it is a pure read stream, with read_bytes = 0
 * a pure write stream, with equal sizes a copy, and with the byte mix of a
 * preprocessing launch (for example 83 % reads, 17 % writes for 1080p frames
 * reduced to 224 x 224 fp16) the ceiling that launch can be compared with.
 * Timing is the caller's (events around launches on `stream`).
 */
#ifndef SMOL_STREAM_H
#define SMOL_STREAM_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Flags of smol_stream_probe. */
#define SMOL_STREAM_NT_LOADS 1  /* nontemporal loads (else ordinary loads)   */
#define SMOL_STREAM_NT_STORES 2 /* nontemporal stores (else ordinary stores) */
#define SMOL_STREAM_DEEP 4      /* 8 loads in flight per lane (else 4)       */

/* Enqueue one streaming launch on `stream` (a hipStream_t; NULL = the null
 * stream).
 *   src, read_bytes    DEVICE buffer read whole; read_bytes a multiple of 16
 *                      (0: no reads, src may be NULL); 16-byte aligned
 *   dst, write_bytes   DEVICE buffer written whole; a multiple of 16 (0: no
 *                      writes, dst may be NULL); 16-byte aligned. The
 *                      written values depend on the data read (a fixed
 *                      pattern when nothing is read).
 *   waves              number of 64-lane waves of the launch (1 .. 2^20)
 *   flags              SMOL_STREAM_* bits
 * Both buffers are owned by the caller and must stay alive until the work on
 * `stream` completes. Returns SMOL_OK, SMOL_ERR_INVALID_ARG (sizes not
 * multiples of 16, misaligned or NULL pointers for nonzero sizes, waves out
 * of range, both sizes 0) or SMOL_ERR_HIP; nothing is enqueued on error. */
int smol_stream_probe(const void *src, uint64_t read_bytes, void *dst, uint64_t write_bytes,
                      int32_t waves, int32_t flags, void *stream);

/* Instruction kinds of smol_valu_probe. */
#define SMOL_VALU_MUL_F32 0     /* v_mul_f32          */
#define SMOL_VALU_ADD_F32 1     /* v_add_f32          */
#define SMOL_VALU_FMA_F32 2     /* v_fma_f32          */
#define SMOL_VALU_PERM 3        /* v_perm_b32         */
#define SMOL_VALU_ALIGNBYTE 4   /* v_alignbyte_b32    */
#define SMOL_VALU_DOT4 5        /* v_dot4_u32_u8      */
#define SMOL_VALU_MED3_F32 6    /* v_med3_f32         */
#define SMOL_VALU_CVT_F32_I32 7 /* v_cvt_f32_i32      */
#define SMOL_VALU_MUL_U24 8     /* v_mul_u32_u24      */
#define SMOL_VALU_MUL_LO_U32 9  /* v_mul_lo_u32       */
#define SMOL_VALU_MAX_F32 10    /* v_max_f32          */
#define SMOL_VALU_ADD_U32 11    /* v_add_u32          */
#define SMOL_VALU_CNDMASK 12    /* v_cndmask_b32      */
#define SMOL_VALU_CVT_F32_UBYTE0 13 /* v_cvt_f32_ubyte0 */
#define SMOL_VALU_AND_B32 14    /* v_and_b32          */
#define SMOL_VALU_ADD_F32_SALU 15 /* v_add_f32, each followed by an s_add_u32 */
#define SMOL_VALU_KINDS 16

/* The issue rate of one kind of VALU instruction, the other ceiling of the
 * preprocessing kernels (the I420 path and the block decoder spend more time
 * issuing VALU instructions than moving bytes). Enqueue one launch of
 * `waves` one-wave workgroups; each wave issues `iters` x 8 instructions of
 * `kind` on eight independent register chains (inline assembly, so nothing
 * is folded away) and writes the time it took, in ticks of the 100 MHz
 * real-time counter, to ticks[w] for its index w.
 *   kind    SMOL_VALU_*
 *   waves   1 .. 2^20 (the device's SIMDs take them round robin: 1024 waves
 *           put one on each SIMD of a 256-CU part)
 *   iters   1 .. 2^20
 *   ticks   DEVICE buffer of `waves` uint64 values, owned by the caller
 * Returns SMOL_OK, SMOL_ERR_INVALID_ARG (kind unknown, waves or iters out of
 * range, ticks NULL) or SMOL_ERR_HIP; nothing is enqueued on error. */
int smol_valu_probe(int32_t kind, int32_t waves, int32_t iters, uint64_t *ticks, void *stream);

#ifdef __cplusplus
}
#endif

#endif /* SMOL_STREAM_H */
