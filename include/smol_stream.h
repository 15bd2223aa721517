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

#ifdef __cplusplus
}
#endif

#endif /* SMOL_STREAM_H */
