/*
 * smol_pipeline.h -- pipelined ingest around the fused preprocessing calls of
 * smol.h: reused pinned host buffers, host-to-device copies on several HIP
 * streams overlapped with the preprocessing kernels of earlier batches, and a
 * caller-supplied consumer (the DNN) enqueued behind each batch.
 *
 * What it follows: section 6.1 ("Efficient Use of Hardware") -- producers
 * that decode into buffers and consumers that execute the DNN, linked by a
 * multi-producer multi-consumer queue; several streams; pinned memory that is
 * reused rather than handed to the caller; more buffers than consumers so
 * that producers do not wait on them -- and the cost model of section 4
 * ("Corrected throughput estimation", Eq. 4): with the stages pipelined, the
 * throughput is about the minimum of the stages' throughputs.
 *
 * Model. A pipeline owns `slots` buffer sets, each a pinned host input buffer
 * of `input_bytes`, a device input buffer of the same size and a device output
 * buffer of `output_bytes`, `streams` compute streams and `copy_streams`
 * copy streams (HIP streams of default priority on the device current at
 * creation). A producer thread acquires a free slot, writes a batch of
 * images into its host buffer (the decoder's output) and submits it; the
 * submission enqueues the copy of the batch's bytes to the device on the
 * next copy stream, and on the next compute stream (both in round-robin
 * order) a wait for that copy, the preprocessing call into the slot's device
 * output and then the consumer, and returns. Copies of later batches thus
 * run while earlier batches are preprocessed and consumed. A slot becomes
 * free again when all of its work has completed on the device; acquiring a
 * slot when none is free waits for the oldest submission.
 *
 * Threading. Every call is thread-safe: any number of producer threads may
 * acquire and submit concurrently (the queue is multi-producer; the streams
 * are its consumers). A slot belongs to the thread that acquired it until it
 * submits or releases it.
 *
 * Errors. Calls return SMOL_OK or a negative status of smol.h, with a
 * message in smol_last_error(). A submission whose own arguments (slot,
 * byte count, output size) are invalid enqueues nothing and leaves the slot
 * acquired. Once the copy is enqueued, a failure of the preprocessing call
 * (its validation included) or of the consumer is returned, and the slot
 * still completes in stream order and is recycled.
 */
#ifndef SMOL_PIPELINE_H
#define SMOL_PIPELINE_H

#include <stdint.h>

#include "smol.h"

#ifdef __cplusplus
extern "C" {
#endif

typedef struct smol_pipeline smol_pipeline;

/* Pipeline sizes.
 *   slots         buffer sets, 1 .. 64 (more than `streams` lets producers
 *                 fill one while the others are in flight)
 *   streams       compute streams, 1 .. 16
 *   input_bytes   bytes of each host / device input buffer, >= 1
 *   output_bytes  bytes of each device output buffer, >= 16
 *   copy_streams  copy streams, 0 .. 4 (0: one)
 *   workspace_bytes  device workspace per slot for smol_pipeline_submit_jpeg
 *                 (at least smol_jpeg_workspace_bytes of its batches), >= 0
 * Device memory held: slots * (input_bytes + output_bytes + workspace_bytes);
 * pinned host memory: slots * input_bytes. */
typedef struct smol_pipeline_config {
    int32_t slots;
    int32_t streams;
    int64_t input_bytes;
    int64_t output_bytes;
    int32_t copy_streams;
    int32_t reserved;  /* must be zero */
    int64_t workspace_bytes;
} smol_pipeline_config;

/* The DNN stage, called on the submitting thread right after the
 * preprocessing launch: it must enqueue its work on `stream` (a hipStream_t)
 * reading the n preprocessed images at `output` (DEVICE, the slot's output
 * buffer, valid in stream order until the work enqueued here completes) and
 * return 0, or nonzero to report a failure.
 *
 * Contract (the submitting thread still holds the slot while the consumer
 * runs):
 *   - all of its device work goes on `stream`: the slot is recycled when the
 *     work on `stream` up to the submission's end completes, so work put on
 *     other streams is not covered by the slot and is not throttled by the
 *     pool of slots;
 *   - it must not wait on the host for device work, and must not call
 *     smol_pipeline_acquire, _submit*, _drain or _destroy of the same
 *     pipeline: with every slot held by producers inside their consumers, a
 *     consumer waiting for a slot or for completions waits forever;
 *   - it may call the library's batch calls on `stream` (they only enqueue).
 * The Python binding runs Python consumers with torch's current stream set to
 * `stream` and refuses those pipeline calls from inside a consumer. */
typedef int (*smol_consumer_fn)(void *user, const void *output, int32_t n, void *stream);

/* smol_pipeline_create -- allocate the buffers, streams and events on the
 * current device. *out receives the pipeline (NULL on failure). Returns
 * SMOL_OK, SMOL_ERR_INVALID_ARG (a size out of range, reserved nonzero) or
 * SMOL_ERR_HIP (an allocation failed; nothing is kept). */
int smol_pipeline_create(const smol_pipeline_config *config, smol_pipeline **out);

/* smol_pipeline_destroy -- wait for every submission to complete, then free
 * everything. NULL is a no-op. No other call on the pipeline may run
 * concurrently or follow. */
int smol_pipeline_destroy(smol_pipeline *p);

/* smol_pipeline_acquire -- a free slot for the calling producer: *slot its
 * index, *host its pinned host input buffer (input_bytes, HOST-writable
 * until the slot is submitted), *output its device output buffer. Waits for
 * the oldest in-flight submission when no slot is free, and for another
 * producer's submit or release when every slot is acquired (a thread that
 * holds every slot itself would wait forever). */
int smol_pipeline_acquire(smol_pipeline *p, int32_t *slot, void **host, void **output);

/* smol_pipeline_release -- give back an acquired slot without submitting. */
int smol_pipeline_release(smol_pipeline *p, int32_t slot);

/* smol_pipeline_submit -- enqueue the slot's batch: copy the first `bytes`
 * (1 .. input_bytes) bytes of its host buffer to its device input buffer,
 * preprocess them with smol_preprocess_batch_ex into the slot's output
 * buffer (tables and offsets relative to the start of the buffer, src_bytes
 * = bytes), then call `consumer` (may be NULL). The n images' output must
 * fit output_bytes. Host tables are read before the call returns. Returns as
 * smol_preprocess_batch_ex; see Errors above for the slot's state. */
int smol_pipeline_submit(smol_pipeline *p, int32_t slot, int64_t bytes, const int64_t *offsets,
                         const int32_t *widths, const int32_t *heights,
                         const int32_t *row_pitch, const int32_t *rois, int32_t n,
                         const smol_params *params, const smol_options *opts,
                         smol_consumer_fn consumer, void *user);

/* smol_pipeline_submit_yuv420 -- the same for planar I420 frames
 * (smol_yuv420_preprocess_batch_ex). */
int smol_pipeline_submit_yuv420(smol_pipeline *p, int32_t slot, int64_t bytes,
                                const int64_t *y_offsets, const int64_t *cb_offsets,
                                const int64_t *cr_offsets, const int32_t *widths,
                                const int32_t *heights, const int32_t *rois, int32_t n,
                                const smol_params *params, const smol_options *opts,
                                smol_consumer_fn consumer, void *user);

/* smol_pipeline_submit_jpeg -- the same for entropy-decoded JPEG batches
 * (smol_jpeg_roi_preprocess_batch): the slot's host buffer holds the int16
 * coefficients (`bytes` even) as smol_jpeg_entropy_decode_batch wrote them,
 * tables relative to its start; the slot's workspace (workspace_bytes at
 * creation, nonzero) takes the decoded planes. Producer threads can thus
 * entropy-decode straight into the pinned slot they acquired (section 6.1's
 * decoder threads feeding the queue). */
int smol_pipeline_submit_jpeg(smol_pipeline *p, int32_t slot, int64_t bytes,
                              const int64_t *coef_offsets, const uint16_t *qtables,
                              int32_t n_qtables, const int32_t *widths, const int32_t *heights,
                              int32_t n, int32_t coef_layout, const smol_params *params,
                              const smol_options *opts, smol_consumer_fn consumer, void *user);

/* smol_pipeline_drain -- wait until every submission so far has completed
 * and its slot is free. */
int smol_pipeline_drain(smol_pipeline *p);

/* Counters since creation. */
typedef struct smol_pipeline_stats {
    int64_t submitted;      /* batches submitted                           */
    int64_t completed;      /* batches whose slot has been recycled        */
    int64_t images;         /* images submitted                            */
    int64_t bytes_copied;   /* host-to-device bytes submitted              */
    int64_t acquire_waits;  /* acquisitions that had to wait for a slot    */
    int64_t reserved[3];
} smol_pipeline_stats;

int smol_pipeline_get_stats(smol_pipeline *p, smol_pipeline_stats *stats);

#ifdef __cplusplus
}
#endif

#endif /* SMOL_PIPELINE_H */
