// smol_pipeline.cpp -- pipelined ingest: a pool of buffer sets (pinned host
// input, device input, device output), producer threads that acquire and
// submit them, copy streams that move each batch to the device, and compute
// streams on which its preprocessing and consumer run once its copy is done,
// while the copy streams already move later batches (section 6.1; Eq. 4 is
// the throughput model this overlap serves).
#include <hip/hip_runtime.h>

#include <condition_variable>
#include <cstdint>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "smol.h"
#include "smol_internal.h"
#include "smol_jpeg.h"
#include "smol_pipeline.h"

namespace {

enum SlotState { kFree, kAcquired, kInFlight };

struct Slot {
    uint8_t *host = nullptr;    // pinned, input_bytes
    uint8_t *dev_in = nullptr;  // input_bytes
    uint8_t *dev_out = nullptr; // output_bytes
    uint8_t *dev_ws = nullptr;  // workspace_bytes (JPEG submissions)
    hipEvent_t copied = nullptr; // after the slot's input copy
    hipEvent_t done = nullptr;  // after the slot's last consumer
    SlotState state = kFree;
    uint64_t seq = 0;           // submission number while in flight
};

constexpr int kMaxSlots = 64;
constexpr int kMaxStreams = 16;
constexpr int kMaxCopyStreams = 4;

}  // namespace

struct smol_pipeline {
    int device = 0;
    int64_t input_bytes = 0;
    int64_t output_bytes = 0;
    int64_t workspace_bytes = 0;
    std::vector<hipStream_t> streams;       // preprocessing and consumers
    std::vector<hipStream_t> copy_streams;  // host-to-device copies
    std::vector<Slot> slots;
    std::mutex mu;
    std::condition_variable cv;  // a slot was submitted or released
    uint64_t next_seq = 0;
    smol_pipeline_stats stats = {};
};

namespace {

int hip_error(hipError_t e, const char *what)
{
    return smol::set_error(SMOL_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

void free_all(smol_pipeline *p)
{
    for (Slot &s : p->slots) {
        if (s.done)
            (void)hipEventDestroy(s.done);
        if (s.copied)
            (void)hipEventDestroy(s.copied);
        if (s.host)
            (void)hipHostFree(s.host);
        if (s.dev_in)
            (void)hipFree(s.dev_in);
        if (s.dev_out)
            (void)hipFree(s.dev_out);
        if (s.dev_ws)
            (void)hipFree(s.dev_ws);
    }
    for (hipStream_t st : p->streams)
        if (st)
            (void)hipStreamDestroy(st);
    for (hipStream_t st : p->copy_streams)
        if (st)
            (void)hipStreamDestroy(st);
    p->slots.clear();
    p->streams.clear();
    p->copy_streams.clear();
}

// Marks completed in-flight slots free. Caller holds p->mu.
void reap(smol_pipeline *p)
{
    for (Slot &s : p->slots)
        if (s.state == kInFlight && hipEventQuery(s.done) == hipSuccess) {
            s.state = kFree;
            ++p->stats.completed;
        }
}

// Waits on the host for the oldest in-flight slot and frees it; false when
// none is in flight. Caller holds `lk` on p->mu (released while waiting).
bool wait_oldest(smol_pipeline *p, std::unique_lock<std::mutex> &lk, hipError_t *err)
{
    int oldest = -1;
    for (int i = 0; i < (int)p->slots.size(); ++i)
        if (p->slots[i].state == kInFlight &&
            (oldest < 0 || p->slots[i].seq < p->slots[oldest].seq))
            oldest = i;
    *err = hipSuccess;
    if (oldest < 0)
        return false;
    const hipEvent_t ev = p->slots[oldest].done;
    const uint64_t seq = p->slots[oldest].seq;
    lk.unlock();
    *err = hipEventSynchronize(ev);
    lk.lock();
    Slot &s = p->slots[oldest];
    if (*err == hipSuccess && s.state == kInFlight && s.seq == seq) {
        s.state = kFree;
        ++p->stats.completed;
    }
    return true;
}

// Makes the pipeline's device current for the calling thread for the
// lifetime of the guard.
struct DeviceGuard {
    int old = -1;
    hipError_t err = hipSuccess;
    explicit DeviceGuard(int device)
    {
        int cur = -1;
        err = hipGetDevice(&cur);
        if (err == hipSuccess && cur != device) {
            err = hipSetDevice(device);
            if (err == hipSuccess)
                old = cur;
        }
    }
    ~DeviceGuard()
    {
        if (old >= 0)
            (void)hipSetDevice(old);
    }
};

int64_t output_bytes_of(const smol_params *params, int32_t n)
{
    const int64_t esz = params->out_dtype == SMOL_OUT_F32   ? 4
                        : params->out_dtype == SMOL_OUT_F16 ? 2
                                                            : 1;
    return (int64_t)n * 3 * params->crop_h * params->crop_w * esz;
}

// Shared part of the submissions: argument checks, the copy, the
// preprocessing call `pre(src, bytes, out, workspace, stream)`, the consumer
// and the completion event.
template <class Pre>
int submit(smol_pipeline *p, int32_t slot, int64_t bytes, int32_t n, const smol_params *params,
           smol_consumer_fn consumer, void *user, Pre pre)
{
    smol::clear_error();
    if (!p)
        return smol::set_error(SMOL_ERR_INVALID_ARG, "pipeline is NULL");
    if (slot < 0 || slot >= (int32_t)p->slots.size())
        return smol::set_error(SMOL_ERR_INVALID_ARG, "slot %d outside 0..%d", slot,
                               (int)p->slots.size() - 1);
    if (bytes < 1 || bytes > p->input_bytes)
        return smol::set_error(SMOL_ERR_INVALID_ARG, "bytes %lld outside 1..%lld",
                               (long long)bytes, (long long)p->input_bytes);
    if (!params || n < 0)
        return smol::set_error(SMOL_ERR_INVALID_ARG, "params is NULL or n < 0");
    if (output_bytes_of(params, n) > p->output_bytes)
        return smol::set_error(SMOL_ERR_INVALID_ARG, "output of %lld bytes exceeds the slot's %lld",
                               (long long)output_bytes_of(params, n), (long long)p->output_bytes);
    hipStream_t s, cs;
    uint64_t seq;
    {
        std::lock_guard<std::mutex> lk(p->mu);
        if (p->slots[slot].state != kAcquired)
            return smol::set_error(SMOL_ERR_INVALID_ARG, "slot %d is not acquired", slot);
        seq = p->next_seq++;
        s = p->streams[seq % p->streams.size()];
        cs = p->copy_streams[seq % p->copy_streams.size()];
    }
    DeviceGuard dg(p->device);
    if (dg.err != hipSuccess)
        return hip_error(dg.err, "hipSetDevice");
    Slot &sl = p->slots[slot];
    // the copy on a copy stream; the compute stream waits for it
    hipError_t e = hipMemcpyAsync(sl.dev_in, sl.host, (size_t)bytes, hipMemcpyHostToDevice, cs);
    if (e != hipSuccess)
        return hip_error(e, "hipMemcpyAsync(input)");
    e = hipEventRecord(sl.copied, cs);
    if (e == hipSuccess)
        e = hipStreamWaitEvent(s, sl.copied, 0);
    if (e != hipSuccess) {
        // the copy is enqueued: wait for it so that the slot is free again
        const hipError_t e2 = hipStreamSynchronize(cs);
        std::lock_guard<std::mutex> lk(p->mu);
        sl.state = kFree;
        p->cv.notify_all();
        return hip_error(e2 != hipSuccess ? e2 : e, "copy event");
    }
    int rc = pre(sl.dev_in, bytes, sl.dev_out, sl.dev_ws, s);
    std::string msg = rc ? smol_last_error() : "";
    if (!rc && consumer) {
        const int c = consumer(user, sl.dev_out, n, s);
        if (c) {
            rc = SMOL_ERR_INVALID_ARG;
            msg = "consumer returned " + std::to_string(c);
        }
    }
    e = hipEventRecord(sl.done, s);
    if (e != hipSuccess) {
        // without the event the slot's completion is the stream's
        const hipError_t e2 = hipStreamSynchronize(s);
        std::lock_guard<std::mutex> lk(p->mu);
        sl.state = kFree;
        p->cv.notify_all();
        return hip_error(e2 != hipSuccess ? e2 : e, "hipEventRecord(slot)");
    }
    {
        std::lock_guard<std::mutex> lk(p->mu);
        sl.seq = seq;
        sl.state = kInFlight;
        p->stats.submitted += 1;
        p->stats.images += n;
        p->stats.bytes_copied += bytes;
    }
    p->cv.notify_all();
    if (rc)
        return smol::set_error(rc, "%s", msg.c_str());
    return SMOL_OK;
}

}  // namespace

extern "C" {

int smol_pipeline_create(const smol_pipeline_config *c, smol_pipeline **out)
{
    smol::clear_error();
    if (!out)
        return smol::set_error(SMOL_ERR_INVALID_ARG, "out is NULL");
    *out = nullptr;
    if (!c)
        return smol::set_error(SMOL_ERR_INVALID_ARG, "config is NULL");
    if (c->slots < 1 || c->slots > kMaxSlots)
        return smol::set_error(SMOL_ERR_INVALID_ARG, "slots %d outside 1..%d", c->slots,
                               kMaxSlots);
    if (c->streams < 1 || c->streams > kMaxStreams)
        return smol::set_error(SMOL_ERR_INVALID_ARG, "streams %d outside 1..%d", c->streams,
                               kMaxStreams);
    if (c->copy_streams < 0 || c->copy_streams > kMaxCopyStreams)
        return smol::set_error(SMOL_ERR_INVALID_ARG, "copy_streams %d outside 0..%d",
                               c->copy_streams, kMaxCopyStreams);
    if (c->input_bytes < 1 || c->output_bytes < 16)
        return smol::set_error(SMOL_ERR_INVALID_ARG, "input_bytes %lld < 1 or output_bytes %lld "
                               "< 16", (long long)c->input_bytes, (long long)c->output_bytes);
    if (c->reserved)
        return smol::set_error(SMOL_ERR_INVALID_ARG, "reserved is not zero");
    if (c->workspace_bytes < 0)
        return smol::set_error(SMOL_ERR_INVALID_ARG, "workspace_bytes %lld < 0",
                               (long long)c->workspace_bytes);
    smol_pipeline *p = new smol_pipeline();
    p->input_bytes = c->input_bytes;
    p->output_bytes = c->output_bytes;
    p->workspace_bytes = c->workspace_bytes;
    hipError_t e = hipGetDevice(&p->device);
    p->slots.resize((size_t)c->slots);
    p->streams.resize((size_t)c->streams, nullptr);
    p->copy_streams.resize((size_t)(c->copy_streams ? c->copy_streams : 1), nullptr);
    for (int i = 0; e == hipSuccess && i < c->streams; ++i)
        e = hipStreamCreateWithFlags(&p->streams[i], hipStreamNonBlocking);
    for (int i = 0; e == hipSuccess && i < (int)p->copy_streams.size(); ++i)
        e = hipStreamCreateWithFlags(&p->copy_streams[i], hipStreamNonBlocking);
    for (int i = 0; e == hipSuccess && i < c->slots; ++i) {
        Slot &s = p->slots[i];
        e = hipHostMalloc((void **)&s.host, (size_t)c->input_bytes, hipHostMallocDefault);
        if (e == hipSuccess)
            e = hipMalloc((void **)&s.dev_in, (size_t)c->input_bytes);
        if (e == hipSuccess)
            e = hipMalloc((void **)&s.dev_out, (size_t)c->output_bytes);
        if (e == hipSuccess && c->workspace_bytes > 0)
            e = hipMalloc((void **)&s.dev_ws, (size_t)c->workspace_bytes);
        if (e == hipSuccess)
            e = hipEventCreateWithFlags(&s.done, hipEventDisableTiming);
        if (e == hipSuccess)
            e = hipEventCreateWithFlags(&s.copied, hipEventDisableTiming);
    }
    if (e != hipSuccess) {
        free_all(p);
        delete p;
        return hip_error(e, "pipeline allocation");
    }
    *out = p;
    return SMOL_OK;
}

int smol_pipeline_drain(smol_pipeline *p)
{
    smol::clear_error();
    if (!p)
        return smol::set_error(SMOL_ERR_INVALID_ARG, "pipeline is NULL");
    std::unique_lock<std::mutex> lk(p->mu);
    hipError_t e;
    while (wait_oldest(p, lk, &e))
        if (e != hipSuccess)
            return hip_error(e, "hipEventSynchronize");
    return SMOL_OK;
}

int smol_pipeline_destroy(smol_pipeline *p)
{
    if (!p)
        return SMOL_OK;
    const int rc = smol_pipeline_drain(p);
    {
        DeviceGuard dg(p->device);
        free_all(p);
    }
    delete p;
    return rc;
}

int smol_pipeline_acquire(smol_pipeline *p, int32_t *slot, void **host, void **output)
{
    smol::clear_error();
    if (!p || !slot || !host || !output)
        return smol::set_error(SMOL_ERR_INVALID_ARG, "a NULL argument");
    std::unique_lock<std::mutex> lk(p->mu);
    bool waited = false;
    for (;;) {
        reap(p);
        for (int i = 0; i < (int)p->slots.size(); ++i) {
            Slot &s = p->slots[i];
            if (s.state == kFree) {
                s.state = kAcquired;
                *slot = i;
                *host = s.host;
                *output = s.dev_out;
                p->stats.acquire_waits += waited ? 1 : 0;
                return SMOL_OK;
            }
        }
        waited = true;
        hipError_t e;
        if (!wait_oldest(p, lk, &e))
            p->cv.wait(lk);  // every slot is held by a producer
        else if (e != hipSuccess)
            return hip_error(e, "hipEventSynchronize");
    }
}

int smol_pipeline_release(smol_pipeline *p, int32_t slot)
{
    smol::clear_error();
    if (!p)
        return smol::set_error(SMOL_ERR_INVALID_ARG, "pipeline is NULL");
    std::lock_guard<std::mutex> lk(p->mu);
    if (slot < 0 || slot >= (int32_t)p->slots.size() || p->slots[slot].state != kAcquired)
        return smol::set_error(SMOL_ERR_INVALID_ARG, "slot %d is not acquired", slot);
    p->slots[slot].state = kFree;
    p->cv.notify_all();
    return SMOL_OK;
}

int smol_pipeline_submit(smol_pipeline *p, int32_t slot, int64_t bytes, const int64_t *offsets,
                         const int32_t *widths, const int32_t *heights,
                         const int32_t *row_pitch, const int32_t *rois, int32_t n,
                         const smol_params *params, const smol_options *opts,
                         smol_consumer_fn consumer, void *user)
{
    return submit(p, slot, bytes, n, params, consumer, user,
                  [&](const uint8_t *src, int64_t nb, void *out, void *, hipStream_t s) {
                      return smol_preprocess_batch_ex(src, nb, offsets, widths, heights,
                                                      row_pitch, rois, n, params, opts, out, s);
                  });
}

int smol_pipeline_submit_yuv420(smol_pipeline *p, int32_t slot, int64_t bytes,
                                const int64_t *y_offsets, const int64_t *cb_offsets,
                                const int64_t *cr_offsets, const int32_t *widths,
                                const int32_t *heights, const int32_t *rois, int32_t n,
                                const smol_params *params, const smol_options *opts,
                                smol_consumer_fn consumer, void *user)
{
    return submit(p, slot, bytes, n, params, consumer, user,
                  [&](const uint8_t *src, int64_t nb, void *out, void *, hipStream_t s) {
                      return smol_yuv420_preprocess_batch_ex(src, nb, y_offsets, cb_offsets,
                                                             cr_offsets, widths, heights, rois,
                                                             n, params, opts, out, s);
                  });
}

int smol_pipeline_submit_jpeg(smol_pipeline *p, int32_t slot, int64_t bytes,
                              const int64_t *coef_offsets, const uint16_t *qtables,
                              int32_t n_qtables, const int32_t *widths, const int32_t *heights,
                              int32_t n, int32_t coef_layout, const smol_params *params,
                              const smol_options *opts, smol_consumer_fn consumer, void *user)
{
    if (p && p->workspace_bytes == 0) {
        smol::clear_error();
        return smol::set_error(SMOL_ERR_INVALID_ARG, "the pipeline has no workspace "
                               "(workspace_bytes 0 at creation)");
    }
    if (bytes % 2)
        return smol::set_error(SMOL_ERR_INVALID_ARG, "bytes %lld: whole int16 coefficients "
                               "needed", (long long)bytes);
    return submit(p, slot, bytes, n, params, consumer, user,
                  [&](const uint8_t *src, int64_t nb, void *out, void *ws, hipStream_t s) {
                      return smol_jpeg_roi_preprocess_batch(
                          (const int16_t *)src, nb / 2, coef_offsets, qtables, n_qtables,
                          widths, heights, n, coef_layout, params, opts, ws,
                          p->workspace_bytes, out, s);
                  });
}

int smol_pipeline_get_stats(smol_pipeline *p, smol_pipeline_stats *stats)
{
    smol::clear_error();
    if (!p || !stats)
        return smol::set_error(SMOL_ERR_INVALID_ARG, "a NULL argument");
    std::lock_guard<std::mutex> lk(p->mu);
    reap(p);
    *stats = p->stats;
    return SMOL_OK;
}

}  // extern "C"
