// The thread-backed HIP stand-in declared in fake_hip/hip/hip_runtime.h, and
// the library's kernel launchers as tasks on it (each takes kernel_us()), so
// that the pipeline and the host code run on the CPU with real concurrency:
// producer threads, stream workers, host waits on events.
#include <hip/hip_runtime.h>

#include <atomic>
#include <chrono>
#include <condition_variable>
#include <cstdlib>
#include <cstring>
#include <deque>
#include <functional>
#include <mutex>
#include <thread>

#include "smol_internal.h"

namespace {

// Duration of a kernel task: 200 us, or FAKE_HIP_KERNEL_US from the
// environment.
unsigned kernel_us()
{
    static const unsigned us = [] {
        const char *e = std::getenv("FAKE_HIP_KERNEL_US");
        return e ? (unsigned)std::atoi(e) : 200u;
    }();
    return us;
}
std::atomic<long> g_pending{0};

}  // namespace

struct ihipStream_t {
    std::mutex mu;
    std::condition_variable cv;
    std::deque<std::function<void()>> q;
    bool stop = false;
    std::thread worker;

    ihipStream_t() : worker([this] { run(); }) {}
    ~ihipStream_t()
    {
        {
            std::lock_guard<std::mutex> lk(mu);
            stop = true;
        }
        cv.notify_all();
        worker.join();
    }
    void run()
    {
        for (;;) {
            std::function<void()> f;
            {
                std::unique_lock<std::mutex> lk(mu);
                cv.wait(lk, [this] { return stop || !q.empty(); });
                if (q.empty())
                    return;
                f = std::move(q.front());
                q.pop_front();
            }
            f();
            --g_pending;
        }
    }
    void push(std::function<void()> f)
    {
        ++g_pending;
        {
            std::lock_guard<std::mutex> lk(mu);
            q.push_back(std::move(f));
        }
        cv.notify_all();
    }
};

struct ihipEvent_t {
    std::mutex mu;
    std::condition_variable cv;
    unsigned long recorded = 0, done = 0;
    void complete(unsigned long gen)
    {
        // notified under the lock: a host waiter may destroy the event as soon
        // as it sees `done`, and only after this returns can it take the lock
        std::lock_guard<std::mutex> lk(mu);
        if (gen > done)
            done = gen;
        cv.notify_all();
    }
    void wait_for(unsigned long gen)
    {
        std::unique_lock<std::mutex> lk(mu);
        cv.wait(lk, [&] { return done >= gen; });
    }
};

namespace {

ihipStream_t &null_stream()
{
    static ihipStream_t s;
    return s;
}

ihipStream_t &stream_of(hipStream_t s) { return s ? *s : null_stream(); }

}  // namespace

hipError_t hipGetDevice(int *device)
{
    *device = 0;
    return hipSuccess;
}
hipError_t hipSetDevice(int device) { return device == 0 ? hipSuccess : hipErrorInvalidDevice; }
hipError_t hipDeviceGetAttribute(int *value, hipDeviceAttribute_t attr, int)
{
    *value = attr == hipDeviceAttributeMultiprocessorCount ? 256
             : attr == hipDeviceAttributeMaxSharedMemoryPerMultiprocessor ? 163840
                                                                           : 65536;
    return hipSuccess;
}
hipError_t hipMemcpyAsync(void *dst, const void *src, size_t bytes, hipMemcpyKind,
                          hipStream_t stream)
{
    stream_of(stream).push([=] { std::memmove(dst, src, bytes); });
    return hipSuccess;
}
hipError_t hipEventRecord(hipEvent_t e, hipStream_t s)
{
    unsigned long gen;
    {
        std::lock_guard<std::mutex> lk(e->mu);
        gen = ++e->recorded;
    }
    stream_of(s).push([e, gen] { e->complete(gen); });
    return hipSuccess;
}
hipError_t hipEventQuery(hipEvent_t e)
{
    std::lock_guard<std::mutex> lk(e->mu);
    return e->done >= e->recorded ? hipSuccess : hipErrorNotReady;
}
hipError_t hipEventSynchronize(hipEvent_t e)
{
    unsigned long gen;
    {
        std::lock_guard<std::mutex> lk(e->mu);
        gen = e->recorded;
    }
    e->wait_for(gen);
    return hipSuccess;
}
hipError_t hipStreamWaitEvent(hipStream_t s, hipEvent_t e, unsigned)
{
    unsigned long gen;
    {
        std::lock_guard<std::mutex> lk(e->mu);
        gen = e->recorded;
    }
    stream_of(s).push([e, gen] { e->wait_for(gen); });
    return hipSuccess;
}
hipError_t hipStreamSynchronize(hipStream_t s)
{
    ihipEvent_t e;
    hipEventRecord(&e, s);
    return hipEventSynchronize(&e);
}
const char *hipGetErrorString(hipError_t e)
{
    return e == hipSuccess ? "no error" : "fake runtime error";
}
hipError_t hipEventCreateWithFlags(hipEvent_t *e, unsigned)
{
    *e = new ihipEvent_t();
    return hipSuccess;
}
hipError_t hipEventDestroy(hipEvent_t e)
{
    delete e;
    return hipSuccess;
}
hipError_t hipStreamCreateWithFlags(hipStream_t *s, unsigned)
{
    *s = new ihipStream_t();
    return hipSuccess;
}
hipError_t hipStreamDestroy(hipStream_t s)
{
    hipStreamSynchronize(s);
    delete s;
    return hipSuccess;
}
hipError_t hipMalloc(void **p, size_t bytes)
{
    *p = std::aligned_alloc(256, (bytes + 255) / 256 * 256);
    return *p ? hipSuccess : hipErrorInvalidValue;
}
hipError_t hipFree(void *p)
{
    std::free(p);
    return hipSuccess;
}
hipError_t hipHostMalloc(void **p, size_t bytes, unsigned) { return hipMalloc(p, bytes); }
hipError_t hipHostFree(void *p) { return hipFree(p); }
hipError_t hipHostGetDevicePointer(void **dev, void *host, unsigned)
{
    *dev = host;
    return hipSuccess;
}

void fake_hip_enqueue_task(hipStream_t s, unsigned us)
{
    stream_of(s).push([us] {
        if (us)
            std::this_thread::sleep_for(std::chrono::microseconds(us));
    });
}

long fake_hip_pending(void) { return g_pending.load(); }

namespace smol {
namespace {
int task(void *stream, void *done = nullptr)
{
    fake_hip_enqueue_task((hipStream_t)stream, kernel_us());
    // the completion event of the launch: recorded right behind the task
    return done ? hipEventRecord((hipEvent_t)done, (hipStream_t)stream) : hipSuccess;
}
uint8_t g_scratch[kNoallocTableBytes];
}  // namespace

int launch_jpeg_idct(const JpegArgs &, int, void *s) { return task(s); }
int scratch_table(int, void **t)
{
    *t = g_scratch;
    return hipSuccess;
}
int launch_table_copy(const void *src, void *dst, size_t bytes, void *s)
{
    return hipMemcpyAsync(dst, src, bytes, hipMemcpyHostToDevice, (hipStream_t)s);
}
int launch_rgb_direct(const BatchArgs &, int, void *s, void *d) { return task(s, d); }
int launch_rgb_lds(const BatchArgs &, int, size_t, void *s, void *d) { return task(s, d); }
int launch_rgb_gather(const BatchArgs &, int, size_t, void *s, void *d) { return task(s, d); }
int launch_rgb_rows(const BatchArgs &, int, size_t, void *s, void *d) { return task(s, d); }
int occupancy_rgb_rows(const BatchArgs &, int, size_t, int *b)
{
    *b = 2;
    return hipSuccess;
}
int occupancy_rgb_gather(int, size_t, int *b)
{
    *b = 2;
    return hipSuccess;
}
int occupancy_rgb_lds(int, size_t, int *b)
{
    *b = 2;
    return hipSuccess;
}
int launch_yuv_direct(const BatchArgs &, int, void *s, void *d) { return task(s, d); }
int launch_yuv_rows(const BatchArgs &, int, size_t, void *s, void *d) { return task(s, d); }
int occupancy_yuv_rows(const BatchArgs &, int, size_t, int *b)
{
    *b = 2;
    return hipSuccess;
}
}  // namespace smol

extern "C" {
void fake_hip_task(void *stream, unsigned us) { fake_hip_enqueue_task((hipStream_t)stream, us); }
long fake_hip_pending_ops(void) { return fake_hip_pending(); }
}
