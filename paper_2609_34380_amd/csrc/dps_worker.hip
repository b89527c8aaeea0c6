// dps_worker.hip -- the SUM manager's restore worker (Sec. IV-B "SUM
// manager": a background thread drains the restore queue; Sec. IV-C
// restoration paragraph: the copies run on their own stream, in 4 MiB
// pieces, beside fast-mode passes).
//
// A host thread sleeps until it is woken (dps_restore_worker_kick, e.g. after
// the serving loop freed KV blocks).  Then, for as long as the manager hands
// out a restore (dps_sum_restore_begin: an evicted residual and a FREE unit
// held for it), the thread rewrites that residual's device chunk table to
// the unit's slots, copies the residual's host backup into them
// (dps::launch_restore) on its own stream, waits for the copies and reports
// dps_sum_restore_done; when the last evicted residual is back the manager's
// mode is full again.  The thread never touches the compute stream: kernels
// that read a residual run in full mode only, after the mode says so, and by
// then its copies have completed.
//
// Host code only (no kernels).  The worker's stream has the default priority.
#include <hip/hip_runtime.h>
#include <stdio.h>
#include <string.h>

#include <chrono>
#include <condition_variable>
#include <mutex>
#include <new>
#include <thread>
#include <vector>

#include "dps.h"
#include "dps_internal.h"

#define DPS_EXPORT extern "C" __attribute__((visibility("default")))

struct dps_restore_worker {
    dps_sum *sum = nullptr;
    std::vector<dps_restore_target> targets;
    int64_t chunks_per_unit = 0;
    int64_t copy_bytes = 0;
    int device = 0;
    hipStream_t stream = nullptr;
    std::thread thread;
    std::mutex mu;
    std::condition_variable wake, idle;
    bool stop = false;
    bool busy = false;
    uint64_t kicks = 0, served = 0;  // kicks asked for / taken up by the thread
    int64_t restored = 0;
    dps_status error = DPS_OK;
    char err[256] = "";
};

namespace {

thread_local char g_worker_err[256] = "";

dps::ResidualView view_of_target(const dps_restore_target &t)
{
    dps::ResidualView v;
    v.pool = t.res.pool;
    v.slots = t.res.slots;
    v.log2c = t.res.log2_chunk;
    v.n_pool_slots = t.res.pool_bytes >> t.res.log2_chunk;
    v.n_chunks = t.res.n_chunks;
    return v;
}

// One restore: residual r into unit u.  Returns DPS_OK or the failure.
dps_status restore_one(dps_restore_worker *w, int64_t r, std::vector<int32_t> &slots)
{
    const dps_restore_target &t = w->targets[(size_t)r];
    const int64_t n_chunks = t.res.n_chunks;
    slots.resize((size_t)n_chunks);
    dps_status s = dps_sum_slots(w->sum, r, w->chunks_per_unit, n_chunks, slots.data());
    if (s != DPS_OK) {
        snprintf(w->err, sizeof(w->err), "dps_sum_slots failed for residual %lld", (long long)r);
        return s;
    }
    for (int64_t c = 0; c < n_chunks; ++c)
        if (slots[(size_t)c] >= (t.res.pool_bytes >> t.res.log2_chunk)) {
            snprintf(w->err, sizeof(w->err), "unit slots of residual %lld lie outside its pool",
                     (long long)r);
            return DPS_ERR_INVALID_ARG;
        }
    hipError_t e = hipMemcpyAsync(const_cast<int32_t *>(t.res.slots), slots.data(),
                                  (size_t)n_chunks * sizeof(int32_t), hipMemcpyHostToDevice,
                                  w->stream);
    if (e == hipSuccess)
        e = dps::launch_restore(t.backup, t.numel, view_of_target(t), slots.data(), 0, n_chunks,
                                w->copy_bytes, w->stream);
    if (e == hipSuccess)
        e = hipStreamSynchronize(w->stream);  // the table and the bytes are in place
    if (e != hipSuccess) {
        snprintf(w->err, sizeof(w->err), "restore of residual %lld: %s", (long long)r,
                 hipGetErrorString(e));
        return DPS_ERR_HIP;
    }
    return dps_sum_restore_done(w->sum, r);
}

void worker_main(dps_restore_worker *w)
{
    (void)hipSetDevice(w->device);
    std::vector<int32_t> slots;
    std::unique_lock<std::mutex> lock(w->mu);
    for (;;) {
        w->wake.wait(lock, [&] { return w->stop || w->kicks != w->served; });
        if (w->stop)
            break;
        w->served = w->kicks;
        if (w->error != DPS_OK)
            continue;  // a failed worker restores nothing more
        w->busy = true;
        lock.unlock();
        dps_status s = DPS_OK;
        int64_t done = 0;
        for (;;) {
            int64_t r = -1, u = -1;
            s = dps_sum_restore_begin(w->sum, &r, &u);
            if (s != DPS_OK || r < 0)
                break;
            if (r >= (int64_t)w->targets.size()) {
                snprintf(w->err, sizeof(w->err), "residual %lld has no restore target",
                         (long long)r);
                s = DPS_ERR_INVALID_ARG;
                break;
            }
            s = restore_one(w, r, slots);
            if (s != DPS_OK)
                break;
            ++done;
        }
        lock.lock();
        w->restored += done;
        if (s != DPS_OK)
            w->error = s;
        w->busy = false;
        w->idle.notify_all();
    }
}

}  // namespace

DPS_EXPORT const char *dps_restore_worker_last_error(void) { return g_worker_err; }

DPS_EXPORT dps_status dps_restore_worker_create(dps_sum *sum, const dps_restore_target *targets,
                                                int64_t n_targets, int64_t chunks_per_unit,
                                                int64_t copy_bytes, dps_restore_worker **out)
{
    g_worker_err[0] = 0;
    if (out == nullptr || sum == nullptr || targets == nullptr || n_targets < 1 ||
        chunks_per_unit < 1 || copy_bytes <= 0) {
        snprintf(g_worker_err, sizeof(g_worker_err), "%s", "bad argument");
        return DPS_ERR_INVALID_ARG;
    }
    *out = nullptr;
    for (int64_t r = 0; r < n_targets; ++r) {
        const dps_restore_target &t = targets[r];
        const bool ok = t.backup != nullptr && t.numel >= 0 && t.res.pool != nullptr &&
                        t.res.slots != nullptr && t.res.log2_chunk >= 4 &&
                        t.res.log2_chunk <= 30 && t.res.n_chunks >= 1 &&
                        t.res.n_chunks <= chunks_per_unit &&
                        t.numel <= (t.res.n_chunks << t.res.log2_chunk);
        if (!ok) {
            snprintf(g_worker_err, sizeof(g_worker_err), "bad restore target %lld", (long long)r);
            return DPS_ERR_INVALID_ARG;
        }
    }
    dps_restore_worker *w = new (std::nothrow) dps_restore_worker();
    if (w == nullptr)
        return DPS_ERR_NO_SPACE;
    w->sum = sum;
    w->targets.assign(targets, targets + n_targets);
    w->chunks_per_unit = chunks_per_unit;
    w->copy_bytes = copy_bytes;
    hipError_t e = hipGetDevice(&w->device);
    if (e == hipSuccess)
        e = hipStreamCreateWithFlags(&w->stream, hipStreamNonBlocking);
    if (e != hipSuccess) {
        snprintf(g_worker_err, sizeof(g_worker_err), "%s", hipGetErrorString(e));
        delete w;
        return DPS_ERR_HIP;
    }
    try {
        w->thread = std::thread(worker_main, w);
    } catch (...) {
        (void)hipStreamDestroy(w->stream);
        delete w;
        snprintf(g_worker_err, sizeof(g_worker_err), "%s", "cannot start the worker thread");
        return DPS_ERR_NO_SPACE;
    }
    *out = w;
    return DPS_OK;
}

DPS_EXPORT dps_status dps_restore_worker_kick(dps_restore_worker *w)
{
    if (w == nullptr)
        return DPS_ERR_INVALID_ARG;
    std::lock_guard<std::mutex> lock(w->mu);
    ++w->kicks;
    w->wake.notify_one();
    return DPS_OK;
}

DPS_EXPORT dps_status dps_restore_worker_wait_idle(dps_restore_worker *w, int64_t timeout_ms)
{
    g_worker_err[0] = 0;
    if (w == nullptr || timeout_ms < 0)
        return DPS_ERR_INVALID_ARG;
    std::unique_lock<std::mutex> lock(w->mu);
    const bool idle = w->idle.wait_for(lock, std::chrono::milliseconds(timeout_ms), [&] {
        return !w->busy && w->kicks == w->served;
    });
    if (w->error != DPS_OK) {
        snprintf(g_worker_err, sizeof(g_worker_err), "%s", w->err);
        return w->error;
    }
    if (!idle) {
        snprintf(g_worker_err, sizeof(g_worker_err), "%s", "restores still running");
        return DPS_ERR_TIMEOUT;
    }
    return DPS_OK;
}

DPS_EXPORT int64_t dps_restore_worker_restored(dps_restore_worker *w)
{
    if (w == nullptr)
        return -1;
    std::lock_guard<std::mutex> lock(w->mu);
    return w->restored;
}

DPS_EXPORT void dps_restore_worker_destroy(dps_restore_worker *w)
{
    if (w == nullptr)
        return;
    {
        std::lock_guard<std::mutex> lock(w->mu);
        w->stop = true;
        w->wake.notify_one();
    }
    w->thread.join();  // a restore in progress finishes first
    (void)hipStreamDestroy(w->stream);
    delete w;
}
