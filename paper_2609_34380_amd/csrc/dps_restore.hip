// dps_restore.hip -- residual backup and restore between a host copy of a
// residual's logical byte stream and its chunk slots in the device pool
// (Sec. IV-B "Residual Backup"; Sec. IV-C, restoration paragraph).
//
// This is data movement only: the copies run on the DMA engines through
// hipMemcpyAsync, so they take no compute units from the decode kernels they
// overlap.  A restore is cut into copies of at most `copy_bytes` (the paper
// uses 4 MiB) enqueued in order on the caller's stream; between two of them
// the engines are free for other streams' transfers.  Chunks whose slots
// are consecutive in the pool are joined before cutting, so an identity
// table restores in copy_bytes pieces whatever the chunk size.
#include "dps_internal.h"

namespace dps {

namespace {

// One contiguous run: `len` bytes at logical offset `lo` <-> pool offset `po`.
struct Run {
    int64_t lo, po, len;
};

template <typename Emit>
hipError_t for_each_copy(const ResidualView &r, const int32_t *slots_host, int64_t numel,
                         int64_t c0, int64_t c1, int64_t copy_bytes, Emit emit)
{
    const int64_t chunk = int64_t(1) << r.log2c;
    Run cur = {0, 0, 0};
    auto flush = [&](const Run &run) -> hipError_t {
        for (int64_t off = 0; off < run.len; off += copy_bytes) {
            const int64_t n = run.len - off < copy_bytes ? run.len - off : copy_bytes;
            const hipError_t e = emit(run.lo + off, run.po + off, n);
            if (e != hipSuccess)
                return e;
        }
        return hipSuccess;
    };
    for (int64_t c = c0; c < c1; ++c) {
        const int64_t lo = c * chunk;
        const int64_t len = numel - lo < chunk ? numel - lo : chunk;
        const int64_t po = (int64_t)slots_host[c] << r.log2c;
        if (cur.len > 0 && cur.lo + cur.len == lo && cur.po + cur.len == po) {
            cur.len += len;
            continue;
        }
        if (cur.len > 0) {
            const hipError_t e = flush(cur);
            if (e != hipSuccess)
                return e;
        }
        cur = Run{lo, po, len};
    }
    return cur.len > 0 ? flush(cur) : hipSuccess;
}

}  // namespace

hipError_t launch_restore(const uint8_t *backup, int64_t numel, const ResidualView &r,
                          const int32_t *slots_host, int64_t c0, int64_t c1,
                          int64_t copy_bytes, hipStream_t stream)
{
    uint8_t *pool = const_cast<uint8_t *>(r.pool);
    return for_each_copy(r, slots_host, numel, c0, c1, copy_bytes,
                         [&](int64_t lo, int64_t po, int64_t n) {
                             return hipMemcpyAsync(pool + po, backup + lo, (size_t)n,
                                                   hipMemcpyHostToDevice, stream);
                         });
}

hipError_t launch_backup(const ResidualView &r, const int32_t *slots_host, int64_t numel,
                         uint8_t *backup, int64_t copy_bytes, hipStream_t stream)
{
    const int64_t used = numel == 0 ? 0 : ((numel - 1) >> r.log2c) + 1;
    return for_each_copy(r, slots_host, numel, 0, used, copy_bytes,
                         [&](int64_t lo, int64_t po, int64_t n) {
                             return hipMemcpyAsync(backup + lo, r.pool + po, (size_t)n,
                                                   hipMemcpyDeviceToHost, stream);
                         });
}

}  // namespace dps
