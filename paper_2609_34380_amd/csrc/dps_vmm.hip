// dps_vmm.hip -- the shared region's physical units mapped twice through the
// HIP virtual memory API (Sec. IV-B "Shared Region", dual-mapping property).
//
// n_units physical units (hipMemCreate) are mapped once, in unit order, into
// the KV view, and again into residual views: one virtual range per residual
// tensor, whose i-th unit-sized piece maps the unit that holds the tensor's
// chunk i.  A residual view is contiguous, so the linear kernels address it
// through an identity chunk table, and a byte written through either view is
// the same physical byte.  When a unit is taken for KV blocks, the residual
// view still maps it (the residual is stale, as the SUM manager records);
// restoring into another unit remaps that piece of the view
// (dps_vmm_remap) before the backup is copied back through it.
//
// Host code only (no kernels).  Every call works on the device that was
// current at dps_vmm_create.  Mapping changes are not ordered with queued
// work: the caller makes sure nothing that uses a view runs while it is
// unmapped or remapped.
#include <hip/hip_runtime.h>
#include <stdio.h>
#include <string.h>

#include <mutex>
#include <new>
#include <vector>

#include "dps.h"

#define DPS_EXPORT extern "C" __attribute__((visibility("default")))

struct dps_vmm {
    int device;
    int64_t n_units;
    int64_t unit_bytes;
    std::vector<hipMemGenericAllocationHandle_t> units;
    hipDeviceptr_t kv = nullptr;
    struct View {
        hipDeviceptr_t base;
        std::vector<int32_t> units;  // unit mapped at each piece, -1: none
    };
    std::vector<View> views;
    std::mutex mu;
};

namespace {

thread_local char g_vmm_err[256] = "";

dps_status vmm_fail(dps_status s, const char *what, hipError_t e)
{
    snprintf(g_vmm_err, sizeof(g_vmm_err), "%s: %s", what, hipGetErrorString(e));
    return e == hipErrorNotSupported ? DPS_ERR_UNSUPPORTED : s;
}

#define VMM_REQUIRE(cond, status, msg)                                  \
    do {                                                                \
        if (!(cond)) {                                                  \
            snprintf(g_vmm_err, sizeof(g_vmm_err), "%s", msg);          \
            return status;                                              \
        }                                                               \
    } while (0)

#define VMM_HIP(call, what)                                             \
    do {                                                                \
        hipError_t e_ = (call);                                         \
        if (e_ != hipSuccess)                                           \
            return vmm_fail(DPS_ERR_HIP, what, e_);                     \
    } while (0)

// Makes v's device current for a call and restores the caller's afterwards.
struct DeviceGuard {
    int prev = -1;
    hipError_t err;
    explicit DeviceGuard(int device)
    {
        err = hipGetDevice(&prev);
        if (err == hipSuccess && prev != device)
            err = hipSetDevice(device);
    }
    ~DeviceGuard()
    {
        if (prev >= 0)
            (void)hipSetDevice(prev);
    }
};

hipMemAllocationProp unit_prop(int device)
{
    hipMemAllocationProp p;
    memset(&p, 0, sizeof(p));
    p.type = hipMemAllocationTypePinned;
    p.location.type = hipMemLocationTypeDevice;
    p.location.id = device;
    return p;
}

// Map unit u of v at va (unit_bytes) with read/write access on v's device.
dps_status map_unit(dps_vmm *v, hipDeviceptr_t va, int32_t u)
{
    VMM_HIP(hipMemMap(va, (size_t)v->unit_bytes, 0, v->units[u], 0), "hipMemMap");
    hipMemAccessDesc acc;
    memset(&acc, 0, sizeof(acc));
    acc.location.type = hipMemLocationTypeDevice;
    acc.location.id = v->device;
    acc.flags = hipMemAccessFlagsProtReadWrite;
    VMM_HIP(hipMemSetAccess(va, (size_t)v->unit_bytes, &acc, 1), "hipMemSetAccess");
    return DPS_OK;
}

// Unmap every piece of a view and free its range (errors ignored: teardown).
void drop_view(dps_vmm *v, dps_vmm::View &w)
{
    for (size_t i = 0; i < w.units.size(); ++i)
        if (w.units[i] >= 0)
            (void)hipMemUnmap((char *)w.base + i * v->unit_bytes, (size_t)v->unit_bytes);
    (void)hipMemAddressFree(w.base, w.units.size() * (size_t)v->unit_bytes);
}

void release_all(dps_vmm *v)
{
    for (auto &w : v->views)
        drop_view(v, w);
    v->views.clear();
    if (v->kv) {
        for (int64_t u = 0; u < (int64_t)v->units.size(); ++u)
            (void)hipMemUnmap((char *)v->kv + u * v->unit_bytes, (size_t)v->unit_bytes);
        (void)hipMemAddressFree(v->kv, (size_t)(v->n_units * v->unit_bytes));
        v->kv = nullptr;
    }
    for (auto h : v->units)
        (void)hipMemRelease(h);
    v->units.clear();
}

dps_vmm::View *find_view(dps_vmm *v, const void *view)
{
    for (auto &w : v->views)
        if (w.base == view)
            return &w;
    return nullptr;
}

}  // namespace

DPS_EXPORT const char *dps_vmm_last_error(void) { return g_vmm_err; }

DPS_EXPORT dps_status dps_vmm_granularity(int64_t *bytes_out)
{
    g_vmm_err[0] = 0;
    VMM_REQUIRE(bytes_out != nullptr, DPS_ERR_INVALID_ARG, "bytes_out is NULL");
    int dev = 0;
    VMM_HIP(hipGetDevice(&dev), "hipGetDevice");
    const hipMemAllocationProp p = unit_prop(dev);
    size_t g = 0;
    VMM_HIP(hipMemGetAllocationGranularity(&g, &p, hipMemAllocationGranularityMinimum),
            "hipMemGetAllocationGranularity");
    *bytes_out = (int64_t)g;
    return DPS_OK;
}

DPS_EXPORT dps_status dps_vmm_create(int64_t n_units, int64_t unit_bytes, dps_vmm **out)
{
    g_vmm_err[0] = 0;
    VMM_REQUIRE(out != nullptr, DPS_ERR_INVALID_ARG, "out is NULL");
    *out = nullptr;
    VMM_REQUIRE(n_units >= 1 && n_units <= (1 << 20), DPS_ERR_INVALID_ARG,
                "n_units must be in 1..2^20");
    VMM_REQUIRE(unit_bytes >= 4096 && (unit_bytes & (unit_bytes - 1)) == 0 &&
                    unit_bytes <= (int64_t(1) << 30),
                DPS_ERR_INVALID_ARG, "unit_bytes must be a power of two in 4 KiB..1 GiB");
    int64_t gran = 0;
    dps_status s = dps_vmm_granularity(&gran);
    if (s != DPS_OK)
        return s;
    VMM_REQUIRE(gran > 0 && unit_bytes % gran == 0, DPS_ERR_INVALID_ARG,
                "unit_bytes is not a multiple of the VMM allocation granularity");
    int dev = 0;
    VMM_HIP(hipGetDevice(&dev), "hipGetDevice");
    dps_vmm *v = new (std::nothrow) dps_vmm();
    VMM_REQUIRE(v != nullptr, DPS_ERR_NO_SPACE, "out of host memory");
    v->device = dev;
    v->n_units = n_units;
    v->unit_bytes = unit_bytes;
    const hipMemAllocationProp p = unit_prop(v->device);
    v->units.reserve((size_t)n_units);
    for (int64_t u = 0; u < n_units; ++u) {
        hipMemGenericAllocationHandle_t h;
        const hipError_t e = hipMemCreate(&h, (size_t)unit_bytes, &p, 0);
        if (e != hipSuccess) {
            release_all(v);
            delete v;
            return vmm_fail(DPS_ERR_HIP, "hipMemCreate", e);
        }
        v->units.push_back(h);
    }
    hipError_t e = hipMemAddressReserve(&v->kv, (size_t)(n_units * unit_bytes),
                                        (size_t)unit_bytes, nullptr, 0);
    if (e != hipSuccess) {
        v->kv = nullptr;
        release_all(v);
        delete v;
        return vmm_fail(DPS_ERR_HIP, "hipMemAddressReserve", e);
    }
    for (int64_t u = 0; u < n_units; ++u) {
        s = map_unit(v, (char *)v->kv + u * unit_bytes, (int32_t)u);
        if (s != DPS_OK) {
            // units before u are mapped; release_all unmaps all, ignoring errors
            release_all(v);
            delete v;
            return s;
        }
    }
    *out = v;
    return DPS_OK;
}

DPS_EXPORT void *dps_vmm_kv_view(const dps_vmm *v) { return v ? v->kv : nullptr; }

DPS_EXPORT int64_t dps_vmm_unit_bytes(const dps_vmm *v) { return v ? v->unit_bytes : 0; }

DPS_EXPORT dps_status dps_vmm_map_residual(dps_vmm *v, const int32_t *units_host, int64_t count,
                                           void **view_out)
{
    g_vmm_err[0] = 0;
    VMM_REQUIRE(v != nullptr && view_out != nullptr, DPS_ERR_INVALID_ARG,
                "vmm or view_out is NULL");
    *view_out = nullptr;
    VMM_REQUIRE(count >= 1 && count <= v->n_units * 64, DPS_ERR_INVALID_ARG,
                "count must be in 1..64 * n_units");
    VMM_REQUIRE(units_host != nullptr, DPS_ERR_INVALID_ARG, "units_host is NULL");
    for (int64_t i = 0; i < count; ++i)
        VMM_REQUIRE(units_host[i] >= 0 && units_host[i] < v->n_units, DPS_ERR_INVALID_ARG,
                    "unit index outside 0..n_units-1");
    std::lock_guard<std::mutex> lock(v->mu);
    DeviceGuard dg(v->device);
    VMM_HIP(dg.err, "hipSetDevice");
    dps_vmm::View w;
    VMM_HIP(hipMemAddressReserve(&w.base, (size_t)(count * v->unit_bytes),
                                 (size_t)v->unit_bytes, nullptr, 0),
            "hipMemAddressReserve");
    w.units.assign((size_t)count, -1);
    for (int64_t i = 0; i < count; ++i) {
        const dps_status s = map_unit(v, (char *)w.base + i * v->unit_bytes, units_host[i]);
        if (s != DPS_OK) {
            drop_view(v, w);
            return s;
        }
        w.units[(size_t)i] = units_host[i];
    }
    v->views.push_back(w);
    *view_out = w.base;
    return DPS_OK;
}

DPS_EXPORT dps_status dps_vmm_remap(dps_vmm *v, void *view, int64_t piece, int32_t unit)
{
    g_vmm_err[0] = 0;
    VMM_REQUIRE(v != nullptr && view != nullptr, DPS_ERR_INVALID_ARG, "vmm or view is NULL");
    VMM_REQUIRE(unit >= 0 && unit < v->n_units, DPS_ERR_INVALID_ARG,
                "unit index outside 0..n_units-1");
    std::lock_guard<std::mutex> lock(v->mu);
    dps_vmm::View *w = find_view(v, view);
    VMM_REQUIRE(w != nullptr, DPS_ERR_INVALID_ARG, "not a residual view of this region");
    VMM_REQUIRE(piece >= 0 && piece < (int64_t)w->units.size(), DPS_ERR_INVALID_ARG,
                "piece outside the view");
    DeviceGuard dg(v->device);
    VMM_HIP(dg.err, "hipSetDevice");
    char *va = (char *)w->base + piece * v->unit_bytes;
    if (w->units[(size_t)piece] >= 0) {
        VMM_HIP(hipMemUnmap(va, (size_t)v->unit_bytes), "hipMemUnmap");
        w->units[(size_t)piece] = -1;
    }
    const dps_status s = map_unit(v, va, unit);
    if (s == DPS_OK)
        w->units[(size_t)piece] = unit;
    return s;
}

DPS_EXPORT dps_status dps_vmm_unmap_residual(dps_vmm *v, void *view)
{
    g_vmm_err[0] = 0;
    VMM_REQUIRE(v != nullptr && view != nullptr, DPS_ERR_INVALID_ARG, "vmm or view is NULL");
    std::lock_guard<std::mutex> lock(v->mu);
    for (size_t i = 0; i < v->views.size(); ++i) {
        if (v->views[i].base == view) {
            DeviceGuard dg(v->device);
            VMM_HIP(dg.err, "hipSetDevice");
            drop_view(v, v->views[i]);
            v->views.erase(v->views.begin() + (long)i);
            return DPS_OK;
        }
    }
    snprintf(g_vmm_err, sizeof(g_vmm_err), "%s", "not a residual view of this region");
    return DPS_ERR_INVALID_ARG;
}

DPS_EXPORT void dps_vmm_destroy(dps_vmm *v)
{
    if (v == nullptr)
        return;
    {
        std::lock_guard<std::mutex> lock(v->mu);
        DeviceGuard dg(v->device);
        release_all(v);
    }
    delete v;
}
