// dps_sum.cpp -- the SUM manager's unit bookkeeping (Sec. IV-B "SUM
// manager"; Sec. IV-D, Algorithm 1): which physical units of the shared
// region hold a residual, which hold KV blocks, which residuals were
// evicted, and the precision mode that follows from it.  Host-only C++; the
// copies a restore needs are dps_restore's.
//
// Every call locks the manager, so a restore worker thread may drive the
// restores while the serving loop allocates and frees KV blocks.
//
// Units are numbered 0 .. n_units-1, each with blocks_per_unit KV blocks
// (block id = unit * blocks_per_unit + index).  Residual r starts bound to
// unit r.  Every state set is ordered by unit id and "pop" takes the lowest
// id; a unit gives out its lowest free block indices first.
#include <stdint.h>
#include <string.h>

#include <mutex>
#include <new>
#include <set>
#include <vector>

#include "dps.h"

#define DPS_EXPORT extern "C" __attribute__((visibility("default")))

struct dps_sum {
    int64_t n_units, blocks_per_unit, n_res;
    int32_t mode;
    std::set<int64_t> free_, backed, avail, full, restoring;  // units
    std::set<int64_t> stale, evicted;                         // residuals
    std::vector<int32_t> state;            // per unit: a DPS_UNIT_* value
    std::vector<int64_t> used;             // per unit: allocated KV blocks
    std::vector<std::vector<uint8_t>> taken;  // per unit: block index -> allocated
    std::vector<int64_t> unit_of;          // per residual: bound or restoring unit, or -1
    std::vector<int64_t> resident;         // per unit: residual bound to it, or -1
    // every call holds it: the serving loop and a restore worker thread
    // (dps_restore_worker_*) may call at the same time
    mutable std::mutex mu;
};

namespace {

void move_unit(dps_sum *s, int64_t u, int32_t to)
{
    switch (s->state[u]) {
    case DPS_UNIT_FREE: s->free_.erase(u); break;
    case DPS_UNIT_BACKED: s->backed.erase(u); break;
    case DPS_UNIT_AVAIL: s->avail.erase(u); break;
    case DPS_UNIT_FULL: s->full.erase(u); break;
    case DPS_UNIT_RESTORING: s->restoring.erase(u); break;
    }
    switch (to) {
    case DPS_UNIT_FREE: s->free_.insert(u); break;
    case DPS_UNIT_BACKED: s->backed.insert(u); break;
    case DPS_UNIT_AVAIL: s->avail.insert(u); break;
    case DPS_UNIT_FULL: s->full.insert(u); break;
    case DPS_UNIT_RESTORING: s->restoring.insert(u); break;
    }
    s->state[u] = to;
}

int64_t pop_lowest(std::set<int64_t> &set)
{
    const int64_t u = *set.begin();
    set.erase(set.begin());
    return u;
}

}  // namespace

DPS_EXPORT dps_status dps_sum_create(int64_t n_units, int64_t blocks_per_unit, int64_t n_res,
                                     dps_sum **out)
{
    if (out == nullptr)
        return DPS_ERR_INVALID_ARG;
    *out = nullptr;
    if (n_units < 1 || blocks_per_unit < 1 || n_res < 0 || n_res > n_units ||
        n_units > (int64_t(1) << 40) / blocks_per_unit)
        return DPS_ERR_INVALID_ARG;
    dps_sum *s = new (std::nothrow) dps_sum;
    if (s == nullptr)
        return DPS_ERR_INVALID_ARG;
    s->n_units = n_units;
    s->blocks_per_unit = blocks_per_unit;
    s->n_res = n_res;
    s->mode = DPS_MODE_FULL;
    s->state.assign(n_units, DPS_UNIT_FREE);
    s->used.assign(n_units, 0);
    s->taken.assign(n_units, std::vector<uint8_t>(blocks_per_unit, 0));
    s->unit_of.assign(n_res, -1);
    s->resident.assign(n_units, -1);
    for (int64_t u = 0; u < n_units; ++u)
        s->free_.insert(u);
    for (int64_t r = 0; r < n_res; ++r) {
        move_unit(s, r, DPS_UNIT_BACKED);
        s->unit_of[r] = r;
        s->resident[r] = r;
    }
    *out = s;
    return DPS_OK;
}

DPS_EXPORT void dps_sum_destroy(dps_sum *s) { delete s; }

// Algorithm 1, AllocKVBlock.  A request larger than the room left in AVAIL,
// FREE and BACKED units together takes nothing (the loop would only fail
// after taking what it found).
DPS_EXPORT dps_status dps_sum_alloc(dps_sum *s, int64_t n, int64_t *blocks)
{
    if (s == nullptr || n < 0 || (n > 0 && blocks == nullptr))
        return DPS_ERR_INVALID_ARG;
    std::lock_guard<std::mutex> lock(s->mu);
    int64_t room = (int64_t)(s->free_.size() + s->backed.size()) * s->blocks_per_unit;
    for (int64_t u : s->avail)
        room += s->blocks_per_unit - s->used[u];
    if (n > room)
        return DPS_ERR_NO_SPACE;
    int64_t got = 0;
    while (got < n) {
        if (s->avail.empty()) {
            int64_t u;
            if (!s->free_.empty()) {
                u = pop_lowest(s->free_);
            } else {
                u = pop_lowest(s->backed);
                // the unit's residual mapping goes stale and its data now lives
                // only in the host backup: serve in fast mode until restored
                const int64_t r = s->resident[u];
                s->resident[u] = -1;
                s->unit_of[r] = -1;
                s->stale.insert(r);
                s->evicted.insert(r);
                s->mode = DPS_MODE_FAST;
            }
            s->state[u] = DPS_UNIT_AVAIL;
            s->avail.insert(u);
        }
        const int64_t u = pop_lowest(s->avail);  // state stays AVAIL until re-filed below
        std::vector<uint8_t> &t = s->taken[u];
        for (int64_t i = 0; i < s->blocks_per_unit && got < n; ++i) {
            if (!t[i]) {
                t[i] = 1;
                ++s->used[u];
                blocks[got++] = u * s->blocks_per_unit + i;
            }
        }
        const int32_t to = s->used[u] == s->blocks_per_unit ? DPS_UNIT_FULL : DPS_UNIT_AVAIL;
        s->state[u] = to;
        (to == DPS_UNIT_FULL ? s->full : s->avail).insert(u);
    }
    return DPS_OK;
}

// Algorithm 1, FreeKVBlock.  Every block must be allocated and listed once;
// otherwise nothing changes.  *wake (optional) is set to 1 when a unit became
// free while residuals wait for restoration.
DPS_EXPORT dps_status dps_sum_free(dps_sum *s, const int64_t *blocks, int64_t n, int32_t *wake)
{
    if (s == nullptr || n < 0 || (n > 0 && blocks == nullptr))
        return DPS_ERR_INVALID_ARG;
    std::lock_guard<std::mutex> lock(s->mu);
    if (wake)
        *wake = 0;
    const int64_t total = s->n_units * s->blocks_per_unit;
    std::set<int64_t> seen;
    for (int64_t j = 0; j < n; ++j) {
        const int64_t b = blocks[j];
        if (b < 0 || b >= total || !seen.insert(b).second)
            return DPS_ERR_INVALID_ARG;
        const int64_t u = b / s->blocks_per_unit;
        if (!s->taken[u][b % s->blocks_per_unit] ||
            (s->state[u] != DPS_UNIT_AVAIL && s->state[u] != DPS_UNIT_FULL))
            return DPS_ERR_INVALID_ARG;
    }
    for (int64_t j = 0; j < n; ++j) {
        const int64_t b = blocks[j];
        const int64_t u = b / s->blocks_per_unit;
        s->taken[u][b % s->blocks_per_unit] = 0;
        --s->used[u];
        if (s->state[u] == DPS_UNIT_FULL)
            move_unit(s, u, DPS_UNIT_AVAIL);
        if (s->used[u] == 0) {
            move_unit(s, u, DPS_UNIT_FREE);
            if (!s->evicted.empty() && wake)
                *wake = 1;
        }
    }
    return DPS_OK;
}

// The restore worker's first step (Sec. IV-B "SUM manager"): the lowest stale
// residual is unmapped and bound to the lowest FREE unit, which is held for
// it (RESTORING) while the caller copies the data in (dps_restore into the
// slots dps_sum_slots names).  *residual = -1 when no residual is stale or
// no unit is free.
DPS_EXPORT dps_status dps_sum_restore_begin(dps_sum *s, int64_t *residual, int64_t *unit)
{
    if (s == nullptr || residual == nullptr || unit == nullptr)
        return DPS_ERR_INVALID_ARG;
    std::lock_guard<std::mutex> lock(s->mu);
    *residual = -1;
    *unit = -1;
    if (s->stale.empty() || s->free_.empty())
        return DPS_OK;
    const int64_t r = pop_lowest(s->stale);
    const int64_t u = *s->free_.begin();
    move_unit(s, u, DPS_UNIT_RESTORING);
    s->unit_of[r] = u;
    s->resident[u] = r;
    *residual = r;
    *unit = u;
    return DPS_OK;
}

// The copy of residual r has completed: its unit becomes BACKED, and once no
// residual is evicted the mode returns to full.
DPS_EXPORT dps_status dps_sum_restore_done(dps_sum *s, int64_t residual)
{
    if (s == nullptr || residual < 0 || residual >= s->n_res)
        return DPS_ERR_INVALID_ARG;
    std::lock_guard<std::mutex> lock(s->mu);
    const int64_t u = s->unit_of[residual];
    if (u < 0 || s->state[u] != DPS_UNIT_RESTORING || !s->evicted.count(residual))
        return DPS_ERR_INVALID_ARG;
    move_unit(s, u, DPS_UNIT_BACKED);
    s->evicted.erase(residual);
    if (s->evicted.empty())
        s->mode = DPS_MODE_FULL;
    return DPS_OK;
}

DPS_EXPORT int32_t dps_sum_mode(const dps_sum *s)
{
    if (s == nullptr)
        return -1;
    std::lock_guard<std::mutex> lock(s->mu);
    return s->mode;
}

DPS_EXPORT int32_t dps_sum_unit_state(const dps_sum *s, int64_t unit)
{
    if (s == nullptr || unit < 0 || unit >= s->n_units)
        return -1;
    std::lock_guard<std::mutex> lock(s->mu);
    return s->state[unit];
}

DPS_EXPORT int64_t dps_sum_unit_of(const dps_sum *s, int64_t residual)
{
    if (s == nullptr || residual < 0 || residual >= s->n_res)
        return -1;
    std::lock_guard<std::mutex> lock(s->mu);
    return s->unit_of[residual];
}

DPS_EXPORT dps_status dps_sum_counts(const dps_sum *s, int64_t *counts)
{
    if (s == nullptr || counts == nullptr)
        return DPS_ERR_INVALID_ARG;
    std::lock_guard<std::mutex> lock(s->mu);
    int64_t free_blocks = 0;
    for (int64_t u : s->avail)
        free_blocks += s->blocks_per_unit - s->used[u];
    counts[0] = (int64_t)s->free_.size();
    counts[1] = (int64_t)s->backed.size();
    counts[2] = (int64_t)s->avail.size();
    counts[3] = (int64_t)s->full.size();
    counts[4] = (int64_t)s->restoring.size();
    counts[5] = (int64_t)s->stale.size();
    counts[6] = (int64_t)s->evicted.size();
    counts[7] = free_blocks;
    return DPS_OK;
}

// Host slot table of residual r (n_chunks chunks of the pool's chunk size)
// in the unit it is bound to or being restored into: unit u spans pool slots
// [u * chunks_per_unit, (u + 1) * chunks_per_unit).
DPS_EXPORT dps_status dps_sum_slots(const dps_sum *s, int64_t residual, int64_t chunks_per_unit,
                                    int64_t n_chunks, int32_t *slots_host)
{
    if (s == nullptr || residual < 0 || residual >= s->n_res || chunks_per_unit < 1 ||
        n_chunks < 0 || n_chunks > chunks_per_unit || (n_chunks > 0 && slots_host == nullptr))
        return DPS_ERR_INVALID_ARG;
    std::lock_guard<std::mutex> lock(s->mu);
    const int64_t u = s->unit_of[residual];
    if (u < 0)
        return DPS_ERR_INVALID_ARG;
    if ((u + 1) * chunks_per_unit > INT32_MAX)
        return DPS_ERR_INVALID_ARG;
    for (int64_t c = 0; c < n_chunks; ++c)
        slots_host[c] = (int32_t)(u * chunks_per_unit + c);
    return DPS_OK;
}
