// Model-state store: the GMS ownership protocol (paper section 3.2, Figure 4).
//
// A writer populates allocations under an exclusive read-write lease and
// commits them; commit records the layout and the hash of every 4 KiB block
// and makes the state immutable by mapping it read-only.  Readers attach
// read-only, optionally after the committed state has been re-hashed and
// compared with the commit-time hashes.  A writer that leaves before commit
// discards its incomplete state; readers that leave only end their leases;
// exclusive write access returns once the last reader has left.  Section 4
// adds that the layout is recorded before commit and that a separate writer
// repopulates a cold store from storage before the engine reattaches.
//
// The state machine is host logic under one mutex; the data-plane work it
// triggers (hashing, comparison) is the library's verify kernel, and access
// changes go through the pool's HIP virtual-memory mappings.

#include <algorithm>
#include <mutex>
#include <new>
#include <set>
#include <vector>

#include "gms_host.h"

using gms::DeviceGuard;
using gms::fail;
using gms::fail_hip;

struct gms_store {
    int device = GMS_HOST_ONLY;
    gms_pool *pool = nullptr;
    std::mutex mu;
    int state = GMS_STORE_EMPTY;
    bool invalid = false;
    uint64_t next_lease = 1;
    uint64_t writer = 0;          // lease id of the writer, 0 if none
    std::set<uint64_t> readers;   // lease ids of the readers
    gms_manifest *layout = nullptr;
    uint64_t *d_hash = nullptr;   // commit-time block hashes (device)
    uint64_t *d_count = nullptr;  // mismatch counter for verification (device)
};

namespace {

void drop_layout(gms_store *s)
{
    if (s->layout) gms_manifest_destroy(s->layout);
    s->layout = nullptr;
    if (s->d_hash) (void)hipFree(s->d_hash);
    s->d_hash = nullptr;
}

// Hashes the blocks of `m` (into `hash_out`) and compares them with
// `expected` when given; returns the mismatch count through *count.
int hash_and_compare(gms_store *s, const gms_manifest *m, const uint64_t *expected, uint64_t *hash_out,
                     uint64_t *list, uint64_t cap, uint64_t *count, void *stream)
{
    *count = 0;
    int rc = gms::refuse_capture((hipStream_t)stream, "a store verification");
    if (rc != GMS_OK) return rc;
    if (gms_num_blocks(m) == 0) return GMS_OK;
    rc = gms_verify(m, expected, hash_out, nullptr, expected ? s->d_count : nullptr, expected ? list : nullptr,
                    expected ? cap : 0, stream);
    if (rc != GMS_OK) return rc;
    hipStream_t st = (hipStream_t)stream;
    hipError_t e;
    if (expected && (e = hipMemcpyAsync(count, s->d_count, sizeof(uint64_t), hipMemcpyDeviceToHost, st)) != hipSuccess)
        return fail_hip(e, "mismatch count");
    if ((e = hipStreamSynchronize(st)) != hipSuccess) return fail_hip(e, "store verification");
    return GMS_OK;
}

// The caller holds s->mu.  Discards allocations and layout: EMPTY.
int discard(gms_store *s)
{
    drop_layout(s);
    s->writer = 0;
    s->invalid = false;
    s->state = GMS_STORE_EMPTY;
    if (s->pool) {
        DeviceGuard g(s->device);
        return gms::pool_reset(s->pool);
    }
    return GMS_OK;
}

int check_writer(gms_store *s, uint64_t lease)
{
    if (s->state != GMS_STORE_RW || lease == 0 || lease != s->writer)
        return fail(GMS_ERR_INVALID, "lease %llu is not the store's writer", (unsigned long long)lease);
    return GMS_OK;
}

}  // namespace

extern "C" {

int gms_store_create(int device, uint64_t va_bytes, uint64_t slab_bytes, gms_store **out)
{
    gms::clear_error();
    if (!out) return fail(GMS_ERR_INVALID, "out is null");
    *out = nullptr;
    gms_store *s = new (std::nothrow) gms_store;
    if (!s) return fail(GMS_ERR_NOMEM, "store");
    s->device = device;
    if (device != GMS_HOST_ONLY) {
        int rc = gms_pool_create(device, va_bytes, slab_bytes, &s->pool);
        if (rc != GMS_OK) {
            delete s;
            return rc;
        }
        DeviceGuard g(device);
        hipError_t e = hipMalloc((void **)&s->d_count, sizeof(uint64_t));
        if (e != hipSuccess) {
            (void)hipGetLastError();
            gms_pool_destroy(s->pool);
            delete s;
            return fail(GMS_ERR_NOMEM, "store counter: %s", hipGetErrorString(e));
        }
    }
    *out = s;
    return GMS_OK;
}

void gms_store_destroy(gms_store *s)
{
    if (!s) return;
    if (s->device != GMS_HOST_ONLY) {
        DeviceGuard g(s->device);
        (void)hipDeviceSynchronize();
        drop_layout(s);
        if (s->d_count) (void)hipFree(s->d_count);
        gms_pool_destroy(s->pool);
    } else {
        drop_layout(s);
    }
    delete s;
}

int gms_store_state(const gms_store *cs, int *state, uint32_t *readers, int *invalid)
{
    if (!cs) return fail(GMS_ERR_INVALID, "store is null");
    gms_store *s = const_cast<gms_store *>(cs);
    std::lock_guard<std::mutex> lock(s->mu);
    if (state) *state = s->state;
    if (readers) *readers = (uint32_t)s->readers.size();
    if (invalid) *invalid = s->invalid ? 1 : 0;
    return GMS_OK;
}

gms_pool *gms_store_pool(gms_store *s) { return s ? s->pool : nullptr; }

int gms_store_connect_rw(gms_store *s, uint64_t *lease_out)
{
    gms::clear_error();
    if (!s || !lease_out) return fail(GMS_ERR_INVALID, "store or lease_out is null");
    std::lock_guard<std::mutex> lock(s->mu);
    if (s->state != GMS_STORE_EMPTY && s->state != GMS_STORE_COMMITTED)
        return fail(GMS_ERR_STATE, "store is %s", s->state == GMS_STORE_RW ? "held by a writer" : "held by readers");
    if (s->state == GMS_STORE_COMMITTED && s->pool) {  // the writer reuses the allocation set
        DeviceGuard g(s->device);
        int rc = gms::pool_set_access_all(s->pool, false);
        if (rc != GMS_OK) return rc;
    }
    s->writer = s->next_lease++;
    s->state = GMS_STORE_RW;
    *lease_out = s->writer;
    return GMS_OK;
}

int gms_store_alloc(gms_store *s, uint64_t lease, uint64_t bytes, uint64_t align, uint64_t *addr_out)
{
    gms::clear_error();
    if (!s) return fail(GMS_ERR_INVALID, "store is null");
    std::lock_guard<std::mutex> lock(s->mu);
    int rc = check_writer(s, lease);
    if (rc != GMS_OK) return rc;
    if (!s->pool) return fail(GMS_ERR_STATE, "host-only store has no memory");
    return gms_pool_alloc(s->pool, bytes, align, addr_out);
}

int gms_store_free(gms_store *s, uint64_t lease, uint64_t addr)
{
    gms::clear_error();
    if (!s) return fail(GMS_ERR_INVALID, "store is null");
    std::lock_guard<std::mutex> lock(s->mu);
    int rc = check_writer(s, lease);
    if (rc != GMS_OK) return rc;
    if (!s->pool) return fail(GMS_ERR_STATE, "host-only store has no memory");
    return gms_pool_free(s->pool, addr);
}

int gms_store_commit(gms_store *s, uint64_t lease, const gms_entry *entries, uint64_t n, const uint64_t *expected_blk,
                     uint64_t *mismatch_count_out, void *stream)
{
    gms::clear_error();
    if (mismatch_count_out) *mismatch_count_out = 0;
    if (!s) return fail(GMS_ERR_INVALID, "store is null");
    std::lock_guard<std::mutex> lock(s->mu);
    int rc = check_writer(s, lease);
    if (rc != GMS_OK) return rc;
    if (n && !entries) return fail(GMS_ERR_INVALID, "entries is null");
    if (!s->pool) {
        if (n || expected_blk) return fail(GMS_ERR_STATE, "host-only store commits no entries");
        drop_layout(s);
        s->writer = 0;
        s->invalid = false;
        s->state = GMS_STORE_COMMITTED;
        return GMS_OK;
    }
    for (uint64_t i = 0; i < n; ++i)
        if (entries[i].nbytes && !gms::pool_holds(s->pool, entries[i].addr, entries[i].nbytes))
            return fail(GMS_ERR_INVALID, "entry %llu [%#llx, +%llu) is not inside one store allocation",
                        (unsigned long long)i, (unsigned long long)entries[i].addr,
                        (unsigned long long)entries[i].nbytes);
    gms_manifest *m = nullptr;
    if ((rc = gms_manifest_create(entries, n, s->device, 0, &m)) != GMS_OK) return rc;
    DeviceGuard g(s->device);
    uint64_t *hash = nullptr;
    const uint64_t nb = gms_num_blocks(m);
    hipError_t e = hipMalloc((void **)&hash, std::max<uint64_t>(nb, 1) * sizeof(uint64_t));
    if (e != hipSuccess) {
        (void)hipGetLastError();
        gms_manifest_destroy(m);
        return fail(GMS_ERR_NOMEM, "store block hashes (%llu): %s", (unsigned long long)nb, hipGetErrorString(e));
    }
    uint64_t count = 0;
    // every device write of the writer, on any stream, lands before it is hashed
    if ((e = hipDeviceSynchronize()) != hipSuccess) rc = fail_hip(e, "hipDeviceSynchronize");
    if (rc == GMS_OK) rc = hash_and_compare(s, m, expected_blk, hash, nullptr, 0, &count, stream);
    if (rc == GMS_OK && count) {
        rc = fail(GMS_ERR_INTEGRITY, "%llu blocks differ from the expected hashes; commit refused",
                  (unsigned long long)count);
        if (mismatch_count_out) *mismatch_count_out = count;
    }
    if (rc == GMS_OK) rc = gms::pool_set_access_all(s->pool, true);
    if (rc != GMS_OK) {
        (void)hipFree(hash);
        gms_manifest_destroy(m);
        return rc;  // the writer keeps its lease
    }
    drop_layout(s);
    s->layout = m;
    s->d_hash = hash;
    s->writer = 0;
    s->invalid = false;
    s->state = GMS_STORE_COMMITTED;
    return GMS_OK;
}

int gms_store_abort(gms_store *s, uint64_t lease)
{
    gms::clear_error();
    if (!s) return fail(GMS_ERR_INVALID, "store is null");
    std::lock_guard<std::mutex> lock(s->mu);
    int rc = check_writer(s, lease);
    if (rc != GMS_OK) return rc;
    return discard(s);
}

int gms_store_connect_ro(gms_store *s, uint32_t flags, uint64_t *lease_out, uint64_t *mismatch_count_out, void *stream)
{
    gms::clear_error();
    if (mismatch_count_out) *mismatch_count_out = 0;
    if (!s || !lease_out) return fail(GMS_ERR_INVALID, "store or lease_out is null");
    if (flags & ~(uint32_t)GMS_CONNECT_VERIFY) return fail(GMS_ERR_INVALID, "flags %#x", flags);
    std::lock_guard<std::mutex> lock(s->mu);
    if (s->state != GMS_STORE_COMMITTED && s->state != GMS_STORE_RO)
        return fail(GMS_ERR_STATE, "store has %s", s->state == GMS_STORE_RW ? "a writer connected" : "no committed state");
    if (s->invalid) return fail(GMS_ERR_INTEGRITY, "committed state is invalid; a writer must repopulate it");
    if ((flags & GMS_CONNECT_VERIFY) && s->layout) {
        DeviceGuard g(s->device);
        uint64_t count = 0;
        int rc = hash_and_compare(s, s->layout, s->d_hash, nullptr, nullptr, 0, &count, stream);
        if (rc != GMS_OK) return rc;
        if (count) {
            s->invalid = true;
            if (mismatch_count_out) *mismatch_count_out = count;
            return fail(GMS_ERR_INTEGRITY, "%llu committed blocks changed; read-only lease refused",
                        (unsigned long long)count);
        }
    }
    const uint64_t id = s->next_lease++;
    s->readers.insert(id);
    s->state = GMS_STORE_RO;
    *lease_out = id;
    return GMS_OK;
}

int gms_store_verify(gms_store *s, uint64_t *mismatch_count_out, uint64_t *mismatch_list_out, uint64_t cap,
                     void *stream)
{
    gms::clear_error();
    if (!s || !mismatch_count_out) return fail(GMS_ERR_INVALID, "store or mismatch_count_out is null");
    *mismatch_count_out = 0;
    std::lock_guard<std::mutex> lock(s->mu);
    if (s->state != GMS_STORE_COMMITTED && s->state != GMS_STORE_RO)
        return fail(GMS_ERR_STATE, "nothing committed");
    if (!s->layout) return GMS_OK;
    DeviceGuard g(s->device);
    int rc = hash_and_compare(s, s->layout, s->d_hash, nullptr, mismatch_list_out, cap, mismatch_count_out, stream);
    if (rc != GMS_OK) return rc;
    if (*mismatch_count_out) s->invalid = true;
    return GMS_OK;
}

int gms_store_disconnect(gms_store *s, uint64_t lease)
{
    gms::clear_error();
    if (!s) return fail(GMS_ERR_INVALID, "store is null");
    std::lock_guard<std::mutex> lock(s->mu);
    if (lease != 0 && lease == s->writer) return discard(s);  // a writer leaving before commit
    auto it = s->readers.find(lease);
    if (it == s->readers.end()) return fail(GMS_ERR_INVALID, "lease %llu is not held", (unsigned long long)lease);
    s->readers.erase(it);
    if (s->readers.empty()) s->state = GMS_STORE_COMMITTED;
    return GMS_OK;
}

const gms_manifest *gms_store_layout(const gms_store *s) { return s ? s->layout : nullptr; }

const uint64_t *gms_store_block_hashes(const gms_store *s) { return s ? s->d_hash : nullptr; }

}  // extern "C"
