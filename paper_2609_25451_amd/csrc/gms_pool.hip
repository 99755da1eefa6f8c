// Device memory pool over HIP virtual memory management.
//
// GMS owns physical allocations and maps them for engines, amortising the
// virtual-memory operations with a first-fit suballocator over 2 GiB slabs and
// dedicated slabs for larger allocations (paper section 4, GMS); mapped ranges
// can be made read-only so that readers cannot modify shared state (section
// 3.2).  Before a checkpoint the engine releases its KV pages but keeps their
// virtual-address reservations, so addresses captured in graphs and tensors
// stay valid, and fresh pages are mapped at the same addresses after restore
// (section 3.1, section 3.3).  A mapping (slab or dedicated) is the unit of
// release, remap and access change, and each mapping has a VA reservation of
// its own: when mappings of different sizes share one reservation, HIP's
// access changes on one of them fail at random (measured on this ROCm, where
// one reservation per mapping never failed).  Reservations are placed one
// after another in the pool's address window while the address space allows,
// so consecutive allocations stay contiguous.

#include <algorithm>
#include <cstdio>
#include <map>
#include <mutex>
#include <new>
#include <vector>

#include "gms_host.h"

using gms::DeviceGuard;
using gms::fail;
using gms::fail_hip;

namespace {

struct Mapping {
    uint64_t bytes = 0;
    hipMemGenericAllocationHandle_t handle{};
    bool mapped = false;
    bool read_only = false;
    bool dedicated = false;
    std::map<uint64_t, uint64_t> free;  // slab only: offset -> bytes, coalesced
};

struct Alloc {
    uint64_t bytes;
    uint64_t map_va;  // mapping that holds it
};

uint64_t round_up(uint64_t v, uint64_t a) { return (v + a - 1) / a * a; }

}  // namespace

struct gms_pool {
    int device = 0;
    uint64_t base = 0, reserved = 0;  // address window (placement hint) and VA budget
    uint64_t next = 0;                // window offset where the next mapping is placed
    uint64_t used = 0;                // VA held by the mappings' reservations
    uint64_t gran = 0, slab_bytes = 0;
    std::map<uint64_t, Mapping> maps;   // by VA
    std::map<uint64_t, Alloc> allocs;   // by address
    std::mutex mu;
};

namespace {

hipMemAllocationProp device_prop(int device)
{
    hipMemAllocationProp prop = {};
    prop.type = hipMemAllocationTypePinned;
    prop.location.type = hipMemLocationTypeDevice;
    prop.location.id = device;
    return prop;
}

int set_access(gms_pool *p, uint64_t va, uint64_t bytes, bool read_only)
{
    hipMemAccessDesc acc = {};
    acc.location = device_prop(p->device).location;
    acc.flags = read_only ? hipMemAccessFlagsProtRead : hipMemAccessFlagsProtReadWrite;
    hipError_t e = hipMemSetAccess((void *)(uintptr_t)va, bytes, &acc, 1);
    if (e == hipSuccess) return GMS_OK;
    (void)hipGetLastError();
    return fail(GMS_ERR_HIP, "hipMemSetAccess(va %#llx, %llu bytes, %s; granularity %llu): %s (%d)",
                (unsigned long long)va, (unsigned long long)bytes, read_only ? "read-only" : "read-write",
                (unsigned long long)p->gran, hipGetErrorString(e), (int)e);
}

// Creates physical memory for mapping `m` at `va` and maps it read-write.
int back(gms_pool *p, uint64_t va, Mapping &m)
{
    hipMemAllocationProp prop = device_prop(p->device);
    hipError_t e = hipMemCreate(&m.handle, m.bytes, &prop, 0);
    if (e != hipSuccess) {
        (void)hipGetLastError();
        return fail(GMS_ERR_NOMEM, "hipMemCreate(%llu): %s", (unsigned long long)m.bytes, hipGetErrorString(e));
    }
    if ((e = hipMemMap((void *)(uintptr_t)va, m.bytes, 0, m.handle, 0)) != hipSuccess) {
        (void)hipMemRelease(m.handle);
        (void)hipGetLastError();
        return fail(GMS_ERR_HIP, "hipMemMap(va %#llx, %llu bytes): %s (%d)", (unsigned long long)va,
                    (unsigned long long)m.bytes, hipGetErrorString(e), (int)e);
    }
    int rc = set_access(p, va, m.bytes, false);
    if (rc != GMS_OK) {
        (void)hipMemUnmap((void *)(uintptr_t)va, m.bytes);
        (void)hipMemRelease(m.handle);
        return rc;
    }
    m.mapped = true;
    m.read_only = false;
    return GMS_OK;
}

int unback(uint64_t va, Mapping &m)
{
    hipError_t e = hipMemUnmap((void *)(uintptr_t)va, m.bytes);
    if (e != hipSuccess) return fail_hip(e, "hipMemUnmap");
    if ((e = hipMemRelease(m.handle)) != hipSuccess) return fail_hip(e, "hipMemRelease");
    m.mapped = false;
    return GMS_OK;
}

constexpr uint64_t kLargePage = 2ull << 20;

// New mapping of `bytes` with a reservation of its own, at the next address of
// the window when that is free, elsewhere otherwise.
int new_mapping(gms_pool *p, uint64_t bytes, bool dedicated, uint64_t *va_out)
{
    if (p->used + bytes > p->reserved || p->used + bytes < p->used)
        return fail(GMS_ERR_NOMEM, "pool VA budget of %llu bytes exhausted", (unsigned long long)p->reserved);
    const uint64_t align = bytes % kLargePage == 0 ? std::max(kLargePage, p->gran) : p->gran;
    const uint64_t off = round_up(p->next, align);
    void *want = off + bytes <= p->reserved ? (void *)(uintptr_t)(p->base + off) : nullptr;
    void *res = nullptr;
    hipError_t e = hipMemAddressReserve(&res, bytes, align, want, 0);
    if (e != hipSuccess && want) {
        (void)hipGetLastError();
        e = hipMemAddressReserve(&res, bytes, align, nullptr, 0);
    }
    if (e != hipSuccess) {
        (void)hipGetLastError();
        return fail(GMS_ERR_NOMEM, "hipMemAddressReserve(%llu): %s", (unsigned long long)bytes, hipGetErrorString(e));
    }
    const uint64_t va = (uint64_t)(uintptr_t)res;
    Mapping m;
    m.bytes = bytes;
    m.dedicated = dedicated;
    int rc = back(p, va, m);
    if (rc != GMS_OK) {
        (void)hipMemAddressFree(res, bytes);
        return rc;
    }
    if (!dedicated) m.free[0] = bytes;
    p->maps[va] = std::move(m);
    p->used += bytes;
    if (res == want) p->next = off + bytes;
    *va_out = va;
    return GMS_OK;
}

// Unmaps (if backed) and frees the reservation of the mapping at `va`.
int drop_mapping(gms_pool *p, uint64_t va, Mapping &m)
{
    if (m.mapped) {
        int rc = unback(va, m);
        if (rc != GMS_OK) return rc;
    }
    hipError_t e = hipMemAddressFree((void *)(uintptr_t)va, m.bytes);
    if (e != hipSuccess) return fail_hip(e, "hipMemAddressFree");
    p->used -= m.bytes;
    return GMS_OK;
}

// The mappings that exactly tile [addr, addr + bytes); GMS_ERR_INVALID otherwise.
int whole_mappings(gms_pool *p, uint64_t addr, uint64_t bytes, std::vector<uint64_t> *out)
{
    uint64_t cur = addr;
    const uint64_t end = addr + bytes;
    auto it = p->maps.find(addr);
    while (cur < end) {
        if (it == p->maps.end() || it->first != cur)
            return fail(GMS_ERR_INVALID, "range [%#llx, %#llx) does not tile whole pool mappings",
                        (unsigned long long)addr, (unsigned long long)end);
        out->push_back(cur);
        cur += it->second.bytes;
        ++it;
    }
    if (cur != end || bytes == 0)
        return fail(GMS_ERR_INVALID, "range [%#llx, %#llx) does not tile whole pool mappings",
                    (unsigned long long)addr, (unsigned long long)end);
    return GMS_OK;
}

}  // namespace

namespace gms {

// Discards every allocation: unmaps and releases all physical memory and
// rewinds the reservation, which the pool keeps.
int pool_reset(gms_pool *p)
{
    std::lock_guard<std::mutex> lock(p->mu);
    DeviceGuard g(p->device);
    if (g.err != hipSuccess) return fail_hip(g.err, "hipSetDevice");
    hipError_t e = hipDeviceSynchronize();  // no kernel may still touch the pages
    if (e != hipSuccess) return fail_hip(e, "hipDeviceSynchronize");
    while (!p->maps.empty()) {
        auto it = p->maps.begin();
        int rc = drop_mapping(p, it->first, it->second);
        if (rc != GMS_OK) return rc;
        p->maps.erase(it);
    }
    p->allocs.clear();
    p->next = 0;
    return GMS_OK;
}

// Read-only or read-write device access for every backed mapping.
int pool_set_access_all(gms_pool *p, bool read_only)
{
    std::lock_guard<std::mutex> lock(p->mu);
    DeviceGuard g(p->device);
    if (g.err != hipSuccess) return fail_hip(g.err, "hipSetDevice");
    // device writes still in flight, on any stream, must land before their pages turn read-only
    if (read_only) {
        hipError_t e = hipDeviceSynchronize();
        if (e != hipSuccess) return fail_hip(e, "hipDeviceSynchronize");
    }
    for (auto &kv : p->maps) {
        Mapping &m = kv.second;
        if (!m.mapped) continue;
        int rc = set_access(p, kv.first, m.bytes, read_only);
        if (rc != GMS_OK) return rc;
        m.read_only = read_only;
    }
    return GMS_OK;
}

// True when [addr, addr + bytes) lies inside one allocation of the pool.
bool pool_holds(gms_pool *p, uint64_t addr, uint64_t bytes)
{
    std::lock_guard<std::mutex> lock(p->mu);
    auto it = p->allocs.upper_bound(addr);
    if (it == p->allocs.begin()) return false;
    --it;
    return addr + bytes >= addr && addr + bytes <= it->first + it->second.bytes;
}

int pool_device(const gms_pool *p) { return p->device; }

}  // namespace gms

extern "C" {

int gms_pool_create(int device, uint64_t va_bytes, uint64_t slab_bytes, gms_pool **out)
{
    gms::clear_error();
    if (!out) return fail(GMS_ERR_INVALID, "out is null");
    *out = nullptr;
    if (device < 0) return fail(GMS_ERR_INVALID, "device %d", device);
    DeviceGuard g(device);
    if (g.err != hipSuccess) return fail_hip(g.err, "hipSetDevice");
    int vmm = 0;
    hipError_t e = hipDeviceGetAttribute(&vmm, hipDeviceAttributeVirtualMemoryManagementSupported, device);
    if (e != hipSuccess) return fail_hip(e, "hipDeviceGetAttribute");
    if (!vmm) return fail(GMS_ERR_STATE, "device %d has no virtual memory management", device);
    hipMemAllocationProp prop = device_prop(device);
    size_t gran = 0;
    if ((e = hipMemGetAllocationGranularity(&gran, &prop, hipMemAllocationGranularityRecommended)) != hipSuccess)
        return fail_hip(e, "hipMemGetAllocationGranularity");
    if (slab_bytes == 0) slab_bytes = 2ull << 30;
    if (slab_bytes % gran || va_bytes == 0 || va_bytes % gran)
        return fail(GMS_ERR_INVALID, "va_bytes %llu and slab_bytes %llu must be non-zero multiples of %zu",
                    (unsigned long long)va_bytes, (unsigned long long)slab_bytes, gran);
    gms_pool *p = new (std::nothrow) gms_pool;
    if (!p) return fail(GMS_ERR_NOMEM, "pool");
    // find a free window of va_bytes; mappings reserve their own ranges in it
    void *va = nullptr;
    if ((e = hipMemAddressReserve(&va, va_bytes, std::max<uint64_t>(kLargePage, gran), nullptr, 0)) != hipSuccess) {
        delete p;
        (void)hipGetLastError();
        return fail(GMS_ERR_NOMEM, "hipMemAddressReserve(%llu): %s", (unsigned long long)va_bytes,
                    hipGetErrorString(e));
    }
    if ((e = hipMemAddressFree(va, va_bytes)) != hipSuccess) {
        delete p;
        return fail_hip(e, "hipMemAddressFree");
    }
    p->device = device;
    p->base = (uint64_t)(uintptr_t)va;
    p->reserved = va_bytes;
    p->gran = gran;
    p->slab_bytes = slab_bytes;
    *out = p;
    return GMS_OK;
}

void gms_pool_destroy(gms_pool *p)
{
    if (!p) return;
    {
        DeviceGuard g(p->device);
        (void)hipDeviceSynchronize();
        for (auto &kv : p->maps) (void)drop_mapping(p, kv.first, kv.second);
        (void)hipGetLastError();
    }
    delete p;
}

int gms_pool_alloc(gms_pool *p, uint64_t bytes, uint64_t align, uint64_t *addr_out)
{
    gms::clear_error();
    if (!p || !addr_out) return fail(GMS_ERR_INVALID, "pool or addr_out is null");
    if (align == 0) align = 256;
    if (bytes == 0 || (align & (align - 1)) || align > p->gran)
        return fail(GMS_ERR_INVALID, "bytes %llu / align %llu (power of two <= %llu)", (unsigned long long)bytes,
                    (unsigned long long)align, (unsigned long long)p->gran);
    if (bytes > p->reserved)
        return fail(GMS_ERR_NOMEM, "%llu bytes exceed the pool's VA budget of %llu", (unsigned long long)bytes,
                    (unsigned long long)p->reserved);
    std::lock_guard<std::mutex> lock(p->mu);
    DeviceGuard g(p->device);
    if (g.err != hipSuccess) return fail_hip(g.err, "hipSetDevice");
    const uint64_t need = round_up(bytes, align);
    if (need > p->slab_bytes) {  // dedicated mapping
        uint64_t va = 0;
        int rc = new_mapping(p, round_up(bytes, p->gran), true, &va);
        if (rc != GMS_OK) return rc;
        p->allocs[va] = Alloc{bytes, va};
        *addr_out = va;
        return GMS_OK;
    }
    for (int attempt = 0; attempt < 2; ++attempt) {
        for (auto &kv : p->maps) {  // first fit, in VA order
            Mapping &m = kv.second;
            if (m.dedicated || !m.mapped) continue;
            for (auto f = m.free.begin(); f != m.free.end(); ++f) {
                const uint64_t start = round_up(kv.first + f->first, align) - kv.first;
                if (start + need > f->first + f->second) continue;
                const uint64_t f_off = f->first, f_len = f->second;
                m.free.erase(f);
                if (start > f_off) m.free[f_off] = start - f_off;
                if (start + need < f_off + f_len) m.free[start + need] = f_off + f_len - (start + need);
                const uint64_t addr = kv.first + start;
                p->allocs[addr] = Alloc{need, kv.first};
                *addr_out = addr;
                return GMS_OK;
            }
        }
        if (attempt == 0) {
            uint64_t va = 0;
            int rc = new_mapping(p, p->slab_bytes, false, &va);
            if (rc != GMS_OK) return rc;
        }
    }
    return fail(GMS_ERR_NOMEM, "no slab space for %llu bytes", (unsigned long long)bytes);
}

int gms_pool_free(gms_pool *p, uint64_t addr)
{
    gms::clear_error();
    if (!p) return fail(GMS_ERR_INVALID, "pool is null");
    std::lock_guard<std::mutex> lock(p->mu);
    auto a = p->allocs.find(addr);
    if (a == p->allocs.end()) return fail(GMS_ERR_INVALID, "%#llx is not a pool allocation", (unsigned long long)addr);
    Mapping &m = p->maps[a->second.map_va];
    if (m.dedicated) {
        DeviceGuard g(p->device);
        if (m.mapped) (void)hipDeviceSynchronize();
        int rc = drop_mapping(p, a->second.map_va, m);
        if (rc != GMS_OK) return rc;
        p->maps.erase(a->second.map_va);
    } else {
        uint64_t off = addr - a->second.map_va, len = a->second.bytes;
        auto nx = m.free.lower_bound(off);
        if (nx != m.free.end() && off + len == nx->first) {  // merge with the next free block
            len += nx->second;
            nx = m.free.erase(nx);
        }
        if (nx != m.free.begin()) {  // and with the previous one
            auto pv = std::prev(nx);
            if (pv->first + pv->second == off) {
                off = pv->first;
                len += pv->second;
                m.free.erase(pv);
            }
        }
        m.free[off] = len;
    }
    p->allocs.erase(a);
    return GMS_OK;
}

int gms_pool_release(gms_pool *p, uint64_t addr, uint64_t bytes)
{
    gms::clear_error();
    if (!p) return fail(GMS_ERR_INVALID, "pool is null");
    std::lock_guard<std::mutex> lock(p->mu);
    std::vector<uint64_t> vas;
    int rc = whole_mappings(p, addr, bytes, &vas);
    if (rc != GMS_OK) return rc;
    DeviceGuard g(p->device);
    if (g.err != hipSuccess) return fail_hip(g.err, "hipSetDevice");
    hipError_t e = hipDeviceSynchronize();  // no kernel may still touch the pages
    if (e != hipSuccess) return fail_hip(e, "hipDeviceSynchronize");
    for (uint64_t va : vas) {
        Mapping &m = p->maps[va];
        if (m.mapped && (rc = unback(va, m)) != GMS_OK) return rc;
    }
    return GMS_OK;
}

int gms_pool_remap(gms_pool *p, uint64_t addr, uint64_t bytes)
{
    gms::clear_error();
    if (!p) return fail(GMS_ERR_INVALID, "pool is null");
    std::lock_guard<std::mutex> lock(p->mu);
    std::vector<uint64_t> vas;
    int rc = whole_mappings(p, addr, bytes, &vas);
    if (rc != GMS_OK) return rc;
    DeviceGuard g(p->device);
    if (g.err != hipSuccess) return fail_hip(g.err, "hipSetDevice");
    for (uint64_t va : vas) {
        Mapping &m = p->maps[va];
        if (!m.mapped && (rc = back(p, va, m)) != GMS_OK) return rc;
    }
    return GMS_OK;
}

int gms_pool_set_access(gms_pool *p, uint64_t addr, uint64_t bytes, int read_only)
{
    gms::clear_error();
    if (!p) return fail(GMS_ERR_INVALID, "pool is null");
    std::lock_guard<std::mutex> lock(p->mu);
    std::vector<uint64_t> vas;
    int rc = whole_mappings(p, addr, bytes, &vas);
    if (rc != GMS_OK) return rc;
    DeviceGuard g(p->device);
    if (g.err != hipSuccess) return fail_hip(g.err, "hipSetDevice");
    for (uint64_t va : vas)
        if (!p->maps[va].mapped) return fail(GMS_ERR_STATE, "mapping at %#llx is released", (unsigned long long)va);
    // device writes still in flight, on any stream, must land before their pages turn read-only
    if (read_only) {
        hipError_t e = hipDeviceSynchronize();
        if (e != hipSuccess) return fail_hip(e, "hipDeviceSynchronize");
    }
    for (uint64_t va : vas) {
        Mapping &m = p->maps[va];
        if ((rc = set_access(p, va, m.bytes, read_only != 0)) != GMS_OK) return rc;
        m.read_only = read_only != 0;
    }
    return GMS_OK;
}

int gms_pool_info(const gms_pool *cp, uint64_t *base, uint64_t *reserved, uint64_t *mapped_bytes,
                  uint64_t *mappings, uint64_t *granularity)
{
    if (!cp) return fail(GMS_ERR_INVALID, "pool is null");
    gms_pool *p = const_cast<gms_pool *>(cp);
    std::lock_guard<std::mutex> lock(p->mu);
    uint64_t mapped = 0, n = 0;
    for (auto &kv : p->maps) {
        ++n;
        if (kv.second.mapped) mapped += kv.second.bytes;
    }
    if (base) *base = p->base;
    if (reserved) *reserved = p->reserved;
    if (mapped_bytes) *mapped_bytes = mapped;
    if (mappings) *mappings = n;
    if (granularity) *granularity = p->gran;
    return GMS_OK;
}

// The mapping that holds `addr`: its start and size, and whether it is backed.
int gms_pool_mapping_of(const gms_pool *cp, uint64_t addr, uint64_t *map_addr, uint64_t *map_bytes, int *mapped)
{
    if (!cp) return fail(GMS_ERR_INVALID, "pool is null");
    gms_pool *p = const_cast<gms_pool *>(cp);
    std::lock_guard<std::mutex> lock(p->mu);
    auto it = p->maps.upper_bound(addr);
    if (it == p->maps.begin()) return fail(GMS_ERR_INVALID, "%#llx is outside every mapping", (unsigned long long)addr);
    --it;
    if (addr >= it->first + it->second.bytes)
        return fail(GMS_ERR_INVALID, "%#llx is outside every mapping", (unsigned long long)addr);
    if (map_addr) *map_addr = it->first;
    if (map_bytes) *map_bytes = it->second.bytes;
    if (mapped) *mapped = it->second.mapped ? 1 : 0;
    return GMS_OK;
}

}  // extern "C"
