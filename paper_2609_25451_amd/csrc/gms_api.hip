// Host side of libgms: manifest validation and layout, the chunked work
// list, argument checks, and the pinned-host staging ring.  Every exported
// function is declared in include/gms.h, which documents its contract.

#include <algorithm>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <new>
#include <string>
#include <vector>

#include "gms_host.h"

using gms::Chunk;
using gms::HashOut;
using gms::ceil_div;
using gms::DeviceGuard;
using gms::fail;
using gms::fail_hip;
using gms::kMaxChunk;
using gms::kDefaultSlice;
using gms::kMaxSlots;
using gms::kMaxSlice;

namespace {
thread_local std::string g_last_error;
}  // namespace

namespace gms {

int fail(int status, const char *fmt, ...)
{
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    g_last_error = buf;
    return status;
}

int fail_hip(hipError_t e, const char *what)
{
    (void)hipGetLastError();  // reported here: keep it from resurfacing in a later launch check
    return fail(GMS_ERR_HIP, "%s: %s (%d)", what, hipGetErrorString(e), (int)e);
}

void clear_error() { g_last_error.clear(); }

void free_ring(gms_manifest *m)
{
    if (m->copy_stream) (void)hipStreamSynchronize(m->copy_stream);
    if (m->ev_done && m->done_recorded) (void)hipEventSynchronize(m->ev_done);
    for (uint32_t i = 0; i < kMaxSlots; ++i) {
        if (m->ev_filled[i]) (void)hipEventDestroy(m->ev_filled[i]);
        if (m->ev_free[i]) (void)hipEventDestroy(m->ev_free[i]);
        if (m->ev_host[i]) (void)hipEventDestroy(m->ev_host[i]);
        m->ev_filled[i] = m->ev_free[i] = m->ev_host[i] = nullptr;
    }
    if (m->h_ring) (void)hipHostFree(m->h_ring);
    m->h_ring = nullptr;
    m->host_slots = 0;
    if (m->ev_entry) (void)hipEventDestroy(m->ev_entry);
    if (m->ev_done) (void)hipEventDestroy(m->ev_done);
    if (m->copy_stream) (void)hipStreamDestroy(m->copy_stream);
    if (m->d_ring) (void)hipFree(m->d_ring);
    m->ev_entry = m->ev_done = nullptr;
    m->copy_stream = nullptr;
    m->d_ring = nullptr;
    m->ring_slice = 0;
    m->ring_slots = 0;
    m->done_recorded = false;
    m->slice_first.clear();
}

// Ring geometry actually used: slice rounded down to whole chunks.
uint64_t effective_slice(const gms_manifest *m)
{
    uint64_t s = m->slice_bytes / m->chunk_bytes * m->chunk_bytes;
    return s ? s : m->chunk_bytes;
}

int ensure_ring(gms_manifest *m)
{
    const uint64_t slice = effective_slice(m);
    if (m->slots == 0) return GMS_OK;  // zero-copy mode
    if (m->d_ring && m->ring_slice == slice && m->ring_slots == m->slots) return GMS_OK;
    free_ring(m);
    hipError_t e = hipMalloc((void **)&m->d_ring, slice * m->slots);
    if (e != hipSuccess) {
        m->d_ring = nullptr;
        (void)hipGetLastError();
        return fail(GMS_ERR_NOMEM, "staging ring: hipMalloc(%llu) failed: %s",
                    (unsigned long long)(slice * m->slots), hipGetErrorString(e));
    }
    if ((e = hipStreamCreateWithFlags(&m->copy_stream, hipStreamNonBlocking)) != hipSuccess)
        return free_ring(m), fail_hip(e, "staging ring: hipStreamCreate");
    for (uint32_t i = 0; i < m->slots; ++i) {
        if ((e = hipEventCreateWithFlags(&m->ev_filled[i], hipEventDisableTiming)) != hipSuccess ||
            (e = hipEventCreateWithFlags(&m->ev_free[i], hipEventDisableTiming)) != hipSuccess)
            return free_ring(m), fail_hip(e, "staging ring: hipEventCreate");
    }
    if ((e = hipEventCreateWithFlags(&m->ev_entry, hipEventDisableTiming)) != hipSuccess ||
        (e = hipEventCreateWithFlags(&m->ev_done, hipEventDisableTiming)) != hipSuccess)
        return free_ring(m), fail_hip(e, "staging ring: hipEventCreate");
    m->ring_slice = slice;
    m->ring_slots = m->slots;
    // chunk ranges per group and slice; chunks never straddle a slice
    // (slice % chunk == 0) and are in image order within a group
    const uint64_t nslices = ceil_div(m->image_bytes, slice);
    m->slice_first.assign(m->groups.size() * (nslices + 1), 0);
    for (size_t g = 0; g < m->groups.size(); ++g) {
        const gms::LaunchGroup &lg = m->groups[g];
        uint64_t ci = lg.first;
        for (uint64_t s = 0; s < nslices; ++s) {
            while (ci < lg.first + lg.count && m->chunks[ci].img < s * slice) ++ci;
            m->slice_first[g * (nslices + 1) + s] = ci;
        }
        m->slice_first[g * (nslices + 1) + nslices] = lg.first + lg.count;
    }
    return GMS_OK;
}

// Work units a chunk needs as a power of two: the smallest s with 2^s units of
// kBlocksPerUnit blocks covering it.
uint32_t unit_class(uint32_t len)
{
    const uint64_t units = ceil_div(ceil_div(len, kBlockBytes), kBlocksPerUnit);
    uint32_t s = 0;
    while ((1ull << s) < units) ++s;
    return s;
}

// Idle work units that justify one more launch: an idle workgroup costs about
// 0.7 ns of the whole chip (measured: 1.4 M of them added 1.0 ms to a restore),
// a launch some microseconds.
constexpr uint64_t kSplitUnits = 16384;

void plan_launch_groups(gms_manifest *m)
{
    // One launch covers a set of chunks with the units of the largest, so a
    // chunk that needs fewer units leaves the rest idle.  Walking the classes
    // from the largest down, a class gets a launch of its own (shared with the
    // smaller classes after it) once the idle units it would leave reach
    // kSplitUnits; a manifest of similar chunks stays one launch.  Chunks of
    // entries that are not 16-byte aligned then get launches of their own
    // beside the aligned ones of the same size, so that each kernel carries
    // only one of the two access paths.
    const uint64_t n = m->chunks.size();
    std::vector<uint8_t> cls(n);
    uint64_t count[kMaxUnitShift + 1] = {};
    for (uint64_t i = 0; i < n; ++i) ++count[cls[i] = (uint8_t)unit_class(m->chunks[i].len)];
    uint32_t group_of[kMaxUnitShift + 1] = {};
    int top = kMaxUnitShift;
    while (top > 0 && count[top] == 0) --top;
    uint32_t g = (uint32_t)top;
    std::vector<uint32_t> shifts;  // group shifts, largest first
    for (int s = top; s >= 0; --s) {
        if (count[s] && (uint32_t)s < g && count[s] * ((1ull << g) - (1ull << s)) >= kSplitUnits) g = (uint32_t)s;
        group_of[s] = g;
        if (count[s] && (shifts.empty() || shifts.back() != g)) shifts.push_back(g);
    }
    auto shifted = [&](uint64_t i) { return (m->chunks[i].addr & 15) != 0; };
    bool present[kMaxUnitShift + 1][2] = {};
    for (uint64_t i = 0; i < n; ++i) present[group_of[cls[i]]][shifted(i) ? 1 : 0] = true;
    // groups: (shift, aligned) for each shift, largest first, aligned before shifted
    std::vector<LaunchGroup> plan;
    for (uint32_t sh : shifts)
        for (int k = 0; k < 2; ++k)
            if (present[sh][k]) plan.push_back(LaunchGroup{0, 0, sh, k == 1});
    m->groups.clear();
    if (plan.size() == 1) {
        plan[0].count = n;
        m->groups.push_back(plan[0]);
    } else {
        // chunks by group, in image order within a group
        std::vector<Chunk> sorted;
        sorted.reserve(n);
        for (LaunchGroup lg : plan) {
            lg.first = sorted.size();
            for (uint64_t i = 0; i < n; ++i)
                if (group_of[cls[i]] == lg.shift && shifted(i) == lg.shifted) sorted.push_back(m->chunks[i]);
            lg.count = sorted.size() - lg.first;
            m->groups.push_back(lg);
        }
        m->chunks.swap(sorted);
    }
    // A group whose chunks are mostly whole entries of their own (a KV pool's
    // live units: entries scattered over the pool) restores and snapshots in
    // the striped unit order; one of large tensors cut into many chunks keeps
    // the contiguous eighths.  The chunks of an entry are adjacent in a group.
    // Paired launches (one unit per chunk) keep their own order.
    for (LaunchGroup &lg : m->groups) {
        uint64_t entries = 0;
        for (uint64_t i = lg.first; i < lg.first + lg.count; ++i)
            entries += i == lg.first || m->chunks[i].entry != m->chunks[i - 1].entry;
        lg.striped = lg.shift > 0 && lg.count && 2 * entries >= lg.count;
    }
}

hipError_t launch_all(const gms_manifest *m, int op, const HashOut &h, uint8_t *img_base, hipStream_t s)
{
    for (const LaunchGroup &g : m->groups) {
        hipError_t e =
            launch_stream(op, h.any(), g.shifted, g.striped, m->d_chunks, g.first, g.count, g.shift, img_base, 0, h, s);
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

hipError_t launch_slice(const gms_manifest *m, int op, const HashOut &h, uint64_t sl, uint8_t *slot, hipStream_t s)
{
    const uint64_t stride = ceil_div(m->image_bytes, m->ring_slice) + 1;
    for (size_t g = 0; g < m->groups.size(); ++g) {
        const uint64_t c0 = m->slice_first[g * stride + sl], c1 = m->slice_first[g * stride + sl + 1];
        hipError_t e =
            launch_stream(op, h.any(), m->groups[g].shifted, m->groups[g].striped, m->d_chunks, c0, c1 - c0,
                          m->groups[g].shift, slot, sl * m->ring_slice, h, s);
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

int refuse_capture(hipStream_t s, const char *what)
{
    hipStreamCaptureStatus cap = hipStreamCaptureStatusNone;
    hipError_t e = hipStreamIsCapturing(s, &cap);
    if (e != hipSuccess) return fail_hip(e, "hipStreamIsCapturing");
    if (cap != hipStreamCaptureStatusNone) return fail(GMS_ERR_STATE, "%s: not allowed under stream capture", what);
    return GMS_OK;
}

int ensure_host_ring(gms_manifest *m)
{
    int rc = ensure_ring(m);
    if (rc != GMS_OK) return rc;
    if (!m->d_ring) return fail(GMS_ERR_STATE, "image-file and host-image calls need the staging ring (slots > 0)");
    if (m->h_ring) return GMS_OK;
    const uint32_t hk = std::min<uint32_t>(kMaxSlots, 2 * m->ring_slots);
    hipError_t e = hipHostMalloc((void **)&m->h_ring, m->ring_slice * hk, hipHostMallocDefault);
    if (e != hipSuccess) {
        m->h_ring = nullptr;
        (void)hipGetLastError();
        return fail(GMS_ERR_NOMEM, "pinned host ring: hipHostMalloc(%llu) failed: %s",
                    (unsigned long long)(m->ring_slice * hk), hipGetErrorString(e));
    }
    for (uint32_t i = 0; i < hk; ++i)
        if ((e = hipEventCreateWithFlags(&m->ev_host[i], hipEventDisableTiming)) != hipSuccess) {
            for (uint32_t j = 0; j < i; ++j) (void)hipEventDestroy(m->ev_host[j]), m->ev_host[j] = nullptr;
            (void)hipHostFree(m->h_ring);
            m->h_ring = nullptr;
            return fail_hip(e, "pinned host ring: hipEventCreate");
        }
    m->host_slots = hk;
    return GMS_OK;
}

// [ptr, ptr + bytes) must lie inside one device allocation of `device`.
int check_device_range(const void *ptr, uint64_t bytes, int device, const char *what)
{
    if (!ptr) return fail(GMS_ERR_INVALID, "%s: null pointer", what);
    hipPointerAttribute_t attr;
    hipError_t e = hipPointerGetAttributes(&attr, ptr);
    if (e != hipSuccess || attr.type != hipMemoryTypeDevice) {
        (void)hipGetLastError();
        return fail(GMS_ERR_INVALID, "%s: %p is not device memory", what, ptr);
    }
    if (attr.device != device)
        return fail(GMS_ERR_INVALID, "%s: %p belongs to device %d, manifest is on %d", what, ptr, attr.device,
                    device);
    hipDeviceptr_t base = nullptr;
    size_t size = 0;
    e = hipMemGetAddressRange(&base, &size, (hipDeviceptr_t)ptr);
    if (e != hipSuccess) {
        (void)hipGetLastError();
        return fail(GMS_ERR_INVALID, "%s: no allocation contains %p", what, ptr);
    }
    const uint64_t lo = (uint64_t)(uintptr_t)ptr, b = (uint64_t)(uintptr_t)base;
    if (lo + bytes > b + size)
        return fail(GMS_ERR_SIZE, "%s: %llu bytes at %p run past the end of its allocation", what,
                    (unsigned long long)bytes, ptr);
    return GMS_OK;
}

// [ptr, ptr + bytes) must lie inside one pinned host allocation.
int check_pinned(const void *ptr, uint64_t bytes, const char *what)
{
    if (!ptr) return fail(GMS_ERR_INVALID, "%s: null pointer", what);
    hipPointerAttribute_t attr;
    hipError_t e = hipPointerGetAttributes(&attr, ptr);
    if (e != hipSuccess || attr.type != hipMemoryTypeHost) {
        (void)hipGetLastError();
        return fail(GMS_ERR_INVALID, "%s: %p is not pinned host memory", what, ptr);
    }
    hipDeviceptr_t base = nullptr;
    size_t size = 0;
    e = hipMemGetAddressRange(&base, &size, (hipDeviceptr_t)ptr);
    if (e != hipSuccess) {
        (void)hipGetLastError();
        return fail(GMS_ERR_INVALID, "%s: no pinned allocation contains %p", what, ptr);
    }
    const uint64_t lo = (uint64_t)(uintptr_t)ptr, b = (uint64_t)(uintptr_t)base;
    if (lo + bytes > b + size)
        return fail(GMS_ERR_SIZE, "%s: %llu bytes at %p run past the end of its pinned allocation", what,
                    (unsigned long long)bytes, ptr);
    return GMS_OK;
}

int check_common(const gms_manifest *m, const void *image, uint64_t image_bytes, int kind, bool need_image)
{
    if (!m) return fail(GMS_ERR_INVALID, "manifest is null");
    if (m->device < 0) return fail(GMS_ERR_STATE, "host-only manifest has no device");
    if (!need_image) return GMS_OK;
    if (kind != GMS_MEM_DEVICE && kind != GMS_MEM_HOST_PINNED)
        return fail(GMS_ERR_INVALID, "image kind %d is neither device nor pinned host", kind);
    if (image_bytes < m->image_bytes)
        return fail(GMS_ERR_SIZE, "image has %llu bytes, layout needs %llu", (unsigned long long)image_bytes,
                    (unsigned long long)m->image_bytes);
    if (m->image_bytes == 0) return GMS_OK;
    if (((uintptr_t)image & 15) != 0) return fail(GMS_ERR_INVALID, "image %p is not 16-byte aligned", image);
    if (kind == GMS_MEM_DEVICE) return check_device_range(image, m->image_bytes, m->device, "image");
    return check_pinned(image, m->image_bytes, "image");
}

int check_outputs(const gms_manifest *m, const HashOut &h)
{
    int rc;
    if (h.blk && (rc = check_device_range(h.blk, m->num_blocks * 8, m->device, "blk_hash")) != GMS_OK) return rc;
    if (h.ten && (rc = check_device_range(h.ten, m->n * 8, m->device, "ten_hash")) != GMS_OK) return rc;
    if (h.expected) {
        if ((rc = check_device_range(h.expected, m->num_blocks * 8, m->device, "expected_blk")) != GMS_OK) return rc;
        if (!h.mm_count) return fail(GMS_ERR_INVALID, "expected_blk given without mismatch_count_out");
        if ((rc = check_device_range(h.mm_count, 8, m->device, "mismatch_count")) != GMS_OK) return rc;
        // a call records each block at most once, so at most min(cap, blocks) list entries are written
        const uint64_t written = std::min<uint64_t>(h.mm_cap, m->num_blocks);
        if (h.mm_list && written &&
            (rc = check_device_range(h.mm_list, written * 8, m->device, "mismatch_list")) != GMS_OK)
            return rc;
    }
    return GMS_OK;
}

HashOut make_hash(const uint64_t *expected, uint64_t *blk, uint64_t *ten, uint64_t *cnt, uint64_t *list,
                  uint64_t cap)
{
    HashOut h;
    h.blk = blk;
    h.ten = ten;
    h.expected = expected;
    h.mm_count = expected ? cnt : nullptr;
    h.mm_list = (expected && cap) ? list : nullptr;
    h.mm_cap = (expected && list) ? cap : 0;
    return h;
}

}  // namespace gms

namespace {

using gms::make_hash;
using gms::check_common;
using gms::check_outputs;
using gms::ensure_ring;

// Device-resident image, or zero-copy access to a pinned one: one launch per
// launch group.
int run_direct(const gms_manifest *m, int op, uint8_t *image, const HashOut &h, hipStream_t s)
{
    hipError_t e = gms::launch_all(m, op, h, image, s);
    return e == hipSuccess ? GMS_OK : fail_hip(e, "kernel launch");
}

// A pinned image through the staging ring.  Restore: the copy kernel moves a
// slice into a device slot on the copy stream, then the scatter kernel reads
// the slot on the caller's stream.  Snapshot: the gather kernel fills the slot
// on the caller's stream, then the copy stream copies it to the host image.  The slot's producer reuses
// it only after its consumer is done with it.
int run_ring(gms_manifest *m, int op, const HashOut &h, uint8_t *host_image, hipStream_t s)
{
    int rc = ensure_ring(m);
    if (rc != GMS_OK) return rc;
    const uint64_t slice = m->ring_slice;
    const uint32_t k = m->ring_slots;
    const uint64_t nslices = ceil_div(m->image_bytes, slice);
    const bool to_host = op == gms::kSnapshot;
    hipStream_t producer = to_host ? s : m->copy_stream;
    hipStream_t consumer = to_host ? m->copy_stream : s;
    hipError_t e;
#define GMS_TRY(call)                                   \
    do {                                                \
        if ((e = (call)) != hipSuccess) return fail_hip(e, #call); \
    } while (0)

    // order after the caller's earlier work and after the previous ring call
    GMS_TRY(hipEventRecord(m->ev_entry, s));
    GMS_TRY(hipStreamWaitEvent(m->copy_stream, m->ev_entry, 0));
    if (m->done_recorded) {
        GMS_TRY(hipStreamWaitEvent(m->copy_stream, m->ev_done, 0));
        GMS_TRY(hipStreamWaitEvent(s, m->ev_done, 0));
    }
    uint8_t *host_dev = nullptr;  // the pinned image as the copy kernel sees it
    if (!to_host) GMS_TRY(hipHostGetDevicePointer((void **)&host_dev, host_image, 0));
    gms::RingFence fence(m, s);
    fence.armed = true;
    for (uint64_t sl = 0; sl < nslices; ++sl) {
        const uint32_t slot = (uint32_t)(sl % k);
        uint8_t *dev = m->d_ring + (uint64_t)slot * slice;
        const uint64_t lo = sl * slice;
        const uint64_t bytes = std::min(slice, m->image_bytes - lo);
        if (sl >= k) GMS_TRY(hipStreamWaitEvent(producer, m->ev_free[slot], 0));
        if (to_host)
            GMS_TRY(gms::launch_slice(m, op, h, sl, dev, s));
        else
            GMS_TRY(gms::launch_host_copy(host_dev + lo, dev, bytes, m->copy_stream));
        GMS_TRY(hipEventRecord(m->ev_filled[slot], producer));
        GMS_TRY(hipStreamWaitEvent(consumer, m->ev_filled[slot], 0));
        if (to_host)
            GMS_TRY(hipMemcpyAsync(host_image + lo, dev, bytes, hipMemcpyDeviceToHost, m->copy_stream));
        else
            GMS_TRY(gms::launch_slice(m, op, h, sl, dev, s));
        GMS_TRY(hipEventRecord(m->ev_free[slot], consumer));
    }
    // the call ends on the caller's stream once the last slot is consumed
    GMS_TRY(fence.close());
#undef GMS_TRY
    return GMS_OK;
}

// Device images take one launch per launch group.  A pinned image goes through
// the staging ring, except with no ring slots, and except a snapshot with slices below
// gms::kRingSnapshotMinSlice: those access the image zero-copy over the host link.
int run_op(const gms_manifest *cm, int op, void *image, int kind, const HashOut &h, void *stream)
{
    gms_manifest *m = const_cast<gms_manifest *>(cm);
    DeviceGuard g(m->device);
    if (g.err != hipSuccess) return fail_hip(g.err, "hipSetDevice");
    hipStream_t s = (hipStream_t)stream;
    hipError_t e;
    const bool pinned = op != gms::kVerify && kind != GMS_MEM_DEVICE;
    // the pinned-host paths order themselves across calls with events on the
    // library's copy stream, which a captured graph could not replay faithfully
    int rc;
    if (pinned && (rc = gms::refuse_capture(s, "a pinned-host image (device images can be captured)")) != GMS_OK)
        return rc;
    if ((e = gms::launch_prologue(h, m->n, s)) != hipSuccess) return fail_hip(e, "prologue launch");
    if (m->chunks.empty()) return GMS_OK;
    if (!pinned) return run_direct(m, op, (uint8_t *)image, h, s);
    std::lock_guard<std::mutex> lock(m->ring_mu);
    const bool zero_copy =
        m->slots == 0 || (op == gms::kSnapshot && gms::effective_slice(m) < gms::kRingSnapshotMinSlice);
    if (zero_copy) {
        void *dev = nullptr;
        e = hipHostGetDevicePointer(&dev, image, 0);
        if (e != hipSuccess) return fail_hip(e, "hipHostGetDevicePointer");
        if (m->done_recorded && (e = hipStreamWaitEvent(s, m->ev_done, 0)) != hipSuccess)
            return fail_hip(e, "ring order");
        return run_direct(m, op, (uint8_t *)dev, h, s);
    }
    return run_ring(m, op, h, (uint8_t *)image, s);
}

}  // namespace

using gms::check_common;
using gms::check_device_range;
using gms::check_outputs;
using gms::free_ring;
using gms::make_hash;

extern "C" {

int gms_abi_version(void) { return 5; }

const char *gms_status_str(int status)
{
    switch (status) {
    case GMS_OK: return "ok";
    case GMS_ERR_INVALID: return "invalid argument";
    case GMS_ERR_OVERLAP: return "overlapping entries";
    case GMS_ERR_SIZE: return "buffer too small";
    case GMS_ERR_HIP: return "HIP runtime error";
    case GMS_ERR_NOMEM: return "out of memory";
    case GMS_ERR_STATE: return "operation not valid for this manifest";
    case GMS_ERR_IO: return "file I/O error";
    case GMS_ERR_INTEGRITY: return "contents differ from their recorded hashes";
    default: return "unknown status";
    }
}

const char *gms_last_error(void) { return g_last_error.c_str(); }

int gms_manifest_create(const gms_entry *entries, uint64_t n, int device, uint64_t chunk_bytes,
                        gms_manifest **out)
{
    gms::clear_error();
    return gms::manifest_create(entries, n, device, chunk_bytes, true, out);
}

}  // extern "C"

int gms::manifest_create(const gms_entry *entries, uint64_t n, int device, uint64_t chunk_bytes, bool check_ranges,
                         gms_manifest **out)
{
    if (!out) return fail(GMS_ERR_INVALID, "out is null");
    *out = nullptr;
    if (n && !entries) return fail(GMS_ERR_INVALID, "entries is null");
    if (n >= (1ull << 32)) return fail(GMS_ERR_INVALID, "too many entries (%llu)", (unsigned long long)n);
    if (chunk_bytes == 0) chunk_bytes = GMS_DEFAULT_CHUNK_BYTES;
    if (chunk_bytes % GMS_BLOCK_BYTES || chunk_bytes > kMaxChunk)
        return fail(GMS_ERR_INVALID, "chunk_bytes %llu is not a multiple of 4096 in [4096, 64 MiB]",
                    (unsigned long long)chunk_bytes);
    if (device < GMS_HOST_ONLY) return fail(GMS_ERR_INVALID, "device %d", device);

    // ranges: non-null, no address overflow, pairwise disjoint
    std::vector<uint64_t> order;
    order.reserve(n);
    for (uint64_t i = 0; i < n; ++i) {
        const gms_entry &e = entries[i];
        if (!e.nbytes) continue;
        if (!e.addr) return fail(GMS_ERR_INVALID, "entry %llu: null address", (unsigned long long)i);
        if (e.addr + e.nbytes < e.addr) return fail(GMS_ERR_INVALID, "entry %llu: range wraps", (unsigned long long)i);
        order.push_back(i);
    }
    std::sort(order.begin(), order.end(), [&](uint64_t a, uint64_t b) { return entries[a].addr < entries[b].addr; });
    for (size_t k = 1; k < order.size(); ++k) {
        const gms_entry &p = entries[order[k - 1]], &q = entries[order[k]];
        if (q.addr < p.addr + p.nbytes)
            return fail(GMS_ERR_OVERLAP, "entries %llu and %llu overlap", (unsigned long long)order[k - 1],
                        (unsigned long long)order[k]);
    }

    if (device >= 0) {
        int count = 0;
        hipError_t e = hipGetDeviceCount(&count);
        if (e != hipSuccess) return fail_hip(e, "hipGetDeviceCount");
        if (device >= count) return fail(GMS_ERR_INVALID, "device %d of %d", device, count);
        // every range inside one allocation of `device` (walk in address order,
        // reusing the previous allocation's bounds)
        uint64_t cur_lo = 0, cur_hi = 0;
        for (uint64_t i : order) {
            if (!check_ranges) break;
            const gms_entry &r = entries[i];
            if (r.addr >= cur_lo && r.addr + r.nbytes <= cur_hi) continue;
            char what[48];
            snprintf(what, sizeof what, "entry %llu", (unsigned long long)i);
            int rc = check_device_range((const void *)(uintptr_t)r.addr, r.nbytes, device, what);
            if (rc != GMS_OK) return rc;
            hipDeviceptr_t base = nullptr;
            size_t size = 0;
            (void)hipMemGetAddressRange(&base, &size, (hipDeviceptr_t)(uintptr_t)r.addr);
            cur_lo = (uint64_t)(uintptr_t)base;
            cur_hi = cur_lo + size;
        }
    }

    gms_manifest *m = new (std::nothrow) gms_manifest;
    if (!m) return fail(GMS_ERR_NOMEM, "manifest");
    try {
        m->device = device;
        m->n = n;
        m->chunk_bytes = chunk_bytes;
        m->img_off.resize(n);
        uint64_t most = 0;  // an entry splits into at most nbytes / chunk_bytes + 2 chunks
        for (uint64_t i = 0; i < n; ++i) most += entries[i].nbytes ? entries[i].nbytes / chunk_bytes + 2 : 0;
        m->chunks.reserve(most);
        uint64_t off = 0;
        for (uint64_t i = 0; i < n; ++i) {
            const uint64_t nb = entries[i].nbytes;
            m->img_off[i] = off;
            m->payload += nb;
            uint64_t pos = 0;
            while (pos < nb) {
                const uint64_t img = off + pos;
                const uint64_t lim = (img / chunk_bytes + 1) * chunk_bytes;
                const uint64_t len = std::min(nb - pos, lim - img);
                Chunk c;
                c.addr = entries[i].addr + pos;
                c.img = img;
                c.off = pos;
                c.len = (uint32_t)len;
                c.entry = (uint32_t)i;
                m->chunks.push_back(c);
                pos += len;
            }
            off += ceil_div(nb, GMS_BLOCK_BYTES) * GMS_BLOCK_BYTES;
        }
        m->image_bytes = off;
        m->num_blocks = off / GMS_BLOCK_BYTES;
        gms::plan_launch_groups(m);
    } catch (const std::bad_alloc &) {
        delete m;
        return fail(GMS_ERR_NOMEM, "manifest tables");
    }

    if (device >= 0 && !m->chunks.empty()) {
        DeviceGuard g(device);
        if (g.err != hipSuccess) {
            delete m;
            return fail_hip(g.err, "hipSetDevice");
        }
        const size_t bytes = m->chunks.size() * sizeof(Chunk);
        hipError_t e = hipMalloc((void **)&m->d_chunks, bytes);
        if (e != hipSuccess) {
            (void)hipGetLastError();
            m->d_chunks = nullptr;
            delete m;
            return fail(GMS_ERR_NOMEM, "work list: hipMalloc(%zu): %s", bytes, hipGetErrorString(e));
        }
        e = hipMemcpy(m->d_chunks, m->chunks.data(), bytes, hipMemcpyHostToDevice);
        if (e != hipSuccess) {
            (void)hipFree(m->d_chunks);
            delete m;
            return fail_hip(e, "work list upload");
        }
    }
    *out = m;
    return GMS_OK;
}

extern "C" {

void gms_manifest_destroy(gms_manifest *m)
{
    if (!m) return;
    if (m->device >= 0) {
        DeviceGuard g(m->device);
        free_ring(m);
        if (m->d_chunks) (void)hipFree(m->d_chunks);
    }
    delete m;
}

uint64_t gms_num_entries(const gms_manifest *m) { return m ? m->n : 0; }
uint64_t gms_payload_bytes(const gms_manifest *m) { return m ? m->payload : 0; }
uint64_t gms_image_bytes(const gms_manifest *m) { return m ? m->image_bytes : 0; }
uint64_t gms_num_blocks(const gms_manifest *m) { return m ? m->num_blocks : 0; }
uint64_t gms_num_chunks(const gms_manifest *m) { return m ? (uint64_t)m->chunks.size() : 0; }
uint64_t gms_num_launch_groups(const gms_manifest *m) { return m ? (uint64_t)m->groups.size() : 0; }

int gms_launch_group(const gms_manifest *m, uint64_t g, uint64_t *chunks_out, uint32_t *unit_shift_out,
                     uint32_t *flags_out)
{
    gms::clear_error();
    if (!m || g >= m->groups.size())
        return fail(GMS_ERR_INVALID, "launch group %llu of %llu", (unsigned long long)g,
                    (unsigned long long)(m ? m->groups.size() : 0));
    const gms::LaunchGroup &lg = m->groups[g];
    if (chunks_out) *chunks_out = lg.count;
    if (unit_shift_out) *unit_shift_out = lg.shift;
    if (flags_out) *flags_out = (lg.shifted ? GMS_GROUP_SHIFTED : 0u) | (lg.striped ? GMS_GROUP_STRIPED : 0u);
    return GMS_OK;
}
int gms_manifest_device(const gms_manifest *m) { return m ? m->device : GMS_HOST_ONLY; }

int gms_layout(const gms_manifest *m, uint64_t *img_off, uint64_t *blk_base)
{
    if (!m) return fail(GMS_ERR_INVALID, "manifest is null");
    for (uint64_t i = 0; i < m->n; ++i) {
        if (img_off) img_off[i] = m->img_off[i];
        if (blk_base) blk_base[i] = m->img_off[i] / GMS_BLOCK_BYTES;
    }
    return GMS_OK;
}

int gms_manifest_set_staging(gms_manifest *m, uint64_t slice_bytes, uint32_t slots)
{
    if (!m) return fail(GMS_ERR_INVALID, "manifest is null");
    if (m->device < 0) return fail(GMS_ERR_STATE, "host-only manifest has no device");
    if (slots > kMaxSlots) return fail(GMS_ERR_INVALID, "slots %u > %u", slots, kMaxSlots);
    if (slice_bytes && (slice_bytes < GMS_BLOCK_BYTES || slice_bytes > kMaxSlice))
        return fail(GMS_ERR_INVALID, "slice_bytes %llu is outside [4096, 64 GiB]", (unsigned long long)slice_bytes);
    std::lock_guard<std::mutex> lock(m->ring_mu);
    DeviceGuard g(m->device);
    free_ring(m);
    m->slice_bytes = slice_bytes ? slice_bytes : kDefaultSlice;
    m->slots = slots;
    return GMS_OK;
}

int gms_snapshot(const gms_manifest *m, void *image, uint64_t image_bytes, int image_kind, uint64_t *blk_hash_out,
                 uint64_t *ten_hash_out, void *stream)
{
    gms::clear_error();
    int rc = check_common(m, image, image_bytes, image_kind, true);
    if (rc != GMS_OK) return rc;
    HashOut h = make_hash(nullptr, blk_hash_out, ten_hash_out, nullptr, nullptr, 0);
    if ((rc = check_outputs(m, h)) != GMS_OK) return rc;
    return run_op(m, gms::kSnapshot, image, image_kind, h, stream);
}

int gms_restore(const gms_manifest *m, const void *image, uint64_t image_bytes, int image_kind,
                const uint64_t *expected_blk, uint64_t *blk_hash_out, uint64_t *ten_hash_out,
                uint64_t *mismatch_count_out, uint64_t *mismatch_list_out, uint64_t mismatch_cap, void *stream)
{
    gms::clear_error();
    int rc = check_common(m, image, image_bytes, image_kind, true);
    if (rc != GMS_OK) return rc;
    HashOut h = make_hash(expected_blk, blk_hash_out, ten_hash_out, mismatch_count_out, mismatch_list_out,
                          mismatch_cap);
    if ((rc = check_outputs(m, h)) != GMS_OK) return rc;
    return run_op(m, gms::kRestore, const_cast<void *>(image), image_kind, h, stream);
}

int gms_verify(const gms_manifest *m, const uint64_t *expected_blk, uint64_t *blk_hash_out, uint64_t *ten_hash_out,
               uint64_t *mismatch_count_out, uint64_t *mismatch_list_out, uint64_t mismatch_cap, void *stream)
{
    gms::clear_error();
    int rc = check_common(m, nullptr, 0, GMS_MEM_DEVICE, false);
    if (rc != GMS_OK) return rc;
    HashOut h = make_hash(expected_blk, blk_hash_out, ten_hash_out, mismatch_count_out, mismatch_list_out,
                          mismatch_cap);
    if (!h.any()) return fail(GMS_ERR_INVALID, "verify needs blk_hash_out, ten_hash_out or expected_blk");
    if ((rc = check_outputs(m, h)) != GMS_OK) return rc;
    return run_op(m, gms::kVerify, nullptr, GMS_MEM_DEVICE, h, stream);
}

}  // extern "C"
