// Host-side internals shared by the C-ABI implementation files (gms_api.hip,
// gms_hostio.hip, gms_pool.hip, gms_store.hip): the manifest object, error reporting and the helpers that
// validate arguments and drive the staging rings.  Not installed.
#pragma once

#include <cstdint>
#include <mutex>
#include <string>
#include <vector>

#include "gms.h"
#include "gms_internal.h"

namespace gms {

constexpr uint64_t kMaxChunk = 64ull << 20;
constexpr uint64_t kDefaultSlice = GMS_DEFAULT_SLICE_BYTES;
constexpr uint32_t kDefaultSlots = GMS_DEFAULT_SLOTS;
constexpr uint32_t kMaxSlots = 16;
constexpr uint64_t kMaxSlice = 64ull << 30;
// Slices below this size make a snapshot's device-to-host copies erratic (half the
// link and less with 64 MiB pieces); from 128 MiB up it holds about 99% of the
// link, ahead of zero-copy stores from the gather kernel (about 96%).
constexpr uint64_t kRingSnapshotMinSlice = 128ull << 20;

inline uint64_t ceil_div(uint64_t a, uint64_t b) { return a / b + (a % b != 0); }

// Records a message for gms_last_error() and returns `status`.
int fail(int status, const char *fmt, ...) __attribute__((format(printf, 2, 3)));
int fail_hip(hipError_t e, const char *what);
void clear_error();

// Makes `device` current for the lifetime of the guard, restoring the
// caller's current device afterwards.
struct DeviceGuard {
    int prev = -1;
    hipError_t err = hipSuccess;
    explicit DeviceGuard(int device)
    {
        err = hipGetDevice(&prev);
        if (err == hipSuccess && prev != device) err = hipSetDevice(device);
    }
    ~DeviceGuard()
    {
        int cur = -1;
        if (prev >= 0 && hipGetDevice(&cur) == hipSuccess && cur != prev) (void)hipSetDevice(prev);
    }
};

}  // namespace gms

namespace gms {
// Chunks launched together: chunks[first, first + count), each needing at most
// 2^shift work units; `shifted` when their entry addresses are not 16-byte
// aligned (all of them), clear when all are.
struct LaunchGroup {
    uint64_t first = 0, count = 0;
    uint32_t shift = 0;
    bool shifted = false;
    bool striped = false;  // restore and snapshot in the striped unit order (chunks of mostly separate entries)
};
}  // namespace gms

struct gms_manifest {
    int device = GMS_HOST_ONLY;
    uint64_t n = 0;
    uint64_t chunk_bytes = 0;
    uint64_t payload = 0, image_bytes = 0, num_blocks = 0;
    std::vector<uint64_t> img_off;
    std::vector<gms::Chunk> chunks;  // host copy: by launch group, then by image offset
    std::vector<gms::LaunchGroup> groups;
    gms::Chunk *d_chunks = nullptr;

    // staging rings, created lazily: device slots for pinned-host images, and
    // pinned host slots for image files.  ring_mu serialises their users.
    std::mutex ring_mu;
    uint64_t slice_bytes = gms::kDefaultSlice;
    uint32_t slots = gms::kDefaultSlots;
    uint8_t *d_ring = nullptr;
    uint64_t ring_slice = 0;
    uint32_t ring_slots = 0;
    uint8_t *h_ring = nullptr;  // pinned host slots (file paths only), host_slots x ring_slice
    uint32_t host_slots = 0;    // twice the device slots (capped), so reads run ahead of the link copies
    hipStream_t copy_stream = nullptr;
    hipEvent_t ev_filled[gms::kMaxSlots] = {};
    hipEvent_t ev_free[gms::kMaxSlots] = {};
    hipEvent_t ev_host[gms::kMaxSlots] = {};  // link copy that last touched a host slot finished
    hipEvent_t ev_entry = nullptr;
    hipEvent_t ev_done = nullptr;
    bool done_recorded = false;
    // per launch group g and ring slice s, the first chunk of g at or after the
    // slice's start, at [g * (nslices + 1) + s]; s = nslices gives the group's end
    std::vector<uint64_t> slice_first;
};

namespace gms {

// Ends a ring call: joins the caller's stream and the copy stream and records
// ev_done after both, so the next ring call on the manifest, from any stream,
// waits until this one no longer uses a slot.  Once armed, a call that fails
// half-way still fences what it had enqueued (best effort, in the destructor).
struct RingFence {
    gms_manifest *m;
    hipStream_t s;
    bool armed = false;
    RingFence(gms_manifest *m_, hipStream_t s_) : m(m_), s(s_) {}
    // success path: the call's work then completes on `s`
    hipError_t close()
    {
        armed = false;
        hipError_t e;
        if ((e = hipEventRecord(m->ev_entry, s)) != hipSuccess) return e;
        if ((e = hipStreamWaitEvent(m->copy_stream, m->ev_entry, 0)) != hipSuccess) return e;
        if ((e = hipEventRecord(m->ev_done, m->copy_stream)) != hipSuccess) return e;
        m->done_recorded = true;
        return hipStreamWaitEvent(s, m->ev_done, 0);
    }
    ~RingFence()
    {
        if (armed && close() != hipSuccess) (void)hipGetLastError();
    }
    RingFence(const RingFence &) = delete;
    RingFence &operator=(const RingFence &) = delete;
};

// pool internals used by the model-state store
int pool_reset(gms_pool *p);
int pool_set_access_all(gms_pool *p, bool read_only);
bool pool_holds(gms_pool *p, uint64_t addr, uint64_t bytes);
int pool_device(const gms_pool *p);

// gms_manifest_create; with check_ranges false the ranges are not checked
// against the runtime's allocations (for mappings the runtime does not report
// whole, such as imported external memory, which the caller has checked).
int manifest_create(const gms_entry *entries, uint64_t n, int device, uint64_t chunk_bytes, bool check_ranges,
                    gms_manifest **out);
void free_ring(gms_manifest *m);
int ensure_ring(gms_manifest *m);       // device slots, copy stream, events, slice table
int ensure_host_ring(gms_manifest *m);  // plus pinned host slots
int check_common(const gms_manifest *m, const void *image, uint64_t image_bytes, int kind, bool need_image);
int check_outputs(const gms_manifest *m, const HashOut &h);
// `op` over every chunk (one launch per group), image byte x at img_base + x.
hipError_t launch_all(const gms_manifest *m, int op, const HashOut &h, uint8_t *img_base, hipStream_t s);
// `op` over the chunks of ring slice `sl`, image byte x at slot + (x - sl * ring_slice).
hipError_t launch_slice(const gms_manifest *m, int op, const HashOut &h, uint64_t sl, uint8_t *slot, hipStream_t s);
// GMS_ERR_STATE if `s` is capturing a graph: for calls that synchronize or
// order themselves with library-owned streams and events.
int refuse_capture(hipStream_t s, const char *what);
HashOut make_hash(const uint64_t *expected, uint64_t *blk, uint64_t *ten, uint64_t *cnt, uint64_t *list,
                  uint64_t cap);

}  // namespace gms
