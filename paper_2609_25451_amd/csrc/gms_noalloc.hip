// Restore from a pinned host image without allocating: gms_restore_pinned_noalloc.
//
// gms_restore moves a pinned image through a staging ring that it allocates on
// first use (device slots, a copy stream and events).  Callers that cannot
// allocate device memory (code under graph capture, tight serving loops,
// harnesses that forbid it) get this variant instead: the staging area is a
// fixed device array of this file, and every step runs on the caller's stream.
// Each slice of the image is copied into the array by the host-copy kernel and
// then scattered (hashed, compared) by the same kernels as gms_restore, one
// after the other, so no event and no second stream is needed.

#include <algorithm>
#include <mutex>

#include "gms_host.h"

// The staging area, one per device, held until the process ends.  In host code
// its name is only a stand-in for the device symbol: kernels and copies use the
// per-device address that hipGetSymbolAddress returns.
static __device__ __align__(256) uint8_t scratch[GMS_NOALLOC_STAGING_BYTES];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
uint8_t *g_scratch[kMaxDevices] = {};

// The device address of `scratch` on `device` (current when called), looked up
// once per device.
int scratch_on(int device, uint8_t **out)
{
    if (device < 0 || device >= kMaxDevices) return gms::fail(GMS_ERR_INVALID, "device %d out of range", device);
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch[device]) {
        void *p = nullptr;
        hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return gms::fail_hip(e, "hipGetSymbolAddress(staging area)");
        g_scratch[device] = (uint8_t *)p;
    }
    *out = g_scratch[device];
    return GMS_OK;
}

// First chunk of launch group `g` whose image offset is at or past `pos` (chunks
// of a group are in image order).
uint64_t first_at(const gms_manifest *m, const gms::LaunchGroup &g, uint64_t pos)
{
    const gms::Chunk *lo = m->chunks.data() + g.first, *hi = lo + g.count;
    return (uint64_t)(std::lower_bound(lo, hi, pos, [](const gms::Chunk &c, uint64_t p) { return c.img < p; }) -
                      m->chunks.data());
}

}  // namespace

extern "C" int gms_restore_pinned_noalloc(const gms_manifest *m, const void *image, uint64_t image_bytes,
                                          uint64_t staging_bytes, const uint64_t *expected_blk,
                                          uint64_t *blk_hash_out, uint64_t *ten_hash_out,
                                          uint64_t *mismatch_count_out, uint64_t *mismatch_list_out,
                                          uint64_t mismatch_cap, void *stream)
{
    gms::clear_error();
    int rc = gms::check_common(m, image, image_bytes, GMS_MEM_HOST_PINNED, true);
    if (rc != GMS_OK) return rc;
    if (staging_bytes > GMS_NOALLOC_STAGING_BYTES)
        return gms::fail(GMS_ERR_SIZE, "staging_bytes %llu exceeds the fixed staging area of %llu bytes",
                         (unsigned long long)staging_bytes, (unsigned long long)GMS_NOALLOC_STAGING_BYTES);
    const uint64_t want = staging_bytes ? staging_bytes : GMS_NOALLOC_STAGING_BYTES;
    const uint64_t slice = want / m->chunk_bytes * m->chunk_bytes;  // whole chunks: none straddles a slice
    if (slice == 0)
        return gms::fail(GMS_ERR_SIZE, "staging of %llu bytes holds no chunk of the manifest (%llu bytes)",
                         (unsigned long long)want, (unsigned long long)m->chunk_bytes);
    gms::HashOut h = gms::make_hash(expected_blk, blk_hash_out, ten_hash_out, mismatch_count_out, mismatch_list_out,
                                    mismatch_cap);
    if ((rc = gms::check_outputs(m, h)) != GMS_OK) return rc;

    gms::DeviceGuard g(m->device);
    if (g.err != hipSuccess) return gms::fail_hip(g.err, "hipSetDevice");
    uint8_t *stage = nullptr;
    if ((rc = scratch_on(m->device, &stage)) != GMS_OK) return rc;
    hipStream_t s = (hipStream_t)stream;
    hipError_t e;
    gms_manifest *mm = const_cast<gms_manifest *>(m);
    std::lock_guard<std::mutex> lock(mm->ring_mu);
    // after any earlier staging-ring call on this manifest; a graph cannot wait on
    // that call's event, so a capturing stream is refused once there was one
    if (m->done_recorded) {
        hipStreamCaptureStatus cap = hipStreamCaptureStatusNone;
        if ((e = hipStreamIsCapturing(s, &cap)) != hipSuccess) return gms::fail_hip(e, "hipStreamIsCapturing");
        if (cap != hipStreamCaptureStatusNone)
            return gms::fail(GMS_ERR_STATE, "capturing after a staging-ring call on this manifest");
        if ((e = hipStreamWaitEvent(s, m->ev_done, 0)) != hipSuccess) return gms::fail_hip(e, "ring order");
    }
    if ((e = gms::launch_prologue(h, m->n, s)) != hipSuccess) return gms::fail_hip(e, "prologue launch");
    if (m->chunks.empty()) return GMS_OK;
    uint8_t *host_dev = nullptr;  // the pinned image as the copy kernel sees it
    if ((e = hipHostGetDevicePointer((void **)&host_dev, const_cast<void *>(image), 0)) != hipSuccess)
        return gms::fail_hip(e, "hipHostGetDevicePointer");
    const uint64_t nslices = gms::ceil_div(m->image_bytes, slice);
    for (uint64_t sl = 0; sl < nslices; ++sl) {
        const uint64_t lo = sl * slice, bytes = std::min(slice, m->image_bytes - lo);
        if ((e = gms::launch_host_copy(host_dev + lo, stage, bytes, s)) != hipSuccess)
            return gms::fail_hip(e, "staging copy launch");
        for (const gms::LaunchGroup &lg : m->groups) {
            const uint64_t c0 = first_at(m, lg, lo), c1 = first_at(m, lg, lo + slice);
            if ((e = gms::launch_stream(gms::kRestore, h.any(), lg.shifted, lg.striped, m->d_chunks, c0, c1 - c0,
                                        lg.shift, stage, lo, h, s)) != hipSuccess)
                return gms::fail_hip(e, "kernel launch");
        }
    }
    return GMS_OK;
}
