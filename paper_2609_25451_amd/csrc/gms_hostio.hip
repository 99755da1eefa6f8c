// Host-side images: the packed image in a file, or in ordinary (pageable) host
// memory.
//
// A cold replacement repopulates model state from storage while the engine's
// runtime is restored (paper section 3.3 and section 4, cold GMS repopulation);
// a process snapshot stages device state in the host memory of the
// checkpointed process and reinstates it on restore, a copy that the paper's
// checkpoint tool performs serially without saturating PCIe (section 3.1,
// section 5.2).  Either way the end-to-end cost is the artifact size over the
// effective bandwidth (section 3.1).
//
// Restore runs a three-stage pipeline per staging slice: parallel workers move
// the slice's pieces into a pinned host slot (pread, through per-worker
// bounce buffers with O_DIRECT, or memcpy from a memory image), a copy kernel
// moves that slot into a device slot on the manifest's copy stream, and the
// scatter(+hash) kernel runs on the caller's stream.  One pool of workers
// takes pieces in image order from a shared counter, so every worker keeps a
// large request in flight and none waits for a slower slice; a host slot is
// refilled once the copy that read it has finished, so the source, the host
// link and HBM all stay busy.  Snapshot runs the mirror image: the gather
// kernel fills a slice (into a device slot that hipMemcpyAsync then copies to the host
// slot, or straight into the host slot zero-copy when slices are small) and
// the workers write its pieces out.

#include <fcntl.h>
#include <sys/stat.h>
#include <unistd.h>

#include <algorithm>
#include <atomic>
#include <cerrno>
#include <condition_variable>
#include <cstdint>
#include <cstdlib>
#include <cstring>
#include <mutex>
#include <thread>
#include <vector>

#include "gms_host.h"

using gms::ceil_div;
using gms::DeviceGuard;
using gms::fail;
using gms::fail_hip;
using gms::HashOut;

namespace {

constexpr unsigned kDefaultIoThreads = 16;
constexpr unsigned kMaxIoThreads = 64;
constexpr uint64_t kDirectAlign = 4096;
// One pread/pwrite/memcpy.  Direct I/O loses storage bandwidth below 16 MiB
// per request; buffered reads go through the page cache's readahead and copy,
// which run best at 64 MiB per request (at most one slice).
constexpr uint64_t kDirectPieceBytes = 16ull << 20;
constexpr uint64_t kBufferedPieceBytes = 64ull << 20;
constexpr uint64_t kMemoryPieceBytes = 16ull << 20;

struct FileHandle {
    int fd = -1;
    bool direct = false;
    ~FileHandle()
    {
        if (fd >= 0) close(fd);
    }
};

// The host side of a transfer: a file at `file_offset` (image byte 0), or a
// memory image when `mem` is set.
struct HostImage {
    int fd = -1;
    const char *path = nullptr;
    bool direct = false;
    uint64_t file_offset = 0;
    uint8_t *mem = nullptr;
    const char *name() const { return mem ? "the host image" : path; }
};

// Moves `len` bytes between the host slot `slot` and image offset `lo`.
// Direct I/O cannot target the pinned slots (the kernel refuses to pin
// driver-mapped pages: EFAULT), so with O_DIRECT the bytes go through the
// worker's page-aligned bounce buffer.  Returns 0 or an errno value (EIO for
// a file that ends early).
int transfer_piece(const HostImage &img, int fd, uint8_t *bounce, uint8_t *slot, uint64_t len, uint64_t lo,
                   bool write)
{
    if (img.mem) {
        if (write)
            memcpy(img.mem + lo, slot, len);
        else
            memcpy(slot, img.mem + lo, len);
        return 0;
    }
    uint8_t *buf = bounce ? bounce : slot;
    if (write && bounce) memcpy(bounce, slot, len);
    const uint64_t off = img.file_offset + lo;
    uint64_t done = 0;
    while (done < len) {
        ssize_t r = write ? pwrite(fd, buf + done, len - done, (off_t)(off + done))
                          : pread(fd, buf + done, len - done, (off_t)(off + done));
        if (r < 0) {
            if (errno == EINTR) continue;
            return errno;
        }
        if (r == 0) return EIO;
        done += (uint64_t)r;
    }
    if (!write && bounce) memcpy(slot, bounce, len);
    return 0;
}

// The image cut into slices (one host slot each) and each slice into pieces of
// at most `piece` bytes, numbered in image order.  `enqueued` counts the slices
// whose device-side step the caller's thread has enqueued; `left[s]` counts
// the pieces of slice s not yet transferred.  The first error stops every
// worker.
struct PiecePool {
    uint64_t slice = 0, image_bytes = 0, piece = 0, per_slice = 0, nslices = 0, npieces = 0;
    std::atomic<uint64_t> next{0};
    std::mutex mu;
    std::condition_variable cv;
    std::vector<uint32_t> left;
    uint64_t enqueued = 0;
    int err = 0;        // errno of the first failed transfer
    bool hip_err = false;
    bool stop = false;

    PiecePool(uint64_t slice_, uint64_t image_bytes_, uint64_t piece_)
        : slice(slice_), image_bytes(image_bytes_), piece(std::min(piece_, slice_))
    {
        per_slice = ceil_div(slice, piece);
        nslices = ceil_div(image_bytes, slice);
        npieces = nslices * per_slice;
        left.resize(nslices);
        for (uint64_t s = 0; s < nslices; ++s)
            left[s] = (uint32_t)ceil_div(std::min(slice, image_bytes - s * slice), piece);
    }
    // image range of piece p; empty for the padding pieces of a short last slice
    void range(uint64_t p, uint64_t &s, uint64_t &lo, uint64_t &bytes) const
    {
        s = p / per_slice;
        lo = s * slice + (p % per_slice) * piece;
        const uint64_t end = std::min((s + 1) * slice, image_bytes);
        bytes = lo < end ? std::min(piece, end - lo) : 0;
    }
    void fail_stop(int e, bool hip)
    {
        std::lock_guard<std::mutex> l(mu);
        if (!err && !hip_err) {
            err = e;
            hip_err = hip;
        }
        stop = true;
        cv.notify_all();
    }
    // blocks until `enqueued > s`; false once the pool has stopped
    bool wait_enqueued(uint64_t s)
    {
        std::unique_lock<std::mutex> l(mu);
        cv.wait(l, [&] { return stop || enqueued > s; });
        return !stop;
    }
    void set_enqueued(uint64_t n)
    {
        std::lock_guard<std::mutex> l(mu);
        enqueued = n;
        cv.notify_all();
    }
    void piece_done(uint64_t s)
    {
        std::lock_guard<std::mutex> l(mu);
        if (--left[s] == 0) cv.notify_all();
    }
    // blocks until every piece of slice s is done; false once the pool has stopped
    bool wait_slice(uint64_t s)
    {
        std::unique_lock<std::mutex> l(mu);
        cv.wait(l, [&] { return stop || left[s] == 0; });
        return !stop;
    }
};

// Runs `threads` workers over the pool.  A worker takes piece p of slice s in
// host slot s % hslots; to fill the slot (restore) it first waits until the
// copy out of that slot for slice s - hslots has been enqueued and has
// finished; to drain it (snapshot) it waits until slice s has been enqueued
// and has landed in the slot.
class Workers {
public:
    Workers(PiecePool &pool, const HostImage &img, bool write, uint8_t *h_ring, uint32_t hslots,
            const hipEvent_t *ev_host, unsigned threads)
    {
        for (unsigned t = 0; t < threads; ++t) {
            try {
                pool_.emplace_back([=, &pool] { run(pool, img, write, h_ring, hslots, ev_host); });
            } catch (...) {  // no thread: stop the pool rather than wait for work nobody does
                pool.fail_stop(EAGAIN, false);
                break;
            }
        }
    }
    ~Workers() { join(); }
    void join()
    {
        for (auto &t : pool_)
            if (t.joinable()) t.join();
    }

private:
    static void run(PiecePool &pool, HostImage img, bool write, uint8_t *h_ring, uint32_t hslots,
                    const hipEvent_t *ev_host)
    {
        uint8_t *bounce = nullptr;
        if (img.direct && posix_memalign((void **)&bounce, kDirectAlign, pool.piece) != 0) {
            pool.fail_stop(ENOMEM, false);
            return;
        }
        // Buffered file reads: the kernel keeps readahead state per open file,
        // and workers taking interleaved pieces through one descriptor defeat
        // it, so each worker reads through a descriptor of its own (the shared
        // one if the file cannot be opened again).
        const int own = (!img.mem && !write && !img.direct && img.path) ? open(img.path, O_RDONLY | O_CLOEXEC) : -1;
        for (;;) {
            const uint64_t p = pool.next.fetch_add(1, std::memory_order_relaxed);
            if (p >= pool.npieces) break;
            uint64_t s, lo, bytes;
            pool.range(p, s, lo, bytes);
            if (bytes == 0) continue;
            const uint32_t slot = (uint32_t)(s % hslots);
            if (write || s >= hslots) {
                if (!pool.wait_enqueued(write ? s : s - hslots)) break;
                if (hipEventSynchronize(ev_host[slot]) != hipSuccess) {
                    pool.fail_stop(0, true);
                    break;
                }
            }
            uint8_t *host = h_ring + (uint64_t)slot * pool.slice + (lo - s * pool.slice);
            const int e = transfer_piece(img, own >= 0 ? own : img.fd, bounce, host, bytes, lo, write);
            if (e) {
                pool.fail_stop(e, false);
                break;
            }
            pool.piece_done(s);
        }
        if (own >= 0) close(own);
        free(bounce);
    }
    std::vector<std::thread> pool_;
};

int open_file(FileHandle &f, const char *path, bool write, bool want_direct, uint64_t offset)
{
    const bool direct = want_direct && offset % kDirectAlign == 0;
    int flags = write ? (O_WRONLY | O_CREAT | O_TRUNC) : O_RDONLY;
    f.fd = open(path, flags | (direct ? O_DIRECT : 0) | O_CLOEXEC, 0644);
    f.direct = direct && f.fd >= 0;
    if (f.fd < 0 && direct && errno == EINVAL) {  // file system without O_DIRECT: buffered I/O
        f.fd = open(path, flags | O_CLOEXEC, 0644);
        f.direct = false;
    }
    if (f.fd < 0) return fail(GMS_ERR_IO, "open(%s): %s", path, strerror(errno));
    return GMS_OK;
}

int check_manifest(const gms_manifest *m, unsigned threads)
{
    if (!m) return fail(GMS_ERR_INVALID, "manifest is null");
    if (m->device < 0) return fail(GMS_ERR_STATE, "host-only manifest has no device");
    if (threads > kMaxIoThreads) return fail(GMS_ERR_INVALID, "io_threads %u > %u", threads, kMaxIoThreads);
    return GMS_OK;
}

// A memory image: non-null when the layout has bytes, at least as long as the
// layout, and not device memory (which host threads cannot copy).
int check_memory_image(const gms_manifest *m, const void *image, uint64_t image_bytes)
{
    if (image_bytes < m->image_bytes)
        return fail(GMS_ERR_SIZE, "image has %llu bytes, layout needs %llu", (unsigned long long)image_bytes,
                    (unsigned long long)m->image_bytes);
    if (m->image_bytes == 0) return GMS_OK;
    if (!image) return fail(GMS_ERR_INVALID, "image is null");
    if ((uint64_t)(uintptr_t)image + m->image_bytes < (uint64_t)(uintptr_t)image)
        return fail(GMS_ERR_INVALID, "image range wraps");
    hipPointerAttribute_t attr;
    if (hipPointerGetAttributes(&attr, image) == hipSuccess && attr.type == hipMemoryTypeDevice)
        return fail(GMS_ERR_INVALID, "image %p is device memory; gms_snapshot / gms_restore take device images", image);
    (void)hipGetLastError();  // pageable memory is unknown to HIP
    return GMS_OK;
}

// Waits until every earlier ring call of this manifest has finished on the
// device, so that its host and device slots are free.
int drain_ring(gms_manifest *m)
{
    hipError_t e;
    if (m->copy_stream && (e = hipStreamSynchronize(m->copy_stream)) != hipSuccess) return fail_hip(e, "copy stream");
    if (m->done_recorded && (e = hipEventSynchronize(m->ev_done)) != hipSuccess) return fail_hip(e, "ring drain");
    return GMS_OK;
}

// Stops and joins the workers, then reports the pool's first error (or `rc`).
int finish(PiecePool &pool, Workers &w, int rc, const HostImage &img, bool write)
{
    if (rc != GMS_OK) pool.fail_stop(0, false);
    w.join();
    if (rc != GMS_OK) return rc;
    if (pool.hip_err) return fail(GMS_ERR_HIP, "waiting for a staging slot of %s", img.name());
    if (pool.err) return fail(GMS_ERR_IO, "%s %s: %s", write ? "writing" : "reading", img.name(), strerror(pool.err));
    return GMS_OK;
}

#define GMS_TRY(call)                                              \
    do {                                                           \
        hipError_t e_ = (call);                                    \
        if (e_ != hipSuccess) return fail_hip(e_, #call);          \
    } while (0)

// Device set-up common to both directions; *done is set when nothing is left
// to move (an empty layout).
int begin(gms_manifest *m, const HashOut &h, hipStream_t s, const char *what, bool *done)
{
    int rc = gms::refuse_capture(s, what);
    if (rc != GMS_OK) return rc;
    GMS_TRY(gms::launch_prologue(h, m->n, s));
    *done = m->chunks.empty();
    return GMS_OK;
}

// Restore from a host image through the pinned host ring, the device ring and
// the scatter kernel.  The caller holds the device guard.
int restore_pipeline(gms_manifest *m, const HostImage &src, const HashOut &h, unsigned threads, uint64_t piece,
                     hipStream_t s)
{
    std::lock_guard<std::mutex> lock(m->ring_mu);
    int rc;
    if ((rc = gms::ensure_host_ring(m)) != GMS_OK) return rc;
    if ((rc = drain_ring(m)) != GMS_OK) return rc;
    const uint64_t slice = m->ring_slice;
    const uint32_t k = m->ring_slots, hk = m->host_slots;
    uint8_t *h_dev = nullptr;  // the pinned host ring as the copy kernel sees it
    GMS_TRY(hipHostGetDevicePointer((void **)&h_dev, m->h_ring, 0));
    GMS_TRY(hipEventRecord(m->ev_entry, s));
    GMS_TRY(hipStreamWaitEvent(m->copy_stream, m->ev_entry, 0));
    gms::RingFence fence(m, s);
    fence.armed = true;

    PiecePool pool(slice, m->image_bytes, piece);
    Workers w(pool, src, false, m->h_ring, hk, m->ev_host, (unsigned)std::min<uint64_t>(threads, pool.npieces));
    for (uint64_t sl = 0; sl < pool.nslices && rc == GMS_OK; ++sl) {
        if (!pool.wait_slice(sl)) break;  // a worker failed
        const uint32_t slot = (uint32_t)(sl % k), hslot = (uint32_t)(sl % hk);
        uint8_t *dev = m->d_ring + (uint64_t)slot * slice;
        const uint64_t lo = sl * slice;
        const uint64_t bytes = std::min(slice, m->image_bytes - lo);
        hipError_t e;
        if ((sl >= k && (e = hipStreamWaitEvent(m->copy_stream, m->ev_free[slot], 0)) != hipSuccess) ||
            (e = gms::launch_host_copy(h_dev + (uint64_t)hslot * slice, dev, bytes, m->copy_stream)) != hipSuccess ||
            (e = hipEventRecord(m->ev_host[hslot], m->copy_stream)) != hipSuccess ||
            (e = hipEventRecord(m->ev_filled[slot], m->copy_stream)) != hipSuccess ||
            (e = hipStreamWaitEvent(s, m->ev_filled[slot], 0)) != hipSuccess ||
            (e = gms::launch_slice(m, gms::kRestore, h, sl, dev, s)) != hipSuccess ||
            (e = hipEventRecord(m->ev_free[slot], s)) != hipSuccess) {
            rc = fail_hip(e, "host restore slice");
            break;
        }
        pool.set_enqueued(sl + 1);
    }
    if ((rc = finish(pool, w, rc, src, false)) != GMS_OK) return rc;
    GMS_TRY(fence.close());
    return GMS_OK;
}

// Snapshot into a host image: the gather kernel fills each slice, which lands
// in its pinned host slot, and the workers write the slot out.  With slices of
// gms::kRingSnapshotMinSlice and up the kernel gathers into a device slot and
// the copy stream copies it to the host slot; smaller slices are gathered
// straight into the host slot over the link.  Returns when every byte is out.
int snapshot_pipeline(gms_manifest *m, const HostImage &dst, const HashOut &h, unsigned threads, uint64_t piece,
                      hipStream_t s)
{
    std::lock_guard<std::mutex> lock(m->ring_mu);
    int rc;
    if ((rc = gms::ensure_host_ring(m)) != GMS_OK) return rc;
    if ((rc = drain_ring(m)) != GMS_OK) return rc;
    const uint64_t slice = m->ring_slice;
    const uint32_t k = m->ring_slots, hk = m->host_slots;
    const bool via_device = slice >= gms::kRingSnapshotMinSlice;
    uint8_t *h_dev = nullptr;  // device view of the pinned host ring
    GMS_TRY(hipHostGetDevicePointer((void **)&h_dev, m->h_ring, 0));

    auto enqueue = [&](uint64_t sl) -> int {
        const uint32_t hslot = (uint32_t)(sl % hk);
        const uint64_t lo = sl * slice;
        if (!via_device) {
            GMS_TRY(gms::launch_slice(m, gms::kSnapshot, h, sl, h_dev + (uint64_t)hslot * slice, s));
            GMS_TRY(hipEventRecord(m->ev_host[hslot], s));
            return GMS_OK;
        }
        const uint32_t slot = (uint32_t)(sl % k);
        uint8_t *dev = m->d_ring + (uint64_t)slot * slice;
        if (sl >= k) GMS_TRY(hipStreamWaitEvent(s, m->ev_free[slot], 0));
        GMS_TRY(gms::launch_slice(m, gms::kSnapshot, h, sl, dev, s));
        GMS_TRY(hipEventRecord(m->ev_filled[slot], s));
        GMS_TRY(hipStreamWaitEvent(m->copy_stream, m->ev_filled[slot], 0));
        GMS_TRY(hipMemcpyAsync(m->h_ring + (uint64_t)hslot * slice, dev, std::min(slice, m->image_bytes - lo),
                               hipMemcpyDeviceToHost, m->copy_stream));
        GMS_TRY(hipEventRecord(m->ev_host[hslot], m->copy_stream));
        GMS_TRY(hipEventRecord(m->ev_free[slot], m->copy_stream));
        return GMS_OK;
    };

    gms::RingFence fence(m, s);
    fence.armed = true;
    PiecePool pool(slice, m->image_bytes, piece);
    Workers w(pool, dst, true, m->h_ring, hk, m->ev_host, (unsigned)std::min<uint64_t>(threads, pool.npieces));
    const uint64_t first = std::min<uint64_t>(hk, pool.nslices);
    for (uint64_t sl = 0; sl < first && rc == GMS_OK; ++sl) rc = enqueue(sl);
    if (rc == GMS_OK) pool.set_enqueued(first);
    for (uint64_t sl = 0; sl + hk < pool.nslices && rc == GMS_OK; ++sl) {
        if (!pool.wait_slice(sl)) break;  // host slot sl % hk is written out: refill it
        if ((rc = enqueue(sl + hk)) == GMS_OK) pool.set_enqueued(sl + hk + 1);
    }
    if ((rc = finish(pool, w, rc, dst, true)) != GMS_OK) return rc;
    GMS_TRY(fence.close());
    return GMS_OK;
}

}  // namespace

extern "C" {

int gms_restore_from_file(const gms_manifest *cm, const char *path, uint64_t file_offset, uint32_t flags,
                          uint32_t io_threads, const uint64_t *expected_blk, uint64_t *blk_hash_out,
                          uint64_t *ten_hash_out, uint64_t *mismatch_count_out, uint64_t *mismatch_list_out,
                          uint64_t mismatch_cap, void *stream)
{
    gms::clear_error();
    int rc = check_manifest(cm, io_threads);
    if (rc != GMS_OK) return rc;
    if (!path) return fail(GMS_ERR_INVALID, "path is null");
    const HashOut h = gms::make_hash(expected_blk, blk_hash_out, ten_hash_out, mismatch_count_out,
                                     mismatch_list_out, mismatch_cap);
    if ((rc = gms::check_outputs(cm, h)) != GMS_OK) return rc;
    gms_manifest *m = const_cast<gms_manifest *>(cm);
    if (file_offset > (uint64_t)INT64_MAX - m->image_bytes)
        return fail(GMS_ERR_INVALID, "file_offset %llu is past any file position", (unsigned long long)file_offset);

    FileHandle f;
    if ((rc = open_file(f, path, false, flags & GMS_FILE_DIRECT, file_offset)) != GMS_OK) return rc;
    struct stat st;
    if (fstat(f.fd, &st) != 0) return fail(GMS_ERR_IO, "fstat(%s): %s", path, strerror(errno));
    if ((uint64_t)st.st_size < file_offset + m->image_bytes)
        return fail(GMS_ERR_SIZE, "%s holds %lld bytes, needs %llu from offset %llu", path, (long long)st.st_size,
                    (unsigned long long)m->image_bytes, (unsigned long long)file_offset);

    DeviceGuard g(m->device);
    if (g.err != hipSuccess) return fail_hip(g.err, "hipSetDevice");
    hipStream_t s = (hipStream_t)stream;
    bool done = false;
    if ((rc = begin(m, h, s, "an image-file call", &done)) != GMS_OK || done) return rc;
    HostImage src;
    src.fd = f.fd;
    src.path = path;
    src.direct = f.direct;
    src.file_offset = file_offset;
    return restore_pipeline(m, src, h, io_threads ? io_threads : kDefaultIoThreads,
                            f.direct ? kDirectPieceBytes : kBufferedPieceBytes, s);
}

int gms_snapshot_to_file(const gms_manifest *cm, const char *path, uint32_t flags, uint32_t io_threads,
                         uint64_t *blk_hash_out, uint64_t *ten_hash_out, void *stream)
{
    gms::clear_error();
    int rc = check_manifest(cm, io_threads);
    if (rc != GMS_OK) return rc;
    if (!path) return fail(GMS_ERR_INVALID, "path is null");
    const HashOut h = gms::make_hash(nullptr, blk_hash_out, ten_hash_out, nullptr, nullptr, 0);
    if ((rc = gms::check_outputs(cm, h)) != GMS_OK) return rc;
    gms_manifest *m = const_cast<gms_manifest *>(cm);

    FileHandle f;
    if ((rc = open_file(f, path, true, flags & GMS_FILE_DIRECT, 0)) != GMS_OK) return rc;

    DeviceGuard g(m->device);
    if (g.err != hipSuccess) return fail_hip(g.err, "hipSetDevice");
    hipStream_t s = (hipStream_t)stream;
    bool done = false;
    if ((rc = begin(m, h, s, "an image-file call", &done)) != GMS_OK) return rc;
    if (done) {
        GMS_TRY(hipStreamSynchronize(s));
    } else {
        HostImage dst;
        dst.fd = f.fd;
        dst.path = path;
        dst.direct = f.direct;
        if ((rc = snapshot_pipeline(m, dst, h, io_threads ? io_threads : kDefaultIoThreads, kDirectPieceBytes, s)) !=
            GMS_OK)
            return rc;
    }
    if ((flags & GMS_FILE_SYNC) && fsync(f.fd) != 0) return fail(GMS_ERR_IO, "fsync(%s): %s", path, strerror(errno));
    return GMS_OK;
}

int gms_restore_from_host(const gms_manifest *cm, const void *image, uint64_t image_bytes, uint32_t threads,
                          const uint64_t *expected_blk, uint64_t *blk_hash_out, uint64_t *ten_hash_out,
                          uint64_t *mismatch_count_out, uint64_t *mismatch_list_out, uint64_t mismatch_cap,
                          void *stream)
{
    gms::clear_error();
    int rc = check_manifest(cm, threads);
    if (rc != GMS_OK) return rc;
    if ((rc = check_memory_image(cm, image, image_bytes)) != GMS_OK) return rc;
    const HashOut h = gms::make_hash(expected_blk, blk_hash_out, ten_hash_out, mismatch_count_out,
                                     mismatch_list_out, mismatch_cap);
    if ((rc = gms::check_outputs(cm, h)) != GMS_OK) return rc;
    gms_manifest *m = const_cast<gms_manifest *>(cm);

    DeviceGuard g(m->device);
    if (g.err != hipSuccess) return fail_hip(g.err, "hipSetDevice");
    hipStream_t s = (hipStream_t)stream;
    bool done = false;
    if ((rc = begin(m, h, s, "a host-image call", &done)) != GMS_OK || done) return rc;
    HostImage src;
    src.mem = const_cast<uint8_t *>(static_cast<const uint8_t *>(image));
    return restore_pipeline(m, src, h, threads ? threads : kDefaultIoThreads, kMemoryPieceBytes, s);
}

int gms_snapshot_to_host(const gms_manifest *cm, void *image, uint64_t image_bytes, uint32_t threads,
                         uint64_t *blk_hash_out, uint64_t *ten_hash_out, void *stream)
{
    gms::clear_error();
    int rc = check_manifest(cm, threads);
    if (rc != GMS_OK) return rc;
    if ((rc = check_memory_image(cm, image, image_bytes)) != GMS_OK) return rc;
    const HashOut h = gms::make_hash(nullptr, blk_hash_out, ten_hash_out, nullptr, nullptr, 0);
    if ((rc = gms::check_outputs(cm, h)) != GMS_OK) return rc;
    gms_manifest *m = const_cast<gms_manifest *>(cm);

    DeviceGuard g(m->device);
    if (g.err != hipSuccess) return fail_hip(g.err, "hipSetDevice");
    hipStream_t s = (hipStream_t)stream;
    bool done = false;
    if ((rc = begin(m, h, s, "a host-image call", &done)) != GMS_OK) return rc;
    if (done) {
        GMS_TRY(hipStreamSynchronize(s));
        return GMS_OK;
    }
    HostImage dst;
    dst.mem = static_cast<uint8_t *>(image);
    return snapshot_pipeline(m, dst, h, threads ? threads : kDefaultIoThreads, kMemoryPieceBytes, s);
}

}  // extern "C"
