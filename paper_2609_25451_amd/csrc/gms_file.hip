// Image files: the packed image written to and streamed back from storage.
//
// A cold replacement repopulates model state from storage while the engine's
// runtime is restored (paper section 3.3 and section 4, cold GMS repopulation);
// the end-to-end cost is the artifact size over the effective bandwidth
// (section 3.1).  Restore runs a three-stage pipeline per staging slice:
// parallel pread (O_DIRECT through per-worker bounce buffers when the file
// system allows it, buffered otherwise) into a pinned host slot, a DMA of
// that slot into a device slot on the manifest's copy stream, and the
// scatter(+hash) kernel on the caller's stream.  One pool of I/O workers
// takes pieces (16 MiB direct, up to 64 MiB buffered) in file order from a
// shared counter, so every worker keeps a large request in flight and none
// waits for a slower slice; a host slot is refilled once the DMA that read it
// has finished, so storage, the host link and HBM all stay busy.  Snapshot runs the mirror image: the
// gather kernel writes each slice straight into a pinned host slot (zero-copy)
// and the workers write its pieces to the file.

#include <fcntl.h>
#include <sys/stat.h>
#include <unistd.h>

#include <algorithm>
#include <atomic>
#include <cerrno>
#include <cstdint>
#include <condition_variable>
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
// One pread/pwrite.  Direct I/O loses storage bandwidth below 16 MiB per
// request; buffered reads go through the page cache's readahead and copy,
// which run best at 64 MiB per request (at most one slice).
constexpr uint64_t kDirectPieceBytes = 16ull << 20;
constexpr uint64_t kBufferedPieceBytes = 64ull << 20;

struct FileHandle {
    int fd = -1;
    bool direct = false;
    ~FileHandle()
    {
        if (fd >= 0) close(fd);
    }
};

// Moves `len` bytes between `buf` and file offset `off`.  Direct I/O cannot
// target the pinned slots (the kernel refuses to pin driver-mapped pages:
// EFAULT), so with O_DIRECT the bytes go through the worker's page-aligned
// bounce buffer.  Returns 0 or an errno value (EIO for a file that ends early).
int transfer_piece(int fd, uint8_t *bounce, uint8_t *buf, uint64_t len, uint64_t off, bool write)
{
    uint8_t *mem = bounce ? bounce : buf;
    if (write && bounce) memcpy(bounce, buf, len);
    uint64_t done = 0;
    while (done < len) {
        ssize_t r = write ? pwrite(fd, mem + done, len - done, (off_t)(off + done))
                          : pread(fd, mem + done, len - done, (off_t)(off + done));
        if (r < 0) {
            if (errno == EINTR) continue;
            return errno;
        }
        if (r == 0) return EIO;
        done += (uint64_t)r;
    }
    if (!write && bounce) memcpy(buf, bounce, len);
    return 0;
}

// The image cut into slices (one host slot each) and each slice into pieces of
// at most `piece` bytes, numbered in file order.  `enqueued` counts the slices
// whose device-side step the caller's thread has enqueued; `left[s]` counts
// the pieces of slice s not yet transferred.  The first error stops every
// worker.
struct PiecePool {
    uint64_t slice = 0, image_bytes = 0, piece = 0, per_slice = 0, nslices = 0, npieces = 0;
    uint64_t file_offset = 0;  // file position of image byte 0
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
// host slot s % hslots; for a read it first waits until the DMA out of that
// slot for slice s - hslots has been enqueued and has finished; for a write it
// waits until the gather of slice s has been enqueued and has finished.
class Workers {
public:
    Workers(PiecePool &pool, int fd, const char *path, bool direct, bool write, uint8_t *h_ring, uint32_t hslots,
            const hipEvent_t *ev_host, unsigned threads)
    {
        for (unsigned t = 0; t < threads; ++t) {
            try {
                pool_.emplace_back([=, &pool] { run(pool, fd, path, direct, write, h_ring, hslots, ev_host); });
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
    static void run(PiecePool &pool, int fd, const char *path, bool direct, bool write, uint8_t *h_ring,
                    uint32_t hslots, const hipEvent_t *ev_host)
    {
        uint8_t *bounce = nullptr;
        if (direct && posix_memalign((void **)&bounce, kDirectAlign, pool.piece) != 0) {
            pool.fail_stop(ENOMEM, false);
            return;
        }
        // Buffered reads: the kernel keeps readahead state per open file, and
        // workers taking interleaved pieces through one descriptor defeat it,
        // so each worker reads through a descriptor of its own (the shared
        // one if the file cannot be opened again).
        const int own = (!write && !direct && path) ? open(path, O_RDONLY | O_CLOEXEC) : -1;
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
            const int e = transfer_piece(own >= 0 ? own : fd, bounce, host, bytes, pool.file_offset + lo, write);
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

int check_file_args(const gms_manifest *m, const char *path, unsigned io_threads)
{
    if (!m) return fail(GMS_ERR_INVALID, "manifest is null");
    if (m->device < 0) return fail(GMS_ERR_STATE, "host-only manifest has no device");
    if (!path) return fail(GMS_ERR_INVALID, "path is null");
    if (io_threads > kMaxIoThreads) return fail(GMS_ERR_INVALID, "io_threads %u > %u", io_threads, kMaxIoThreads);
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
int finish(PiecePool &pool, Workers &w, int rc, const char *path, bool write)
{
    if (rc != GMS_OK) pool.fail_stop(0, false);
    w.join();
    if (rc != GMS_OK) return rc;
    if (pool.hip_err) return fail(GMS_ERR_HIP, "waiting for a staging slot of %s", path);
    if (pool.err) return fail(GMS_ERR_IO, "%s %s: %s", write ? "writing" : "reading", path, strerror(pool.err));
    return GMS_OK;
}

#define GMS_TRY(call)                                              \
    do {                                                           \
        hipError_t e_ = (call);                                    \
        if (e_ != hipSuccess) return fail_hip(e_, #call);          \
    } while (0)

}  // namespace

extern "C" {

int gms_restore_from_file(const gms_manifest *cm, const char *path, uint64_t file_offset, uint32_t flags,
                          uint32_t io_threads, const uint64_t *expected_blk, uint64_t *blk_hash_out,
                          uint64_t *ten_hash_out, uint64_t *mismatch_count_out, uint64_t *mismatch_list_out,
                          uint64_t mismatch_cap, void *stream)
{
    gms::clear_error();
    int rc = check_file_args(cm, path, io_threads);
    if (rc != GMS_OK) return rc;
    const HashOut h = gms::make_hash(expected_blk, blk_hash_out, ten_hash_out, mismatch_count_out,
                                     mismatch_list_out, mismatch_cap);
    if ((rc = gms::check_outputs(cm, h)) != GMS_OK) return rc;
    gms_manifest *m = const_cast<gms_manifest *>(cm);
    const unsigned threads = io_threads ? io_threads : kDefaultIoThreads;

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
    if ((rc = gms::refuse_capture(s, "an image-file call")) != GMS_OK) return rc;
    GMS_TRY(gms::launch_prologue(h, m->n, s));
    if (m->chunks.empty()) return GMS_OK;

    std::lock_guard<std::mutex> lock(m->ring_mu);
    if ((rc = gms::ensure_host_ring(m)) != GMS_OK) return rc;
    if ((rc = drain_ring(m)) != GMS_OK) return rc;
    const uint64_t slice = m->ring_slice;
    const uint32_t k = m->ring_slots, hk = m->host_slots;
    GMS_TRY(hipEventRecord(m->ev_entry, s));
    GMS_TRY(hipStreamWaitEvent(m->copy_stream, m->ev_entry, 0));

    PiecePool pool(slice, m->image_bytes, f.direct ? kDirectPieceBytes : kBufferedPieceBytes);
    pool.file_offset = file_offset;
    Workers w(pool, f.fd, path, f.direct, false, m->h_ring, hk, m->ev_host,
              (unsigned)std::min<uint64_t>(threads, pool.npieces));
    for (uint64_t sl = 0; sl < pool.nslices && rc == GMS_OK; ++sl) {
        if (!pool.wait_slice(sl)) break;  // a worker failed
        const uint32_t slot = (uint32_t)(sl % k), hslot = (uint32_t)(sl % hk);
        uint8_t *host = m->h_ring + (uint64_t)hslot * slice;
        uint8_t *dev = m->d_ring + (uint64_t)slot * slice;
        const uint64_t lo = sl * slice;
        const uint64_t bytes = std::min(slice, m->image_bytes - lo);
        hipError_t e;
        if ((sl >= k && (e = hipStreamWaitEvent(m->copy_stream, m->ev_free[slot], 0)) != hipSuccess) ||
            (e = hipMemcpyAsync(dev, host, bytes, hipMemcpyHostToDevice, m->copy_stream)) != hipSuccess ||
            (e = hipEventRecord(m->ev_host[hslot], m->copy_stream)) != hipSuccess ||
            (e = hipEventRecord(m->ev_filled[slot], m->copy_stream)) != hipSuccess ||
            (e = hipStreamWaitEvent(s, m->ev_filled[slot], 0)) != hipSuccess ||
            (e = gms::launch_stream(gms::kRestore, h.any(), m->d_chunks, m->slice_first[sl],
                                    m->slice_first[sl + 1] - m->slice_first[sl], m->max_chunk, dev, lo, h, s)) !=
                hipSuccess ||
            (e = hipEventRecord(m->ev_free[slot], s)) != hipSuccess) {
            rc = fail_hip(e, "file restore slice");
            break;
        }
        pool.set_enqueued(sl + 1);
    }
    if ((rc = finish(pool, w, rc, path, false)) != GMS_OK) return rc;
    GMS_TRY(hipEventRecord(m->ev_done, s));
    m->done_recorded = true;
    return GMS_OK;
}

int gms_snapshot_to_file(const gms_manifest *cm, const char *path, uint32_t flags, uint32_t io_threads,
                         uint64_t *blk_hash_out, uint64_t *ten_hash_out, void *stream)
{
    gms::clear_error();
    int rc = check_file_args(cm, path, io_threads);
    if (rc != GMS_OK) return rc;
    const HashOut h = gms::make_hash(nullptr, blk_hash_out, ten_hash_out, nullptr, nullptr, 0);
    if ((rc = gms::check_outputs(cm, h)) != GMS_OK) return rc;
    gms_manifest *m = const_cast<gms_manifest *>(cm);
    const unsigned threads = io_threads ? io_threads : kDefaultIoThreads;

    FileHandle f;
    if ((rc = open_file(f, path, true, flags & GMS_FILE_DIRECT, 0)) != GMS_OK) return rc;

    DeviceGuard g(m->device);
    if (g.err != hipSuccess) return fail_hip(g.err, "hipSetDevice");
    hipStream_t s = (hipStream_t)stream;
    if ((rc = gms::refuse_capture(s, "an image-file call")) != GMS_OK) return rc;
    GMS_TRY(gms::launch_prologue(h, m->n, s));
    if (m->chunks.empty()) {
        GMS_TRY(hipStreamSynchronize(s));
        return GMS_OK;
    }

    std::lock_guard<std::mutex> lock(m->ring_mu);
    if ((rc = gms::ensure_host_ring(m)) != GMS_OK) return rc;
    if ((rc = drain_ring(m)) != GMS_OK) return rc;
    const uint64_t slice = m->ring_slice;
    const uint32_t hk = m->host_slots;
    uint8_t *h_dev = nullptr;  // device view of the pinned host ring
    GMS_TRY(hipHostGetDevicePointer((void **)&h_dev, m->h_ring, 0));

    // gather slice `sl` straight into its pinned host slot (zero-copy writes
    // over the host link keep it saturated more steadily than a device slot
    // plus DMA)
    auto enqueue = [&](uint64_t sl) -> int {
        const uint32_t hslot = (uint32_t)(sl % hk);
        const uint64_t c0 = m->slice_first[sl], c1 = m->slice_first[sl + 1];
        GMS_TRY(gms::launch_stream(gms::kSnapshot, h.any(), m->d_chunks, c0, c1 - c0, m->max_chunk,
                                   h_dev + (uint64_t)hslot * slice, sl * slice, h, s));
        GMS_TRY(hipEventRecord(m->ev_host[hslot], s));
        return GMS_OK;
    };

    PiecePool pool(slice, m->image_bytes, kDirectPieceBytes);
    Workers w(pool, f.fd, path, f.direct, true, m->h_ring, hk, m->ev_host,
              (unsigned)std::min<uint64_t>(threads, pool.npieces));
    const uint64_t first = std::min<uint64_t>(hk, pool.nslices);
    for (uint64_t sl = 0; sl < first && rc == GMS_OK; ++sl) rc = enqueue(sl);
    if (rc == GMS_OK) pool.set_enqueued(first);
    for (uint64_t sl = 0; sl + hk < pool.nslices && rc == GMS_OK; ++sl) {
        if (!pool.wait_slice(sl)) break;  // host slot sl % hk is written out: refill it
        if ((rc = enqueue(sl + hk)) == GMS_OK) pool.set_enqueued(sl + hk + 1);
    }
    if ((rc = finish(pool, w, rc, path, true)) != GMS_OK) return rc;
    GMS_TRY(hipEventRecord(m->ev_done, s));
    m->done_recorded = true;
    if ((flags & GMS_FILE_SYNC) && fsync(f.fd) != 0) return fail(GMS_ERR_IO, "fsync(%s): %s", path, strerror(errno));
    return GMS_OK;
}

}  // extern "C"
