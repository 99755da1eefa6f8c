// Image files: the packed image written to and streamed back from storage.
//
// A cold replacement repopulates model state from storage while the engine's
// runtime is restored (paper section 3.3 and section 4, cold GMS repopulation);
// the end-to-end cost is the artifact size over the effective bandwidth
// (section 3.1).  Restore runs a three-stage pipeline per 64 MiB slice:
// parallel pread (O_DIRECT through per-worker bounce buffers when the file
// system allows it, buffered otherwise) into a pinned host slot, a DMA of
// that slot into a device slot on the manifest's copy stream, and the
// scatter(+hash) kernel on the caller's stream.  Host slots are reused
// once the DMA that read them has finished, so storage, the host link and HBM
// all stay busy.  Snapshot gathers each slice straight into a pinned host slot
// (zero-copy) and writes it with pwrite.

#include <fcntl.h>
#include <sys/stat.h>
#include <unistd.h>

#include <algorithm>
#include <atomic>
#include <cerrno>
#include <cstdlib>
#include <cstring>
#include <future>
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

constexpr unsigned kDefaultIoThreads = 8;
constexpr unsigned kMaxIoThreads = 64;
constexpr uint64_t kDirectAlign = 4096;

struct FileHandle {
    int fd = -1;
    bool direct = false;
    ~FileHandle()
    {
        if (fd >= 0) close(fd);
    }
};

// Per-call I/O context: `lanes` independent transfers (one per ring slot in
// flight) of `threads` workers each.  Direct I/O cannot target the pinned
// slots (the kernel refuses to pin driver-mapped pages: EFAULT), so with
// O_DIRECT every worker moves data through a private page-aligned bounce
// buffer and copies to or from the pinned slot; buffered I/O reads and writes
// the slot itself.
struct IoCtx {
    int fd = -1;
    bool direct = false;
    unsigned threads = 1;
    uint64_t bounce_bytes = 0;
    std::vector<uint8_t *> bounce;  // [lane * threads + worker]
    ~IoCtx()
    {
        for (uint8_t *b : bounce) free(b);
    }
    int init(int fd_, bool direct_, unsigned lanes, unsigned threads_, uint64_t slice)
    {
        fd = fd_;
        direct = direct_;
        threads = threads_;
        if (!direct) return GMS_OK;
        bounce_bytes = std::min<uint64_t>(16ull << 20, ceil_div(ceil_div(slice, threads), kDirectAlign) * kDirectAlign);
        for (unsigned t = 0; t < lanes * threads; ++t) {
            void *b = nullptr;
            if (posix_memalign(&b, kDirectAlign, bounce_bytes) != 0) return fail(GMS_ERR_NOMEM, "bounce buffer");
            bounce.push_back((uint8_t *)b);
        }
        return GMS_OK;
    }
};

// One worker's share: bytes [lo, hi) of buf <-> file offset off + lo, using
// bounce buffer `b` for direct I/O.  Returns 0 or an errno value (EIO for a
// file that ends early).
int transfer_range(const IoCtx &io, uint8_t *b, uint8_t *buf, uint64_t lo, uint64_t hi, uint64_t off, bool write,
                   const std::atomic<int> &stop)
{
    uint64_t p = lo;
    while (p < hi && !stop.load(std::memory_order_relaxed)) {
        const uint64_t want = io.direct ? std::min(hi - p, io.bounce_bytes) : hi - p;
        uint8_t *mem = io.direct ? b : buf + p;
        if (write && io.direct) memcpy(mem, buf + p, want);
        uint64_t done = 0;
        while (done < want) {
            ssize_t r = write ? pwrite(io.fd, mem + done, want - done, (off_t)(off + p + done))
                              : pread(io.fd, mem + done, want - done, (off_t)(off + p + done));
            if (r < 0) {
                if (errno == EINTR) continue;
                return errno;
            }
            if (r == 0) return EIO;
            done += (uint64_t)r;
        }
        if (!write && io.direct) memcpy(buf + p, mem, want);
        p += want;
    }
    return 0;
}

// Moves exactly `len` bytes between buf and file offset `off` with lane
// `lane`'s workers on disjoint 4 KiB-aligned ranges.
int transfer(const IoCtx &io, unsigned lane, uint8_t *buf, uint64_t len, uint64_t off, bool write)
{
    std::atomic<int> err{0};
    uint64_t per = ceil_div(len, io.threads);
    per = ceil_div(per, kDirectAlign) * kDirectAlign;
    auto work = [&](unsigned t, uint64_t lo, uint64_t hi) {
        uint8_t *b = io.direct ? io.bounce[lane * io.threads + t] : nullptr;
        int e = transfer_range(io, b, buf, lo, hi, off, write, err);
        if (e) err = e;
    };
    std::vector<std::thread> pool;
    for (unsigned t = 1; t < io.threads && t * per < len; ++t)
        pool.emplace_back(work, t, t * per, std::min(len, (t + 1) * per));
    work(0, 0, std::min(len, per));
    for (auto &t : pool) t.join();
    return err.load();
}

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
    GMS_TRY(gms::launch_prologue(h, m->n, s));
    if (m->chunks.empty()) return GMS_OK;

    std::lock_guard<std::mutex> lock(m->ring_mu);
    if ((rc = gms::ensure_host_ring(m)) != GMS_OK) return rc;
    if ((rc = drain_ring(m)) != GMS_OK) return rc;
    const uint64_t slice = m->ring_slice;
    const uint32_t k = m->ring_slots;
    const uint64_t nslices = ceil_div(m->image_bytes, slice);
    // every host slot has its own read in flight; the workers are shared out
    const unsigned per_slot = std::max(1u, threads / k);
    IoCtx io;
    if ((rc = io.init(f.fd, f.direct, k, per_slot, slice)) != GMS_OK) return rc;
    std::vector<std::future<int>> reads(k);
    auto start_read = [&](uint64_t sl) -> int {
        const uint32_t slot = (uint32_t)(sl % k);
        if (sl >= k) GMS_TRY(hipEventSynchronize(m->ev_host[slot]));  // the DMA out of this slot is done
        uint8_t *host = m->h_ring + (uint64_t)slot * slice;
        const uint64_t lo = sl * slice;
        const uint64_t bytes = std::min(slice, m->image_bytes - lo);
        reads[slot] = std::async(std::launch::async, [&io, slot, host, bytes, lo, file_offset] {
            return transfer(io, slot, host, bytes, file_offset + lo, false);
        });
        return GMS_OK;
    };
    // joins every read still in flight (they use `io` and the host slots)
    auto join_reads = [&] {
        for (auto &r : reads)
            if (r.valid()) r.wait();
    };

    GMS_TRY(hipEventRecord(m->ev_entry, s));
    GMS_TRY(hipStreamWaitEvent(m->copy_stream, m->ev_entry, 0));
    for (uint64_t sl = 0; sl < std::min<uint64_t>(k, nslices); ++sl)
        if ((rc = start_read(sl)) != GMS_OK) return join_reads(), rc;
    for (uint64_t sl = 0; sl < nslices; ++sl) {
        const uint32_t slot = (uint32_t)(sl % k);
        uint8_t *host = m->h_ring + (uint64_t)slot * slice;
        uint8_t *dev = m->d_ring + (uint64_t)slot * slice;
        const uint64_t lo = sl * slice;
        const uint64_t bytes = std::min(slice, m->image_bytes - lo);
        const int err = reads[slot].get();
        if (err) {
            join_reads();
            return fail(GMS_ERR_IO, "reading %s at %llu: %s", path, (unsigned long long)(file_offset + lo),
                        strerror(err));
        }
        hipError_t e;
        if ((sl >= k && (e = hipStreamWaitEvent(m->copy_stream, m->ev_free[slot], 0)) != hipSuccess) ||
            (e = hipMemcpyAsync(dev, host, bytes, hipMemcpyHostToDevice, m->copy_stream)) != hipSuccess ||
            (e = hipEventRecord(m->ev_host[slot], m->copy_stream)) != hipSuccess ||
            (e = hipEventRecord(m->ev_filled[slot], m->copy_stream)) != hipSuccess ||
            (e = hipStreamWaitEvent(s, m->ev_filled[slot], 0)) != hipSuccess ||
            (e = gms::launch_stream(gms::kRestore, h.any(), m->d_chunks, m->slice_first[sl],
                                    m->slice_first[sl + 1] - m->slice_first[sl], dev, lo, h, s)) != hipSuccess ||
            (e = hipEventRecord(m->ev_free[slot], s)) != hipSuccess) {
            join_reads();
            return fail_hip(e, "file restore slice");
        }
        if (sl + k < nslices && (rc = start_read(sl + k)) != GMS_OK) return join_reads(), rc;
    }
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
    GMS_TRY(gms::launch_prologue(h, m->n, s));
    if (m->chunks.empty()) {
        GMS_TRY(hipStreamSynchronize(s));
        return GMS_OK;
    }

    std::lock_guard<std::mutex> lock(m->ring_mu);
    if ((rc = gms::ensure_host_ring(m)) != GMS_OK) return rc;
    if ((rc = drain_ring(m)) != GMS_OK) return rc;
    const uint64_t slice = m->ring_slice;
    const uint32_t k = m->ring_slots;
    const uint64_t nslices = ceil_div(m->image_bytes, slice);
    IoCtx io;
    if ((rc = io.init(f.fd, f.direct, 1, threads, slice)) != GMS_OK) return rc;
    uint8_t *h_dev = nullptr;  // device view of the pinned host ring
    GMS_TRY(hipHostGetDevicePointer((void **)&h_dev, m->h_ring, 0));

    // gather slice `sl` straight into its pinned host slot (zero-copy writes
    // over the host link keep it saturated more steadily than a device slot
    // plus DMA)
    auto enqueue = [&](uint64_t sl) -> int {
        const uint32_t slot = (uint32_t)(sl % k);
        const uint64_t c0 = m->slice_first[sl], c1 = m->slice_first[sl + 1];
        GMS_TRY(gms::launch_stream(gms::kSnapshot, h.any(), m->d_chunks, c0, c1 - c0,
                                   h_dev + (uint64_t)slot * slice, sl * slice, h, s));
        GMS_TRY(hipEventRecord(m->ev_host[slot], s));
        return GMS_OK;
    };

    for (uint64_t sl = 0; sl < std::min<uint64_t>(k, nslices); ++sl)
        if ((rc = enqueue(sl)) != GMS_OK) return rc;
    for (uint64_t sl = 0; sl < nslices; ++sl) {
        const uint32_t slot = (uint32_t)(sl % k);
        const uint64_t lo = sl * slice;
        const uint64_t bytes = std::min(slice, m->image_bytes - lo);
        GMS_TRY(hipEventSynchronize(m->ev_host[slot]));
        int err = transfer(io, 0, m->h_ring + (uint64_t)slot * slice, bytes, lo, true);
        if (err) return fail(GMS_ERR_IO, "writing %s at %llu: %s", path, (unsigned long long)lo, strerror(err));
        if (sl + k < nslices && (rc = enqueue(sl + k)) != GMS_OK) return rc;
    }
    GMS_TRY(hipEventRecord(m->ev_done, s));
    m->done_recorded = true;
    if ((flags & GMS_FILE_SYNC) && fsync(f.fd) != 0) return fail(GMS_ERR_IO, "fsync(%s): %s", path, strerror(errno));
    return GMS_OK;
}

}  // extern "C"
