// GMS across processes: an owner process that holds a GPU's model-state
// allocations, and the engines that attach to them (paper section 3.2, GMS
// and Figure 4; section 4, GMS implementation).
//
// The owner creates physical device memory (HIP virtual memory) and never maps
// it; an engine's crash therefore cannot take the allocations with it.  It
// hands allocations to clients as POSIX file descriptors (dma-buf) over a
// Unix-domain socket, and it runs the lease protocol: one writer populates the
// state under an exclusive read-write lease and commits it, readers attach,
// a writer that leaves before commit (its connection closes, whether by
// disconnect or by death) has its incomplete state discarded, and a reader
// that leaves only ends its own lease.
//
// Clients map each descriptor as external memory.  On this ROCm a virtual-
// memory handle imports only in the process that exported it (in any other
// process the runtime refuses the same descriptor, measured), while the
// external-memory import of the descriptor works in every process; such a
// mapping has no access flags, so a reader's read-only use is the library's
// contract (no call writes through a reader's mapping) rather than the page
// tables', and readers check the state before they use it.
//
// The owner never touches the pages, so the checks that need the contents run
// in the clients with the library's kernels: at commit the writer hashes every
// 4 KiB block of the committed layout (and can compare with hashes recorded at
// snapshot), and the owner keeps those hashes; a reader that asks for it
// re-hashes the state it mapped before it uses it, and a mismatch invalidates
// the committed state at the owner (section 3.2: integrity errors invalidate
// GMS state) until a writer repopulates and commits again.
//
// An allocation travels as one descriptor of at most GMS_IPC_PIECE_BYTES
// (1 GiB); larger requests are refused.

#include <errno.h>
#include <fcntl.h>
#include <stdio.h>
#include <poll.h>
#include <signal.h>
#include <sys/mman.h>
#include <sys/resource.h>
#include <sys/socket.h>
#include <sys/types.h>
#include <sys/un.h>
#include <unistd.h>

#include <algorithm>
#include <atomic>
#include <cstring>
#include <map>
#include <mutex>
#include <new>
#include <optional>
#include <string>
#include <vector>

#include "gms_host.h"

using gms::DeviceGuard;
using gms::fail;
using gms::fail_hip;

namespace {

constexpr uint32_t kMagic = 0x31534D47u;  // "GMS1"
constexpr uint32_t kMaxFdsPerMsg = 128;
constexpr uint64_t kMaxPayload = 1ull << 32;  // refuse absurd lengths from a broken peer
constexpr uint64_t kRecvPiece = 1ull << 20;   // payload bytes received per step

enum Op : uint32_t {
    kHelloRW = 1,
    kHelloRO = 2,
    kAlloc = 3,
    kFree = 4,
    kCommit = 5,
    kAbort = 6,
    kInvalidate = 7,
    kBye = 8,
    kStatus = 9,
    kFds = 10,
};

// Every message: this header, then `payload` bytes; `nfds` descriptors ride
// with the header (SCM_RIGHTS).
struct Wire {
    uint32_t magic = kMagic;
    uint32_t op = 0;
    int32_t status = GMS_OK;
    uint32_t nfds = 0;
    uint64_t lease = 0;
    uint64_t arg[4] = {};
    uint64_t payload = 0;
};

// ---------------------------------------------------------------- socket I/O

int send_all(int fd, const void *p, size_t n)
{
    const uint8_t *b = (const uint8_t *)p;
    while (n) {
        ssize_t k = send(fd, b, n, MSG_NOSIGNAL);
        if (k < 0 && errno == EINTR) continue;
        if (k <= 0) return -1;
        b += k;
        n -= (size_t)k;
    }
    return 0;
}

int recv_all(int fd, void *p, size_t n)
{
    uint8_t *b = (uint8_t *)p;
    while (n) {
        ssize_t k = recv(fd, b, n, 0);
        if (k < 0 && errno == EINTR) continue;
        if (k <= 0) return -1;
        b += k;
        n -= (size_t)k;
    }
    return 0;
}

// Sends a header (with up to kMaxFdsPerMsg descriptors) and its payload.
int send_msg(int fd, Wire w, const void *payload, const std::vector<int> &fds)
{
    w.nfds = (uint32_t)fds.size();
    struct iovec iov = {&w, sizeof w};
    struct msghdr mh = {};
    mh.msg_iov = &iov;
    mh.msg_iovlen = 1;
    std::vector<uint8_t> ctl;
    if (!fds.empty()) {
        ctl.assign(CMSG_SPACE(fds.size() * sizeof(int)), 0);
        mh.msg_control = ctl.data();
        mh.msg_controllen = ctl.size();
        struct cmsghdr *c = CMSG_FIRSTHDR(&mh);
        c->cmsg_level = SOL_SOCKET;
        c->cmsg_type = SCM_RIGHTS;
        c->cmsg_len = CMSG_LEN(fds.size() * sizeof(int));
        memcpy(CMSG_DATA(c), fds.data(), fds.size() * sizeof(int));
    }
    ssize_t k;
    do {
        k = sendmsg(fd, &mh, MSG_NOSIGNAL);
    } while (k < 0 && errno == EINTR);
    if (k <= 0) return -1;
    if ((size_t)k < sizeof w && send_all(fd, (const uint8_t *)&w + k, sizeof w - (size_t)k)) return -1;
    return w.payload ? send_all(fd, payload, w.payload) : 0;
}

// Receives one message; descriptors are appended to `fds` (the caller owns them).
int recv_msg(int fd, Wire &w, std::vector<uint8_t> &payload, std::vector<int> &fds)
{
    struct iovec iov = {&w, sizeof w};
    struct msghdr mh = {};
    mh.msg_iov = &iov;
    mh.msg_iovlen = 1;
    std::vector<uint8_t> ctl(CMSG_SPACE(kMaxFdsPerMsg * sizeof(int)));
    mh.msg_control = ctl.data();
    mh.msg_controllen = ctl.size();
    ssize_t k;
    do {
        k = recvmsg(fd, &mh, MSG_CMSG_CLOEXEC);
    } while (k < 0 && errno == EINTR);
    if (k <= 0) return -1;
    for (struct cmsghdr *c = CMSG_FIRSTHDR(&mh); c; c = CMSG_NXTHDR(&mh, c))
        if (c->cmsg_level == SOL_SOCKET && c->cmsg_type == SCM_RIGHTS) {
            const size_t nfd = (c->cmsg_len - CMSG_LEN(0)) / sizeof(int);
            const int *p = (const int *)CMSG_DATA(c);
            fds.insert(fds.end(), p, p + nfd);
        }
    if ((size_t)k < sizeof w && recv_all(fd, (uint8_t *)&w + k, sizeof w - (size_t)k)) return -1;
    if (w.magic != kMagic || w.payload > kMaxPayload) return -1;
    // the buffer grows with the bytes that arrive, so a length alone reserves nothing
    payload.clear();
    for (uint64_t got = 0; got < w.payload;) {
        const uint64_t part = std::min<uint64_t>(w.payload - got, kRecvPiece);
        payload.resize(got + part);
        if (recv_all(fd, payload.data() + got, part)) return -1;
        got += part;
    }
    return 0;
}

void close_all(std::vector<int> &fds)
{
    for (int f : fds) close(f);
    fds.clear();
}

// Appends POD values to a payload, and reads them back.
struct Out {
    std::vector<uint8_t> b;
    template <class T> void put(const T &v)
    {
        const uint8_t *p = (const uint8_t *)&v;
        b.insert(b.end(), p, p + sizeof v);
    }
    void put_raw(const void *p, size_t n) { b.insert(b.end(), (const uint8_t *)p, (const uint8_t *)p + n); }
};

struct In {
    const uint8_t *p, *end;
    explicit In(const std::vector<uint8_t> &v) : p(v.data()), end(v.data() + v.size()) {}
    template <class T> bool get(T &v)
    {
        if ((size_t)(end - p) < sizeof v) return false;
        memcpy(&v, p, sizeof v);
        p += sizeof v;
        return true;
    }
    bool get_raw(void *d, size_t n)
    {
        if ((size_t)(end - p) < n) return false;
        if (n) memcpy(d, p, n);  // an empty table's buffer may be null
        p += n;
        return true;
    }
};

int connect_to(const char *path, int *out)
{
    struct sockaddr_un sa = {};
    if (!path || strlen(path) >= sizeof sa.sun_path) return fail(GMS_ERR_INVALID, "socket path is null or too long");
    int fd = socket(AF_UNIX, SOCK_STREAM | SOCK_CLOEXEC, 0);
    if (fd < 0) return fail(GMS_ERR_IO, "socket: %s", strerror(errno));
    sa.sun_family = AF_UNIX;
    strcpy(sa.sun_path, path);
    if (connect(fd, (struct sockaddr *)&sa, sizeof sa) != 0) {
        const int err = errno;
        close(fd);
        return fail(GMS_ERR_IO, "connect(%s): %s", path, strerror(err));
    }
    *out = fd;
    return GMS_OK;
}

hipMemAllocationProp shareable_prop(int device)
{
    hipMemAllocationProp prop = {};
    prop.type = hipMemAllocationTypePinned;
    prop.requestedHandleTypes = hipMemHandleTypePosixFileDescriptor;
    prop.location.type = hipMemLocationTypeDevice;
    prop.location.id = device;
    return prop;
}

uint64_t round_up(uint64_t v, uint64_t a) { return (v + a - 1) / a * a; }

}  // namespace

// ====================================================================== owner

namespace {

constexpr uint64_t kAllocSlab = 1;  // allocation flag: the writer suballocates it

struct OwnedAlloc {
    uint64_t bytes = 0;  // as requested; the handle holds them rounded to the granularity
    uint64_t size = 0;   // the handle's size
    uint64_t flags = 0;  // kAllocSlab, as the writer asked; kept for later writers
    hipMemGenericAllocationHandle_t handle{};
};

struct LayoutRec {
    uint64_t alloc, off, nbytes;
};

struct Conn {
    int fd = -1;
    int role = 0;  // 0 none, 1 writer, 2 reader
    uint64_t lease = 0;
};

}  // namespace

struct gms_owner {
    int device = GMS_HOST_ONLY;
    uint64_t gran = 4096;
    std::string path;
    int listen_fd = -1;
    int wake[2] = {-1, -1};
    std::atomic<bool> stop{false};
    int state = GMS_STORE_EMPTY;
    bool invalid = false;
    uint64_t next_lease = 1, next_alloc = 1;
    std::map<uint64_t, OwnedAlloc> allocs;
    std::vector<LayoutRec> layout;
    std::vector<uint64_t> hashes;  // commit-time block hashes of the layout
    std::vector<Conn> conns;
    std::mutex mu;  // guards the fields gms_owner_status reads from another thread
};

namespace {

uint32_t readers_of(const gms_owner *o)
{
    uint32_t r = 0;
    for (const Conn &c : o->conns) r += c.role == 2;
    return r;
}

void release_alloc(gms_owner *o, OwnedAlloc &a)
{
    if (o->device != GMS_HOST_ONLY && a.size) {
        DeviceGuard g(o->device);
        (void)hipMemRelease(a.handle);
    }
    a.size = 0;
}

void discard(gms_owner *o)
{
    for (auto &kv : o->allocs) release_alloc(o, kv.second);
    o->allocs.clear();
    o->layout.clear();
    o->hashes.clear();
    o->invalid = false;
    o->state = GMS_STORE_EMPTY;
}

// A POSIX descriptor for handle h.  The descriptor is written through the
// pointer; a 64-bit buffer keeps a wider write than an int from running past it.
hipError_t export_fd(hipMemGenericAllocationHandle_t h, int *fd)
{
    uint64_t buf = ~0ull;
    hipError_t e = hipMemExportToShareableHandle(&buf, h, hipMemHandleTypePosixFileDescriptor, 0);
    if (e != hipSuccess) {
        (void)hipGetLastError();
        return e;
    }
    *fd = (int)(uint32_t)buf;
    return hipSuccess;
}

// A descriptor per allocation, in allocation-id order, with the table
// {id, bytes, size, flags} in `out`.
int export_all(gms_owner *o, Out &out, std::vector<int> &fds)
{
    out.put((uint64_t)o->allocs.size());
    for (auto &kv : o->allocs) {
        const OwnedAlloc &a = kv.second;
        out.put(kv.first);
        out.put(a.bytes);
        out.put(a.size);
        out.put(a.flags);
        int fd = -1;
        DeviceGuard g(o->device);
        hipError_t e = export_fd(a.handle, &fd);
        if (e != hipSuccess) {
            close_all(fds);
            return fail_hip(e, "hipMemExportToShareableHandle");
        }
        fds.push_back(fd);
    }
    return GMS_OK;
}

void put_layout(const gms_owner *o, Out &out)
{
    out.put((uint64_t)o->layout.size());
    out.put_raw(o->layout.data(), o->layout.size() * sizeof(LayoutRec));
    out.put((uint64_t)o->hashes.size());
    out.put_raw(o->hashes.data(), o->hashes.size() * sizeof(uint64_t));
}

// Sends a reply whose descriptors may exceed one message: the reply carries the
// first kMaxFdsPerMsg, kFds messages the rest.  Closes the owner's copies.
int reply_with_fds(int fd, Wire w, const Out &out, std::vector<int> &fds)
{
    w.arg[3] = fds.size();
    w.payload = out.b.size();
    std::vector<int> first(fds.begin(), fds.begin() + std::min<size_t>(fds.size(), kMaxFdsPerMsg));
    int rc = send_msg(fd, w, out.b.data(), first);
    for (size_t i = first.size(); rc == 0 && i < fds.size(); i += kMaxFdsPerMsg) {
        std::vector<int> part(fds.begin() + i, fds.begin() + std::min<size_t>(fds.size(), i + kMaxFdsPerMsg));
        Wire f;
        f.op = kFds;
        rc = send_msg(fd, f, nullptr, part);
    }
    close_all(fds);
    return rc;
}

int reply(int fd, uint32_t op, int status, uint64_t lease = 0, uint64_t a0 = 0, uint64_t a1 = 0, uint64_t a2 = 0,
          uint64_t a3 = 0)
{
    Wire w;
    w.op = op;
    w.status = status;
    w.lease = lease;
    w.arg[0] = a0;
    w.arg[1] = a1;
    w.arg[2] = a2;
    w.arg[3] = a3;
    return send_msg(fd, w, nullptr, {});
}

// A connection ended (disconnect or death): a writer before commit discards the
// incomplete state, a reader releases its lease.
void drop_role(gms_owner *o, Conn &c)
{
    if (c.role == 1) {
        discard(o);
    } else if (c.role == 2) {
        c.role = 0;
        if (readers_of(o) == 0) o->state = GMS_STORE_COMMITTED;
    }
    c.role = 0;
    c.lease = 0;
}

int handle(gms_owner *o, Conn &c, const Wire &w, const std::vector<uint8_t> &payload)
{
    std::lock_guard<std::mutex> lock(o->mu);
    switch (w.op) {
    case kStatus: {
        uint64_t mapped = 0;
        for (auto &kv : o->allocs) mapped += kv.second.size;
        return reply(c.fd, kStatus, GMS_OK, 0, (uint64_t)o->state | ((uint64_t)o->invalid << 8), readers_of(o),
                     o->allocs.size(), mapped);
    }
    case kHelloRW: {
        if (c.role) return reply(c.fd, w.op, GMS_ERR_STATE);
        if (o->state != GMS_STORE_EMPTY && o->state != GMS_STORE_COMMITTED)
            return reply(c.fd, w.op, GMS_ERR_STATE, 0, o->state);
        Out out;
        std::vector<int> fds;
        int rc = export_all(o, out, fds);
        if (rc != GMS_OK) return reply(c.fd, w.op, rc);
        put_layout(o, out);  // from COMMITTED: the layout the writer may repopulate
        c.role = 1;
        c.lease = o->next_lease++;
        o->state = GMS_STORE_RW;
        Wire r;
        r.op = w.op;
        r.lease = c.lease;
        r.arg[0] = (uint64_t)(int64_t)o->device;
        r.arg[1] = o->gran;
        return reply_with_fds(c.fd, r, out, fds);
    }
    case kHelloRO: {
        if (c.role) return reply(c.fd, w.op, GMS_ERR_STATE);
        if (o->state != GMS_STORE_COMMITTED && o->state != GMS_STORE_RO)
            return reply(c.fd, w.op, GMS_ERR_STATE, 0, o->state);
        if (o->invalid) return reply(c.fd, w.op, GMS_ERR_INTEGRITY, 0, o->state);
        Out out;
        std::vector<int> fds;
        int rc = export_all(o, out, fds);
        if (rc != GMS_OK) return reply(c.fd, w.op, rc);
        put_layout(o, out);
        c.role = 2;
        c.lease = o->next_lease++;
        o->state = GMS_STORE_RO;
        Wire r;
        r.op = w.op;
        r.lease = c.lease;
        r.arg[0] = (uint64_t)(int64_t)o->device;
        r.arg[1] = o->gran;
        return reply_with_fds(c.fd, r, out, fds);
    }
    case kAlloc: {
        if (c.role != 1) return reply(c.fd, w.op, GMS_ERR_STATE);
        if (o->device == GMS_HOST_ONLY) return reply(c.fd, w.op, GMS_ERR_STATE);
        const uint64_t bytes = w.arg[0];
        if (bytes == 0) return reply(c.fd, w.op, GMS_ERR_INVALID);
        if (bytes > GMS_IPC_PIECE_BYTES) return reply(c.fd, w.op, GMS_ERR_SIZE);
        OwnedAlloc a;
        a.bytes = bytes;
        a.size = round_up(bytes, o->gran);
        a.flags = w.arg[1] & kAllocSlab;
        hipMemAllocationProp prop = shareable_prop(o->device);
        DeviceGuard g(o->device);
        hipError_t e = hipMemCreate(&a.handle, a.size, &prop, 0);
        if (e != hipSuccess) {
            (void)hipGetLastError();
            return reply(c.fd, w.op, GMS_ERR_NOMEM);
        }
        std::vector<int> fds(1, -1);
        if ((e = export_fd(a.handle, &fds[0])) != hipSuccess) {
            release_alloc(o, a);
            return reply(c.fd, w.op, GMS_ERR_HIP, 0, (uint64_t)e);
        }
        const uint64_t id = o->next_alloc++;
        Out out;
        out.put(id);
        out.put(a.bytes);
        out.put(a.size);
        out.put(a.flags);
        o->allocs[id] = a;
        Wire r;
        r.op = w.op;
        r.lease = c.lease;
        r.arg[0] = id;
        return reply_with_fds(c.fd, r, out, fds);
    }
    case kFree: {
        if (c.role != 1) return reply(c.fd, w.op, GMS_ERR_STATE);
        auto it = o->allocs.find(w.arg[0]);
        if (it == o->allocs.end()) return reply(c.fd, w.op, GMS_ERR_INVALID);
        release_alloc(o, it->second);
        o->allocs.erase(it);
        return reply(c.fd, w.op, GMS_OK);
    }
    case kCommit: {
        if (c.role != 1) return reply(c.fd, w.op, GMS_ERR_STATE);
        In in(payload);
        uint64_t n = 0, nh = 0;
        std::vector<LayoutRec> lay;
        if (!in.get(n) || n > (payload.size() / sizeof(LayoutRec))) return reply(c.fd, w.op, GMS_ERR_INVALID);
        lay.resize(n);
        if (!in.get_raw(lay.data(), n * sizeof(LayoutRec))) return reply(c.fd, w.op, GMS_ERR_INVALID);
        if (!in.get(nh) || nh > payload.size() / 8) return reply(c.fd, w.op, GMS_ERR_INVALID);
        std::vector<uint64_t> hs(nh);
        if (!in.get_raw(hs.data(), nh * 8)) return reply(c.fd, w.op, GMS_ERR_INVALID);
        uint64_t blocks = 0;
        for (const LayoutRec &r : lay) {
            auto it = o->allocs.find(r.alloc);
            if (r.nbytes && (it == o->allocs.end() || r.off + r.nbytes > it->second.bytes || r.off + r.nbytes < r.off))
                return reply(c.fd, w.op, GMS_ERR_INVALID);
            blocks += gms::ceil_div(r.nbytes, GMS_BLOCK_BYTES);
        }
        if (blocks != nh) return reply(c.fd, w.op, GMS_ERR_INVALID);
        o->layout.swap(lay);
        o->hashes.swap(hs);
        o->invalid = false;
        o->state = GMS_STORE_COMMITTED;
        c.role = 0;  // the write lease ends at commit
        c.lease = 0;
        return reply(c.fd, w.op, GMS_OK);
    }
    case kAbort: {
        if (c.role != 1) return reply(c.fd, w.op, GMS_ERR_STATE);
        drop_role(o, c);
        return reply(c.fd, w.op, GMS_OK);
    }
    case kInvalidate: {
        if (c.role != 2) return reply(c.fd, w.op, GMS_ERR_STATE);
        o->invalid = true;
        if (w.arg[0]) drop_role(o, c);  // the reader's lease is refused
        return reply(c.fd, w.op, GMS_OK);
    }
    case kBye: {
        drop_role(o, c);
        return reply(c.fd, w.op, GMS_OK);
    }
    default:
        return reply(c.fd, w.op, GMS_ERR_INVALID);
    }
}

}  // namespace

extern "C" {

int gms_owner_create(const char *socket_path, int device, gms_owner **out)
{
    gms::clear_error();
    if (!out) return fail(GMS_ERR_INVALID, "out is null");
    *out = nullptr;
    struct sockaddr_un sa = {};
    if (!socket_path || !*socket_path || strlen(socket_path) >= sizeof sa.sun_path)
        return fail(GMS_ERR_INVALID, "socket path is empty or longer than %zu bytes", sizeof sa.sun_path - 1);
    gms_owner *o = new (std::nothrow) gms_owner;
    if (!o) return fail(GMS_ERR_NOMEM, "owner");
    o->device = device;
    o->path = socket_path;
    if (device != GMS_HOST_ONLY) {
        DeviceGuard g(device);
        if (g.err != hipSuccess) {
            delete o;
            return fail_hip(g.err, "hipSetDevice");
        }
        size_t gran = 0;
        hipMemAllocationProp prop = shareable_prop(device);
        hipError_t e = hipMemGetAllocationGranularity(&gran, &prop, hipMemAllocationGranularityMinimum);
        if (e != hipSuccess || gran == 0) {
            delete o;
            return e != hipSuccess ? fail_hip(e, "hipMemGetAllocationGranularity")
                                   : fail(GMS_ERR_STATE, "device %d has no VMM support", device);
        }
        o->gran = gran;
    }
    o->listen_fd = socket(AF_UNIX, SOCK_STREAM | SOCK_CLOEXEC, 0);
    if (o->listen_fd < 0 || pipe2(o->wake, O_CLOEXEC | O_NONBLOCK) != 0) {
        const int err = errno;
        gms_owner_destroy(o);
        return fail(GMS_ERR_IO, "socket/pipe: %s", strerror(err));
    }
    sa.sun_family = AF_UNIX;
    strcpy(sa.sun_path, socket_path);
    unlink(socket_path);
    if (bind(o->listen_fd, (struct sockaddr *)&sa, sizeof sa) != 0 || listen(o->listen_fd, 64) != 0) {
        const int err = errno;
        o->path.clear();  // not ours to unlink
        gms_owner_destroy(o);
        return fail(GMS_ERR_IO, "bind/listen(%s): %s", socket_path, strerror(err));
    }
    *out = o;
    return GMS_OK;
}

int gms_owner_run(gms_owner *o)
{
    gms::clear_error();
    if (!o) return fail(GMS_ERR_INVALID, "owner is null");
    while (!o->stop.load()) {
        std::vector<struct pollfd> pf;
        pf.push_back({o->wake[0], POLLIN, 0});
        pf.push_back({o->listen_fd, POLLIN, 0});
        for (const Conn &c : o->conns) pf.push_back({c.fd, POLLIN, 0});
        int k = poll(pf.data(), pf.size(), 1000);
        if (k < 0 && errno == EINTR) continue;
        if (k < 0) return fail(GMS_ERR_IO, "poll: %s", strerror(errno));
        if (pf[0].revents) break;
        std::vector<int> gone;
        for (size_t i = 2; i < pf.size(); ++i) {
            if (!pf[i].revents) continue;
            Conn &c = o->conns[i - 2];
            Wire w;
            std::vector<uint8_t> payload;
            std::vector<int> fds;
            const bool ok = (pf[i].revents & POLLIN) && recv_msg(c.fd, w, payload, fds) == 0;
            close_all(fds);  // clients send no descriptors
            if (!ok || handle(o, c, w, payload) != 0 || w.op == kBye) gone.push_back(c.fd);
        }
        for (int fd : gone) {
            std::lock_guard<std::mutex> lock(o->mu);
            auto it = std::find_if(o->conns.begin(), o->conns.end(), [fd](const Conn &c) { return c.fd == fd; });
            if (it == o->conns.end()) continue;
            drop_role(o, *it);
            close(it->fd);
            o->conns.erase(it);
        }
        if (pf[1].revents & POLLIN) {
            int fd = accept4(o->listen_fd, nullptr, nullptr, SOCK_CLOEXEC);
            if (fd >= 0) {
                struct timeval tv = {30, 0};  // a stalled peer cannot hold the owner longer
                setsockopt(fd, SOL_SOCKET, SO_RCVTIMEO, &tv, sizeof tv);
                setsockopt(fd, SOL_SOCKET, SO_SNDTIMEO, &tv, sizeof tv);
                Conn c;
                c.fd = fd;
                std::lock_guard<std::mutex> lock(o->mu);
                o->conns.push_back(c);
            }
        }
    }
    return GMS_OK;
}

void gms_owner_stop(gms_owner *o)
{
    if (!o) return;
    o->stop.store(true);
    const char b = 1;
    (void)!write(o->wake[1], &b, 1);
}

int gms_owner_status(gms_owner *o, int *state, uint32_t *readers, int *invalid, uint64_t *allocations)
{
    if (!o) return fail(GMS_ERR_INVALID, "owner is null");
    std::lock_guard<std::mutex> lock(o->mu);
    if (state) *state = o->state;
    if (readers) *readers = readers_of(o);
    if (invalid) *invalid = o->invalid ? 1 : 0;
    if (allocations) *allocations = o->allocs.size();
    return GMS_OK;
}

void gms_owner_destroy(gms_owner *o)
{
    if (!o) return;
    for (Conn &c : o->conns) close(c.fd);
    o->conns.clear();
    discard(o);
    if (o->listen_fd >= 0) close(o->listen_fd);
    for (int f : o->wake)
        if (f >= 0) close(f);
    if (!o->path.empty()) unlink(o->path.c_str());
    delete o;
}

}  // extern "C"

// ===================================================================== client

namespace {

struct ClientAlloc {
    uint64_t id = 0, bytes = 0, size = 0;
    uint64_t va = 0;                     // the mapping of the owner's memory in this process
    hipExternalMemory_t ext = nullptr;
    bool slab = false;                   // suballocated by the writer (first fit)
    std::map<uint64_t, uint64_t> free;   // slab: offset -> bytes, coalesced
    std::map<uint64_t, uint64_t> parts;  // slab: offset -> bytes handed out
};

}  // namespace

struct gms_client {
    int fd = -1;
    int mode = 0;  // GMS_LEASE_RW or GMS_LEASE_RO
    bool leased = false;
    uint64_t lease = 0;
    int device = GMS_HOST_ONLY;
    uint64_t gran = 4096;
    std::map<uint64_t, ClientAlloc> allocs;  // by id
    std::vector<gms_entry> layout;           // committed entries at this process's addresses
    gms_manifest *m = nullptr;               // manifest over `layout`
    uint64_t *d_hash = nullptr;              // commit-time block hashes (device)
    uint64_t *d_count = nullptr;
};

namespace {

void unmap(gms_client *c, ClientAlloc &a)
{
    if (c->device == GMS_HOST_ONLY) return;
    if (a.va) (void)hipFree((void *)(uintptr_t)a.va);
    if (a.ext) (void)hipDestroyExternalMemory(a.ext);
    a.va = 0;
    a.ext = nullptr;
}

// Maps the owner's allocation behind descriptor `fd` as external memory.  The
// descriptor stays the caller's (the runtime keeps its own reference).
int map_alloc(gms_client *c, ClientAlloc &a, int fd)
{
    hipExternalMemoryHandleDesc d = {};
    d.type = hipExternalMemoryHandleTypeOpaqueFd;
    d.handle.fd = fd;
    d.size = a.size;
    hipError_t e = hipImportExternalMemory(&a.ext, &d);
    if (e != hipSuccess) {
        a.ext = nullptr;
        return fail_hip(e, "hipImportExternalMemory");
    }
    hipExternalMemoryBufferDesc bd = {};
    bd.offset = 0;
    bd.size = a.size;
    void *va = nullptr;
    if ((e = hipExternalMemoryGetMappedBuffer(&va, a.ext, &bd)) != hipSuccess) {
        (void)hipDestroyExternalMemory(a.ext);
        a.ext = nullptr;
        return fail_hip(e, "hipExternalMemoryGetMappedBuffer");
    }
    a.va = (uint64_t)(uintptr_t)va;
    return GMS_OK;
}

// Reads an allocation table {count, then id, bytes, size, flags each} and maps every
// allocation, taking the descriptors from `fds` in order (more arrive in kFds
// messages when needed).
int map_table(gms_client *c, In &in, std::vector<int> &fds, uint64_t nfds)
{
    while (fds.size() < nfds) {
        Wire w;
        std::vector<uint8_t> pl;
        if (recv_msg(c->fd, w, pl, fds) != 0 || w.op != kFds) return fail(GMS_ERR_IO, "owner closed the connection");
    }
    uint64_t n = 0;
    if (!in.get(n) || n > fds.size()) return fail(GMS_ERR_IO, "short reply from the owner");
    for (uint64_t i = 0; i < n; ++i) {
        ClientAlloc a;
        uint64_t flags = 0;
        if (!in.get(a.id) || !in.get(a.bytes) || !in.get(a.size) || !in.get(flags) || a.bytes > a.size)
            return fail(GMS_ERR_IO, "short reply from the owner");
        a.slab = (flags & kAllocSlab) != 0;
        if (c->device != GMS_HOST_ONLY) {
            int rc = map_alloc(c, a, fds[i]);
            if (rc != GMS_OK) return rc;
        }
        c->allocs[a.id] = a;
    }
    return GMS_OK;
}

int request(gms_client *c, Wire w, const Out *payload, Wire &r, std::vector<uint8_t> &rp, std::vector<int> &fds)
{
    w.lease = c->lease;
    w.payload = payload ? payload->b.size() : 0;
    if (send_msg(c->fd, w, payload ? payload->b.data() : nullptr, {}) != 0 || recv_msg(c->fd, r, rp, fds) != 0)
        return fail(GMS_ERR_IO, "owner connection lost");
    return GMS_OK;
}

void teardown(gms_client *c)
{
    if (c->device != GMS_HOST_ONLY) {
        DeviceGuard g(c->device);
        (void)hipDeviceSynchronize();  // no kernel of this process still uses the mappings
        if (c->m) gms_manifest_destroy(c->m);
        if (c->d_hash) (void)hipFree(c->d_hash);
        if (c->d_count) (void)hipFree(c->d_count);
        for (auto &kv : c->allocs) unmap(c, kv.second);
    }
    c->m = nullptr;
    c->d_hash = c->d_count = nullptr;
    c->allocs.clear();
    c->layout.clear();
}

// Forgets the committed layout (its manifest and hashes): a writer that frees memory the
// layout uses no longer has it whole.
void drop_committed(gms_client *c)
{
    if (c->device != GMS_HOST_ONLY) {
        DeviceGuard g(c->device);
        (void)hipDeviceSynchronize();
        if (c->m) gms_manifest_destroy(c->m);
        if (c->d_hash) (void)hipFree(c->d_hash);
    }
    c->m = nullptr;
    c->d_hash = nullptr;
    c->layout.clear();
}

bool layout_touches(const gms_client *c, uint64_t lo, uint64_t hi)
{
    for (const gms_entry &e : c->layout)
        if (e.nbytes && e.addr < hi && e.addr + e.nbytes > lo) return true;
    return false;
}

// A writer that took over committed state: the parts of its slabs are the
// committed entries in them (rounded up to the default alignment, short of the
// next entry), the rest is free.
void rebuild_slabs(gms_client *c)
{
    for (auto &kv : c->allocs) {
        ClientAlloc &a = kv.second;
        if (!a.slab) continue;
        a.parts.clear();
        a.free.clear();
        std::map<uint64_t, uint64_t> in;  // offset -> bytes of the entries in this slab
        for (const gms_entry &e : c->layout)
            if (e.nbytes && e.addr >= a.va && e.addr < a.va + a.bytes) in[e.addr - a.va] = e.nbytes;
        for (auto it = in.begin(); it != in.end(); ++it) {
            auto nx = std::next(it);
            const uint64_t end = nx == in.end() ? a.bytes : nx->first;  // entries do not overlap
            a.parts[it->first] = std::min(round_up(it->second, 256), end - it->first);
        }
        uint64_t at = 0;
        for (const auto &p : a.parts) {
            if (p.first > at) a.free[at] = p.first - at;
            at = std::max(at, p.first + p.second);
        }
        if (a.bytes > at) a.free[at] = a.bytes - at;
    }
}

// Verify the mapped state against the commit-time hashes.
int verify_state(gms_client *c, uint64_t *count, uint64_t *list, uint64_t cap, void *stream)
{
    *count = 0;
    if (!c->m || gms_num_blocks(c->m) == 0) return GMS_OK;
    int rc = gms::refuse_capture((hipStream_t)stream, "a client verification");
    if (rc != GMS_OK) return rc;
    rc = gms_verify(c->m, c->d_hash, nullptr, nullptr, c->d_count, list, list ? cap : 0, stream);
    if (rc != GMS_OK) return rc;
    hipError_t e = hipMemcpyAsync(count, c->d_count, 8, hipMemcpyDeviceToHost, (hipStream_t)stream);
    if (e == hipSuccess) e = hipStreamSynchronize((hipStream_t)stream);
    return e == hipSuccess ? GMS_OK : fail_hip(e, "client verification");
}

}  // namespace

extern "C" {

int gms_client_connect(const char *socket_path, int mode, uint32_t flags, void *stream, gms_client **out,
                       uint64_t *mismatch_count_out)
{
    gms::clear_error();
    if (mismatch_count_out) *mismatch_count_out = 0;
    if (!out) return fail(GMS_ERR_INVALID, "out is null");
    *out = nullptr;
    if (mode != GMS_LEASE_RW && mode != GMS_LEASE_RO) return fail(GMS_ERR_INVALID, "mode %d", mode);
    if (flags & ~(uint32_t)GMS_CONNECT_VERIFY) return fail(GMS_ERR_INVALID, "flags %#x", flags);
    gms_client *c = new (std::nothrow) gms_client;
    if (!c) return fail(GMS_ERR_NOMEM, "client");
    int rc = connect_to(socket_path, &c->fd);
    if (rc != GMS_OK) {
        delete c;
        return rc;
    }
    c->mode = mode;
    Wire w, r;
    w.op = mode == GMS_LEASE_RW ? kHelloRW : kHelloRO;
    w.arg[0] = (uint64_t)getpid();
    std::vector<uint8_t> rp;
    std::vector<int> fds;
    if ((rc = request(c, w, nullptr, r, rp, fds)) != GMS_OK || (rc = r.status) != GMS_OK) {
        close_all(fds);
        if (rc == r.status && rc != GMS_OK)
            fail(rc, "owner refused the %s lease (state %llu)", mode == GMS_LEASE_RW ? "read-write" : "read-only",
                 (unsigned long long)r.arg[0]);
        close(c->fd);
        delete c;
        return rc;
    }
    c->leased = true;
    c->lease = r.lease;
    c->device = (int)(int64_t)r.arg[0];
    c->gran = r.arg[1];
    In in(rp);
    {
        std::optional<DeviceGuard> g;  // a host-only owner: no HIP call at all
        if (c->device != GMS_HOST_ONLY && g.emplace(c->device).err != hipSuccess) rc = fail_hip(g->err, "hipSetDevice");
        if (rc == GMS_OK) rc = map_table(c, in, fds, r.arg[3]);
        close_all(fds);
        if (rc == GMS_OK) {
            uint64_t n = 0, nh = 0;
            std::vector<LayoutRec> lay;
            bool ok = in.get(n) && n <= rp.size() / sizeof(LayoutRec);
            if (ok) {
                lay.resize(n);
                ok = in.get_raw(lay.data(), n * sizeof(LayoutRec)) && in.get(nh) && nh <= rp.size() / 8;
            }
            std::vector<uint64_t> hs(ok ? nh : 0);
            if (ok) ok = in.get_raw(hs.data(), nh * 8);
            if (!ok) rc = fail(GMS_ERR_IO, "short layout from the owner");
            for (size_t i = 0; rc == GMS_OK && i < lay.size(); ++i) {
                auto it = c->allocs.find(lay[i].alloc);
                if (lay[i].nbytes && it == c->allocs.end())
                    rc = fail(GMS_ERR_IO, "layout names an unknown allocation");
                else
                    c->layout.push_back(gms_entry{lay[i].nbytes ? it->second.va + lay[i].off : 0, lay[i].nbytes});
            }
            if (rc == GMS_OK && c->device != GMS_HOST_ONLY && !lay.empty()) {
                if ((rc = gms::manifest_create(c->layout.data(), c->layout.size(), c->device, 0, false, &c->m)) == GMS_OK &&
                    gms_num_blocks(c->m) != hs.size())
                    rc = fail(GMS_ERR_IO, "owner's hashes do not match the layout");
                hipError_t e = hipSuccess;
                if (rc == GMS_OK) e = hipMalloc((void **)&c->d_hash, std::max<size_t>(hs.size(), 1) * 8);
                if (rc == GMS_OK && e == hipSuccess) e = hipMalloc((void **)&c->d_count, 8);
                if (rc == GMS_OK && e == hipSuccess && !hs.empty())
                    e = hipMemcpy(c->d_hash, hs.data(), hs.size() * 8, hipMemcpyHostToDevice);
                if (rc == GMS_OK && e != hipSuccess) rc = fail_hip(e, "commit-time hashes");
                uint64_t count = 0;
                if (rc == GMS_OK && mode == GMS_LEASE_RO && (flags & GMS_CONNECT_VERIFY))
                    rc = verify_state(c, &count, nullptr, 0, stream);
                if (rc == GMS_OK && count) {
                    if (mismatch_count_out) *mismatch_count_out = count;
                    Wire iv, ir;
                    iv.op = kInvalidate;
                    iv.arg[0] = 1;  // and refuse this reader's lease
                    std::vector<uint8_t> ip;
                    std::vector<int> ifd;
                    (void)request(c, iv, nullptr, ir, ip, ifd);
                    close_all(ifd);
                    c->leased = false;
                    rc = fail(GMS_ERR_INTEGRITY, "%llu committed blocks changed; read-only lease refused",
                              (unsigned long long)count);
                }
            }
        }
    }
    if (rc != GMS_OK) {
        teardown(c);
        close(c->fd);  // the owner ends the lease with the connection
        delete c;
        return rc;
    }
    if (mode == GMS_LEASE_RW) rebuild_slabs(c);
    *out = c;
    return GMS_OK;
}

int gms_client_lease(const gms_client *c, uint64_t *lease_out, int *device_out)
{
    if (!c) return fail(GMS_ERR_INVALID, "client is null");
    if (lease_out) *lease_out = c->leased ? c->lease : 0;
    if (device_out) *device_out = c->device;
    return GMS_OK;
}

int gms_client_alloc(gms_client *c, uint64_t bytes, uint64_t align, uint64_t *addr_out)
{
    gms::clear_error();
    if (!c || !addr_out) return fail(GMS_ERR_INVALID, "client or addr_out is null");
    if (c->mode != GMS_LEASE_RW || !c->leased) return fail(GMS_ERR_STATE, "only a connected writer allocates");
    if (c->device == GMS_HOST_ONLY) return fail(GMS_ERR_STATE, "the owner has no device memory");
    if (bytes == 0) return fail(GMS_ERR_INVALID, "zero bytes");
    if (align == 0) align = 256;
    if (align & (align - 1) || align > c->gran) return fail(GMS_ERR_INVALID, "align %llu", (unsigned long long)align);
    const uint64_t need = round_up(bytes, align);
    if (need > GMS_IPC_PIECE_BYTES)
        return fail(GMS_ERR_SIZE, "%llu bytes exceed the largest shared allocation (%llu)", (unsigned long long)need,
                    (unsigned long long)GMS_IPC_PIECE_BYTES);
    // requests up to half a slab: first fit in the slabs already held
    const bool slab = need <= GMS_IPC_PIECE_BYTES / 2;
    for (auto &kv : c->allocs) {
        ClientAlloc &a = kv.second;
        if (!slab || !a.slab) continue;
        for (auto f = a.free.begin(); f != a.free.end(); ++f) {
            const uint64_t off = round_up(f->first, align);
            if (off + need > f->first + f->second) continue;
            const uint64_t lo = f->first, len = f->second;
            a.free.erase(f);
            if (off > lo) a.free[lo] = off - lo;
            if (lo + len > off + need) a.free[off + need] = lo + len - off - need;
            a.parts[off] = need;
            *addr_out = a.va + off;
            return GMS_OK;
        }
    }
    // a new allocation from the owner: a slab of GMS_IPC_PIECE_BYTES, or one of its own
    Wire w, r;
    w.op = kAlloc;
    w.arg[0] = slab ? GMS_IPC_PIECE_BYTES : need;
    w.arg[1] = slab ? kAllocSlab : 0;
    std::vector<uint8_t> rp;
    std::vector<int> fds;
    int rc = request(c, w, nullptr, r, rp, fds);
    if (rc == GMS_OK && r.status != GMS_OK)
        rc = fail(r.status, "owner refused an allocation of %llu bytes", (unsigned long long)w.arg[0]);
    if (rc != GMS_OK) {
        close_all(fds);
        return rc;
    }
    DeviceGuard g(c->device);
    Out one;
    one.put((uint64_t)1);
    one.b.insert(one.b.end(), rp.begin(), rp.end());
    In in(one.b);
    rc = map_table(c, in, fds, r.arg[3]);
    close_all(fds);
    if (rc != GMS_OK) return rc;
    auto it = c->allocs.find(r.arg[0]);
    if (it == c->allocs.end()) return fail(GMS_ERR_IO, "owner sent no allocation");
    ClientAlloc &a = it->second;
    a.slab = slab;
    if (slab) {
        a.parts[0] = need;
        if (a.bytes > need) a.free[need] = a.bytes - need;
    }
    *addr_out = a.va;
    return GMS_OK;
}

int gms_client_free(gms_client *c, uint64_t addr)
{
    gms::clear_error();
    if (!c) return fail(GMS_ERR_INVALID, "client is null");
    if (c->mode != GMS_LEASE_RW || !c->leased) return fail(GMS_ERR_STATE, "only a connected writer frees");
    for (auto &kv : c->allocs) {
        ClientAlloc &a = kv.second;
        if (addr < a.va || addr >= a.va + a.bytes) continue;
        if (a.slab) {
            auto p = a.parts.find(addr - a.va);
            if (p == a.parts.end()) break;
            uint64_t off = p->first, len = p->second;
            if (layout_touches(c, a.va + off, a.va + off + len)) drop_committed(c);
            a.parts.erase(p);
            auto nx = a.free.lower_bound(off);
            if (nx != a.free.end() && nx->first == off + len) {
                len += nx->second;
                nx = a.free.erase(nx);
            }
            if (nx != a.free.begin()) {
                auto pv = std::prev(nx);
                if (pv->first + pv->second == off) {
                    pv->second += len;
                    return GMS_OK;
                }
            }
            a.free[off] = len;
            return GMS_OK;
        }
        if (addr != a.va) break;
        const uint64_t id = kv.first;
        if (layout_touches(c, a.va, a.va + a.bytes)) drop_committed(c);
        {
            DeviceGuard g(c->device);
            (void)hipDeviceSynchronize();
            unmap(c, a);
        }
        c->allocs.erase(id);
        Wire w, r;
        w.op = kFree;
        w.arg[0] = id;
        std::vector<uint8_t> rp;
        std::vector<int> fds;
        int rc = request(c, w, nullptr, r, rp, fds);
        close_all(fds);
        return rc != GMS_OK ? rc : r.status != GMS_OK ? fail(r.status, "owner refused the free") : GMS_OK;
    }
    return fail(GMS_ERR_INVALID, "%#llx is not an allocation of this client", (unsigned long long)addr);
}

int gms_client_commit(gms_client *c, const gms_entry *entries, uint64_t n, const uint64_t *expected_blk,
                      uint64_t *mismatch_count_out, void *stream)
{
    gms::clear_error();
    if (mismatch_count_out) *mismatch_count_out = 0;
    if (!c) return fail(GMS_ERR_INVALID, "client is null");
    if (c->mode != GMS_LEASE_RW || !c->leased) return fail(GMS_ERR_STATE, "only a connected writer commits");
    if (n && !entries) return fail(GMS_ERR_INVALID, "entries is null");
    if (c->device == GMS_HOST_ONLY && (n || expected_blk))
        return fail(GMS_ERR_STATE, "the owner has no device memory: commit takes no entries");
    Out out;
    out.put(n);
    for (uint64_t i = 0; i < n; ++i) {
        LayoutRec rec = {0, 0, entries[i].nbytes};
        bool found = entries[i].nbytes == 0;
        for (auto &kv : c->allocs) {
            const ClientAlloc &a = kv.second;
            if (entries[i].addr >= a.va && entries[i].addr + entries[i].nbytes <= a.va + a.bytes &&
                entries[i].addr + entries[i].nbytes >= entries[i].addr && entries[i].nbytes) {
                rec.alloc = kv.first;
                rec.off = entries[i].addr - a.va;
                found = true;
                break;
            }
        }
        if (!found)
            return fail(GMS_ERR_INVALID, "entry %llu [%#llx, +%llu) is not inside one allocation of the owner",
                        (unsigned long long)i, (unsigned long long)entries[i].addr,
                        (unsigned long long)entries[i].nbytes);
        out.put(rec);
    }
    std::vector<uint64_t> hs;
    if (c->device != GMS_HOST_ONLY && n) {
        DeviceGuard g(c->device);
        gms_manifest *m = nullptr;
        int rc = gms::manifest_create(entries, n, c->device, 0, false, &m);  // entries checked above
        if (rc != GMS_OK) return rc;
        // every device write of this process, on any stream, lands before it is hashed
        hipError_t e = hipDeviceSynchronize();
        if (e != hipSuccess) {
            gms_manifest_destroy(m);
            return fail_hip(e, "hipDeviceSynchronize");
        }
        const uint64_t nb = gms_num_blocks(m);
        uint64_t *d = nullptr, *cnt = nullptr;
        e = hipMalloc((void **)&d, std::max<uint64_t>(nb, 1) * 8);
        if (e == hipSuccess) e = hipMalloc((void **)&cnt, 8);
        if (e != hipSuccess) {
            (void)hipGetLastError();
            if (d) (void)hipFree(d);
            gms_manifest_destroy(m);
            return fail(GMS_ERR_NOMEM, "commit hashes");
        }
        uint64_t count = 0;
        rc = gms::refuse_capture((hipStream_t)stream, "a commit");
        if (rc == GMS_OK && nb)
            rc = gms_verify(m, expected_blk, d, nullptr, expected_blk ? cnt : nullptr, nullptr, 0, stream);
        hs.resize(nb);
        if (rc == GMS_OK && nb) e = hipMemcpyAsync(hs.data(), d, nb * 8, hipMemcpyDeviceToHost, (hipStream_t)stream);
        if (rc == GMS_OK && nb && expected_blk && e == hipSuccess)
            e = hipMemcpyAsync(&count, cnt, 8, hipMemcpyDeviceToHost, (hipStream_t)stream);
        if (rc == GMS_OK && e == hipSuccess) e = hipStreamSynchronize((hipStream_t)stream);
        if (rc == GMS_OK && e != hipSuccess) rc = fail_hip(e, "commit hashes");
        (void)hipFree(d);
        (void)hipFree(cnt);
        gms_manifest_destroy(m);
        if (rc != GMS_OK) return rc;
        if (count) {
            if (mismatch_count_out) *mismatch_count_out = count;
            return fail(GMS_ERR_INTEGRITY, "%llu blocks differ from the expected hashes; commit refused",
                        (unsigned long long)count);
        }
    }
    out.put((uint64_t)hs.size());
    out.put_raw(hs.data(), hs.size() * 8);
    Wire w, r;
    w.op = kCommit;
    std::vector<uint8_t> rp;
    std::vector<int> fds;
    int rc = request(c, w, &out, r, rp, fds);
    close_all(fds);
    if (rc != GMS_OK) return rc;
    if (r.status != GMS_OK) return fail(r.status, "owner refused the commit");
    c->leased = false;  // the write lease ends at commit
    drop_committed(c);  // the layout it took over is gone; a read-only reconnect gets the new one
    return GMS_OK;
}

int gms_client_abort(gms_client *c)
{
    gms::clear_error();
    if (!c) return fail(GMS_ERR_INVALID, "client is null");
    if (c->mode != GMS_LEASE_RW || !c->leased) return fail(GMS_ERR_STATE, "only a connected writer aborts");
    teardown(c);  // unmapped before the owner releases the memory
    Wire w, r;
    w.op = kAbort;
    std::vector<uint8_t> rp;
    std::vector<int> fds;
    int rc = request(c, w, nullptr, r, rp, fds);
    close_all(fds);
    c->leased = false;
    return rc != GMS_OK ? rc : r.status != GMS_OK ? fail(r.status, "owner refused the abort") : GMS_OK;
}

int gms_client_layout(const gms_client *c, gms_entry *entries_out, uint64_t cap, uint64_t *n_out)
{
    if (!c) return fail(GMS_ERR_INVALID, "client is null");
    if (n_out) *n_out = c->layout.size();
    if (entries_out)
        for (uint64_t i = 0; i < std::min<uint64_t>(cap, c->layout.size()); ++i) entries_out[i] = c->layout[i];
    return GMS_OK;
}

const gms_manifest *gms_client_manifest(const gms_client *c) { return c ? c->m : nullptr; }

int gms_client_manifest_create(const gms_client *c, const gms_entry *entries, uint64_t n, uint64_t chunk_bytes,
                               gms_manifest **out)
{
    gms::clear_error();
    if (!c || !out) return fail(GMS_ERR_INVALID, "client or out is null");
    *out = nullptr;
    if (n && !entries) return fail(GMS_ERR_INVALID, "entries is null");
    if (c->device == GMS_HOST_ONLY) return fail(GMS_ERR_STATE, "the owner has no device memory");
    for (uint64_t i = 0; i < n; ++i) {
        const gms_entry &e = entries[i];
        if (!e.nbytes) continue;
        bool inside = false;
        for (const auto &kv : c->allocs) {
            const ClientAlloc &a = kv.second;
            if (e.addr >= a.va && e.addr + e.nbytes >= e.addr && e.addr + e.nbytes <= a.va + a.bytes) {
                inside = true;
                break;
            }
        }
        if (!inside)
            return fail(GMS_ERR_INVALID, "entry %llu [%#llx, +%llu) is not inside one allocation of this client",
                        (unsigned long long)i, (unsigned long long)e.addr, (unsigned long long)e.nbytes);
    }
    return gms::manifest_create(entries, n, c->device, chunk_bytes, false, out);
}

const uint64_t *gms_client_block_hashes(const gms_client *c) { return c ? c->d_hash : nullptr; }

int gms_client_verify(gms_client *c, uint64_t *mismatch_count_out, uint64_t *mismatch_list_out, uint64_t cap,
                      void *stream)
{
    gms::clear_error();
    if (!c || !mismatch_count_out) return fail(GMS_ERR_INVALID, "client or mismatch_count_out is null");
    *mismatch_count_out = 0;
    if (c->mode != GMS_LEASE_RO || !c->leased) return fail(GMS_ERR_STATE, "only a connected reader verifies");
    if (c->device == GMS_HOST_ONLY) return GMS_OK;
    DeviceGuard g(c->device);
    int rc = verify_state(c, mismatch_count_out, mismatch_list_out, cap, stream);
    if (rc != GMS_OK || *mismatch_count_out == 0) return rc;
    Wire w, r;  // integrity errors invalidate the committed state; this reader keeps its lease
    w.op = kInvalidate;
    std::vector<uint8_t> rp;
    std::vector<int> fds;
    rc = request(c, w, nullptr, r, rp, fds);
    close_all(fds);
    return rc;
}

int gms_client_disconnect(gms_client *c)
{
    gms::clear_error();
    if (!c) return GMS_OK;
    teardown(c);  // unmapped before a writer's abort releases the memory
    int rc = GMS_OK;
    if (c->fd >= 0) {
        Wire w, r;
        w.op = kBye;
        std::vector<uint8_t> rp;
        std::vector<int> fds;
        rc = request(c, w, nullptr, r, rp, fds);
        close_all(fds);
        close(c->fd);
    }
    delete c;
    return rc;
}

int gms_owner_query(const char *socket_path, int *state, uint32_t *readers, int *invalid, uint64_t *allocations)
{
    gms::clear_error();
    int fd = -1;
    int rc = connect_to(socket_path, &fd);
    if (rc != GMS_OK) return rc;
    Wire w, r;
    w.op = kStatus;
    std::vector<uint8_t> rp;
    std::vector<int> fds;
    if (send_msg(fd, w, nullptr, {}) != 0 || recv_msg(fd, r, rp, fds) != 0) rc = fail(GMS_ERR_IO, "owner query");
    close_all(fds);
    close(fd);
    if (rc != GMS_OK) return rc;
    if (state) *state = (int)(r.arg[0] & 0xFF);
    if (invalid) *invalid = (int)((r.arg[0] >> 8) & 1);
    if (readers) *readers = (uint32_t)r.arg[1];
    if (allocations) *allocations = r.arg[2];
    return GMS_OK;
}

}  // extern "C"
