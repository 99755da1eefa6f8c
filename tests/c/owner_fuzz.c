/*
 * The owner process's message handling against hostile peers, built with the
 * library under AddressSanitizer/UndefinedBehaviorSanitizer by a CPU test: a
 * host-only owner runs in a thread while this program connects thousands of
 * times with random bytes, headers with random operations and lengths (most
 * announcing more payload than they send), descriptors passed with them, and
 * random commit payloads from a connection that holds the write lease; valid
 * clients of the C-ABI run the protocol in between; then random calls with
 * random leases on a host-only in-process store.  Exits non-zero on any
 * failed check; the sanitizers abort on any memory or UB error.
 */
#define _GNU_SOURCE
#include <poll.h>
#include <pthread.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>
#include <sys/socket.h>
#include <sys/un.h>
#include <unistd.h>

#include "gms.h"

#define CHECK(c)                                                                    \
    do {                                                                            \
        if (!(c)) {                                                                 \
            fprintf(stderr, "%s:%d: check failed: %s\n", __FILE__, __LINE__, #c);   \
            exit(1);                                                                \
        }                                                                           \
    } while (0)

/* The message header on the socket: magic, operation, status, descriptor count,
 * lease, four arguments, payload length (64 bytes, little-endian). */
enum { HDR = 64, OFF_OP = 4, OFF_ARG = 24, OFF_PAYLOAD = 56 };
static const uint32_t kMagic = 0x31534D47u;

static uint64_t rng_state = 0x9E3779B97F4A7C15ull;
static uint64_t rnd(void)
{
    rng_state ^= rng_state << 13;
    rng_state ^= rng_state >> 7;
    rng_state ^= rng_state << 17;
    return rng_state;
}

static void *run_owner(void *o)
{
    CHECK(gms_owner_run((gms_owner *)o) == GMS_OK);
    return NULL;
}

static int dial(const char *path)
{
    struct sockaddr_un sa;
    memset(&sa, 0, sizeof sa);
    sa.sun_family = AF_UNIX;
    strncpy(sa.sun_path, path, sizeof sa.sun_path - 1);
    int fd = socket(AF_UNIX, SOCK_STREAM, 0);
    CHECK(fd >= 0);
    CHECK(connect(fd, (struct sockaddr *)&sa, sizeof sa) == 0);
    return fd;
}

/* Sends n bytes, with one descriptor attached when pass_fd >= 0. */
static void send_bytes(int fd, const uint8_t *b, size_t n, int pass_fd)
{
    struct iovec iov = {(void *)b, n};
    struct msghdr mh;
    memset(&mh, 0, sizeof mh);
    mh.msg_iov = &iov;
    mh.msg_iovlen = 1;
    char ctl[CMSG_SPACE(sizeof(int))];
    if (pass_fd >= 0) {
        memset(ctl, 0, sizeof ctl);
        mh.msg_control = ctl;
        mh.msg_controllen = sizeof ctl;
        struct cmsghdr *c = CMSG_FIRSTHDR(&mh);
        c->cmsg_level = SOL_SOCKET;
        c->cmsg_type = SCM_RIGHTS;
        c->cmsg_len = CMSG_LEN(sizeof(int));
        memcpy(CMSG_DATA(c), &pass_fd, sizeof(int));
    }
    (void)sendmsg(fd, &mh, MSG_NOSIGNAL);
}

/* Reads whatever arrives within a few milliseconds (the owner's reply, if any). */
static void drain(int fd)
{
    uint8_t sink[4096];
    struct pollfd p = {fd, POLLIN, 0};
    while (poll(&p, 1, 5) > 0 && (p.revents & POLLIN)) {
        ssize_t k = recv(fd, sink, sizeof sink, MSG_DONTWAIT);
        if (k <= 0) break;
    }
}

static void header(uint8_t *b, uint32_t op, uint64_t payload)
{
    memset(b, 0, HDR);
    memcpy(b, &kMagic, 4);
    memcpy(b + OFF_OP, &op, 4);
    for (int i = 0; i < 4; ++i) {
        uint64_t a = rnd() % 4 == 0 ? rnd() : rnd() % 8;
        memcpy(b + OFF_ARG + 8 * i, &a, 8);
    }
    memcpy(b + OFF_PAYLOAD, &payload, 8);
}

static void state_of(gms_owner *o, int *st, uint32_t *rd, int *inv)
{
    uint64_t al = 0;
    CHECK(gms_owner_status(o, st, rd, inv, &al) == GMS_OK);
    CHECK(al == 0); /* a host-only owner never holds memory */
}

int main(int argc, char **argv)
{
    CHECK(argc == 2);
    const char *path = argv[1];
    gms_owner *o = NULL;
    CHECK(gms_owner_create(path, GMS_HOST_ONLY, &o) == GMS_OK);
    pthread_t th;
    CHECK(pthread_create(&th, NULL, run_owner, o) == 0);
    int pipefd[2];
    CHECK(pipe(pipefd) == 0);

    for (int it = 0; it < 3000; ++it) {
        uint8_t b[HDR + 512];
        const int kind = (int)(rnd() % 4);
        int fd = dial(path);
        if (kind == 0) { /* raw random bytes, any length up to a header and more */
            const size_t n = (size_t)(rnd() % (HDR + 64));
            for (size_t i = 0; i < n; ++i) b[i] = (uint8_t)rnd();
            send_bytes(fd, b, n, rnd() % 8 == 0 ? pipefd[0] : -1);
        } else if (kind == 1) { /* a header with a random operation and a payload length it breaks */
            const uint64_t announced = rnd() % 3 == 0 ? rnd() % ((uint64_t)1 << 33) : rnd() % 600;
            header(b, (uint32_t)(rnd() % 14), announced);
            const size_t extra = (size_t)(rnd() % 512);
            for (size_t i = 0; i < extra; ++i) b[HDR + i] = (uint8_t)rnd();
            send_bytes(fd, b, HDR + extra, rnd() % 8 == 0 ? pipefd[0] : -1);
            drain(fd);
        } else { /* the write lease (from EMPTY or COMMITTED), then a random commit, alloc or free */
            header(b, 1 /* hello read-write */, 0);
            send_bytes(fd, b, HDR, -1);
            drain(fd);
            const uint32_t ops[4] = {5 /* commit */, 5, 3 /* alloc */, 4 /* free */};
            const size_t len = (size_t)(rnd() % 400);
            header(b, ops[rnd() % 4], len);
            uint64_t words[64];
            for (int i = 0; i < 64; ++i) words[i] = rnd() % 3 == 0 ? rnd() : rnd() % 5;
            memcpy(b + HDR, words, len < sizeof words ? len : sizeof words);
            if (len > sizeof words) memset(b + HDR + sizeof words, 0, len - sizeof words);
            send_bytes(fd, b, HDR + len, -1);
            drain(fd);
        }
        close(fd);

        if (it % 100 == 99) { /* the protocol still works for well-behaved clients */
            int st, inv;
            uint32_t rd;
            gms_client *w = NULL, *r1 = NULL, *r2 = NULL;
            uint64_t mm = 1;
            /* a garbage peer's connection may not be closed at the owner yet: retry briefly */
            int rc = GMS_ERR_STATE;
            for (int t = 0; t < 200 && rc == GMS_ERR_STATE; ++t) {
                rc = gms_client_connect(path, GMS_LEASE_RW, 0, NULL, &w, &mm);
                if (rc == GMS_ERR_STATE) usleep(1000);
            }
            CHECK(rc == GMS_OK && w != NULL);
            state_of(o, &st, &rd, &inv);
            CHECK(st == GMS_STORE_RW && rd == 0);
            CHECK(gms_client_commit(w, NULL, 0, NULL, &mm, NULL) == GMS_OK && mm == 0);
            CHECK(gms_client_disconnect(w) == GMS_OK);
            CHECK(gms_client_connect(path, GMS_LEASE_RO, 0, NULL, &r1, &mm) == GMS_OK);
            CHECK(gms_client_connect(path, GMS_LEASE_RO, 0, NULL, &r2, &mm) == GMS_OK);
            state_of(o, &st, &rd, &inv);
            CHECK(st == GMS_STORE_RO && rd == 2 && inv == 0);
            CHECK(gms_client_connect(path, GMS_LEASE_RW, 0, NULL, &w, &mm) == GMS_ERR_STATE);
            CHECK(gms_client_disconnect(r1) == GMS_OK && gms_client_disconnect(r2) == GMS_OK);
            state_of(o, &st, &rd, &inv);
            CHECK(st == GMS_STORE_COMMITTED && rd == 0);
        }
    }
    close(pipefd[0]);
    close(pipefd[1]);

    /* the in-process store's protocol, host-only, under random calls with random leases: every
     * call returns a status, and the reader count never exceeds the leases handed out */
    gms_store *st = NULL;
    CHECK(gms_store_create(GMS_HOST_ONLY, 0, 0, &st) == GMS_OK);
    uint64_t leases[16] = {0};
    int nl = 0;
    for (int it = 0; it < 20000; ++it) {
        uint64_t lease = 0, mm = 0, any = nl && rnd() % 4 ? leases[rnd() % (uint64_t)nl] : rnd() % 64;
        int rc = GMS_OK;
        switch (rnd() % 7) {
        case 0: rc = gms_store_connect_rw(st, &lease); break;
        case 1: rc = gms_store_connect_ro(st, rnd() % 2 ? GMS_CONNECT_VERIFY : 0, &lease, &mm, NULL); break;
        case 2: rc = gms_store_commit(st, any, NULL, 0, NULL, &mm, NULL); break;
        case 3: rc = gms_store_abort(st, any); break;
        case 4: rc = gms_store_disconnect(st, any); break;
        case 5: rc = gms_store_verify(st, &mm, NULL, 0, NULL); break;
        default: {
            uint64_t addr = 0;
            rc = gms_store_alloc(st, any, 1 + rnd() % 4096, 0, &addr);
            CHECK(rc != GMS_OK); /* a host-only store has no memory */
        }
        }
        CHECK(rc <= 0 && rc >= GMS_ERR_INTEGRITY);
        if (rc == GMS_OK && lease && nl < 16) leases[nl++] = lease;
        int state = 0, inv = 0;
        uint32_t rd = 0;
        CHECK(gms_store_state(st, &state, &rd, &inv) == GMS_OK);
        CHECK(state >= GMS_STORE_EMPTY && state <= GMS_STORE_RO && rd <= 16u + (uint32_t)it);
        CHECK((state == GMS_STORE_RO) == (rd > 0));
        if (nl == 16) nl = 0; /* forget old leases; the store keeps them */
    }
    gms_store_destroy(st);

    gms_owner_stop(o);
    CHECK(pthread_join(th, NULL) == 0);
    gms_owner_destroy(o);
    puts("owner fuzz ok");
    return 0;
}
