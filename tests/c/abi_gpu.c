/*
 * C99 client of include/gms.h on the GPU, with no Python or torch: device
 * memory from hipMalloc, streams as plain HIP handles.  Snapshot, restore and
 * verify results are compared with the C oracle (linked beside the library,
 * sharing nothing with it) on the same host bytes, for device images, a pinned
 * image through a small staging ring, an image file and a pageable host image;
 * the model-state store is driven through one commit and one verified
 * read-only lease.  Exits non-zero
 * on the first failed check, printing it.
 */
#define _POSIX_C_SOURCE 200809L /* mkstemp, close, unlink */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>
#include <unistd.h>

#include <hip/hip_runtime_api.h>

#include "gms.h"
#include "oracle.h"

#define CHECK(c)                                                                  \
    do {                                                                          \
        if (!(c)) {                                                               \
            fprintf(stderr, "%s:%d: check failed: %s (%s)\n", __FILE__, __LINE__, #c, \
                    gms_last_error());                                            \
            return 1;                                                             \
        }                                                                         \
    } while (0)

#define N 4

int main(void)
{
    const uint64_t sizes[N] = {(1u << 20) + 7, 4096, 13, 3 * 4096 + 100};
    const uint64_t mis[N] = {0, 0, 3, 16}; /* byte offsets inside each allocation */
    uint8_t *host[N], *back[N], *dev[N];
    gms_entry e[N];
    uint64_t state = 0x243F6A8885A308D3ull;
    CHECK(hipSetDevice(0) == hipSuccess);
    for (int i = 0; i < N; ++i) {
        host[i] = malloc(sizes[i]);
        back[i] = malloc(sizes[i] + 32);
        CHECK(host[i] && back[i]);
        for (uint64_t k = 0; k < sizes[i]; ++k) {
            state = state * 6364136223846793005ull + 1442695040888963407ull;
            host[i][k] = (uint8_t)(state >> 56);
        }
        CHECK(hipMalloc((void **)&dev[i], sizes[i] + 32) == hipSuccess);
        CHECK(hipMemset(dev[i], 0xA5, sizes[i] + 32) == hipSuccess);
        CHECK(hipMemcpy(dev[i] + mis[i], host[i], sizes[i], hipMemcpyHostToDevice) == hipSuccess);
        e[i].addr = (uint64_t)(uintptr_t)(dev[i] + mis[i]);
        e[i].nbytes = sizes[i];
    }

    /* the oracle's image and hashes of the same host bytes */
    uint64_t off[N], base[N], ib = 0, nb = 0;
    oracle_layout(sizes, N, off, base, &ib, &nb);
    uint8_t *o_img = malloc(ib), *g_img = malloc(ib);
    uint64_t *o_blk = malloc(nb * 8), *g_blk = malloc(nb * 8), o_ten[N], g_ten[N];
    CHECK(o_img && g_img && o_blk && g_blk);
    oracle_pack((const uint8_t *const *)host, sizes, N, o_img);
    oracle_hash((const uint8_t *const *)host, sizes, N, o_blk, o_ten);

    gms_manifest *m = NULL;
    CHECK(gms_manifest_create(e, N, 0, 0, &m) == GMS_OK);
    CHECK(gms_image_bytes(m) == ib && gms_num_blocks(m) == nb);
    hipStream_t s;
    CHECK(hipStreamCreate(&s) == hipSuccess);
    uint8_t *d_img;
    uint64_t *d_blk, *d_ten, *d_cnt, *d_list;
    CHECK(hipMalloc((void **)&d_img, ib) == hipSuccess);
    CHECK(hipMalloc((void **)&d_blk, nb * 8) == hipSuccess && hipMalloc((void **)&d_ten, N * 8) == hipSuccess);
    CHECK(hipMalloc((void **)&d_cnt, 8) == hipSuccess && hipMalloc((void **)&d_list, 8 * 8) == hipSuccess);

    /* snapshot: image and hashes equal the oracle's */
    CHECK(gms_snapshot(m, d_img, ib, GMS_MEM_DEVICE, d_blk, d_ten, s) == GMS_OK);
    CHECK(hipStreamSynchronize(s) == hipSuccess);
    CHECK(hipMemcpy(g_img, d_img, ib, hipMemcpyDeviceToHost) == hipSuccess);
    CHECK(hipMemcpy(g_blk, d_blk, nb * 8, hipMemcpyDeviceToHost) == hipSuccess);
    CHECK(hipMemcpy(g_ten, d_ten, N * 8, hipMemcpyDeviceToHost) == hipSuccess);
    CHECK(memcmp(g_img, o_img, ib) == 0);
    CHECK(memcmp(g_blk, o_blk, nb * 8) == 0 && memcmp(g_ten, o_ten, N * 8) == 0);

    /* poison, fused restore against the oracle's hashes: no mismatch, bytes back, nothing else written */
    uint64_t *d_exp, cnt = 99;
    CHECK(hipMalloc((void **)&d_exp, nb * 8) == hipSuccess);
    CHECK(hipMemcpy(d_exp, o_blk, nb * 8, hipMemcpyHostToDevice) == hipSuccess);
    for (int i = 0; i < N; ++i) CHECK(hipMemset(dev[i], 0x5A, sizes[i] + 32) == hipSuccess);
    for (int i = 0; i < N; ++i) CHECK(hipMemset(dev[i] + mis[i], 0xA5, sizes[i]) == hipSuccess);
    CHECK(gms_restore(m, d_img, ib, GMS_MEM_DEVICE, d_exp, NULL, NULL, d_cnt, d_list, 8, s) == GMS_OK);
    CHECK(hipStreamSynchronize(s) == hipSuccess);
    CHECK(hipMemcpy(&cnt, d_cnt, 8, hipMemcpyDeviceToHost) == hipSuccess && cnt == 0);
    for (int i = 0; i < N; ++i) {
        CHECK(hipMemcpy(back[i], dev[i], sizes[i] + 32, hipMemcpyDeviceToHost) == hipSuccess);
        CHECK(memcmp(back[i] + mis[i], host[i], sizes[i]) == 0);
        for (uint64_t k = 0; k < mis[i]; ++k) CHECK(back[i][k] == 0x5A);
        for (uint64_t k = mis[i] + sizes[i]; k < sizes[i] + 32; ++k) CHECK(back[i][k] == 0x5A);
    }

    /* one flipped byte in entry 3, block 2: verify flags exactly that block */
    uint8_t byte = host[3][2 * 4096 + 50] ^ 0x10;
    CHECK(hipMemcpy(dev[3] + mis[3] + 2 * 4096 + 50, &byte, 1, hipMemcpyHostToDevice) == hipSuccess);
    uint64_t list[8];
    CHECK(gms_verify(m, d_exp, NULL, NULL, d_cnt, d_list, 8, s) == GMS_OK);
    CHECK(hipStreamSynchronize(s) == hipSuccess);
    CHECK(hipMemcpy(&cnt, d_cnt, 8, hipMemcpyDeviceToHost) == hipSuccess && cnt == 1);
    CHECK(hipMemcpy(list, d_list, 8, hipMemcpyDeviceToHost) == hipSuccess && list[0] == base[3] + 2);
    CHECK(gms_verify(m, NULL, NULL, NULL, NULL, NULL, 0, s) == GMS_ERR_INVALID); /* nothing to do */

    /* pageable host image: snapshot into malloc'd memory, then restore from it with the oracle's hashes */
    uint8_t *h_img = malloc(ib);
    CHECK(h_img);
    memset(h_img, 0xEE, ib);
    CHECK(hipMemcpy(dev[3] + mis[3] + 2 * 4096 + 50, &host[3][2 * 4096 + 50], 1, hipMemcpyHostToDevice) == hipSuccess);
    CHECK(gms_snapshot_to_host(m, h_img, ib, 3, d_blk, NULL, s) == GMS_OK);
    CHECK(memcmp(h_img, o_img, ib) == 0);
    CHECK(hipMemcpy(g_blk, d_blk, nb * 8, hipMemcpyDeviceToHost) == hipSuccess && memcmp(g_blk, o_blk, nb * 8) == 0);
    for (int i = 0; i < N; ++i) CHECK(hipMemset(dev[i] + mis[i], 0x33, sizes[i]) == hipSuccess);
    CHECK(gms_restore_from_host(m, h_img, ib, 0, d_exp, NULL, NULL, d_cnt, d_list, 8, s) == GMS_OK);
    memset(h_img, 0, ib); /* the image may be reused once the call returns */
    CHECK(hipStreamSynchronize(s) == hipSuccess);
    CHECK(hipMemcpy(&cnt, d_cnt, 8, hipMemcpyDeviceToHost) == hipSuccess && cnt == 0);
    for (int i = 0; i < N; ++i) {
        CHECK(hipMemcpy(back[i], dev[i] + mis[i], sizes[i], hipMemcpyDeviceToHost) == hipSuccess);
        CHECK(memcmp(back[i], host[i], sizes[i]) == 0);
    }
    CHECK(gms_restore_from_host(m, h_img, ib - 1, 0, NULL, NULL, NULL, NULL, NULL, 0, s) == GMS_ERR_SIZE);
    CHECK(gms_snapshot_to_host(m, d_img, ib, 0, NULL, NULL, s) == GMS_ERR_INVALID); /* device memory */
    free(h_img);

    /* pinned host image through a staging ring of 64 KiB slices (many slices, the ring wraps) */
    uint8_t *p_img = NULL;
    CHECK(hipHostMalloc((void **)&p_img, ib, 0) == hipSuccess);
    memcpy(p_img, o_img, ib);
    CHECK(gms_manifest_set_staging(m, 64 * 1024, 2) == GMS_OK);
    for (int i = 0; i < N; ++i) CHECK(hipMemset(dev[i] + mis[i], 0x44, sizes[i]) == hipSuccess);
    CHECK(gms_restore(m, p_img, ib, GMS_MEM_HOST_PINNED, d_exp, NULL, NULL, d_cnt, NULL, 0, s) == GMS_OK);
    CHECK(hipStreamSynchronize(s) == hipSuccess);
    CHECK(hipMemcpy(&cnt, d_cnt, 8, hipMemcpyDeviceToHost) == hipSuccess && cnt == 0);
    for (int i = 0; i < N; ++i) {
        CHECK(hipMemcpy(back[i], dev[i] + mis[i], sizes[i], hipMemcpyDeviceToHost) == hipSuccess);
        CHECK(memcmp(back[i], host[i], sizes[i]) == 0);
    }
    memset(p_img, 0, ib);
    CHECK(gms_snapshot(m, p_img, ib, GMS_MEM_HOST_PINNED, NULL, NULL, s) == GMS_OK);
    CHECK(hipStreamSynchronize(s) == hipSuccess && memcmp(p_img, o_img, ib) == 0);
    CHECK(hipHostFree(p_img) == hipSuccess);

    /* an image file, buffered I/O, 3 workers */
    char path[] = "/tmp/gms_abi_gpu_XXXXXX";
    int fd = mkstemp(path);
    CHECK(fd >= 0);
    close(fd);
    CHECK(gms_snapshot_to_file(m, path, 0, 3, NULL, NULL, s) == GMS_OK);
    for (int i = 0; i < N; ++i) CHECK(hipMemset(dev[i] + mis[i], 0x55, sizes[i]) == hipSuccess);
    CHECK(gms_restore_from_file(m, path, 0, 0, 3, d_exp, NULL, NULL, d_cnt, NULL, 0, s) == GMS_OK);
    CHECK(hipStreamSynchronize(s) == hipSuccess);
    CHECK(hipMemcpy(&cnt, d_cnt, 8, hipMemcpyDeviceToHost) == hipSuccess && cnt == 0);
    for (int i = 0; i < N; ++i) {
        CHECK(hipMemcpy(back[i], dev[i] + mis[i], sizes[i], hipMemcpyDeviceToHost) == hipSuccess);
        CHECK(memcmp(back[i], host[i], sizes[i]) == 0);
    }
    unlink(path);

    /* the model-state store: populate, commit, verified read-only lease */
    gms_store *st = NULL;
    uint64_t w = 0, r = 0, a = 0, mm = 0;
    int state_now = -1;
    uint32_t readers = 0;
    CHECK(gms_store_create(0, 1u << 30, 8u << 20, &st) == GMS_OK);
    CHECK(gms_store_connect_rw(st, &w) == GMS_OK);
    CHECK(gms_store_alloc(st, w, sizes[0], 0, &a) == GMS_OK);
    CHECK(hipMemcpy((void *)(uintptr_t)a, host[0], sizes[0], hipMemcpyHostToDevice) == hipSuccess);
    gms_entry se = {a, sizes[0]};
    CHECK(gms_store_commit(st, w, &se, 1, NULL, &mm, s) == GMS_OK);
    CHECK(gms_store_connect_ro(st, GMS_CONNECT_VERIFY, &r, &mm, s) == GMS_OK && mm == 0);
    CHECK(gms_store_state(st, &state_now, &readers, NULL) == GMS_OK);
    CHECK(state_now == GMS_STORE_RO && readers == 1);
    uint64_t sb[260];
    CHECK(gms_num_blocks(gms_store_layout(st)) == 257);
    CHECK(hipMemcpy(sb, gms_store_block_hashes(st), 257 * 8, hipMemcpyDeviceToHost) == hipSuccess);
    CHECK(memcmp(sb, o_blk, 257 * 8) == 0); /* entry 0's blocks come first in both layouts */
    CHECK(gms_store_disconnect(st, r) == GMS_OK);
    gms_store_destroy(st);

    gms_manifest_destroy(m);
    CHECK(hipStreamDestroy(s) == hipSuccess);
    puts("abi_gpu ok");
    return 0;
}
