/*
 * Randomised host-only manifests through the C-ABI: layout invariants,
 * overlap detection against a brute-force pairwise check, chunk bounds.
 * Built with the library's host code under ASan/UBSan by a CPU test.
 */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>

#include "gms.h"

static uint64_t st = 88172645463325252ull;
static uint64_t rnd(void)
{
    st ^= st << 13;
    st ^= st >> 7;
    st ^= st << 17;
    return st;
}

int main(void)
{
    for (int rep = 0; rep < 3000; ++rep) {
        uint64_t n = rnd() % 64;
        gms_entry *e = calloc(n + 1, sizeof *e);
        int expect_overlap = 0;
        for (uint64_t i = 0; i < n; ++i) {
            e[i].addr = (1ull << 36) + (rnd() % 4096) * 4096 + (rnd() % 64);
            e[i].nbytes = (rnd() % 4 == 0) ? 0 : rnd() % (3 * 4096 * 64);
        }
        for (uint64_t i = 0; i < n; ++i)
            for (uint64_t j = i + 1; j < n; ++j)
                if (e[i].nbytes && e[j].nbytes && e[i].addr < e[j].addr + e[j].nbytes &&
                    e[j].addr < e[i].addr + e[i].nbytes)
                    expect_overlap = 1;
        uint64_t cb = (rnd() % 3 == 0) ? 0 : 4096 * (1 + rnd() % 64);
        gms_manifest *m = NULL;
        int rc = gms_manifest_create(e, n, GMS_HOST_ONLY, cb, &m);
        if (expect_overlap) {
            if (rc != GMS_ERR_OVERLAP || m) { fprintf(stderr, "rep %d: overlap not reported (%d)\n", rep, rc); return 1; }
            free(e);
            continue;
        }
        if (rc != GMS_OK) { fprintf(stderr, "rep %d: create failed %d %s\n", rep, rc, gms_last_error()); return 1; }
        uint64_t *off = calloc(n + 1, 8), *base = calloc(n + 1, 8);
        gms_layout(m, off, base);
        uint64_t acc = 0, payload = 0, chunks_min = 0, chunks_max = 0;
        const uint64_t chunk = cb ? cb : GMS_DEFAULT_CHUNK_BYTES;
        for (uint64_t i = 0; i < n; ++i) {
            if (off[i] != acc || base[i] * 4096 != off[i]) { fprintf(stderr, "rep %d: layout\n", rep); return 1; }
            acc += (e[i].nbytes + 4095) / 4096 * 4096;
            payload += e[i].nbytes;
            chunks_min += (e[i].nbytes + chunk - 1) / chunk;
            chunks_max += e[i].nbytes ? (e[i].nbytes + chunk - 1) / chunk + 1 : 0;
        }
        if (gms_image_bytes(m) != acc || gms_payload_bytes(m) != payload || gms_num_blocks(m) * 4096 != acc ||
            gms_num_chunks(m) < chunks_min || gms_num_chunks(m) > chunks_max) {
            fprintf(stderr, "rep %d: totals\n", rep);
            return 1;
        }
        gms_manifest_destroy(m);
        free(off);
        free(base);
        free(e);
    }
    puts("manifest fuzz ok");
    return 0;
}
