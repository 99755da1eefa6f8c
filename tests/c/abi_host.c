/*
 * C99 client of include/gms.h: builds host-only manifests (no GPU needed) and
 * checks the layout queries and argument errors.  Compiled by a CPU test with
 * gcc -std=c99 -Wall -Werror against libgms.so; exits non-zero on failure.
 */
#include <stdint.h>
#include <stdio.h>
#include <string.h>

#include "gms.h"

#define CHECK(c)                                                          \
    do {                                                                  \
        if (!(c)) {                                                       \
            fprintf(stderr, "%s:%d: check failed: %s\n", __FILE__, __LINE__, #c); \
            return 1;                                                     \
        }                                                                 \
    } while (0)

int main(void)
{
    gms_entry e[4] = {{1u << 20, 5000}, {2u << 20, 0}, {3u << 20, 8192}, {4u << 20, 1}};
    gms_manifest *m = NULL;
    CHECK(gms_abi_version() == 5);
    CHECK(gms_manifest_create(e, 4, GMS_HOST_ONLY, 0, &m) == GMS_OK && m != NULL);
    CHECK(gms_num_entries(m) == 4);
    CHECK(gms_payload_bytes(m) == 5000 + 8192 + 1);
    CHECK(gms_image_bytes(m) == 8192 + 0 + 8192 + 4096);
    CHECK(gms_num_blocks(m) == 2 + 0 + 2 + 1);
    CHECK(gms_num_chunks(m) == 3);
    CHECK(gms_manifest_device(m) == GMS_HOST_ONLY);
    uint64_t off[4], base[4];
    CHECK(gms_layout(m, off, base) == GMS_OK);
    CHECK(off[0] == 0 && off[1] == 8192 && off[2] == 8192 && off[3] == 16384);
    CHECK(base[0] == 0 && base[1] == 2 && base[2] == 2 && base[3] == 4);
    CHECK(gms_restore(m, (void *)(uintptr_t)0x1000, 1 << 20, GMS_MEM_DEVICE, NULL, NULL, NULL, NULL, NULL, 0, NULL)
          == GMS_ERR_STATE);
    CHECK(strlen(gms_last_error()) > 0);
    gms_manifest_destroy(m);

    gms_entry ov[2] = {{1u << 20, 100}, {(1u << 20) + 50, 100}};
    m = NULL;
    CHECK(gms_manifest_create(ov, 2, GMS_HOST_ONLY, 0, &m) == GMS_ERR_OVERLAP && m == NULL);
    CHECK(gms_manifest_create(e, 4, GMS_HOST_ONLY, 1000, &m) == GMS_ERR_INVALID);
    CHECK(strcmp(gms_status_str(GMS_ERR_IO), "file I/O error") == 0);
    gms_manifest_destroy(NULL);
    puts("abi_host ok");
    return 0;
}
