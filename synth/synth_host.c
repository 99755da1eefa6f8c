/*
 * Host side of the synthetic-input generator (see philox.h).  Plain C, built
 * with gcc into libsynth_host.so; the GPU side (synth_dev.hip) compiles the
 * same philox.h, so a tensor generated on either side has the same bits.
 */
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define SYNTH_FN static inline
#include "philox.h"

/* Raw Philox4x32-10 block, for the published known-answer vectors. */
void synth_philox(const uint32_t ctr[4], const uint32_t key[2], uint32_t out[4])
{
    synth_u32x4 c = {{ctr[0], ctr[1], ctr[2], ctr[3]}};
    synth_u32x4 r = synth_philox4x32_10(c, key[0], key[1]);
    memcpy(out, r.v, sizeof r.v);
}

/* 64-bit value number `index` of stream `stream` (low two words of a draw). */
uint64_t synth_u64(uint64_t seed, uint64_t stream, uint64_t index)
{
    synth_u32x4 r = synth_draw(seed, stream, index);
    return (uint64_t)r.v[0] | ((uint64_t)r.v[1] << 32);
}

/* out[i] = bf16 element (first + i) of tensor `tensor` under `seed`. */
void synth_fill_bf16(uint16_t *out, uint64_t n, uint64_t seed, uint64_t tensor, uint64_t first)
{
    for (uint64_t i = 0; i < n; ++i)
        out[i] = synth_bf16(seed, tensor, first + i);
}

/* out[i] = byte (first + i) of byte stream `stream`: byte k is byte k%16 of draw k/16. */
void synth_fill_bytes(uint8_t *out, uint64_t n, uint64_t seed, uint64_t stream, uint64_t first)
{
    uint64_t i = 0;
    while (i < n) {
        uint64_t k = first + i;
        synth_u32x4 r = synth_draw(seed, stream, k >> 4);
        uint8_t b[16];
        memcpy(b, r.v, 16);
        for (uint64_t q = k & 15; q < 16 && i < n; ++q, ++i)
            out[i] = b[q];
    }
}

/*
 * Fragmented live map of a paged pool: Fisher-Yates over ids 0..nblocks-1,
 * step i (from nblocks-1 down to 1) swaps ids i and j = u64 mod (i + 1),
 * drawing value number (nblocks-1-i) of stream `stream`.  The first `nlive`
 * ids of the shuffled order, sorted ascending, are written to live_out.
 * Returns 0, or -1 on bad arguments / allocation failure.
 */
static int cmp_u32(const void *a, const void *b)
{
    uint32_t x = *(const uint32_t *)a, y = *(const uint32_t *)b;
    return (x > y) - (x < y);
}

int synth_live_map(uint32_t *live_out, uint32_t nblocks, uint32_t nlive, uint64_t seed, uint64_t stream)
{
    if (!live_out || nlive > nblocks) return -1;
    uint32_t *perm = (uint32_t *)malloc((size_t)nblocks * sizeof *perm + 1);
    if (!perm) return -1;
    for (uint32_t i = 0; i < nblocks; ++i) perm[i] = i;
    for (uint32_t i = nblocks ? nblocks - 1 : 0; i >= 1; --i) {
        uint64_t r = synth_u64(seed, stream, (uint64_t)(nblocks - 1 - i));
        uint32_t j = (uint32_t)(r % ((uint64_t)i + 1));
        uint32_t t = perm[i]; perm[i] = perm[j]; perm[j] = t;
    }
    memcpy(live_out, perm, (size_t)nlive * sizeof *perm);
    qsort(live_out, nlive, sizeof *live_out, cmp_u32);
    free(perm);
    return 0;
}
