/*
 * CPU oracle -- TEST INFRASTRUCTURE ONLY (see oracle.h for the definitions).
 *
 * What is computed, and where it comes from:
 *  - Pack/unpack model the device-state image of a checkpoint: capture stages
 *    the engine's remaining device state into one artifact and recovery
 *    reverses it, re-creating the allocations (paper section 3.1, Snapshots,
 *    capture step 3 and the restore that reverses it).  The transfer cost of
 *    recovery is the artifact size over the effective bandwidth, S / B_eff
 *    (section 3.1).  The allocations are the recorded tensor layouts a GMS
 *    client captures before commit (section 4, GMS).
 *  - The block/tensor hashes back the check that surviving allocations are
 *    safe to reattach read-only: the paper notes that a schedulable device or
 *    the absence of fault reports does not prove resident state intact
 *    (section 2.2, Failure model) before a replacement re-imports it
 *    (section 3.2, GMS).  The paper fixes no hash; the one here is the
 *    library's own fixed definition.
 *
 * Nothing here is blocked, fused or reordered: every word is read byte by
 * byte and mixed in definition order.
 */
#include "oracle.h"

#include <string.h>

#define ORACLE_G  0x9E3779B97F4A7C15ull
#define ORACLE_C1 0xBF58476D1CE4E5B9ull
#define ORACLE_C2 0x94D049BB133111EBull

uint64_t oracle_fmix(uint64_t z)
{
    z ^= z >> 30;
    z *= ORACLE_C1;
    z ^= z >> 27;
    z *= ORACLE_C2;
    z ^= z >> 31;
    return z;
}

/* W[j]: bytes 8j..8j+7 as a little-endian integer, bytes at or past n read 0. */
uint64_t oracle_word(const uint8_t *x, uint64_t n, uint64_t j)
{
    uint64_t w = 0;
    for (uint64_t k = 0; k < 8; ++k) {
        uint64_t pos = 8 * j + k;
        uint64_t byte = pos < n ? x[pos] : 0;
        w |= byte << (8 * k);
    }
    return w;
}

static uint64_t ceil_div(uint64_t a, uint64_t b) { return a / b + (a % b != 0); }

/* Hb of a block whose `len` (<= 4096) real bytes start at blk and whose first
 * word has entry-relative index j0. */
static uint64_t hash_block_bytes(const uint8_t *blk, uint64_t len, uint64_t j0)
{
    uint64_t h = 0;
    for (uint64_t q = 0; q < ceil_div(len, 8); ++q)
        h ^= oracle_fmix(oracle_word(blk, len, q) ^ ((j0 + q) * ORACLE_G));
    return h;
}

/* Real bytes of block b of an n-byte entry (0 past the last block). */
static uint64_t block_len(uint64_t n, uint64_t b)
{
    uint64_t lo = ORACLE_BLOCK * b;
    if (lo >= n) return 0;
    return n - lo < ORACLE_BLOCK ? n - lo : ORACLE_BLOCK;
}

uint64_t oracle_block_hash(const uint8_t *x, uint64_t n, uint64_t b)
{
    uint64_t len = block_len(n, b);
    return len ? hash_block_bytes(x + ORACLE_BLOCK * b, len, ORACLE_BLOCK * b / 8) : 0;
}

/* Same as oracle_block_hash, given only block b's bytes (blk) of an n-byte entry. */
uint64_t oracle_block_hash_at(const uint8_t *blk, uint64_t n, uint64_t b)
{
    uint64_t len = block_len(n, b);
    return len ? hash_block_bytes(blk, len, ORACLE_BLOCK * b / 8) : 0;
}

/* Writes ceil(n/4096) block hashes (if blk_out) and returns the tensor hash. */
uint64_t oracle_entry_hashes(const uint8_t *x, uint64_t n, uint64_t *blk_out)
{
    uint64_t nblk = ceil_div(n, ORACLE_BLOCK);
    uint64_t t = 0;
    for (uint64_t b = 0; b < nblk; ++b) {
        uint64_t hb = oracle_block_hash(x, n, b);
        if (blk_out) blk_out[b] = hb;
        t ^= hb;
    }
    return t;
}

void oracle_layout(const uint64_t *nbytes, uint64_t count, uint64_t *img_off, uint64_t *blk_base,
                   uint64_t *image_bytes, uint64_t *num_blocks)
{
    uint64_t off = 0, blk = 0;
    for (uint64_t i = 0; i < count; ++i) {
        if (img_off) img_off[i] = off;
        if (blk_base) blk_base[i] = blk;
        off += ceil_div(nbytes[i], ORACLE_BLOCK) * ORACLE_BLOCK;
        blk += ceil_div(nbytes[i], ORACLE_BLOCK);
    }
    if (image_bytes) *image_bytes = off;
    if (num_blocks) *num_blocks = blk;
}

void oracle_pack(const uint8_t *const *src, const uint64_t *nbytes, uint64_t count, uint8_t *image)
{
    uint64_t off = 0;
    for (uint64_t i = 0; i < count; ++i) {
        uint64_t slot = ceil_div(nbytes[i], ORACLE_BLOCK) * ORACLE_BLOCK;
        if (nbytes[i]) memcpy(image + off, src[i], nbytes[i]);
        memset(image + off + nbytes[i], 0, slot - nbytes[i]);
        off += slot;
    }
}

void oracle_unpack(const uint8_t *image, uint8_t *const *dst, const uint64_t *nbytes, uint64_t count)
{
    uint64_t off = 0;
    for (uint64_t i = 0; i < count; ++i) {
        if (nbytes[i]) memcpy(dst[i], image + off, nbytes[i]);
        off += ceil_div(nbytes[i], ORACLE_BLOCK) * ORACLE_BLOCK;
    }
}

void oracle_hash(const uint8_t *const *src, const uint64_t *nbytes, uint64_t count,
                 uint64_t *blk_hash, uint64_t *ten_hash)
{
    uint64_t blk = 0;
    for (uint64_t i = 0; i < count; ++i) {
        uint64_t t = oracle_entry_hashes(src[i], nbytes[i], blk_hash ? blk_hash + blk : 0);
        if (ten_hash) ten_hash[i] = t;
        blk += ceil_div(nbytes[i], ORACLE_BLOCK);
    }
}

/* Returns |M|; writes the first min(|M|, cap) indices of M, ascending. */
uint64_t oracle_verify(const uint8_t *const *src, const uint64_t *nbytes, uint64_t count,
                       const uint64_t *expected, uint64_t *mismatch_list, uint64_t cap)
{
    uint64_t blk = 0, found = 0;
    for (uint64_t i = 0; i < count; ++i) {
        uint64_t nblk = ceil_div(nbytes[i], ORACLE_BLOCK);
        for (uint64_t b = 0; b < nblk; ++b) {
            if (oracle_block_hash(src[i], nbytes[i], b) != expected[blk + b]) {
                if (found < cap && mismatch_list) mismatch_list[found] = blk + b;
                ++found;
            }
        }
        blk += nblk;
    }
    return found;
}
