/*
 * CPU oracle for the image/restore/verify path -- TEST INFRASTRUCTURE ONLY.
 *
 * Plain, slow, obviously correct C that states what the GPU library computes.
 * Only the tests, the smoke check and the benchmark's CPU-baseline leg may
 * load it; the product path never does.  It shares no code, header, table or
 * constant generator with the GPU library.
 *
 * Definitions (all integers little-endian, arithmetic mod 2^64):
 *   Layout   img_off[0] = 0, img_off[i+1] = img_off[i] + roundup(n_i, 4096);
 *            blk_base[0] = 0, blk_base[i+1] = blk_base[i] + ceil(n_i / 4096).
 *   Pack     image[img_off[i] + k] = X_i[k] for k < n_i; the rest of entry i's
 *            4 KiB slots is zero.
 *   Unpack   X_i[k] = image[img_off[i] + k] for k < n_i; nothing else written.
 *   Word     W_i[j] = bytes 8j..8j+7 of X_i, little-endian, bytes >= n_i read 0,
 *            for j < ceil(n_i / 8); j is the entry-relative word index.
 *   Mixer    fmix(z): z ^= z>>30; z *= C1; z ^= z>>27; z *= C2; z ^= z>>31
 *            (the splitmix64 output function; C1 = 0xBF58476D1CE4E5B9,
 *            C2 = 0x94D049BB133111EB).
 *   Block    Hb(i,b) = XOR over words j of block b (512 words per 4 KiB
 *            block, the last block only its real words) of
 *            fmix(W_i[j] XOR j*G), G = 0x9E3779B97F4A7C15.
 *   Tensor   Ht(i) = XOR_b Hb(i,b); an empty entry hashes to 0.
 *   Verify   M = ascending { blk_base[i] + b : Hb(i,b) != E[blk_base[i] + b] }.
 */
#ifndef GMS_ORACLE_H
#define GMS_ORACLE_H

#include <stdint.h>

#define ORACLE_BLOCK 4096u

uint64_t oracle_fmix(uint64_t z);
uint64_t oracle_word(const uint8_t *x, uint64_t n, uint64_t j);
uint64_t oracle_block_hash(const uint8_t *x, uint64_t n, uint64_t b);
uint64_t oracle_block_hash_at(const uint8_t *blk, uint64_t n, uint64_t b);
uint64_t oracle_entry_hashes(const uint8_t *x, uint64_t n, uint64_t *blk_out);
void oracle_layout(const uint64_t *nbytes, uint64_t count, uint64_t *img_off, uint64_t *blk_base,
                   uint64_t *image_bytes, uint64_t *num_blocks);
void oracle_pack(const uint8_t *const *src, const uint64_t *nbytes, uint64_t count, uint8_t *image);
void oracle_unpack(const uint8_t *image, uint8_t *const *dst, const uint64_t *nbytes, uint64_t count);
void oracle_hash(const uint8_t *const *src, const uint64_t *nbytes, uint64_t count,
                 uint64_t *blk_hash, uint64_t *ten_hash);
uint64_t oracle_verify(const uint8_t *const *src, const uint64_t *nbytes, uint64_t count,
                       const uint64_t *expected, uint64_t *mismatch_list, uint64_t cap);

#endif
