// Gather / scatter / verify kernels for gfx950.
//
// The unit of work is two 4 KiB blocks of one chunk of the manifest's work
// list, taken by one 2-wave workgroup: each wave moves and hashes one block
// (k_stream).  Launches of chunks of at most two blocks give each wave a whole
// chunk instead (k_pair).
// For a block a lane moves four 16-byte segments at byte offsets
// k*1024 + lane*16 (k = 0..3), so every load and store instruction of the
// wave covers 1 KiB contiguously.  Small, short-lived workgroups let the
// dispatcher keep every CU's few resident waves busy; restore and snapshot
// launches reserve LDS so that six workgroups (12 waves) are resident per CU,
// which measured best for the mixed read/write stream across weight sets,
// shards and KV pools, and the unit order is XCD-aware (striped for verify and for
// scattered units, contiguous per XCD otherwise).  Hashing happens on
// the registers that were just moved: each lane mixes its eight 8-byte words,
// the wave XOR-reduces its 64 partials with DPP row operations plus four lane
// reads, and lane 0 stores / compares the block hash.  Tensor hashes combine
// the two waves' XORs in LDS and take one 64-bit atomic XOR per unit (k_pair:
// one per chunk, from its wave).
//
// Bandwidth path: no MFMA; 16-byte non-temporal loads and stores for the
// streaming side, also for entries at any byte alignment (bytes are shifted
// between lanes in registers); byte stores only where a partial 16-byte
// granule has to be written.

#include <cstdlib>

#include "gms_internal.h"

namespace gms {
namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
// Entry addresses arrive as integers; these global-address-space views let the
// compiler emit global_* rather than flat_* memory instructions for them.
typedef __attribute__((address_space(1))) uint8_t gbyte;
typedef __attribute__((address_space(1))) u32x4 gvec;

constexpr uint64_t kG = 0x9E3779B97F4A7C15ull;   // index multiplier
constexpr uint64_t kMulA = 0xBF58476D1CE4E5B9ull;
constexpr uint64_t kMulB = 0x94D049BB133111EBull;
constexpr uint64_t kSegStrideG = 128ull * kG;    // word-index step between a lane's segments
constexpr uint64_t kBlockStrideG = 512ull * kG;  // word-index step between blocks
constexpr int kWaves = kBlocksPerUnit;           // waves per workgroup, one block each
constexpr int kUnitThreads = kWaves * 64;
constexpr uint32_t kXcds = 8;                    // accelerator complex dies on MI355X

__device__ __forceinline__ uint64_t mix64(uint64_t z)
{
    z ^= z >> 30;
    z *= kMulA;
    z ^= z >> 27;
    z *= kMulB;
    z ^= z >> 31;
    return z;
}

// Hash of the two little-endian words in v, at word indices j and j+1 (jg = j*G).
__device__ __forceinline__ uint64_t seg_hash(u32x4 v, uint64_t jg)
{
    uint64_t w0 = (uint64_t)v.x | ((uint64_t)v.y << 32);
    uint64_t w1 = (uint64_t)v.z | ((uint64_t)v.w << 32);
    return mix64(w0 ^ jg) ^ mix64(w1 ^ (jg + kG));
}

// XOR of v over the 64 lanes, returned uniformly.  Two quad permutes and two
// row rotations leave every lane with its 16-lane row's XOR; four lane reads
// combine the rows.
__device__ __forceinline__ uint32_t wave_xor32(uint32_t v)
{
    v ^= (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0xB1, 0xF, 0xF, false);  // quad_perm 1,0,3,2
    v ^= (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0x4E, 0xF, 0xF, false);  // quad_perm 2,3,0,1
    v ^= (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0x124, 0xF, 0xF, false); // row_ror 4
    v ^= (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0x128, 0xF, 0xF, false); // row_ror 8
    return (uint32_t)(__builtin_amdgcn_readlane((int)v, 0) ^ __builtin_amdgcn_readlane((int)v, 16) ^
                      __builtin_amdgcn_readlane((int)v, 32) ^ __builtin_amdgcn_readlane((int)v, 48));
}

__device__ __forceinline__ uint64_t wave_xor64(uint64_t v)
{
    uint32_t lo = wave_xor32((uint32_t)v);
    uint32_t hi = wave_xor32((uint32_t)(v >> 32));
    return (uint64_t)lo | ((uint64_t)hi << 32);
}

// Keeps the first `valid` (0..16) bytes of v, zeroes the rest.
__device__ __forceinline__ u32x4 keep_bytes(u32x4 v, uint32_t valid)
{
    uint64_t w0 = (uint64_t)v.x | ((uint64_t)v.y << 32);
    uint64_t w1 = (uint64_t)v.z | ((uint64_t)v.w << 32);
    if (valid < 8) {
        w0 = valid ? (w0 & (~0ull >> (64 - 8 * valid))) : 0;
        w1 = 0;
    } else if (valid < 16) {
        uint32_t r = valid - 8;
        w1 = r ? (w1 & (~0ull >> (64 - 8 * r))) : 0;
    }
    u32x4 o;
    o.x = (uint32_t)w0;
    o.y = (uint32_t)(w0 >> 32);
    o.z = (uint32_t)w1;
    o.w = (uint32_t)(w1 >> 32);
    return o;
}

// Reads `valid` bytes at the 16-byte-aligned p, zero-extended to 16.
__device__ __forceinline__ u32x4 load_part(const gbyte *p, uint32_t valid)
{
    if (valid == 16) return *(const gvec *)p;
    uint64_t w0 = 0, w1 = 0;
    for (uint32_t q = 0; q < valid; ++q) {
        uint64_t b = p[q];
        if (q < 8)
            w0 |= b << (8 * q);
        else
            w1 |= b << (8 * (q - 8));
    }
    u32x4 o;
    o.x = (uint32_t)w0;
    o.y = (uint32_t)(w0 >> 32);
    o.z = (uint32_t)w1;
    o.w = (uint32_t)(w1 >> 32);
    return o;
}

// Writes the first `valid` bytes of v to the 16-byte-aligned p.
__device__ __forceinline__ void store_part(gbyte *p, u32x4 v, uint32_t valid)
{
    if (valid == 16) {
        __builtin_nontemporal_store(v, (gvec *)p);
        return;
    }
    uint64_t w0 = (uint64_t)v.x | ((uint64_t)v.y << 32);
    uint64_t w1 = (uint64_t)v.z | ((uint64_t)v.w << 32);
    for (uint32_t q = 0; q < valid; ++q)
        p[q] = (uint8_t)(q < 8 ? (w0 >> (8 * q)) : (w1 >> (8 * (q - 8))));
}

// Bytes o .. o + 15 (o = 1..15, wave-uniform) of the 32 bytes lo:hi, lo first.
template <int D>
__device__ __forceinline__ u32x4 join_at(u32x4 lo, u32x4 hi, uint32_t r)
{
    const uint32_t x[8] = {lo.x, lo.y, lo.z, lo.w, hi.x, hi.y, hi.z, hi.w};
    u32x4 o;
    o.x = __builtin_amdgcn_alignbyte(x[D + 1], x[D], r);
    o.y = __builtin_amdgcn_alignbyte(x[D + 2], x[D + 1], r);
    o.z = __builtin_amdgcn_alignbyte(x[D + 3], x[D + 2], r);
    o.w = __builtin_amdgcn_alignbyte(x[D + 4], x[D + 3], r);
    return o;
}

__device__ __forceinline__ u32x4 join(u32x4 lo, u32x4 hi, uint32_t o)
{
    switch (o >> 2) {  // uniform: the shift is fixed per chunk
    case 0: return join_at<0>(lo, hi, o & 3);
    case 1: return join_at<1>(lo, hi, o & 3);
    case 2: return join_at<2>(lo, hi, o & 3);
    default: return join_at<3>(lo, hi, o & 3);
    }
}

// Whole-wave rotations by one lane (DPP wave_ror:1 / wave_rol:1, a GFX9 feature):
// ror gives lane l the value of lane l - 1 (lane 0 that of lane 63), rol the
// value of lane l + 1 (lane 63 that of lane 0).
template <int CTRL>
__device__ __forceinline__ u32x4 rotate(u32x4 v)
{
    u32x4 o;
    o.x = (uint32_t)__builtin_amdgcn_mov_dpp((int)v.x, CTRL, 0xF, 0xF, false);
    o.y = (uint32_t)__builtin_amdgcn_mov_dpp((int)v.y, CTRL, 0xF, 0xF, false);
    o.z = (uint32_t)__builtin_amdgcn_mov_dpp((int)v.z, CTRL, 0xF, 0xF, false);
    o.w = (uint32_t)__builtin_amdgcn_mov_dpp((int)v.w, CTRL, 0xF, 0xF, false);
    return o;
}
constexpr int kWaveRor1 = 0x13C;
constexpr int kWaveRol1 = 0x134;

// Writes bytes [lo, hi) of v into the 16-byte-aligned granule p, in naturally
// aligned pieces of 8, 4, 2 and 1 bytes.
__device__ __forceinline__ void store_range(gbyte *p, u32x4 v, int lo, int hi)
{
    const uint64_t w0 = (uint64_t)v.x | ((uint64_t)v.y << 32);
    const uint64_t w1 = (uint64_t)v.z | ((uint64_t)v.w << 32);
#pragma unroll 1
    for (int q = lo; q < hi;) {
        const uint64_t w = q < 8 ? w0 : w1;
        const int sh = 8 * (q & 7);
        if ((q & 7) == 0 && q + 8 <= hi) {
            *(__attribute__((address_space(1))) uint64_t *)(p + q) = w;
            q += 8;
        } else if ((q & 3) == 0 && q + 4 <= hi) {
            *(__attribute__((address_space(1))) uint32_t *)(p + q) = (uint32_t)(w >> sh);
            q += 4;
        } else if ((q & 1) == 0 && q + 2 <= hi) {
            *(__attribute__((address_space(1))) uint16_t *)(p + q) = (uint16_t)(w >> sh);
            q += 2;
        } else {
            p[q] = (uint8_t)(w >> sh);
            q += 1;
        }
    }
}

// Block epilogue.  `hl` is the lane's partial hash; with `check` set, lane 0
// folds the expected hash `want` into the reduction, so the reduced value is
// zero exactly when the block matches and `want` never has to leave its vector
// register.  Lane 0 stores the block hash / records a mismatch.  Returns the
// block hash in a vector register (meaningful in lane 0).
__device__ __forceinline__ uint64_t finish_block(uint64_t hl, uint64_t gblk, const HashOut &h, uint32_t lane,
                                                 bool check, uint64_t want)
{
    const uint64_t fold = (check && lane == 0) ? want : 0;
    const uint64_t red = wave_xor64(hl ^ fold);  // block hash, XOR want when checking
    const uint64_t hb = red ^ fold;
    if (lane == 0) {
        if (h.blk) h.blk[gblk] = hb;
        if (check && red != 0) {
            const uint64_t at = atomicAdd((unsigned long long *)h.mm_count, 1ull);
            if (h.mm_list && at < h.mm_cap) h.mm_list[at] = gblk;
        }
    }
    return hb;
}

// The lane's four 16-byte segments of the full 4 KiB block at p.
__device__ __forceinline__ void load_block(u32x4 v[4], const gbyte *p)
{
#pragma unroll
    for (int k = 0; k < 4; ++k) v[k] = __builtin_nontemporal_load((const gvec *)(p + k * 1024));
}

__device__ __forceinline__ void store_block(const u32x4 v[4], gbyte *p)
{
#pragma unroll
    for (int k = 0; k < 4; ++k) __builtin_nontemporal_store(v[k], (gvec *)(p + k * 1024));
}

// A snapshot wave pauses about 512 cycles after storing its block, before it
// hashes or exits.  The image it writes is one contiguous stream, and without
// the pause the next workgroup's gather reads start while that stream's
// stores are still in flight: an unhashed snapshot of the llama8b set read
// 78.5 to 79.3% of HBM peak without it and 80.4 to 81.3% with a pause of 128 to
// 2048 cycles; with hashes, 81.2 to 81.5% without and 81.7% at 512 cycles
// (79.9% at 2048).  Restores gained nothing from it.
constexpr int kSnapshotPause = 8;  // s_sleep units of 64 cycles

// An interior block of the shifted path (see move_block_shifted): a restore's
// full block that is not its chunk's last, or any full block of a snapshot or
// verify.  Every granule is whole (bar a chunk's first, for a restore), so no
// segment needs bounds.  The join takes bytes o .. o + 15 of each segment pair,
// o = 4 * D + r, o = 16 - a for a restore and a otherwise.
template <int OP, bool HASH, int D>
__device__ __forceinline__ uint64_t interior_block(uint32_t b, gbyte *img, gbyte *gran, uint64_t jg0, uint64_t gblk,
                                                   const HashOut &h, uint32_t lane, bool check, uint32_t a,
                                                   uint32_t r)
{
    const u32x4 zero = {0u, 0u, 0u, 0u};
    u32x4 seg[4];
    if (OP == kRestore) {
#pragma unroll
        for (int k = 0; k < 4; ++k) seg[k] = __builtin_nontemporal_load((const gvec *)(img + k * 1024));
        const bool inner = b > 0;  // the chunk's previous block shares granule 0
        u32x4 before = zero;
        if (inner && lane == 0) before = *(const gvec *)(img - 16);
        u32x4 rot[4];
#pragma unroll
        for (int k = 0; k < 4; ++k) rot[k] = rotate<kWaveRor1>(seg[k]);
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            const u32x4 prev = lane == 0 ? (k > 0 ? rot[k - 1] : before) : rot[k];
            const u32x4 gv = join_at<D>(prev, seg[k], r);
            if (k == 0 && !inner && lane == 0)
                store_range(gran, gv, (int)a, 16);
            else
                __builtin_nontemporal_store(gv, (gvec *)(gran + k * 1024));
        }
    } else {
        u32x4 g[4];
#pragma unroll
        for (int k = 0; k < 4; ++k) g[k] = __builtin_nontemporal_load((const gvec *)(gran + k * 1024));
        u32x4 tail = zero;  // the granule after the block, for lane 63
        if (lane == 63) tail = *(const gvec *)(gran + 3 * 1024 + 16);
        u32x4 rot[4];
#pragma unroll
        for (int k = 0; k < 4; ++k) rot[k] = rotate<kWaveRol1>(g[k]);
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            const u32x4 next = lane == 63 ? (k < 3 ? rot[k + 1] : tail) : rot[k];
            seg[k] = join_at<D>(g[k], next, r);
            if (OP == kSnapshot) __builtin_nontemporal_store(seg[k], (gvec *)(img + k * 1024));
        }
        if (OP == kSnapshot) __builtin_amdgcn_s_sleep(kSnapshotPause);
    }
    uint64_t tacc = 0;
    if (HASH) {
        uint64_t hl = 0;
#pragma unroll
        for (int k = 0; k < 4; ++k) hl ^= seg_hash(seg[k], jg0 + (uint64_t)k * kSegStrideG);
        tacc = finish_block(hl, gblk, h, lane, check, check ? h.expected[gblk] : 0);
    }
    return tacc;
}

// Block b of a chunk whose entry address is not 16-byte aligned (a = addr mod
// 16, 1..15).  Image slots are 4096-aligned, so the image side stays in
// 16-byte segments that hold whole entry words: lane l's segment s = 64k + l
// holds entry bytes [16s, 16s + 16) of the block and is hashed exactly as on
// the aligned path.  The entry side is covered by aligned 16-byte granules:
// granule s starts a bytes before segment s, so it takes the last a bytes of
// segment s - 1 and the first 16 - a of segment s, which a whole-wave DPP
// rotation brings from the neighbouring lane (lane 0 takes lane 63 of the
// previous k).
//  - A restore writes every granule with one 16-byte store.  The granule a
//    block shares with the one before it is written by the later block, which
//    also loads the earlier block's last image segment (same chunk, so the
//    same image slot); only at a chunk's first and last byte, and at the
//    entry's end, are granules written in part, with the widest aligned
//    stores that fit, so no byte outside the entry is touched.
//  - Snapshot and verify load the granules that hold a byte of the block
//    (whole granules never leave the entry's pages) and rotate the other way.
// Returns the block hash (in lane 0).
template <int OP, bool HASH>
__device__ __forceinline__ uint64_t move_block_shifted(const Chunk &c, uint32_t b, gbyte *img, uint64_t jg0,
                                                       uint64_t gblk, const HashOut &h, uint32_t lane, bool check)
{
    const uint32_t a = (uint32_t)(c.addr & 15);
    const uint32_t bs = b * kBlockBytes;
    const int bv = (int)min(kBlockBytes, c.len - bs);            // real bytes of the block
    gbyte *const gran = (gbyte *)(c.addr - a) + bs + lane * 16;  // the lane's granule of k = 0
    const u32x4 zero = {0u, 0u, 0u, 0u};
    u32x4 seg[4];

    // Interior blocks, most of any entry, skip the per-segment bounds below: for a
    // restore, a full block that is not the chunk's last writes whole granules
    // only (bar a chunk's first granule) and leaves the granule after it to the
    // next block; snapshot and verify of any full block load every granule and
    // the one after it, which holds the block's last a bytes.
    const bool interior = OP == kRestore ? bs + kBlockBytes < c.len : bs + kBlockBytes <= c.len;
    if (interior) {
        // one straight-line body per dword shift of the join (the shift is fixed per chunk)
        const uint32_t o = OP == kRestore ? 16 - a : a;
        switch (o >> 2) {
        case 0: return interior_block<OP, HASH, 0>(b, img, gran, jg0, gblk, h, lane, check, a, o & 3);
        case 1: return interior_block<OP, HASH, 1>(b, img, gran, jg0, gblk, h, lane, check, a, o & 3);
        case 2: return interior_block<OP, HASH, 2>(b, img, gran, jg0, gblk, h, lane, check, a, o & 3);
        default: return interior_block<OP, HASH, 3>(b, img, gran, jg0, gblk, h, lane, check, a, o & 3);
        }
    }

    if (OP == kRestore) {
#pragma unroll
        for (int k = 0; k < 4; ++k) seg[k] = __builtin_nontemporal_load((const gvec *)(img + k * 1024));
        const bool inner = b > 0;  // the chunk's previous block shares granule 0
        u32x4 before = zero;       // that block's last image segment, for lane 0
        if (inner && lane == 0) before = *(const gvec *)(img - 16);
        u32x4 r[4];
#pragma unroll
        for (int k = 0; k < 4; ++k) r[k] = rotate<kWaveRor1>(seg[k]);
        // at most two partial granules per lane, written after the loop
        u32x4 head = zero, part = zero;
        int head_hi = 0, part_hi = 0;
        gbyte *part_at = gran;
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            const u32x4 prev = lane == 0 ? (k > 0 ? r[k - 1] : before) : r[k];
            const int s = 64 * k + (int)lane;
            const int hi = min(16, bv + (int)a - 16 * s);
            const u32x4 gv = join(prev, seg[k], 16 - a);
            if (s == 0 && !inner) {
                head = gv;
                head_hi = hi;
            } else if (hi >= 16) {
                __builtin_nontemporal_store(gv, (gvec *)(gran + k * 1024));
            } else if (hi > 0) {
                part = gv;
                part_hi = hi;
                part_at = gran + k * 1024;
            }
        }
        // the granule after the block: the next block writes it, unless this is the chunk's last
        const bool last = bs + kBlockBytes >= c.len;
        if (last && lane == 63 && bv + (int)a > (int)kBlockBytes) {
            part = join(seg[3], zero, 16 - a);
            part_hi = bv + (int)a - (int)kBlockBytes;
            part_at = gran + 3 * 1024 + 16;
        }
        if (lane == 0 && !inner) store_range(gran, head, (int)a, head_hi);
        if (part_hi > 0) store_range(part_at, part, 0, part_hi);
    } else {
        u32x4 g[4];
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            const int s = 64 * k + (int)lane;
            g[k] = 16 * s < bv + (int)a ? __builtin_nontemporal_load((const gvec *)(gran + k * 1024)) : zero;
        }
        u32x4 tail = zero;  // the granule after the block, for lane 63
        if (lane == 63 && bv + (int)a > (int)kBlockBytes) tail = *(const gvec *)(gran + 3 * 1024 + 16);
        u32x4 n[4];
#pragma unroll
        for (int k = 0; k < 4; ++k) n[k] = rotate<kWaveRol1>(g[k]);
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            const u32x4 next = lane == 63 ? (k < 3 ? n[k + 1] : tail) : n[k];
            const int s = 64 * k + (int)lane;
            const uint32_t valid = (uint32_t)max(0, min(16, bv - 16 * s));
            seg[k] = keep_bytes(join(g[k], next, a), valid);
            if (OP == kSnapshot) __builtin_nontemporal_store(seg[k], (gvec *)(img + k * 1024));
        }
    }
    uint64_t tacc = 0;
    if (HASH) {
        uint64_t hl = 0;
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            const int s = 64 * k + (int)lane;
            const int valid = max(0, min(16, bv - 16 * s));
            const u32x4 v = OP == kRestore ? keep_bytes(seg[k], (uint32_t)valid) : seg[k];
            const uint64_t jg = jg0 + (uint64_t)k * kSegStrideG;
            const uint64_t w0 = (uint64_t)v.x | ((uint64_t)v.y << 32);
            const uint64_t w1 = (uint64_t)v.z | ((uint64_t)v.w << 32);
            if (valid > 0) hl ^= mix64(w0 ^ jg);
            if (valid > 8) hl ^= mix64(w1 ^ (jg + kG));
        }
        tacc = finish_block(hl, gblk, h, lane, check, check ? h.expected[gblk] : 0);
    }
    return tacc;
}

// Block b of chunk c, by one wave.  Chunks of entries at a 16-byte-aligned
// address (SHIFTED false; launches never mix the two kinds) move a full block
// with 16-byte non-temporal loads, store and hash it from the same registers;
// its expected hash is loaded branch-free (a harmless address when not
// checking) just before its data and folded into the wave reduction.  The
// ragged last block of an entry masks its partial segments.  Other chunks take
// move_block_shifted.  Returns the block hash (in lane 0), or 0 past the
// chunk's end.
template <int OP, bool HASH, bool SHIFTED>
__device__ __forceinline__ uint64_t move_block(const Chunk &c, uint32_t b, gbyte *img_base, uint64_t img_origin,
                                               const HashOut &h, uint32_t lane, bool check,
                                               const uint64_t *exp_dummy)
{
    const uint32_t nblk = (c.len + kBlockBytes - 1) / kBlockBytes;
    gbyte *const img = img_base + (c.img - img_origin) + (size_t)b * kBlockBytes + lane * 16;
    gbyte *const ent = (gbyte *)c.addr + (size_t)b * kBlockBytes + lane * 16;
    const uint64_t jg0 = (c.off >> 3) * kG + (uint64_t)b * kBlockStrideG + 2ull * lane * kG;
    const uint64_t gblk = (c.img >> 12) + b;
    uint64_t tacc = 0;

    if (SHIFTED) {
        if (b < nblk) tacc = move_block_shifted<OP, HASH>(c, b, img, jg0, gblk, h, lane, check);
    } else if (b < c.len / kBlockBytes) {  // full block
        uint64_t want = 0;
        if (HASH) want = *(check ? h.expected + gblk : exp_dummy);
        u32x4 v[4];
        load_block(v, OP == kRestore ? img : ent);
        if (OP != kVerify) store_block(v, OP == kRestore ? ent : img);
        if (OP == kSnapshot) __builtin_amdgcn_s_sleep(kSnapshotPause);
        if (HASH) {
            uint64_t hl = 0;
#pragma unroll
            for (int k = 0; k < 4; ++k) hl ^= seg_hash(v[k], jg0 + (uint64_t)k * kSegStrideG);
            tacc = finish_block(hl, gblk, h, lane, check, want);
        }
    } else if (b < nblk) {  // ragged last block
        const uint32_t boff = b * kBlockBytes;
        uint64_t hl = 0;
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            const uint32_t p = boff + k * 1024 + lane * 16;  // chunk-relative
            const uint32_t valid = p >= c.len ? 0u : min(16u, c.len - p);
            u32x4 v;
            if (OP == kRestore) {
                v = keep_bytes(*(const gvec *)(img + k * 1024), valid);
                store_part(ent + k * 1024, v, valid);
            } else {
                v = load_part(ent + k * 1024, valid);
                if (OP == kSnapshot) *(gvec *)(img + k * 1024) = v;
            }
            if (HASH) {
                const uint64_t jg = jg0 + (uint64_t)k * kSegStrideG;
                uint64_t w0 = (uint64_t)v.x | ((uint64_t)v.y << 32);
                uint64_t w1 = (uint64_t)v.z | ((uint64_t)v.w << 32);
                if (valid > 0) hl ^= mix64(w0 ^ jg);
                if (valid > 8) hl ^= mix64(w1 ^ (jg + kG));
            }
        }
        if (HASH) tacc = finish_block(hl, gblk, h, lane, check, check ? h.expected[gblk] : 0);
    }
    return tacc;
}

// XCD-aware order: the dispatcher hands workgroup IDs to the 8 XCDs round
// robin, so within each grid-sized round, XCD x takes the x-th contiguous
// eighth of the units and every XCD streams its own contiguous region of the
// image and of the entries.
__device__ __forceinline__ uint64_t xcd_slot()
{
    const uint64_t per_xcd = gridDim.x / kXcds;  // the grid is a multiple of kXcds
    return (blockIdx.x % kXcds) * per_xcd + blockIdx.x / kXcds;
}

// Striped order for verify, which only reads: XCD x takes stripes x, x + 8, ...
// of kVerifyStripe units (1 MiB), so the eight XCDs read one moving window of
// the entries together.  The last, partial round of stripes is split into eight
// contiguous pieces, which keeps the order a permutation of the round's slots.
// Measured on the llama8b set over six image allocations: 90.4 to 91.8% of HBM
// peak against 86.8 to 88.8% with contiguous eighths.  Restores and snapshots of
// launch groups whose chunks are mostly entries of their own (`striped`, set by
// the manifest: a KV pool's live units) take it too, 1.2 to 1.6 points above the
// eighths on the KV pool for either; weight sets keep the eighths, where striping
// moved llama8b by -1.0 to +0.0 points and the 70B shard by -2.9 to +1.5.
constexpr uint64_t kVerifyStripe = 128;

__device__ __forceinline__ uint64_t striped_slot()
{
    const uint64_t per_xcd = gridDim.x / kXcds, x = blockIdx.x % kXcds, i = blockIdx.x / kXcds;
    const uint64_t striped = per_xcd / kVerifyStripe * kVerifyStripe;  // slots per XCD in whole stripes
    if (i < striped) return ((i / kVerifyStripe) * kXcds + x) * kVerifyStripe + i % kVerifyStripe;
    return striped * kXcds + x * (per_xcd - striped) + (i - striped);
}

// Unit u is blocks [(u mod 2^shift) * kWaves, +kWaves) of chunk u >> shift
// (2^shift units cover the launch's longest chunk); wave w of the workgroup
// takes the unit's block w.  Tensor hashes combine the two waves' block
// hashes in LDS and take one atomic XOR per unit.  `striped` (uniform) selects
// the striped unit order for a restore or snapshot.
template <int OP, bool HASH, bool SHIFTED>
__global__ void __launch_bounds__(kUnitThreads)
k_stream(const Chunk *__restrict__ chunks, uint64_t count, uint32_t unit_shift, gbyte *__restrict__ img_base,
         uint64_t img_origin, HashOut h, uint32_t striped)
{
    extern __shared__ uint64_t wave_part[];  // kWaves words used
    const uint32_t lane = threadIdx.x & 63;
    const uint32_t wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);  // wave-uniform
    const bool check = HASH && h.expected != nullptr;
    const uint64_t *const exp_dummy = (const uint64_t *)chunks;  // any readable word
    const uint64_t units = count << unit_shift;
    const uint32_t unit_mask = (1u << unit_shift) - 1;
    const uint64_t slot_in_round = OP == kVerify || striped ? striped_slot() : xcd_slot();
    for (uint64_t round = 0; round < units; round += gridDim.x) {
        const uint64_t u = round + slot_in_round;
        if (u >= units) break;  // uniform across the workgroup
        const Chunk c = chunks[u >> unit_shift];
        const uint32_t b = ((uint32_t)u & unit_mask) * kWaves + wave;  // the wave's block of the chunk
        const uint64_t tacc = move_block<OP, HASH, SHIFTED>(c, b, img_base, img_origin, h, lane, check, exp_dummy);

        // ---- tensor hash: XOR of the workgroup's block hashes, one atomic per unit
        if (HASH && h.ten) {
            if (lane == 0) wave_part[wave] = tacc;
            __syncthreads();
            if (threadIdx.x == 0) {
                uint64_t t = 0;
#pragma unroll
                for (int w = 0; w < kWaves; ++w) t ^= wave_part[w];
                if (t) atomicXor((unsigned long long *)(h.ten + c.entry), (unsigned long long)t);
            }
            __syncthreads();
        }
    }
}

// Launches of one unit per chunk (chunks of at most kWaves blocks): a
// one-block chunk would leave the unit's second wave idle, so instead wave w
// of unit u takes all of chunk 2u + w, and each wave adds its chunk's hash to
// the tensor hash itself.  No barrier: a wave past the last chunk just skips.
template <int OP, bool HASH, bool SHIFTED>
__global__ void __launch_bounds__(kUnitThreads)
k_pair(const Chunk *__restrict__ chunks, uint64_t count, gbyte *__restrict__ img_base, uint64_t img_origin,
       HashOut h)
{
    const uint32_t lane = threadIdx.x & 63;
    const uint32_t wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);  // wave-uniform
    const bool check = HASH && h.expected != nullptr;
    const uint64_t *const exp_dummy = (const uint64_t *)chunks;
    const uint64_t units = (count + kWaves - 1) / kWaves;
    const uint64_t slot_in_round = xcd_slot();
    for (uint64_t round = 0; round < units; round += gridDim.x) {
        const uint64_t u = round + slot_in_round;
        if (u >= units) break;
        const uint64_t ci = u * kWaves + wave;
        if (ci >= count) continue;  // wave-uniform
        const Chunk c = chunks[ci];
        const uint32_t nblk = (c.len + kBlockBytes - 1) / kBlockBytes;  // at most kWaves
        uint64_t tacc = 0;
        for (uint32_t b = 0; b < nblk; ++b)
            tacc ^= move_block<OP, HASH, SHIFTED>(c, b, img_base, img_origin, h, lane, check, exp_dummy);
        if (HASH && h.ten && lane == 0 && tacc)
            atomicXor((unsigned long long *)(h.ten + c.entry), (unsigned long long)tacc);
    }
}

// Host-to-device copies of staging slices run as a kernel, not on a DMA
// engine.  The copy stream's DMA engine is shared with work the driver starts
// when device memory is remapped, or freed and allocated again, and for up to a
// second then H2D DMAs ran at 34 to 46 of 57 GB/s; a kernel reading the pinned
// slice over the link is not slowed.  32 workgroups, each taking 64 KiB spans in
// turn with 16-byte non-temporal loads two deep per thread, keep 256 KiB of
// host reads in flight: the link's bandwidth-latency product, and no more.
// Every read beyond it only waits in queues that HBM traffic from other
// kernels shares: with 1 MiB in flight (64 workgroups, four deep) the link
// gained 0.2% while a device-image restore running beside the copy fell from
// 81% to 28% of HBM peak; at 256 KiB it runs at 78%.  Grids that do not divide
// the spans evenly (20, 24 or 48 workgroups) lose 2 to 3% of the link.
constexpr uint32_t kCopyThreads = 256;
constexpr uint32_t kCopyGroups = 32;
constexpr int kCopyDepth = 2;                   // loads in flight per thread
constexpr uint64_t kCopySpan = 64 * 1024 / 16;  // 16-byte elements per span

__global__ void __launch_bounds__(kCopyThreads)
k_host_copy(const gvec *__restrict__ src, gvec *__restrict__ dst, uint64_t n16)
{
    for (uint64_t lo = (uint64_t)blockIdx.x * kCopySpan; lo < n16; lo += (uint64_t)gridDim.x * kCopySpan) {
        const uint64_t hi = lo + kCopySpan < n16 ? lo + kCopySpan : n16;
#pragma unroll kCopyDepth
        for (uint64_t i = lo + threadIdx.x; i < hi; i += kCopyThreads) dst[i] = __builtin_nontemporal_load(src + i);
    }
}

__global__ void __launch_bounds__(kUnitThreads)
k_prologue(uint64_t *__restrict__ ten, uint64_t n, uint64_t *__restrict__ mm_count)
{
    const uint64_t tid = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const uint64_t stride = (uint64_t)gridDim.x * blockDim.x;
    if (ten)
        for (uint64_t i = tid; i < n; i += stride) ten[i] = 0;
    if (mm_count && tid == 0) *mm_count = 0;
}

// A dispatch counts its grid in work-items with 32 bits, so a launch holds at
// most 2^24 workgroups of kUnitThreads (2^31 work-items, a multiple of kXcds);
// larger launches loop over grid-sized rounds.  GMS_MAX_GRID (a multiple of 8,
// read once) lowers the cap so that tests can run many rounds on small inputs.
constexpr uint64_t kMaxGrid = 1ull << 24;
static_assert(kMaxGrid * kUnitThreads <= (1ull << 32) - 1, "grid in work-items must fit 32 bits");

uint64_t max_grid()
{
    static const uint64_t cap = [] {
        const char *v = getenv("GMS_MAX_GRID");
        if (!v || !*v) return kMaxGrid;
        const unsigned long long x = strtoull(v, nullptr, 10);
        if (x < kXcds || x > kMaxGrid || x % kXcds) return kMaxGrid;
        return (uint64_t)x;
    }();
    return cap;
}
// Dynamic LDS per workgroup: restore and snapshot ask for a sixth of a CU's
// 160 KiB so that six 2-wave workgroups are resident per CU; verify
// (read-only, heavier on VALU per byte) only needs the wave partials and runs
// at full occupancy.  So do launches of one unit per chunk (chunks of at most
// two blocks, k_pair): each wave then moves at most 8 KiB behind two dependent
// loads, and more of them in flight hide that latency (200,000 one-block
// entries: 0.52 ms at six workgroups per CU, 0.24 ms at full occupancy).
constexpr size_t kLdsCopy = 26 * 1024;
constexpr size_t kLdsVerify = kWaves * sizeof(uint64_t);

uint64_t grid_for(uint64_t units)
{
    const uint64_t cap = max_grid();
    return ((units < cap ? units : cap) + kXcds - 1) / kXcds * kXcds;
}

template <int OP, bool HASH, bool SHIFTED>
hipError_t launch_t(const Chunk *chunks, uint64_t first, uint64_t count, uint32_t unit_shift, uint8_t *img_base,
                    uint64_t img_origin, const HashOut &h, bool striped, hipStream_t s)
{
    if (unit_shift == 0) {
        const uint64_t grid = grid_for((count + kWaves - 1) / kWaves);
        hipLaunchKernelGGL((k_pair<OP, HASH, SHIFTED>), dim3((uint32_t)grid), dim3(kUnitThreads), 0, s, chunks + first, count,
                           (gbyte *)img_base, img_origin, h);
        return hipGetLastError();
    }
    constexpr size_t lds = OP == kVerify ? kLdsVerify : kLdsCopy;
    static_assert(lds <= 64 * 1024, "above 64 KiB the launch would have to opt in per device");
    hipLaunchKernelGGL((k_stream<OP, HASH, SHIFTED>), dim3((uint32_t)grid_for(count << unit_shift)), dim3(kUnitThreads), lds,
                       s, chunks + first, count, unit_shift, (gbyte *)img_base, img_origin, h, striped ? 1u : 0u);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_host_copy(const uint8_t *src, uint8_t *dst, uint64_t bytes, hipStream_t s)
{
    if (bytes == 0) return hipSuccess;
    if (bytes % 16) return hipErrorInvalidValue;
    const uint64_t spans = (bytes / 16 + kCopySpan - 1) / kCopySpan;
    const uint32_t grid = (uint32_t)(spans < kCopyGroups ? spans : kCopyGroups);
    hipLaunchKernelGGL(k_host_copy, dim3(grid), dim3(kCopyThreads), 0, s, (const gvec *)src, (gvec *)dst, bytes / 16);
    return hipGetLastError();
}

hipError_t launch_prologue(const HashOut &h, uint64_t n_entries, hipStream_t s)
{
    uint64_t *ten = h.ten;
    uint64_t *cnt = h.expected ? h.mm_count : nullptr;
    if (!ten && !cnt) return hipSuccess;
    uint64_t items = ten ? n_entries : 1;
    uint64_t grid = (items + kUnitThreads - 1) / kUnitThreads;
    if (grid == 0) grid = 1;
    if (grid > 4096) grid = 4096;
    hipLaunchKernelGGL(k_prologue, dim3((uint32_t)grid), dim3(kUnitThreads), 0, s, ten, ten ? n_entries : 0, cnt);
    return hipGetLastError();
}

template <bool SHIFTED>
hipError_t launch_op(int op, bool hash, const Chunk *chunks, uint64_t first, uint64_t count, uint32_t shift,
                     uint8_t *img_base, uint64_t img_origin, const HashOut &h, bool striped, hipStream_t s)
{
#define GMS_LAUNCH(OP, HASH) launch_t<OP, HASH, SHIFTED>(chunks, first, count, shift, img_base, img_origin, h, striped, s)
    switch (op * 2 + (hash ? 1 : 0)) {
    case kRestore * 2: return GMS_LAUNCH(kRestore, false);
    case kRestore * 2 + 1: return GMS_LAUNCH(kRestore, true);
    case kSnapshot * 2: return GMS_LAUNCH(kSnapshot, false);
    case kSnapshot * 2 + 1: return GMS_LAUNCH(kSnapshot, true);
    case kVerify * 2 + 1: return GMS_LAUNCH(kVerify, true);
    default: return hipErrorInvalidValue;
    }
#undef GMS_LAUNCH
}

hipError_t launch_stream(int op, bool hash, bool shifted, bool striped, const Chunk *chunks, uint64_t first,
                         uint64_t count, uint32_t shift, uint8_t *img_base, uint64_t img_origin, const HashOut &h,
                         hipStream_t s)
{
    if (count == 0) return hipSuccess;
    if (shift > kMaxUnitShift || (count << shift) >> shift != count) return hipErrorInvalidValue;
    return shifted ? launch_op<true>(op, hash, chunks, first, count, shift, img_base, img_origin, h, striped, s)
                   : launch_op<false>(op, hash, chunks, first, count, shift, img_base, img_origin, h, striped, s);
}

}  // namespace gms
