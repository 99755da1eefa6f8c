// Gather / scatter / verify kernels for gfx950.
//
// One workgroup (4 wave64s) takes one chunk of the manifest's work list; each
// wave walks the chunk's 4 KiB blocks with stride 4.  For one block a lane
// moves four 16-byte segments at byte offsets k*1024 + lane*16 (k = 0..3), so
// every load and store instruction of the wave covers 1 KiB contiguously.
// Hashing happens on the registers that were just moved: each lane mixes its
// eight 8-byte words, the wave XOR-reduces its 64 partials with DPP row
// operations plus four lane reads, and lane 0 stores / compares the block
// hash.  Tensor hashes combine the four waves' XORs in LDS and take one 64-bit
// atomic XOR per chunk.
//
// Bandwidth path: no MFMA; 16-byte non-temporal loads and stores for the
// streaming side; byte-granular code only for unaligned entries and the ragged
// last block of an entry.

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

// Reads `valid` bytes at p (any alignment), zero-extended to 16.
__device__ __forceinline__ u32x4 load_part(const gbyte *p, uint32_t valid, bool aligned)
{
    if (aligned && valid == 16) return *(const gvec *)p;
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

// Writes the first `valid` bytes of v to p (any alignment).
__device__ __forceinline__ void store_part(gbyte *p, u32x4 v, uint32_t valid, bool aligned)
{
    if (aligned && valid == 16) {
        __builtin_nontemporal_store(v, (gvec *)p);
        return;
    }
    uint64_t w0 = (uint64_t)v.x | ((uint64_t)v.y << 32);
    uint64_t w1 = (uint64_t)v.z | ((uint64_t)v.w << 32);
    for (uint32_t q = 0; q < valid; ++q)
        p[q] = (uint8_t)(q < 8 ? (w0 >> (8 * q)) : (w1 >> (8 * (q - 8))));
}

template <int OP, bool HASH>
__global__ void __launch_bounds__(kThreads)
k_stream(const Chunk *__restrict__ chunks, uint64_t count, gbyte *__restrict__ img_base,
         uint64_t img_origin, HashOut h)
{
    __shared__ uint64_t wave_part[kThreads / 64];
    const uint32_t lane = threadIdx.x & 63;
    const uint32_t wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);  // wave-uniform

    for (uint64_t ci = blockIdx.x; ci < count; ci += gridDim.x) {
        const Chunk c = chunks[ci];
        const uint32_t nblk = (c.len + kBlockBytes - 1) / kBlockBytes;
        const bool aligned = (c.addr & 15) == 0;
        gbyte *const img = img_base + (c.img - img_origin);
        uint64_t tacc = 0;

        for (uint32_t b = wave; b < nblk; b += kThreads / 64) {
            const uint32_t boff = b * kBlockBytes;
            gbyte *const ip = img + boff + lane * 16;
            gbyte *const ep = (gbyte *)(c.addr + boff) + lane * 16;
            // j*G of the lane's first word in segment 0
            const uint64_t jg0 = (((c.off + boff) >> 3) + 2 * lane) * kG;
            uint64_t hl = 0;

            if (aligned && boff + kBlockBytes <= c.len) {
                u32x4 v[4];
                if (OP == kRestore) {
#pragma unroll
                    for (int k = 0; k < 4; ++k) v[k] = __builtin_nontemporal_load((const gvec *)(ip + k * 1024));
#pragma unroll
                    for (int k = 0; k < 4; ++k) __builtin_nontemporal_store(v[k], (gvec *)(ep + k * 1024));
                } else {
#pragma unroll
                    for (int k = 0; k < 4; ++k) v[k] = __builtin_nontemporal_load((const gvec *)(ep + k * 1024));
                    if (OP == kSnapshot) {
#pragma unroll
                        for (int k = 0; k < 4; ++k) __builtin_nontemporal_store(v[k], (gvec *)(ip + k * 1024));
                    }
                }
                if (HASH) {
#pragma unroll
                    for (int k = 0; k < 4; ++k) hl ^= seg_hash(v[k], jg0 + (uint64_t)k * kSegStrideG);
                }
            } else {
                // ragged last block and/or unaligned entry
#pragma unroll
                for (int k = 0; k < 4; ++k) {
                    const uint32_t p = boff + k * 1024 + lane * 16;  // chunk-relative
                    const uint32_t valid = p >= c.len ? 0u : min(16u, c.len - p);
                    u32x4 v;
                    if (OP == kRestore) {
                        v = keep_bytes(*(const gvec *)(ip + k * 1024), valid);
                        store_part(ep + k * 1024, v, valid, aligned);
                    } else {
                        v = load_part(ep + k * 1024, valid, aligned);
                        if (OP == kSnapshot) *(gvec *)(ip + k * 1024) = v;
                    }
                    if (HASH) {
                        const uint64_t jg = jg0 + (uint64_t)k * kSegStrideG;
                        uint64_t w0 = (uint64_t)v.x | ((uint64_t)v.y << 32);
                        uint64_t w1 = (uint64_t)v.z | ((uint64_t)v.w << 32);
                        if (valid > 0) hl ^= mix64(w0 ^ jg);
                        if (valid > 8) hl ^= mix64(w1 ^ (jg + kG));
                    }
                }
            }

            if (HASH) {
                const uint64_t hb = wave_xor64(hl);
                tacc ^= hb;
                if (lane == 0) {
                    const uint64_t gblk = (c.img >> 12) + b;
                    if (h.blk) h.blk[gblk] = hb;
                    if (h.expected && h.expected[gblk] != hb) {
                        const uint64_t at = atomicAdd((unsigned long long *)h.mm_count, 1ull);
                        if (h.mm_list && at < h.mm_cap) h.mm_list[at] = gblk;
                    }
                }
            }
        }

        if (HASH && h.ten) {
            if (lane == 0) wave_part[wave] = tacc;
            __syncthreads();
            if (threadIdx.x == 0) {
                uint64_t t = 0;
#pragma unroll
                for (int w = 0; w < kThreads / 64; ++w) t ^= wave_part[w];
                if (t) atomicXor((unsigned long long *)(h.ten + c.entry), (unsigned long long)t);
            }
            __syncthreads();
        }
    }
}

__global__ void __launch_bounds__(kThreads)
k_prologue(uint64_t *__restrict__ ten, uint64_t n, uint64_t *__restrict__ mm_count)
{
    const uint64_t tid = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const uint64_t stride = (uint64_t)gridDim.x * blockDim.x;
    if (ten)
        for (uint64_t i = tid; i < n; i += stride) ten[i] = 0;
    if (mm_count && tid == 0) *mm_count = 0;
}

constexpr uint64_t kMaxGrid = 1u << 20;

template <int OP, bool HASH>
hipError_t launch_t(const Chunk *chunks, uint64_t first, uint64_t count, uint8_t *img_base,
                    uint64_t img_origin, const HashOut &h, hipStream_t s)
{
    const uint64_t grid = count < kMaxGrid ? count : kMaxGrid;
    hipLaunchKernelGGL((k_stream<OP, HASH>), dim3((uint32_t)grid), dim3(kThreads), 0, s, chunks + first, count,
                       (gbyte *)img_base, img_origin, h);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_prologue(const HashOut &h, uint64_t n_entries, hipStream_t s)
{
    uint64_t *ten = h.ten;
    uint64_t *cnt = h.expected ? h.mm_count : nullptr;
    if (!ten && !cnt) return hipSuccess;
    uint64_t items = ten ? n_entries : 1;
    uint64_t grid = (items + kThreads - 1) / kThreads;
    if (grid == 0) grid = 1;
    if (grid > 4096) grid = 4096;
    hipLaunchKernelGGL(k_prologue, dim3((uint32_t)grid), dim3(kThreads), 0, s, ten, ten ? n_entries : 0, cnt);
    return hipGetLastError();
}

hipError_t launch_stream(int op, bool hash, const Chunk *chunks, uint64_t first, uint64_t count,
                         uint8_t *img_base, uint64_t img_origin, const HashOut &h, hipStream_t s)
{
    if (count == 0) return hipSuccess;
    switch (op * 2 + (hash ? 1 : 0)) {
    case kRestore * 2: return launch_t<kRestore, false>(chunks, first, count, img_base, img_origin, h, s);
    case kRestore * 2 + 1: return launch_t<kRestore, true>(chunks, first, count, img_base, img_origin, h, s);
    case kSnapshot * 2: return launch_t<kSnapshot, false>(chunks, first, count, img_base, img_origin, h, s);
    case kSnapshot * 2 + 1: return launch_t<kSnapshot, true>(chunks, first, count, img_base, img_origin, h, s);
    case kVerify * 2 + 1: return launch_t<kVerify, true>(chunks, first, count, img_base, img_origin, h, s);
    default: return hipErrorInvalidValue;
    }
}

}  // namespace gms
