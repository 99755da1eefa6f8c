// Internal interface between the host side (gms_api.hip) and the kernels
// (gms_kernels.hip).  Not installed; the public surface is include/gms.h.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace gms {

constexpr uint32_t kBlockBytes = 4096;  // hash block and image alignment
constexpr uint32_t kBlocksPerUnit = 2;  // 4 KiB blocks per work unit (one per wave of a workgroup)
constexpr uint32_t kMaxUnitShift = 13;  // a 64 MiB chunk needs 2^13 units

// An entry of the work list: a piece of one entry that never crosses an image
// offset that is a multiple of the manifest's chunk size.
struct Chunk {
    uint64_t addr;   // device address of the piece's first byte
    uint64_t img;    // image offset of the piece's first byte (multiple of 4096)
    uint64_t off;    // entry-relative byte offset (multiple of 4096)
    uint32_t len;    // bytes of entry data in the piece (>= 1)
    uint32_t entry;  // entry index
};
static_assert(sizeof(Chunk) == 32, "Chunk is 32 bytes");

enum Op : int { kRestore = 0, kSnapshot = 1, kVerify = 2 };

struct HashOut {
    uint64_t *blk;             // block hashes by global block index, or null
    uint64_t *ten;             // tensor hashes by entry, or null
    const uint64_t *expected;  // expected block hashes, or null
    uint64_t *mm_count;        // mismatch counter (required with expected)
    uint64_t *mm_list;         // mismatch indices, or null
    uint64_t mm_cap;
    bool any() const { return blk || ten || expected; }
};

// Copies `bytes` (a multiple of 16) from `src`, pinned host memory mapped into
// the device, to device memory `dst`, with a kernel on `s` rather than a DMA
// engine.
hipError_t launch_host_copy(const uint8_t *src, uint8_t *dst, uint64_t bytes, hipStream_t s);

// Zeroes the tensor-hash array and the mismatch counter (either may be null).
hipError_t launch_prologue(const HashOut &h, uint64_t n_entries, hipStream_t s);

// Runs `op` over chunks[first, first + count), each of which needs at most
// 2^unit_shift work units of kBlocksPerUnit blocks (unit_shift <= kMaxUnitShift).
// The image byte at offset x lives at img_base + (x - img_origin).  `hash`
// selects the hashing variant; `shifted` is set when the chunks' entry
// addresses are not 16-byte aligned and clear when they all are (a launch
// never mixes the two).
hipError_t launch_stream(int op, bool hash, bool shifted, bool striped, const Chunk *chunks, uint64_t first,
                         uint64_t count, uint32_t unit_shift, uint8_t *img_base, uint64_t img_origin, const HashOut &h,
                         hipStream_t s);

}  // namespace gms
