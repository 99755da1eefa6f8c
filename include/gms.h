/*
 * libgms: packed device-state image, restore and verify on one AMD Instinct
 * MI355X (gfx950).
 *
 * An engine's GPU-resident state (weight tensors and a fixed pool of mutable
 * state such as live KV blocks) is described by a manifest of device address
 * ranges.  gms_snapshot gathers those ranges into one packed image,
 * gms_restore scatters an image (device-resident or in pinned host memory)
 * back into the ranges, and gms_verify hashes the live ranges so that
 * surviving allocations can be checked before they are reattached.
 *
 * Where the operations come from (arXiv 2609.25451):
 *  - Capture stages the engine's remaining device state into host memory and
 *    recovery reverses the steps, re-creating the allocations
 *    (section 3.1, Snapshots, capture steps 3-4 and restore).  The data
 *    transfer part of recovery is about S / B_eff for an artifact of size S
 *    (section 3.1); the library exists to drive B_eff to the HBM or host-link
 *    limit, which the paper leaves as future work (section 6, Limitations).
 *  - The manifest is the recorded tensor layout a GMS client captures before
 *    commit (section 4, GMS implementation).
 *  - Verify serves the reattach of surviving allocations by a replacement
 *    engine (section 3.2, GMS): a schedulable device and the absence of fault
 *    reports do not show that resident state is intact (section 2.2).
 *  - Restoring only the live blocks of a fixed private pool follows the
 *    shadow engine's fixed runtime pool (section 5.3) and KV pages that stay
 *    reattachable (section 6, Preserving KV state).
 *
 * Image layout (the paper fixes none; this is the library's definition):
 *   entries keep the caller's order; entry i occupies image bytes
 *   [img_off[i], img_off[i] + roundup(n_i, 4096)), img_off[0] = 0,
 *   img_off[i+1] = img_off[i] + roundup(n_i, 4096); bytes past n_i in that
 *   slot are zero after a snapshot.  There is no in-band header: the manifest
 *   and the hashes travel beside the image.
 *
 * Hash (the paper fixes none; this is the library's definition):
 *   all integers little-endian, arithmetic mod 2^64,
 *   G = 0x9E3779B97F4A7C15, mix(z) = splitmix64's output function
 *   (z ^= z>>30; z *= 0xBF58476D1CE4E5B9; z ^= z>>27; z *= 0x94D049BB133111EB;
 *   z ^= z>>31).  W_i[j] = bytes 8j..8j+7 of entry i, bytes past n_i read as 0,
 *   j < ceil(n_i/8) the entry-relative word index.
 *   Block hash Hb(i,b) = XOR of mix(W_i[j] ^ j*G) over the words of 4 KiB block
 *   b (the last block only its real words); it is stored at global block index
 *   blk_base[i] + b, blk_base[i] = img_off[i] / 4096.
 *   Tensor hash Ht(i) = XOR_b Hb(i,b); an empty entry hashes to 0.
 *   mix is a bijection, so any change confined to one 8-byte word changes that
 *   block's hash.
 *
 * Conventions for every data-plane call (gms_snapshot, gms_restore,
 * gms_verify):
 *  - Asynchronous on `stream` (a hipStream_t passed as void*, NULL = the
 *    device's null stream); outputs are valid once the stream has drained.
 *    The call returns after enqueueing; argument errors are reported before
 *    anything is enqueued.
 *  - Device pointers must be hipMalloc'd memory of the manifest's device
 *    (sub-ranges of a caching allocator's blocks are fine); the library checks
 *    every range against its allocation and returns GMS_ERR_INVALID if it
 *    falls outside one.  The image base must be 16-byte aligned; entries may
 *    start at any byte address (entries off a 16-byte boundary are moved by
 *    byte-shifting kernels with the same 16-byte accesses, and no byte outside
 *    an entry is written).
 *  - Hash/mismatch arrays are uint64_t device arrays: blk_hash has
 *    gms_num_blocks() entries, ten_hash gms_num_entries(), mismatch_count one,
 *    mismatch_list min(mismatch_cap, gms_num_blocks()) (a call records each
 *    block at most once).  Every output pointer may be NULL unless
 *    stated otherwise; with all of them NULL the call is a plain copy.
 *  - A verify mismatch is not an error: the call returns GMS_OK and the count
 *    is > 0.  The mismatch list holds min(count, cap) global block indices in
 *    an unspecified order (sort it for a unique result).
 *  - Calls on one manifest that use the pinned-host staging ring are ordered
 *    by the library; other calls that write the same memory from different
 *    streams race, as any two kernels would.
 *  - Snapshot, restore and verify on device images only launch kernels on
 *    `stream` (the zeroing of outputs included), so they can be captured into
 *    a HIP graph and replayed; each replay recomputes every output.  Calls on
 *    pinned-host images, the image-file calls and the store's verifications
 *    return GMS_ERR_STATE while `stream` is capturing, and record nothing.
 *  - No exception, abort or hipMalloc failure crosses the ABI: each call
 *    returns a status; gms_last_error() gives the calling thread's last
 *    message.
 */
#ifndef GMS_H
#define GMS_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define GMS_BLOCK_BYTES 4096u
#define GMS_DEFAULT_CHUNK_BYTES (64u * 1024u)
#define GMS_DEFAULT_SLICE_BYTES (256ull << 20) /* staging ring slice (gms_manifest_set_staging) */
#define GMS_DEFAULT_SLOTS 2u                   /* staging ring device slots */
#define GMS_HOST_ONLY (-1)

/* One device address range of engine state: [addr, addr + nbytes). */
typedef struct gms_entry {
    uint64_t addr;
    uint64_t nbytes;
} gms_entry;

/* Opaque; owns the layout, the device-side work list and the staging ring. */
typedef struct gms_manifest gms_manifest;

enum gms_status {
    GMS_OK = 0,
    GMS_ERR_INVALID = -1, /* bad pointer, size, alignment, kind or device  */
    GMS_ERR_OVERLAP = -2, /* two non-empty entries share bytes             */
    GMS_ERR_SIZE = -3,    /* image (or output array) smaller than required */
    GMS_ERR_HIP = -4,     /* a HIP runtime call failed (see last error)     */
    GMS_ERR_NOMEM = -5,   /* host or device allocation failed              */
    GMS_ERR_STATE = -6,   /* call not allowed in the object's current state
                             (host-only manifest; store lease protocol)     */
    GMS_ERR_IO = -7,      /* a file could not be opened, read or written   */
    GMS_ERR_INTEGRITY = -8 /* store: contents differ from their hashes      */
};

enum gms_mem_kind {
    GMS_MEM_DEVICE = 0,      /* image is device memory of the manifest's GPU       */
    GMS_MEM_HOST_PINNED = 1  /* image is pinned host memory (hipHostMalloc / torch
                                pin_memory), moved through the staging ring       */
};

/*
 * Build a manifest over `n` entries (caller order is the image order).
 *  entries      host array of n ranges; zero-length entries are allowed and
 *               occupy no image bytes.
 *  device       HIP device ordinal that owns every range, or GMS_HOST_ONLY for
 *               a manifest that only answers layout queries (no HIP call is
 *               made; data-plane calls return GMS_ERR_STATE).
 *  chunk_bytes  work-item size: entries are cut at image offsets that are
 *               multiples of it; 0 selects GMS_DEFAULT_CHUNK_BYTES; otherwise a
 *               multiple of 4096 in [4096, 64 MiB].
 *  out          receives the manifest (caller frees with gms_manifest_destroy).
 * Errors: GMS_ERR_INVALID (NULL pointers, n >= 2^32, address overflow, a range
 * that is not inside one allocation of `device`), GMS_ERR_OVERLAP, GMS_ERR_NOMEM,
 * GMS_ERR_HIP.  Synchronous (uploads the work list).
 */
int gms_manifest_create(const gms_entry *entries, uint64_t n, int device, uint64_t chunk_bytes,
                        gms_manifest **out);

/* Frees the manifest and its device work list / staging ring.  NULL is a no-op.
 * The caller must have drained every stream that still uses the manifest. */
void gms_manifest_destroy(gms_manifest *m);

/* Layout queries (valid for host-only manifests too; 0 for NULL). */
uint64_t gms_num_entries(const gms_manifest *m);
uint64_t gms_payload_bytes(const gms_manifest *m); /* sum of n_i                 */
uint64_t gms_image_bytes(const gms_manifest *m);   /* sum of roundup(n_i, 4096)  */
uint64_t gms_num_blocks(const gms_manifest *m);    /* sum of ceil(n_i / 4096)    */
uint64_t gms_num_chunks(const gms_manifest *m);    /* work items                 */
/* Kernel launches per data-plane call on a device image.  Chunks that need
 * far fewer work units than the largest (tiny entries beside large ones) are
 * launched apart once the idle units they would otherwise leave outweigh a
 * launch; a manifest of similar chunks is one launch. */
uint64_t gms_num_launch_groups(const gms_manifest *m);
/* Launch group g (0 <= g < gms_num_launch_groups): its chunks, its work units per
 * chunk as a power of two (0: one unit per chunk, a paired launch), and flags:
 * GMS_GROUP_SHIFTED (entries off a 16-byte boundary, the byte-shifting kernels) and
 * GMS_GROUP_STRIPED (restores and snapshots take the striped unit order, as verify
 * always does: the group's chunks span several work units and are mostly entries of
 * their own, such as a KV pool's live units).  Outputs may be NULL.
 * Errors: GMS_ERR_INVALID (manifest null, g out of range). */
enum gms_group_flags {
    GMS_GROUP_SHIFTED = 1,
    GMS_GROUP_STRIPED = 2
};
int gms_launch_group(const gms_manifest *m, uint64_t g, uint64_t *chunks_out, uint32_t *unit_shift_out,
                     uint32_t *flags_out);
int gms_manifest_device(const gms_manifest *m);

/* Copies img_off[n] and blk_base[n] (host arrays; either may be NULL). */
int gms_layout(const gms_manifest *m, uint64_t *img_off, uint64_t *blk_base);

/*
 * Staging ring: `slots` device buffers of `slice_bytes` (rounded down to a
 * multiple of the chunk size, at least one chunk).  A restore from a pinned
 * host image copies host slices into free slots with a copy kernel on a
 * library-owned copy stream (a kernel rather than a DMA engine, whose rate
 * drops for up to a second after device memory is remapped or re-allocated)
 * while the scatter kernel drains filled slots on the caller's stream; with
 * slots == 0 it reads the pinned image directly over the host link
 * (zero-copy) instead.  A snapshot into pinned host memory runs the other
 * way: the gather kernel fills a slot on the caller's stream and the copy
 * stream copies it to the host image (hipMemcpyAsync); with slots == 0, or
 * slices below 128 MiB (where those copies lose half the link and more), it writes the
 * image zero-copy.  The image-file and host-image calls also use the ring (and
 * a pinned host ring of twice the slots) and need slots > 0.  slice_bytes is 0, which selects
 * GMS_DEFAULT_SLICE_BYTES, or in [4096, 64 GiB]; slots at most 16; a new manifest starts with GMS_DEFAULT_SLICE_BYTES x
 * GMS_DEFAULT_SLOTS (256 MiB slices keep the host link at about 99% of its
 * peak; 64 MiB slices reach about 97.5%).  Takes effect at the next ring
 * call; frees the old rings after draining them.  Synchronous.
 */
int gms_manifest_set_staging(gms_manifest *m, uint64_t slice_bytes, uint32_t slots);

/*
 * Snapshot (gather): image[img_off[i] + k] = entry_i[k] for k < n_i, zero in
 * the rest of each slot.  Optionally emits the block / tensor hashes of the
 * gathered bytes in the same pass (the expected hashes for later checks).
 *  image, image_bytes, image_kind  destination image (>= gms_image_bytes).
 *  blk_hash_out, ten_hash_out      optional device outputs.
 * Errors: GMS_ERR_STATE, GMS_ERR_INVALID, GMS_ERR_SIZE, GMS_ERR_HIP, GMS_ERR_NOMEM.
 */
int gms_snapshot(const gms_manifest *m, void *image, uint64_t image_bytes, int image_kind,
                 uint64_t *blk_hash_out, uint64_t *ten_hash_out, void *stream);

/*
 * Restore (scatter): entry_i[k] = image[img_off[i] + k] for k < n_i.  No other
 * byte of any allocation is written.  With hashing requested the words are
 * hashed in registers as they are stored (no extra HBM traffic): the block
 * hashes of the restored bytes go to blk_hash_out, the tensor hashes to
 * ten_hash_out, and if expected_blk is given each block is compared with it;
 * mismatching global block indices are counted in *mismatch_count_out
 * (required when expected_blk is set; zeroed by the call) and up to
 * mismatch_cap of them, in any order, written to mismatch_list_out.
 * Errors: as gms_snapshot.
 */
int gms_restore(const gms_manifest *m, const void *image, uint64_t image_bytes, int image_kind,
                const uint64_t *expected_blk, uint64_t *blk_hash_out, uint64_t *ten_hash_out,
                uint64_t *mismatch_count_out, uint64_t *mismatch_list_out, uint64_t mismatch_cap,
                void *stream);

/*
 * Verify (read-only): hashes the live entries in place.  Outputs as
 * gms_restore; at least one of blk_hash_out, ten_hash_out, expected_blk must be
 * given.  Verifying an image needs no separate call: a manifest whose entries
 * are image + img_off[i] with the same sizes hashes identically.
 * Errors: GMS_ERR_STATE, GMS_ERR_INVALID, GMS_ERR_HIP.
 */
int gms_verify(const gms_manifest *m, const uint64_t *expected_blk, uint64_t *blk_hash_out,
               uint64_t *ten_hash_out, uint64_t *mismatch_count_out, uint64_t *mismatch_list_out,
               uint64_t mismatch_cap, void *stream);

/*
 * For callers that cannot allocate (code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc): gms_restore from a pinned host image without any
 * allocation.  gms_restore's staging ring is allocated on first use; here the staging area
 * is a fixed device array of GMS_NOALLOC_STAGING_BYTES that the library holds on each
 * device it runs on until the process ends, and every step runs on `stream`: each slice
 * of the image (staging_bytes rounded down to whole chunks of the manifest; 0 = the whole
 * area) is copied into the area by a kernel reading the pinned image over the host link,
 * then scattered, hashed and compared by the kernels of gms_restore.  Arguments, outputs
 * and results are those of gms_restore with image_kind GMS_MEM_HOST_PINNED; no hipMalloc,
 * hipFree, stream or event is created, and only kernels are enqueued on `stream`, so the
 * call can be captured into a HIP graph (each replay reads the pinned image anew) after
 * one call outside capture on the device; on a manifest that an earlier staging-ring call
 * used, a capturing call returns GMS_ERR_STATE (the graph could not wait for it).  The
 * area is shared by every call on a device: calls that overlap on one device (different
 * streams or threads) race, so a caller serializes them, for example on one stream.
 * Errors: as gms_restore, plus GMS_ERR_SIZE for staging_bytes above
 * GMS_NOALLOC_STAGING_BYTES or below the manifest's chunk size.
 */
#define GMS_NOALLOC_STAGING_BYTES (64ull << 20)
int gms_restore_pinned_noalloc(const gms_manifest *m, const void *image, uint64_t image_bytes,
                               uint64_t staging_bytes, const uint64_t *expected_blk, uint64_t *blk_hash_out,
                               uint64_t *ten_hash_out, uint64_t *mismatch_count_out,
                               uint64_t *mismatch_list_out, uint64_t mismatch_cap, void *stream);

/* Flags of the image-file calls. */
enum gms_file_flags {
    GMS_FILE_DIRECT = 1, /* O_DIRECT I/O (bypasses the page cache) when the file system and
                            the offset (multiple of 4096) allow it, buffered I/O otherwise */
    GMS_FILE_SYNC = 2    /* snapshot: fsync the file before returning                      */
};

/*
 * Cold repopulation from storage (paper section 3.3 and section 4: a
 * replacement's model state is re-read from storage while its runtime is
 * restored; section 3.1: the transfer costs S / B_eff).  The file holds the
 * packed image (the layout above, no header) starting at `file_offset`.
 * `io_threads` workers (0 = 16) read the image in pieces (16 MiB with
 * O_DIRECT, 64 MiB or one slice buffered), in file order, into the slices of
 * a pinned host ring; the copy kernel moves each full slice into
 * a device slot on the manifest's copy stream and it is scattered (and hashed /
 * compared, as gms_restore) by the kernel on `stream`; a host slot is refilled
 * once the copy out of it has finished.  The call returns when every slice has been read
 * and enqueued; device work completes on `stream`.  The first file call
 * allocates the manifest's pinned host ring: 2 x slots (at most 16) slices.
 * Errors: as gms_restore, plus GMS_ERR_IO (open/read failure) and
 * GMS_ERR_SIZE (file shorter than file_offset + gms_image_bytes), and
 * GMS_ERR_INVALID for a file_offset no file can reach.  After an
 * I/O error, slices already read may have been restored (and counted in the
 * hash outputs): the entries and outputs are then partial and must not be
 * used; the manifest stays usable.
 */
int gms_restore_from_file(const gms_manifest *m, const char *path, uint64_t file_offset, uint32_t flags,
                          uint32_t io_threads, const uint64_t *expected_blk, uint64_t *blk_hash_out,
                          uint64_t *ten_hash_out, uint64_t *mismatch_count_out, uint64_t *mismatch_list_out,
                          uint64_t mismatch_cap, void *stream);

/*
 * Writes the packed image to `path` (created or truncated): the kernel gathers
 * each slice into a slot of the pinned host ring (through a device slot and a
 * device-to-host copy when slices are 128 MiB or more) and `io_threads` workers
 * (0 = 16) write its 16 MiB pieces with pwrite; optionally emits the
 * block / tensor hashes of the gathered bytes.  Synchronous: the file is
 * complete when the call returns (durable too with GMS_FILE_SYNC).
 * Errors: GMS_ERR_STATE, GMS_ERR_INVALID, GMS_ERR_IO, GMS_ERR_HIP, GMS_ERR_NOMEM.
 */
int gms_snapshot_to_file(const gms_manifest *m, const char *path, uint32_t flags, uint32_t io_threads,
                         uint64_t *blk_hash_out, uint64_t *ten_hash_out, void *stream);

/*
 * The packed image in ordinary host memory (pageable, or any host memory the
 * calling process can read and write).  A process snapshot stages device
 * state in the host memory of the checkpointed process and reinstates it on
 * restore (paper section 3.1); the paper's checkpoint tool copies it back
 * serially without saturating PCIe (section 5.2).  Here `threads` workers
 * (0 = 16) copy 16 MiB pieces between `image` and the slots of the pinned host
 * ring, and each slice goes through a device slot and the kernel as in
 * gms_restore_from_file; no part of `image` has to be pinned.
 *
 * gms_restore_from_host returns when every slice has been copied out of
 * `image` and enqueued (the caller may then reuse `image`); device work and
 * the hash / mismatch outputs complete on `stream`, as gms_restore.
 * gms_snapshot_to_host is synchronous: `image` holds the packed image (zero
 * padding included) when it returns, and the optional hashes are complete.
 * `image` is host memory of at least gms_image_bytes(m) bytes (NULL allowed
 * for an empty layout); the library cannot check pageable memory beyond
 * that, so a shorter or unmapped buffer is undefined behaviour.  Device
 * memory is refused (GMS_ERR_INVALID: use gms_restore / gms_snapshot).
 * Errors: GMS_ERR_STATE (host-only manifest, no staging slots, or `stream`
 * capturing a graph), GMS_ERR_INVALID, GMS_ERR_SIZE (image_bytes below the layout), GMS_ERR_HIP,
 * GMS_ERR_NOMEM (staging rings).
 */
int gms_restore_from_host(const gms_manifest *m, const void *image, uint64_t image_bytes, uint32_t threads,
                          const uint64_t *expected_blk, uint64_t *blk_hash_out, uint64_t *ten_hash_out,
                          uint64_t *mismatch_count_out, uint64_t *mismatch_list_out, uint64_t mismatch_cap,
                          void *stream);
int gms_snapshot_to_host(const gms_manifest *m, void *image, uint64_t image_bytes, uint32_t threads,
                         uint64_t *blk_hash_out, uint64_t *ten_hash_out, void *stream);

/*
 * Device memory pool over HIP virtual memory (paper section 4: a first-fit
 * suballocator over 2 GiB slabs, with dedicated slabs for larger allocations,
 * so that mapping and access changes happen per slab rather than per tensor;
 * section 3.2: shared state is mapped read-only for readers; sections 3.1 and
 * 3.3: KV pages are released before a checkpoint while their virtual
 * addresses stay reserved, and fresh pages are mapped at the same addresses
 * after restore).  A mapping (a slab, or a dedicated mapping for an
 * allocation larger than a slab) is the unit of release, remap and access
 * change; each holds a VA reservation of its own, placed one after another in
 * a window of `va_bytes` while the address space allows (so consecutive
 * allocations are contiguous), and together they hold at most `va_bytes` of
 * VA.  Addresses handed out stay valid until freed, across release and
 * remap, and can be used in manifests like any device allocation.  The caller must not let
 * kernels (including snapshot/restore/verify) touch a released range; release
 * synchronises the device first.  Not for use under graph capture.
 */
typedef struct gms_pool gms_pool;

/* A pool on `device` with a VA budget (and placement window) of va_bytes; slab_bytes
 * 0 = 2 GiB.  Both must be multiples of the allocation granularity (gms_pool_info).
 * Errors: GMS_ERR_INVALID, GMS_ERR_STATE (no VMM support), GMS_ERR_NOMEM, GMS_ERR_HIP. */
int gms_pool_create(int device, uint64_t va_bytes, uint64_t slab_bytes, gms_pool **out);

/* Unmaps and releases every mapping and frees the reservations.  NULL is a no-op. */
void gms_pool_destroy(gms_pool *p);

/* First fit in mapped slabs (a new slab is mapped when none fits); an allocation larger
 * than a slab gets a dedicated mapping.  align: power of two <= granularity, 0 = 256.
 * Errors: GMS_ERR_INVALID, GMS_ERR_NOMEM (reservation or device memory exhausted, or
 * bytes above the pool's VA budget). */
int gms_pool_alloc(gms_pool *p, uint64_t bytes, uint64_t align, uint64_t *addr_out);

/* Returns an allocation; a dedicated mapping is unmapped and released, with its VA,
 * after the device has finished its work.  Slab space is handed to the next allocation
 * at once, without waiting for the device: device work that still uses it must have
 * finished, or be ordered before any use of the new allocation.
 * Errors: GMS_ERR_INVALID (not an allocation of this pool). */
int gms_pool_free(gms_pool *p, uint64_t addr);

/* Releases the physical pages of the mappings that exactly tile [addr, addr+bytes),
 * keeping their VA; allocations inside keep their addresses. */
int gms_pool_release(gms_pool *p, uint64_t addr, uint64_t bytes);

/* Backs released mappings in [addr, addr+bytes) with fresh physical pages at the same
 * VA, read-write.  Contents are undefined until written. */
int gms_pool_remap(gms_pool *p, uint64_t addr, uint64_t bytes);

/* Device access to the mapped mappings tiling [addr, addr+bytes): read_only != 0 maps
 * them read-only, 0 read-write.  A switch to read-only first synchronizes the device, so
 * writes that work on any stream still has in flight land before the pages turn read-only.
 * Errors: GMS_ERR_INVALID, GMS_ERR_STATE (released). */
int gms_pool_set_access(gms_pool *p, uint64_t addr, uint64_t bytes, int read_only);

/* Pool facts (base: start of the placement window; reserved: the VA budget); any output
 * may be NULL. */
int gms_pool_info(const gms_pool *p, uint64_t *base, uint64_t *reserved, uint64_t *mapped_bytes,
                  uint64_t *mappings, uint64_t *granularity);

/* The mapping holding addr: its start, size and whether it is currently backed. */
int gms_pool_mapping_of(const gms_pool *p, uint64_t addr, uint64_t *map_addr, uint64_t *map_bytes,
                        int *mapped);

/*
 * Model-state store: the ownership protocol of paper section 3.2 (Figure 4,
 * the GMS model-state state machine) over a pool of this library.
 *
 * States:
 *  EMPTY      no layout.
 *  RW         one writer holds the exclusive read-write lease and populates
 *             allocations it makes through the store.
 *  COMMITTED  committed state, immutable, no readers.
 *  RO         committed state with one or more read-only leases.
 *
 * Transitions:
 *  EMPTY or COMMITTED --connect_rw--> RW (refused while readers hold
 *  leases or another writer does; from COMMITTED the writer reuses the
 *  allocation set and its mappings become writable again).
 *  RW --commit--> COMMITTED: records the layout (a manifest over the
 *  entries given), hashes every 4 KiB block of it and maps every pool
 *  mapping read-only, so device writes into committed state fault instead
 *  of changing it.
 *  RW --abort, or the writer disconnecting before commit--> EMPTY: discards
 *  the incomplete state (every allocation, and its physical memory).
 *  COMMITTED or RO --connect_ro--> RO.  RO --disconnect--> RO, or COMMITTED
 *  after the last reader.  A reader's disconnect leaves committed state
 *  intact.
 *
 * Integrity: with GMS_CONNECT_VERIFY, connect_ro first re-hashes the
 * committed state and compares it with the hashes recorded at commit; any
 * mismatch refuses the lease with GMS_ERR_INTEGRITY and marks the state
 * invalid (section 3.2: integrity errors invalidate GMS state).  An invalid
 * state grants no read-only lease; once no reader holds one, a writer may
 * reconnect, repopulate the same allocations (for example with gms_restore
 * from an image) and commit again, which makes it valid.
 *
 * In one process the store's pool is the engine's own mapping of the
 * allocations; gms_owner_* and gms_client_* below run the same protocol across
 * processes.  A store made with device GMS_HOST_ONLY runs the
 * protocol alone, without memory (no allocations; commit takes no entries).
 * Store calls are thread-safe and synchronous: each returns after the device
 * work it enqueues on `stream` has finished.  Leases are non-zero ids, valid
 * until released; a stale or foreign id is GMS_ERR_INVALID, a call not
 * allowed in the current state is GMS_ERR_STATE.
 */
typedef struct gms_store gms_store;

enum gms_store_state {
    GMS_STORE_EMPTY = 0,
    GMS_STORE_RW = 1,
    GMS_STORE_COMMITTED = 2,
    GMS_STORE_RO = 3
};

/* Flags of gms_store_connect_ro. */
enum gms_connect_flags {
    GMS_CONNECT_VERIFY = 1 /* re-hash the committed state and refuse the lease on any mismatch */
};

/* A store with its own pool (gms_pool_create's arguments); device GMS_HOST_ONLY makes a
 * protocol-only store.  Errors: as gms_pool_create. */
int gms_store_create(int device, uint64_t va_bytes, uint64_t slab_bytes, gms_store **out);

/* Frees the committed layout, every allocation and the pool, whatever leases are held.
 * NULL is a no-op. */
void gms_store_destroy(gms_store *s);

/* Current state, reader count and whether the committed state is invalid; outputs may be NULL. */
int gms_store_state(const gms_store *s, int *state, uint32_t *readers, int *invalid);

/* The store's pool, for queries (gms_pool_info, gms_pool_mapping_of); NULL if host-only.
 * Its mutating calls bypass the protocol. */
gms_pool *gms_store_pool(gms_store *s);

/* Exclusive read-write lease.  Errors: GMS_ERR_STATE (a writer or readers are connected). */
int gms_store_connect_rw(gms_store *s, uint64_t *lease_out);

/* Writer only: an allocation in the store's pool (as gms_pool_alloc), or its return. */
int gms_store_alloc(gms_store *s, uint64_t lease, uint64_t bytes, uint64_t align, uint64_t *addr_out);
int gms_store_free(gms_store *s, uint64_t lease, uint64_t addr);

/*
 * Writer only: commits entries[0..n) (each inside one allocation of the store) as the
 * layout: synchronizes the device (so device work of the writer on any stream has
 * finished), hashes the layout's blocks and maps the pool read-only; the lease ends.  With
 * expected_blk (device, one u64 per block of the layout, as gms_snapshot writes them) the
 * populated contents must match it: on any mismatch the commit is refused with
 * GMS_ERR_INTEGRITY, *mismatch_count_out (host, may be NULL) holds the count, and the
 * writer keeps its lease.  Errors: GMS_ERR_INVALID (lease, entries), GMS_ERR_OVERLAP,
 * GMS_ERR_INTEGRITY, GMS_ERR_HIP, GMS_ERR_NOMEM.
 */
int gms_store_commit(gms_store *s, uint64_t lease, const gms_entry *entries, uint64_t n,
                     const uint64_t *expected_blk, uint64_t *mismatch_count_out, void *stream);

/* Writer only: discards the incomplete state (EMPTY); the lease ends. */
int gms_store_abort(gms_store *s, uint64_t lease);

/* Read-only lease on committed state.  flags: GMS_CONNECT_VERIFY.  *mismatch_count_out
 * (host, may be NULL) receives the blocks that failed verification.  Errors:
 * GMS_ERR_STATE (no committed state, or a writer is connected), GMS_ERR_INTEGRITY. */
int gms_store_connect_ro(gms_store *s, uint32_t flags, uint64_t *lease_out, uint64_t *mismatch_count_out,
                         void *stream);

/* Re-hashes the committed state against its commit-time hashes: *mismatch_count_out (host)
 * gets the count and mismatch_list_out (device, may be NULL) up to `cap` global block
 * indices, in any order.  A mismatch marks the state invalid but is not an error.
 * Errors: GMS_ERR_STATE (nothing committed), GMS_ERR_HIP. */
int gms_store_verify(gms_store *s, uint64_t *mismatch_count_out, uint64_t *mismatch_list_out, uint64_t cap,
                     void *stream);

/* Ends a lease: a reader's leaves committed state intact; a writer's before commit is an
 * abort. */
int gms_store_disconnect(gms_store *s, uint64_t lease);

/* The committed layout (a manifest of the store) and its block hashes (device, one u64 per
 * block); NULL while nothing is committed.  Valid until the next writer connects. */
const gms_manifest *gms_store_layout(const gms_store *s);
const uint64_t *gms_store_block_hashes(const gms_store *s);

/*
 * The model-state store across processes (paper section 3.2, GMS and Figure 4; section 4:
 * a GMS process per GPU owns the allocations and exports them as POSIX file descriptors over
 * a Unix-domain socket, so that an engine's crash cannot take them with it).
 *
 * Owner.  gms_owner_create binds a Unix-domain socket at `socket_path` (an existing socket
 * file there is replaced) for `device`; gms_owner_run serves clients until gms_owner_stop
 * (callable from any thread); gms_owner_destroy releases every allocation and removes the
 * socket file.  The owner creates device memory with HIP virtual memory and never maps it;
 * each allocation (at most GMS_IPC_PIECE_BYTES) travels as one dma-buf descriptor.  It runs
 * the states and transitions of the in-process store above: one writer, then COMMITTED;
 * readers; a writer's connection that closes before commit (disconnect, abort or the
 * process's death) discards every allocation (EMPTY); a reader's connection that closes
 * ends only its lease.  An owner made with device GMS_HOST_ONLY runs the protocol alone,
 * without memory.
 *
 * Clients.  gms_client_connect opens a lease: GMS_LEASE_RW (exclusive; from EMPTY, or from
 * COMMITTED reusing the allocation set) or GMS_LEASE_RO (on committed state).  The client
 * maps every allocation as external memory (hipImportExternalMemory of the descriptor):
 * on this ROCm a virtual-memory handle cannot be imported by a process other than its
 * exporter, so the mappings carry no access flags; a reader's read-only use is this
 * library's contract (nothing here writes through a reader's mapping) and readers verify
 * the state before they use it.  A writer takes memory with gms_client_alloc (first fit in
 * slabs of GMS_IPC_PIECE_BYTES; a request above half a slab gets an allocation of its own;
 * GMS_ERR_SIZE above GMS_IPC_PIECE_BYTES), populates it, and commits entries (each inside
 * one of its allocations): the library synchronizes the device (every write of the writer
 * process, on any stream, has landed), hashes every 4 KiB block of them (and compares with
 * expected_blk when given, refusing the commit on a mismatch with GMS_ERR_INTEGRITY while
 * the writer keeps its lease), and the owner records the layout and the hashes; the write
 * lease ends (the writer must not write after it) and the client's layout is emptied (as the
 * paper's writer does, it reconnects read-only to use the committed state).  A client's
 * layout is the committed entries at its own addresses (gms_client_layout,
 * gms_client_manifest for gms_restore / gms_verify; empty before the first commit): a
 * reader's to use, a writer's to repopulate.  A writer that took over committed state gets
 * its slabs back with the committed entries as their allocated parts (the rest free), and
 * freeing memory that a committed entry uses drops the client's layout and manifest (no
 * later call can then reach the freed memory through them).  With GMS_CONNECT_VERIFY a reader re-hashes
 * the layout against the commit-time hashes before the lease is granted, and any mismatch
 * refuses the lease (GMS_ERR_INTEGRITY, the count in *mismatch_count_out) and invalidates
 * the committed state at the owner until a writer commits again.  gms_client_verify
 * re-hashes later (a mismatch invalidates the state; the reader keeps its lease).
 * gms_client_disconnect unmaps everything and ends the lease.  Client calls are
 * synchronous and not thread-safe on one client object.
 * Errors: GMS_ERR_IO (socket), GMS_ERR_STATE (lease protocol), GMS_ERR_INTEGRITY,
 * GMS_ERR_INVALID, GMS_ERR_SIZE, GMS_ERR_NOMEM, GMS_ERR_HIP.
 */
#define GMS_IPC_PIECE_BYTES (1ull << 30)

enum gms_lease_mode {
    GMS_LEASE_RW = 1,
    GMS_LEASE_RO = 2
};

typedef struct gms_owner gms_owner;
typedef struct gms_client gms_client;

int gms_owner_create(const char *socket_path, int device, gms_owner **out);
int gms_owner_run(gms_owner *o);
void gms_owner_stop(gms_owner *o);
/* State (enum gms_store_state), reader count, invalid flag and live allocations; outputs may
 * be NULL.  gms_owner_query asks a running owner the same over its socket. */
int gms_owner_status(gms_owner *o, int *state, uint32_t *readers, int *invalid, uint64_t *allocations);
int gms_owner_query(const char *socket_path, int *state, uint32_t *readers, int *invalid, uint64_t *allocations);
void gms_owner_destroy(gms_owner *o);

int gms_client_connect(const char *socket_path, int mode, uint32_t flags, void *stream, gms_client **out,
                       uint64_t *mismatch_count_out);
/* The lease id (0 once it ended) and the owner's device; outputs may be NULL. */
int gms_client_lease(const gms_client *c, uint64_t *lease_out, int *device_out);
int gms_client_alloc(gms_client *c, uint64_t bytes, uint64_t align, uint64_t *addr_out);
int gms_client_free(gms_client *c, uint64_t addr);
int gms_client_commit(gms_client *c, const gms_entry *entries, uint64_t n, const uint64_t *expected_blk,
                      uint64_t *mismatch_count_out, void *stream);
int gms_client_abort(gms_client *c);
/* Reader: the committed entries at this process's addresses (up to cap; *n_out the count). */
int gms_client_layout(const gms_client *c, gms_entry *entries_out, uint64_t cap, uint64_t *n_out);
const gms_manifest *gms_client_manifest(const gms_client *c);
/* A manifest over entries inside this client's allocations (gms_manifest_create's arguments and
 * errors; the caller destroys it), for gms_restore into a writer's memory before its first
 * commit, or any other data-plane call on client memory: the runtime does not report the extent
 * of these mappings, so gms_manifest_create cannot check them. */
int gms_client_manifest_create(const gms_client *c, const gms_entry *entries, uint64_t n, uint64_t chunk_bytes,
                               gms_manifest **out);
const uint64_t *gms_client_block_hashes(const gms_client *c);
int gms_client_verify(gms_client *c, uint64_t *mismatch_count_out, uint64_t *mismatch_list_out, uint64_t cap,
                      void *stream);
int gms_client_disconnect(gms_client *c);

/* Static description of a status code. */
const char *gms_status_str(int status);

/* The calling thread's last error message ("" if none); valid until its next call. */
const char *gms_last_error(void);

/* ABI version of this header (2: adds the model-state store and GMS_ERR_INTEGRITY;
 * 3: adds gms_restore_from_host and gms_snapshot_to_host; 4: adds gms_restore_pinned_noalloc,
 * the owner process and its clients; 5: adds gms_launch_group). */
int gms_abi_version(void);

#ifdef __cplusplus
}
#endif

#endif /* GMS_H */
