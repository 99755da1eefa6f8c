"""Seeded random manifests through every combination the launch planner can make: chunk
sizes from 4 KiB to 1 MiB, entries at any byte alignment, sizes from one byte to a few MiB,
mixes that split into paired and unit launches and into striped and contiguous unit orders,
device images and pinned images through small staging rings.  Each case is the oracle round
trip: snapshot image and hashes, a fused restore into poisoned memory with sentinels around
every entry, and verify, all equal to the oracle; the same restore from ordinary host memory
and through the allocation-free path in slices of a random number of chunks, and for every fourth
case from an image file; then bytes flipped at random image offsets
(payload or padding) and a second fused restore, whose mismatch count and list equal the
oracle's verify of the corrupted image unpacked."""
import numpy as np
import pytest
import torch

import oracle
import paper_2609_25451_amd as gms
from gpu_util import Arena, from_u64, need_gpu, random_datas, to_u64, u64_dev
from test_gpu_parity import _round_trip

pytestmark = pytest.mark.gpu

CHUNKS = [4096, 16384, 65536, 262144, 1 << 20]


def _case(seed):
    rng = np.random.default_rng(seed)
    mix = []
    for _ in range(int(rng.integers(1, 4))):  # a few families of sizes
        kind = int(rng.integers(0, 4))
        count = int(rng.integers(1, 400))
        if kind == 0:
            mix += [int(v) for v in rng.integers(1, 9000, count)]        # paired-launch sizes
        elif kind == 1:
            mix += [int(rng.choice([16384, 32768, 65536]))] * count      # one-chunk units
        elif kind == 2:
            mix += [int(v) for v in rng.integers(9000, 300_000, count // 4 + 1)]
        else:
            mix += [int(v) for v in rng.integers(1 << 20, 6 << 20, 3)]  # entries of many chunks
    rng.shuffle(mix)
    p_mis = float(rng.choice([0.0, 0.3, 1.0]))
    chunk = int(rng.choice(CHUNKS))
    pinned = bool(rng.integers(0, 3) == 0)
    return mix, p_mis, chunk, pinned


@pytest.mark.parametrize("seed", range(24))
def test_random_manifest_round_trip(seed, tmp_path):
    need_gpu()
    sizes, p_mis, chunk, pinned = _case(1000 + seed)
    rng_slices = np.random.default_rng(5000 + seed)
    print(f"case {seed}: {len(sizes)} entries, {sum(sizes)} B, chunk {chunk}, misaligned {p_mis}, "
          f"pinned {pinned}", flush=True)
    arena = Arena(sizes, misalign=lambda r: r.integers(1, 16) if r.random() < p_mis else 0, gap=24,
                  seed=2000 + seed)
    datas = random_datas(sizes, seed=3000 + seed)
    arena.fill(datas)
    staging = (max(chunk, 1 << 20), 2) if pinned else None
    m, img = _round_trip(arena, datas, gms.MEM_HOST_PINNED if pinned else gms.MEM_DEVICE, chunk_bytes=chunk,
                       staging=staging)
    groups = m.launch_groups()
    assert sum(g["chunks"] for g in groups) == m.num_chunks
    o_img = oracle.pack(datas)
    o_blk, o_ten = oracle.hashes(datas)
    exp = from_u64(o_blk)

    def check(restore_call, what):
        arena.poison()
        blk, ten, cnt = u64_dev(m.num_blocks), u64_dev(m.num_entries), u64_dev(1)
        restore_call(blk, ten, cnt)
        torch.cuda.synchronize()
        back, whole = arena.read()
        assert all(np.array_equal(a, b) for a, b in zip(back, datas)), what
        assert arena.outside_untouched(whole), what
        assert int(to_u64(cnt)[0]) == 0, what
        assert np.array_equal(to_u64(blk, m.num_blocks), o_blk) and np.array_equal(to_u64(ten, m.num_entries), o_ten)

    # the same image from ordinary host memory (pieces through the host and device rings) ...
    m.set_staging(max(chunk, 1 << 20), 2)
    check(lambda blk, ten, cnt: gms.restore_from_host(m, o_img, expected=exp, blk_hash=blk, ten_hash=ten,
                                                      mismatch_count=cnt), "pageable host image")
    # ... and pinned through the fixed staging area, in slices of a random number of chunks
    pin = torch.from_numpy(o_img.copy()).pin_memory()
    slice_bytes = chunk * int(rng_slices.integers(1, max(2, gms.NOALLOC_STAGING_BYTES // chunk // 8)))
    check(lambda blk, ten, cnt: gms.restore_pinned_noalloc(m, pin, staging_bytes=slice_bytes, expected=exp,
                                                           blk_hash=blk, ten_hash=ten, mismatch_count=cnt),
          f"allocation-free restore, {slice_bytes} B slices")
    if seed % 4 == 0:  # an image file at an offset, direct or buffered, with a random worker count
        path = tmp_path / "image.bin"
        off = 4096 * int(rng_slices.integers(0, 4))
        with open(path, "wb") as f:
            f.write(b"\0" * off)
            f.write(o_img.tobytes())
        flags = gms.FILE_DIRECT if seed % 8 == 0 else 0
        threads = int(rng_slices.integers(1, 9))
        check(lambda blk, ten, cnt: gms.restore_from_file(m, path, file_offset=off, flags=flags, io_threads=threads,
                                                          expected=exp, blk_hash=blk, ten_hash=ten,
                                                          mismatch_count=cnt),
              f"image file, offset {off}, flags {flags}, {threads} workers")

    # corruption: flip bytes anywhere in the image, padding included (padding is neither
    # restored nor hashed, so a flip there must flag nothing)
    rng = np.random.default_rng(4000 + seed)
    host = img.cpu().numpy()[: m.image_bytes].copy() if not pinned else img.numpy()[: m.image_bytes]
    for pos in rng.integers(0, m.image_bytes, int(rng.integers(1, 6))):
        host[pos] ^= np.uint8(1 << int(rng.integers(0, 8)))
    if not pinned:
        img[: m.image_bytes].copy_(torch.from_numpy(host))
    bad = oracle.unpack(host, sizes)
    o_blk, _ = oracle.hashes(datas)
    o_cnt, o_lst = oracle.verify(bad, o_blk)
    arena.poison()
    cnt, lst = u64_dev(1), u64_dev(16)
    gms.restore(m, img, m.image_bytes, gms.MEM_HOST_PINNED if pinned else gms.MEM_DEVICE, expected=from_u64(o_blk),
                mismatch_count=cnt, mismatch_list=lst, mismatch_cap=16)
    torch.cuda.synchronize()
    back, _ = arena.read()
    assert all(np.array_equal(a, b) for a, b in zip(back, bad))
    got = int(to_u64(cnt)[0])
    assert got == o_cnt
    assert sorted(to_u64(lst)[: min(got, 16)].tolist()) == o_lst[:16].tolist()
    m.close()
