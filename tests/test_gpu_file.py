"""Image files: snapshot to a file and cold restore from it, against the oracle.

The file holds the packed image (no header) at a given offset; restore streams
it through pinned host slots, the host link and the device ring into the
entries, hashing and comparing as the in-memory restore does.
"""
import os

import numpy as np
import pytest
import torch

import oracle
import paper_2609_25451_amd as gms
import synth
from gpu_util import Arena, from_u64, need_gpu, random_datas, to_u64, u64_dev

pytestmark = pytest.mark.gpu


def _case(seed, misalign=True):
    rng = np.random.default_rng(900 + seed)
    sizes = [int(v) for v in rng.integers(0, 300_000, 25)] + [2 << 20, 0, 13, 4096 * 3 + 1]
    arena = Arena(sizes, misalign=(lambda r: r.integers(0, 16)) if misalign else None, seed=seed)
    datas = random_datas(sizes, seed=seed + 50)
    arena.fill(datas)
    return arena, datas


@pytest.mark.parametrize("flags", [0, gms.FILE_DIRECT, gms.FILE_DIRECT | gms.FILE_SYNC])
@pytest.mark.parametrize("staging", [None, (256 * 1024, 2), (1 << 20, 3)], ids=["ring_default", "ring256K", "ring1M"])
def test_file_round_trip(tmp_path, flags, staging):
    need_gpu()
    arena, datas = _case(1)
    m = gms.Manifest(arena.entries, device=0)
    if staging:
        m.set_staging(*staging)
    path = tmp_path / "image.bin"
    blk, ten = u64_dev(m.num_blocks), u64_dev(m.num_entries)
    gms.snapshot_to_file(m, path, flags=flags, io_threads=3, blk_hash=blk, ten_hash=ten)
    torch.cuda.synchronize()
    o_img = oracle.pack(datas)
    o_blk, o_ten = oracle.hashes(datas)
    assert np.array_equal(np.fromfile(path, dtype=np.uint8), o_img), "file != oracle image"
    assert np.array_equal(to_u64(blk, m.num_blocks), o_blk) and np.array_equal(to_u64(ten, m.num_entries), o_ten)

    arena.poison()
    blk2, ten2, cnt = u64_dev(m.num_blocks), u64_dev(m.num_entries), u64_dev(1)
    cnt.fill_(5)
    gms.restore_from_file(m, path, flags=flags, io_threads=5, expected=from_u64(o_blk), blk_hash=blk2,
                          ten_hash=ten2, mismatch_count=cnt)
    torch.cuda.synchronize()
    back, whole = arena.read()
    assert all(np.array_equal(a, b) for a, b in zip(back, datas)) and arena.outside_untouched(whole)
    assert to_u64(cnt)[0] == 0
    assert np.array_equal(to_u64(blk2, m.num_blocks), o_blk) and np.array_equal(to_u64(ten2, m.num_entries), o_ten)


@pytest.mark.parametrize("io_threads", [1, 7, 64])
def test_file_pieces_and_short_slices(tmp_path, io_threads):
    """Slices of several 16 MiB pieces plus a short one, a single device slot
    (two host slots), and worker counts from one to more than there are pieces."""
    need_gpu()
    sizes = [33 << 20, 5, (21 << 20) + 12345, 0, 4096 * 7 + 3, 36 << 20]
    arena = Arena(sizes, misalign=[0, 1, 0, 0, 8, 0], seed=11)
    datas = random_datas(sizes, seed=61)
    arena.fill(datas)
    m = gms.Manifest(arena.entries, device=0)
    m.set_staging(40 << 20, 1)  # pieces 16 + 16 + 8 MiB per slice; last slice shorter
    path = tmp_path / "pieces.bin"
    blk = u64_dev(m.num_blocks)
    gms.snapshot_to_file(m, path, flags=gms.FILE_DIRECT, io_threads=io_threads, blk_hash=blk)
    torch.cuda.synchronize()
    o_img = oracle.pack(datas)
    o_blk, o_ten = oracle.hashes(datas)
    assert m.image_bytes > 2 * (40 << 20) and m.image_bytes % (40 << 20) != 0
    assert np.array_equal(np.fromfile(path, dtype=np.uint8), o_img), "file != oracle image"
    assert np.array_equal(to_u64(blk, m.num_blocks), o_blk)
    for flags in (gms.FILE_DIRECT, 0):
        arena.poison()
        ten, cnt = u64_dev(m.num_entries), u64_dev(1)
        gms.restore_from_file(m, path, flags=flags, io_threads=io_threads, expected=from_u64(o_blk), ten_hash=ten,
                              mismatch_count=cnt)
        torch.cuda.synchronize()
        back, whole = arena.read()
        assert all(np.array_equal(a, b) for a, b in zip(back, datas)) and arena.outside_untouched(whole)
        assert to_u64(cnt)[0] == 0 and np.array_equal(to_u64(ten, m.num_entries), o_ten)


@pytest.mark.parametrize("offset", [8192, 100])
def test_file_offset_and_corruption(tmp_path, offset):
    need_gpu()
    arena, datas = _case(2, misalign=False)
    m = gms.Manifest(arena.entries, device=0)
    m.set_staging(512 * 1024, 2)
    o_img = oracle.pack(datas)
    o_blk, _ = oracle.hashes(datas)
    off, _ = m.layout()
    rng = np.random.default_rng(offset)
    img = o_img.copy()
    bad = [d.copy() for d in datas]
    for _ in range(4):
        e = int(rng.integers(0, len(datas)))
        while not datas[e].size:
            e = int(rng.integers(0, len(datas)))
        byte = int(rng.integers(0, datas[e].size))
        img[off[e] + byte] ^= 0x40
        bad[e][byte] ^= 0x40
    path = tmp_path / "image_off.bin"
    with open(path, "wb") as f:
        f.write(b"\x77" * offset)
        f.write(img.tobytes())
        f.write(b"\x55" * 1000)
    want_cnt, want = oracle.verify(bad, o_blk)
    arena.poison()
    cnt, lst = u64_dev(1), u64_dev(16)
    gms.restore_from_file(m, path, file_offset=offset, expected=from_u64(o_blk), mismatch_count=cnt,
                          mismatch_list=lst, mismatch_cap=16)
    torch.cuda.synchronize()
    c = int(to_u64(cnt)[0])
    assert c == want_cnt and np.array_equal(np.sort(to_u64(lst, c)), want)
    back, whole = arena.read()
    assert all(np.array_equal(a, b) for a, b in zip(back, bad)) and arena.outside_untouched(whole)


def test_file_and_pinned_ring_interleave(tmp_path):
    """File and pinned-host calls share the manifest's ring; back-to-back calls on two streams."""
    need_gpu()
    seed, specs = synth.weight_set("tiny")
    ts = [torch.empty(sp.shape, dtype=torch.bfloat16, device="cuda") for sp in specs]
    for i, t in enumerate(ts):
        synth.dev_fill_bf16(t.data_ptr(), t.numel(), seed, i)
    datas = [synth.bf16_bits(sp.numel, seed, i).view(np.uint8) for i, sp in enumerate(specs)]
    m = gms.Manifest(ts, device=0)
    m.set_staging(1 << 20, 2)
    path = tmp_path / "tiny.bin"
    gms.snapshot_to_file(m, path)
    pinned = torch.empty(m.image_bytes, dtype=torch.uint8, pin_memory=True)
    s2 = torch.cuda.Stream()
    for rep in range(3):
        for t in ts:
            t.view(torch.uint8).fill_(0xA5)
        if rep % 2 == 0:
            gms.restore_from_file(m, path)
            with torch.cuda.stream(s2):
                gms.snapshot(m, pinned, m.image_bytes, gms.MEM_HOST_PINNED)
        else:
            with torch.cuda.stream(s2):
                gms.restore_from_file(m, path, flags=0)
            gms.snapshot(m, pinned, m.image_bytes, gms.MEM_HOST_PINNED)
        torch.cuda.synchronize()
        assert np.array_equal(pinned.numpy(), oracle.pack(datas))
        for t, d in zip(ts, datas):
            assert np.array_equal(t.view(torch.uint8).reshape(-1).cpu().numpy(), d)


def test_file_errors(tmp_path):
    need_gpu()
    arena, datas = _case(3, misalign=False)
    m = gms.Manifest(arena.entries, device=0)
    with pytest.raises(gms.GmsError) as e:
        gms.restore_from_file(m, tmp_path / "missing.bin")
    assert e.value.status == gms.GMS_ERR_IO
    short = tmp_path / "short.bin"
    short.write_bytes(b"\0" * (m.image_bytes - 1))
    with pytest.raises(gms.GmsError) as e:
        gms.restore_from_file(m, short)
    assert e.value.status == gms.GMS_ERR_SIZE
    with pytest.raises(gms.GmsError) as e:
        gms.snapshot_to_file(m, tmp_path / "no_such_dir" / "x.bin")
    assert e.value.status == gms.GMS_ERR_IO
    m.set_staging(0, 0)  # zero-copy manifests have no ring for files
    with pytest.raises(gms.GmsError) as e:
        gms.snapshot_to_file(m, tmp_path / "x.bin")
    assert e.value.status == gms.GMS_ERR_STATE


@pytest.mark.parametrize("seed", range(8))
def test_random_file_round_trips(tmp_path, seed):
    """Seeded random manifests through image files: ring geometry (slice 64 KiB to 8 MiB, 1 to 3
    slots), I/O workers (1 to 24), direct or buffered I/O and the file offset all drawn at random;
    the file equals the oracle's image and the verified restore brings every byte back."""
    need_gpu()
    rng = np.random.default_rng(4000 + seed)
    n = int(rng.integers(1, 30))
    sizes = [int(v) for v in rng.choice([0, 7, 4096, 4099, 70_000, 1 << 20, (3 << 20) + 5], size=n)]
    arena = Arena(sizes, misalign=lambda r: r.integers(0, 16) if r.random() < 0.5 else 0, seed=seed)
    datas = random_datas(sizes, seed=700 + seed)
    arena.fill(datas)
    m = gms.Manifest(arena.entries, device=0)
    m.set_staging(int(rng.choice([64 << 10, 1 << 20, 3 << 20, 8 << 20])), int(rng.integers(1, 4)))
    threads = int(rng.integers(1, 25))
    flags = gms.FILE_DIRECT if seed % 2 == 0 else 0
    path = tmp_path / "img.bin"
    gms.snapshot_to_file(m, path, flags=flags, io_threads=threads)
    torch.cuda.synchronize()
    o_img = oracle.pack(datas)
    o_blk, _ = oracle.hashes(datas)
    assert np.array_equal(np.fromfile(path, dtype=np.uint8), o_img)
    offset = 4096 * int(rng.integers(0, 3)) if flags else int(rng.integers(0, 5000))
    shifted = tmp_path / "img_off.bin"
    with open(shifted, "wb") as f:
        f.write(b"\x33" * offset)
        f.write(o_img.tobytes())
    arena.poison()
    cnt = u64_dev(1)
    gms.restore_from_file(m, shifted, file_offset=offset, flags=flags, io_threads=threads,
                          expected=from_u64(o_blk), mismatch_count=cnt)
    torch.cuda.synchronize()
    back, whole = arena.read()
    assert all(np.array_equal(a, b) for a, b in zip(back, datas)) and arena.outside_untouched(whole)
    assert to_u64(cnt)[0] == 0
