"""GPU path vs the CPU oracle, element by element, at sizes the oracle finishes quickly.

Every case: snapshot image == oracle pack; restored bytes == source with every
byte outside the entries untouched; block / tensor hashes == oracle; mismatch
lists == oracle verify.  Inputs come from the seeded generator on the host
(or the GPU generator, itself checked against the host one).
"""
import ctypes

import numpy as np
import pytest
import torch

import oracle
import paper_2609_25451_amd as gms
import synth
from gpu_util import SENTINEL, Arena, from_u64, host_bytes, need_gpu, random_datas, to_u64, u64_dev

pytestmark = pytest.mark.gpu


def _image(nbytes, kind, sentinel=0x5A):
    if kind == gms.MEM_DEVICE:
        return torch.full((max(nbytes, 16),), sentinel, dtype=torch.uint8, device="cuda")
    t = torch.empty((max(nbytes, 16),), dtype=torch.uint8, pin_memory=True)
    t.fill_(sentinel)
    return t


def _round_trip(arena: Arena, datas, kind, chunk_bytes=0, staging=None, check_outside=True):
    """snapshot -> poison -> fused restore -> verify, all compared with the oracle."""
    m = gms.Manifest(arena.entries, device=0, chunk_bytes=chunk_bytes)
    if staging is not None:
        m.set_staging(*staging)
    o_img = oracle.pack(datas)
    o_blk, o_ten = oracle.hashes(datas)
    nb, n = m.num_blocks, m.num_entries
    assert m.image_bytes == o_img.nbytes and nb == o_blk.size

    img = _image(m.image_bytes, kind)
    blk, ten = u64_dev(nb), u64_dev(n)
    gms.snapshot(m, img, m.image_bytes, kind, blk_hash=blk, ten_hash=ten)
    torch.cuda.synchronize()
    got = (img.cpu() if kind == gms.MEM_DEVICE else img).numpy()[: m.image_bytes]
    assert np.array_equal(got, o_img), "snapshot image differs from the oracle"
    assert np.array_equal(to_u64(blk, nb), o_blk) and np.array_equal(to_u64(ten, n), o_ten)

    arena.poison()
    exp = from_u64(o_blk)
    blk2, ten2, cnt, lst = u64_dev(nb), u64_dev(n), u64_dev(1), u64_dev(8)
    cnt.fill_(12345)
    gms.restore(m, img, m.image_bytes, kind, expected=exp, blk_hash=blk2, ten_hash=ten2,
                mismatch_count=cnt, mismatch_list=lst, mismatch_cap=8)
    torch.cuda.synchronize()
    back, whole = arena.read()
    for i, (a, b) in enumerate(zip(back, datas)):
        assert np.array_equal(a, b), f"entry {i} restored wrong"
    if check_outside:
        assert arena.outside_untouched(whole), "restore wrote outside the manifest"
    assert to_u64(cnt)[0] == 0
    assert np.array_equal(to_u64(blk2, nb), o_blk) and np.array_equal(to_u64(ten2, n), o_ten)

    blk3, ten3, cnt3 = u64_dev(nb), u64_dev(n), u64_dev(1)
    gms.verify(m, expected=exp, blk_hash=blk3, ten_hash=ten3, mismatch_count=cnt3)
    torch.cuda.synchronize()
    assert to_u64(cnt3)[0] == 0
    assert np.array_equal(to_u64(blk3, nb), o_blk) and np.array_equal(to_u64(ten3, n), o_ten)
    return m, img


def test_gpu_generator_matches_host():
    need_gpu()
    seed, ts = synth.weight_set("tiny")
    for t_id in (0, 1, 5, 20):
        n = ts[t_id].numel
        d = torch.empty(n, dtype=torch.int16, device="cuda")
        synth.dev_fill_bf16(d.data_ptr(), n, seed, t_id)
        torch.cuda.synchronize()
        assert np.array_equal(d.cpu().numpy().view(np.uint16), synth.bf16_bits(n, seed, t_id))
    # odd offsets and lengths
    d = torch.empty(1001, dtype=torch.int16, device="cuda")
    synth.dev_fill_bf16(d.data_ptr(), 1001, 9, 3, first=77)
    b = torch.empty(999, dtype=torch.uint8, device="cuda")
    synth.dev_fill_bytes(b.data_ptr(), 999, 4, 6, first=13)
    torch.cuda.synchronize()
    assert np.array_equal(d.cpu().numpy().view(np.uint16), synth.bf16_bits(1001, 9, 3, 77))
    assert np.array_equal(b.cpu().numpy(), synth.random_bytes(999, 4, 6, 13))


@pytest.mark.parametrize("kind", [gms.MEM_DEVICE, gms.MEM_HOST_PINNED])
def test_tiny_weights_round_trip(kind):
    need_gpu()
    seed, ts = synth.weight_set("tiny")
    tensors = [torch.empty(t.shape, dtype=torch.bfloat16, device="cuda") for t in ts]
    for i, t in enumerate(tensors):
        synth.dev_fill_bf16(t.data_ptr(), t.numel(), seed, i)
    datas = [synth.bf16_bits(t.numel, seed, i).view(np.uint8) for i, t in enumerate(ts)]
    m = gms.Manifest(tensors, device=0)
    img = _image(m.image_bytes, kind)
    blk, ten = u64_dev(m.num_blocks), u64_dev(m.num_entries)
    gms.snapshot(m, img, m.image_bytes, kind, blk_hash=blk, ten_hash=ten)
    torch.cuda.synchronize()
    got = (img.cpu() if kind == gms.MEM_DEVICE else img).numpy()[: m.image_bytes]
    assert np.array_equal(got, oracle.pack(datas))
    o_blk, o_ten = oracle.hashes(datas)
    assert np.array_equal(to_u64(blk), o_blk) and np.array_equal(to_u64(ten), o_ten)
    for t in tensors:
        t.view(torch.uint8).fill_(0xA5)
    cnt = u64_dev(1)
    gms.restore(m, img, m.image_bytes, kind, expected=from_u64(o_blk), mismatch_count=cnt)
    torch.cuda.synchronize()
    assert to_u64(cnt)[0] == 0
    for t, d in zip(tensors, datas):
        assert np.array_equal(host_bytes(t), d)


RAGGED_SEEDS = list(range(6))


@pytest.mark.parametrize("seed", RAGGED_SEEDS)
@pytest.mark.parametrize("aligned", [True, False])
def test_ragged_manifest_device(seed, aligned):
    need_gpu()
    rng = np.random.default_rng(500 + seed)
    k = int(rng.integers(1, 40))
    sizes = [int(v) for v in rng.integers(0, 70_000, k)]
    sizes[0] = 300_000 + int(rng.integers(0, 5000))  # spans several chunks and a ragged tail
    if k > 2:
        sizes[1] = 0
    arena = Arena(sizes, misalign=None if aligned else (lambda r: r.integers(0, 16)), seed=seed)
    datas = random_datas(sizes, seed=seed)
    arena.fill(datas)
    _round_trip(arena, datas, gms.MEM_DEVICE, chunk_bytes=int(rng.choice([0, 4096, 12288, 1 << 20])))


@pytest.mark.parametrize("chunk_kib", [4, 8, 20, 36, 64, 196, 64 * 1024])
def test_chunk_geometries(chunk_kib):
    """Chunk sizes whose block counts split unevenly into the kernel's work units (a unit's
    second block past the chunk's end), up to the 64 MiB maximum, with ragged and unaligned
    entries: snapshot, restore and verify all equal the oracle."""
    need_gpu()
    rng = np.random.default_rng(700 + chunk_kib)
    sizes = [int(v) for v in rng.integers(1, 90_000, 12)] + [(5 << 20) + 4099, 0, 4096 * 9, 17, (chunk_kib << 10) + 1]
    misalign = [0 if i % 3 else int(rng.integers(1, 16)) for i in range(len(sizes))]
    arena = Arena(sizes, misalign=misalign, seed=chunk_kib)
    datas = random_datas(sizes, seed=chunk_kib + 1)
    arena.fill(datas)
    _round_trip(arena, datas, gms.MEM_DEVICE, chunk_bytes=chunk_kib << 10)


@pytest.mark.parametrize("seed", range(25))
def test_random_manifests(seed):
    """Seeded random manifests: entry counts, sizes (empty, a few bytes, around a block, several
    MiB), alignments, chunk sizes and image kinds all drawn at random; snapshot, restore and
    verify equal the oracle."""
    need_gpu()
    rng = np.random.default_rng(9000 + seed)
    n = int(rng.integers(1, 61))
    kinds = rng.choice(["zero", "tiny", "block", "mid", "big"], size=n, p=[0.1, 0.25, 0.3, 0.25, 0.1])
    draw = {"zero": lambda: 0, "tiny": lambda: int(rng.integers(1, 64)),
            "block": lambda: 4096 * int(rng.integers(1, 4)) + int(rng.integers(-3, 4)),
            "mid": lambda: int(rng.integers(5000, 300_000)), "big": lambda: int(rng.integers(1 << 20, 6 << 20))}
    sizes = [max(0, draw[k]()) for k in kinds]
    arena = Arena(sizes, misalign=lambda r: r.integers(0, 16) if r.random() < 0.4 else 0, seed=seed)
    datas = random_datas(sizes, seed=300 + seed)
    arena.fill(datas)
    chunk = 4096 * int(rng.choice([1, 2, 3, 5, 16, 17, 64, 256]))
    mode = seed % 3
    if mode == 0:
        _round_trip(arena, datas, gms.MEM_DEVICE, chunk_bytes=chunk)
    else:  # pinned host image through the staging ring (1) or zero-copy (2); default chunking
        staging = (int(rng.choice([1, 2, 4])) << 20, int(rng.integers(1, 4))) if mode == 1 else (0, 0)
        _round_trip(arena, datas, gms.MEM_HOST_PINNED, staging=staging)


def test_many_tiny_entries():
    """200,000 entries of 1 to 300 bytes at every alignment: every block is a partial one (the
    unaligned ones through the shifted path) and most of each chunk's work units are empty."""
    need_gpu()
    rng = np.random.default_rng(808)
    sizes = [int(v) for v in rng.integers(1, 301, 200_000)]
    sizes[::1000] = [0] * len(sizes[::1000])
    arena = Arena(sizes, misalign=lambda r: r.integers(0, 16), gap=8, seed=8)
    datas = [synth.random_bytes(n, 88, i) for i, n in enumerate(sizes)]
    host = np.full(arena.total, SENTINEL, dtype=np.uint8)
    for o, d in zip(arena.offsets, datas):
        host[o:o + d.size] = d
    arena.buf.copy_(torch.from_numpy(host))
    _round_trip(arena, datas, gms.MEM_DEVICE)


@pytest.mark.parametrize("staging", [None, (256 * 1024, 2), (1 << 20, 3), (0, 0)],
                         ids=["ring_default", "ring_256k_x2", "ring_1m_x3", "zero_copy"])
def test_ragged_manifest_pinned(staging):
    need_gpu()
    rng = np.random.default_rng(42)
    sizes = [int(v) for v in rng.integers(0, 200_000, 30)] + [3 << 20, 5, 0, 4096]
    arena = Arena(sizes, misalign=lambda r: r.integers(0, 16) * int(r.integers(0, 2)), seed=3)
    datas = random_datas(sizes, seed=11)
    arena.fill(datas)
    m, img = _round_trip(arena, datas, gms.MEM_HOST_PINNED, staging=staging)
    # a second call through the same ring, on another stream
    arena.poison()
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        gms.restore(m, img, m.image_bytes, gms.MEM_HOST_PINNED)
    s.synchronize()
    back, whole = arena.read()
    assert all(np.array_equal(a, b) for a, b in zip(back, datas)) and arena.outside_untouched(whole)


def test_pinned_snapshot_ring_across_slices():
    """A 340 MiB ragged image through 128 MiB x 2 slots: three slices, the ring wraps and slice
    edges fall inside entries.  Snapshot (gather kernel into a device slot, device-to-host copy to
    the host image), restore and verify equal the oracle; with 64 MiB slices the snapshot writes
    zero-copy instead and gives the same image and hashes."""
    need_gpu()
    sizes = [(100 << 20) + 7, 13, (150 << 20) + 3 * 4096 + 5, 0, (90 << 20) + 4095]
    arena = Arena(sizes, misalign=lambda r: r.integers(0, 16), seed=21)
    datas = random_datas(sizes, seed=21)
    arena.fill(datas)
    m, img = _round_trip(arena, datas, gms.MEM_HOST_PINNED, staging=(128 << 20, 2))
    assert m.image_bytes > 2 * (128 << 20)
    o_blk, o_ten = oracle.hashes(datas)
    m.set_staging(64 << 20, 2)
    img2 = _image(m.image_bytes, gms.MEM_HOST_PINNED)
    blk, ten = u64_dev(m.num_blocks), u64_dev(m.num_entries)
    gms.snapshot(m, img2, m.image_bytes, gms.MEM_HOST_PINNED, blk_hash=blk, ten_hash=ten)
    torch.cuda.synchronize()
    assert np.array_equal(img2.numpy()[: m.image_bytes], img.numpy()[: m.image_bytes])
    assert np.array_equal(to_u64(blk, m.num_blocks), o_blk)
    assert np.array_equal(to_u64(ten, m.num_entries), o_ten)
    m.close()


def test_plain_copy_without_hashes():
    need_gpu()
    sizes = [1 << 20, 4097, 123, 8 << 20]
    arena = Arena(sizes, misalign=[0, 3, 1, 0])
    datas = random_datas(sizes, seed=21)
    arena.fill(datas)
    m = gms.Manifest(arena.entries, device=0)
    img = _image(m.image_bytes, gms.MEM_DEVICE)
    gms.snapshot(m, img, m.image_bytes)
    arena.poison()
    gms.restore(m, img, m.image_bytes)
    torch.cuda.synchronize()
    assert np.array_equal(img.cpu().numpy()[: m.image_bytes], oracle.pack(datas))
    back, whole = arena.read()
    assert all(np.array_equal(a, b) for a, b in zip(back, datas)) and arena.outside_untouched(whole)


def test_corruption_flags_exact_blocks():
    need_gpu()
    sizes = [5 * 4096, 100, 0, 3 * 4096 + 9, 4096, 700_001]
    arena = Arena(sizes, misalign=[0, 0, 0, 5, 0, 8])
    datas = random_datas(sizes, seed=31)
    arena.fill(datas)
    m = gms.Manifest(arena.entries, device=0)
    o_blk, _ = oracle.hashes(datas)
    exp = from_u64(o_blk)
    img = _image(m.image_bytes, gms.MEM_DEVICE)
    gms.snapshot(m, img, m.image_bytes)
    torch.cuda.synchronize()
    off, _ = m.layout()
    rng = np.random.default_rng(8)
    flips = []
    for ent in (0, 3, 1, 5, 5):
        byte = int(rng.integers(0, sizes[ent]))
        flips.append((ent, byte, int(rng.integers(0, 8))))
    # flip bits in the image: the fused restore must flag exactly those blocks
    bad = [d.copy() for d in datas]
    himg = img.cpu()
    for ent, byte, bit in flips:
        himg[off[ent] + byte] ^= 1 << bit
        bad[ent][byte] ^= np.uint8(1 << bit)
    img.copy_(himg)
    want_cnt, want = oracle.verify(bad, o_blk)
    assert want_cnt >= 4
    cnt, lst = u64_dev(1), u64_dev(64)
    gms.restore(m, img, m.image_bytes, expected=exp, mismatch_count=cnt, mismatch_list=lst, mismatch_cap=64)
    torch.cuda.synchronize()
    c = int(to_u64(cnt)[0])
    assert c == want_cnt and np.array_equal(np.sort(to_u64(lst, c)), want)
    # the restored (corrupted) entries: verify must agree; a small cap truncates
    cnt2, lst2 = u64_dev(1), u64_dev(2)
    gms.verify(m, expected=exp, mismatch_count=cnt2, mismatch_list=lst2, mismatch_cap=2)
    torch.cuda.synchronize()
    assert int(to_u64(cnt2)[0]) == want_cnt
    assert set(to_u64(lst2, 2).tolist()) <= set(want.tolist())
    # the padding of an image slot is not part of any hash
    himg[off[1] + 200] ^= 0xFF
    img.copy_(himg)
    gms.restore(m, img, m.image_bytes, expected=exp, mismatch_count=cnt)
    torch.cuda.synchronize()
    assert int(to_u64(cnt)[0]) == want_cnt


@pytest.mark.parametrize("chunks,tail", [(127, 0), (128, 0), (129, 0), (293, 5), (1025, 4097)],
                         ids=["per127", "per128", "per129", "per294", "per1026"])
def test_verify_unit_order_stripe_edges(chunks, tail):
    """Verify walks units in 1 MiB stripes per XCD, with the last partial round of stripes split
    into eight contiguous pieces.  One entry of `chunks` 64 KiB chunks (+ a ragged tail) gives a
    launch whose grid holds exactly 8 slots per chunk, so each XCD's share of slots lands below, at
    and above a stripe boundary.  A unit skipped or visited twice would change a block hash, the
    tensor hash or the mismatch list against the oracle."""
    need_gpu()
    size = chunks * 65536 + tail
    arena = Arena([size])
    datas = random_datas([size], seed=chunks)
    arena.fill(datas)
    m = gms.Manifest(arena.entries, device=0, chunk_bytes=65536)
    assert m.num_chunks == chunks + (tail > 0) and m.num_launch_groups == 1
    o_blk, o_ten = oracle.hashes(datas)
    nb = m.num_blocks
    blk, ten = u64_dev(nb), u64_dev(1)
    gms.verify(m, blk_hash=blk, ten_hash=ten)
    torch.cuda.synchronize()
    assert np.array_equal(to_u64(blk, nb), o_blk) and np.array_equal(to_u64(ten, 1), o_ten)
    # corrupt the first block, a block of the last whole chunk and the last block
    spots = sorted({0, (chunks - 1) * 65536 + 3 * 4096 + 17, size - 1})
    bad = datas[0].copy()
    v = arena.view(0)
    for b in spots:
        v[b:b + 1].bitwise_xor_(0x10)
        bad[b] ^= 0x10
    want_cnt, want = oracle.verify([bad], o_blk)
    assert want_cnt == len(spots)
    cnt, lst = u64_dev(1), u64_dev(8)
    gms.verify(m, expected=from_u64(o_blk), blk_hash=blk, mismatch_count=cnt, mismatch_list=lst, mismatch_cap=8)
    torch.cuda.synchronize()
    c = int(to_u64(cnt)[0])
    assert c == want_cnt and np.array_equal(np.sort(to_u64(lst, c)), want)
    assert np.array_equal(to_u64(blk, nb), oracle.hashes([bad])[0])
    m.close()


def test_empty_and_zero_length_manifests():
    need_gpu()
    cnt = u64_dev(1)
    cnt.fill_(99)
    m = gms.Manifest([], device=0)
    img = _image(16, gms.MEM_DEVICE)
    gms.snapshot(m, img, 16)
    gms.restore(m, img, 16, expected=u64_dev(1), mismatch_count=cnt)
    torch.cuda.synchronize()
    assert to_u64(cnt)[0] == 0
    buf = torch.zeros(64, dtype=torch.uint8, device="cuda")
    m2 = gms.Manifest([(buf.data_ptr(), 0), (buf.data_ptr() + 8, 0)], device=0)
    ten = u64_dev(2)
    ten.fill_(7)
    gms.verify(m2, ten_hash=ten)
    torch.cuda.synchronize()
    assert to_u64(ten, 2).tolist() == [0, 0]


def test_argument_errors_on_gpu():
    need_gpu()
    buf = torch.zeros(10_000, dtype=torch.uint8, device="cuda")
    m = gms.Manifest([(buf.data_ptr(), 5000), (buf.data_ptr() + 5000, 3000)], device=0)
    small = torch.zeros(4096, dtype=torch.uint8, device="cuda")
    with pytest.raises(gms.GmsError) as e:
        gms.restore(m, small, small.numel())
    assert e.value.status == gms.GMS_ERR_SIZE
    big = torch.zeros(m.image_bytes + 64, dtype=torch.uint8, device="cuda")
    with pytest.raises(gms.GmsError) as e:
        gms.restore(m, big.data_ptr() + 1, m.image_bytes)
    assert e.value.status == gms.GMS_ERR_INVALID
    host = np.zeros(m.image_bytes, dtype=np.uint8)
    with pytest.raises(gms.GmsError) as e:
        gms.restore(m, host.ctypes.data, m.image_bytes, gms.MEM_DEVICE)
    assert e.value.status == gms.GMS_ERR_INVALID
    with pytest.raises(gms.GmsError) as e:  # pageable memory is not pinned
        gms.restore(m, host.ctypes.data, m.image_bytes, gms.MEM_HOST_PINNED)
    assert e.value.status == gms.GMS_ERR_INVALID
    # entry running past its allocation (an exact hipMalloc, so the bound is known)
    hip = ctypes.CDLL("libamdhip64.so.7")
    raw = ctypes.c_void_p()
    assert hip.hipMalloc(ctypes.byref(raw), ctypes.c_size_t(1 << 20)) == 0
    try:
        with pytest.raises(gms.GmsError) as e:
            gms.Manifest([(raw.value + (1 << 20) - 100, 4 << 20)], device=0)
        assert e.value.status == gms.GMS_ERR_SIZE
        gms.Manifest([(raw.value + 100, (1 << 20) - 100)], device=0).close()
    finally:
        hip.hipFree(raw)
    # a pinned image smaller than the size the caller claims
    small_pinned = ctypes.c_void_p()
    assert hip.hipHostMalloc(ctypes.byref(small_pinned), ctypes.c_size_t(m.image_bytes - 4096), 0) == 0
    try:
        with pytest.raises(gms.GmsError) as e:
            gms.restore(m, small_pinned.value, m.image_bytes, gms.MEM_HOST_PINNED)
        assert e.value.status == gms.GMS_ERR_SIZE
    finally:
        hip.hipHostFree(small_pinned)
    with pytest.raises(gms.GmsError) as e:  # host memory as an entry
        gms.Manifest([(host.ctypes.data, 100)], device=0)
    assert e.value.status == gms.GMS_ERR_INVALID
    with pytest.raises(gms.GmsError) as e:  # expected without a counter
        gms.verify(m, expected=u64_dev(m.num_blocks))
    assert e.value.status == gms.GMS_ERR_INVALID
    with pytest.raises(gms.GmsError) as e:
        gms.verify(m)
    assert e.value.status == gms.GMS_ERR_INVALID


def test_sizes_that_would_wrap_are_refused():
    """Byte counts that would overflow 64 bits are refused before anything is enqueued."""
    need_gpu()
    hip = ctypes.CDLL("libamdhip64.so.7")
    ent = torch.zeros(1 << 30, dtype=torch.uint8, device="cuda")
    m = gms.Manifest([(ent.data_ptr(), 1 << 30)], device=0)  # 2^18 blocks
    exp, cnt = u64_dev(m.num_blocks), u64_dev(1)
    gms.verify(m, blk_hash=exp)
    lists = []
    for nbytes in (1 << 20, 2 << 20):  # exact allocations: 2^17 and 2^18 list entries
        raw = ctypes.c_void_p()
        assert hip.hipMalloc(ctypes.byref(raw), ctypes.c_size_t(nbytes)) == 0
        lists.append(raw.value)
    try:
        # a capacity whose byte count wraps to 8: the list holds half the entries one call can write
        with pytest.raises(gms.GmsError) as e:
            gms.verify(m, expected=exp, mismatch_count=cnt, mismatch_list=lists[0], mismatch_cap=(1 << 61) + 1)
        assert e.value.status == gms.GMS_ERR_SIZE
        # a list as long as the block count takes any capacity
        gms.verify(m, expected=exp, mismatch_count=cnt, mismatch_list=lists[1], mismatch_cap=(1 << 64) - 1)
        torch.cuda.synchronize()
        assert to_u64(cnt)[0] == 0
    finally:
        for a in lists:
            hip.hipFree(ctypes.c_void_p(a))
    for slice_bytes, slots in ((100, 1), (128 << 30, 1), (1 << 63, 2), (4096, 17)):
        with pytest.raises(gms.GmsError) as e:
            m.set_staging(slice_bytes, slots)
        assert e.value.status == gms.GMS_ERR_INVALID, (slice_bytes, slots)
    with pytest.raises(gms.GmsError) as e:
        gms.restore_from_file(m, "/nonexistent/image", file_offset=(1 << 64) - 4096)
    assert e.value.status == gms.GMS_ERR_INVALID
    m.close()
    del ent
    pool = gms.Pool(va_bytes=1 << 30, slab_bytes=8 << 20)
    for nbytes in ((1 << 64) - 1, (1 << 30) + 1):
        with pytest.raises(gms.GmsError) as e:
            pool.alloc(nbytes)
        assert e.value.status == gms.GMS_ERR_NOMEM, nbytes
    pool.close()


def test_staging_slice_zero_selects_the_default():
    need_gpu()
    sizes = [300_000, 5, 4096 * 3]
    arena = Arena(sizes, seed=4)
    datas = random_datas(sizes, seed=4)
    arena.fill(datas)
    _round_trip(arena, datas, gms.MEM_HOST_PINNED, staging=(0, 3))


@pytest.mark.parametrize("kind,staging", [(gms.MEM_DEVICE, None), (gms.MEM_HOST_PINNED, (1 << 20, 2)),
                                          (gms.MEM_HOST_PINNED, (0, 0))], ids=["device", "ring_1m_x2", "zero_copy"])
def test_mixed_manifest_takes_several_launch_groups(kind, staging):
    """Large entries among 40,000 tiny ones (and some mid-sized): the tiny chunks need one work
    unit where a 64 KiB chunk needs eight, so the library launches them apart; results equal the
    oracle, slices of the ring holding chunks of several groups included."""
    need_gpu()
    rng = np.random.default_rng(99)
    sizes = [int(v) for v in rng.integers(1, 4097, 40_000)]
    for i, v in zip(rng.choice(len(sizes), 12, replace=False), [(3 << 20) + 5, 1 << 20, 65536 * 3 + 7, 9000] * 3):
        sizes[int(i)] = int(v)
    sizes[::997] = [0] * len(sizes[::997])
    arena = Arena(sizes, misalign=lambda r: r.integers(0, 16) if r.random() < 0.3 else 0, gap=16, seed=99)
    datas = random_datas(sizes, seed=99)
    host = np.full(arena.total, SENTINEL, dtype=np.uint8)
    for o, d in zip(arena.offsets, datas):
        host[o:o + d.size] = d
    arena.buf.copy_(torch.from_numpy(host))
    m, _ = _round_trip(arena, datas, kind, staging=staging)
    # tiny and large chunks launch apart, and so do aligned and unaligned entries of a class
    assert m.num_launch_groups >= 3
    # the host-image path over the same groups (it needs ring slots)
    m.set_staging(1 << 20, 2)
    o_img = oracle.pack(datas)
    arena.poison()
    cnt = u64_dev(1)
    gms.restore_from_host(m, o_img, expected=from_u64(oracle.hashes(datas)[0]), mismatch_count=cnt)
    torch.cuda.synchronize()
    back, whole = arena.read()
    assert all(np.array_equal(a, b) for a, b in zip(back, datas)) and arena.outside_untouched(whole)
    assert to_u64(cnt)[0] == 0
    m.close()


@pytest.mark.parametrize("kind,staging", [(gms.MEM_DEVICE, None), (gms.MEM_HOST_PINNED, (64 << 10, 2))],
                         ids=["device", "ring_64k_x2"])
def test_shifted_path_edges(kind, staging):
    """Entries at every byte offset 1..15 from a 16-byte boundary, with sizes around the
    granules a block shares with its neighbours (a block's last bytes short of, at and past the
    next granule), single granules, several chunks and ragged tails: snapshot, restore and
    verify equal the oracle and no byte outside an entry is written."""
    need_gpu()
    sizes, mis = [], []
    for a in range(1, 16):
        for n in (1, 15 - a, 16 - a, 17 - a, 4096 - a - 1, 4096 - a, 4096 - a + 1, 4096, 4097, 8192 - a,
                  8192 + 16 - a, 2 * 65536 + 4096 - a, 65536 * 3 + 5, 300_001):
            if n > 0:
                sizes.append(n)
                mis.append(a)
    arena = Arena(sizes, misalign=mis, gap=40, seed=515)
    datas = random_datas(sizes, seed=515)
    arena.fill(datas)
    m, _ = _round_trip(arena, datas, kind, staging=staging)
    m.close()


_ROUNDS_CHILD = r"""
import sys
sys.path[:0] = [sys.argv[1], sys.argv[1] + "/tests"]
import numpy as np, torch
import paper_2609_25451_amd as gms
from gpu_util import Arena, random_datas
import test_gpu_parity as t
rng = np.random.default_rng(77)
# first, 3,100 entries of 16 KiB: one two-unit chunk each, a launch group of their own that restores
# in the striped order
sizes = [16384] * 3100
sizes += [int(v) for v in rng.integers(1, 200_000, 60)] + [3 << 20, 1 << 20] + [int(v) for v in rng.integers(1, 5000, 3000)]
arena = Arena(sizes, misalign=lambda r: r.integers(0, 16) if r.random() < 0.3 else 0, gap=16, seed=77)
datas = random_datas(sizes, seed=77)
host = np.full(arena.total, 0xA5, dtype=np.uint8)
for o, d in zip(arena.offsets, datas):
    host[o:o + d.size] = d
arena.buf.copy_(torch.from_numpy(host))
m, _ = t._round_trip(arena, datas, gms.MEM_DEVICE)
gs = m.launch_groups()
assert any(g["striped"] for g in gs) and any(g["unit_shift"] and not g["striped"] for g in gs), gs
print("rounds ok", m.num_blocks, m.num_launch_groups, flush=True)
"""


@pytest.mark.parametrize("cap", [8, 64, 2048])
def test_launches_loop_over_grid_rounds(cap):
    """With the grid capped at `cap` workgroups (GMS_MAX_GRID, read once per process, so the
    case runs in a child process), every launch loops over many grid-sized rounds: contiguous
    and striped unit orders, paired and unit kernels, aligned and shifted entries; results
    equal the oracle as with an uncapped grid."""
    import os
    import subprocess
    import sys

    need_gpu()
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    env = dict(os.environ, GMS_MAX_GRID=str(cap))
    print(f"child: GMS_MAX_GRID={cap}", flush=True)
    r = subprocess.run([sys.executable, "-c", _ROUNDS_CHILD, root], env=env, capture_output=True, text=True,
                       timeout=300)
    assert r.returncode == 0, r.stdout[-2000:] + r.stderr[-4000:]
    assert "rounds ok" in r.stdout
