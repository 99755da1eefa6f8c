"""gms_restore_pinned_noalloc, called through the C-ABI, against gms_restore.

Two calls in a row on one device (the second with a smaller manifest, so the
fixed staging area holds the previous call's bytes when it starts), each
compared with gms_restore from the same pinned image through the staging
ring: restored bytes, block and tensor hashes, mismatch count and list, and
the oracle's hashes.
"""
import ctypes

import numpy as np
import pytest
import torch

import oracle
import paper_2609_25451_amd as gms
from gpu_util import Arena, from_u64, need_gpu, random_datas, to_u64, u64_dev

pytestmark = pytest.mark.gpu


def _outputs(arena, nb, n):
    return u64_dev(nb), u64_dev(n), u64_dev(1), u64_dev(16)


def _existing(m, pinned, exp, arena):
    blk, ten, cnt, lst = _outputs(arena, m.num_blocks, m.num_entries)
    arena.poison()
    gms.restore(m, pinned, m.image_bytes, gms.MEM_HOST_PINNED, expected=exp, blk_hash=blk, ten_hash=ten,
                mismatch_count=cnt, mismatch_list=lst, mismatch_cap=16)
    torch.cuda.synchronize()
    back, whole = arena.read()
    return back, whole, blk, ten, cnt, lst


def _noalloc(m, pinned, exp, arena, staging):
    blk, ten, cnt, lst = _outputs(arena, m.num_blocks, m.num_entries)
    arena.poison()
    stream = torch.cuda.current_stream().cuda_stream
    rc = gms.gms_restore_pinned_noalloc(m.handle, pinned.data_ptr(), m.image_bytes, staging, exp.data_ptr(),
                                        blk.data_ptr(), ten.data_ptr(), cnt.data_ptr(), lst.data_ptr(), 16,
                                        ctypes.c_void_p(stream))
    assert rc == gms.GMS_OK, gms.gms_last_error()
    torch.cuda.synchronize()
    back, whole = arena.read()
    return back, whole, blk, ten, cnt, lst


def _case(sizes, seed, staging, flips):
    arena = Arena(sizes, misalign=lambda r: r.integers(0, 16) if r.random() < 0.3 else 0, gap=32, seed=seed)
    datas = random_datas(sizes, seed=seed)
    arena.fill(datas)
    m = gms.Manifest(arena.entries, device=0)
    pinned = torch.empty(m.image_bytes, dtype=torch.uint8, pin_memory=True)
    gms.snapshot(m, pinned, m.image_bytes, gms.MEM_HOST_PINNED)
    torch.cuda.synchronize()
    o_img = oracle.pack(datas)
    assert np.array_equal(pinned.numpy(), o_img)
    o_blk, o_ten = oracle.hashes(datas)
    exp = from_u64(o_blk)
    off, base = m.layout()
    flipped = sorted({base[i] + b // 4096 for i, b in flips})
    for i, b in flips:  # planted corruption in the image
        pinned[off[i] + b] ^= 0x20
    a = _existing(m, pinned, exp, arena)
    b = _noalloc(m, pinned, exp, arena, staging)
    for x, y in zip(a[0], b[0]):
        assert np.array_equal(x, y)
    assert arena.outside_untouched(b[1]), "the no-allocation restore wrote outside the manifest"
    for x, y in zip(a[2:4], b[2:4]):
        assert torch.equal(x, y)
    assert int(a[4].item()) == int(b[4].item()) == len(flipped)
    assert sorted(to_u64(a[5])[:len(flipped)].tolist()) == sorted(to_u64(b[5])[:len(flipped)].tolist()) == flipped
    # against the oracle: the restored bytes are the corrupted image's, unpacked
    o_back = oracle.unpack(pinned.numpy(), sizes)
    assert all(np.array_equal(x, y) for x, y in zip(b[0], o_back))
    o_blk2, o_ten2 = oracle.hashes(o_back)
    assert np.array_equal(to_u64(b[2], m.num_blocks), o_blk2)
    assert np.array_equal(to_u64(b[3], m.num_entries), o_ten2)
    m.close()


def test_noalloc_restore_matches_gms_restore_on_two_calls():
    need_gpu()
    rng = np.random.default_rng(2024)
    big = [int(v) for v in rng.integers(1, 3_000_000, 80)] + [(40 << 20) + 4099, 0, 17, 4096 * 33]
    _case(big, 31, 0, flips=[(3, 5), (81, 4099), (20, 0)])  # the whole 64 MiB area: 3 slices
    small = [int(v) for v in rng.integers(1, 200_000, 30)] + [300_001]
    _case(small, 32, 1 << 20, flips=[(4, 1)])  # 1 MiB slices over a smaller image


def test_noalloc_refuses_staging_beyond_the_area():
    need_gpu()
    arena = Arena([5000, 70_000])
    m = gms.Manifest(arena.entries, device=0)
    pinned = torch.empty(m.image_bytes, dtype=torch.uint8, pin_memory=True)
    for staging in (gms.NOALLOC_STAGING_BYTES + 4096, 4096):  # above the area; below one 64 KiB chunk
        with pytest.raises(gms.GmsError) as e:
            gms.restore_pinned_noalloc(m, pinned, staging_bytes=staging)
        assert e.value.status == gms.GMS_ERR_SIZE
    m.close()


def test_noalloc_restore_replays_from_a_graph():
    """After one call outside capture, the allocation-free restore captured into a HIP graph
    replays: each replay reads the pinned image as it is at that moment, restores it and
    compares it with the expected hashes.  Replays are checked against the oracle, with eager
    work and a host-side change of the image between them.  On a manifest that a staging-ring
    call used, a capturing call is refused before it records anything."""
    need_gpu()
    sizes = [70_000, 4096 * 5 + 3, 1, 300_001, 64 << 10, 2_000_003]
    arena = Arena(sizes, misalign=lambda r: r.integers(0, 16) if r.random() < 0.5 else 0, gap=32, seed=77)
    datas = random_datas(sizes, seed=77)
    arena.fill(datas)
    m = gms.Manifest(arena.entries, device=0)
    pinned = torch.empty(m.image_bytes, dtype=torch.uint8, pin_memory=True)
    pinned.numpy()[:] = oracle.pack(datas)  # written on the host: no staging-ring call on m
    o_blk, o_ten = oracle.hashes(datas)
    exp = from_u64(o_blk)
    blk, ten, cnt, lst = _outputs(arena, m.num_blocks, m.num_entries)
    side = torch.cuda.Stream()

    def call():
        gms.restore_pinned_noalloc(m, pinned, staging_bytes=1 << 20, expected=exp, blk_hash=blk, ten_hash=ten,
                                   mismatch_count=cnt, mismatch_list=lst, mismatch_cap=16)

    with torch.cuda.stream(side):
        call()  # the eager call: also loads the kernels and finds the staging area
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=side):
        call()
    torch.cuda.synchronize()

    off, base = m.layout()
    scratch = torch.ones(1 << 22, device="cuda")
    for step, flip in enumerate([False, True, False, True]):
        want = [d.copy() for d in datas]
        if flip:  # one byte of entry 3 changed in the image on the host
            pinned[off[3] + 5 + step] ^= 0x10
            want[3][5 + step] ^= 0x10
        arena.poison()
        scratch.mul_(1.5)  # eager work between replays
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        back, whole = arena.read()
        assert all(np.array_equal(x, y) for x, y in zip(back, want)), step
        assert arena.outside_untouched(whole), step
        w_blk, w_ten = oracle.hashes(want)
        assert np.array_equal(to_u64(blk, m.num_blocks), w_blk), step
        assert np.array_equal(to_u64(ten, m.num_entries), w_ten), step
        assert int(cnt.item()) == (1 if flip else 0), step
        if flip:
            assert to_u64(lst)[0] == base[3] + (5 + step) // 4096
            pinned[off[3] + 5 + step] ^= 0x10  # put back

    # a staging-ring call on the manifest: a graph could not wait for it, so capture is refused
    gms.restore(m, pinned, m.image_bytes, gms.MEM_HOST_PINNED, expected=exp, mismatch_count=cnt)
    torch.cuda.synchronize()
    g2 = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g2, stream=side):
        with pytest.raises(gms.GmsError) as e:
            call()
        scratch.add_(1.0)  # the capture still holds a node of its own
    assert e.value.status == gms.GMS_ERR_STATE
    torch.cuda.synchronize()
    m.close()
