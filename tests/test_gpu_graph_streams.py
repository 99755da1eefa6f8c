"""Capture in a HIP graph and concurrent streams.

A device-image restore, snapshot or verify launches only kernels (the prologue
that zeroes the counters is a kernel, not a memset), so it can be captured
once and replayed; every replay is checked against the oracle for the bytes
the memory holds at that moment, with eager work in between.  Calls that
cannot be captured (pinned-host images, image files, store verification)
refuse with GMS_ERR_STATE and leave the capture usable.  Independent
manifests restored on two streams at once must not interfere.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2609_25451_amd as gms
from gpu_util import Arena, from_u64, need_gpu, random_datas, to_u64, u64_dev

pytestmark = pytest.mark.gpu

SIZES = [70_000, 13, 0, 3 * 4096, (2 << 20) + 5, 4095, 200_001]


def _arena(seed):
    arena = Arena(SIZES, misalign=lambda r: r.integers(0, 16), seed=seed)
    datas = random_datas(SIZES, seed=seed)
    arena.fill(datas)
    return arena, datas


def _setup(seed, sizes):
    arena = Arena(sizes, misalign=[0] * len(sizes), seed=seed)
    datas = random_datas(sizes, seed=seed)
    arena.fill(datas)
    m = gms.Manifest(arena.entries, device=0)
    img = torch.empty(m.image_bytes, dtype=torch.uint8, device="cuda")
    gms.snapshot(m, img, m.image_bytes)
    torch.cuda.synchronize()
    o_blk, o_ten = oracle.hashes(datas)
    return arena, datas, m, img, o_blk, o_ten


def test_restore_captured_in_a_graph_and_replayed():
    need_gpu()
    sizes = [700_000, 4096 * 5, 13, 300_001, 1 << 20]
    arena, datas, m, img, o_blk, o_ten = _setup(61, sizes)
    exp = from_u64(o_blk)
    cnt, lst, ten = u64_dev(1), u64_dev(4), u64_dev(m.num_entries)
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):  # warm the kernels and the LDS opt-in outside capture
        gms.restore(m, img, m.image_bytes, expected=exp, ten_hash=ten, mismatch_count=cnt, mismatch_list=lst,
                    mismatch_cap=4)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s):
        gms.restore(m, img, m.image_bytes, expected=exp, ten_hash=ten, mismatch_count=cnt, mismatch_list=lst,
                    mismatch_cap=4)
    off, base = m.layout()
    for rep in range(4):
        arena.poison()
        cnt.fill_(123)
        ten.fill_(7)
        flip = rep == 2
        if flip:  # eager corruption of the image between replays
            img[off[3] + 5000] ^= 0x01
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        back, whole = arena.read()
        want = [d.copy() for d in datas]
        if flip:
            want[3][5000] ^= 0x01
        assert all(np.array_equal(a, b) for a, b in zip(back, want)) and arena.outside_untouched(whole)
        c = int(to_u64(cnt)[0])
        if flip:
            assert c == 1 and int(to_u64(lst)[0]) == base[3] + 5000 // 4096
            img[off[3] + 5000] ^= 0x01
        else:
            assert c == 0 and np.array_equal(to_u64(ten, m.num_entries), o_ten)


def test_independent_manifests_on_two_streams():
    need_gpu()
    a = _setup(71, [3 << 20, 123_457, 4096])
    b = _setup(72, [1 << 20, 99, 2 << 20, 77_777])
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    outs = []
    for (arena, datas, m, img, o_blk, o_ten), s in ((a, s1), (b, s2)):
        arena.poison()
        outs.append((u64_dev(1), u64_dev(m.num_blocks), u64_dev(m.num_entries)))
    torch.cuda.synchronize()
    for rep in range(3):
        for ((arena, datas, m, img, o_blk, o_ten), s), (cnt, blk, ten) in zip(((a, s1), (b, s2)), outs):
            with torch.cuda.stream(s):
                gms.restore(m, img, m.image_bytes, expected=from_u64(o_blk), blk_hash=blk, ten_hash=ten,
                            mismatch_count=cnt)
                gms.verify(m, expected=from_u64(o_blk), mismatch_count=cnt)
        torch.cuda.synchronize()
        for (arena, datas, m, img, o_blk, o_ten), (cnt, blk, ten) in zip((a, b), outs):
            back, whole = arena.read()
            assert all(np.array_equal(x, y) for x, y in zip(back, datas)) and arena.outside_untouched(whole)
            assert to_u64(cnt)[0] == 0
            assert np.array_equal(to_u64(blk, m.num_blocks), o_blk)
            assert np.array_equal(to_u64(ten, m.num_entries), o_ten)


def test_captured_snapshot_and_verify_follow_the_data():
    """One graph holds a snapshot (image, block and tensor hashes) and a verify against an
    earlier hash array; the entries change eagerly between replays."""
    need_gpu()
    arena, datas = _arena(62)
    m = gms.Manifest(arena.entries)
    o_blk0, _ = oracle.hashes(datas)
    exp = from_u64(o_blk0)
    img = torch.empty(m.image_bytes, dtype=torch.uint8, device="cuda")
    blk, ten, vcnt = u64_dev(m.num_blocks), u64_dev(m.num_entries), u64_dev(1)

    def step():
        gms.snapshot(m, img, m.image_bytes, blk_hash=blk, ten_hash=ten)
        gms.verify(m, expected=exp, mismatch_count=vcnt)

    step()  # warm the kernels outside capture
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step()
    torch.cuda.synchronize()

    rng = np.random.default_rng(5)
    cur = [d.copy() for d in datas]
    for rep in range(4):
        if rep:  # rewrite a few bytes of random non-empty entries
            for _ in range(rep):
                i = int(rng.choice([k for k, n in enumerate(SIZES) if n]))
                j = int(rng.integers(0, SIZES[i]))
                cur[i][j] ^= 0xFF
                arena.view(i)[j] = int(cur[i][j])
        img.fill_(0xEE)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        o_blk, o_ten = oracle.hashes(cur)
        assert np.array_equal(img.cpu().numpy(), oracle.pack(cur)), f"replay {rep}: image"
        assert np.array_equal(to_u64(blk, m.num_blocks), o_blk), f"replay {rep}: block hashes"
        assert np.array_equal(to_u64(ten, m.num_entries), o_ten), f"replay {rep}: tensor hashes"
        assert to_u64(vcnt)[0] == oracle.verify(cur, o_blk0)[0], f"replay {rep}: verify count"
    del g
    m.close()


def test_uncapturable_calls_refuse_and_leave_the_capture_usable(tmp_path):
    need_gpu()
    arena, datas = _arena(63)
    m = gms.Manifest(arena.entries)
    o_img = oracle.pack(datas)
    pinned = torch.from_numpy(o_img.copy()).pin_memory()
    path = tmp_path / "image.bin"
    o_img.tofile(path)
    dev_img = torch.from_numpy(o_img).cuda()
    s = gms.Store(va_bytes=1 << 30, slab_bytes=8 << 20)
    with s.connect_rw() as w:
        a = w.alloc(4096)
        w.commit([(a, 4096)])
    reader = s.connect_ro()

    refused = []
    gms.restore(m, dev_img, m.image_bytes)  # warm the kernels outside capture
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        for name, call in (
            ("pinned restore", lambda: gms.restore(m, pinned, m.image_bytes, gms.MEM_HOST_PINNED)),
            ("pinned snapshot", lambda: gms.snapshot(m, pinned, m.image_bytes, gms.MEM_HOST_PINNED)),
            ("file restore", lambda: gms.restore_from_file(m, path, flags=0)),
            ("store verify", lambda: s.verify()),
        ):
            try:
                call()
            except gms.GmsError as e:
                refused.append((name, e.status))
        gms.restore(m, dev_img, m.image_bytes)
    torch.cuda.synchronize()
    assert refused == [(n, gms.GMS_ERR_STATE) for n in
                       ("pinned restore", "pinned snapshot", "file restore", "store verify")]
    arena.poison()
    torch.cuda.synchronize()
    g.replay()
    torch.cuda.synchronize()
    back, whole = arena.read()
    assert all(np.array_equal(a, b) for a, b in zip(back, datas)) and arena.outside_untouched(whole)
    # the same calls work again outside capture
    arena.poison()
    gms.restore(m, pinned, m.image_bytes, gms.MEM_HOST_PINNED)
    torch.cuda.synchronize()
    assert all(np.array_equal(a, b) for a, b in zip(arena.read()[0], datas))
    assert s.verify() == 0
    reader.close()
    del g
    m.close()
    s.close()
