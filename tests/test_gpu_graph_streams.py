"""Capture in a HIP graph and concurrent streams.

A device-image restore launches only kernels (the prologue that zeroes the
counters is a kernel, not a memset), so it can be captured once and replayed;
every replay is checked against the oracle with eager work in between.
Independent manifests restored on two streams at once must not interfere.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2609_25451_amd as gms
from gpu_util import Arena, from_u64, need_gpu, random_datas, to_u64, u64_dev

pytestmark = pytest.mark.gpu


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
