"""The model-state store on the GPU: commit-time hashes against the oracle,
read-only leases gated on verification, integrity failures and their repair.

No test writes to committed (read-only) memory: corruption is planted while
a writer holds the lease, or by replacing a mapping's physical pages through
the pool, which is what a lost page looks like to the store.
"""
import ctypes

import numpy as np
import pytest
import torch

import oracle
import paper_2609_25451_amd as gms
import synth
from gpu_util import d2h, from_u64, memset, need_gpu, to_u64, u64_dev

pytestmark = pytest.mark.gpu

SLAB = 8 << 20


def _populate(w, seed):
    """The tiny transformer weight set plus one tensor larger than a slab (a dedicated
    mapping), allocated through the writer's lease and filled on the device."""
    _, specs = synth.weight_set("tiny")
    sizes = [sp.nbytes for sp in specs] + [(20 << 20) + 4098]
    entries, datas = [], []
    for i, n in enumerate(sizes):
        a = w.alloc(n)
        synth.dev_fill_bf16(a, n // 2, seed, i)
        entries.append((a, n))
        datas.append(synth.bf16_bits(n // 2, seed, i).view(np.uint8))
    torch.cuda.synchronize()
    return entries, datas


def _store_hashes(s, m):
    return to_u64_addr(s.block_hashes_ptr(), m.num_blocks)


def to_u64_addr(addr, n):
    return d2h(addr, 8 * n).view(np.uint64)


def test_commit_readers_and_rewrite():
    need_gpu()
    s = gms.Store(va_bytes=1 << 30, slab_bytes=SLAB)
    w = s.connect_rw()
    entries, datas = _populate(w, seed=31)
    w.commit(entries)
    assert s.state() == ("COMMITTED", 0, False)
    m = s.layout()
    o_blk, o_ten = oracle.hashes(datas)
    assert m.num_entries == len(entries) and np.array_equal(_store_hashes(s, m), o_blk)

    r1 = s.connect_ro(verify=True)
    r2 = s.connect_ro(verify=True)
    assert s.state() == ("RO", 2, False) and s.verify() == 0
    # readers read through the committed layout: a snapshot of it is the oracle's image
    image = torch.empty(m.image_bytes, dtype=torch.uint8, device="cuda")
    ten = u64_dev(m.num_entries)
    gms.snapshot(m, image, m.image_bytes, ten_hash=ten)
    torch.cuda.synchronize()
    assert np.array_equal(image.cpu().numpy(), oracle.pack(datas))
    assert np.array_equal(to_u64(ten, m.num_entries), o_ten)
    with pytest.raises(gms.GmsError) as e:
        s.connect_rw()
    assert e.value.status == gms.GMS_ERR_STATE
    r1.close()
    r2.close()
    assert s.state() == ("COMMITTED", 0, False)

    # a writer reacquires the allocation set (writable again), changes a byte and recommits
    w2 = s.connect_rw()
    a3, _ = entries[3]
    memset(a3 + 777, 0x3C, 1)
    datas[3] = datas[3].copy()
    datas[3][777] = 0x3C
    w2.commit(entries)
    assert np.array_equal(_store_hashes(s, s.layout()), oracle.hashes(datas)[0])
    with s.connect_ro():
        assert s.verify() == 0

    # abort discards every allocation and its physical memory
    w3 = s.connect_rw()
    assert s.pool_info()["mapped_bytes"] > 0
    w3.abort()
    assert s.state() == ("EMPTY", 0, False) and s.layout() is None
    info = s.pool_info()
    assert info["mapped_bytes"] == 0 and info["mappings"] == 0
    with s.connect_rw() as w4:  # the rewound reservation serves a new writer
        w4.alloc(1 << 20)
    assert s.state() == ("EMPTY", 0, False) and s.pool_info()["mappings"] == 0
    s.close()


def test_commit_waits_for_writes_still_queued_on_other_streams():
    """Commit turns every mapping of the store read-only.  Device writes the writer queued on
    another stream land first, also with an empty committed layout (no hashing launch to
    order them), and then the pages hold exactly what those writes left."""
    need_gpu()
    s = gms.Store(va_bytes=1 << 30, slab_bytes=SLAB)
    w = s.connect_rw()
    n = 128 << 20
    a = w.alloc(n)
    side = torch.cuda.Stream()
    for seed in range(12):  # a queue of whole-range writes, still running at commit
        synth.dev_fill_bytes(a, n, seed, 9, stream=side)
    w.commit([])
    assert s.state() == ("COMMITTED", 0, False)
    assert np.array_equal(d2h(a, n), synth.random_bytes(n, 11, 9))
    # the same with the range in the layout: commit hashes what the last write left
    w = s.connect_rw()
    a = w.alloc(n)
    want = synth.random_bytes(n, 23, 9)
    o_blk, _ = oracle.hashes([want])
    exp = torch.from_numpy(o_blk.view(np.int64)).cuda()
    torch.cuda.synchronize()
    for seed in range(12, 24):
        synth.dev_fill_bytes(a, n, seed, 9, stream=side)
    w.commit([(a, n)], expected=exp)
    assert s.state() == ("COMMITTED", 0, False)
    assert np.array_equal(_store_hashes(s, s.layout()), o_blk)
    w.close()
    s.close()


def test_commit_refused_on_expected_hash_mismatch():
    """A writer that populated from an image commits against the image's hashes;
    a corrupted byte refuses the commit and the writer keeps its lease."""
    need_gpu()
    s = gms.Store(va_bytes=1 << 30, slab_bytes=SLAB)
    w = s.connect_rw()
    entries, datas = _populate(w, seed=32)
    m = gms.Manifest(entries)
    image = torch.empty(m.image_bytes, dtype=torch.uint8, device="cuda")
    expected = u64_dev(m.num_blocks)
    gms.snapshot(m, image, m.image_bytes, blk_hash=expected)
    torch.cuda.synchronize()
    a5, n5 = entries[5]
    memset(a5 + n5 - 1, 0xFF ^ int(datas[5][-1]), 1)
    with pytest.raises(gms.GmsError) as e:
        w.commit(entries, expected=expected)
    assert e.value.status == gms.GMS_ERR_INTEGRITY and e.value.mismatches == 1
    assert s.state() == ("RW", 0, False)
    gms.restore(m, image, m.image_bytes)  # repopulate from the image
    w.commit(entries, expected=expected)
    assert s.state() == ("COMMITTED", 0, False)
    assert np.array_equal(_store_hashes(s, s.layout()), oracle.hashes(datas)[0])
    m.close()
    s.close()


def test_lost_pages_refuse_readers_until_repopulated():
    need_gpu()
    s = gms.Store(va_bytes=1 << 30, slab_bytes=SLAB)
    w = s.connect_rw()
    entries, datas = _populate(w, seed=33)
    m = gms.Manifest(entries)
    image = torch.empty(m.image_bytes, dtype=torch.uint8, device="cuda")
    expected = u64_dev(m.num_blocks)
    gms.snapshot(m, image, m.image_bytes, blk_hash=expected)
    w.commit(entries, expected=expected)
    with s.connect_ro():
        pass

    # the pages of the mapping holding entry 0 are replaced and hold other bytes
    pool = ctypes.c_void_p(s.pool_handle)
    ma, mb, mapped = ctypes.c_uint64(), ctypes.c_uint64(), ctypes.c_int()
    lib = gms._lib
    assert lib.gms_pool_mapping_of(pool, entries[0][0], ctypes.byref(ma), ctypes.byref(mb), ctypes.byref(mapped)) == 0
    lo, hi = ma.value, ma.value + mb.value
    assert lib.gms_pool_release(pool, ctypes.c_uint64(lo), ctypes.c_uint64(hi - lo)) == 0
    assert lib.gms_pool_remap(pool, ctypes.c_uint64(lo), ctypes.c_uint64(hi - lo)) == 0
    memset(lo, 0x5A, hi - lo)
    o_blk, _ = oracle.hashes(datas)
    assert np.array_equal(to_u64(expected, m.num_blocks), o_blk)
    bad = [np.full(n, 0x5A, np.uint8) if lo <= a < hi else d for (a, n), d in zip(entries, datas)]
    want_cnt, want = oracle.verify(bad, o_blk)
    assert want_cnt > 0

    with pytest.raises(gms.GmsError) as e:
        s.connect_ro(verify=True)
    assert e.value.status == gms.GMS_ERR_INTEGRITY and e.value.mismatches == want_cnt
    assert s.state() == ("COMMITTED", 0, True)
    with pytest.raises(gms.GmsError) as e:
        s.connect_ro(verify=False)
    assert e.value.status == gms.GMS_ERR_INTEGRITY, "an invalid state grants no read lease"
    lst = u64_dev(want_cnt)
    assert s.verify(mismatch_list=lst, mismatch_cap=want_cnt) == want_cnt
    assert np.array_equal(np.sort(to_u64(lst, want_cnt)), want)

    # repair: a writer reuses the allocation set, restores it from the image and recommits
    w2 = s.connect_rw()
    gms.restore(m, image, m.image_bytes)
    w2.commit(entries, expected=expected)
    assert s.state() == ("COMMITTED", 0, False)
    with s.connect_ro(verify=True):
        assert s.verify() == 0
    m.close()
    s.close()


def test_commit_rejects_ranges_outside_the_store():
    need_gpu()
    s = gms.Store(va_bytes=1 << 30, slab_bytes=SLAB)
    outside = torch.empty(4096, dtype=torch.uint8, device="cuda")
    with s.connect_rw() as w:
        a = w.alloc(10_000)  # holds 10,240 bytes: sizes round up to the 256-byte alignment
        b = w.alloc(4096)
        assert b == a + 10_240, "first fit places the next allocation right after"
        for bad in ([(int(outside.data_ptr()), 4096)], [(a, 10_241)], [(a + 10_239, 2)], [(a + 10_000, 1000)]):
            with pytest.raises(gms.GmsError) as e:
                w.commit(bad)
            assert e.value.status == gms.GMS_ERR_INVALID
        w.commit([(a, 10_000), (a, 0)])
    assert s.state() == ("COMMITTED", 0, False)
    s.close()


def test_cold_repopulation_from_file(tmp_path):
    """A cold store repopulated from storage by a separate writer, then attached read-only:
    the weights are snapshotted to an image file with their block hashes; a writer lease
    allocates the same layout in the store, streams the file into it (restore with verify),
    commits against the file's hashes and a reader attaches after re-hashing.  A file with one
    flipped byte is refused at commit with exactly one mismatching block."""
    need_gpu()
    seed, specs = synth.weight_set("tiny")
    src = [torch.empty(sp.shape, dtype=torch.bfloat16, device="cuda") for sp in specs]
    for i, t in enumerate(src):
        synth.dev_fill_bf16(t.data_ptr(), t.numel(), seed, i)
    datas = [synth.bf16_bits(sp.numel, seed, i).view(np.uint8) for i, sp in enumerate(specs)]
    o_blk, _ = oracle.hashes(datas)
    m0 = gms.Manifest(src)
    path = tmp_path / "weights.img"
    blk = u64_dev(m0.num_blocks)
    gms.snapshot_to_file(m0, path, flags=gms.FILE_DIRECT | gms.FILE_SYNC, blk_hash=blk)
    torch.cuda.synchronize()
    assert np.array_equal(to_u64(blk, m0.num_blocks), o_blk)
    sizes = [sp.nbytes for sp in specs]
    m0.close()
    del src

    s = gms.Store(va_bytes=1 << 30, slab_bytes=SLAB)
    w = s.connect_rw()
    addrs = [w.alloc(n) for n in sizes]
    m = gms.Manifest(list(zip(addrs, sizes)))
    expected = from_u64(o_blk)
    cnt = u64_dev(1)
    gms.restore_from_file(m, path, flags=gms.FILE_DIRECT, expected=expected, mismatch_count=cnt)
    torch.cuda.synchronize()
    assert to_u64(cnt)[0] == 0
    w.commit(list(zip(addrs, sizes)), expected=expected)
    with s.connect_ro(verify=True):
        assert np.array_equal(_store_hashes(s, s.layout()), o_blk)

    # a damaged file: the writer's commit is refused, the store stays with the writer
    img = np.fromfile(path, dtype=np.uint8)
    off, _ = m.layout()
    img[off[5] + 100] ^= 0x01
    bad = tmp_path / "weights_bad.img"
    img.tofile(bad)
    w2 = s.connect_rw()
    gms.restore_from_file(m, bad, flags=0, expected=expected, mismatch_count=cnt)
    torch.cuda.synchronize()
    assert to_u64(cnt)[0] == 1
    with pytest.raises(gms.GmsError) as e:
        w2.commit(list(zip(addrs, sizes)), expected=expected)
    assert e.value.status == gms.GMS_ERR_INTEGRITY and e.value.mismatches == 1
    assert s.state() == ("RW", 0, False)
    gms.restore_from_file(m, path, expected=expected, mismatch_count=cnt)  # the good copy
    torch.cuda.synchronize()
    w2.commit(list(zip(addrs, sizes)), expected=expected)
    assert s.state() == ("COMMITTED", 0, False)
    m.close()
    s.close()


def test_recovery_sequence_weights_resident_kv_from_host():
    """The recovery data path at small scale.  The weights stay resident in the committed store;
    the live KV units were saved with their hashes to pageable host memory and the engine's KV
    pages released.  The replacement attaches to the weights after re-hashing them, remaps the
    KV pages at the same addresses and restores the live units from the host image with fused
    verification: live units equal the oracle's bytes, dead units keep what the fresh pages
    held, and a damaged host image is flagged at exactly its block."""
    need_gpu()
    s = gms.Store(va_bytes=1 << 30, slab_bytes=SLAB)
    w = s.connect_rw()
    entries, datas = _populate(w, seed=34)
    o_blk, _ = oracle.hashes(datas)
    w.commit(entries, expected=from_u64(o_blk))
    engine = s.connect_ro()

    layers, blocks, unit = 4, 64, 64 << 10
    slab = blocks * unit
    pool = gms.Pool(va_bytes=layers * slab + (64 << 20), slab_bytes=slab)
    kv = [pool.alloc(slab) for _ in range(layers)]
    kv_data = []
    for l, a in enumerate(kv):
        synth.dev_fill_bf16(a, slab // 2, 35, l)
        kv_data.append(synth.bf16_bits(slab // 2, 35, l).view(np.uint8))
    live = np.sort(np.random.default_rng(36).choice(blocks, blocks // 2, replace=False))
    ents = [(kv[l] + int(b) * unit, unit) for l in range(layers) for b in live]
    want = [kv_data[l][int(b) * unit:(int(b) + 1) * unit] for l in range(layers) for b in live]
    km = gms.Manifest(ents)
    host = np.zeros(km.image_bytes, dtype=np.uint8)
    kv_exp = u64_dev(km.num_blocks)
    gms.snapshot_to_host(km, host, blk_hash=kv_exp)
    assert np.array_equal(host, oracle.pack(want))
    o_kv = oracle.hashes(want)[0]
    assert np.array_equal(to_u64(kv_exp, km.num_blocks), o_kv)

    # the failure: the engine's lease ends, its KV pages are released
    engine.close()
    for a in kv:
        pool.release(a, slab)

    # recovery
    r = s.connect_ro(verify=True)
    assert s.state() == ("RO", 1, False)
    for a in kv:
        pool.remap(a, slab)
        memset(a, 0x5A, slab)  # what the fresh pages hold before the restore
    cnt = u64_dev(1)
    gms.restore_from_host(km, host, expected=from_u64(o_kv), mismatch_count=cnt)
    torch.cuda.synchronize()
    assert to_u64(cnt)[0] == 0
    dead = np.setdiff1d(np.arange(blocks), live)
    for l, a in enumerate(kv):
        got = d2h(a, slab).reshape(blocks, unit)
        for b in live:
            assert np.array_equal(got[b], kv_data[l][int(b) * unit:(int(b) + 1) * unit]), (l, b)
        assert (got[dead] == 0x5A).all(), f"layer {l}: a dead unit was written"

    # a damaged host image: exactly its block is flagged
    off, base = km.layout()
    e = len(ents) // 3
    host[off[e] + 5 * 4096 + 77] ^= 0x08
    lst = u64_dev(4)
    gms.restore_from_host(km, host, expected=from_u64(o_kv), mismatch_count=cnt, mismatch_list=lst, mismatch_cap=4)
    torch.cuda.synchronize()
    assert to_u64(cnt)[0] == 1 and int(to_u64(lst, 1)[0]) == int(base[e]) + 5
    r.close()
    km.close()
    pool.close()
    s.close()
