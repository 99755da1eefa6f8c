"""VMM pool: slab suballocation, KV release/remap at retained addresses, read-only access.

Manifests over pool addresses go through the same snapshot/restore/verify path
and are checked against the oracle; between release and remap no kernel
touches the released range.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2609_25451_amd as gms
import synth
from gpu_util import d2h, from_u64, h2d, memset, need_gpu, to_u64, u64_dev

pytestmark = pytest.mark.gpu


def test_pool_suballocation_round_trip():
    need_gpu()
    pool = gms.Pool(va_bytes=1 << 30, slab_bytes=8 << 20)
    info = pool.info()
    assert info["granularity"] and info["mappings"] == 0
    seed, specs = synth.weight_set("tiny")
    sizes = [sp.nbytes for sp in specs] + [20 << 20, 5, 4097, 100_003]
    addrs = [pool.alloc(n) for n in sizes]
    assert all(a % 256 == 0 for a in addrs)
    iv = sorted(zip(addrs, sizes))
    assert all(a + n <= b for (a, n), (b, _) in zip(iv, iv[1:])), "allocations overlap"
    assert all(info["base"] <= a and a + n <= info["base"] + info["reserved"] for a, n in iv)
    big = addrs[len(specs)]
    start, nbytes, mapped = pool.mapping_of(big)
    assert start == big and nbytes >= 20 << 20 and mapped, "a larger-than-slab allocation gets its own mapping"

    datas = []
    for i, sp in enumerate(specs):
        synth.dev_fill_bf16(addrs[i], sp.numel, seed, i)
        datas.append(synth.bf16_bits(sp.numel, seed, i).view(np.uint8))
    for k, n in enumerate(sizes[len(specs):]):
        d = synth.random_bytes(n, 77, 1000 + k)
        h2d(addrs[len(specs) + k], d)
        datas.append(d)
    torch.cuda.synchronize()

    m = gms.Manifest(list(zip(addrs, sizes)), device=0)
    img = torch.empty(m.image_bytes, dtype=torch.uint8, device="cuda")
    blk, ten = u64_dev(m.num_blocks), u64_dev(m.num_entries)
    gms.snapshot(m, img, m.image_bytes, blk_hash=blk, ten_hash=ten)
    torch.cuda.synchronize()
    o_blk, o_ten = oracle.hashes(datas)
    assert np.array_equal(img.cpu().numpy(), oracle.pack(datas))
    assert np.array_equal(to_u64(blk), o_blk) and np.array_equal(to_u64(ten), o_ten)
    for a, n in zip(addrs, sizes):
        memset(a, 0xA5, n)
    cnt = u64_dev(1)
    gms.restore(m, img, m.image_bytes, expected=from_u64(o_blk), mismatch_count=cnt)
    torch.cuda.synchronize()
    assert to_u64(cnt)[0] == 0
    for a, n, d in zip(addrs, sizes, datas):
        assert np.array_equal(d2h(a, n), d)

    # first fit: a freed block is handed out again; a freed dedicated mapping goes away
    m.close()
    pool.free(addrs[3])
    assert pool.alloc(sizes[3]) == addrs[3]
    before = pool.info()["mappings"]
    pool.free(big)
    assert pool.info()["mappings"] == before - 1
    with pytest.raises(gms.GmsError) as e:
        pool.free(big)
    assert e.value.status == gms.GMS_ERR_INVALID
    pool.close()


def test_kv_pages_released_and_remapped_at_same_addresses():
    need_gpu()
    layers, blocks, unit = 4, 256, 65536
    layer_bytes = blocks * unit
    pool = gms.Pool(va_bytes=1 << 30, slab_bytes=layer_bytes)
    kv = [pool.alloc(layer_bytes) for _ in range(layers)]
    assert kv == [kv[0] + l * layer_bytes for l in range(layers)], "one slab per layer, contiguous"
    for l, a in enumerate(kv):
        synth.dev_fill_bf16(a, layer_bytes // 2, 5, l)
    live = synth.live_map(blocks, blocks * 3 // 5, 1005, 1)
    ents = [(kv[l] + int(b) * unit, unit) for l in range(layers) for b in live]
    m = gms.Manifest(ents, device=0)
    img = torch.empty(m.image_bytes, dtype=torch.uint8, device="cuda")
    exp = u64_dev(m.num_blocks)
    gms.snapshot(m, img, m.image_bytes, blk_hash=exp)
    torch.cuda.synchronize()
    datas = []
    for l in range(layers):
        full = synth.bf16_bits(layer_bytes // 2, 5, l).view(np.uint8)
        datas += [full[int(b) * unit:(int(b) + 1) * unit] for b in live]
    o_blk, _ = oracle.hashes(datas)
    assert np.array_equal(to_u64(exp), o_blk)

    # release the KV pages: VA stays reserved, physical memory goes back
    free0, _ = torch.cuda.mem_get_info()
    pool.release(kv[0], layers * layer_bytes)
    free1, _ = torch.cuda.mem_get_info()
    assert pool.info()["mapped_bytes"] == 0
    assert all(not pool.mapping_of(a)[2] for a in kv)
    assert free1 - free0 >= layers * layer_bytes - (2 << 20)
    with pytest.raises(gms.GmsError) as e:
        pool.set_access(kv[0], layer_bytes, True)
    assert e.value.status == gms.GMS_ERR_STATE

    # fresh pages at the same addresses; restore the live blocks into them
    pool.remap(kv[0], layers * layer_bytes)
    assert all(pool.mapping_of(a) == (a, layer_bytes, True) for a in kv)
    for a in kv:
        memset(a, 0xA5, layer_bytes)
    cnt, lst = u64_dev(1), u64_dev(4)
    gms.restore(m, img, m.image_bytes, expected=exp, mismatch_count=cnt, mismatch_list=lst, mismatch_cap=4)
    torch.cuda.synchronize()
    assert to_u64(cnt)[0] == 0
    dead = np.setdiff1d(np.arange(blocks), live)
    for l, a in enumerate(kv):
        got = d2h(a, layer_bytes).reshape(blocks, unit)
        full = synth.bf16_bits(layer_bytes // 2, 5, l).view(np.uint8).reshape(blocks, unit)
        assert np.array_equal(got[live], full[live]) and (got[dead] == 0xA5).all()

    # read-only for readers: verify still reads the state
    pool.set_access(kv[0], layers * layer_bytes, True)
    gms.verify(m, expected=exp, mismatch_count=cnt)
    torch.cuda.synchronize()
    assert to_u64(cnt)[0] == 0
    pool.set_access(kv[0], layers * layer_bytes, False)

    with pytest.raises(gms.GmsError) as e:  # a range that does not tile whole mappings
        pool.release(kv[0] + 4096, layer_bytes)
    assert e.value.status == gms.GMS_ERR_INVALID
    m.close()
    pool.close()


def test_pool_argument_errors():
    need_gpu()
    with pytest.raises(gms.GmsError) as e:
        gms.Pool(va_bytes=(1 << 30) + 1)
    assert e.value.status == gms.GMS_ERR_INVALID
    pool = gms.Pool(va_bytes=64 << 20, slab_bytes=16 << 20)
    for bad in ((0, 0), (100, 3), (100, 1 << 40)):
        with pytest.raises(gms.GmsError) as e:
            pool.alloc(*bad)
        assert e.value.status == gms.GMS_ERR_INVALID
    with pytest.raises(gms.GmsError) as e:  # reservation exhausted
        pool.alloc(128 << 20)
    assert e.value.status == gms.GMS_ERR_NOMEM
    pool.close()
