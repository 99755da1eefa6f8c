"""Full-size workloads, in the launch configuration bench.py times, compared with
the CPU oracle element by element.

Every workload streams through tests/full_parity.py: the seeded generator's
bytes of each batch of entries go through the oracle, whose packed image must
equal the library's image byte for byte and whose block and tensor hashes must
equal every hash array the library produced (snapshot, fused restore, verify,
pinned-host and pageable-host legs), whole arrays; the restored entries must
equal the generator's bytes.  Mismatch counts and lists of planted bit flips
are the oracle's verify of the flipped entry.  The KV pool's dead units must
keep their poison.
"""
import gc

import numpy as np
import pytest
import torch

import oracle
import paper_2609_25451_amd as gms
import synth
from full_parity import entry_bytes, weight_parity
from gpu_util import need_gpu, to_u64


pytestmark = pytest.mark.gpu


def _free():
    gc.collect()
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    torch._C._host_emptyCache()  # pinned host blocks torch keeps cached for reuse


def _alloc_or_skip(fn):
    try:
        return fn()
    except torch.OutOfMemoryError as e:  # pragma: no cover - depends on the box
        _free()
        pytest.skip(f"not enough device memory: {e}")


def _weights(name):
    seed, specs = synth.weight_set(name)
    ts = [torch.empty(sp.shape, dtype=torch.bfloat16, device="cuda") for sp in specs]
    torch.cuda.synchronize()
    synth.dev_fill_tensors(ts, seed)  # one launch for the whole set
    return seed, specs, ts


def _weight_gen(seed, sizes):
    """gen(lo, hi, dst): generator bytes of tensors lo..hi-1 (bf16 stream k for tensor k)."""
    def gen(lo, hi, dst):
        ranges, o = [], 0
        for k in range(lo, hi):
            ranges.append((dst.data_ptr() + o, sizes[k] // 2, k))
            o += sizes[k]
        synth.dev_fill_bf16_many(ranges, seed)
    return gen


def _restored(ts):
    def cat(lo, hi):
        return torch.cat([ts[k].view(torch.uint8).reshape(-1) for k in range(lo, hi)])
    return cat


def _oracle_flip(gen, sizes, base, o_blk, i, byte, mask):
    """The oracle's verify of entry i with one bit flipped: (count, ascending global indices)."""
    x = entry_bytes(gen, sizes, i)
    x[byte] ^= mask
    nb = -(-sizes[i] // 4096)
    cnt, lst = oracle.verify([x], o_blk[base[i]:base[i] + nb])
    return cnt, [int(v) + base[i] for v in lst], oracle.entry_hashes(x)[0]


def _u64(t):
    torch.cuda.synchronize()
    return to_u64(t)


@pytest.mark.timeout(900)
@pytest.mark.parametrize("name", ["llama8b", "llama70b_tp8"])
def test_full_weight_set(name):
    need_gpu()
    _free()
    seed, specs, ts = _alloc_or_skip(lambda: _weights(name))
    sizes = [sp.nbytes for sp in specs]
    gen = _weight_gen(seed, sizes)
    m = gms.Manifest(ts, device=0)
    _, _, o_ib, o_nb = oracle.layout(sizes)
    assert m.image_bytes == o_ib and m.num_blocks == o_nb
    off, base = m.layout()
    img = _alloc_or_skip(lambda: torch.empty(m.image_bytes, dtype=torch.uint8, device="cuda"))
    z = lambda n: torch.zeros(n, dtype=torch.int64, device="cuda")  # noqa: E731
    blk, ten, blk2, ten2, blk3, ten3 = z(m.num_blocks), z(m.num_entries), z(m.num_blocks), z(m.num_entries), \
        z(m.num_blocks), z(m.num_entries)
    cnt = torch.full((1,), 99, dtype=torch.int64, device="cuda")
    gms.snapshot(m, img, m.image_bytes, blk_hash=blk, ten_hash=ten)
    for t in ts:
        t.view(torch.uint8).fill_(0xA5)
    gms.restore(m, img, m.image_bytes, expected=blk, blk_hash=blk2, ten_hash=ten2, mismatch_count=cnt)
    assert int(cnt.item()) == 0
    gms.verify(m, expected=blk, blk_hash=blk3, ten_hash=ten3, mismatch_count=cnt)
    assert int(cnt.item()) == 0

    # the pinned-host image through the staging ring: snapshot, poison, restore
    pinned = torch.empty(m.image_bytes, dtype=torch.uint8, pin_memory=True)
    blk_ps, blk_pr = z(m.num_blocks), z(m.num_blocks)
    gms.snapshot(m, pinned, m.image_bytes, gms.MEM_HOST_PINNED, blk_hash=blk_ps)
    for t in ts:
        t.view(torch.uint8).fill_(0xA5)
    gms.restore(m, pinned, m.image_bytes, gms.MEM_HOST_PINNED, expected=blk, blk_hash=blk_pr, mismatch_count=cnt)
    assert int(cnt.item()) == 0

    # every image byte, block hash and tensor hash against the oracle; restored bytes
    o_blk, o_ten = weight_parity(
        m, sizes, gen, {"device": img, "pinned": pinned},
        {"snapshot": _u64(blk), "restore": _u64(blk2), "verify": _u64(blk3), "pinned snapshot": _u64(blk_ps),
         "pinned restore": _u64(blk_pr)},
        {"snapshot": _u64(ten), "restore": _u64(ten2), "verify": _u64(ten3)},
        restored=_restored(ts))
    del pinned
    _free()

    # a planted bit flip in the image: the mismatch list is the oracle's verify of that entry
    rng = np.random.default_rng(sum(map(ord, name)))
    i = int(rng.integers(0, len(ts)))
    byte = int(rng.integers(0, sizes[i]))
    img[off[i] + byte] ^= 0x04
    lst = torch.zeros(4, dtype=torch.int64, device="cuda")
    blk_f = z(m.num_blocks)
    gms.restore(m, img, m.image_bytes, expected=blk, blk_hash=blk_f, mismatch_count=cnt, mismatch_list=lst,
                mismatch_cap=4)
    o_cnt, o_lst, o_flipped = _oracle_flip(gen, sizes, base, o_blk, i, byte, 0x04)
    assert int(cnt.item()) == o_cnt == 1 and sorted(_u64(lst)[:1].tolist()) == o_lst
    want = o_blk.copy()
    want[base[i]:base[i] + o_flipped.size] = o_flipped
    assert np.array_equal(_u64(blk_f), want)
    img[off[i] + byte] ^= 0x04
    gms.restore(m, img, m.image_bytes)  # the tensors took the flipped bit; restore the clean image
    m.close()
    del ts, img, blk, blk2, blk3, ten, ten2, ten3, blk_ps, blk_pr, blk_f
    _free()


@pytest.mark.timeout(900)
def test_full_kv_pool_live_blocks_and_corruption():
    need_gpu()
    _free()
    p = synth.kv_pool()
    pool = _alloc_or_skip(lambda: [torch.empty(p.layer_bytes, dtype=torch.uint8, device="cuda")
                                   for _ in range(p.layers)])
    for l, t in enumerate(pool):
        synth.dev_fill_bf16(t.data_ptr(), p.layer_bytes // 2, p.seed, l)
    live = synth.live_map(p.blocks, p.n_live, p.map_seed, p.map_stream)
    live_t = torch.from_numpy(live.astype(np.int64)).cuda()
    ents = [(pool[l].data_ptr() + int(b) * p.unit_bytes, p.unit_bytes) for l in range(p.layers) for b in live]
    m = gms.Manifest(ents, device=0)
    assert m.num_entries == 78_624 and m.payload_bytes == 5_152_702_464
    sizes = [p.unit_bytes] * m.num_entries
    off, base = m.layout()
    layer = torch.empty(p.layer_bytes, dtype=torch.uint8, device="cuda")

    def gen(lo, hi, dst):  # generator bytes of live units lo..hi-1 (layer-major, ids ascending)
        o, e = 0, lo
        while e < hi:
            l, j0 = divmod(e, p.n_live)
            j1 = min(p.n_live, j0 + hi - e)
            synth.dev_fill_bf16(layer.data_ptr(), p.layer_bytes // 2, p.seed, l)
            u = layer.view(p.blocks, p.unit_bytes)[live_t[j0:j1]].reshape(-1)
            dst[o:o + u.numel()].copy_(u)
            o, e = o + u.numel(), e + j1 - j0

    def restored(lo, hi):
        parts, e = [], lo
        while e < hi:
            l, j0 = divmod(e, p.n_live)
            j1 = min(p.n_live, j0 + hi - e)
            parts.append(pool[l].view(p.blocks, p.unit_bytes)[live_t[j0:j1]].reshape(-1))
            e += j1 - j0
        return torch.cat(parts)

    z = lambda n: torch.zeros(n, dtype=torch.int64, device="cuda")  # noqa: E731
    img = torch.empty(m.image_bytes, dtype=torch.uint8, device="cuda")
    exp, ten, blk2 = z(m.num_blocks), z(m.num_entries), z(m.num_blocks)
    cnt = torch.zeros(1, dtype=torch.int64, device="cuda")
    lst = torch.zeros(8, dtype=torch.int64, device="cuda")
    gms.snapshot(m, img, m.image_bytes, blk_hash=exp, ten_hash=ten)
    for t in pool:
        t.fill_(0xA5)
    gms.restore(m, img, m.image_bytes, expected=exp, blk_hash=blk2, mismatch_count=cnt)
    assert int(cnt.item()) == 0
    dead = torch.from_numpy(np.setdiff1d(np.arange(p.blocks), live)).cuda()
    for l, t in enumerate(pool):
        assert bool((t.view(p.blocks, p.unit_bytes)[dead] == 0xA5).all()), f"layer {l}: a dead unit was written"

    # whole image, block and tensor hashes against the oracle; restored live units
    o_blk, o_ten = weight_parity(m, sizes, gen, {"device": img}, {"snapshot": _u64(exp), "restore": _u64(blk2)},
                                 {"snapshot": _u64(ten)}, restored=restored)

    # the planted corruption (seeded), in the image: the oracle's verify decides the list
    e = synth.u64(p.corrupt_seed, p.corrupt_stream, 0) % m.num_entries
    bl = synth.u64(p.corrupt_seed, p.corrupt_stream, 1) % 16
    bit = synth.u64(p.corrupt_seed, p.corrupt_stream, 2) % (4096 * 8)
    byte, mask = bl * 4096 + bit // 8, 1 << (bit % 8)
    o_cnt, o_lst, o_flipped = _oracle_flip(gen, sizes, base, o_blk, e, byte, mask)
    want = o_blk.copy()
    want[base[e]:base[e] + 16] = o_flipped
    img[off[e] + byte] ^= mask
    for t in pool:
        t.fill_(0xA5)
    blk_f = z(m.num_blocks)
    gms.restore(m, img, m.image_bytes, expected=exp, blk_hash=blk_f, mismatch_count=cnt, mismatch_list=lst,
                mismatch_cap=8)
    assert int(cnt.item()) == o_cnt == 1 and _u64(lst)[:1].tolist() == o_lst == [base[e] + bl]
    assert np.array_equal(_u64(blk_f), want)
    for l, t in enumerate(pool):
        assert bool((t.view(p.blocks, p.unit_bytes)[dead] == 0xA5).all()), f"layer {l}: a dead unit was written"
    img[off[e] + byte] ^= mask

    # the same through a pinned host image and the staging ring
    pinned = torch.empty(m.image_bytes, dtype=torch.uint8, pin_memory=True)
    blk_ps, blk_pr = z(m.num_blocks), z(m.num_blocks)
    gms.restore(m, img, m.image_bytes)
    gms.snapshot(m, pinned, m.image_bytes, gms.MEM_HOST_PINNED, blk_hash=blk_ps)
    torch.cuda.synchronize()
    assert np.array_equal(_u64(blk_ps), o_blk)
    for lo in range(0, m.image_bytes, 1 << 30):  # the pinned image equals the (oracle-checked) device image
        hi = min(m.image_bytes, lo + (1 << 30))
        assert torch.equal(pinned[lo:hi].cuda(), img[lo:hi]), f"pinned image bytes {lo}..{hi}"
    pinned[off[e] + byte] ^= mask
    for t in pool:
        t.fill_(0xA5)
    gms.restore(m, pinned, m.image_bytes, gms.MEM_HOST_PINNED, expected=exp, blk_hash=blk_pr, mismatch_count=cnt,
                mismatch_list=lst, mismatch_cap=8)
    assert int(cnt.item()) == 1 and _u64(lst)[:1].tolist() == o_lst
    assert np.array_equal(_u64(blk_pr), want)
    del pinned
    _free()

    # verify before reattach: a flipped bit in the pool itself
    gms.restore(m, img, m.image_bytes)
    rng = np.random.default_rng(5)
    e2 = int(rng.integers(0, m.num_entries))
    b2 = int(rng.integers(0, p.unit_bytes))
    layer2, bid2 = e2 // p.n_live, int(live[e2 % p.n_live])
    pool[layer2][bid2 * p.unit_bytes + b2] ^= 0x80
    gms.verify(m, expected=exp, mismatch_count=cnt, mismatch_list=lst, mismatch_cap=8)
    o_cnt2, o_lst2, _ = _oracle_flip(gen, sizes, base, o_blk, e2, b2, 0x80)
    assert int(cnt.item()) == o_cnt2 == 1 and _u64(lst)[:1].tolist() == o_lst2
    m.close()
    del pool, img, exp, layer
    _free()


@pytest.mark.timeout(1200)
def test_full_moe_shard_device_and_host_image():
    """122 GB over 18,771 tensors: the device-image leg needs about 245 GB of HBM
    (allocations + image); the pageable-host leg then restores from 122 GB of host memory."""
    need_gpu()
    _free()
    free, _ = torch.cuda.mem_get_info()
    _, specs = synth.weight_set("moe")
    P = sum(sp.nbytes for sp in specs)
    if free < 2 * P + (8 << 30):
        pytest.skip(f"needs {2 * P / 1e9:.0f} GB free, have {free / 1e9:.0f} GB")
    seed, specs, ts = _alloc_or_skip(lambda: _weights("moe"))
    sizes = [sp.nbytes for sp in specs]
    gen = _weight_gen(seed, sizes)
    m = gms.Manifest(ts, device=0)
    assert m.num_entries == 18_771 and m.payload_bytes == 122_143_121_408
    z = lambda n: torch.zeros(n, dtype=torch.int64, device="cuda")  # noqa: E731
    img = _alloc_or_skip(lambda: torch.empty(m.image_bytes, dtype=torch.uint8, device="cuda"))
    blk, ten, blk2 = z(m.num_blocks), z(m.num_entries), z(m.num_blocks)
    cnt = torch.full((1,), 9, dtype=torch.int64, device="cuda")
    gms.snapshot(m, img, m.image_bytes, blk_hash=blk, ten_hash=ten)
    for t in ts:
        t.view(torch.uint8).fill_(0xA5)
    gms.restore(m, img, m.image_bytes, expected=blk, blk_hash=blk2, mismatch_count=cnt)
    assert int(cnt.item()) == 0
    h_blk, h_ten, h_blk2 = _u64(blk), _u64(ten), _u64(blk2)
    del img
    _free()
    o_blk, _ = weight_parity(m, sizes, gen, {}, {"snapshot": h_blk, "restore": h_blk2}, {"snapshot": h_ten},
                             restored=_restored(ts))

    # the pageable host image: snapshot into ordinary host memory, poison, restore from it
    host = np.empty(m.image_bytes, dtype=np.uint8)
    blk_hs, blk_hr = z(m.num_blocks), z(m.num_blocks)
    gms.snapshot_to_host(m, host, blk_hash=blk_hs)
    for t in ts:
        t.view(torch.uint8).fill_(0xA5)
    gms.restore_from_host(m, host, expected=blk, blk_hash=blk_hr, mismatch_count=cnt)
    assert int(cnt.item()) == 0
    weight_parity(m, sizes, gen, {"host": host}, {"host snapshot": _u64(blk_hs), "host restore": _u64(blk_hr)}, {},
                  restored=_restored(ts))
    assert np.array_equal(h_blk, o_blk)
    del host
    m.close()
    del ts, blk, blk2, blk_hs, blk_hr
    _free()


def test_entry_larger_than_4gib():
    """One 4 GiB + 12,345-byte entry (byte offsets and word indices past 32 bits), a small
    one behind it: every block hash and both tensor hashes equal the oracle's, and the fused
    restore of the whole entry verifies against them."""
    need_gpu()
    big = (4 << 30) + 12_345
    sizes = [big, 5000]
    ts = _alloc_or_skip(lambda: [torch.empty(n, dtype=torch.uint8, device="cuda") for n in sizes])
    for i, (t, n) in enumerate(zip(ts, sizes)):
        synth.dev_fill_bytes(t.data_ptr(), n, 41, i)
    datas = [synth.random_bytes(n, 41, i) for i, n in enumerate(sizes)]
    o_blk, o_ten = oracle.hashes(datas)
    m = gms.Manifest(ts, device=0)
    assert m.num_blocks == o_blk.size
    img = _alloc_or_skip(lambda: torch.empty(m.image_bytes, dtype=torch.uint8, device="cuda"))
    blk = torch.zeros(m.num_blocks, dtype=torch.int64, device="cuda")
    ten = torch.zeros(2, dtype=torch.int64, device="cuda")
    gms.snapshot(m, img, m.image_bytes, blk_hash=blk, ten_hash=ten)
    torch.cuda.synchronize()
    assert np.array_equal(to_u64(blk), o_blk) and np.array_equal(to_u64(ten), o_ten)
    # image bytes at sampled offsets, including the last ones of the big entry and the pad
    off, _ = m.layout()
    h_img = {}
    for o in (0, (1 << 32) - 16, (1 << 32) + 4096, big - 7, off[1] + 4999):
        h_img[o] = img[o:o + 8].cpu().numpy()
    assert np.array_equal(h_img[0], datas[0][:8])
    assert np.array_equal(h_img[(1 << 32) - 16], datas[0][(1 << 32) - 16:(1 << 32) - 8])
    assert np.array_equal(h_img[(1 << 32) + 4096], datas[0][(1 << 32) + 4096:(1 << 32) + 4104])
    assert np.array_equal(h_img[big - 7][:7], datas[0][-7:]) and not h_img[big - 7][7:].any()
    assert h_img[off[1] + 4999][0] == datas[1][-1] and not h_img[off[1] + 4999][1:].any()
    for t in ts:
        t.fill_(0xA5)
    cnt = torch.zeros(1, dtype=torch.int64, device="cuda")
    ten2 = torch.zeros(2, dtype=torch.int64, device="cuda")
    gms.restore(m, img, m.image_bytes, expected=torch.from_numpy(o_blk.view(np.int64)).cuda(), ten_hash=ten2,
                mismatch_count=cnt)
    torch.cuda.synchronize()
    assert int(cnt.item()) == 0 and np.array_equal(to_u64(ten2), o_ten)
    assert np.array_equal(ts[0][-4096:].cpu().numpy(), datas[0][-4096:])
    assert np.array_equal(ts[1].cpu().numpy(), datas[1])
    m.close()
    del ts, img, blk
    _free()
