"""C-ABI surface on the CPU: symbols, layout queries, argument validation.

Host-only manifests (device = -1) exercise every host-side rule without a GPU;
no data-plane call here reaches a kernel.
"""
import ctypes
import subprocess

import numpy as np
import pytest

import oracle
import paper_2609_25451_amd as gms
import synth


def test_exports_every_declared_symbol():
    declared = gms.exported_symbols_declared()
    assert "gms_restore" in declared and "gms_manifest_create" in declared
    out = subprocess.run(["nm", "-D", "--defined-only", gms.LIB_PATH], capture_output=True, text=True,
                         check=True).stdout
    exported = {line.split()[-1] for line in out.splitlines() if line.strip()}
    missing = [s for s in declared if s not in exported]
    assert not missing, f"declared but not exported: {missing}"
    assert gms.abi_version() == 5


def _host_manifest(sizes, base=1 << 40, gap=0, chunk_bytes=0, align=1):
    ents, a = [], base
    for s in sizes:
        a = (a + align - 1) // align * align
        ents.append((a, s))
        a += s + gap
    return gms.Manifest(ents, device=gms.HOST_ONLY, chunk_bytes=chunk_bytes)


def test_layout_matches_oracle():
    rng = np.random.default_rng(1)
    for _ in range(30):
        sizes = [int(v) for v in rng.integers(0, 50_000, rng.integers(0, 40))]
        m = _host_manifest(sizes, gap=int(rng.integers(0, 9)))
        off, base = m.layout()
        o_off, o_base, o_ib, o_nb = oracle.layout(sizes)
        assert off == [int(v) for v in o_off] and base == [int(v) for v in o_base]
        assert m.image_bytes == o_ib and m.num_blocks == o_nb and m.payload_bytes == sum(sizes)
        assert m.num_entries == len(sizes)


def _expected_chunks(sizes, cb):
    n, off = 0, 0
    for s in sizes:
        pos = 0
        while pos < s:
            img = off + pos
            pos += min(s - pos, (img // cb + 1) * cb - img)
            n += 1
        off += -(-s // 4096) * 4096
    return n


@pytest.mark.parametrize("name", ["tiny", "llama8b", "llama70b_tp8"])
def test_workload_layouts(name):
    _, ts = synth.weight_set(name)
    sizes = [t.nbytes for t in ts]
    m = _host_manifest(sizes)
    _, _, ib, nb = oracle.layout(sizes)
    assert m.image_bytes == ib and m.num_blocks == nb
    assert m.num_chunks == _expected_chunks(sizes, 64 * 1024)
    m4 = _host_manifest(sizes, chunk_bytes=1 << 20)
    assert m4.num_chunks == _expected_chunks(sizes, 1 << 20)


def test_kv_pool_layout():
    p = synth.kv_pool()
    live = synth.live_map(p.blocks, p.n_live, p.map_seed, p.map_stream)
    ents = [((1 << 40) + l * p.layer_bytes + int(b) * p.unit_bytes, p.unit_bytes)
            for l in range(p.layers) for b in live]
    m = gms.Manifest(ents, device=gms.HOST_ONLY)
    assert m.num_entries == 78_624 and m.payload_bytes == 5_152_702_464 == m.image_bytes
    assert m.num_blocks == 78_624 * 16 and m.num_chunks == 78_624


def test_overlap_and_bad_ranges_rejected():
    with pytest.raises(gms.GmsError) as e:
        gms.Manifest([(4096, 100), (4096 + 99, 10)], device=gms.HOST_ONLY)
    assert e.value.status == gms.GMS_ERR_OVERLAP
    # touching ranges and zero-length entries anywhere are fine
    m = gms.Manifest([(4096, 100), (4196, 10), (4150, 0), (0, 0)], device=gms.HOST_ONLY)
    assert m.num_entries == 4 and m.num_blocks == 2
    for bad in ([(0, 8)], [((1 << 64) - 8, 16)]):
        with pytest.raises(gms.GmsError) as e:
            gms.Manifest(bad, device=gms.HOST_ONLY)
        assert e.value.status == gms.GMS_ERR_INVALID
    for cb in (1000, 4096 * 3 + 1, 128 << 20):
        with pytest.raises(gms.GmsError) as e:
            gms.Manifest([(4096, 10)], device=gms.HOST_ONLY, chunk_bytes=cb)
        assert e.value.status == gms.GMS_ERR_INVALID


def test_empty_manifest():
    m = gms.Manifest([], device=gms.HOST_ONLY)
    assert m.num_entries == 0 and m.image_bytes == 0 and m.num_blocks == 0 and m.num_chunks == 0
    assert m.layout() == ([], [])


def test_data_plane_refused_on_host_only_manifest():
    m = _host_manifest([5000, 3])
    for call in (lambda: gms.snapshot(m, 1 << 30, m.image_bytes, stream=0),
                 lambda: gms.restore(m, 1 << 30, m.image_bytes, stream=0),
                 lambda: gms.verify(m, blk_hash=1 << 30, stream=0)):
        with pytest.raises(gms.GmsError) as e:
            call()
        assert e.value.status == gms.GMS_ERR_STATE
    with pytest.raises(gms.GmsError) as e:
        m.set_staging(1 << 20, 2)
    assert e.value.status == gms.GMS_ERR_STATE
    host = np.zeros(m.image_bytes, dtype=np.uint8)
    for call in (lambda: gms.restore_from_file(m, "/nonexistent"),
                 lambda: gms.snapshot_to_file(m, "/nonexistent"),
                 lambda: gms.restore_from_host(m, host, stream=0),
                 lambda: gms.snapshot_to_host(m, host, stream=0)):
        with pytest.raises(gms.GmsError) as e:
            call()
        assert e.value.status == gms.GMS_ERR_STATE
    with pytest.raises(ValueError, match="non-contiguous"):  # refused by the binding before the call
        gms.snapshot_to_host(m, np.zeros((2, m.image_bytes), np.uint8)[:, ::2], stream=0)
    with pytest.raises(ValueError, match="image_bytes"):
        gms.restore_from_host(m, 1 << 30, stream=0)


def test_null_arguments():
    out = ctypes.c_void_p()
    assert gms.gms_manifest_create(None, 3, gms.HOST_ONLY, 0, ctypes.byref(out)) == gms.GMS_ERR_INVALID
    assert gms.gms_manifest_create(None, 0, gms.HOST_ONLY, 0, None) == gms.GMS_ERR_INVALID
    assert gms.gms_snapshot(None, None, 0, 0, None, None, None) == gms.GMS_ERR_INVALID
    assert gms.gms_restore(None, None, 0, 0, None, None, None, None, None, 0, None) == gms.GMS_ERR_INVALID
    assert gms.gms_verify(None, None, None, None, None, None, 0, None) == gms.GMS_ERR_INVALID
    assert b"null" in gms.gms_last_error()
    assert gms.gms_restore_from_file(None, b"x", 0, 0, 0, None, None, None, None, None, 0, None) == gms.GMS_ERR_INVALID
    assert gms.gms_snapshot_to_file(None, b"x", 0, 0, None, None, None) == gms.GMS_ERR_INVALID
    m = gms.Manifest([(4096, 10)], device=gms.HOST_ONLY)
    assert gms.gms_restore_from_file(m.handle, None, 0, 0, 0, None, None, None, None, None, 0, None) == gms.GMS_ERR_STATE
    for rc in (0, -1, -2, -3, -4, -5, -6, -7, 7):
        assert gms.status_str(rc)


def test_non_contiguous_tensors_refused_by_the_binding():
    """A strided view is not the byte range [data_ptr, data_ptr + nbytes): the binding refuses it
    as an entry, an image or an output array before any library call."""
    import torch

    t = torch.zeros(64, 64, dtype=torch.bfloat16)
    col = t[:, 3]
    assert not col.is_contiguous()
    with pytest.raises(ValueError, match="non-contiguous"):
        gms.Manifest([col], device=gms.HOST_ONLY)
    m = gms.Manifest([t], device=gms.HOST_ONLY)
    assert m.payload_bytes == t.numel() * 2
    with pytest.raises(ValueError, match="non-contiguous"):
        gms.snapshot(m, torch.zeros(4, 8192, dtype=torch.uint8)[:, ::2], m.image_bytes, stream=0)
    with pytest.raises(ValueError, match="non-contiguous"):
        gms.verify(m, blk_hash=torch.zeros(8, 2, dtype=torch.int64)[:, 0], stream=0)
    m.close()


def test_launch_groups_split_only_when_idle_units_pay_for_a_launch():
    """A chunk of at most 8 KiB needs one work unit (two 4 KiB blocks); a 64 KiB chunk needs
    eight.  Tiny chunks beside large ones get a launch of their own once the idle units they would
    leave (7 each) reach 16,384; a manifest of similar chunks is a single launch."""
    big = [64 << 20] * 4
    hm = lambda sizes: _host_manifest(sizes, align=256)  # noqa: E731  (torch-like 256-byte alignment)
    assert hm(big).num_launch_groups == 1
    assert hm(big + [100] * 2340).num_launch_groups == 1  # 16,380 idle units
    assert hm(big + [100] * 2341).num_launch_groups == 2  # 16,387
    assert hm([100] * 200_000).num_launch_groups == 1
    assert hm([]).num_launch_groups == 0
    # a middle class too small to pay for a launch stays in the large chunks' launch
    m = hm(big + [100] * 3000 + [20_000] * 10)  # 20,000 B: 5 blocks, 3 units -> 4
    assert m.num_launch_groups == 2
    # the weight sets and the KV pool
    for name, groups in (("tiny", 1), ("llama8b", 1), ("llama70b_tp8", 1), ("moe", 3)):
        _, ts = synth.weight_set(name)
        assert hm([t.nbytes for t in ts]).num_launch_groups == groups, name
    # entries off a 16-byte boundary get launches of their own beside aligned ones of the same
    # size class; a manifest of only one kind stays one launch per class
    assert _host_manifest(big, base=(1 << 40) + 2).num_launch_groups == 1
    assert _host_manifest([100] * 1000, base=(1 << 40) + 3, align=256).num_launch_groups == 1
    assert _host_manifest([100] * 1000).num_launch_groups == 2  # 100-byte steps: a quarter aligned
    assert _host_manifest(big + [100] * 3000, gap=2).num_launch_groups == 4
    m = _host_manifest(big + [100] * 3000, gap=2)
    assert m.image_bytes == hm(big + [100] * 3000).image_bytes
    # the layout does not depend on the grouping
    sizes = big + [100] * 3000
    m, m1 = _host_manifest(sizes), _host_manifest(sizes[:4])
    off, _ = m.layout()
    assert off[:4] == m1.layout()[0] and m.image_bytes == m1.image_bytes + 3000 * 4096


def test_scattered_units_take_the_striped_order():
    """A launch group whose chunks are mostly entries of their own (the KV pool's 64 KiB live
    units) restores and snapshots in the striped unit order; weight sets, whose tensors span many chunks,
    keep the contiguous eighths.  The query reports every group of a manifest."""
    p = synth.kv_pool()
    live = synth.live_map(p.blocks, p.n_live, p.map_seed, p.map_stream)
    ents = [((1 << 40) + l * p.layer_bytes + int(b) * p.unit_bytes, p.unit_bytes) for l in range(4) for b in live]
    kv = gms.Manifest(ents, device=gms.HOST_ONLY)
    assert kv.launch_groups() == [{"chunks": len(ents), "unit_shift": 3, "shifted": False, "striped": True}]
    kv.close()
    for name in ("llama8b", "llama70b_tp8", "moe"):
        _, ts = synth.weight_set(name)
        gs = _host_manifest([t.nbytes for t in ts], align=256).launch_groups()
        assert not gs[0]["striped"] and sum(g["chunks"] for g in gs) > 0, name
    # mixed: the large tensors' groups keep the eighths, the tiny buffers' groups are paired
    # launches, which have an order of their own
    gs = _host_manifest([64 << 20] * 4 + [100] * 3000, gap=2).launch_groups()
    assert [(g["unit_shift"] > 0, g["shifted"], g["striped"]) for g in gs] == [
        (True, False, False), (True, True, False), (False, False, False), (False, True, False)]
    m = _host_manifest([4096])
    assert gms._launch_group(m._h, 1, None, None, None) == gms.GMS_ERR_INVALID
    assert gms._launch_group(None, 0, None, None, None) == gms.GMS_ERR_INVALID


def test_binding_refuses_short_or_mistyped_outputs():
    """The C side can only check that a pointer range lies inside one allocation, and under a
    caching allocator that is a whole segment; the binding therefore checks each tensor or
    array against its own size and element type before the call (nothing reaches the library)."""
    import torch

    m = _host_manifest([5000, 3000, 0, 12_288])  # 2 + 1 + 0 + 3 blocks, 4 entries
    nb, ne = m.num_blocks, m.num_entries
    assert (nb, ne) == (6, 4)
    short = [np.zeros(nb - 1, np.uint64), torch.zeros(nb - 1, dtype=torch.int64)]
    mistyped = [np.zeros(nb, np.int32), np.zeros(nb, np.float64), torch.zeros(2 * nb, dtype=torch.int32),
                torch.zeros(nb, dtype=torch.float64)]
    for bad in short:
        for call in (lambda: gms.verify(m, blk_hash=bad, stream=0),
                     lambda: gms.verify(m, expected=bad, mismatch_count=np.zeros(1, np.uint64), stream=0),
                     lambda: gms.snapshot(m, np.zeros(m.image_bytes, np.uint8), blk_hash=bad, stream=0),
                     lambda: gms.restore(m, np.zeros(m.image_bytes, np.uint8), expected=bad,
                                         mismatch_count=np.zeros(1, np.uint64), stream=0)):
            with pytest.raises(ValueError, match="holds"):
                call()
    for bad in mistyped:
        with pytest.raises(ValueError, match="64-bit integer"):
            gms.verify(m, blk_hash=bad, stream=0)
    with pytest.raises(ValueError, match="ten_hash"):
        gms.verify(m, ten_hash=np.zeros(ne - 1, np.uint64), stream=0)
    with pytest.raises(ValueError, match="mismatch_count"):
        gms.verify(m, expected=np.zeros(nb, np.uint64), mismatch_count=np.zeros(0, np.uint64), stream=0)
    # the list must hold min(cap, blocks) entries
    with pytest.raises(ValueError, match="mismatch_list"):
        gms.verify(m, expected=np.zeros(nb, np.uint64), mismatch_count=np.zeros(1, np.uint64),
                   mismatch_list=np.zeros(3, np.uint64), mismatch_cap=4, stream=0)
    # a claimed image size beyond the buffer
    with pytest.raises(ValueError, match="image_bytes"):
        gms.restore(m, np.zeros(m.image_bytes, np.uint8), m.image_bytes + 1, stream=0)
    with pytest.raises(ValueError, match="image_bytes"):
        gms.snapshot_to_host(m, torch.zeros(m.image_bytes - 1, dtype=torch.uint8), m.image_bytes, stream=0)
    # well-formed outputs pass the binding and reach the library (which refuses a host-only manifest)
    ok = dict(expected=np.zeros(nb, np.uint64), blk_hash=torch.zeros(nb, dtype=torch.int64),
              ten_hash=np.zeros(ne, np.int64), mismatch_count=np.zeros(1, np.uint64),
              mismatch_list=np.zeros(2, np.uint64), mismatch_cap=2)
    with pytest.raises(gms.GmsError) as e:
        gms.verify(m, stream=0, **ok)
    assert e.value.status == gms.GMS_ERR_STATE
    with pytest.raises(gms.GmsError) as e:
        gms.restore(m, np.zeros(m.image_bytes, np.uint8), stream=0, **ok)
    assert e.value.status == gms.GMS_ERR_STATE
