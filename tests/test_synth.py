"""The seeded input generator: published Philox vectors, distribution, live map."""
import os

import numpy as np
import torch

import synth

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def test_philox_known_answers():
    n = 0
    with open(os.path.join(GOLDEN, "philox4x32_10_kat.txt")) as f:
        for line in f:
            if not line.strip() or line.startswith("#"):
                continue
            v = [int(t, 16) for t in line.split()]
            assert synth.philox(v[0:4], v[4:6]) == v[6:10]
            n += 1
    assert n == 3


def test_bf16_matches_float_rounding():
    """Integer RNE of (f32 sum * f32 scale) equals torch's f32 -> bf16 conversion."""
    n = 4096
    bits = synth.bf16_bits(n, seed=1, tensor=3)
    scale = np.array([0x350DE3BD], dtype=np.uint32).view(np.float32)[0]
    assert abs(float(scale) - 0.02 / 37837.227237) < 1e-12
    s = []
    for e in range(n):
        d = synth.philox([(e >> 1) & 0xFFFFFFFF, e >> 33, 3, 0], [1, 0])
        a, b = (d[0], d[1]) if e % 2 == 0 else (d[2], d[3])
        s.append((a & 0xFFFF) + (a >> 16) + (b & 0xFFFF) + (b >> 16) - 131070)
    f = np.array(s, dtype=np.float32) * scale
    ref = torch.from_numpy(f).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(bits, ref)


def test_bf16_distribution():
    bits = synth.bf16_bits(1_000_000, seed=2, tensor=0)
    f = torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16).float().numpy()
    assert abs(f.mean()) < 1e-4
    assert abs(f.std() / 0.02 - 1) < 0.01
    assert np.abs(f).max() < 0.0694  # support of the scaled Irwin-Hall sum


def test_offsets_and_streams():
    a = synth.bf16_bits(100, 7, 4)
    assert np.array_equal(synth.bf16_bits(37, 7, 4, first=63), a[63:])
    assert not np.array_equal(synth.bf16_bits(100, 7, 5), a)
    assert not np.array_equal(synth.bf16_bits(100, 8, 4), a)
    b = synth.random_bytes(1000, 3, 9)
    assert np.array_equal(synth.random_bytes(500, 3, 9, first=333), b[333:833])


def test_live_map():
    p = synth.kv_pool()
    live = synth.live_map(p.blocks, p.n_live, p.map_seed, p.map_stream)
    assert live.size == 2457 and np.all(np.diff(live.astype(np.int64)) > 0)
    assert live[0] >= 0 and live[-1] < p.blocks
    runs = 1 + int(np.count_nonzero(np.diff(live.astype(np.int64)) > 1))
    # a uniform 60% subset of 4096 ids has about 4096*0.6*0.4 ~ 983 runs
    assert 900 < runs < 1070
    again = synth.live_map(p.blocks, p.n_live, p.map_seed, p.map_stream)
    assert np.array_equal(live, again)
    assert not np.array_equal(live, synth.live_map(p.blocks, p.n_live, p.map_seed + 1, p.map_stream))


def test_workload_sizes():
    want = {
        "tiny": (21, 8_391_168),
        "llama8b": (291, 16_060_522_496),
        "llama70b_tp8": (723, 17_640_734_720),
        "moe": (18_771, 122_143_121_408),
    }
    for name, (n, b) in want.items():
        _, ts = synth.weight_set(name)
        assert len(ts) == n and sum(t.nbytes for t in ts) == b
    p = synth.kv_pool()
    assert p.layers * p.layer_bytes == 8 << 30 and p.unit_bytes == 65536
    assert p.n_live * p.layers * p.unit_bytes == 5_152_702_464


# An independent evaluation of the generator's definition, for golden vectors: Philox4x32-10
# (Salmon, Moraes, Dror and Shaw, SC'11) in plain Python integers, and the live map's
# Fisher-Yates shuffle.  It shares no code with synth/.
_M0, _M1, _W0, _W1, _MASK = 0xD2511F53, 0xCD9E8D57, 0x9E3779B9, 0xBB67AE85, 0xFFFFFFFF


def _py_philox(c, k):
    c, (k0, k1) = list(c), k
    for _ in range(10):
        p0, p1 = _M0 * c[0], _M1 * c[2]
        c = [((p1 >> 32) ^ c[1] ^ k0) & _MASK, p1 & _MASK, ((p0 >> 32) ^ c[3] ^ k1) & _MASK, p0 & _MASK]
        k0, k1 = (k0 + _W0) & _MASK, (k1 + _W1) & _MASK
    return c


def _py_u64(seed, stream, index):
    r = _py_philox([index & _MASK, index >> 32, stream & _MASK, stream >> 32], [seed & _MASK, seed >> 32])
    return r[0] | (r[1] << 32)


def _py_live_map(nblocks, nlive, seed, stream):
    perm = list(range(nblocks))
    for i in range(nblocks - 1, 0, -1):
        j = _py_u64(seed, stream, nblocks - 1 - i) % (i + 1)
        perm[i], perm[j] = perm[j], perm[i]
    return sorted(perm[:nlive])


def _golden_kv():
    out = {}
    with open(os.path.join(GOLDEN, "kv_pool_default.txt")) as f:
        for line in f:
            if line.strip() and not line.startswith("#"):
                key, *vals = line.split()
                out[key] = [int(v) for v in vals]
    return out


def test_kv_pool_golden_vectors():
    """The default pool's live map and planted corruption site: the pure-Python evaluation of
    the generator's definition, the golden file and the generator library all agree, and the
    expected mismatch index is the corrupted unit's global block (16 blocks per 64 KiB unit)."""
    g = _golden_kv()
    p = synth.kv_pool()
    py_live = _py_live_map(p.blocks, p.n_live, p.map_seed, p.map_stream)
    runs = 1 + sum(1 for a, b in zip(py_live, py_live[1:]) if b - a > 1)
    assert [len(py_live)] == g["live_count"]
    assert py_live[:8] == g["live_first"] and py_live[-4:] == g["live_last"]
    assert [runs] == g["live_runs"] and [sum(py_live)] == g["live_id_sum"]
    assert synth.live_map(p.blocks, p.n_live, p.map_seed, p.map_stream).tolist() == py_live
    n_entries = p.layers * p.n_live
    units_blocks = p.unit_bytes // 4096
    e = _py_u64(p.corrupt_seed, p.corrupt_stream, 0) % n_entries
    bl = _py_u64(p.corrupt_seed, p.corrupt_stream, 1) % units_blocks
    bit = _py_u64(p.corrupt_seed, p.corrupt_stream, 2) % (4096 * 8)
    assert ([e], [bl], [bit]) == (g["corrupt_entry"], g["corrupt_block"], g["corrupt_bit"])
    assert [synth.u64(p.corrupt_seed, p.corrupt_stream, k) for k in range(3)] == \
        [_py_u64(p.corrupt_seed, p.corrupt_stream, k) for k in range(3)]
    assert [e * units_blocks + bl] == g["mismatch_index"]
    # the known-answer vectors hold for the Python evaluation too
    with open(os.path.join(GOLDEN, "philox4x32_10_kat.txt")) as f:
        for line in f:
            if line.strip() and not line.startswith("#"):
                v = [int(t, 16) for t in line.split()]
                assert _py_philox(v[0:4], v[4:6]) == v[6:10]
