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
