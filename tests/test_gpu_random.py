"""Seeded random manifests through every combination the launch planner can make: chunk
sizes from 4 KiB to 1 MiB, entries at any byte alignment, sizes from one byte to a few MiB,
mixes that split into paired and unit launches and into striped and contiguous unit orders,
device images and pinned images through small staging rings.  Each case is the oracle round
trip: snapshot image and hashes, a fused restore into poisoned memory with sentinels around
every entry, and verify, all equal to the oracle."""
import numpy as np
import pytest

import paper_2609_25451_amd as gms
from gpu_util import Arena, need_gpu, random_datas
from test_gpu_parity import _round_trip

pytestmark = pytest.mark.gpu

CHUNKS = [4096, 16384, 65536, 262144, 1 << 20]


def _case(seed):
    rng = np.random.default_rng(seed)
    mix = []
    for _ in range(int(rng.integers(1, 4))):  # a few families of sizes
        kind = int(rng.integers(0, 4))
        count = int(rng.integers(1, 400))
        if kind == 0:
            mix += [int(v) for v in rng.integers(1, 9000, count)]        # paired-launch sizes
        elif kind == 1:
            mix += [int(rng.choice([16384, 32768, 65536]))] * count      # one-chunk units
        elif kind == 2:
            mix += [int(v) for v in rng.integers(9000, 300_000, count // 4 + 1)]
        else:
            mix += [int(v) for v in rng.integers(1 << 20, 6 << 20, 3)]  # entries of many chunks
    rng.shuffle(mix)
    p_mis = float(rng.choice([0.0, 0.3, 1.0]))
    chunk = int(rng.choice(CHUNKS))
    pinned = bool(rng.integers(0, 3) == 0)
    return mix, p_mis, chunk, pinned


@pytest.mark.parametrize("seed", range(24))
def test_random_manifest_round_trip(seed):
    need_gpu()
    sizes, p_mis, chunk, pinned = _case(1000 + seed)
    print(f"case {seed}: {len(sizes)} entries, {sum(sizes)} B, chunk {chunk}, misaligned {p_mis}, "
          f"pinned {pinned}", flush=True)
    arena = Arena(sizes, misalign=lambda r: r.integers(1, 16) if r.random() < p_mis else 0, gap=24,
                  seed=2000 + seed)
    datas = random_datas(sizes, seed=3000 + seed)
    arena.fill(datas)
    staging = (max(chunk, 1 << 20), 2) if pinned else None
    m, _ = _round_trip(arena, datas, gms.MEM_HOST_PINNED if pinned else gms.MEM_DEVICE, chunk_bytes=chunk,
                       staging=staging)
    groups = m.launch_groups()
    assert sum(g["chunks"] for g in groups) == m.num_chunks
    m.close()
