"""Pins of the CPU oracle against facts fixed outside it.

Each ``pin_*`` takes an ``oracle.Oracle`` and raises AssertionError when the
oracle disagrees with a published value, a closed form, an invariant of the
definition, or brute force.  test_oracle.py runs them on the real oracle;
test_oracle_mutants.py runs them on builds of the oracle with planted
mistakes and requires every mistake to be caught.
"""
from __future__ import annotations

import os

import numpy as np

M64 = (1 << 64) - 1
G = 0x9E3779B97F4A7C15
C1 = 0xBF58476D1CE4E5B9
C2 = 0x94D049BB133111EB
GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")
BLOCK = 4096


def splitmix64_published():
    vals = {}
    with open(os.path.join(GOLDEN, "splitmix64_seed0.txt")) as f:
        for line in f:
            if line.strip() and not line.startswith("#"):
                k, v = line.split()
                vals[int(k)] = int(v, 16)
    return vals


def _le64(v: int) -> bytes:
    return int(v & M64).to_bytes(8, "little")


def _unxorshift(z: int, s: int) -> int:
    y = z
    for _ in range(64 // s + 1):
        y = z ^ (y >> s)
    return y & M64


def fmix_inverse(z: int) -> int:
    """Inverse of the mixer, from the inverses of its steps (odd multipliers are units mod 2^64)."""
    z = _unxorshift(z, 31)
    z = (z * pow(C2, -1, 1 << 64)) & M64
    z = _unxorshift(z, 27)
    z = (z * pow(C1, -1, 1 << 64)) & M64
    z = _unxorshift(z, 30)
    return z


def splitmix64_stream(count: int):
    """splitmix64 outputs 1..count from state 0, by the published algorithm."""
    out, s = [], 0
    for _ in range(count):
        s = (s + G) & M64
        z = s
        z = ((z ^ (z >> 30)) * C1) & M64
        z = ((z ^ (z >> 27)) * C2) & M64
        out.append(z ^ (z >> 31))
    return out


# --------------------------------------------------------------------------- pins


def pin_splitmix_published(o):
    pub = splitmix64_published()
    for k, v in pub.items():
        assert o.fmix((k * G) & M64) == v, f"mix({k}G) != published splitmix64 output {k}"
    assert o.fmix(0) == 0


def pin_fmix_bijective(o):
    rng = np.random.default_rng(7)
    for z in [0, 1, G, M64] + [int(x) for x in rng.integers(0, 1 << 63, 300, dtype=np.uint64)]:
        assert fmix_inverse(o.fmix(z)) == z, f"mixer does not invert at {z:#x}"


def pin_word_order_and_index(o):
    """Words chosen so that word j XOR j*G = (j+1)*G: each h is a published output."""
    pub = splitmix64_published()
    raw = b"".join(_le64(((j + 1) * G) ^ (j * G)) for j in range(3))
    x = np.frombuffer(raw, dtype=np.uint8)
    assert o.word(x, 0) == G, "little-endian word assembly"
    blk, ten = o.entry_hashes(x)
    want = pub[1] ^ pub[2] ^ pub[3]
    assert len(blk) == 1 and int(blk[0]) == want and ten == want


def pin_block_membership(o):
    """W_j = j*G makes every word hash to mix(0) = 0, except planted words whose
    h is a published splitmix64 output; only their blocks may be non-zero."""
    pub = splitmix64_published()
    nwords = 3 * 512 + 5
    words = [(j * G) & M64 for j in range(nwords)]
    plant = {0: 1, 511: 2, 512: 3, 1023: 1, 1024 + 7: 2, nwords - 1: 3}
    for j, k in plant.items():
        words[j] ^= (k * G) & M64
    x = np.frombuffer(b"".join(_le64(w) for w in words), dtype=np.uint8)
    blk, ten = o.entry_hashes(x)
    want = [0, 0, 0, 0]
    for j, k in plant.items():
        want[j // 512] ^= pub[k]
    assert [int(b) for b in blk] == want, f"block membership {[hex(int(b)) for b in blk]}"
    acc = 0
    for v in want:
        acc ^= v
    assert ten == acc


def pin_zero_extension(o):
    rng = np.random.default_rng(11)
    for n in [1, 5, 7, 8, 9, 15, 4095, 4097, 6001]:
        x = rng.integers(0, 256, n, dtype=np.uint8)
        pad = (-n) % 8
        same = np.concatenate([x, np.zeros(pad, np.uint8)])
        longer = np.concatenate([x, np.zeros(pad + 8, np.uint8)])
        bx, tx = o.entry_hashes(x)
        bs, ts = o.entry_hashes(same)
        assert tx == ts and np.array_equal(bx, bs), f"partial final word must read as zero-extended (n={n})"
        _, tl = o.entry_hashes(longer)
        assert tl != tx, f"an extra zero word must change the hash (n={n})"


def pin_zero_blocks_closed_form(o):
    s = splitmix64_stream(1023)  # s[k-1] = mix(k*G)
    z = np.zeros(2 * BLOCK, dtype=np.uint8)
    blk, ten = o.entry_hashes(z)
    b0 = 0
    for k in range(1, 512):
        b0 ^= s[k - 1]
    b1 = 0
    for k in range(512, 1024):
        b1 ^= s[k - 1]
    assert int(blk[0]) == b0 and int(blk[1]) == b1 and ten == b0 ^ b1


def pin_bitflip_exhaustive(o):
    """mix is a bijection, so any single-word change alters its block hash."""
    rng = np.random.default_rng(3)
    x = rng.integers(0, 256, BLOCK, dtype=np.uint8)
    base = o.block_hash(x, 0)
    y = x.copy()
    for bit in range(BLOCK * 8):
        y[bit >> 3] ^= np.uint8(1 << (bit & 7))
        assert o.block_hash(y, 0) != base, f"flip of bit {bit} undetected"
        y[bit >> 3] ^= np.uint8(1 << (bit & 7))


def pin_swaps_and_positions(o):
    rng = np.random.default_rng(5)
    x = rng.integers(0, 256, 3 * BLOCK, dtype=np.uint8)
    blk, _ = o.entry_hashes(x)
    w = x.view(np.uint64).copy()
    w[[3, 200]] = w[[200, 3]]
    assert o.entry_hashes(w.view(np.uint8))[0][0] != blk[0], "word swap undetected"
    y = x.copy()
    y[:BLOCK], y[BLOCK:2 * BLOCK] = x[BLOCK:2 * BLOCK].copy(), x[:BLOCK].copy()
    by, _ = o.entry_hashes(y)
    assert by[0] != blk[1] and by[1] != blk[0], "block swap undetected"
    rep = np.tile(x[:BLOCK], 2)
    br, _ = o.entry_hashes(rep)
    assert br[0] != br[1], "identical blocks at different positions must hash differently"


def pin_entry_relative_and_xor(o):
    rng = np.random.default_rng(9)
    a = rng.integers(0, 256, 3 * BLOCK + 100, dtype=np.uint8)
    b = rng.integers(0, 256, 777, dtype=np.uint8)
    blk, ten = o.hashes([b, a, a, np.zeros(0, np.uint8)])
    ba, ta = o.entry_hashes(a)
    bb, tb = o.entry_hashes(b)
    assert ten[1] == ta and ten[2] == ta and ten[0] == tb and ten[3] == 0
    assert np.array_equal(blk, np.concatenate([bb, ba, ba]))
    acc = 0
    for v in rng.permutation(ba):
        acc ^= int(v)
    assert acc == ta, "tensor hash is the XOR of its block hashes, in any order"


def pin_block_hash_at(o):
    """The by-position block hash agrees with the whole-entry one, including ragged tails."""
    rng = np.random.default_rng(19)
    for n in [1, 8, 4095, 4096, 4097, 3 * BLOCK + 123, 5 * BLOCK]:
        x = rng.integers(0, 256, n, dtype=np.uint8)
        for b in range(-(-n // BLOCK)):
            assert o.block_hash_at(x[BLOCK * b: BLOCK * (b + 1)].copy(), n, b) == o.block_hash(x, b)
        assert o.block_hash(x, -(-n // BLOCK)) == 0


def pin_layout(o):
    rng = np.random.default_rng(13)
    for _ in range(50):
        n = rng.integers(0, 20000, rng.integers(0, 30)).astype(np.uint64)
        off, base, ib, nb = o.layout(n)
        slots = [(-(-int(v) // BLOCK)) * BLOCK for v in n]
        assert ib == sum(slots) and nb == sum(s // BLOCK for s in slots)
        assert [int(v) for v in off] == [sum(slots[:i]) for i in range(len(n))]
        assert np.array_equal(off, base * np.uint64(BLOCK))
    # tiny transformer set: 21 tensors; norms are 512 B, matrices whole 4 KiB multiples
    sizes = [2 * 4096 * 256] + 2 * ([512] + [2 * 256 * 256] * 4 + [512] + [2 * 1024 * 256] * 3) + [512, 2 * 4096 * 256]
    _, _, ib, nb = o.layout(sizes)
    assert sum(sizes) == 8_391_168 and ib == 8_409_088 and nb == 2053


def pin_roundtrip(o):
    for seed in range(200):
        rng = np.random.default_rng(1000 + seed)
        k = int(rng.integers(0, 12))
        sizes = [int(v) for v in rng.integers(0, 10_001, k)]
        if k and seed % 3 == 0:
            sizes[int(rng.integers(0, k))] = 0
        ents = [rng.integers(0, 256, s, dtype=np.uint8) for s in sizes]
        img = o.pack(ents)
        off, _, ib, _ = o.layout(sizes)
        assert img.nbytes == ib
        for e, s, a in zip(ents, sizes, off):
            a = int(a)
            slot = (-(-s // BLOCK)) * BLOCK
            assert np.array_equal(img[a:a + s], e)
            assert not img[a + s:a + slot].any(), "pad bytes must be zero"
        guard = 64
        bufs = [np.full(s + 2 * guard, 0xA5, np.uint8) for s in sizes]
        o.unpack_into(img, [b[guard:guard + s] for b, s in zip(bufs, sizes)])
        for b, e, s in zip(bufs, ents, sizes):
            assert np.array_equal(b[guard:guard + s], e)
            assert (b[:guard] == 0xA5).all() and (b[guard + s:] == 0xA5).all(), "write outside entry"


def pin_verify(o):
    rng = np.random.default_rng(17)
    sizes = [5 * BLOCK, 100, 0, 3 * BLOCK + 9, BLOCK]
    ents = [rng.integers(0, 256, s, dtype=np.uint8) for s in sizes]
    exp, _ = o.hashes(ents)
    cnt, lst = o.verify(ents, exp)
    assert cnt == 0 and lst.size == 0
    bad = [e.copy() for e in ents]
    # global blocks: entry0 -> 0..4, entry1 -> 5, entry3 -> 6..9, entry4 -> 10
    for ent, byte in [(0, 2 * BLOCK + 17), (3, 3 * BLOCK + 8), (1, 99), (4, 0)]:
        bad[ent][byte] ^= 0x10
    cnt, lst = o.verify(bad, exp)
    assert cnt == 4 and [int(v) for v in lst] == [2, 5, 9, 10]
    cnt, lst = o.verify(bad, exp, cap=2)
    assert cnt == 4 and [int(v) for v in lst] == [2, 5]


def _recipe(r: str) -> np.ndarray:
    p = r.split(":")
    if p[0] == "zeros":
        return np.zeros(int(p[1]), np.uint8)
    if p[0] == "ramp":
        x = (np.arange(int(p[1])) & 0xFF).astype(np.uint8)
        if len(p) > 2 and p[2] == "flipbit":
            bit = int(p[3])
            x[bit >> 3] ^= np.uint8(1 << (bit & 7))
        if len(p) > 2 and p[2] == "swapwords":
            w = x.view(np.uint64).copy()
            a, b = int(p[3]), int(p[4])
            w[[a, b]] = w[[b, a]]
            x = w.view(np.uint8)
        return x
    if p[0] == "seq":
        return np.arange(1, int(p[1]) + 1, dtype=np.uint8)
    if p[0] == "bf16words":
        return np.array([int(v, 16) for v in p[1].split(",")], dtype="<u2").view(np.uint8)
    if p[0] == "affine":
        n, a, c = int(p[1]), int(p[2]), int(p[3])
        return ((a * np.arange(n) + c) & 0xFF).astype(np.uint8)
    raise ValueError(r)


def golden_vectors():
    out = []
    with open(os.path.join(GOLDEN, "hash_vectors.txt")) as f:
        for line in f:
            if line.strip() and not line.startswith("#"):
                r, b, t = [s.strip() for s in line.split("|")]
                out.append((r, [int(v, 16) for v in b.split(",")], int(t, 16)))
    return out


def pin_golden_vectors(o):
    for r, blks, ten in golden_vectors():
        b, t = o.entry_hashes(_recipe(r))
        assert [int(v) for v in b] == blks and t == ten, f"golden vector {r}"


ALL_PINS = [
    pin_splitmix_published,
    pin_fmix_bijective,
    pin_word_order_and_index,
    pin_block_membership,
    pin_zero_extension,
    pin_zero_blocks_closed_form,
    pin_swaps_and_positions,
    pin_entry_relative_and_xor,
    pin_block_hash_at,
    pin_layout,
    pin_roundtrip,
    pin_verify,
    pin_golden_vectors,
    pin_bitflip_exhaustive,
]
