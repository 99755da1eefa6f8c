"""CPU oracle of the image/restore/verify path -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the benchmark's CPU-baseline
leg may import this package.  It wraps ``liboracle.so`` (plain C, see
``oracle.h`` for the definitions) with numpy-facing helpers; it shares nothing
with the GPU library.

``Oracle(path)`` binds one build of the C oracle; the module-level functions
use the default build next to this file.  The tests also bind deliberately
broken builds of the same source to show that the pins catch such mistakes.
"""
from __future__ import annotations

import ctypes
import os
from typing import Sequence

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
SOURCE = os.path.join(HERE, "oracle.c")
DEFAULT_LIB = os.path.join(HERE, "liboracle.so")
U64 = ctypes.c_uint64
VP = ctypes.c_void_p

BLOCK = 4096


def _u8(a) -> np.ndarray:
    a = np.ascontiguousarray(a)
    return a.view(np.uint8).reshape(-1)


def _ptrs(arrays):
    return (VP * max(len(arrays), 1))(*[a.ctypes.data for a in arrays])


def _sizes(arrays):
    return np.array([a.nbytes for a in arrays], dtype=np.uint64)


class Oracle:
    def __init__(self, path: str = DEFAULT_LIB):
        if not os.path.exists(path):
            raise RuntimeError(f"{path} is not built; run __graft_entry__.build()")
        lib = ctypes.CDLL(path)
        lib.oracle_fmix.argtypes = [U64]
        lib.oracle_fmix.restype = U64
        lib.oracle_word.argtypes = [VP, U64, U64]
        lib.oracle_word.restype = U64
        lib.oracle_block_hash.argtypes = [VP, U64, U64]
        lib.oracle_block_hash.restype = U64
        lib.oracle_block_hash_at.argtypes = [VP, U64, U64]
        lib.oracle_block_hash_at.restype = U64
        lib.oracle_entry_hashes.argtypes = [VP, U64, VP]
        lib.oracle_entry_hashes.restype = U64
        lib.oracle_layout.argtypes = [VP, U64, VP, VP, VP, VP]
        lib.oracle_pack.argtypes = [VP, VP, U64, VP]
        lib.oracle_unpack.argtypes = [VP, VP, VP, U64]
        lib.oracle_hash.argtypes = [VP, VP, U64, VP, VP]
        lib.oracle_verify.argtypes = [VP, VP, U64, VP, VP, U64]
        lib.oracle_verify.restype = U64
        self.lib = lib
        self.path = path

    def fmix(self, z: int) -> int:
        return int(self.lib.oracle_fmix(z))

    def word(self, x, j: int) -> int:
        x = _u8(x)
        return int(self.lib.oracle_word(x.ctypes.data, x.nbytes, j))

    def block_hash(self, x, b: int) -> int:
        x = _u8(x)
        return int(self.lib.oracle_block_hash(x.ctypes.data, x.nbytes, b))

    def block_hash_at(self, blk, n: int, b: int) -> int:
        """Hash of block b of an n-byte entry, given only that block's bytes."""
        blk = _u8(blk)
        if blk.nbytes < min(BLOCK, max(n - BLOCK * b, 0)):
            raise ValueError("block buffer shorter than the block")
        return int(self.lib.oracle_block_hash_at(blk.ctypes.data, n, b))

    def entry_hashes(self, x):
        """(block hashes [ceil(n/4096)] uint64, tensor hash int) of one entry."""
        x = _u8(x)
        nb = -(-x.nbytes // BLOCK)
        blk = np.zeros(max(nb, 1), dtype=np.uint64)
        t = self.lib.oracle_entry_hashes(x.ctypes.data, x.nbytes, blk.ctypes.data)
        return blk[:nb], int(t)

    def layout(self, nbytes: Sequence[int]):
        """(img_off, blk_base, image_bytes, num_blocks) for entry sizes ``nbytes``."""
        n = np.ascontiguousarray(nbytes, dtype=np.uint64)
        k = len(n)
        off = np.zeros(max(k, 1), dtype=np.uint64)
        base = np.zeros(max(k, 1), dtype=np.uint64)
        ib, nb = U64(), U64()
        self.lib.oracle_layout(n.ctypes.data, k, off.ctypes.data, base.ctypes.data,
                               ctypes.byref(ib), ctypes.byref(nb))
        return off[:k], base[:k], int(ib.value), int(nb.value)

    def pack(self, entries) -> np.ndarray:
        arrs = [_u8(e) for e in entries]
        sizes = _sizes(arrs)
        _, _, ib, _ = self.layout(sizes)
        image = np.empty(ib, dtype=np.uint8)
        self.lib.oracle_pack(_ptrs(arrs), sizes.ctypes.data, len(arrs), image.ctypes.data)
        return image

    def unpack_into(self, image, dsts) -> None:
        """Write each entry's bytes from ``image`` into the writable contiguous arrays ``dsts``."""
        image = _u8(image)
        arrs = [d.view(np.uint8).reshape(-1) for d in dsts]
        sizes = _sizes(arrs)
        _, _, ib, _ = self.layout(sizes)
        if image.nbytes < ib:
            raise ValueError("image smaller than the layout")
        self.lib.oracle_unpack(image.ctypes.data, _ptrs(arrs), sizes.ctypes.data, len(arrs))

    def unpack(self, image, nbytes: Sequence[int]):
        dsts = [np.empty(int(n), dtype=np.uint8) for n in nbytes]
        self.unpack_into(image, dsts)
        return dsts

    def hashes(self, entries):
        """(block hashes [num_blocks] uint64, tensor hashes [n] uint64)."""
        arrs = [_u8(e) for e in entries]
        sizes = _sizes(arrs)
        _, _, _, nb = self.layout(sizes)
        blk = np.zeros(max(nb, 1), dtype=np.uint64)
        ten = np.zeros(max(len(arrs), 1), dtype=np.uint64)
        self.lib.oracle_hash(_ptrs(arrs), sizes.ctypes.data, len(arrs), blk.ctypes.data, ten.ctypes.data)
        return blk[:nb], ten[: len(arrs)]

    def verify(self, entries, expected, cap: int | None = None):
        """(mismatch count, ascending mismatch indices [min(count, cap)])."""
        arrs = [_u8(e) for e in entries]
        sizes = _sizes(arrs)
        _, _, _, nb = self.layout(sizes)
        exp = np.ascontiguousarray(expected, dtype=np.uint64)
        if exp.size < nb:
            raise ValueError("expected hash array shorter than the block count")
        cap = nb if cap is None else cap
        lst = np.zeros(max(cap, 1), dtype=np.uint64)
        cnt = self.lib.oracle_verify(_ptrs(arrs), sizes.ctypes.data, len(arrs), exp.ctypes.data,
                                     lst.ctypes.data, cap)
        return int(cnt), lst[: min(int(cnt), cap)]


_default: Oracle | None = None


def default() -> Oracle:
    global _default
    if _default is None:
        _default = Oracle()
    return _default


def fmix(z):
    return default().fmix(z)


def word(x, j):
    return default().word(x, j)


def block_hash(x, b):
    return default().block_hash(x, b)


def block_hash_at(blk, n, b):
    return default().block_hash_at(blk, n, b)


def entry_hashes(x):
    return default().entry_hashes(x)


def layout(nbytes):
    return default().layout(nbytes)


def pack(entries):
    return default().pack(entries)


def unpack_into(image, dsts):
    return default().unpack_into(image, dsts)


def unpack(image, nbytes):
    return default().unpack(image, nbytes)


def hashes(entries):
    return default().hashes(entries)


def verify(entries, expected, cap=None):
    return default().verify(entries, expected, cap)


def build(out_path: str = DEFAULT_LIB, source: str = SOURCE, defines=()) -> str:
    """Compile the C oracle with gcc (plain -O2) into ``out_path``."""
    import subprocess

    cmd = ["gcc", "-O2", "-Wall", "-Wextra", "-fPIC", "-shared", "-I", HERE, source, "-o", out_path]
    cmd[1:1] = [f"-D{d}" for d in defines]
    subprocess.run(cmd, check=True)
    return out_path
