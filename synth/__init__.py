"""Seeded synthetic inputs shared by the tests, the smoke check and the benchmark.

Holds the counter-based generator (Philox4x32-10, see ``philox.h``) and the
workload shapes; none of the restore/verify arithmetic lives here.  The host
generator is ``libsynth_host.so`` (gcc); the GPU generator is ``libsynth_dev.so``
(hipcc), which fills device buffers with the same bits so multi-GB inputs are
made in HBM.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

from .configs import (  # noqa: F401
    BF16,
    KVPool,
    TensorSpec,
    WEIGHT_CONFIGS,
    kv_pool,
    weight_set,
)

_HERE = os.path.dirname(os.path.abspath(__file__))
_host = None
_dev = None

U64 = ctypes.c_uint64
VP = ctypes.c_void_p


def _load_host():
    global _host
    if _host is None:
        path = os.path.join(_HERE, "libsynth_host.so")
        if not os.path.exists(path):
            raise RuntimeError(f"{path} is not built; run __graft_entry__.build()")
        lib = ctypes.CDLL(path)
        lib.synth_philox.argtypes = [VP, VP, VP]
        lib.synth_u64.argtypes = [U64, U64, U64]
        lib.synth_u64.restype = U64
        lib.synth_fill_bf16.argtypes = [VP, U64, U64, U64, U64]
        lib.synth_fill_bytes.argtypes = [VP, U64, U64, U64, U64]
        lib.synth_live_map.argtypes = [VP, ctypes.c_uint32, ctypes.c_uint32, U64, U64]
        lib.synth_live_map.restype = ctypes.c_int
        _host = lib
    return _host


def _load_dev():
    global _dev
    if _dev is None:
        import torch  # noqa: F401  (load torch's HIP runtime before the generator's)
        path = os.path.join(_HERE, "libsynth_dev.so")
        if not os.path.exists(path):
            raise RuntimeError(f"{path} is not built; run __graft_entry__.build()")
        lib = ctypes.CDLL(path)
        lib.synth_dev_fill_bf16.argtypes = [VP, U64, U64, U64, U64, VP]
        lib.synth_dev_fill_bf16.restype = ctypes.c_int
        lib.synth_dev_fill_bytes.argtypes = [VP, U64, U64, U64, U64, VP]
        lib.synth_dev_fill_bytes.restype = ctypes.c_int
        lib.synth_dev_fill_bf16_pieces.argtypes = [VP, U64, U64, VP]
        lib.synth_dev_fill_bf16_pieces.restype = ctypes.c_int
        _dev = lib
    return _dev


def philox(ctr, key):
    """Raw Philox4x32-10 of a 4-word counter under a 2-word key."""
    c = (ctypes.c_uint32 * 4)(*ctr)
    k = (ctypes.c_uint32 * 2)(*key)
    out = (ctypes.c_uint32 * 4)()
    _load_host().synth_philox(c, k, out)
    return list(out)


def u64(seed: int, stream: int, index: int) -> int:
    return int(_load_host().synth_u64(seed, stream, index))


def bf16_bits(n: int, seed: int, tensor: int, first: int = 0) -> np.ndarray:
    """bf16 bit patterns of elements first..first+n-1 of ``tensor`` under ``seed``."""
    out = np.empty(n, dtype=np.uint16)
    if n:
        _load_host().synth_fill_bf16(out.ctypes.data, n, seed, tensor, first)
    return out


def random_bytes(n: int, seed: int, stream: int, first: int = 0) -> np.ndarray:
    out = np.empty(n, dtype=np.uint8)
    if n:
        _load_host().synth_fill_bytes(out.ctypes.data, n, seed, stream, first)
    return out


def live_map(nblocks: int, nlive: int, seed: int, stream: int) -> np.ndarray:
    out = np.empty(max(nlive, 1), dtype=np.uint32)
    if _load_host().synth_live_map(out.ctypes.data, nblocks, nlive, seed, stream) != 0:
        raise ValueError("bad live-map arguments")
    return out[:nlive]


def _stream_handle(stream) -> int:
    if stream is None:
        return 0
    return int(getattr(stream, "cuda_stream", stream))


def dev_fill_bf16(ptr: int, n: int, seed: int, tensor: int, first: int = 0, stream=None) -> None:
    rc = _load_dev().synth_dev_fill_bf16(ptr, n, seed, tensor, first, _stream_handle(stream))
    if rc != 0:
        raise RuntimeError(f"synth_dev_fill_bf16 failed ({rc})")


def dev_fill_bytes(ptr: int, n: int, seed: int, stream_id: int, first: int = 0, stream=None) -> None:
    rc = _load_dev().synth_dev_fill_bytes(ptr, n, seed, stream_id, first, _stream_handle(stream))
    if rc != 0:
        raise RuntimeError(f"synth_dev_fill_bytes failed ({rc})")


PIECE_ELEMS = 1 << 20  # elements per piece of a batched fill (2 MiB of bf16)


def dev_fill_bf16_many(ranges, seed: int, stream=None) -> None:
    """Fills device ranges [(address, elements, tensor id)] (elements 0.. of each tensor)
    with one launch; returns once they are filled."""
    rows = []
    for ptr, n, tid in ranges:
        for first in range(0, int(n), PIECE_ELEMS):
            rows.append((int(ptr) + 2 * first, min(PIECE_ELEMS, int(n) - first), int(tid), first))
    if not rows:
        return
    table = np.array(rows, dtype=np.uint64)
    rc = _load_dev().synth_dev_fill_bf16_pieces(table.ctypes.data, len(rows), seed, _stream_handle(stream))
    if rc != 0:
        raise RuntimeError(f"synth_dev_fill_bf16_pieces failed ({rc})")


def dev_fill_tensors(tensors, seed: int, ids=None, stream=None) -> None:
    """Every tensor t_k gets the bf16 stream of tensor id ids[k] (default k), in one launch."""
    ids = range(len(tensors)) if ids is None else ids
    dev_fill_bf16_many([(t.data_ptr(), t.numel() * t.element_size() // 2, i) for t, i in zip(tensors, ids)],
                       seed, stream)
