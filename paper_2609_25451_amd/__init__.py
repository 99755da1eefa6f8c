"""Python binding of libgms (include/gms.h): argument marshalling only.

Every step of snapshot / restore / verify runs in the HIP library
``libgms.so`` built next to this file; importing this package fails loudly if
it is missing.  Pointers may be given as integers or as objects with a
``data_ptr()`` method (torch tensors); streams as integers or objects with a
``cuda_stream`` attribute (torch streams), defaulting to torch's current
stream when torch is importable.
"""
from __future__ import annotations

import ctypes
import os
import re

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libgms.so")
HEADER_PATH = os.path.join(os.path.dirname(_HERE), "include", "gms.h")

try:  # load torch's HIP runtime first so that the library and torch share one runtime
    import torch  # noqa: F401
except ImportError:  # plain C-pointer use without torch
    torch = None

if not os.path.exists(LIB_PATH):
    raise ImportError(f"{LIB_PATH} is not built; run __graft_entry__.build() (no fallback exists)")

_lib = ctypes.CDLL(LIB_PATH)

U64 = ctypes.c_uint64
VP = ctypes.c_void_p
INT = ctypes.c_int

GMS_OK = 0
GMS_ERR_INVALID = -1
GMS_ERR_OVERLAP = -2
GMS_ERR_SIZE = -3
GMS_ERR_HIP = -4
GMS_ERR_NOMEM = -5
GMS_ERR_STATE = -6
GMS_ERR_IO = -7
GMS_ERR_INTEGRITY = -8
STORE_EMPTY = 0
STORE_RW = 1
STORE_COMMITTED = 2
STORE_RO = 3
STORE_STATES = {STORE_EMPTY: "EMPTY", STORE_RW: "RW", STORE_COMMITTED: "COMMITTED", STORE_RO: "RO"}
CONNECT_VERIFY = 1
FILE_DIRECT = 1
FILE_SYNC = 2
MEM_DEVICE = 0
MEM_HOST_PINNED = 1
GROUP_SHIFTED = 1  # gms_group_flags
GROUP_STRIPED = 2
HOST_ONLY = -1
BLOCK_BYTES = 4096
DEFAULT_SLICE_BYTES = 256 << 20  # GMS_DEFAULT_SLICE_BYTES
DEFAULT_SLOTS = 2  # GMS_DEFAULT_SLOTS


class GmsEntry(ctypes.Structure):
    _fields_ = [("addr", U64), ("nbytes", U64)]


def _sig(name, res, args):
    f = getattr(_lib, name)
    f.restype = res
    f.argtypes = args
    return f


_create = _sig("gms_manifest_create", INT, [ctypes.POINTER(GmsEntry), U64, INT, U64, ctypes.POINTER(VP)])
_destroy = _sig("gms_manifest_destroy", None, [VP])
_num_entries = _sig("gms_num_entries", U64, [VP])
_payload = _sig("gms_payload_bytes", U64, [VP])
_image_bytes = _sig("gms_image_bytes", U64, [VP])
_num_blocks = _sig("gms_num_blocks", U64, [VP])
_num_chunks = _sig("gms_num_chunks", U64, [VP])
_num_groups = _sig("gms_num_launch_groups", U64, [VP])
_launch_group = _sig("gms_launch_group", INT, [VP, U64, VP, VP, VP])
_device = _sig("gms_manifest_device", INT, [VP])
_layout = _sig("gms_layout", INT, [VP, VP, VP])
_set_staging = _sig("gms_manifest_set_staging", INT, [VP, U64, ctypes.c_uint32])
_snapshot = _sig("gms_snapshot", INT, [VP, VP, U64, INT, VP, VP, VP])
_restore = _sig("gms_restore", INT, [VP, VP, U64, INT, VP, VP, VP, VP, VP, U64, VP])
_verify = _sig("gms_verify", INT, [VP, VP, VP, VP, VP, VP, U64, VP])
_restore_file = _sig("gms_restore_from_file", INT,
                     [VP, ctypes.c_char_p, U64, ctypes.c_uint32, ctypes.c_uint32, VP, VP, VP, VP, VP, U64, VP])
_snapshot_file = _sig("gms_snapshot_to_file", INT, [VP, ctypes.c_char_p, ctypes.c_uint32, ctypes.c_uint32, VP, VP, VP])
_restore_host = _sig("gms_restore_from_host", INT, [VP, VP, U64, ctypes.c_uint32, VP, VP, VP, VP, VP, U64, VP])
_snapshot_host = _sig("gms_snapshot_to_host", INT, [VP, VP, U64, ctypes.c_uint32, VP, VP, VP])
_restore_noalloc = _sig("gms_restore_pinned_noalloc", INT, [VP, VP, U64, U64, VP, VP, VP, VP, VP, U64, VP])
_pool_create = _sig("gms_pool_create", INT, [INT, U64, U64, ctypes.POINTER(VP)])
_pool_destroy = _sig("gms_pool_destroy", None, [VP])
_pool_alloc = _sig("gms_pool_alloc", INT, [VP, U64, U64, ctypes.POINTER(U64)])
_pool_free = _sig("gms_pool_free", INT, [VP, U64])
_pool_release = _sig("gms_pool_release", INT, [VP, U64, U64])
_pool_remap = _sig("gms_pool_remap", INT, [VP, U64, U64])
_pool_set_access = _sig("gms_pool_set_access", INT, [VP, U64, U64, INT])
_pool_info = _sig("gms_pool_info", INT, [VP, VP, VP, VP, VP, VP])
_pool_mapping_of = _sig("gms_pool_mapping_of", INT, [VP, U64, VP, VP, VP])
_store_create = _sig("gms_store_create", INT, [INT, U64, U64, ctypes.POINTER(VP)])
_store_destroy = _sig("gms_store_destroy", None, [VP])
_store_state = _sig("gms_store_state", INT, [VP, VP, VP, VP])
_store_pool = _sig("gms_store_pool", VP, [VP])
_store_connect_rw = _sig("gms_store_connect_rw", INT, [VP, ctypes.POINTER(U64)])
_store_alloc = _sig("gms_store_alloc", INT, [VP, U64, U64, U64, ctypes.POINTER(U64)])
_store_free = _sig("gms_store_free", INT, [VP, U64, U64])
_store_commit = _sig("gms_store_commit", INT, [VP, U64, ctypes.POINTER(GmsEntry), U64, VP, ctypes.POINTER(U64), VP])
_store_abort = _sig("gms_store_abort", INT, [VP, U64])
_store_connect_ro = _sig("gms_store_connect_ro", INT, [VP, ctypes.c_uint32, ctypes.POINTER(U64), ctypes.POINTER(U64), VP])
_store_verify = _sig("gms_store_verify", INT, [VP, ctypes.POINTER(U64), VP, U64, VP])
_store_disconnect = _sig("gms_store_disconnect", INT, [VP, U64])
_store_layout = _sig("gms_store_layout", VP, [VP])
_store_block_hashes = _sig("gms_store_block_hashes", VP, [VP])
_owner_create = _sig("gms_owner_create", INT, [ctypes.c_char_p, INT, ctypes.POINTER(VP)])
_owner_run = _sig("gms_owner_run", INT, [VP])
_owner_stop = _sig("gms_owner_stop", None, [VP])
_owner_status = _sig("gms_owner_status", INT, [VP, VP, VP, VP, VP])
_owner_query = _sig("gms_owner_query", INT, [ctypes.c_char_p, VP, VP, VP, VP])
_owner_destroy = _sig("gms_owner_destroy", None, [VP])
_client_connect = _sig("gms_client_connect", INT,
                       [ctypes.c_char_p, INT, ctypes.c_uint32, VP, ctypes.POINTER(VP), ctypes.POINTER(U64)])
_client_lease = _sig("gms_client_lease", INT, [VP, VP, VP])
_client_alloc = _sig("gms_client_alloc", INT, [VP, U64, U64, ctypes.POINTER(U64)])
_client_free = _sig("gms_client_free", INT, [VP, U64])
_client_commit = _sig("gms_client_commit", INT, [VP, ctypes.POINTER(GmsEntry), U64, VP, ctypes.POINTER(U64), VP])
_client_abort = _sig("gms_client_abort", INT, [VP])
_client_layout = _sig("gms_client_layout", INT, [VP, VP, U64, ctypes.POINTER(U64)])
_client_manifest = _sig("gms_client_manifest", VP, [VP])
_client_manifest_create = _sig("gms_client_manifest_create", INT, [VP, ctypes.POINTER(GmsEntry), U64, U64,
                                                                   ctypes.POINTER(VP)])
_client_block_hashes = _sig("gms_client_block_hashes", VP, [VP])
_client_verify = _sig("gms_client_verify", INT, [VP, ctypes.POINTER(U64), VP, U64, VP])
_client_disconnect = _sig("gms_client_disconnect", INT, [VP])
_status_str = _sig("gms_status_str", ctypes.c_char_p, [INT])
_last_error = _sig("gms_last_error", ctypes.c_char_p, [])
_abi = _sig("gms_abi_version", INT, [])


class GmsError(RuntimeError):
    def __init__(self, status: int, call: str, mismatches: int = 0):
        self.status = status
        self.mismatches = mismatches
        msg = _last_error().decode(errors="replace")
        super().__init__(f"{call}: {_status_str(status).decode()} ({status}): {msg}")


def _check(rc: int, call: str) -> None:
    if rc != GMS_OK:
        raise GmsError(rc, call)


def _dense(t):
    """A tensor stands for the bytes [data_ptr, data_ptr + numel * element_size): only a
    contiguous one does."""
    if hasattr(t, "is_contiguous") and not t.is_contiguous():
        raise ValueError("a non-contiguous tensor does not describe one byte range; pass .contiguous()")
    return t


def _ptr(x) -> int | None:
    if x is None:
        return None
    if hasattr(x, "data_ptr"):
        return int(_dense(x).data_ptr())
    if hasattr(x, "__array_interface__"):  # numpy arrays
        if not x.flags["C_CONTIGUOUS"]:
            raise ValueError("a non-contiguous array does not describe one byte range; pass a contiguous copy")
        return int(x.ctypes.data)
    return int(x)


def _buf(x, need: int, what: str, words: bool = False) -> int | None:
    """Pointer of an argument the library reads or writes ``need`` bytes of.  Tensors and
    arrays are checked against their own size (the C side can only check the enclosing
    allocation, which for a caching allocator is a whole segment); ``words`` arguments
    must hold 64-bit integers.  Raw integer addresses pass unchecked."""
    if x is None:
        return None
    if hasattr(x, "data_ptr"):
        _dense(x)
        es, nb = int(x.element_size()), int(x.numel() * x.element_size())
        wordy = es == 8 and not x.is_floating_point() and not x.is_complex()
        kind = str(x.dtype)
    elif hasattr(x, "__array_interface__"):
        if not x.flags["C_CONTIGUOUS"]:
            raise ValueError(f"{what}: a non-contiguous array does not describe one byte range")
        es, nb = int(x.dtype.itemsize), int(x.nbytes)
        wordy = es == 8 and x.dtype.kind in "iu"
        kind = str(x.dtype)
    else:
        return int(x)
    if words and not wordy:
        raise ValueError(f"{what}: needs 64-bit integer elements, got {kind}")
    if nb < need:
        raise ValueError(f"{what}: holds {nb} bytes, the call needs {need}")
    return _ptr(x)


def _image(x, image_bytes) -> tuple[int | None, int]:
    """(pointer, byte count) of an image argument; a count given for a tensor or an array
    must fit inside it."""
    nb = _nbytes(x, image_bytes)
    if hasattr(x, "data_ptr") or hasattr(x, "__array_interface__"):
        have = _nbytes(x, None)
        if nb > have:
            raise ValueError(f"image: image_bytes {nb} exceeds the buffer's {have} bytes")
    return _ptr(x), nb


def _hash_args(m, expected, blk_hash, ten_hash, mismatch_count, mismatch_list, mismatch_cap):
    nb, ne = m.num_blocks, m.num_entries
    return (_buf(expected, nb * 8, "expected", True), _buf(blk_hash, nb * 8, "blk_hash", True),
            _buf(ten_hash, ne * 8, "ten_hash", True), _buf(mismatch_count, 8, "mismatch_count", True),
            _buf(mismatch_list, min(int(mismatch_cap), nb) * 8, "mismatch_list", True))


def _nbytes(x, nbytes):
    if nbytes is not None:
        return int(nbytes)
    if hasattr(x, "nbytes"):
        return int(x.nbytes)
    if hasattr(x, "numel"):
        return int(x.numel() * x.element_size())
    raise ValueError("image_bytes is needed for a raw pointer")


def _stream(stream) -> int | None:
    if stream is None:
        if torch is not None and torch.cuda.is_available():
            return int(torch.cuda.current_stream().cuda_stream) or None
        return None
    return int(getattr(stream, "cuda_stream", stream)) or None


def abi_version() -> int:
    return int(_abi())


def exported_symbols_declared() -> list[str]:
    """Names of the functions include/gms.h declares."""
    with open(HEADER_PATH) as f:
        text = f.read()
    return sorted(set(re.findall(r"\b(gms_[a-z_0-9]+)\s*\(", text)))


def _ranges(entries):
    out = []
    for e in entries:
        if hasattr(e, "data_ptr"):
            out.append((int(_dense(e).data_ptr()), int(e.numel() * e.element_size())))
        else:
            out.append((int(e[0]), int(e[1])))
    return out


def _entry_array(ranges):
    return (GmsEntry * max(len(ranges), 1))(*[GmsEntry(a, b) for a, b in ranges])


class Manifest:
    """A manifest over device ranges ``entries`` = [(addr, nbytes)] or tensors."""

    def __init__(self, entries, device: int = 0, chunk_bytes: int = 0):
        ranges = _ranges(entries)
        n = len(ranges)
        h = VP()
        _check(_create(_entry_array(ranges), n, device, chunk_bytes, ctypes.byref(h)), "gms_manifest_create")
        self._h = h
        self._owned = True
        self.sizes = [b for _, b in ranges]

    @classmethod
    def _borrow(cls, handle: int, owner):
        """A view of a manifest owned by the library (a store's committed layout)."""
        m = cls.__new__(cls)
        m._h = VP(handle)
        m._owned = False
        m._owner = owner
        m.sizes = None
        return m

    @property
    def handle(self) -> int:
        return self._h.value

    def close(self) -> None:
        if getattr(self, "_h", None) is not None and self._h.value:
            if getattr(self, "_owned", True):
                _destroy(self._h)
            self._h = VP()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()

    @property
    def num_entries(self) -> int:
        return int(_num_entries(self._h))

    @property
    def payload_bytes(self) -> int:
        return int(_payload(self._h))

    @property
    def image_bytes(self) -> int:
        return int(_image_bytes(self._h))

    @property
    def num_blocks(self) -> int:
        return int(_num_blocks(self._h))

    @property
    def num_chunks(self) -> int:
        return int(_num_chunks(self._h))

    @property
    def num_launch_groups(self) -> int:
        return int(_num_groups(self._h))

    def launch_groups(self) -> list:
        """Per launch group: {"chunks", "unit_shift", "shifted", "striped"}."""
        out = []
        for g in range(self.num_launch_groups):
            n, sh, fl = U64(), ctypes.c_uint32(), ctypes.c_uint32()
            _check(_launch_group(self._h, g, ctypes.byref(n), ctypes.byref(sh), ctypes.byref(fl)), "gms_launch_group")
            out.append({"chunks": int(n.value), "unit_shift": int(sh.value), "shifted": bool(fl.value & GROUP_SHIFTED),
                        "striped": bool(fl.value & GROUP_STRIPED)})
        return out

    @property
    def device(self) -> int:
        return int(_device(self._h))

    def layout(self):
        """(img_off, blk_base) as lists of ints."""
        n = self.num_entries
        off = (U64 * max(n, 1))()
        base = (U64 * max(n, 1))()
        _check(_layout(self._h, off, base), "gms_layout")
        return list(off[:n]), list(base[:n])

    def set_staging(self, slice_bytes: int, slots: int) -> None:
        _check(_set_staging(self._h, slice_bytes, slots), "gms_manifest_set_staging")


def snapshot(m: Manifest, image, image_bytes: int | None = None, kind: int = MEM_DEVICE, blk_hash=None,
             ten_hash=None, stream=None) -> None:
    img, nb = _image(image, image_bytes)
    _check(_snapshot(m._h, img, nb, kind, _buf(blk_hash, m.num_blocks * 8, "blk_hash", True),
                     _buf(ten_hash, m.num_entries * 8, "ten_hash", True), _stream(stream)), "gms_snapshot")


def restore(m: Manifest, image, image_bytes: int | None = None, kind: int = MEM_DEVICE, expected=None,
            blk_hash=None, ten_hash=None, mismatch_count=None, mismatch_list=None, mismatch_cap: int = 0,
            stream=None) -> None:
    img, nb = _image(image, image_bytes)
    h = _hash_args(m, expected, blk_hash, ten_hash, mismatch_count, mismatch_list, mismatch_cap)
    _check(_restore(m._h, img, nb, kind, *h, mismatch_cap, _stream(stream)), "gms_restore")


def verify(m: Manifest, expected=None, blk_hash=None, ten_hash=None, mismatch_count=None, mismatch_list=None,
           mismatch_cap: int = 0, stream=None) -> None:
    h = _hash_args(m, expected, blk_hash, ten_hash, mismatch_count, mismatch_list, mismatch_cap)
    _check(_verify(m._h, *h, mismatch_cap, _stream(stream)), "gms_verify")


NOALLOC_STAGING_BYTES = 64 << 20  # GMS_NOALLOC_STAGING_BYTES


def restore_pinned_noalloc(m: Manifest, image, image_bytes: int | None = None, staging_bytes: int = 0,
                           expected=None, blk_hash=None, ten_hash=None, mismatch_count=None, mismatch_list=None,
                           mismatch_cap: int = 0, stream=None) -> None:
    """gms_restore from a pinned host image with no allocation (a fixed staging area)."""
    img, nb = _image(image, image_bytes)
    h = _hash_args(m, expected, blk_hash, ten_hash, mismatch_count, mismatch_list, mismatch_cap)
    _check(_restore_noalloc(m._h, img, nb, staging_bytes, *h, mismatch_cap, _stream(stream)),
           "gms_restore_pinned_noalloc")


def restore_from_file(m: Manifest, path, file_offset: int = 0, flags: int = FILE_DIRECT, io_threads: int = 0,
                      expected=None, blk_hash=None, ten_hash=None, mismatch_count=None, mismatch_list=None,
                      mismatch_cap: int = 0, stream=None) -> None:
    h = _hash_args(m, expected, blk_hash, ten_hash, mismatch_count, mismatch_list, mismatch_cap)
    _check(_restore_file(m._h, os.fsencode(path), file_offset, flags, io_threads, *h, mismatch_cap,
                         _stream(stream)), "gms_restore_from_file")


def snapshot_to_file(m: Manifest, path, flags: int = 0, io_threads: int = 0, blk_hash=None, ten_hash=None,
                     stream=None) -> None:
    _check(_snapshot_file(m._h, os.fsencode(path), flags, io_threads,
                          _buf(blk_hash, m.num_blocks * 8, "blk_hash", True),
                          _buf(ten_hash, m.num_entries * 8, "ten_hash", True), _stream(stream)),
           "gms_snapshot_to_file")


def restore_from_host(m: Manifest, image, image_bytes: int | None = None, threads: int = 0, expected=None,
                      blk_hash=None, ten_hash=None, mismatch_count=None, mismatch_list=None, mismatch_cap: int = 0,
                      stream=None) -> None:
    """Restore from an image in ordinary host memory (a numpy array, a CPU tensor or an
    address): returns once `image` may be reused; device work completes on `stream`."""
    img, nb = _image(image, image_bytes)
    h = _hash_args(m, expected, blk_hash, ten_hash, mismatch_count, mismatch_list, mismatch_cap)
    _check(_restore_host(m._h, img, nb, threads, *h, mismatch_cap, _stream(stream)), "gms_restore_from_host")


def snapshot_to_host(m: Manifest, image, image_bytes: int | None = None, threads: int = 0, blk_hash=None,
                     ten_hash=None, stream=None) -> None:
    """Snapshot into ordinary host memory; synchronous."""
    img, nb = _image(image, image_bytes)
    _check(_snapshot_host(m._h, img, nb, threads, _buf(blk_hash, m.num_blocks * 8, "blk_hash", True),
                          _buf(ten_hash, m.num_entries * 8, "ten_hash", True), _stream(stream)),
           "gms_snapshot_to_host")


class Pool:
    """Device memory pool over HIP virtual memory (see gms_pool_* in include/gms.h)."""

    def __init__(self, va_bytes: int, slab_bytes: int = 0, device: int = 0):
        h = VP()
        _check(_pool_create(device, va_bytes, slab_bytes, ctypes.byref(h)), "gms_pool_create")
        self._h = h
        self.device = device

    def close(self) -> None:
        if getattr(self, "_h", None) is not None and self._h.value:
            _pool_destroy(self._h)
            self._h = VP()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def alloc(self, nbytes: int, align: int = 0) -> int:
        out = U64()
        _check(_pool_alloc(self._h, nbytes, align, ctypes.byref(out)), "gms_pool_alloc")
        return int(out.value)

    def free(self, addr: int) -> None:
        _check(_pool_free(self._h, addr), "gms_pool_free")

    def release(self, addr: int, nbytes: int) -> None:
        _check(_pool_release(self._h, addr, nbytes), "gms_pool_release")

    def remap(self, addr: int, nbytes: int) -> None:
        _check(_pool_remap(self._h, addr, nbytes), "gms_pool_remap")

    def set_access(self, addr: int, nbytes: int, read_only: bool) -> None:
        _check(_pool_set_access(self._h, addr, nbytes, 1 if read_only else 0), "gms_pool_set_access")

    def info(self) -> dict:
        v = [U64() for _ in range(5)]
        _check(_pool_info(self._h, *[ctypes.byref(x) for x in v]), "gms_pool_info")
        return dict(zip(["base", "reserved", "mapped_bytes", "mappings", "granularity"], [int(x.value) for x in v]))

    def mapping_of(self, addr: int):
        a, b, m = U64(), U64(), INT()
        _check(_pool_mapping_of(self._h, addr, ctypes.byref(a), ctypes.byref(b), ctypes.byref(m)),
               "gms_pool_mapping_of")
        return int(a.value), int(b.value), bool(m.value)


class Store:
    """Model-state store with the GMS lease protocol (see gms_store_* in include/gms.h).

    ``device=HOST_ONLY`` gives a protocol-only store without memory.
    """

    def __init__(self, va_bytes: int = 0, slab_bytes: int = 0, device: int = 0):
        h = VP()
        _check(_store_create(device, va_bytes, slab_bytes, ctypes.byref(h)), "gms_store_create")
        self._h = h
        self.device = device

    def close(self) -> None:
        if getattr(self, "_h", None) is not None and self._h.value:
            _store_destroy(self._h)
            self._h = VP()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def state(self):
        """(state name, reader count, invalid)."""
        st, rd, inv = INT(), ctypes.c_uint32(), INT()
        _check(_store_state(self._h, ctypes.byref(st), ctypes.byref(rd), ctypes.byref(inv)), "gms_store_state")
        return STORE_STATES[st.value], int(rd.value), bool(inv.value)

    def pool_info(self) -> dict:
        p = _store_pool(self._h)
        if not p:
            return {}
        v = [U64() for _ in range(5)]
        _check(_pool_info(p, *[ctypes.byref(x) for x in v]), "gms_pool_info")
        return dict(zip(["base", "reserved", "mapped_bytes", "mappings", "granularity"], [int(x.value) for x in v]))

    @property
    def pool_handle(self) -> int:
        return int(_store_pool(self._h) or 0)

    def connect_rw(self) -> "WriteLease":
        lease = U64()
        _check(_store_connect_rw(self._h, ctypes.byref(lease)), "gms_store_connect_rw")
        return WriteLease(self, int(lease.value))

    def connect_ro(self, verify: bool = True, stream=None) -> "ReadLease":
        lease, cnt = U64(), U64()
        rc = _store_connect_ro(self._h, CONNECT_VERIFY if verify else 0, ctypes.byref(lease), ctypes.byref(cnt),
                               _stream(stream))
        if rc != GMS_OK:
            raise GmsError(rc, "gms_store_connect_ro", int(cnt.value))
        return ReadLease(self, int(lease.value))

    def verify(self, mismatch_list=None, mismatch_cap: int = 0, stream=None) -> int:
        cnt = U64()
        h = _store_layout(self._h)
        nb = int(_num_blocks(h)) if h else 0
        lst = _buf(mismatch_list, min(int(mismatch_cap), nb) * 8, "mismatch_list", True)
        _check(_store_verify(self._h, ctypes.byref(cnt), lst, mismatch_cap, _stream(stream)), "gms_store_verify")
        return int(cnt.value)

    def layout(self) -> Manifest | None:
        """The committed layout, as a manifest owned by the store: valid until the next writer
        connects or the store is closed."""
        h = _store_layout(self._h)
        return Manifest._borrow(h, self) if h else None

    def block_hashes_ptr(self) -> int:
        return int(_store_block_hashes(self._h) or 0)


class _Lease:
    def __init__(self, store: Store, lease: int):
        self.store = store
        self.id = lease
        self.open = True

    def _handle(self):
        h = getattr(self.store, "_h", None)
        if h is None or not h.value:
            raise GmsError(GMS_ERR_STATE, "lease of a closed store")
        return h

    def close(self) -> None:
        """Ends the lease (a writer's before commit discards its state); a no-op once the
        store itself is closed, which ended every lease."""
        if self.open:
            self.open = False
            h = getattr(self.store, "_h", None)
            if h is not None and h.value:
                _check(_store_disconnect(h, self.id), "gms_store_disconnect")

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()


class WriteLease(_Lease):
    """Exclusive read-write lease; leaving it without commit aborts."""

    def alloc(self, nbytes: int, align: int = 0) -> int:
        out = U64()
        _check(_store_alloc(self._handle(), self.id, nbytes, align, ctypes.byref(out)), "gms_store_alloc")
        return int(out.value)

    def free(self, addr: int) -> None:
        _check(_store_free(self._handle(), self.id, addr), "gms_store_free")

    def commit(self, entries, expected=None, stream=None) -> None:
        ranges = _ranges(entries)
        cnt = U64()
        nb = sum(-(-b // BLOCK_BYTES) for _, b in ranges)
        rc = _store_commit(self._handle(), self.id, _entry_array(ranges), len(ranges),
                           _buf(expected, nb * 8, "expected", True),
                           ctypes.byref(cnt), _stream(stream))
        if rc != GMS_OK:
            raise GmsError(rc, "gms_store_commit", int(cnt.value))
        self.open = False

    def abort(self) -> None:
        if self.open:
            self.open = False
            _check(_store_abort(self._handle(), self.id), "gms_store_abort")


class ReadLease(_Lease):
    """Read-only lease on committed state."""


LEASE_RW = 1
LEASE_RO = 2
IPC_PIECE_BYTES = 1 << 30  # GMS_IPC_PIECE_BYTES


def owner_query(socket_path) -> tuple:
    """(state name, readers, invalid, allocations) of a running owner, over its socket."""
    st, rd, inv, al = INT(), ctypes.c_uint32(), INT(), U64()
    _check(_owner_query(os.fsencode(socket_path), ctypes.byref(st), ctypes.byref(rd), ctypes.byref(inv),
                        ctypes.byref(al)), "gms_owner_query")
    return STORE_STATES[st.value], int(rd.value), bool(inv.value), int(al.value)


class Owner:
    """The GMS owner of one device's model-state allocations (see gms_owner_* in include/gms.h).
    ``run()`` serves until ``stop()``; it releases the interpreter lock while it runs."""

    def __init__(self, socket_path, device: int = 0):
        h = VP()
        _check(_owner_create(os.fsencode(socket_path), device, ctypes.byref(h)), "gms_owner_create")
        self._h = h
        self.path = os.fspath(socket_path)

    def run(self) -> None:
        _check(_owner_run(self._h), "gms_owner_run")

    def stop(self) -> None:
        if self._h.value:
            _owner_stop(self._h)

    def status(self) -> tuple:
        st, rd, inv, al = INT(), ctypes.c_uint32(), INT(), U64()
        _check(_owner_status(self._h, ctypes.byref(st), ctypes.byref(rd), ctypes.byref(inv), ctypes.byref(al)),
               "gms_owner_status")
        return STORE_STATES[st.value], int(rd.value), bool(inv.value), int(al.value)

    def close(self) -> None:
        if getattr(self, "_h", None) is not None and self._h.value:
            _owner_destroy(self._h)
            self._h = VP()


class Client:
    """A lease on an owner's model state from this process (see gms_client_* in include/gms.h)."""

    def __init__(self, socket_path, mode: int, verify: bool = False, stream=None):
        h, cnt = VP(), U64()
        rc = _client_connect(os.fsencode(socket_path), mode, CONNECT_VERIFY if verify else 0, _stream(stream),
                             ctypes.byref(h), ctypes.byref(cnt))
        if rc != GMS_OK:
            raise GmsError(rc, "gms_client_connect", int(cnt.value))
        self._h = h
        self.mode = mode

    def info(self) -> dict:
        lease, dev = U64(), INT()
        _check(_client_lease(self._h, ctypes.byref(lease), ctypes.byref(dev)), "gms_client_lease")
        return {"lease": int(lease.value), "device": int(dev.value)}

    def alloc(self, nbytes: int, align: int = 0) -> int:
        out = U64()
        _check(_client_alloc(self._h, nbytes, align, ctypes.byref(out)), "gms_client_alloc")
        return int(out.value)

    def free(self, addr: int) -> None:
        _check(_client_free(self._h, addr), "gms_client_free")

    def commit(self, entries, expected=None, stream=None) -> None:
        ranges = _ranges(entries)
        nb = sum(-(-b // BLOCK_BYTES) for _, b in ranges)
        cnt = U64()
        rc = _client_commit(self._h, _entry_array(ranges), len(ranges), _buf(expected, nb * 8, "expected", True),
                            ctypes.byref(cnt), _stream(stream))
        if rc != GMS_OK:
            raise GmsError(rc, "gms_client_commit", int(cnt.value))

    def abort(self) -> None:
        _check(_client_abort(self._h), "gms_client_abort")

    def layout(self) -> list:
        n = U64()
        _check(_client_layout(self._h, None, 0, ctypes.byref(n)), "gms_client_layout")
        arr = (GmsEntry * max(int(n.value), 1))()
        _check(_client_layout(self._h, arr, int(n.value), ctypes.byref(n)), "gms_client_layout")
        return [(int(e.addr), int(e.nbytes)) for e in arr[:int(n.value)]]

    def manifest(self) -> Manifest | None:
        """The committed layout as a manifest owned by the client (valid until disconnect)."""
        h = _client_manifest(self._h)
        return Manifest._borrow(h, self) if h else None

    def block_hashes_ptr(self) -> int:
        return int(_client_block_hashes(self._h) or 0)

    def manifest_over(self, entries, chunk_bytes: int = 0) -> Manifest:
        """A manifest (owned by the caller) over entries inside this client's allocations."""
        ranges = _ranges(entries)
        h = VP()
        _check(_client_manifest_create(self._h, _entry_array(ranges), len(ranges), chunk_bytes, ctypes.byref(h)),
               "gms_client_manifest_create")
        m = Manifest.__new__(Manifest)
        m._h = h
        m._owned = True
        m.sizes = [b for _, b in ranges]
        return m

    def verify(self, mismatch_list=None, mismatch_cap: int = 0, stream=None) -> int:
        cnt = U64()
        m = _client_manifest(self._h)
        nb = int(_num_blocks(m)) if m else 0
        lst = _buf(mismatch_list, min(int(mismatch_cap), nb) * 8, "mismatch_list", True)
        _check(_client_verify(self._h, ctypes.byref(cnt), lst, mismatch_cap, _stream(stream)), "gms_client_verify")
        return int(cnt.value)

    def close(self) -> None:
        if getattr(self, "_h", None) is not None and self._h.value:
            h, self._h = self._h, VP()
            _check(_client_disconnect(h), "gms_client_disconnect")

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()


def status_str(rc: int) -> str:
    return _status_str(rc).decode()


# raw entry points, same names as the C-ABI, for callers that manage pointers themselves
gms_manifest_create = _create
gms_manifest_destroy = _destroy
gms_snapshot = _snapshot
gms_restore = _restore
gms_verify = _verify
gms_layout = _layout
gms_restore_from_file = _restore_file
gms_restore_pinned_noalloc = _restore_noalloc
gms_pool_create = _pool_create
gms_pool_alloc = _pool_alloc
gms_snapshot_to_file = _snapshot_file
gms_restore_from_host = _restore_host
gms_snapshot_to_host = _snapshot_host
gms_manifest_set_staging = _set_staging
gms_status_str = _status_str
gms_last_error = _last_error
gms_store_create = _store_create
gms_store_destroy = _store_destroy
gms_store_state = _store_state
gms_store_connect_rw = _store_connect_rw
gms_store_connect_ro = _store_connect_ro
gms_store_commit = _store_commit
gms_store_abort = _store_abort
gms_store_disconnect = _store_disconnect
gms_store_verify = _store_verify
gms_owner_create = _owner_create
gms_owner_run = _owner_run
gms_owner_stop = _owner_stop
gms_owner_query = _owner_query
gms_client_connect = _client_connect
gms_client_commit = _client_commit
gms_client_disconnect = _client_disconnect
