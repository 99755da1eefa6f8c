"""The model-state lease protocol (paper section 3.2, Figure 4) on the CPU.

A store made without a device runs the protocol alone, through the same
C-ABI calls as a device store.  Pins: the scenarios the paper states in
words, each as a fixed call sequence with its expected states; then seeded
random walks checked step by step against the reference model in
``oracle/lease_fsm.py``; then lease-id hygiene and concurrent readers.
"""
import ctypes
import threading

import numpy as np
import pytest

import paper_2609_25451_amd as gms
from oracle.lease_fsm import LeaseModel

RC = {gms.GMS_OK: "ok", gms.GMS_ERR_STATE: "state", gms.GMS_ERR_INVALID: "invalid",
      gms.GMS_ERR_INTEGRITY: "integrity"}


class Raw:
    """Host-only store driven through the raw entry points (status codes, no exceptions)."""

    def __init__(self):
        h = ctypes.c_void_p()
        assert gms.gms_store_create(gms.HOST_ONLY, 0, 0, ctypes.byref(h)) == 0
        self.h = h

    def close(self):
        gms.gms_store_destroy(self.h)

    def state(self):
        st, rd, inv = ctypes.c_int(), ctypes.c_uint32(), ctypes.c_int()
        assert gms.gms_store_state(self.h, ctypes.byref(st), ctypes.byref(rd), ctypes.byref(inv)) == 0
        return gms.STORE_STATES[st.value], int(rd.value), bool(inv.value)

    def connect_rw(self):
        lease = ctypes.c_uint64()
        rc = gms.gms_store_connect_rw(self.h, ctypes.byref(lease))
        return RC[rc], (int(lease.value) if rc == 0 else None)

    def connect_ro(self):
        lease, cnt = ctypes.c_uint64(), ctypes.c_uint64()
        rc = gms.gms_store_connect_ro(self.h, gms.CONNECT_VERIFY, ctypes.byref(lease), ctypes.byref(cnt), None)
        return RC[rc], (int(lease.value) if rc == 0 else None)

    def commit(self, lease):
        return RC[gms.gms_store_commit(self.h, lease, None, 0, None, None, None)]

    def abort(self, lease):
        return RC[gms.gms_store_abort(self.h, lease)]

    def disconnect(self, lease):
        return RC[gms.gms_store_disconnect(self.h, lease)]


class Model(LeaseModel):
    """The reference model behind the same interface, so the scenario pins hold it too."""

    def state(self):
        return self.state_name, len(self.readers), self.invalid

    def close(self):
        pass


@pytest.fixture(params=["store", "model"])
def store(request):
    s = Raw() if request.param == "store" else Model()
    yield s
    s.close()


def test_cold_start_then_readers(store):
    """A cold engine takes the write lease, populates and commits; the writer
    reconnects read-only and more engines attach as readers."""
    assert store.state() == ("EMPTY", 0, False)
    rc, w = store.connect_rw()
    assert rc == "ok" and store.state() == ("RW", 0, False)
    assert store.commit(w) == "ok" and store.state() == ("COMMITTED", 0, False)
    rcs = [store.connect_ro() for _ in range(3)]
    assert all(rc == "ok" for rc, _ in rcs) and store.state() == ("RO", 3, False)
    assert len({lease for _, lease in rcs} | {w}) == 4, "lease ids are unique"


def test_writer_failure_before_commit_discards(store):
    """A writer that fails before commit leaves nothing behind."""
    _, w = store.connect_rw()
    assert store.disconnect(w) == "ok" and store.state() == ("EMPTY", 0, False)
    assert store.connect_ro() == ("state", None), "no committed state to read"
    _, w = store.connect_rw()
    assert store.abort(w) == "ok" and store.state() == ("EMPTY", 0, False)


def test_reader_failure_keeps_committed_state(store):
    _, w = store.connect_rw()
    store.commit(w)
    _, r1 = store.connect_ro()
    _, r2 = store.connect_ro()
    assert store.disconnect(r1) == "ok" and store.state() == ("RO", 1, False)
    assert store.disconnect(r2) == "ok" and store.state() == ("COMMITTED", 0, False)


def test_exclusive_write_only_after_last_reader(store):
    _, w = store.connect_rw()
    assert store.connect_rw() == ("state", None), "one writer at a time"
    assert store.connect_ro() == ("state", None), "no reader while a writer populates"
    store.commit(w)
    _, r = store.connect_ro()
    assert store.connect_rw() == ("state", None), "readers hold the committed state"
    store.disconnect(r)
    rc, w2 = store.connect_rw()
    assert rc == "ok" and store.state() == ("RW", 0, False), "writer reacquires after the last reader"
    assert store.commit(w2) == "ok" and store.state() == ("COMMITTED", 0, False)


def test_stale_and_foreign_leases(store):
    _, w = store.connect_rw()
    assert store.commit(w + 1000) == "invalid" and store.abort(0) == "invalid"
    store.commit(w)
    assert store.commit(w) == "invalid", "a committed writer's lease has ended"
    assert store.abort(w) == "invalid" and store.disconnect(w) == "invalid"
    _, r = store.connect_ro()
    assert store.commit(r) == "invalid" and store.abort(r) == "invalid"
    assert store.disconnect(r) == "ok" and store.disconnect(r) == "invalid", "double disconnect"
    assert store.disconnect(0) == "invalid"


@pytest.mark.parametrize("seed", range(20))
def test_random_walk_matches_model(seed):
    """Seeded random call sequences: the store and the model agree on every status and state."""
    store = Raw()
    rng = np.random.default_rng(seed)
    model = LeaseModel()
    real_of = {}  # model lease -> store lease
    for step in range(400):
        op = rng.choice(["rw", "ro", "commit", "abort", "disc", "disc", "bogus"])
        known = list(real_of)
        if op == "rw":
            (ms, ml), (rs, rl) = model.connect_rw(), store.connect_rw()
            assert ms == rs
            if ms == "ok":
                real_of[ml] = rl
        elif op == "ro":
            (ms, ml), (rs, rl) = model.connect_ro(), store.connect_ro()
            assert ms == rs
            if ms == "ok":
                real_of[ml] = rl
        elif op in ("commit", "abort", "disc") and known:
            ml = known[int(rng.integers(0, len(known)))]
            rl = real_of[ml]
            if op == "commit":
                assert model.commit(ml) == store.commit(rl)
            elif op == "abort":
                assert model.abort(ml) == store.abort(rl)
            else:
                assert model.disconnect(ml) == store.disconnect(rl)
        elif op == "bogus":
            assert store.disconnect(10 ** 9 + step) == "invalid"
        name, readers, invalid = store.state()
        assert (name, readers, invalid) == (model.state_name, len(model.readers), model.invalid), f"step {step} ({op})"
    store.close()


def test_concurrent_readers_and_python_leases():
    s = gms.Store(device=gms.HOST_ONLY)
    with s.connect_rw() as w:
        w.commit([])
    leases = []
    lock = threading.Lock()

    def reader():
        for _ in range(50):
            lease = s.connect_ro()
            with lock:
                leases.append(lease)

    ts = [threading.Thread(target=reader) for _ in range(8)]
    for t in ts:
        t.start()
    for t in ts:
        t.join()
    assert s.state() == ("RO", 400, False) and len({x.id for x in leases}) == 400
    for x in leases:
        x.close()
    assert s.state() == ("COMMITTED", 0, False)
    # a writer whose `with` body raises leaves the store EMPTY (failure before commit)
    with pytest.raises(RuntimeError):
        with s.connect_rw():
            raise RuntimeError("writer crashed while populating")
    assert s.state() == ("EMPTY", 0, False)
    with pytest.raises(gms.GmsError) as e:
        s.connect_ro()
    assert e.value.status == gms.GMS_ERR_STATE
    with pytest.raises(gms.GmsError) as e:
        with s.connect_rw() as w:
            w.alloc(4096)
    assert e.value.status == gms.GMS_ERR_STATE, "a host-only store has no memory"
    with s.connect_rw() as w:
        with pytest.raises(gms.GmsError) as e:
            w.commit([(0x1000, 16)])
        assert e.value.status == gms.GMS_ERR_STATE
    s.close()


def test_leases_outlive_a_closed_store():
    s = gms.Store(device=gms.HOST_ONLY)
    w = s.connect_rw()
    s.close()
    w.close()  # the store ended every lease when it closed: nothing left to release
    w2 = gms.WriteLease(s, 1)
    with pytest.raises(gms.GmsError) as e:
        w2.commit([])
    assert e.value.status == gms.GMS_ERR_STATE


# -- plausible mistakes in the reference model, each caught by the scenario pins ---------------

class _RwWhileReaders(Model):
    def connect_rw(self):
        if self.state_name == "RO":
            self.writer, self.state_name = self._lease(), "RW"
            return "ok", self.writer
        return super().connect_rw()


class _LastReaderStaysRO(Model):
    def disconnect(self, lease):
        if lease in self.readers and len(self.readers) == 1:
            self.readers.remove(lease)
            return "ok"
        return super().disconnect(lease)


class _WriterLeaveKeepsState(Model):
    def disconnect(self, lease):
        if lease is not None and lease == self.writer:
            return "ok"
        return super().disconnect(lease)


class _CommitKeepsWriter(Model):
    def commit(self, lease):
        w = self.writer
        rc = super().commit(lease)
        self.writer = w
        return rc


class _ReaderDuringWrite(Model):
    def connect_ro(self):
        if self.state_name == "RW":
            lease = self._lease()
            self.readers.add(lease)
            return "ok", lease
        return super().connect_ro()


class _ReusedLeaseIds(Model):
    def _lease(self):
        return 1


class _AbortToCommitted(Model):
    def abort(self, lease):
        rc = super().abort(lease)
        if rc == "ok":
            self.state_name = "COMMITTED"
        return rc


SCENARIOS = [test_cold_start_then_readers, test_writer_failure_before_commit_discards,
             test_reader_failure_keeps_committed_state, test_exclusive_write_only_after_last_reader,
             test_stale_and_foreign_leases]


@pytest.mark.parametrize("mutant", [_RwWhileReaders, _LastReaderStaysRO, _WriterLeaveKeepsState, _CommitKeepsWriter,
                                    _ReaderDuringWrite, _ReusedLeaseIds, _AbortToCommitted],
                         ids=lambda c: c.__name__.lstrip("_"))
def test_model_mutants_are_caught(mutant):
    caught = []
    for scenario in SCENARIOS:
        try:
            scenario(mutant())
        except AssertionError:
            caught.append(scenario.__name__)
    assert caught, f"{mutant.__name__} passes every scenario pin"
