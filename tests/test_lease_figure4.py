"""The lease protocol's transitions as the paper draws them (section 3.2, Figure 4), from a
fixture written from the figure and its text (tests/golden/lease_transitions_figure4.txt),
replayed against the reference model, the in-process store and the owner process, each
without device memory.  The fixture, not the model, is the authority here: the model was
written together with the store, and this pins both to the figure."""
import os
import signal
import subprocess
import sys

import pytest

import paper_2609_25451_amd as gms
from oracle.lease_fsm import LeaseModel

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
FIXTURE = os.path.join(ROOT, "tests", "golden", "lease_transitions_figure4.txt")


def _rows():
    rows = []
    for line in open(FIXTURE):
        line = line.split("#", 1)[0].strip()
        if line:
            start, event, result = line.split()
            rows.append((start, event, result))
    return rows


ROWS = _rows()
NAMES = {"EMPTY": ("EMPTY", 0), "RW": ("RW", 0), "COMMITTED": ("COMMITTED", 0), "RO1": ("RO", 1), "RO2": ("RO", 2)}


class ModelSide:
    def __init__(self):
        self.m = LeaseModel()

    def rw(self):
        st, lease = self.m.connect_rw()
        return lease if st == "ok" else None

    def ro(self):
        st, lease = self.m.connect_ro()
        return lease if st == "ok" else None

    def commit(self, w):
        return self.m.commit(w) == "ok"

    def abort(self, w):
        return self.m.abort(w) == "ok"

    def leave(self, lease):
        return self.m.disconnect(lease) == "ok"

    def state(self):
        return self.m.state_name, len(self.m.readers)


class StoreSide:
    def __init__(self):
        self.s = gms.Store(device=gms.HOST_ONLY)

    def rw(self):
        try:
            return self.s.connect_rw()
        except gms.GmsError:
            return None

    def ro(self):
        try:
            return self.s.connect_ro(verify=False)
        except gms.GmsError:
            return None

    def commit(self, w):
        w.commit([])
        return True

    def abort(self, w):
        w.abort()
        return True

    def leave(self, lease):
        lease.close()
        return True

    def state(self):
        st, rd, _ = self.s.state()
        return st, rd


class OwnerSide:
    def __init__(self, sock):
        self.sock = sock

    def rw(self):
        try:
            return gms.Client(self.sock, gms.LEASE_RW)
        except gms.GmsError:
            return None

    def ro(self):
        try:
            return gms.Client(self.sock, gms.LEASE_RO)
        except gms.GmsError:
            return None

    def commit(self, w):
        w.commit([])
        return True

    def abort(self, w):
        w.abort()
        return True

    def leave(self, c):  # the connection closes: for the owner a departure and a death look alike
        c.close()
        return True

    def state(self):
        st, rd, _, _ = gms.owner_query(self.sock)
        return st, rd


def _replay(side, start, event, result):
    """Reaches `start`, applies `event`, checks `result`; returns the handles it opened."""
    writer, readers, opened = None, [], []
    if start != "EMPTY":  # reach the start state: a writer, its commit, then readers
        writer = side.rw()
        assert writer is not None
        opened.append(writer)
        if start != "RW":
            assert side.commit(writer)
            writer = None
            for _ in range({"COMMITTED": 0, "RO1": 1, "RO2": 2}[start]):
                r = side.ro()
                assert r is not None
                readers.append(r)
                opened.append(r)
    assert side.state() == NAMES[start], (start, side.state())
    ok = True
    if event in ("rw_connect", "ro_connect"):
        got = side.rw() if event == "rw_connect" else side.ro()
        ok = got is not None
        if ok:
            opened.append(got)
    elif event == "commit":
        ok = side.commit(writer)
    elif event == "abort":
        ok = side.abort(writer)
    elif event == "writer_leaves":
        ok = side.leave(writer)
    elif event == "reader_leaves":
        ok = side.leave(readers.pop())
    else:
        raise AssertionError(event)
    if result == "refused":
        assert not ok, (start, event)
        assert side.state() == NAMES[start], (start, event, side.state())
    else:
        assert ok, (start, event)
        assert side.state() == NAMES[result], (start, event, side.state())
    return opened


def test_fixture_covers_every_edge_of_the_figure():
    edges = {(s, e) for s, e, r in ROWS if r != "refused"}
    assert {("EMPTY", "rw_connect"), ("RW", "commit"), ("RW", "abort"), ("COMMITTED", "rw_connect"),
            ("COMMITTED", "ro_connect"), ("RO1", "ro_connect"), ("RO2", "reader_leaves"),
            ("RO1", "reader_leaves")} <= edges


@pytest.mark.parametrize("row", ROWS, ids=[" ".join(r) for r in ROWS])
def test_reference_model(row):
    _replay(ModelSide(), *row)


@pytest.mark.parametrize("row", ROWS, ids=[" ".join(r) for r in ROWS])
def test_in_process_store(row):
    side = StoreSide()
    try:
        _replay(side, *row)
    finally:
        side.s.close()


@pytest.fixture(scope="module")
def owner_sock(tmp_path_factory):
    sock = str(tmp_path_factory.mktemp("fig4") / "gms.sock")
    p = subprocess.Popen([sys.executable, "-m", "paper_2609_25451_amd.owner", sock, "--device", "-1"], cwd=ROOT,
                         stdout=subprocess.PIPE, stderr=subprocess.PIPE, text=True)
    line = p.stdout.readline()
    assert line.startswith("owner ready"), line + p.stderr.read()
    yield sock
    p.send_signal(signal.SIGTERM)
    try:
        assert p.wait(timeout=20) == 0
    finally:
        if p.poll() is None:
            p.kill()
            p.wait()


@pytest.mark.parametrize("row", ROWS, ids=[" ".join(r) for r in ROWS])
def test_owner_process(owner_sock, row):
    # each row starts from EMPTY: a writer that connects and leaves discards whatever was there
    c = gms.Client(owner_sock, gms.LEASE_RW) if gms.owner_query(owner_sock)[0] in ("EMPTY", "COMMITTED") else None
    assert c is not None, gms.owner_query(owner_sock)
    c.close()
    assert gms.owner_query(owner_sock)[:2] == ("EMPTY", 0)
    for c in _replay(OwnerSide(owner_sock), *row):
        c.close()  # a connection that already ended closes as a no-op
