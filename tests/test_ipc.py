"""The lease protocol across processes, on the CPU: a host-only owner process serving
clients over its Unix-domain socket (paper section 3.2, Figure 4; section 4).

The owner runs as its own process (``python -m paper_2609_25451_amd.owner``);
clients are connections from this process or from child processes that the
tests kill with SIGKILL.  States are read back over the socket and checked
against the reference model in oracle/lease_fsm.py.
"""
import os
import signal
import subprocess
import sys
import time

import numpy as np
import pytest

import paper_2609_25451_amd as gms
from oracle.lease_fsm import COMMITTED, EMPTY, RO, RW, LeaseModel

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture()
def owner(tmp_path):
    sock = str(tmp_path / "gms.sock")
    p = subprocess.Popen([sys.executable, "-m", "paper_2609_25451_amd.owner", sock, "--device", "-1"], cwd=ROOT,
                         stdout=subprocess.PIPE, stderr=subprocess.PIPE, text=True)
    line = p.stdout.readline()
    assert line.startswith("owner ready"), line + p.stderr.read()
    yield sock
    p.send_signal(signal.SIGTERM)
    try:
        assert p.wait(timeout=20) == 0, p.stderr.read()
    finally:
        if p.poll() is None:
            p.kill()
            p.wait()
    assert not os.path.exists(sock), "the owner left its socket file behind"


def state(sock):
    return gms.owner_query(sock)[:3]


def wait_state(sock, want, timeout=10.0):
    t0 = time.time()
    while time.time() - t0 < timeout:
        if state(sock) == want:
            return
        time.sleep(0.02)
    assert state(sock) == want


_CHILD = r"""
import sys, time
sys.path.insert(0, sys.argv[1])
import paper_2609_25451_amd as gms
mode = gms.LEASE_RW if sys.argv[3] == "rw" else gms.LEASE_RO
c = gms.Client(sys.argv[2], mode)
print("connected", c.info()["lease"], flush=True)
time.sleep(120)
"""


def child(sock, mode):
    p = subprocess.Popen([sys.executable, "-c", _CHILD, ROOT, sock, mode], stdout=subprocess.PIPE,
                         stderr=subprocess.PIPE, text=True)
    line = p.stdout.readline()
    assert line.startswith("connected"), line + p.stderr.read()
    return p


def kill(p):
    p.kill()
    p.wait()


def test_cold_start_readers_and_exclusive_write(owner):
    assert state(owner) == ("EMPTY", 0, False)
    w = gms.Client(owner, gms.LEASE_RW)
    assert state(owner) == ("RW", 0, False) and w.info()["lease"] > 0 and w.info()["device"] == -1
    with pytest.raises(gms.GmsError) as e:  # one writer at a time
        gms.Client(owner, gms.LEASE_RW)
    assert e.value.status == gms.GMS_ERR_STATE
    with pytest.raises(gms.GmsError) as e:  # no reader before commit
        gms.Client(owner, gms.LEASE_RO)
    assert e.value.status == gms.GMS_ERR_STATE
    with pytest.raises(gms.GmsError) as e:  # a host-only owner has no memory
        w.alloc(4096)
    assert e.value.status == gms.GMS_ERR_STATE
    w.commit([])
    assert state(owner) == ("COMMITTED", 0, False) and w.info()["lease"] == 0
    w.close()  # a committed writer leaving changes nothing
    assert state(owner) == ("COMMITTED", 0, False)
    r1, r2 = gms.Client(owner, gms.LEASE_RO), gms.Client(owner, gms.LEASE_RO)
    assert state(owner) == ("RO", 2, False) and r1.layout() == [] and r1.info()["lease"] != r2.info()["lease"]
    with pytest.raises(gms.GmsError) as e:  # exclusive write only after the last reader
        gms.Client(owner, gms.LEASE_RW)
    assert e.value.status == gms.GMS_ERR_STATE
    r1.close()
    assert state(owner) == ("RO", 1, False)
    r2.close()
    assert state(owner) == ("COMMITTED", 0, False)
    w2 = gms.Client(owner, gms.LEASE_RW)  # a writer reacquires the committed state
    assert state(owner) == ("RW", 0, False)
    w2.abort()
    assert state(owner) == ("EMPTY", 0, False)
    w2.close()


def test_writer_killed_before_commit_leaves_empty(owner):
    """A writer process that dies before commit: the owner discards its incomplete state."""
    p = child(owner, "rw")
    assert state(owner) == ("RW", 0, False)
    kill(p)
    wait_state(owner, ("EMPTY", 0, False))
    # and from committed state: a new writer that dies also leaves EMPTY (its writes are unknown)
    w = gms.Client(owner, gms.LEASE_RW)
    w.commit([])
    w.close()
    p = child(owner, "rw")
    assert state(owner) == ("RW", 0, False)
    kill(p)
    wait_state(owner, ("EMPTY", 0, False))


def test_dead_reader_releases_only_its_lease(owner):
    w = gms.Client(owner, gms.LEASE_RW)
    w.commit([])
    w.close()
    a, b = child(owner, "ro"), child(owner, "ro")
    local = gms.Client(owner, gms.LEASE_RO)
    assert state(owner) == ("RO", 3, False)
    kill(a)
    wait_state(owner, ("RO", 2, False))
    kill(b)
    wait_state(owner, ("RO", 1, False))
    local.close()
    assert state(owner) == ("COMMITTED", 0, False)
    r = gms.Client(owner, gms.LEASE_RO)  # committed state survived every reader
    assert state(owner) == ("RO", 1, False)
    r.close()


def test_owner_survives_clients_that_vanish_mid_message(owner, tmp_path):
    """A peer that connects and closes, or sends garbage, costs only its own connection."""
    import socket

    for junk in (b"", b"x" * 7, b"\0" * 64, b"GMS1" + b"\xff" * 60):
        s = socket.socket(socket.AF_UNIX, socket.SOCK_STREAM)
        s.connect(owner)
        if junk:
            s.sendall(junk)
        s.close()
    assert state(owner) == ("EMPTY", 0, False)
    w = gms.Client(owner, gms.LEASE_RW)
    w.commit([])
    w.close()
    assert state(owner) == ("COMMITTED", 0, False)


@pytest.mark.parametrize("seed", range(6))
def test_random_walks_follow_the_model(owner, seed):
    """Seeded walks of connects, commits, aborts and disconnects against the reference model
    of the protocol (the deaths of writer and reader processes are the tests above)."""
    rng = np.random.default_rng(seed)
    model = LeaseModel()
    names = {EMPTY: "EMPTY", RW: "RW", COMMITTED: "COMMITTED", RO: "RO"}
    clients = {}  # model lease -> (client, kind)
    spent = []    # writers whose lease ended at commit or abort: connections only
    for _ in range(80):
        op = rng.choice(["rw", "ro", "ro", "commit", "abort", "bye", "bye"])
        if op in ("rw", "ro"):
            want, lease = model.connect_rw() if op == "rw" else model.connect_ro()
            try:
                c = gms.Client(owner, gms.LEASE_RW if op == "rw" else gms.LEASE_RO)
                got = "ok"
            except gms.GmsError as e:
                got = "state" if e.status == gms.GMS_ERR_STATE else str(e.status)
            assert got == want, (op, model.state_name)
            if lease is not None:
                clients[lease] = (c, op)
        elif op in ("commit", "abort") and model.writer is not None:
            lease = model.writer
            c, _ = clients.pop(lease)
            if op == "commit":
                c.commit([])
                assert model.commit(lease) == "ok"
            else:
                c.abort()
                assert model.abort(lease) == "ok"
            spent.append(c)
        elif op == "bye" and clients:
            lease = list(clients)[int(rng.integers(0, len(clients)))]
            c, _ = clients.pop(lease)
            c.close()
            assert model.disconnect(lease) == "ok"
        elif op == "bye" and spent:
            spent.pop(int(rng.integers(0, len(spent)))).close()  # changes nothing
        assert state(owner) == (names[model.state_name], len(model.readers), False)
    for c, _ in clients.values():
        c.close()
    for c in spent:
        c.close()


_CHURN = r"""
import random, sys, time
sys.path.insert(0, sys.argv[1])
import paper_2609_25451_amd as gms
rng = random.Random(int(sys.argv[3]))
held = 0
for _ in range(12):
    c = gms.Client(sys.argv[2], gms.LEASE_RO)
    held += 1
    time.sleep(rng.random() * 0.02)
    if rng.random() < 0.2:
        c._h = None  # leave without a goodbye: the connection closes when the process ends
        break
    c.close()
print("done", held, flush=True)
"""


def test_concurrent_reader_processes_keep_the_count(owner):
    """Six reader processes connect and leave at random, some without saying goodbye, while
    this process watches: the state is RO exactly while the count is positive, the count never
    exceeds the processes, and once they are gone the state is COMMITTED with no reader."""
    w = gms.Client(owner, gms.LEASE_RW)
    w.commit([])
    w.close()
    ps = [subprocess.Popen([sys.executable, "-c", _CHURN, ROOT, owner, str(seed)], stdout=subprocess.PIPE,
                           stderr=subprocess.PIPE, text=True) for seed in range(6)]
    seen = set()
    while any(p.poll() is None for p in ps):
        st, rd, inv = state(owner)
        assert st in ("COMMITTED", "RO") and not inv and rd <= 6
        assert (st == "RO") == (rd > 0)
        seen.add(rd)
        time.sleep(0.01)
    for p in ps:
        out, err = p.communicate()
        assert p.returncode == 0 and out.startswith("done"), out + err
    wait_state(owner, ("COMMITTED", 0, False))
    assert max(seen) >= 2, seen  # the readers did overlap
