"""The model-state store across processes on the GPU (paper section 3.2, Figure 4;
section 4): an owner process holds the allocations, a writer process populates and
commits them and exits, reader processes map them read-only and verify them.

Every process here is a fresh child (never an exec of a process that touched the
GPU): the owner, one writer and one or two readers at a time, next to this test's
own process.  Contents come from the seeded generator; the oracle decides the
expected block and tensor hashes.
"""
import json
import os
import signal
import subprocess
import sys
import time

import pytest

import paper_2609_25451_amd as gms
from gpu_util import need_gpu

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

# Shared by the child scripts: the committed entries and their generated contents.
_COMMON = r"""
import json, sys, numpy as np, torch
sys.path[:0] = [sys.argv[1], sys.argv[1] + "/tests"]
import paper_2609_25451_amd as gms, synth, oracle
from gpu_util import d2h, h2d
SOCK = sys.argv[2]
SEED, SPECS = synth.weight_set("tiny")
BIG = (600 << 20) + 5              # above half a slab: an allocation of its own
ODD = 4000                          # an entry 3 bytes past a 16-byte boundary, inside a slab

def fill(addrs):
    for i, sp in enumerate(SPECS):
        synth.dev_fill_bf16(addrs[i], sp.numel, SEED, i)
    synth.dev_fill_bytes(addrs[-2], BIG, 7, 1)
    synth.dev_fill_bytes(addrs[-1], ODD, 7, 2)
    torch.cuda.synchronize()

def sizes():
    return [sp.nbytes for sp in SPECS] + [BIG, ODD]

def reference():
    # the generator's bytes of every entry, made in scratch device memory and copied back
    out = []
    for n, make in zip(sizes(), range(len(sizes()))):
        t = torch.empty(n, dtype=torch.uint8, device="cuda")
        a = t.data_ptr()
        if make < len(SPECS):
            synth.dev_fill_bf16(a, n // 2, SEED, make)
        else:
            synth.dev_fill_bytes(a, n, 7, 1 if make == len(SPECS) else 2)
        torch.cuda.synchronize()
        out.append(t.cpu().numpy())
    return out
"""

_WRITER = _COMMON + r"""
def step(msg):
    print("writer:", msg, file=sys.stderr, flush=True)
step("connect")
c = gms.Client(SOCK, gms.LEASE_RW)
step("alloc and free")
tmp, own = c.alloc(1000), c.alloc(700 << 20)
c.free(tmp)
c.free(own)
step("alloc slab entries")
addrs = [c.alloc(sp.nbytes) for sp in SPECS]
step("alloc dedicated entry")
addrs.append(c.alloc(BIG))
addrs.append(c.alloc(ODD + 16, align=16) + 3)
step("fill")
fill(addrs)
step("commit")
entries = list(zip(addrs, sizes()))
o_blk, _ = oracle.hashes(reference())
c.commit(entries, expected=torch.from_numpy(o_blk.view(np.int64)).cuda())
assert c.layout() == [] and c.manifest() is None  # the writer reconnects read-only to use it
print("committed", json.dumps({"entries": len(entries), "info": c.info()}), flush=True)
"""

_READER = _COMMON + r"""
import time
c = gms.Client(SOCK, gms.LEASE_RO, verify=True)
lay = c.layout()
assert [n for _, n in lay] == sizes(), lay
ref = reference()
for (a, n), want in zip(lay, ref):
    assert np.array_equal(d2h(a, n), want), "mapped bytes differ from the generator"
o_blk, o_ten = oracle.hashes(ref)
m = c.manifest()
blk = torch.zeros(m.num_blocks, dtype=torch.int64, device="cuda")
ten = torch.zeros(m.num_entries, dtype=torch.int64, device="cuda")
cnt = torch.zeros(1, dtype=torch.int64, device="cuda")
exp = torch.from_numpy(o_blk.view(np.int64)).cuda()
gms.verify(m, expected=exp, blk_hash=blk, ten_hash=ten, mismatch_count=cnt)
torch.cuda.synchronize()
assert int(cnt.item()) == 0
assert np.array_equal(blk.cpu().numpy().view(np.uint64), o_blk), "reader's block hashes differ from the oracle"
assert np.array_equal(ten.cpu().numpy().view(np.uint64), o_ten), "reader's tensor hashes differ from the oracle"
assert c.verify() == 0
print("reader ok", json.dumps(c.info()), flush=True)
if len(sys.argv) > 3 and sys.argv[3] == "stay":
    time.sleep(120)
"""

_REWRITER = _COMMON + r"""
# a writer that reacquires the committed allocation set and its layout, changes one byte and
# commits against the first writer's hashes: refused with exactly one mismatch, and the lease
# is kept; with the byte put back the commit holds
c = gms.Client(SOCK, gms.LEASE_RW)
lay = c.layout()
assert [n for _, n in lay] == sizes(), lay
o_blk, _ = oracle.hashes(reference())
exp = torch.from_numpy(o_blk.view(np.int64)).cuda()
a0, n0 = lay[0]
keep = d2h(a0 + 77, 1)
h2d(a0 + 77, keep ^ np.uint8(0x40))
try:
    c.commit(lay, expected=exp)
    raise SystemExit("a changed byte was committed")
except gms.GmsError as e:
    assert e.status == gms.GMS_ERR_INTEGRITY and e.mismatches == 1, (e.status, e.mismatches)
h2d(a0 + 77, keep)
c.commit(lay, expected=exp)
print("recommitted", flush=True)
"""

_RESHAPER = _COMMON + r"""
# a writer that takes over committed state gets its slabs back with the committed entries as
# their parts: it frees one entry inside a slab and the entry with an allocation of its own,
# allocates both again, repopulates and commits a layout that moved
c = gms.Client(SOCK, gms.LEASE_RW)
lay = c.layout()
assert [n for _, n in lay] == sizes() and c.manifest() is not None
try:  # inside a slab but not the start of a part
    c.free(lay[0][0] + 8)
    raise SystemExit("freed a middle address")
except gms.GmsError as e:
    assert e.status == gms.GMS_ERR_INVALID, e.status
c.free(lay[0][0])
assert c.layout() == [] and c.manifest() is None  # the committed layout is no longer whole
c.free(lay[-2][0])
keep = lay[1:-2] + [lay[-1]]
new0 = c.alloc(sizes()[0])
for a, n in keep:  # the new part lies outside every entry that stays
    assert new0 + sizes()[0] <= a or a + n <= new0, (new0, a, n)
newbig = c.alloc(BIG)
addrs = [new0] + [a for a, _ in lay[1:-2]] + [newbig, lay[-1][0]]
fill(addrs)
o_blk, _ = oracle.hashes(reference())
c.commit(list(zip(addrs, sizes())), expected=torch.from_numpy(o_blk.view(np.int64)).cuda())
print("reshaped", flush=True)
"""

_ALLOCATOR = _COMMON + r"""
# a writer's first-fit suballocation under a random walk of allocs and frees: live parts never
# overlap, each holds its own bytes after every other part was written, and the live set
# commits and verifies in a reader
rng = np.random.default_rng(int(sys.argv[3]))
c = gms.Client(SOCK, gms.LEASE_RW)
live = {}  # addr -> (bytes, stream id)
sid = 10
for step in range(300):
    if live and rng.random() < 0.4:
        a = list(live)[int(rng.integers(0, len(live)))]
        c.free(a)
        del live[a]
        continue
    r = rng.random()
    if r < 0.6:
        n = int(rng.integers(1, 5000))
    elif r < 0.9:
        n = int(rng.integers(5000, 3 << 20))
    elif r < 0.97:
        n = int(rng.integers(300 << 20, 520 << 20))  # up to about half a slab: first fit
    else:
        n = int(rng.integers(600 << 20, 1 << 30))  # an allocation of its own
    align = int(rng.choice([0, 16, 256, 4096]))
    a = c.alloc(n, align=align)
    assert align == 0 or a % align == 0
    for b, (m, _) in live.items():
        assert a + n <= b or b + m <= a, ("overlap", a, n, b, m)
    sid += 1
    live[a] = (n, sid)
for a, (n, k) in live.items():
    synth.dev_fill_bytes(a, n, 5, k)
torch.cuda.synchronize()
entries = sorted((a, n) for a, (n, _) in live.items())
datas = [synth.random_bytes(n, 5, live[a][1]) for a, n in entries]
for (a, n), want in zip(entries, datas):
    if n <= (8 << 20):
        assert np.array_equal(d2h(a, n), want), "a part was overwritten by another"
o_blk, _ = oracle.hashes(datas)
c.commit(entries, expected=torch.from_numpy(o_blk.view(np.int64)).cuda())
print("allocator ok", len(entries), flush=True)
"""

_CORRUPTER = _COMMON + r"""
# stands for a fault that changes committed memory behind the protocol's back: this reader
# writes one byte of entry 3 through its own mapping (nothing in the library would)
c = gms.Client(SOCK, gms.LEASE_RO)
a3, n3 = c.layout()[3]
h2d(a3 + 5, d2h(a3 + 5, 1) ^ np.uint8(0x01))
torch.cuda.synchronize()
print("corrupted", flush=True)
"""

_VERIFY_REFUSED = _COMMON + r"""
try:
    gms.Client(SOCK, gms.LEASE_RO, verify=True)
    raise SystemExit("a changed block was not caught")
except gms.GmsError as e:
    assert e.status == gms.GMS_ERR_INTEGRITY and e.mismatches == 1, (e.status, e.mismatches)
try:  # the committed state is invalid now: no read lease, verified or not
    gms.Client(SOCK, gms.LEASE_RO)
    raise SystemExit("a read lease on invalid state")
except gms.GmsError as e:
    assert e.status == gms.GMS_ERR_INTEGRITY, e.status
print("refused", flush=True)
"""

_REPAIRER = _COMMON + r"""
# a writer repopulates the allocation set from the generator and commits against the oracle
c = gms.Client(SOCK, gms.LEASE_RW)
lay = c.layout()
fill([a for a, _ in lay])
o_blk, _ = oracle.hashes(reference())
c.commit(lay, expected=torch.from_numpy(o_blk.view(np.int64)).cuda())
print("repaired", flush=True)
"""

_KILLED_WRITER = _COMMON + r"""
c = gms.Client(SOCK, gms.LEASE_RW)
try:  # one shared allocation holds at most 1 GiB
    c.alloc((1 << 30) + 1)
    raise SystemExit("an allocation above 1 GiB was granted")
except gms.GmsError as e:
    assert e.status == gms.GMS_ERR_SIZE, e.status
a = [c.alloc(64 << 20) for _ in range(3)] + [c.alloc(BIG)]
synth.dev_fill_bytes(a[0], 64 << 20, 9, 9)
torch.cuda.synchronize()
print("connected", flush=True)
import time
time.sleep(120)
"""


def _spawn(script, sock, *extra):
    # -X faulthandler: a crash in a child names the Python line that was running
    return subprocess.Popen([sys.executable, "-X", "faulthandler", "-c", script, ROOT, sock, *extra],
                            stdout=subprocess.PIPE, stderr=subprocess.PIPE, text=True)


def _finish(p, timeout=240):
    out, err = p.communicate(timeout=timeout)
    assert p.returncode == 0, out[-2000:] + err[-4000:]
    return out


def _wait_line(p, prefix, timeout=240):
    t0 = time.time()
    line = p.stdout.readline()
    assert line.startswith(prefix), line + p.stderr.read()[-4000:]
    assert time.time() - t0 < timeout
    return line


def _wait_state(sock, want, timeout=20.0):
    t0 = time.time()
    while time.time() - t0 < timeout:
        if gms.owner_query(sock)[:3] == want:
            return
        time.sleep(0.05)
    assert gms.owner_query(sock)[:3] == want


@pytest.fixture()
def owner(tmp_path):
    need_gpu()
    sock = str(tmp_path / "gms.sock")
    print(f"owner process on device 0 at {sock}", flush=True)
    p = subprocess.Popen([sys.executable, "-m", "paper_2609_25451_amd.owner", sock, "--device", "0"], cwd=ROOT,
                         stdout=subprocess.PIPE, stderr=subprocess.PIPE, text=True)
    _wait_line(p, "owner ready")
    yield sock
    p.send_signal(signal.SIGTERM)
    try:
        assert p.wait(timeout=60) == 0, p.stderr.read()
    finally:
        if p.poll() is None:
            p.kill()
            p.wait()


def test_writer_commits_and_exits_readers_attach_and_verify(owner):
    print("writer process", flush=True)
    out = _finish(_spawn(_WRITER, owner))
    assert "committed" in out, out
    # the writer has exited: the owner still holds the committed state
    state, readers, invalid, allocs = gms.owner_query(owner)
    assert (state, readers, invalid) == ("COMMITTED", 0, False) and allocs >= 2
    print("reader process", flush=True)
    out = _finish(_spawn(_READER, owner))
    info = json.loads(out.split("reader ok", 1)[1])
    assert info["device"] == 0 and info["lease"] > 0
    assert gms.owner_query(owner)[:3] == ("COMMITTED", 0, False)

    # a reader that dies releases only its lease
    print("two reader processes, one killed", flush=True)
    r1, r2 = _spawn(_READER, owner, "stay"), _spawn(_READER, owner, "stay")
    _wait_line(r1, "reader ok")
    _wait_line(r2, "reader ok")
    assert gms.owner_query(owner)[:3] == ("RO", 2, False)
    r1.kill()
    r1.wait()
    _wait_state(owner, ("RO", 1, False))
    r2.kill()
    r2.wait()
    _wait_state(owner, ("COMMITTED", 0, False))
    print("reader after the deaths", flush=True)
    _finish(_spawn(_READER, owner))

    # a writer reacquires the committed state; a changed byte is refused at commit
    print("rewriter process", flush=True)
    out = _finish(_spawn(_REWRITER, owner))
    assert "recommitted" in out
    assert gms.owner_query(owner)[:3] == ("COMMITTED", 0, False)
    _finish(_spawn(_READER, owner))


def test_writer_killed_before_commit_releases_its_memory(owner):
    print("writer process, killed before commit", flush=True)
    p = _spawn(_KILLED_WRITER, owner)
    _wait_line(p, "connected")
    state, _, _, allocs = gms.owner_query(owner)
    assert state == "RW" and allocs == 2  # one 1 GiB slab holding the three 64 MiB parts, one of its own
    p.kill()
    p.wait()
    _wait_state(owner, ("EMPTY", 0, False))
    assert gms.owner_query(owner)[3] == 0
    with pytest.raises(gms.GmsError) as e:  # nothing to read
        gms.Client(owner, gms.LEASE_RO)
    assert e.value.status == gms.GMS_ERR_STATE
    print("a new writer after the death", flush=True)
    out = _finish(_spawn(_WRITER, owner))
    assert "committed" in out
    _finish(_spawn(_READER, owner))


def test_changed_state_is_refused_until_a_writer_repairs_it(owner):
    """Verify before reattach across processes: committed memory changed behind the
    protocol's back refuses the next verified read lease with exactly one mismatching block,
    invalidates the state for every reader, and a writer's repopulation makes it valid."""
    _finish(_spawn(_WRITER, owner))
    print("corrupting reader", flush=True)
    assert "corrupted" in _finish(_spawn(_CORRUPTER, owner))
    print("verifying reader", flush=True)
    assert "refused" in _finish(_spawn(_VERIFY_REFUSED, owner))
    assert gms.owner_query(owner)[:3] == ("COMMITTED", 0, True)
    print("repairing writer", flush=True)
    assert "repaired" in _finish(_spawn(_REPAIRER, owner))
    assert gms.owner_query(owner)[:3] == ("COMMITTED", 0, False)
    _finish(_spawn(_READER, owner))


def test_writer_takes_over_committed_slabs_frees_and_reallocates(owner):
    """A writer from committed state frees committed entries (one inside a slab, one with an
    allocation of its own) and allocates again; its layout and manifest are dropped at the
    first free, and the new layout commits and verifies in a reader."""
    _finish(_spawn(_WRITER, owner))
    allocs = gms.owner_query(owner)[3]
    print("reshaping writer", flush=True)
    assert "reshaped" in _finish(_spawn(_RESHAPER, owner))
    assert gms.owner_query(owner)[:3] == ("COMMITTED", 0, False) and gms.owner_query(owner)[3] == allocs
    _finish(_spawn(_READER, owner))


def test_writer_suballocation_random_walk(owner):
    """300 random allocs and frees (bytes to 1 GiB, alignments to 4 KiB) in a writer process:
    no two live parts overlap, every part keeps its own bytes, and the surviving set commits
    against the oracle's hashes and verifies in a reader."""
    print("allocating writer", flush=True)
    out = _finish(_spawn(_ALLOCATOR, owner, "7"))
    assert "allocator ok" in out
    assert gms.owner_query(owner)[:3] == ("COMMITTED", 0, False)
    c = gms.Client(owner, gms.LEASE_RO, verify=True)  # re-hashed here against the commit-time hashes
    assert c.verify() == 0
    c.close()
