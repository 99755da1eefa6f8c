"""Reference model of the GMS model-state lease protocol -- TEST INFRASTRUCTURE ONLY.

Only ``tests/`` may import this module.  It writes out the state machine of
paper section 3.2 (Figure 4) and the rules stated beside it, in plain Python,
with no code shared with the library:

* States: EMPTY (no layout), RW (one writer), COMMITTED (committed, no
  readers), RO (committed, one or more readers).
* EMPTY --RW connect--> RW; RW --abort--> EMPTY; RW --commit--> COMMITTED;
  COMMITTED --RW connect--> RW; COMMITTED --RO connect--> RO;
  RO --RO connect / non-last disconnect--> RO; RO --last disconnect-->
  COMMITTED.
* A writer that fails (leaves) before commit has its incomplete state
  discarded: EMPTY.  A reader's failure only releases its lease.
* Exclusive write access is available again only after the last reader
  has disconnected.
* Integrity errors invalidate the committed state (section 3.2); this model
  takes the library's reading: an invalid state grants no read lease, and a
  writer that commits again makes it valid.

Every call returns a status: "ok", "state" (not allowed now), "invalid"
(unknown or foreign lease) or "integrity" (refused on an invalid state).
"""
from __future__ import annotations

EMPTY, RW, COMMITTED, RO = "EMPTY", "RW", "COMMITTED", "RO"


class LeaseModel:
    def __init__(self):
        self.state_name = EMPTY
        self.writer = None
        self.readers: set[int] = set()
        self.invalid = False
        self._next = 1

    def _lease(self) -> int:
        lease = self._next
        self._next += 1
        return lease

    # -- writer -------------------------------------------------------------
    def connect_rw(self):
        if self.state_name not in (EMPTY, COMMITTED):  # a writer, or readers, hold it
            return "state", None
        self.writer = self._lease()
        self.state_name = RW
        return "ok", self.writer

    def commit(self, lease):
        if self.state_name != RW or lease != self.writer:
            return "invalid"
        self.writer = None
        self.state_name = COMMITTED
        self.invalid = False
        return "ok"

    def abort(self, lease):
        if self.state_name != RW or lease != self.writer:
            return "invalid"
        self._discard()
        return "ok"

    def _discard(self):
        self.writer = None
        self.invalid = False
        self.state_name = EMPTY

    # -- readers ------------------------------------------------------------
    def connect_ro(self):
        if self.state_name not in (COMMITTED, RO):
            return "state", None
        if self.invalid:
            return "integrity", None
        lease = self._lease()
        self.readers.add(lease)
        self.state_name = RO
        return "ok", lease

    def integrity_failure(self):
        """A verification found committed blocks changed."""
        if self.state_name in (COMMITTED, RO):
            self.invalid = True

    # -- either -------------------------------------------------------------
    def disconnect(self, lease):
        if lease is not None and lease == self.writer:  # writer leaving before commit
            self._discard()
            return "ok"
        if lease not in self.readers:
            return "invalid"
        self.readers.remove(lease)
        if not self.readers:
            self.state_name = COMMITTED
        return "ok"
