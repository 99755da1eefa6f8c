"""The GMS owner process of one GPU: ``python -m paper_2609_25451_amd.owner SOCKET [--device N]``.

Holds the device's model-state allocations beyond any engine's lifetime and
serves writer and reader leases over a Unix-domain socket (gms_owner_* in
include/gms.h).  Prints ``owner ready <socket>`` once it listens; SIGTERM or
SIGINT stop it, which releases every allocation.  ``--device -1`` runs the
lease protocol alone, without device memory.
"""
from __future__ import annotations

import argparse
import signal
import sys
import threading


def main(argv=None) -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("socket")
    ap.add_argument("--device", type=int, default=0)
    args = ap.parse_args(argv)
    import paper_2609_25451_amd as gms

    owner = gms.Owner(args.socket, device=args.device)
    done = threading.Event()
    err = []

    def serve():
        try:
            owner.run()
        except Exception as e:  # reported after the loop ends
            err.append(e)
        finally:
            done.set()

    t = threading.Thread(target=serve, daemon=True)
    t.start()
    for sig in (signal.SIGTERM, signal.SIGINT):
        signal.signal(sig, lambda *a: owner.stop())
    print(f"owner ready {args.socket}", flush=True)
    while not done.wait(0.2):
        pass
    t.join()
    owner.close()
    if err:
        print(f"owner failed: {err[0]}", file=sys.stderr, flush=True)
        return 1
    return 0


if __name__ == "__main__":
    sys.exit(main())
