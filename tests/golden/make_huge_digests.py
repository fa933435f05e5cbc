"""Write tests/golden/huge_digests.json: the oracle's outputs for whole pools of the 262,144-block
workload (64 pools x 65,536 events), stored as SHA-256 digests.

The oracle needs minutes per pool at this size, too slow for a test run, so this script (calling
only the oracle and the input generator) records what it computes once; the GPU test then compares
the kernel's outputs for the same pools against these digests.  Re-run it whenever the generator or
the contract changes:

    python tests/golden/make_huge_digests.py
"""
import hashlib
import json
import os
import sys
from concurrent.futures import ThreadPoolExecutor

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

import oracle  # noqa: E402
from paper_2605_24259_amd import tracegen as tg  # noqa: E402

POOLS = (0, 21, 42, 63)
OUT = os.path.join(os.path.dirname(os.path.abspath(__file__)), "huge_digests.json")


def sha(a) -> str:
    return hashlib.sha256(np.ascontiguousarray(a, dtype=np.int32).tobytes()).hexdigest()


def one(p):
    tr = tg.generate("huge", n_pools=1, first_pool=p)
    out, ptel, ctel, chk = oracle.replay(tr.desc, tr.events, tr.n_claim_slots)
    assert not chk.any(), oracle.check_names(int(chk[0]))
    return p, dict(events_sha256=sha(tr.events), n_events=int(tr.n_events),
                   n_claim_slots=int(tr.n_claim_slots), outcomes_sha256=sha(out),
                   pool_tel=[int(x) for x in ptel[0]], claim_tel_sha256=sha(ctel))


def main():
    with ThreadPoolExecutor(len(POOLS)) as ex:
        res = dict(ex.map(one, POOLS))
    doc = {"workload": "huge: 64 pools x 262144 usable blocks x 65536 events",
           "made_by": "tests/golden/make_huge_digests.py (oracle only)",
           "pools": {str(p): res[p] for p in POOLS}}
    with open(OUT, "w") as f:
        json.dump(doc, f, indent=1)
    print("wrote", OUT)


if __name__ == "__main__":
    main()
