"""Write tests/golden/full/<workload>.json: the oracle's outputs for EVERY pool of a full-size
workload, stored as SHA-256 digests per chunk of consecutive pools, next to the SHA-256 of the
trace itself (descriptors and events) and the recipe it was drawn from.

A full oracle replay of these workloads takes CPU-minutes to CPU-hours, too slow for a test run, so
this script -- which calls only the oracle and the input generator, never the HIP library --
records what the oracle computes once.  The GPU tests replay the same trace and must reproduce
every chunk digest; a chunk that differs is then replayed by the oracle for an element-wise report.

Re-run it whenever the generator or the contract changes:

    python tests/golden/make_full_digests.py [--threads N] [workload ...]
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time
from concurrent.futures import ThreadPoolExecutor

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

import oracle  # noqa: E402
from paper_2605_24259_amd import tracegen as tg  # noqa: E402

OUT_DIR = os.path.join(os.path.dirname(os.path.abspath(__file__)), "full")

# pools per chunk: about a million events per chunk (one pool per chunk for the 262,144-block pools)
CHUNK_POOLS = {"probe": 4, "small": 4096, "zipf": 1024, "zipf_defer": 1024, "zipf_relax": 1024,
               "zipf_offload": 1024, "nested": 512, "huge": 1}
WORKLOADS = ("probe", "small", "zipf", "zipf_defer", "zipf_relax", "zipf_offload", "nested", "huge")


def sha(a) -> str:
    return hashlib.sha256(np.ascontiguousarray(a, dtype=np.int32).tobytes()).hexdigest()


def draw(name: str, first: int, n: int):
    if name == "probe":
        return tg.probe().subset(range(first, first + n))
    return tg.generate(name, n_pools=n, first_pool=first)


def chunk_digest(name: str, first: int, n: int) -> dict:
    tr = draw(name, first, n)
    out, ptel, ctel, chk = oracle.replay(tr.desc, tr.events, tr.n_claim_slots)
    bad = np.nonzero(chk)[0]
    assert bad.size == 0, f"{name} pool {first + int(bad[0])}: " + ", ".join(
        oracle.check_names(int(chk[bad[0]])))
    return dict(first_pool=first, n_pools=n, n_events=int(tr.n_events),
                n_claim_slots=int(tr.n_claim_slots), events_sha256=sha(tr.events),
                outcomes_sha256=sha(out), pool_tel_sha256=sha(ptel), claim_tel_sha256=sha(ctel))


def make(name: str, threads: int) -> str:
    t0 = time.time()
    full = tg.generate(name)
    trace_sha = full.sha256()
    n_pools, n_events, n_slots = full.n_pools, full.n_events, full.n_claim_slots
    del full
    step = CHUNK_POOLS[name]
    firsts = list(range(0, n_pools, step))
    # finished chunks are kept until the workload's file is written, so an interrupted run resumes
    part = os.path.join(OUT_DIR, ".partial", name)
    os.makedirs(part, exist_ok=True)
    done = [0]

    def one(first):
        cache = os.path.join(part, f"{first}.json")
        if os.path.exists(cache):
            d = json.load(open(cache))
        else:
            d = chunk_digest(name, first, min(step, n_pools - first))
            with open(cache + ".tmp", "w") as f:
                json.dump(d, f)
            os.replace(cache + ".tmp", cache)
        done[0] += 1
        print(f"{name}: chunk {done[0]}/{len(firsts)} (pools {first}..) {time.time() - t0:.0f} s",
              flush=True)
        return d

    with ThreadPoolExecutor(threads) as ex:
        chunks = list(ex.map(one, firsts))
    assert sum(c["n_events"] for c in chunks) == n_events
    assert sum(c["n_claim_slots"] for c in chunks) == n_slots
    if name == "probe":
        recipe = {"pools": "usable 80, policies LRU / soft / no-admit / hard",
                  "events": "CLAIM(chain 0, L 60, T 60, hard, prio 3); PREFILL(70 private)"}
    else:
        recipe = {k: (list(v) if isinstance(v, tuple) else v) for k, v in tg.CONFIGS[name].items()}
    doc = {"workload": name,
           "recipe": recipe,
           "seed0": int(tg.SEED0),
           "n_pools": n_pools, "n_events": n_events, "n_claim_slots": n_slots,
           "trace_sha256": trace_sha,
           "chunk_pools": step,
           "made_by": "tests/golden/make_full_digests.py (oracle and input generator only)",
           "chunks": chunks}
    os.makedirs(OUT_DIR, exist_ok=True)
    path = os.path.join(OUT_DIR, name + ".json")
    head = {k: v for k, v in doc.items() if k != "chunks"}
    text = json.dumps(head, indent=1)[:-2] + ',\n "chunks": [\n'
    text += ",\n".join("  " + json.dumps(c) for c in chunks) + "\n ]\n}\n"
    assert json.loads(text) == doc
    with open(path, "w") as f:
        f.write(text)
    for first in firsts:
        os.remove(os.path.join(part, f"{first}.json"))
    os.rmdir(part)
    print(f"wrote {path} ({time.time() - t0:.0f} s)", flush=True)
    return path


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--threads", type=int, default=max(1, (os.cpu_count() or 2) - 1))
    ap.add_argument("workloads", nargs="*", default=list(WORKLOADS))
    a = ap.parse_args()
    for name in a.workloads:
        make(name, a.threads)


if __name__ == "__main__":
    main()
