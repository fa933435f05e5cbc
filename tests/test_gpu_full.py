"""GPU parity on EVERY pool of the full-size workloads, against the oracle's digests.

tests/golden/make_full_digests.py replays each workload on the oracle once (CPU-minutes to
CPU-hours, calling only the oracle and the input generator) and stores, per chunk of consecutive
pools, SHA-256 digests of the oracle's outcomes, pool telemetry and claim telemetry, plus the
SHA-256 of the trace itself.  Here the same trace is drawn again, checked against its stored
digest, replayed by the HIP path through the C ABI in the launch configuration the benchmark times
(one batch of all pools), and every chunk's digests must be reproduced bit for bit.  A chunk that
differs is replayed by the oracle for an element-wise report of its first differences.
"""
import hashlib
import json
import os

import numpy as np
import pytest

from tests.gpu_util import compare_pools, gpu_replay, say

pytestmark = pytest.mark.gpu

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "full")
WORKLOADS = ("probe", "small", "zipf", "zipf_defer", "zipf_relax", "zipf_offload", "nested", "huge")


def sha(a) -> str:
    return hashlib.sha256(np.ascontiguousarray(a, dtype=np.int32).tobytes()).hexdigest()


def properties(trace, gpu):
    """Identities that hold for every pool at any size."""
    out, pt, ct = gpu
    U = trace.field("usable_blocks").astype(np.int64)
    ne = trace.field("n_events")
    # table-capacity bits (1, 2, 4) are contract outcomes the oracle reports too; anything else is a
    # descriptor or internal fault
    assert (pt[:, 31] & ~7 == 0).all(), "a descriptor or internal-fault status bit is set"
    assert (pt[:, :10].sum(1) + pt[:, 32] + pt[:, 36] == ne).all()
    assert (pt[:, 25] + pt[:, 26] + pt[:, 27] == U).all()
    assert (pt[:, 24] <= U).all() and (pt[:, 24] >= pt[:, 25]).all()
    assert (pt[:, 42:] == 0).all()
    code = out[:, 0] & 255
    ref = (code == 2) | (code == 3) | (code == 10)
    Ue = np.repeat(U, ne)
    assert (out[ref, 2].astype(np.int64) + out[ref, 3] > Ue[ref]).all()


@pytest.mark.parametrize("name", WORKLOADS)
def test_every_pool_matches_oracle_digests(oracle_mod, tg, name):
    path = os.path.join(GOLDEN, name + ".json")
    if not os.path.exists(path):
        pytest.skip(f"{path} not written yet (tests/golden/make_full_digests.py {name})")
    doc = json.load(open(path))
    trace = tg.generate(name)
    say(f"case full {name}: {trace.n_pools} pools, {trace.n_events} events, "
        f"{len(doc['chunks'])} digest chunks")
    assert (trace.n_pools, trace.n_events, trace.n_claim_slots) == \
        (doc["n_pools"], doc["n_events"], doc["n_claim_slots"])
    assert trace.sha256() == doc["trace_sha256"], \
        "the generator changed: re-run tests/golden/make_full_digests.py"
    gpu = gpu_replay(trace)
    out, pt, ct = gpu
    eo, so = trace.field("event_offset"), trace.field("claim_slot_offset")
    bad = []
    for c in doc["chunks"]:
        p0, n = c["first_pool"], c["n_pools"]
        e0, s0 = int(eo[p0]), int(so[p0])
        got = (sha(out[e0: e0 + c["n_events"]]), sha(pt[p0: p0 + n]),
               sha(ct[s0: s0 + c["n_claim_slots"]]))
        want = (c["outcomes_sha256"], c["pool_tel_sha256"], c["claim_tel_sha256"])
        if got != want:
            bad.append(c)
    if bad:
        c = bad[0]
        pools = list(range(c["first_pool"], c["first_pool"] + c["n_pools"]))
        say(f"{len(bad)} chunks differ; oracle replay of pools {pools[0]}..{pools[-1]}")
        ora = oracle_mod.replay(trace.desc, trace.events, trace.n_claim_slots, pools=pools,
                                threads=16)
        compare_pools(trace, gpu, ora, pools=pools)
        pytest.fail(f"{name}: {len(bad)} of {len(doc['chunks'])} chunks differ from the oracle's "
                    f"digests (first at pool {c['first_pool']})")
    properties(trace, gpu)
