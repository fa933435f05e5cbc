"""Helpers for the GPU parity tests: run the HIP path through the C ABI and the oracle on the same
seeded inputs, and report the first mismatching (pool, step, field)."""
from __future__ import annotations

import sys

import numpy as np

OUT_FIELDS = ("code|flags|n16", "id", "a", "b")


def gpu_replay(trace, flags=0):
    import paper_2605_24259_amd as rkc
    db = rkc.DeviceBatch.from_trace(trace, flags=flags)
    db.replay()
    return db.results()


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def compare_pools(trace, gpu, ora, pools=None, prefix_events=None, tel=True):
    """Assert bit-exact equality of outcomes, pool telemetry and claim telemetry for `pools`."""
    g_out, g_pt, g_ct = gpu
    o_out, o_pt, o_ct = ora[:3]
    eo, ne, so, ns = (trace.field(k) for k in ("event_offset", "n_events", "claim_slot_offset",
                                                "n_claim_slots"))
    errs = []
    for i in (range(trace.n_pools) if pools is None else pools):
        n = int(ne[i]) if prefix_events is None else min(int(ne[i]), prefix_events)
        a = g_out[eo[i]: eo[i] + n]
        b = o_out[eo[i]: eo[i] + n]
        if not np.array_equal(a, b):
            rows = np.nonzero((a != b).any(1))[0]
            t = int(rows[0])
            f = int(np.nonzero(a[t] != b[t])[0][0])
            errs.append(f"pool {i} (mode {int(trace.desc[i][1])}) step {t} field {OUT_FIELDS[f]}: "
                        f"gpu {a[t].tolist()} oracle {b[t].tolist()} event "
                        f"{trace.events[eo[i] + t].tolist()} ({len(rows)} rows differ)")
            continue
        if not tel:
            continue
        if not np.array_equal(g_pt[i], o_pt[i]):
            w = np.nonzero(g_pt[i] != o_pt[i])[0]
            errs.append(f"pool {i} pool-telemetry words {w.tolist()}: gpu {g_pt[i][w].tolist()} "
                        f"oracle {o_pt[i][w].tolist()}")
            continue
        ga, gb = g_ct[so[i]: so[i] + ns[i]], o_ct[so[i]: so[i] + ns[i]]
        if not np.array_equal(ga, gb):
            r = int(np.nonzero((ga != gb).any(1))[0][0])
            errs.append(f"pool {i} claim slot {r}: gpu {ga[r].tolist()} oracle {gb[r].tolist()}")
        if len(errs) >= 10:
            break
    assert not errs, "\n".join(errs)
