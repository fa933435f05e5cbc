"""Scheduler-visible refusal records from the outcome stream, as JSON lines.

Every active refusal (and deferral) in the outcome stream carries the capacity proof of the §5.4
refusal record: the smallest blocking claim id and the number of blocking claims, protected resident
blocks (a) and active live blocks required (b).  This module renders those outcomes with the
record's field names (§5.4 canonical refusal event), adding the pool, the step and the usable
blocks of the pool it happened in: resident_plus_active_blocks = a + b, capacity_shortfall_blocks =
a + b - usable_blocks.  The outcome stream holds the smallest blocking id and the count, so
blocking_claim_ids lists every id only when a single claim blocks; otherwise the record names the
smallest one and the count.  Host-side decoding only: it reads outcome arrays already copied back.
"""
from __future__ import annotations

import json

import numpy as np

OC_REFUSED_CLAIM, OC_REFUSED_CAPACITY, OC_DEFERRED = 2, 3, 10
_EVENT = {OC_REFUSED_CLAIM: "active_request_refused", OC_REFUSED_CAPACITY: "active_request_refused",
          OC_DEFERRED: "active_request_deferred"}
_TYPES = {0: "prefill", 1: "extend", 7: "retry"}


def refusal_records(desc, events, outcomes, pools=None):
    """Records of every refused or deferred active event of the given pools (default: all), in pool
    and step order.  desc int32 [P,16] (64-byte descriptors), events and outcomes int32 [E,4]."""
    desc = np.asarray(desc, np.int32).reshape(-1, 16)
    events = np.asarray(events, np.int32).reshape(-1, 4)
    outcomes = np.asarray(outcomes, np.int32).reshape(-1, 4)
    offs = desc[:, 12:14].copy().view(np.int64)[:, 0]
    recs = []
    for p in (range(desc.shape[0]) if pools is None else pools):
        p = int(p)
        U, n = int(desc[p, 0]), int(desc[p, 2])
        o = outcomes[offs[p]: offs[p] + n]
        code = o[:, 0] & 255
        for t in np.nonzero((code == OC_REFUSED_CLAIM) | (code == OC_REFUSED_CAPACITY) | (code == OC_DEFERRED))[0]:
            w0, bid, a, b = (int(x) for x in o[t])
            c, n16 = w0 & 255, (w0 >> 16) & 0xFFFF
            ev = events[offs[p] + t]
            r = {"event": _EVENT[c], "pool": p, "step": int(t),
                 "event_type": _TYPES.get(int(ev[0]) & 15, "other"),
                 "refusal": "capacity" if c == OC_REFUSED_CAPACITY else "claim"}
            if c == OC_REFUSED_CAPACITY:
                r["blocking_claim_ids"] = []
            elif n16 == 1:
                r["blocking_claim_ids"] = [bid]
            else:
                r["first_blocking_claim_id"] = bid
                r["blocking_claim_count"] = n16
            r.update(protected_resident_blocks=a, active_live_blocks_required=b,
                     resident_plus_active_blocks=a + b, usable_blocks=U,
                     capacity_shortfall_blocks=a + b - U,
                     feasibility=("infeasible_preserve_resident_and_active" if c != OC_REFUSED_CAPACITY
                                  else "infeasible_active_alone"))
            recs.append(r)
    return recs


def write_jsonl(path, records) -> int:
    """Write one JSON object per line; returns the number of records written."""
    with open(path, "w") as f:
        for r in records:
            f.write(json.dumps(r) + "\n")
    return len(records)
