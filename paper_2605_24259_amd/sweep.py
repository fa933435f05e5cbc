"""Capacity-sweep heatmap: outcome class of every (policy, resident R, active A, usable U) cell.

The sweep batch (tracegen.sweep) replays, per cell, a resident claim of R blocks followed by an
active prefill of A blocks on a pool of U usable blocks (§5.3 capacity-sweep figure).  This module
only decodes the replay's outcome stream into classes; all replay work happens in the kernels.
"""
from __future__ import annotations

import numpy as np

COEXIST = 0             # claim materialized, active admitted without resident victims
RESIDENT_LOST = 1       # active served by evicting resident blocks (EVICT_RESIDENT)
REFUSED_CLAIM = 2       # active refused, attributed to the resident claim
REFUSED_CAPACITY = 3    # active alone exceeds the pool
CLAIM_FAILED = 4        # the resident claim could not materialize (MATFAIL)
CLASS_NAMES = ("coexist", "resident_lost", "refused_claim", "refused_capacity", "claim_failed")


def heatmap(trace, outcomes: np.ndarray) -> np.ndarray:
    """Classes as an int8 array [mode, R, A, U] from the sweep's outcomes (int32 [2 * cells, 4])."""
    g = trace.meta["grid"]
    shape = (len(g["modes"]), len(g["residents"]), len(g["actives"]), len(g["usables"]))
    o = np.asarray(outcomes).reshape(-1, 2, 4)
    c0 = o[:, 0, 0] & 255
    c1 = o[:, 1, 0] & 255
    cls = np.full(c0.shape, -1, np.int8)
    cls[c1 == 0] = COEXIST
    cls[c1 == 1] = RESIDENT_LOST
    cls[c1 == 2] = REFUSED_CLAIM
    cls[c1 == 3] = REFUSED_CAPACITY
    cls[c0 == 4] = CLAIM_FAILED
    return cls.reshape(shape)
