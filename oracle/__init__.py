"""Reference oracle for the resident-KV-claim replay -- TEST INFRASTRUCTURE.

Only the test suite, ``__graft_entry__.smoke()`` and the CPU-baseline leg of ``bench.py`` may import
this package.  It wraps ``rkc_oracle.c``: a plain, slow, single-threaded C replay that keeps the pool
one block at a time and checks its structural invariants after every step.  It shares no code with
the HIP library.

Pins (what the oracle is checked against, in ``tests/``): the paper's 60/70/80 probe under the four
policies (§5.3 BlockPool probe table; §5.4 checks L1-L7 and C1, refusal record), demotion and expiry
before loss (§5.4 L4/L5), the capacity sweep boundary at 130 usable blocks (§5.3 figure caption), the
chunked-prefill accumulation 20/40/60/70 (§5.2 chunking table), the no-admit repeat 1120 vs 0 tokens
(§5.2 no-admit table), closed forms of the feasibility inequality (§3.4), structural invariants, and
a brute-force enumeration on pools of at most 8 blocks (``oracle/brute.py``).
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from concurrent.futures import ThreadPoolExecutor

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "rkc_oracle.c")
_LIB = os.path.join(_HERE, "librkc_oracle.so")
_lib = None

# invariant check bits reported per pool (see rkc_oracle.c)
CHECK_NAMES = {
    1: "I1 counts",
    2: "I2 hard-protected victim",
    4: "I3 hard claim harmed",
    8: "I4 accepted/harm in shadow pool",
    16: "I6 refusal identity",
    32: "I7 reuse index collision",
    64: "I8 illegal lifecycle transition",
    128: "I9 equal eviction keys",
    256: "prefix shape of registered positions",
    512: "refcount",
    1024: "allocation bookkeeping",
}


def build(force: bool = True) -> str:
    """Compile rkc_oracle.c with gcc into oracle/librkc_oracle.so."""
    global _lib
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", "-O2", "-std=c11", "-Wall", "-Wextra", "-shared", "-fPIC",
                               _SRC, "-o", tmp])
        os.replace(tmp, _LIB)
        _lib = None
    return _LIB


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build(force=True)
        lib = ctypes.CDLL(_LIB)
        p = ctypes.c_void_p
        lib.rkc_oracle_replay.argtypes = [p, ctypes.c_int32, ctypes.c_int32, p, p, p, p, p]
        lib.rkc_oracle_replay.restype = ctypes.c_int
        lib.rkc_oracle_predicate.argtypes = [p, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32]
        lib.rkc_oracle_predicate.restype = ctypes.c_int
        _lib = lib
    return _lib


def _ptr(a: np.ndarray) -> ctypes.c_void_p:
    return ctypes.c_void_p(a.ctypes.data)


def replay(desc: np.ndarray, events: np.ndarray, n_claim_slots_total: int, pools=None,
           threads: int = 1):
    """Replay pools of a batch on the CPU.

    desc: int32 [P, 16] (64-byte pool descriptors), events: int32 [E, 4].
    pools: iterable of pool indices to replay (default: all); other pools' outputs stay zero.
    Returns (outcomes int32 [E,4], pool_tel int32 [P,64], claim_tel int32 [C,10], check int32 [P]).
    """
    lib = _load()
    desc = np.ascontiguousarray(desc, dtype=np.int32).reshape(-1, 16)
    events = np.ascontiguousarray(events, dtype=np.int32).reshape(-1, 4)
    n_pools = desc.shape[0]
    out = np.zeros((events.shape[0], 4), np.int32)
    ptel = np.zeros((n_pools, 64), np.int32)
    ctel = np.zeros((max(int(n_claim_slots_total), 1), 10), np.int32)
    check = np.zeros(n_pools, np.int32)
    todo = list(range(n_pools)) if pools is None else [int(i) for i in pools]

    def run(chunk):
        for i in chunk:
            lib.rkc_oracle_replay(_ptr(desc), i, 1, _ptr(events), _ptr(out), _ptr(ptel), _ptr(ctel),
                                  _ptr(check))

    if threads <= 1 or len(todo) <= 1:
        run(todo)
    else:
        chunks = [todo[k::threads] for k in range(threads)]
        with ThreadPoolExecutor(threads) as ex:
            list(ex.map(run, chunks))
    return out, ptel, ctel[: int(n_claim_slots_total)], check


def predicate(registered_positions, npos: int, L: int, T: int) -> bool:
    """The oracle's materialization predicate on an explicit set of registered positions."""
    flags = np.zeros(max(npos, 1), np.uint8)
    for p in registered_positions:
        flags[p] = 1
    return bool(_load().rkc_oracle_predicate(_ptr(flags), npos, L, T))


def check_names(bits: int) -> list[str]:
    return [name for bit, name in CHECK_NAMES.items() if bits & bit]
