"""Seeded synthetic traces for the batched resident-claim replay (input generation only).

The paper uses no public trace or dataset: its evidence comes from a 60/70/80 allocator probe
(§5.3 BlockPool probe table), the conformance traces L1-L7 (§5.4) and small MicroRuntime scenarios
(§5.2).  The five workloads here are synthetic stand-ins shaped like those probes:

  probe  4 pools x 80 blocks x 2 events: the 60-block resident claim and 70-block active prefill,
         replayed under the four pool policies (LRU, soft, no-admit, hard).
  small  4,096 pools x 80 blocks x 256 events, private prefills, a fresh chain per claim.
  zipf   65,536 pools x 2,048 blocks x 1,024 events, prefixes shared through 256 Zipf(1.1) chains.
  nested 16,384 pools x 16,384 blocks x 2,048 events, nested claims on 64 chains, demotion-heavy.
  huge   64 pools x 262,144 blocks x 65,536 events, the zipf mix scaled x128, <= 4,096 live claims.

This module draws events and lays out descriptors; it holds none of the replay arithmetic.
"""
from __future__ import annotations

import ctypes
import hashlib
import os
import subprocess
from dataclasses import dataclass, field

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "tracegen.c")
_LIB = os.path.join(_HERE, "libtracegen.so")
_lib = None

SEED0 = 260524259

EV_PREFILL, EV_EXTEND, EV_CLAIM, EV_FINISH, EV_RELEASE, EV_DEMOTE, EV_NOP, EV_RETRY = range(8)
MODE_RELAX = 16  # pool mode flag: the runtime demotes demotable hard claims to serve active requests
DESC_WORDS = 16  # int32 words per pool descriptor (64 bytes): event offset at 12:14, slot offset at 14:16
MODE_LRU, MODE_SOFT, MODE_NOADMIT, MODE_HARD = range(4)
MODE_NAMES = ("lru", "soft", "noadmit", "hard")


class GenParams(ctypes.Structure):
    _fields_ = [
        ("cfg_id", ctypes.c_int32),
        ("usable_blocks", ctypes.c_int32),
        ("n_events", ctypes.c_int32),
        ("mix", ctypes.c_int32 * 6),
        ("prefill_dist", ctypes.c_int32),
        ("prefill_min", ctypes.c_int32),
        ("prefill_max", ctypes.c_int32),
        ("chain_pick", ctypes.c_int32),
        ("n_chains", ctypes.c_int32),
        ("chain_len_min", ctypes.c_int32),
        ("chain_len_max", ctypes.c_int32),
        ("claim_len", ctypes.c_int32),
        ("claim_len_min", ctypes.c_int32),
        ("claim_len_max", ctypes.c_int32),
        ("claim_thresh", ctypes.c_int32),
        ("hard_permille", ctypes.c_int32),
        ("prio_max", ctypes.c_int32),
        ("dur_min", ctypes.c_int32),
        ("dur_max", ctypes.c_int32),
        ("extend_k", ctypes.c_int32),
        ("claim_cap", ctypes.c_int32),
        ("max_live_claims", ctypes.c_int32),
        ("max_live_requests", ctypes.c_int32),
        ("retry_permille", ctypes.c_int32),
        ("defer_limit", ctypes.c_int32),
        ("mode", ctypes.c_int32),
        ("demotable_permille", ctypes.c_int32),
        ("offloadable_permille", ctypes.c_int32),
        ("offload_blocks", ctypes.c_int32),
        ("zipf_s", ctypes.c_double),
        ("seed0", ctypes.c_uint64),
    ]


# Workload recipes (see the design notes for the reading behind every number that the workload
# description leaves open).  mix = per-mille of PREFILL, EXTEND, CLAIM, FINISH, RELEASE, DEMOTE.
CONFIGS = {
    "small": dict(cfg_id=2, n_pools=4096, usable_blocks=80, n_events=256,
                  mix=(400, 300, 150, 100, 50, 0), prefill_dist=0, prefill_min=1, prefill_max=96,
                  chain_pick=0, n_chains=0, chain_len_min=0, chain_len_max=0,
                  claim_len=1, claim_len_min=8, claim_len_max=64, claim_thresh=0,
                  hard_permille=500, prio_max=3, dur_min=16, dur_max=128, extend_k=1,
                  claim_cap=0, max_live_claims=64, max_live_requests=64),
    "zipf": dict(cfg_id=3, n_pools=65536, usable_blocks=2048, n_events=1024,
                 mix=(400, 300, 150, 100, 50, 0), prefill_dist=1, prefill_min=4, prefill_max=1536,
                 chain_pick=1, n_chains=256, chain_len_min=32, chain_len_max=512,
                 claim_len=0, claim_len_min=0, claim_len_max=0, claim_thresh=0,
                 hard_permille=250, prio_max=3, dur_min=64, dur_max=512, extend_k=1,
                 claim_cap=0, max_live_claims=64, max_live_requests=256),
    "nested": dict(cfg_id=4, n_pools=16384, usable_blocks=16384, n_events=2048,
                   mix=(300, 250, 200, 100, 50, 100), prefill_dist=1, prefill_min=16,
                   prefill_max=8192,
                   chain_pick=2, n_chains=64, chain_len_min=4096, chain_len_max=4096,
                   claim_len=2, claim_len_min=64, claim_len_max=4096, claim_thresh=1,
                   hard_permille=500, prio_max=3, dur_min=128, dur_max=1024, extend_k=152,
                   claim_cap=0, max_live_claims=256, max_live_requests=256),
    "huge": dict(cfg_id=5, n_pools=64, usable_blocks=262144, n_events=65536,
                 mix=(400, 300, 150, 100, 50, 0), prefill_dist=1, prefill_min=4,
                 prefill_max=196608,
                 chain_pick=1, n_chains=256, chain_len_min=4096, chain_len_max=65536,
                 claim_len=0, claim_len_min=0, claim_len_max=0, claim_thresh=0,
                 hard_permille=250, prio_max=3, dur_min=4096, dur_max=32768, extend_k=1,
                 claim_cap=4096, max_live_claims=4096, max_live_requests=16384),
    # The zipf pools under hard protection with active deferral: a prefill refused on behalf of
    # resident claims waits in the scheduler queue; 10% of the events are scheduler retries of the
    # oldest waiting request, which is deferred at most 4 times before a terminal refusal.
    "zipf_defer": dict(cfg_id=6, n_pools=65536, usable_blocks=2048, n_events=1024,
                       mix=(400, 300, 150, 100, 50, 0), prefill_dist=1, prefill_min=4,
                       prefill_max=1536, chain_pick=1, n_chains=256, chain_len_min=32,
                       chain_len_max=512, claim_len=0, claim_len_min=0, claim_len_max=0,
                       claim_thresh=0, hard_permille=500, prio_max=3, dur_min=64, dur_max=512,
                       extend_k=1, claim_cap=0, max_live_claims=64, max_live_requests=256,
                       mode=3, defer_limit=4, retry_permille=100),
    # The zipf pools under hard protection with runtime relaxation: half of the claims allow
    # demotion, and the runtime demotes blocking ones (lowest priority first) to serve an active
    # request before refusing it.
    "zipf_relax": dict(cfg_id=7, n_pools=65536, usable_blocks=2048, n_events=1024,
                       mix=(400, 300, 150, 100, 50, 0), prefill_dist=1, prefill_min=4,
                       prefill_max=1536, chain_pick=1, n_chains=256, chain_len_min=32,
                       chain_len_max=512, claim_len=0, claim_len_min=0, claim_len_max=0,
                       claim_thresh=0, hard_permille=500, prio_max=3, dur_min=64, dur_max=512,
                       extend_k=1, claim_cap=0, max_live_claims=64, max_live_requests=256,
                       mode=3 | MODE_RELAX, demotable_permille=500),
    # The same pools with a second tier of 1,024 blocks (half the GPU pool): half of the claims
    # allow offload and a quarter allow demotion; a blocking claim is offloaded when it allows it
    # and fits the tier's free room, else demoted when it allows it.
    "zipf_offload": dict(cfg_id=8, n_pools=65536, usable_blocks=2048, n_events=1024,
                         mix=(400, 300, 150, 100, 50, 0), prefill_dist=1, prefill_min=4,
                         prefill_max=1536, chain_pick=1, n_chains=256, chain_len_min=32,
                         chain_len_max=512, claim_len=0, claim_len_min=0, claim_len_max=0,
                         claim_thresh=0, hard_permille=500, prio_max=3, dur_min=64, dur_max=512,
                         extend_k=1, claim_cap=0, max_live_claims=64, max_live_requests=256,
                         mode=3 | MODE_RELAX, demotable_permille=250, offloadable_permille=500,
                         offload_blocks=1024),
}


def build(force: bool = True) -> str:
    global _lib
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", "-O2", "-std=c11", "-Wall", "-shared", "-fPIC", _SRC, "-o",
                               tmp, "-lm"])
        os.replace(tmp, _LIB)
        _lib = None
    return _LIB


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build(force=True)
        lib = ctypes.CDLL(_LIB)
        lib.rkc_tracegen.argtypes = [ctypes.POINTER(GenParams), ctypes.c_int64, ctypes.c_int32,
                                     ctypes.c_void_p, ctypes.c_void_p]
        lib.rkc_tracegen.restype = ctypes.c_int64
        _lib = lib
    return _lib


@dataclass
class Trace:
    """A batch of pools: 64-byte descriptors (int32 [P,16]) and 16-byte events (int32 [E,4])."""
    desc: np.ndarray
    events: np.ndarray
    n_claim_slots: int
    name: str = ""
    meta: dict = field(default_factory=dict)

    @property
    def n_pools(self) -> int:
        return int(self.desc.shape[0])

    @property
    def n_events(self) -> int:
        return int(self.events.shape[0])

    def field(self, name: str) -> np.ndarray:
        cols = {"usable_blocks": 0, "mode": 1, "n_events": 2, "n_chains": 3, "max_live_claims": 4,
                "max_live_requests": 5, "n_claim_slots": 6, "defer_limit": 7,
                "offload_blocks": 8}
        if name in cols:
            return self.desc[:, cols[name]]
        if name == "event_offset":
            return self.desc[:, 12:14].copy().view(np.int64)[:, 0]
        if name == "claim_slot_offset":
            return self.desc[:, 14:16].copy().view(np.int64)[:, 0]
        raise KeyError(name)

    def limits(self) -> dict:
        """Batch-level maxima (the host side of the replay launch needs them)."""
        if self.n_pools == 0:
            return dict(max_usable_blocks=0, max_events=0, max_chains=0, max_live_requests=0,
                        max_live_claims=0, max_claim_slots=0)
        return dict(max_usable_blocks=int(self.field("usable_blocks").max()),
                    max_events=int(self.field("n_events").max()),
                    max_chains=int(self.field("n_chains").max()),
                    max_live_requests=int(self.field("max_live_requests").max()),
                    max_live_claims=int(self.field("max_live_claims").max()),
                    max_claim_slots=int(self.field("n_claim_slots").max()))

    def subset(self, pools) -> "Trace":
        """A new batch holding only the given pools, re-laid out contiguously."""
        pools = [int(p) for p in pools]
        eo = self.field("event_offset")
        co = self.field("claim_slot_offset")
        ne = self.field("n_events")
        ns = self.field("n_claim_slots")
        evs, rows, e_acc, s_acc = [], [], 0, 0
        for p in pools:
            row = self.desc[p].copy()
            evs.append(self.events[eo[p]: eo[p] + ne[p]])
            row[12:14] = np.array([e_acc], np.int64).view(np.int32)
            row[14:16] = np.array([s_acc], np.int64).view(np.int32)
            rows.append(row)
            e_acc += int(ne[p])
            s_acc += int(ns[p])
        desc = np.stack(rows) if rows else np.zeros((0, DESC_WORDS), np.int32)
        events = np.concatenate(evs) if evs else np.zeros((0, 4), np.int32)
        t = Trace(desc, np.ascontiguousarray(events), s_acc, self.name + "[subset]", dict(self.meta))
        t.meta["source_pools"] = pools
        t.meta["source_slot_offsets"] = [int(co[p]) for p in pools]
        return t

    def prefix(self, pools, n_events: int) -> "Trace":
        """A new batch of the given pools, each cut to its first n_events events (claim slots cut to
        the CLAIM events kept).  Replay is causal, so the outcomes of a prefix equal the leading
        outcomes of the full pool."""
        sub = self.subset(pools)
        ne = sub.field("n_events")
        eo = sub.field("event_offset")
        evs, rows, e_acc, s_acc = [], [], 0, 0
        for j in range(sub.n_pools):
            k = int(min(ne[j], n_events))
            ev = sub.events[eo[j]: eo[j] + k]
            row = sub.desc[j].copy()
            n_sl = int(np.sum((ev[:, 0] & 15) == EV_CLAIM))
            row[2] = k
            row[6] = n_sl
            row[12:14] = np.array([e_acc], np.int64).view(np.int32)
            row[14:16] = np.array([s_acc], np.int64).view(np.int32)
            rows.append(row)
            evs.append(ev)
            e_acc += k
            s_acc += n_sl
        desc = np.stack(rows) if rows else np.zeros((0, DESC_WORDS), np.int32)
        events = np.concatenate(evs) if evs else np.zeros((0, 4), np.int32)
        return Trace(desc, np.ascontiguousarray(events), s_acc, self.name + "[prefix]", dict(sub.meta))

    def sha256(self) -> str:
        h = hashlib.sha256()
        h.update(np.ascontiguousarray(self.desc).tobytes())
        h.update(np.ascontiguousarray(self.events).tobytes())
        return h.hexdigest()


def make_desc(pools: list[dict], n_events: list[int], n_slots: list[int]) -> np.ndarray:
    desc = np.zeros((len(pools), DESC_WORDS), np.int32)
    e_acc = s_acc = 0
    for i, p in enumerate(pools):
        desc[i, 0] = p["usable_blocks"]
        desc[i, 1] = p["mode"]
        desc[i, 2] = n_events[i]
        desc[i, 3] = p.get("n_chains", 0)
        desc[i, 4] = p.get("max_live_claims", max(n_slots[i], 1))
        desc[i, 5] = p.get("max_live_requests", max(n_events[i], 1))
        desc[i, 6] = p.get("n_claim_slots", n_slots[i])
        desc[i, 7] = p.get("defer_limit", 0)
        desc[i, 8] = p.get("offload_blocks", 0)
        desc[i, 12:14] = np.array([e_acc], np.int64).view(np.int32)
        desc[i, 14:16] = np.array([s_acc], np.int64).view(np.int32)
        e_acc += n_events[i]
        s_acc += int(desc[i, 6])
    return desc


def ev(type_: int, w1: int = 0, w2: int = 0, w3: int = 0, hard: int = 0, prio: int = 0,
       dur: int = 0, demotable: int = 0, best_effort: int = 0, offloadable: int = 0) -> list[int]:
    """Encode one event (w0 = type | hard << 4 | prio << 5 | demotable << 7 | best_effort << 8 |
    offloadable << 9 | duration << 16)."""
    w0 = ((type_ & 15) | ((hard & 1) << 4) | ((prio & 3) << 5) | ((demotable & 1) << 7)
          | ((best_effort & 1) << 8) | ((offloadable & 1) << 9) | ((dur & 0xFFFF) << 16))
    if w0 >= 1 << 31:
        w0 -= 1 << 32
    w = [w0, w1, w2, w3]
    return [int(np.int64(x).astype(np.int32)) if -(1 << 31) <= x < (1 << 32) else x for x in w]


def prefill(S, c=-1, P=0):
    return ev(EV_PREFILL, S, c, P)


def extend(k, sel=0):
    return ev(EV_EXTEND, k, sel)


def claim(L, c, T=None, hard=0, prio=0, dur=0, demotable=0, best_effort=0, offloadable=0):
    return ev(EV_CLAIM, L, c, L if T is None else T, hard=hard, prio=prio, dur=dur,
              demotable=demotable, best_effort=best_effort, offloadable=offloadable)


def finish(sel=0):
    return ev(EV_FINISH, sel)


def release(sel=0):
    return ev(EV_RELEASE, sel)


def demote(sel=0):
    return ev(EV_DEMOTE, sel)


def nop():
    return ev(EV_NOP)


def retry():
    return ev(EV_RETRY)


def from_pools(pools: list[dict], name: str = "handmade") -> Trace:
    """Batch from explicit pools: each dict has usable_blocks, mode, events (list of 4-int lists),
    optional n_chains / max_live_claims / max_live_requests / n_claim_slots / defer_limit /
    offload_blocks."""
    evs = [np.asarray(p["events"], np.int64).reshape(-1, 4) for p in pools]
    n_ev = [int(e.shape[0]) for e in evs]
    n_sl = [int(np.sum((e[:, 0] & 15) == EV_CLAIM)) if e.size else 0 for e in evs]
    desc = make_desc(pools, n_ev, n_sl)
    events = (np.concatenate(evs) if evs else np.zeros((0, 4), np.int64)).astype(np.int64)
    events = ((events + (1 << 31)) % (1 << 32) - (1 << 31)).astype(np.int32)
    return Trace(desc, np.ascontiguousarray(events), int(desc[:, 6].sum()), name)


def probe(usable_blocks: int = 80, modes=(0, 1, 2, 3)) -> Trace:
    """The paper's 60/70/80 probe (§2.3, §5.3): claim 0 = resident claim of 60 blocks on chain 0
    (hard, priority 3, no expiry, threshold 60); event 1 = active prefill of 70 private blocks."""
    pools = [dict(usable_blocks=usable_blocks, mode=m, n_chains=2,
                  events=[claim(60, 0, 60, hard=1, prio=3), prefill(70, 1, 0)]) for m in modes]
    return from_pools(pools, "probe")


# Capacity sweep (§5.3 capacity-sweep figure, generalized): every combination of resident claim
# footprint R, active prefill size A, usable blocks U and pool policy is one pool replaying
#   t0: CLAIM(L = R, chain 0, T = R, hard, priority 3, no expiry), t1: PREFILL(A private blocks).
SWEEP_GRID = dict(residents=tuple(range(8, 257, 8)), actives=tuple(range(8, 257, 8)),
                  usables=tuple(range(16, 513, 16)), modes=(MODE_LRU, MODE_SOFT, MODE_NOADMIT, MODE_HARD))


def sweep(residents=SWEEP_GRID["residents"], actives=SWEEP_GRID["actives"], usables=SWEEP_GRID["usables"],
          modes=SWEEP_GRID["modes"]) -> Trace:
    """The capacity-sweep batch; pool index = ((mode_i * |R| + r_i) * |A| + a_i) * |U| + u_i."""
    m, r, a, u = np.meshgrid(np.asarray(modes), np.asarray(residents), np.asarray(actives),
                             np.asarray(usables), indexing="ij")
    m, r, a, u = (x.reshape(-1).astype(np.int64) for x in (m, r, a, u))
    n = m.size
    desc = np.zeros((n, DESC_WORDS), np.int32)
    desc[:, 0] = u
    desc[:, 1] = m
    desc[:, 2] = 2
    desc[:, 3] = 2
    desc[:, 4] = 1
    desc[:, 5] = 1
    desc[:, 6] = 1
    idx = np.arange(n, dtype=np.int64)
    desc[:, 12:14] = (2 * idx).view(np.int32).reshape(n, 2)
    desc[:, 14:16] = idx.view(np.int32).reshape(n, 2)
    ev = np.zeros((n, 2, 4), np.int64)
    ev[:, 0, 0] = EV_CLAIM | (1 << 4) | (3 << 5)
    ev[:, 0, 1] = r
    ev[:, 0, 2] = 0
    ev[:, 0, 3] = r
    ev[:, 1, 0] = EV_PREFILL
    ev[:, 1, 1] = a
    ev[:, 1, 2] = 1
    ev[:, 1, 3] = 0
    t = Trace(desc, np.ascontiguousarray(ev.reshape(-1, 4).astype(np.int32)), n, "sweep")
    t.meta["grid"] = dict(modes=tuple(modes), residents=tuple(residents), actives=tuple(actives),
                          usables=tuple(usables))
    return t


def generate(name: str, n_pools: int | None = None, first_pool: int = 0, **overrides) -> Trace:
    """Draw a synthetic workload (see CONFIGS).  n_pools/first_pool select a slice of its pools;
    pool i always gets the same events whatever slice it is drawn in."""
    if name == "probe":
        return probe()
    if name == "sweep":
        return sweep()
    cfg = dict(CONFIGS[name])
    cfg.update(overrides)
    total = cfg.pop("n_pools")
    if n_pools is None:
        n_pools = total - first_pool
    g = GenParams()
    g.mode = -1
    for k, v in cfg.items():
        if k == "mix":
            for i, x in enumerate(v):
                g.mix[i] = x
        else:
            setattr(g, k, v)
    g.zipf_s = 1.1
    g.seed0 = SEED0
    lib = _load()
    desc = np.zeros((n_pools, DESC_WORDS), np.int32)
    events = np.empty((n_pools * cfg["n_events"], 4), np.int32)
    slots = lib.rkc_tracegen(ctypes.byref(g), first_pool, n_pools, ctypes.c_void_p(desc.ctypes.data),
                             ctypes.c_void_p(events.ctypes.data))
    if slots < 0:
        raise ValueError("bad generator parameters")
    return Trace(desc, events, int(slots), name, dict(first_pool=first_pool, params=cfg))
