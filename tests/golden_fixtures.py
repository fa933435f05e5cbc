"""Parser and checker for the paper-cited fixtures in tests/golden/*.txt.

Each fixture file holds one or more ``[pool NAME]`` sections: pool parameters, an ``events:`` list
and an ``expect:`` list.  Expectations name an outcome (``tN``), the pool telemetry (``tel``) or a
claim slot (``claimK``) and give ``field=value`` pairs.  ``flags=a|b`` demands exactly that flag
set (``flags=`` demands none); ``shortfall`` is a + b - U, ``sum`` is a + b, ``tokens`` is 16 * b.
"""
from __future__ import annotations

import glob
import os

import numpy as np

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")

MODES = {"lru": 0, "soft": 1, "noadmit": 2, "hard": 3}
CODES = {"admit": 0, "evict_resident": 1, "refused_claim": 2, "refused_capacity": 3, "matfail": 4,
         "demoted": 5, "released": 6, "finished": 7, "noop": 8, "invalid": 9, "deferred": 10,
         "relaxed": 11}
FLAGS = {"expired": 1, "pred_fail": 2, "harm": 4, "post_release_loss": 8, "evict_unclaimed": 16,
         "noadmit_drop": 32, "lowered": 64, "shadow": 128}
TEL = {"victims": 10, "resident": 11, "post_release": 12, "dropped": 13, "hits": 14,
       "accepted": 15, "approx": 16, "shadow": 17, "rejected": 18, "harm": 19, "pred_fail": 20,
       "expired": 21, "demoted": 22, "released": 23, "peak_active": 24, "active": 25, "cached": 26,
       "free": 27, "protected": 28, "live_requests": 29, "live_claims": 30, "status": 31,
       "n_deferred": 32, "retry_served": 33, "retry_refused": 34, "queued": 35, "n_relaxed": 36,
       "runtime_demoted": 37, "off_claims": 38, "off_blocks": 39, "restored": 40, "t2_peak": 41,
       "n_admit": 0, "n_refused_claim": 2, "n_refused_capacity": 3}
DECISIONS = {"none": 0, "accepted": 1, "approx": 2, "shadow": 3, "rejected": 4}
STATES = {"submitted": 0, "observed": 1, "materialized": 2, "demoted": 3, "expired": 4,
          "released": 5, "harmed": 6, "rejected": 7}
CLAIM_FIELDS = {"id": 0, "accept": 2, "demote": 3, "expire": 4, "release": 5, "pred_fail": 6,
                "harm": 7, "blocked": 8, "lead_end": 9}


def _kv(tokens):
    out = {}
    for tok in tokens:
        k, _, v = tok.partition("=")
        out[k] = v
    return out


def parse(path):
    return parse_text(open(path).read(), os.path.basename(path))


def parse_text(text, name):
    pools = []
    cur = None
    section = None
    for raw in text.splitlines():
        line = raw.split("#", 1)[0].rstrip()
        if not line.strip():
            continue
        s = line.strip()
        if s.startswith("[pool"):
            cur = dict(name=s[5:-1].strip(), events=[], expect=[], file=name)
            pools.append(cur)
            section = None
        elif s == "events:":
            section = "events"
        elif s == "expect:":
            section = "expect"
        elif section == "events":
            kind, *rest = s.split()
            cur["events"].append((kind, _kv(rest)))
        elif section == "expect":
            what, *rest = s.split()
            cur["expect"].append((what, _kv(rest)))
        else:
            k, _, v = s.partition("=")
            cur[k.strip()] = v.strip()
    return pools


def all_fixtures():
    out = []
    for path in sorted(glob.glob(os.path.join(GOLDEN, "*.txt"))):
        out.extend(parse(path))
    return out


def to_trace(tg, fixtures):
    """Build one batch holding every fixture pool."""
    pools = []
    for f in fixtures:
        evs = []
        for kind, kv in f["events"]:
            g = lambda k, d=0: int(kv.get(k, d))
            if kind == "claim":
                evs.append(tg.claim(g("L"), g("c"), g("T", g("L")), hard=g("hard"), prio=g("prio"),
                                    dur=g("dur"), demotable=g("demotable"),
                                    best_effort=g("best_effort"), offloadable=g("offloadable")))
            elif kind == "prefill":
                evs.append(tg.prefill(g("S"), g("c", -1), g("P")))
            elif kind == "extend":
                evs.append(tg.extend(g("k"), g("sel")))
            elif kind == "finish":
                evs.append(tg.finish(g("sel")))
            elif kind == "release":
                evs.append(tg.release(g("sel")))
            elif kind == "demote":
                evs.append(tg.demote(g("sel")))
            elif kind == "nop":
                evs.append(tg.nop())
            elif kind == "retry":
                evs.append(tg.retry())
            else:
                raise ValueError(kind)
        mode = MODES[f["mode"]] | (tg.MODE_RELAX if int(f.get("relax", 0)) else 0)
        pools.append(dict(usable_blocks=int(f["usable"]), mode=mode,
                          n_chains=int(f.get("chains", 0)), events=evs,
                          defer_limit=int(f.get("defer_limit", 0)),
                          offload_blocks=int(f.get("offload", 0)),
                          **({"max_live_requests": int(f["max_requests"])} if "max_requests" in f
                             else {})))
    return tg.from_pools(pools, "golden")


def _flags(v):
    bits = 0
    for name in filter(None, v.split("|")):
        bits |= FLAGS[name]
    return bits


def check(fixtures, trace, outcomes, pool_tel, claim_tel):
    """Return a list of mismatch strings (empty when every expectation holds)."""
    errs = []
    eo = trace.field("event_offset")
    so = trace.field("claim_slot_offset")
    for i, f in enumerate(fixtures):
        U = int(f["usable"])
        tag = f"{f['file']}:{f['name']}"
        for what, kv in f["expect"]:
            if what.startswith("t") and what[1:].isdigit():
                t = int(what[1:])
                o = outcomes[eo[i] + t]
                w0 = int(np.uint32(o[0]))
                got = dict(code=w0 & 255, flags=(w0 >> 8) & 255, n16=w0 >> 16, id=int(o[1]),
                           a=int(o[2]), b=int(o[3]))
                got["shortfall"] = got["a"] + got["b"] - U
                got["sum"] = got["a"] + got["b"]
                got["tokens"] = 16 * got["b"]
                for k, v in kv.items():
                    want = CODES[v] if k == "code" else _flags(v) if k == "flags" else int(v)
                    if got[k] != want:
                        errs.append(f"{tag} {what}.{k}: got {got[k]}, want {want} ({v})")
            elif what == "tel":
                for k, v in kv.items():
                    if int(pool_tel[i][TEL[k]]) != int(v):
                        errs.append(f"{tag} tel.{k}: got {int(pool_tel[i][TEL[k]])}, want {v}")
            elif what.startswith("claim"):
                s = int(what[5:])
                w = claim_tel[so[i] + s]
                packed = int(w[1])
                got = dict(decision=packed & 15, state=(packed >> 4) & 15, hard=(packed >> 8) & 1,
                           prio=(packed >> 9) & 3, eff=(packed >> 11) & 3,
                           demotable=(packed >> 13) & 1, best_effort=(packed >> 14) & 1,
                           relaxed=(packed >> 15) & 1, offloadable=(packed >> 16) & 1)
                for k, idx in CLAIM_FIELDS.items():
                    got[k] = int(w[idx])
                for k, v in kv.items():
                    want = DECISIONS[v] if k == "decision" else STATES[v] if k == "state" else int(v)
                    if got[k] != want:
                        errs.append(f"{tag} {what}.{k}: got {got[k]}, want {want} ({v})")
            else:
                raise ValueError(what)
    return errs
