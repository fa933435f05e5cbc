"""Brute-force model of the resident-claim replay for tiny pools -- TEST INFRASTRUCTURE.

An independent, deliberately different formulation used to pin the C oracle on pools of at most
eight blocks.  Where the C oracle sorts candidates and walks the reuse index, this model:
  * chooses victims by enumerating every subset of the candidates and keeping the one subset whose
    largest key is below the smallest key left behind (and asserts that exactly one exists);
  * decides feasibility by searching for any subset of FREE and candidate blocks of the needed size;
  * attributes a refusal to claims exactly when the allocation would have been feasible had
    hard protection been ignored (the contract's reading of "protection changes the failure mode";
    §5.3 BlockPool probe);
  * evaluates a claim's predicate as set containment: positions 0..T-1 of its chain are all present
    in the reuse index (§3.1 useful resident value; §5.4 L6);
  * counts every quantity from explicit sets rather than counters;
  * keeps deferred requests (active deferral, §3.5) as a plain list whose first element is retried;
  * relaxes (§3.1 demotable; §3.5 relax resident claim) by trying ever longer prefixes of the
    demotion order on a copy of the claim states and recounting the available blocks as sets.
Only meant for tiny inputs: its cost is exponential in the pool size.
"""
from __future__ import annotations

import itertools

FREE, ACTIVE, CACHED = "free", "active", "cached"
LIVE = ("observed", "materialized", "demoted", "expired", "harmed")
STATE_CODE = {"submitted": 0, "observed": 1, "materialized": 2, "demoted": 3, "expired": 4,
              "released": 5, "harmed": 6, "rejected": 7}
DEC_CODE = {None: 0, "accepted": 1, "approx": 2, "shadow": 3, "rejected": 4}
CODES = {"admit": 0, "evict_resident": 1, "refused_claim": 2, "refused_capacity": 3,
         "matfail": 4, "demoted": 5, "released": 6, "finished": 7, "noop": 8, "invalid": 9,
         "deferred": 10, "relaxed": 11}
TEL_WORD = {name: code for name, code in CODES.items()}
TEL_WORD["deferred"] = 32
TEL_WORD["relaxed"] = 36
LRU, SOFT, NOADMIT, HARD = range(4)
MAXF = 1 << 24


def _s32(x: int) -> int:
    x &= 0xFFFFFFFF
    return x - (1 << 32) if x >= 1 << 31 else x


class Pool:
    def __init__(self, U, mode, n_chains, max_claims, max_reqs, n_slots, defer_limit=0, U2=0):
        self.relax_on = bool(mode & 16)
        self.U2, self.t2_used = U2, 0
        mode &= ~16
        self.U, self.mode, self.n_chains = U, mode, n_chains
        self.max_claims, self.max_reqs, self.n_slots = max_claims, max_reqs, n_slots
        self.defer_limit = defer_limit
        self.waiting = []        # deferred requests, oldest first
        self.blocks = [dict(state=FREE) for _ in range(U)]
        self.index = {}          # (chain, pos) -> block id
        self.reqs = {}           # id -> request dict
        self.claims = []         # slot order
        self.tel = [0] * 64
        self.peak = 0

    # -- sets -------------------------------------------------------------------------------
    def ids(self, state):
        return {i for i, b in enumerate(self.blocks) if b["state"] == state}

    def live_claims(self):
        return [q for q in self.claims if q.get("valid") and q["state"] in LIVE]

    def covering(self, i):
        b = self.blocks[i]
        if not b.get("reg"):
            return []
        return [q for q in self.live_claims() if q["chain"] == b["chain"] and b["pos"] < q["L"]]

    def protected(self, i):
        if self.mode != HARD or self.blocks[i]["state"] != CACHED:
            return False
        return any(q["state"] == "materialized" and q["eff"] == 2 for q in self.covering(i))

    def level(self, i):
        if self.mode not in (SOFT, HARD):
            return 0
        lv = [q["prio"] + 1 for q in self.covering(i)
              if (q["state"] == "materialized" and q["eff"] == 1) or q["state"] == "demoted"]
        return max(lv, default=0)

    def key(self, i):
        b = self.blocks[i]
        return (self.level(i), b["lu"], -b["pos"])

    def registered_positions(self, c):
        return {p for (ch, p) in self.index if ch == c}

    def prefix_len(self, c, upto):
        pos = self.registered_positions(c)
        n = 0
        while n < upto and n in pos:
            n += 1
        return n

    def pred(self, q):
        present = self.registered_positions(q["chain"])
        return all(p in present for p in range(q["T"]))

    # -- allocation ---------------------------------------------------------------------------
    def choose(self, need, hits, ignore_protection=False):
        """Return (feasible, victims, F, E) for `need` blocks with hit set `hits`."""
        free = self.ids(FREE)
        cand = {i for i in self.ids(CACHED) - hits if ignore_protection or not self.protected(i)}
        pool = sorted(free | cand)
        feasible = need <= len(pool) and any(True for _ in itertools.combinations(pool, need))
        if not feasible:
            return False, [], len(free), len(cand)
        m = max(0, need - len(free))
        if m == 0:
            return True, [], len(free), len(cand)
        keys = {i: self.key(i) for i in cand}
        found = []
        for combo in itertools.combinations(sorted(cand), m):
            rest = cand - set(combo)
            if not rest or max(keys[i] for i in combo) < min(keys[i] for i in rest):
                found.append(combo)
        assert len(found) == 1, "victim order is not a strict total order"
        return True, list(found[0]), len(free), len(cand)

    def take(self, need, victims):
        """Blocks for a new allocation: FREE blocks first (lowest ids), then the victims."""
        free = sorted(self.ids(FREE))
        out = free[: min(need, len(free))] + list(victims)
        stats = dict(victims=len(victims), resident=0, post=0, unclaimed=0, unreg=0)
        for i in victims:
            cov = [q for q in self.covering(i) if not q.get("offloaded")]
            if cov:
                stats["resident"] += 1
                if all(q["state"] in ("demoted", "expired") for q in cov):
                    stats["post"] += 1
            else:
                stats["unclaimed"] += 1
            b = self.blocks[i]
            if b.get("reg"):
                stats["unreg"] += 1
                del self.index[(b["chain"], b["pos"])]
        for i in out:
            self.blocks[i] = dict(state=FREE)
        return out, stats

    def refusal(self, need, hits):
        active = self.ids(ACTIVE)
        cached = self.ids(CACHED)
        hc = len(cached & hits)
        prot = {i for i in cached - hits if self.protected(i)}
        req = len(active) + hc + need
        ok_without, _, _, _ = self.choose(need, hits, ignore_protection=True)
        if ok_without:
            blocking = [q for q in self.live_claims()
                        if q["state"] == "materialized" and q["eff"] == 2
                        and any(self.blocks[self.index[(q["chain"], p)]]["state"] == CACHED
                                and self.index[(q["chain"], p)] not in hits
                                for p in range(q["L"]) if (q["chain"], p) in self.index)]
            for q in blocking:
                q["blocked"] += 1
            return "refused_claim", min(q["id"] for q in blocking), len(prot), req, len(blocking)
        return "refused_capacity", -1, len(prot), req, 0

    def _available(self, hits):
        free = self.ids(FREE)
        return len(free) + len({i for i in self.ids(CACHED) - hits if not self.protected(i)})

    def relax(self, t, need, hits):
        """Relax the shortest prefix of the blocking claims that allow demotion or offload, ordered
        by (priority, id), that lets `need` blocks be allocated: in that prefix a claim is offloaded
        when it allows it and its footprint fits the second tier's free room, else demoted when it
        allows it, else left alone.  Nothing changes when no prefix suffices."""
        if self.mode != HARD or not self.relax_on or need <= self._available(hits):
            return 0
        cands = []
        for q in self.live_claims():
            if q["state"] != "materialized" or q["eff"] != 2 or not (q["demotable"] or q["offloadable"]):
                continue
            blocks = [self.index[(q["chain"], p)] for p in range(q["L"]) if (q["chain"], p) in self.index]
            if any(self.blocks[i]["state"] == CACHED and i not in hits for i in blocks):
                cands.append(q)
        cands.sort(key=lambda q: (q["prio"], q["id"]))

        def actions(k):
            room, acts = self.U2 - self.t2_used, []
            for q in cands[:k]:
                if q["offloadable"] and q["L"] <= room:
                    acts.append((q, "offload"))
                    room -= q["L"]
                elif q["demotable"]:
                    acts.append((q, "demote"))
            return acts

        for k in range(1, len(cands) + 1):
            acts = actions(k)
            saved = [(q["state"], q["eff"]) for q, _ in acts]
            for q, a in acts:
                if a == "offload":
                    q["eff"] = 3
                else:
                    q["state"] = "demoted"
            ok = need <= self._available(hits)
            for (q, _), (st, eff) in zip(acts, saved):
                q["state"], q["eff"] = st, eff
            if ok:
                for q, a in acts:
                    q["relaxed"] = 1
                    if a == "offload":
                        q["eff"], q["offloaded"] = 3, 1
                        self.t2_used += q["L"]
                        self.tel[38] += 1
                        self.tel[39] += q["L"]
                    else:
                        q["state"], q["demote"] = "demoted", t
                        self.tel[37] += 1
                self.tel[41] = max(self.tel[41], self.t2_used)
                return len(acts)
        return 0

    def _restorable(self, c, h, P):
        e = max([q["L"] for q in self.live_claims() if q.get("offloaded") and q["chain"] == c],
                default=0)
        return max(0, min(P, e) - h)

    def live_request_ids(self):
        return sorted(r for r, q in self.reqs.items() if q["live"])

    # -- one event ------------------------------------------------------------------------------
    def step(self, t, e):
        w0 = e[0] & 0xFFFFFFFF
        typ, hard, prio, dur = w0 & 15, (w0 >> 4) & 1, (w0 >> 5) & 3, w0 >> 16
        flags, n16 = 0, None
        code, oid, a, b = "noop", -1, 0, 0
        expired = 0
        for q in self.claims:
            if q.get("valid") and q["dur"] > 0 and q["state"] in ("materialized", "demoted") \
                    and q["accept"] + q["dur"] <= t:
                q["state"], q["expire"] = "expired", t
                expired += 1
                if q.get("offloaded"):
                    self.t2_used -= q["L"]
                    q["offloaded"], q["eff"] = 0, 0
                    # the predicate held only through the dropped copy
                    if q["pred_fail"] < 0 and not self.pred(q):
                        q["pred_fail"] = t
                        flags |= 2
                        self.tel[20] += 1
        if expired:
            flags |= 1
            self.tel[21] += expired
        invalid = False
        slot = None
        live_req = self.live_request_ids()
        if typ == 0:
            S, c, P = e[1], e[2], e[3]
            if S < 1 or S > MAXF or P < 0 or P > S or (P > 0 and not 0 <= c < self.n_chains):
                invalid = True
            elif len(live_req) >= self.max_reqs:
                invalid = True
                self.tel[31] |= 1
        elif typ == 1:
            invalid = not 1 <= e[1] <= MAXF
        elif typ == 2:
            L, c, T = e[1], e[2], e[3]
            if len(self.claims) >= self.n_slots:
                invalid = True
                self.tel[31] |= 4
            else:
                slot = dict(id=t, valid=False, state="submitted", decision=None, accept=-1,
                            demote=-1, expire=-1, release=-1, pred_fail=-1, harm=-1, blocked=0)
                self.claims.append(slot)
                if L < 1 or L > MAXF or not 0 <= c < self.n_chains or T < 0 or T > L:
                    invalid = True
                elif len(self.live_claims()) >= self.max_claims:
                    invalid = True
                    self.tel[31] |= 2
        elif typ == 7:
            if self.waiting and len(live_req) >= self.max_reqs:
                invalid = True
                self.tel[31] |= 1
        elif typ > 7:
            invalid = True

        unreg = 0
        if invalid:
            code = "invalid"
        elif typ == 0:
            served, rec, fl, unreg = self._prefill(t, t, e[1], e[2], e[3])
            code, oid, a, b, n16 = rec
            flags |= fl
            if not served and code == "refused_claim" and self.defer_limit > 0 \
                    and len(self.waiting) < self.max_reqs:
                self.waiting.append(dict(id=t, S=e[1], c=e[2], P=e[3], times=1))
                code = "deferred"
        elif typ == 7:
            if not self.waiting:
                code = "noop"
            else:
                w = self.waiting[0]
                served, rec, fl, unreg = self._prefill(t, w["id"], w["S"], w["c"], w["P"])
                code, oid, a, b, n16 = rec
                flags |= fl
                if served:
                    self.waiting.pop(0)
                    self.tel[33] += 1
                elif code == "refused_claim" and w["times"] < self.defer_limit:
                    w["times"] += 1
                    code = "deferred"
                else:
                    self.waiting.pop(0)
                    self.tel[34] += 1
        elif typ == 1:
            if not live_req:
                code = "noop"
            else:
                rid = live_req[(e[2] & 0xFFFFFFFF) % len(live_req)]
                rq = self.reqs[rid]
                need = e[1]
                relaxed = self.relax(t, need, set())
                ok, victims, _, _ = self.choose(need, set())
                if not ok:
                    code, oid, a, b, n16 = self.refusal(need, set())
                else:
                    out, st = self.take(need, victims)
                    for j, i in enumerate(out):
                        self.blocks[i] = dict(state=ACTIVE, ref=1, lu=t, prod=rid, chain=None,
                                              pos=rq["len"] + j, reg=False)
                        rq["blocks"].append(i)
                    rq["len"] += need
                    code = "relaxed" if relaxed else "evict_resident" if st["resident"] else "admit"
                    oid, a, b = rid, st["resident"], len(self.ids(ACTIVE))
                    if relaxed:
                        n16 = relaxed
                    flags |= (8 if st["post"] else 0) | (16 if st["unclaimed"] else 0)
                    self._tel_victims(st)
                    unreg = st["unreg"]
        elif typ == 2:
            L, c, T = e[1], e[2], e[3]
            q = slot
            demq, beq, offq = (w0 >> 7) & 1, (w0 >> 8) & 1, (w0 >> 9) & 1
            observe = self.mode in (LRU, NOADMIT) or beq
            q.update(valid=True, chain=c, L=L, T=T, hard=hard, prio=prio, dur=dur, demotable=demq,
                     best_effort=beq, offloadable=offq, offloaded=0, relaxed=0,
                     eff=0 if beq else (2 if hard else 1) if self.mode == HARD
                     else (1 if self.mode == SOFT else 0))
            h = self.prefix_len(c, L)
            hits = {self.index[(c, p)] for p in range(h)}
            need = L - h
            ok, victims, F, E = self.choose(need, hits)
            if not ok:
                q["decision"] = "shadow" if observe else "rejected"
                q["state"] = "rejected"
                code, oid, a, b = "matfail", t, need, F + E
            else:
                out, st = self.take(need, victims)
                for i in hits:
                    self.blocks[i]["lu"] = t
                for j, i in enumerate(out):
                    self.blocks[i] = dict(state=CACHED, ref=0, lu=t, prod=-1, chain=c, pos=h + j,
                                          reg=True)
                    self.index[(c, h + j)] = i
                if observe:
                    q["decision"], q["state"] = "shadow", "observed"
                    flags |= 128
                elif self.mode == SOFT and hard:
                    q["decision"], q["state"] = "approx", "materialized"
                    flags |= 64
                else:
                    q["decision"], q["state"] = "accepted", "materialized"
                q["accept"] = t
                code = "evict_resident" if st["resident"] else "admit"
                oid, a, b = t, st["resident"], need
                flags |= (8 if st["post"] else 0) | (16 if st["unclaimed"] else 0)
                self._tel_victims(st)
                unreg = st["unreg"]
            self.tel[{"accepted": 15, "approx": 16, "shadow": 17, "rejected": 18}[q["decision"]]] += 1
        elif typ == 3:
            if not live_req:
                code = "noop"
            else:
                rid = live_req[(e[1] & 0xFFFFFFFF) % len(live_req)]
                rq = self.reqs[rid]
                turned = dropped = 0
                for i in rq["blocks"]:
                    bl = self.blocks[i]
                    bl["ref"] -= 1
                    bl["lu"] = t
                    if bl["ref"] == 0:
                        if self.mode == NOADMIT and bl["prod"] == rid:
                            self.blocks[i] = dict(state=FREE)
                            dropped += 1
                        else:
                            bl["state"] = CACHED
                            turned += 1
                rq["live"] = False
                code, oid, a, b = "finished", rid, turned, dropped
                if dropped:
                    flags |= 32
                self.tel[13] += dropped
        elif typ == 4:
            live = self.live_claims()
            if not live:
                code = "noop"
            else:
                q = live[(e[1] & 0xFFFFFFFF) % len(live)]
                q["state"], q["release"] = "released", t
                if q.get("offloaded"):
                    self.t2_used -= q["L"]
                    q["offloaded"] = 0
                code, oid = "released", q["id"]
                a, b = self.prefix_len(q["chain"], q["L"]), q["T"]
                self.tel[23] += 1
        elif typ == 5:
            cands = [q for q in self.claims if q.get("valid") and q["state"] == "materialized"
                     and q["hard"] and not q.get("offloaded")] if self.mode in (SOFT, HARD) else []
            if not cands:
                code = "noop"
            else:
                q = cands[(e[1] & 0xFFFFFFFF) % len(cands)]
                q["state"], q["demote"] = "demoted", t
                code, oid = "demoted", q["id"]
                a, b = self.prefix_len(q["chain"], q["L"]), q["T"]
                self.tel[22] += 1
        # the predicate sweep runs on every valid step (the oracle restricts it to steps where blocks
        # left the reuse index; this model does not, so it checks that restriction independently)
        if not invalid:
            for q in self.claims:
                if q.get("valid") and q["pred_fail"] < 0 and \
                        q["state"] in ("observed", "materialized", "demoted", "expired") \
                        and not q.get("offloaded") and not self.pred(q):
                    q["pred_fail"] = t
                    flags |= 2
                    self.tel[20] += 1
                    if q["state"] == "materialized":
                        q["state"], q["harm"] = "harmed", t
                        flags |= 4
                        self.tel[19] += 1
        if code in ("noop", "invalid"):
            oid, a, b = -1, 0, 0
        if n16 is None:
            n16 = expired
        n16 = min(n16, 65535)
        self.tel[TEL_WORD[code]] += 1
        self.peak = max(self.peak, len(self.ids(ACTIVE)))
        return [_s32(CODES[code] | (flags << 8) | (n16 << 16)), oid, a, b]

    def _prefill(self, t, rid, S, c, P):
        """Serve request rid (S blocks, chain c, shared prefix P) at step t.  Returns (served,
        (code, id, a, b, n16), flags, blocks that left the reuse index)."""
        h = self.prefix_len(c, P) if P > 0 else 0
        hits = {self.index[(c, p)] for p in range(h)}
        need = S - h
        relaxed = self.relax(t, need, hits)
        ok, victims, _, _ = self.choose(need, hits)
        if not ok:
            return False, self.refusal(need, hits), 0, 0
        out, st = self.take(need, victims)
        blks = []
        for i in sorted(hits):
            bl = self.blocks[i]
            bl["ref"] += 1
            bl["state"], bl["lu"] = ACTIVE, t
            blks.append(i)
        for j, i in enumerate(out):
            pos = h + j
            if pos < P:
                reg = self.mode != NOADMIT
                self.blocks[i] = dict(state=ACTIVE, ref=1, lu=t, prod=rid, chain=c, pos=pos, reg=reg)
                if reg:
                    assert (c, pos) not in self.index
                    self.index[(c, pos)] = i
            else:
                self.blocks[i] = dict(state=ACTIVE, ref=1, lu=t, prod=rid, chain=None, pos=pos,
                                      reg=False)
            blks.append(i)
        self.reqs[rid] = dict(live=True, blocks=blks, len=S)
        self._tel_victims(st)
        self.tel[14] += h
        if P > h:
            self.tel[40] += self._restorable(c, h, P)
        flags = (8 if st["post"] else 0) | (16 if st["unclaimed"] else 0)
        code = "relaxed" if relaxed else "evict_resident" if st["resident"] else "admit"
        return True, (code, rid, st["resident"], h, relaxed or None), flags, st["unreg"]

    def _tel_victims(self, st):
        self.tel[10] += st["victims"]
        self.tel[11] += st["resident"]
        self.tel[12] += st["post"]

    def finish_telemetry(self):
        tel = list(self.tel)
        tel[24] = self.peak
        tel[25] = len(self.ids(ACTIVE))
        tel[26] = len(self.ids(CACHED))
        tel[27] = len(self.ids(FREE))
        tel[28] = sum(self.protected(i) for i in range(self.U))
        tel[29] = len(self.live_request_ids())
        tel[30] = len(self.live_claims())
        tel[35] = len(self.waiting)
        slots = []
        for s in range(self.n_slots):
            if s >= len(self.claims):
                slots.append([-1, 0, -1, -1, -1, -1, -1, -1, 0, 0])
                continue
            q = self.claims[s]
            if not q["valid"]:
                slots.append([q["id"], 0, -1, -1, -1, -1, -1, -1, 0, 0])
                continue
            packed = DEC_CODE[q["decision"]] | (STATE_CODE[q["state"]] << 4) | (q["hard"] << 8) \
                | (q["prio"] << 9) | (q["eff"] << 11) | (q["demotable"] << 13) \
                | (q["best_effort"] << 14) | (q["relaxed"] << 15) | (q["offloadable"] << 16)
            slots.append([q["id"], packed, q["accept"], q["demote"], q["expire"], q["release"],
                          q["pred_fail"], q["harm"], q["blocked"],
                          self.prefix_len(q["chain"], q["L"])])
        return tel, slots


def replay_pool(desc_row, events):
    """Replay one pool: desc_row = 16 int32 descriptor words, events = list of 4-int lists."""
    U, mode, n_ev, n_chains, max_claims, max_reqs, n_slots, defer_limit, U2 = \
        [int(x) for x in desc_row[:9]]
    if U > 12:
        raise ValueError("the brute-force model enumerates subsets; use it on pools of <= 12 blocks")
    p = Pool(U, mode, n_chains, max_claims, max_reqs, n_slots, defer_limit, U2)
    outs = [p.step(t, [int(x) for x in events[t]]) for t in range(n_ev)]
    tel, slots = p.finish_telemetry()
    return outs, tel, slots
