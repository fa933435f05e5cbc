"""Seeded random pools for invariant, brute-force and parity tests (input generation only)."""
from __future__ import annotations

import numpy as np


def random_pool(rng: np.random.Generator, U: int, mode: int, n_events: int, n_chains: int = 3,
                p_malformed: float = 0.03, tight_tables: bool = False, defer_limit: int = 0,
                p_retry: float = 0.15, relax: bool = False, offload: bool = False) -> dict:
    """One pool of arbitrary events, including malformed ones and table overflows.  With
    defer_limit > 0 the pool defers blocked prefills and a share p_retry of its events are RETRY
    (pools without deferral draw exactly the random numbers they always did).  With relax, claims
    are demotable or best-effort at random (extra draws only then); the caller sets the pool's
    relaxation flag."""
    from paper_2605_24259_amd import tracegen as tg
    evs = []
    for _ in range(n_events):
        r = rng.random()
        sel = int(rng.integers(0, 1 << 32))
        if defer_limit > 0 and rng.random() < p_retry:
            e = tg.retry()
        elif r < 0.26:
            S = int(rng.integers(1, U + 3))
            if rng.random() < 0.3:
                c, P = -1, 0
            else:
                c = int(rng.integers(0, n_chains))
                P = int(rng.integers(0, S + 1))
            e = tg.prefill(S, c, P)
        elif r < 0.40:
            e = tg.extend(int(rng.integers(1, 4)), sel)
        elif r < 0.62:
            L = int(rng.integers(1, U + 2))
            c = int(rng.integers(0, n_chains))
            T = int(rng.integers(0, L + 1))
            dur = 0 if rng.random() < 0.5 else int(rng.integers(1, 8))
            dem = be = off = 0
            if relax:
                dem = int(rng.random() < 0.6)
                be = int(rng.random() < 0.12)
            if offload:
                off = int(rng.random() < 0.6)
            e = tg.claim(L, c, T, hard=int(rng.integers(0, 2)), prio=int(rng.integers(0, 4)),
                         dur=dur, demotable=dem, best_effort=be, offloadable=off)
        elif r < 0.76:
            e = tg.finish(sel)
        elif r < 0.85:
            e = tg.release(sel)
        elif r < 0.96:
            e = tg.demote(sel)
        else:
            e = tg.nop()
        if rng.random() < p_malformed:
            kind = int(rng.integers(0, 6))
            e = list(e)
            if kind == 0:
                e[0] = (e[0] & ~15) | int(rng.integers(7, 16))    # RETRY or an unknown type
            elif kind == 1:
                e[1] = 0                                           # empty size / footprint
            elif kind == 2 and (e[0] & 15) == 0:
                e[3] = e[1] + 1                                    # P > S
            elif kind == 3 and (e[0] & 15) in (0, 2):
                e[2] = n_chains + 1                                # chain out of range
            elif kind == 4 and (e[0] & 15) == 2:
                e[3] = e[1] + 1                                    # T > L
            elif kind == 5:
                e[1] = -5
        evs.append([int(x) for x in e])
    pool = dict(usable_blocks=U, mode=mode, n_chains=n_chains, events=evs, defer_limit=defer_limit)
    if tight_tables:
        pool["max_live_requests"] = int(rng.integers(1, 4))
        pool["max_live_claims"] = int(rng.integers(1, 4))
        n_claims = sum(1 for e in evs if (e[0] & 15) == 2)
        pool["n_claim_slots"] = int(rng.integers(0, n_claims + 2))
    return pool


def random_batch(seed: int, n_pools: int, U_range=(2, 9), n_events=(1, 14), n_chains=3,
                 tight_every: int = 5, p_malformed: float = 0.03, caps=None, defer=False,
                 hard_share: float = 0.0, relax=False, offload=False):
    """caps = (live requests, live claims): table capacities of the pools that are not tight
    (default: one entry per PREFILL / CLAIM event, which never overflows).  defer: every pool
    defers, with a defer limit of 1..3.  hard_share: that share of the pools use hard protection
    (the only policy under which a refusal is attributed to claims), the rest cycle the policies.
    relax: every pool relaxes (mode flag) and claims are demotable / best-effort at random; with
    defer also set, pools both relax and defer.  offload: claims are offloadable at random and each
    pool gets a second tier of 0..U blocks."""
    from paper_2605_24259_amd import tracegen as tg
    rng = np.random.default_rng(seed)
    pools = []
    for i in range(n_pools):
        U = int(rng.integers(U_range[0], U_range[1]))
        ne = int(rng.integers(n_events[0], n_events[1] + 1))
        tight = tight_every > 0 and i % tight_every == tight_every - 1
        mode = i % 4
        dl = 0
        if defer:
            dl = int(rng.integers(1, 4))
        if defer or relax:
            if rng.random() < hard_share:
                mode = 3
        pool = random_pool(rng, U, mode, ne, n_chains=n_chains, p_malformed=p_malformed,
                           tight_tables=tight, defer_limit=dl, relax=relax, offload=offload)
        if relax:
            pool["mode"] = mode | tg.MODE_RELAX
        if offload:
            pool["offload_blocks"] = int(rng.integers(0, U + 1))
        if caps is not None and not tight:
            pool["max_live_requests"], pool["max_live_claims"] = caps
        pools.append(pool)
    return tg.from_pools(pools, f"random{seed}")


def many_claims_batch(seed: int, n_pools: int, n_events=(600, 1500), claim_cap: int = 256,
                      n_chains: int = 16, features: bool = True, claim_share: float = 0.50,
                      release_share: float = 0.05):
    """Pools that keep up to a few hundred claims live at once (small footprints on a few chains,
    few releases), with prefills large enough to be refused, relaxed and deferred, demotions,
    expiry and finishes: the claim tables span several 64-claim sets.  Policies cycle over the
    four; with features, every other hard-protection pool relaxes (demotable / offloadable claims
    and a second tier) and defers (RETRY events)."""
    from paper_2605_24259_amd import tracegen as tg
    rng = np.random.default_rng(seed)
    pools = []
    for i in range(n_pools):
        mode = i % 4
        ext = features and mode == 3 and (i // 4) % 2 == 1
        U = int(rng.integers(500, 4000))
        ne = int(rng.integers(n_events[0], n_events[1] + 1))
        evs = []
        for _ in range(ne):
            r = rng.random()
            sel = int(rng.integers(0, 1 << 31))
            if ext and r < 0.05:
                evs.append(tg.retry())
            elif r < claim_share:
                L = int(rng.integers(1, 24))
                dur = 0 if rng.random() < 0.6 else int(rng.integers(20, 600))
                evs.append(tg.claim(L, int(rng.integers(0, n_chains)), int(rng.integers(0, L + 1)),
                                    hard=int(rng.random() < 0.6), prio=int(rng.integers(0, 4)), dur=dur,
                                    demotable=int(ext and rng.random() < 0.5),
                                    best_effort=int(rng.random() < 0.05),
                                    offloadable=int(ext and rng.random() < 0.4)))
            elif r < claim_share + 0.18:
                S = int(rng.integers(1, U // 2 + 2))
                c = int(rng.integers(0, n_chains))
                evs.append(tg.prefill(S, c, int(rng.integers(0, min(S, 30) + 1))))
            elif r < claim_share + 0.28:
                evs.append(tg.extend(int(rng.integers(1, 60)), sel))
            elif r < claim_share + 0.38:
                evs.append(tg.finish(sel))
            elif r < claim_share + 0.38 + release_share:
                evs.append(tg.release(sel))
            else:
                evs.append(tg.demote(sel))
        pool = dict(usable_blocks=U, mode=mode | (tg.MODE_RELAX if ext else 0), n_chains=n_chains,
                    max_live_requests=256, max_live_claims=claim_cap, events=evs)
        if ext:
            pool["defer_limit"] = int(rng.integers(1, 4))
            pool["offload_blocks"] = int(rng.integers(0, U))
        pools.append(pool)
    return tg.from_pools(pools, f"many-claims{seed}")


def many_requests_batch(seed: int, n_pools: int, n_events=(700, 1200), n_chains: int = 200,
                        req_cap: int = 256):
    """Pools whose live-request lists grow past a few hundred entries (small served prefills, few
    finishes at first), with extends and finishes picking anywhere in the list, claims, and in every
    other hard-protection pool deferral with RETRY events (retried requests enter the list in id
    order); the request table fills and overflows.  Policies cycle over the four."""
    from paper_2605_24259_amd import tracegen as tg
    rng = np.random.default_rng(seed)
    pools = []
    for i in range(n_pools):
        mode = i % 4
        ext = mode == 3 and (i // 4) % 2 == 1
        U = int(rng.integers(600, 3000))
        ne = int(rng.integers(n_events[0], n_events[1] + 1))
        evs = []
        for k in range(ne):
            r = rng.random()
            sel = int(rng.integers(0, 1 << 32))
            # the list grows first, then shrinks
            pre, fin = (0.50, 0.04) if k < ne // 2 else (0.20, 0.34)
            if ext and r < 0.06:
                evs.append(tg.retry())
            elif r < pre:
                S = int(rng.integers(1, 9))
                if rng.random() < 0.3:
                    evs.append(tg.prefill(S, -1, 0))
                else:
                    evs.append(tg.prefill(S, int(rng.integers(0, n_chains)), int(rng.integers(0, S + 1))))
            elif r < pre + 0.12:
                evs.append(tg.extend(int(rng.integers(1, 5)), sel))
            elif r < pre + 0.12 + fin:
                evs.append(tg.finish(sel))
            elif r < pre + 0.12 + fin + 0.08:
                L = int(rng.integers(1, 40))
                evs.append(tg.claim(L, int(rng.integers(0, n_chains)), int(rng.integers(0, L + 1)),
                                    hard=int(rng.random() < 0.6), prio=int(rng.integers(0, 4)),
                                    dur=0 if rng.random() < 0.6 else int(rng.integers(20, 400))))
            elif r < pre + 0.12 + fin + 0.10:
                evs.append(tg.release(sel))
            else:
                evs.append(tg.nop())
        pool = dict(usable_blocks=U, mode=mode, n_chains=n_chains, max_live_requests=req_cap,
                    max_live_claims=64, events=evs)
        if ext:
            pool["defer_limit"] = int(rng.integers(1, 4))
        pools.append(pool)
    return tg.from_pools(pools, f"manyreq{seed}")
