"""Oracle against invariants, metamorphic relations and a brute-force model (no GPU needed).

Invariants (checked by the oracle after every step, reported in its check word):
I1 block counts; I2 no hard-protected victim; I3 no harm of a hard claim under hard protection;
I4 no acceptance or harm in LRU / no-admit pools; I6 refusal identity Pr + req > U and attribution
preconditions; I7 one block per (chain, pos); I8 lifecycle transitions; I9 strict eviction order;
registered positions of a chain always form a leading run; refcounts match live requests.
"""
import numpy as np
import pytest

from tests import randtrace


def _check_clean(oracle_mod, trace, **kw):
    out, ptel, ctel, chk = oracle_mod.replay(trace.desc, trace.events, trace.n_claim_slots, **kw)
    bad = np.nonzero(chk)[0]
    assert bad.size == 0, [(int(i), oracle_mod.check_names(int(chk[i]))) for i in bad[:5]]
    return out, ptel, ctel


@pytest.mark.parametrize("seed", [1, 2, 3])
def test_invariants_random_small(oracle_mod, seed):
    trace = randtrace.random_batch(seed, 600, U_range=(1, 12), n_events=(1, 40), n_chains=3)
    _check_clean(oracle_mod, trace)


@pytest.mark.parametrize("seed", [11, 12])
def test_invariants_random_medium(oracle_mod, seed):
    trace = randtrace.random_batch(seed, 120, U_range=(16, 160), n_events=(50, 200), n_chains=5,
                                   p_malformed=0.01)
    _check_clean(oracle_mod, trace)


def test_invariants_generated_workloads(oracle_mod, tg):
    for name, n in (("small", 64), ("zipf", 8)):
        trace = tg.generate(name, n_pools=n)
        _, ptel, _ = _check_clean(oracle_mod, trace, threads=8)
        assert (ptel[:, 31] == 0).all()


def test_invariant_accounting(oracle_mod):
    """Telemetry identities that hold for every pool: final FREE + ACTIVE + CACHED = U, outcome
    counts sum to the event count, resident >= post-release victims, harm <= predicate failures."""
    trace = randtrace.random_batch(7, 400, U_range=(1, 40), n_events=(1, 60), n_chains=4)
    out, ptel, ctel = _check_clean(oracle_mod, trace)
    U = trace.field("usable_blocks")
    ne = trace.field("n_events")
    assert (ptel[:, 25] + ptel[:, 26] + ptel[:, 27] == U).all()
    assert (ptel[:, :10].sum(1) == ne).all()
    assert (ptel[:, 11] >= ptel[:, 12]).all() and (ptel[:, 10] >= ptel[:, 11]).all()
    assert (ptel[:, 19] <= ptel[:, 20]).all()
    assert (ptel[:, 24] >= ptel[:, 25]).all() and (ptel[:, 24] <= U).all()
    # every refusal satisfies the infeasibility identity a + b > U (§3.4)
    eo = trace.field("event_offset")
    for i in range(trace.n_pools):
        o = out[eo[i]: eo[i] + ne[i]]
        code = o[:, 0] & 255
        ref = (code == 2) | (code == 3)
        assert (o[ref, 2].astype(np.int64) + o[ref, 3] > U[i]).all()
        # attributed refusals only in hard pools, with the active side alone fitting
        att = code == 2
        if att.any():
            assert trace.field("mode")[i] == 3
            assert (o[att, 3] <= U[i]).all() and (o[att, 2] > 0).all()
            assert ((o[att, 0].view(np.uint32) >> 16) >= 1).all()


def test_no_claims_policy_independent(oracle_mod, tg):
    """I11: with no CLAIM events, LRU, soft and hard pools give identical outputs."""
    rng = np.random.default_rng(5)
    pools = []
    for k in range(60):
        base = randtrace.random_pool(rng, int(rng.integers(4, 50)), 0, 60, n_chains=3)
        evs = [e for e in base["events"] if (e[0] & 15) != 2]
        for mode in (0, 1, 3):
            pools.append(dict(base, mode=mode, events=evs))
    trace = tg.from_pools(pools)
    out, ptel, ctel = _check_clean(oracle_mod, trace)
    eo = trace.field("event_offset")
    ne = trace.field("n_events")
    for k in range(60):
        rows = [out[eo[3 * k + j]: eo[3 * k + j] + ne[3 * k + j]] for j in range(3)]
        assert np.array_equal(rows[0], rows[1]) and np.array_equal(rows[0], rows[2])
        assert np.array_equal(ptel[3 * k], ptel[3 * k + 1]) and np.array_equal(ptel[3 * k], ptel[3 * k + 2])


def test_batch_composition_independent(oracle_mod):
    """I10: a pool's outputs do not depend on the other pools of the batch or on their order."""
    trace = randtrace.random_batch(21, 50, U_range=(2, 30), n_events=(1, 50))
    out, ptel, ctel = _check_clean(oracle_mod, trace)
    perm = np.random.default_rng(0).permutation(trace.n_pools)
    sub = trace.subset(perm)
    out2, ptel2, ctel2 = _check_clean(oracle_mod, sub)
    eo, ne, so, ns = (trace.field(k) for k in ("event_offset", "n_events", "claim_slot_offset",
                                                "n_claim_slots"))
    eo2, so2 = sub.field("event_offset"), sub.field("claim_slot_offset")
    for j, i in enumerate(perm):
        assert np.array_equal(out[eo[i]: eo[i] + ne[i]], out2[eo2[j]: eo2[j] + ne[i]])
        assert np.array_equal(ptel[i], ptel2[j])
        assert np.array_equal(ctel[so[i]: so[i] + ns[i]], ctel2[so2[j]: so2[j] + ns[i]])


def _brute_compare(oracle_mod, trace):
    from oracle import brute
    out, ptel, ctel = _check_clean(oracle_mod, trace)
    eo, ne, so, ns = (trace.field(k) for k in ("event_offset", "n_events", "claim_slot_offset",
                                                "n_claim_slots"))
    for i in range(trace.n_pools):
        bo, btel, bsl = brute.replay_pool(trace.desc[i], trace.events[eo[i]: eo[i] + ne[i]])
        got = out[eo[i]: eo[i] + ne[i]]
        if ne[i]:
            assert np.array_equal(np.asarray(bo, np.int64), got.astype(np.int64)), (i, bo, got.tolist())
        assert np.array_equal(np.asarray(btel), ptel[i]), (i, btel, ptel[i].tolist())
        if ns[i]:
            assert np.array_equal(np.asarray(bsl), ctel[so[i]: so[i] + ns[i]]), i


@pytest.mark.parametrize("seed", [101, 102, 103, 104])
def test_bruteforce_random(oracle_mod, seed):
    """Oracle == brute-force model on random pools of <= 8 blocks, all policies, incl. malformed
    events and table overflows."""
    trace = randtrace.random_batch(seed, 400, U_range=(1, 9), n_events=(1, 16), n_chains=3)
    _brute_compare(oracle_mod, trace)


def test_bruteforce_exhaustive_pairs(oracle_mod, tg):
    """Every ordered pair of events from a small alphabet, on a 4-block pool prepared with two
    claims and a live request, under all four policies."""
    prep = [tg.claim(2, 0, 2, hard=1, prio=1), tg.prefill(1, 1, 1), tg.claim(1, 1, 1, prio=2, dur=3)]
    alphabet = [tg.prefill(1), tg.prefill(2, 0, 2), tg.prefill(3, 1, 1), tg.prefill(4),
                tg.extend(1, 0), tg.extend(2, 1), tg.claim(2, 0, 1, hard=1), tg.claim(3, 1, 3, prio=3),
                tg.claim(1, 2, 1, hard=1, dur=1), tg.finish(0), tg.finish(1), tg.release(0),
                tg.release(1), tg.demote(0), tg.nop()]
    pools = []
    for x in alphabet:
        for y in alphabet:
            for mode in range(4):
                pools.append(dict(usable_blocks=4, mode=mode, n_chains=3, events=prep + [x, y]))
    trace = tg.from_pools(pools)
    _brute_compare(oracle_mod, trace)


@pytest.mark.parametrize("seed", [201, 202, 203])
def test_bruteforce_random_deferral(oracle_mod, seed):
    """Oracle == brute-force model on deferring pools (active deferral, §3.5): prefills blocked by
    hard claims are queued, RETRY events serve, defer again or refuse them, tables overflow."""
    trace = randtrace.random_batch(seed, 400, U_range=(1, 9), n_events=(8, 30), n_chains=2,
                                   defer=True, hard_share=0.8)
    _brute_compare(oracle_mod, trace)
    _, ptel, _ = _check_clean(oracle_mod, trace)
    assert ptel[:, 32].sum() > 50 and ptel[:, 33].sum() > 5 and ptel[:, 34].sum() > 5


def test_deferral_accounting(oracle_mod):
    """Identities of the deferral queue on every pool: each deferred request is served, refused or
    still queued at the end; DEFERRED outcomes appear only in hard-protection pools and carry a
    valid refusal record; outcome counts (incl. DEFERRED) sum to the event count."""
    trace = randtrace.random_batch(17, 400, U_range=(4, 60), n_events=(1, 120), n_chains=4,
                                   defer=True, hard_share=0.7, p_malformed=0.01)
    out, ptel, _ = _check_clean(oracle_mod, trace)
    U, ne, eo = trace.field("usable_blocks"), trace.field("n_events"), trace.field("event_offset")
    assert (ptel[:, :10].sum(1) + ptel[:, 32] == ne).all()
    assert (ptel[:, 36:] == 0).all()
    total_queued = 0
    for i in range(trace.n_pools):
        o = out[eo[i]: eo[i] + ne[i]]
        code = o[:, 0] & 255
        ev = trace.events[eo[i]: eo[i] + ne[i]]
        typ = ev[:, 0] & 15
        d = code == 10
        if d.any():
            assert trace.field("mode")[i] == 3
            assert (o[d, 2].astype(np.int64) + o[d, 3] > U[i]).all() and (o[d, 3] <= U[i]).all()
            assert (o[d, 2] > 0).all() and ((o[d, 0].view(np.uint32) >> 16) >= 1).all()
        # distinct requests that entered the queue: the PREFILLs whose outcome was DEFERRED
        entered = int(((typ == 0) & d).sum())
        assert entered == ptel[i, 33] + ptel[i, 34] + ptel[i, 35]
        # a RETRY never reports more DEFERRED outcomes for one request than the limit allows
        assert int(d.sum()) <= entered * int(trace.field("defer_limit")[i])
        total_queued += entered
    assert total_queued > 100


def test_deferral_off_is_plain_refusal(oracle_mod, tg):
    """defer_limit 0 reproduces the outputs of a pool without deferral, and RETRY is then a NOOP."""
    rng = np.random.default_rng(9)
    pools, plain = [], []
    for k in range(80):
        base = randtrace.random_pool(rng, int(rng.integers(4, 40)), 3, 50, n_chains=3,
                                     defer_limit=2)
        pools.append(dict(base, defer_limit=0))
        plain.append(dict(base, defer_limit=0,
                          events=[e if (e[0] & 15) != 7 else tg.nop() for e in base["events"]]))
    a = tg.from_pools(pools)
    b = tg.from_pools(plain)
    oa, pa, ca = _check_clean(oracle_mod, a)
    ob, pb, cb = _check_clean(oracle_mod, b)
    assert np.array_equal(oa, ob) and np.array_equal(pa, pb) and np.array_equal(ca, cb)


@pytest.mark.parametrize("seed", [301, 302, 303])
def test_bruteforce_random_relaxation(oracle_mod, seed):
    """Oracle == brute-force model on relaxing pools (§3.1 demotable / best_effort; §3.5 relax
    resident claim), alone and together with deferral."""
    trace = randtrace.random_batch(seed, 500, U_range=(1, 9), n_events=(8, 30), n_chains=2,
                                   relax=True, defer=seed == 303, hard_share=0.8)
    _brute_compare(oracle_mod, trace)
    _, ptel, _ = _check_clean(oracle_mod, trace)
    assert ptel[:, 36].sum() > 20 and ptel[:, 37].sum() >= ptel[:, 36].sum()


def test_relaxation_accounting(oracle_mod):
    """On relaxing pools: RELAXED outcomes only in hard pools, each demoting at least one claim;
    runtime demotions are counted in both the outcome and the claim records; no hard claim that is
    still materialized is ever harmed (I3 holds with relaxation)."""
    trace = randtrace.random_batch(19, 400, U_range=(4, 60), n_events=(1, 120), n_chains=4,
                                   relax=True, hard_share=0.7, p_malformed=0.01)
    out, ptel, ctel = _check_clean(oracle_mod, trace)
    ne, eo = trace.field("n_events"), trace.field("event_offset")
    so, ns = trace.field("claim_slot_offset"), trace.field("n_claim_slots")
    assert (ptel[:, :10].sum(1) + ptel[:, 32] + ptel[:, 36] == ne).all()
    total = 0
    for i in range(trace.n_pools):
        o = out[eo[i]: eo[i] + ne[i]]
        code = o[:, 0] & 255
        r = code == 11
        n16 = o[:, 0].view(np.uint32) >> 16
        if r.any():
            assert trace.field("mode")[i] & 15 == 3
            assert (n16[r] >= 1).all()
        assert int(n16[r].sum()) == int(ptel[i, 37])
        packed = ctel[so[i]: so[i] + ns[i], 1]
        assert int(((packed >> 15) & 1).sum()) == int(ptel[i, 37])
        total += int(r.sum())
    assert total > 100


@pytest.mark.parametrize("seed", [401, 402, 403])
def test_bruteforce_random_offload(oracle_mod, seed):
    """Oracle == brute-force model on relaxing pools with a second tier and offloadable claims
    (§3.1 offloadable; §3.5 offload resident), with demotable claims and deferral mixed in."""
    trace = randtrace.random_batch(seed, 500, U_range=(1, 9), n_events=(8, 30), n_chains=2,
                                   relax=True, offload=True, defer=seed == 403, hard_share=0.8)
    _brute_compare(oracle_mod, trace)
    _, ptel, _ = _check_clean(oracle_mod, trace)
    assert ptel[:, 38].sum() > 20 and ptel[:, 40].sum() > 0


def test_offload_accounting(oracle_mod):
    """On pools with a second tier: offloaded claims never fail their predicate while offloaded,
    second-tier use never exceeds the capacity, and relaxation counts add up."""
    trace = randtrace.random_batch(23, 400, U_range=(4, 60), n_events=(1, 120), n_chains=4,
                                   relax=True, offload=True, hard_share=0.7, p_malformed=0.01)
    out, ptel, ctel = _check_clean(oracle_mod, trace)
    U2 = trace.field("offload_blocks")
    assert (ptel[:, 41] <= U2).all()
    so, ns = trace.field("claim_slot_offset"), trace.field("n_claim_slots")
    eo, ne = trace.field("event_offset"), trace.field("n_events")
    for i in range(trace.n_pools):
        rec = ctel[so[i]: so[i] + ns[i]]
        packed = rec[:, 1]
        relaxed = int(((packed >> 15) & 1).sum())
        assert relaxed == int(ptel[i, 37] + ptel[i, 38])
        # claims still holding a copy at the end: offloadable, relaxed, never failed or harmed, and
        # no more of them than were offloaded
        held = ((packed >> 11) & 3) == 3
        assert (((packed[held] >> 16) & 1) == 1).all() and (((packed[held] >> 15) & 1) == 1).all()
        assert (rec[held, 6] == -1).all() and (rec[held, 7] == -1).all()
        assert int(held.sum()) <= int(ptel[i, 38])
        o = out[eo[i]: eo[i] + ne[i]]
        r = (o[:, 0] & 255) == 11
        assert int((o[r, 0].view(np.uint32) >> 16).sum()) == relaxed
    assert ptel[:, 38].sum() > 50
