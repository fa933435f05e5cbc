"""GPU parity: the HIP replay (through the C ABI) against the CPU oracle, bit-exact.

Everything on the path is integer, so the bar is exact equality of every outcome word, every pool
telemetry word and every claim telemetry word.  Small cases compare every pool; the full-size
workloads run in the launch configuration the benchmark times and compare a sample of pools that
the oracle replays in seconds (for the 262,144-block pools, the leading events of sampled pools:
the replay is causal, so a prefix of a pool's outcomes is an exact sample).
"""
import numpy as np
import pytest

from tests import deferral_cases, relax_cases
from tests import golden_fixtures as gf
from tests import randtrace
from tests.gpu_util import compare_pools, gpu_replay, say

pytestmark = pytest.mark.gpu

ORACLE_THREADS = 16


def _both(oracle_mod, trace, pools=None):
    say(f"case {trace.name}: {trace.n_pools} pools, {trace.n_events} events")
    gpu = gpu_replay(trace)
    ora = oracle_mod.replay(trace.desc, trace.events, trace.n_claim_slots, pools=pools,
                            threads=ORACLE_THREADS)
    assert not ora[3].any(), "oracle invariant check failed"
    return gpu, ora


def test_probe(oracle_mod, tg):
    trace = tg.probe()
    gpu, ora = _both(oracle_mod, trace)
    compare_pools(trace, gpu, ora)
    codes = gpu[0][:, 0] & 255
    # LRU, soft, no-admit: the active prefill evicts 50 resident blocks; hard: attributed refusal
    assert list(codes[1::2]) == [1, 1, 1, 2]
    assert gpu[0][7].tolist()[1:] == [0, 60, 70]


def test_golden_fixtures(oracle_mod, tg):
    fx = gf.all_fixtures()
    trace = gf.to_trace(tg, fx)
    gpu, ora = _both(oracle_mod, trace)
    errs = gf.check(fx, trace, *gpu)
    assert not errs, "\n".join(errs)
    compare_pools(trace, gpu, ora)


def test_capacity_sweep(oracle_mod, tg):
    pools = [dict(usable_blocks=U, mode=m, n_chains=2,
                  events=[tg.claim(60, 0, 60, hard=1, prio=3), tg.prefill(70, 1, 0)])
             for m in range(4) for U in range(1, 201)]
    trace = tg.from_pools(pools, "capacity-sweep")
    gpu, ora = _both(oracle_mod, trace)
    compare_pools(trace, gpu, ora)


@pytest.mark.parametrize("seed", [1, 2, 3, 4])
def test_random_tiny(oracle_mod, seed):
    """Pools of <= 12 blocks with malformed events and table overflows, all policies."""
    trace = randtrace.random_batch(seed, 3000, U_range=(1, 13), n_events=(0, 40), n_chains=3)
    gpu, ora = _both(oracle_mod, trace)
    compare_pools(trace, gpu, ora)


@pytest.mark.parametrize("seed", [11, 12, 13])
def test_random_medium(oracle_mod, seed):
    """Several tiles of events per pool (up to 400 > 64-event prefetch), ragged tails, up to 9
    chains; tables of 256 requests and 64 claims (the compact kernel's limits) or tighter."""
    trace = randtrace.random_batch(seed, 400, U_range=(8, 300), n_events=(1, 400), n_chains=9,
                                   p_malformed=0.01, tight_every=7, caps=(256, 64))
    gpu, ora = _both(oracle_mod, trace)
    compare_pools(trace, gpu, ora)


@pytest.mark.parametrize("n_chains", [64, 65, 128, 129, 256])
def test_chain_groups(oracle_mod, n_chains):
    """Pools with many shared chains at the edges of the compact kernel's key groups (64 chains per
    lane-wide group: one, two or four groups), so every key group and chain record is in use."""
    trace = randtrace.random_batch(50 + n_chains, 300, U_range=(40, 400), n_events=(100, 500),
                                   n_chains=n_chains, p_malformed=0.01, tight_every=9, caps=(256, 64))
    assert trace.limits()["max_chains"] == n_chains
    gpu, ora = _both(oracle_mod, trace)
    compare_pools(trace, gpu, ora)


def test_edge_cases(oracle_mod, tg):
    """Empty pools, one-block pools, no chains, a maximal pool size, a pool whose events all fail."""
    pools = [
        dict(usable_blocks=1, mode=0, n_chains=0, events=[]),
        dict(usable_blocks=1, mode=3, n_chains=0, events=[tg.prefill(1), tg.extend(1), tg.finish()]),
        dict(usable_blocks=1, mode=1, n_chains=1, events=[tg.claim(1, 0, 1, hard=1), tg.prefill(1),
                                                         tg.release(), tg.prefill(1)]),
        dict(usable_blocks=(1 << 22), mode=3, n_chains=2,
             events=[tg.claim(60, 0, 60, hard=1, prio=3), tg.prefill(70, 1, 0),
                     tg.prefill(1 << 24, -1, 0), tg.extend(1 << 24), tg.finish(7)]),
        dict(usable_blocks=50, mode=2, n_chains=1,
             events=[tg.ev(9), tg.prefill(0), tg.claim(0, 0), tg.claim(5, 3), tg.claim(5, 0, 6),
                     tg.prefill(5, 7, 5), tg.extend(0), tg.nop()]),
        dict(usable_blocks=80, mode=3, n_chains=2, max_live_claims=0, max_live_requests=0,
             n_claim_slots=0, events=[tg.claim(10, 0), tg.prefill(5), tg.claim(10, 1)]),
    ]
    trace = tg.from_pools(pools, "edges")
    gpu, ora = _both(oracle_mod, trace)
    compare_pools(trace, gpu, ora)


def test_small_full(oracle_mod, tg):
    """4,096 pools x 80 blocks x 256 events: every pool compared."""
    trace = tg.generate("small")
    gpu, ora = _both(oracle_mod, trace)
    compare_pools(trace, gpu, ora)


def _sample(n_pools, k):
    idx = np.unique(np.linspace(0, n_pools - 1, k).astype(int))
    return [int(i) for i in idx]


def _properties(trace, gpu):
    """Identities that hold for every pool at any size."""
    out, pt, ct = gpu
    U = trace.field("usable_blocks").astype(np.int64)
    ne = trace.field("n_events")
    assert (pt[:, 31] & ~7 == 0).all(), "internal fault or descriptor status"
    assert (pt[:, :10].sum(1) + pt[:, 32] + pt[:, 36] == ne).all()
    assert (pt[:, 25] + pt[:, 26] + pt[:, 27] == U).all()
    assert (pt[:, 24] <= U).all() and (pt[:, 24] >= pt[:, 25]).all()
    assert (pt[:, 42:] == 0).all()
    code = out[:, 0] & 255
    ref = (code == 2) | (code == 3) | (code == 10)
    Ue = np.repeat(U, ne)
    assert (out[ref, 2].astype(np.int64) + out[ref, 3] > Ue[ref]).all()


def test_zipf_full_sampled(oracle_mod, tg):
    """65,536 pools x 2,048 blocks x 1,024 events (the benchmark workload)."""
    trace = tg.generate("zipf")
    pools = _sample(trace.n_pools, 96)
    gpu, ora = _both(oracle_mod, trace, pools=pools)
    compare_pools(trace, gpu, ora, pools=pools)
    _properties(trace, gpu)


def test_nested_full_sampled(oracle_mod, tg):
    """16,384 pools x 16,384 blocks x 2,048 events, nested claims, demotion-heavy."""
    trace = tg.generate("nested")
    pools = _sample(trace.n_pools, 6)
    gpu, ora = _both(oracle_mod, trace, pools=pools)
    compare_pools(trace, gpu, ora, pools=pools)
    _properties(trace, gpu)


def test_huge_full_prefix_sampled(oracle_mod, tg):
    """64 pools x 262,144 blocks x 65,536 events; the oracle replays the first 1,500 events of
    sampled pools and their outcomes must equal the GPU's first 1,500 outcomes; four whole pools
    must equal the oracle's stored digests."""
    trace = tg.generate("huge")
    say(f"case huge: {trace.n_pools} pools, {trace.n_events} events")
    gpu = gpu_replay(trace)
    _properties(trace, gpu)
    pools = [0, 21, 42, 63]
    sub = trace.subset(pools)
    pre = 1500
    d = sub.desc.copy()
    evs = []
    for j in range(len(pools)):
        d[j, 2] = pre
        d[j, 12:14] = np.array([j * pre], np.int64).view(np.int32)
        evs.append(sub.events[j * 65536: j * 65536 + pre])
    ora = oracle_mod.replay(d, np.concatenate(evs), sub.n_claim_slots, threads=4)
    assert not ora[3].any()
    eo = trace.field("event_offset")
    for j, p in enumerate(pools):
        a = gpu[0][eo[p]: eo[p] + pre]
        b = ora[0][j * pre: (j + 1) * pre]
        assert np.array_equal(a, b), (p, int(np.nonzero((a != b).any(1))[0][0]))
    # whole pools: the oracle's outputs for all 65,536 events of four pools, stored as digests by
    # tests/golden/make_huge_digests.py (minutes of oracle time per pool)
    import hashlib
    import json
    import os

    def sha(x):
        return hashlib.sha256(np.ascontiguousarray(x, dtype=np.int32).tobytes()).hexdigest()

    doc = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "huge_digests.json")))
    ne, so, ns = trace.field("n_events"), trace.field("claim_slot_offset"), trace.field("n_claim_slots")
    for key, dg in doc["pools"].items():
        p = int(key)
        assert sha(trace.events[eo[p]: eo[p] + ne[p]]) == dg["events_sha256"], \
            "the generator changed: re-run tests/golden/make_huge_digests.py"
        assert gpu[1][p].tolist() == dg["pool_tel"], p
        assert sha(gpu[0][eo[p]: eo[p] + ne[p]]) == dg["outcomes_sha256"], p
        assert sha(gpu[2][so[p]: so[p] + ns[p]]) == dg["claim_tel_sha256"], p


def test_batch_order_independent(oracle_mod, tg):
    """I10: reversing and subsetting the batch changes no pool's outputs."""
    trace = randtrace.random_batch(31, 500, U_range=(4, 120), n_events=(1, 150), n_chains=5)
    g1 = gpu_replay(trace)
    perm = list(range(trace.n_pools))[::-1][::2]
    sub = trace.subset(perm)
    g2 = gpu_replay(sub)
    eo, ne = trace.field("event_offset"), trace.field("n_events")
    eo2 = sub.field("event_offset")
    for j, i in enumerate(perm):
        assert np.array_equal(g1[0][eo[i]: eo[i] + ne[i]], g2[0][eo2[j]: eo2[j] + ne[i]])
        assert np.array_equal(g1[1][i], g2[1][j])


def test_repeat_deterministic(tg):
    trace = tg.generate("zipf", n_pools=2048)
    a = gpu_replay(trace)
    b = gpu_replay(trace)
    for x, y in zip(a, b):
        assert np.array_equal(x, y)


def test_abi_queries(oracle_mod, tg):
    import paper_2605_24259_amd as rkc
    trace = tg.generate("small", n_pools=64)
    db = rkc.DeviceBatch.from_trace(trace).replay()
    out, pt, ct = db.results()
    eo, so, ns = trace.field("event_offset"), trace.field("claim_slot_offset"), trace.field("n_claim_slots")
    for p in (0, 17, 63):
        st, o = db.query_outcomes(p, 3, 100)
        assert st == 0 and np.array_equal(o, out[eo[p] + 3: eo[p] + 103])
        st, ptel, ctel, n = db.query_telemetry(p, 1000)
        assert st == 0 and n == ns[p]
        assert np.array_equal(ptel, pt[p]) and np.array_equal(ctel, ct[so[p]: so[p] + ns[p]])
    assert db.query_outcomes(64, 0, 1)[0] == -3
    assert db.query_outcomes(0, 250, 10)[0] == -3
    assert db.query_outcomes(-1, 0, 1)[0] == -3


def test_descriptor_outside_batch_limits(tg):
    """A pool whose descriptor exceeds the launch's declared limits is not replayed: its outcomes
    are INVALID and its status carries the descriptor bit (an ABI fault, not a contract outcome)."""
    import paper_2605_24259_amd as rkc
    trace = tg.from_pools([dict(usable_blocks=80, mode=0, n_chains=2, events=[tg.prefill(5)] * 3),
                           dict(usable_blocks=80, mode=3, n_chains=2, events=[tg.prefill(5)] * 3)])
    lim = trace.limits()
    trace.desc[1, 0] = 81  # U above the batch maximum of 80
    db = rkc.DeviceBatch(trace.desc, trace.events, trace.n_claim_slots, lim).replay()
    out, pt, ct = db.results()
    assert (out[:3, 0] & 255 == 0).all()
    assert (out[3:, 0] & 255 == 9).all() and pt[1, 31] == 256 and pt[1, 9] == 3
    assert db.query_telemetry(1, 0)[0] == -7


@pytest.mark.parametrize("flags", [0, 1], ids=["compact", "general"])
def test_descriptor_offsets_outside_batch(tg, flags):
    """A descriptor whose event or claim-slot offset leaves the batch's arrays: the kernel writes
    nothing of that pool but its telemetry (descriptor status), and the queries refuse to copy
    from outside the arrays instead of reading past them."""
    import paper_2605_24259_amd as rkc
    ev = [tg.claim(10, 0, 10), tg.prefill(5), tg.finish()]
    trace = tg.from_pools([dict(usable_blocks=80, mode=3, n_chains=2, events=ev),
                           dict(usable_blocks=80, mode=3, n_chains=2, events=ev),
                           dict(usable_blocks=80, mode=3, n_chains=2, events=ev)])
    lim = trace.limits()
    trace.desc[1, 12:14] = np.array([trace.n_events + 1000], np.int64).view(np.int32)
    trace.desc[2, 14:16] = np.array([trace.n_claim_slots + 7], np.int64).view(np.int32)
    db = rkc.DeviceBatch(trace.desc, trace.events, trace.n_claim_slots, lim, flags=flags).replay()
    out, pt, ct = db.results()
    assert pt[0, 31] == 0 and pt[1, 31] == 256 and pt[2, 31] == 256
    assert db.query_outcomes(0, 0, 3)[0] == 0
    assert db.query_outcomes(1, 0, 1)[0] == -3
    assert db.query_outcomes(2, 0, 3)[0] == -7  # events in range, status set
    assert db.query_telemetry(1, 1)[0] == -7     # slots in range, status set
    assert db.query_telemetry(2, 1)[0] == -3


@pytest.mark.parametrize("variant", ["narrow", "wide", "wide_global_lists",
                                     "global_lists_small_request_table"])
def test_storage_layouts_agree(oracle_mod, tg, variant):
    """The same pools replayed with 16-bit LDS state, 32-bit LDS state and 32-bit state with the
    lists in global scratch (chosen by the batch's declared limits) match the oracle exactly.  The
    last variant keeps the lists in global scratch with a live-request table of at most 6 entries,
    so the request list's gap closing from both sides wraps back to the start of its arrays."""
    import paper_2605_24259_amd as rkc
    trace = randtrace.random_batch(41, 600, U_range=(2, 200), n_events=(1, 200), n_chains=7,
                                   tight_every=9)
    if variant == "global_lists_small_request_table":
        _small_request_tables(trace)
    lim = dict(trace.limits())
    if variant == "wide":
        lim["max_usable_blocks"] = 40000          # above the 16-bit bound
    elif variant == "wide_global_lists":
        lim["max_usable_blocks"] = 40000
        lim["max_live_requests"] = 20000          # lists no longer fit in LDS
        lim["max_live_claims"] = 4096
    else:
        lim["max_usable_blocks"] = 40000
        lim["max_live_claims"] = 8192             # the claim list no longer fits in LDS
    say(f"case layouts/{variant}")
    gpu = rkc.DeviceBatch(trace.desc, trace.events, trace.n_claim_slots, lim).replay().results()
    ora = oracle_mod.replay(trace.desc, trace.events, trace.n_claim_slots, threads=ORACLE_THREADS)
    compare_pools(trace, gpu, ora)


def _small_request_tables(trace):
    """Cap every pool's live-request table at 6 entries (descriptor field 5)."""
    trace.desc[:, 5] = np.minimum(trace.desc[:, 5], 6)


@pytest.mark.parametrize("case", ["small", "random"])
def test_general_kernel_on_compact_batches(oracle_mod, tg, case):
    """Batches that the compact kernel serves, replayed with the general kernel forced by the batch
    flag: both kernels match the oracle on the same inputs."""
    import paper_2605_24259_amd as rkc
    if case == "small":
        trace = tg.generate("small", n_pools=512)
    else:
        trace = randtrace.random_batch(21, 600, U_range=(1, 120), n_events=(0, 300), n_chains=9,
                                       p_malformed=0.01, tight_every=5, caps=(256, 64))
    say(f"case general-kernel/{case}")
    ora = oracle_mod.replay(trace.desc, trace.events, trace.n_claim_slots, threads=ORACLE_THREADS)
    assert not ora[3].any()
    gen = gpu_replay(trace, flags=rkc.FLAG_GENERAL_KERNEL)
    compare_pools(trace, gen, ora)
    lean = gpu_replay(trace)
    compare_pools(trace, lean, ora)


# ---- active deferral: both kernels ------------------------------------------------------------
KERNELS = ["compact", "general"]


def _kflags(kernel):
    import paper_2605_24259_amd as rkc
    return rkc.FLAG_GENERAL_KERNEL if kernel == "general" else 0


def _both_kernel(oracle_mod, trace, kernel, pools=None):
    say(f"case {trace.name} ({kernel} kernel): {trace.n_pools} pools, {trace.n_events} events")
    gpu = gpu_replay(trace, flags=_kflags(kernel))
    ora = oracle_mod.replay(trace.desc, trace.events, trace.n_claim_slots, pools=pools,
                            threads=ORACLE_THREADS)
    assert not ora[3].any(), "oracle invariant check failed"
    return gpu, ora


@pytest.mark.parametrize("kernel", KERNELS)
def test_deferral_fixtures(oracle_mod, tg, kernel):
    """The paper's live scheduler run (defer once, then a terminal refusal) and the hand-derived
    deferral cases: the expected values and the oracle, on both kernels."""
    fx = [f for f in gf.all_fixtures() if f["file"].startswith("live_scheduler")]
    fx += deferral_cases.fixtures()
    trace = gf.to_trace(tg, fx)
    gpu, ora = _both_kernel(oracle_mod, trace, kernel)
    errs = gf.check(fx, trace, *gpu)
    assert not errs, "\n".join(errs)
    compare_pools(trace, gpu, ora)


@pytest.mark.parametrize("kernel", KERNELS)
@pytest.mark.parametrize("seed", [51, 52])
def test_random_deferral_tiny(oracle_mod, kernel, seed):
    """Deferring pools of <= 12 blocks (mostly hard protection), RETRY events, tight tables
    (queue rings of 1-3 entries wrap), malformed events."""
    trace = randtrace.random_batch(seed, 3000, U_range=(1, 13), n_events=(0, 40), n_chains=3,
                                   defer=True, hard_share=0.8)
    gpu, ora = _both_kernel(oracle_mod, trace, kernel)
    compare_pools(trace, gpu, ora)
    assert gpu[1][:, 32].sum() > 200 and gpu[1][:, 33].sum() > 20


@pytest.mark.parametrize("kernel", KERNELS)
def test_random_deferral_medium(oracle_mod, kernel):
    """Deferring pools up to 300 blocks and 400 events (several 64-event tiles), tables of 256
    requests and 64 claims or tighter: retried requests are inserted into long live lists."""
    trace = randtrace.random_batch(61, 400, U_range=(8, 300), n_events=(1, 400), n_chains=9,
                                   p_malformed=0.01, tight_every=7, caps=(256, 64), defer=True,
                                   hard_share=0.8)
    gpu, ora = _both_kernel(oracle_mod, trace, kernel)
    compare_pools(trace, gpu, ora)
    assert gpu[1][:, 33].sum() > 50


@pytest.mark.parametrize("seed,kw", [
    (201, {}),
    (202, dict(claim_share=0.30, release_share=0.22, n_events=(1500, 3000))),
    (203, dict(features=False, claim_cap=130, claim_share=0.35, release_share=0.15)),
])
def test_claim_sets(oracle_mod, seed, kw):
    """The compact kernel with four 64-claim sets (live claims up to 256 on up to 64 chains, as in
    the nested workload): tables that fill and overflow, releases that close gaps across sets,
    demotions picked across sets, relaxation and offload picking over every set, deferral; against
    the oracle and the general kernel on the same inputs."""
    import paper_2605_24259_amd as rkc
    trace = randtrace.many_claims_batch(seed, 256, **kw)
    gpu, ora = _both(oracle_mod, trace)
    compare_pools(trace, gpu, ora)
    assert gpu[1][:, 30].max() > min(192, kw.get("claim_cap", 256) - 8)  # claims in the last set
    gen = gpu_replay(trace, flags=rkc.FLAG_GENERAL_KERNEL)
    compare_pools(trace, gen, ora)


@pytest.mark.parametrize("seed", [5, 6])
def test_request_list_past_lds(oracle_mod, seed):
    """Live-request lists of up to 256 entries, of which the compact kernel keeps the first 128 in
    LDS and the rest in global scratch: lists that grow past that split, fill the table and shrink
    back below it, with extends and finishes picking anywhere in them and retried requests entering
    in id order; against the oracle and the general kernel on the same inputs."""
    import paper_2605_24259_amd as rkc
    trace = randtrace.many_requests_batch(seed, 256)
    gpu, ora = _both(oracle_mod, trace)
    compare_pools(trace, gpu, ora)
    live = ora[1][:, 29]
    assert (live > 128).any() and (live < 128).any()
    assert (ora[1][:, 31] & 1).any()  # RKC_PS_REQUEST_TABLE: some lists reached the capacity
    gen = gpu_replay(trace, flags=rkc.FLAG_GENERAL_KERNEL)
    compare_pools(trace, gen, ora)


def _edge_selectors(n):
    """u32 selectors at the edges of `sel mod n`: multiples of n (largest one below 2^32
    included), their neighbours, 0 and 2^32 - 1."""
    top = (2**32 - 1) // n * n
    return sorted(x for x in {0, 1, n - 1, n, n + 1, 2 * n, top - n, top - 1, top, 2**32 - 1}
                  if 0 <= x < 2**32)


def test_selector_edges(oracle_mod, tg):
    """Selector arithmetic (the target is the (sel mod count)-th live request or claim) at the edges
    of the u32 range and at exact multiples of the count, for every count up to 256 live requests
    and claims; both kernels against the oracle."""
    import paper_2605_24259_amd as rkc
    pools = []
    for mode in (1, 3):
        ev = []
        for p in range(1, 257):
            ev.append(tg.prefill(1))
            for sel in _edge_selectors(p)[:: 3 if p > 16 else 1]:
                ev.append(tg.extend(1, sel))
        for n in range(256, 0, -1):
            ev.append(tg.finish(_edge_selectors(n)[n % 10 % len(_edge_selectors(n))]))
        pools.append(dict(usable_blocks=30000, mode=mode, n_chains=1, max_live_requests=256,
                          max_live_claims=256, events=ev))
        ev = []
        for p in range(1, 257):
            ev.append(tg.claim(1, 0, 1, hard=1))
            if p % 7 == 0:
                ev.append(tg.demote(_edge_selectors(p)[p % 10 % len(_edge_selectors(p))]))
        for n in range(256, 0, -1):
            ev.append(tg.release(_edge_selectors(n)[(n // 3) % len(_edge_selectors(n))]))
        pools.append(dict(usable_blocks=30000, mode=mode, n_chains=1, max_live_requests=256,
                          max_live_claims=256, events=ev))
    trace = tg.from_pools(pools, "selector-edges")
    gpu, ora = _both(oracle_mod, trace)
    compare_pools(trace, gpu, ora)
    compare_pools(trace, gpu_replay(trace, flags=rkc.FLAG_GENERAL_KERNEL), ora)


def test_regression_capacity_refusal_record_in_deferring_pools(oracle_mod):
    """Regression guard for a wrong record once produced by builds of the compact kernel: in
    deferring hard-protection pools, capacity refusals came out with b (active live required) equal
    to the hit count of the served-prefill record instead of A + cached hits + need.  Every refusal
    must satisfy the feasibility identity a + b > U (protected resident plus required exceeds the
    usable pool, §3.4) and equal the oracle."""
    trace = randtrace.random_batch(61, 400, U_range=(8, 300), n_events=(1, 400), n_chains=9,
                                   p_malformed=0.01, tight_every=7, caps=(256, 64), defer=True,
                                   hard_share=0.8)
    gpu, ora = _both_kernel(oracle_mod, trace, "compact")
    out = gpu[0]
    code = out[:, 0] & 255
    ref = (code == 2) | (code == 3) | (code == 10)
    Ue = np.repeat(trace.field("usable_blocks").astype(np.int64), trace.field("n_events"))
    assert ref.sum() > 1000
    assert (out[ref, 2].astype(np.int64) + out[ref, 3] > Ue[ref]).all()
    compare_pools(trace, gpu, ora)


@pytest.mark.parametrize("offload", [False, True])
@pytest.mark.parametrize("variant", ["wide", "wide_global_lists", "global_lists_small_request_table"])
def test_deferral_storage_layouts(oracle_mod, tg, variant, offload):
    """Deferral and runtime relaxation (with and without a second tier) with 32-bit LDS state and
    with the live lists in global scratch (also with live-request tables of at most 6 entries:
    retried requests enter a list that wraps back to the start of its arrays)."""
    import paper_2605_24259_amd as rkc
    trace = randtrace.random_batch(71, 600, U_range=(2, 200), n_events=(1, 200), n_chains=7,
                                   tight_every=9, defer=True, relax=True, hard_share=0.8,
                                   offload=offload)
    if variant == "global_lists_small_request_table":
        _small_request_tables(trace)
    lim = dict(trace.limits())
    lim["max_usable_blocks"] = 40000
    if variant == "wide_global_lists":
        lim["max_live_requests"] = 20000
        lim["max_live_claims"] = 4096
    elif variant == "global_lists_small_request_table":
        lim["max_live_claims"] = 8192
    say(f"case deferral layouts/{variant} offload={offload}")
    gpu = rkc.DeviceBatch(trace.desc, trace.events, trace.n_claim_slots, lim).replay().results()
    ora = oracle_mod.replay(trace.desc, trace.events, trace.n_claim_slots, threads=ORACLE_THREADS)
    compare_pools(trace, gpu, ora)


def test_zipf_defer_full_sampled(oracle_mod, tg):
    """65,536 hard-protection pools x 2,048 blocks x 1,024 events with deferral and 10% retries,
    in the benchmark's launch configuration; sampled pools against the oracle."""
    trace = tg.generate("zipf_defer")
    pools = _sample(trace.n_pools, 96)
    gpu, ora = _both(oracle_mod, trace, pools=pools)
    compare_pools(trace, gpu, ora, pools=pools)
    _properties(trace, gpu)
    pt = gpu[1]
    assert pt[:, 32].sum() > 20 * trace.n_pools
    assert (pt[:, 35] <= trace.field("max_live_requests")).all()


# ---- runtime relaxation and best-effort claims: both kernels -----------------------------------
@pytest.mark.parametrize("kernel", KERNELS)
def test_relaxation_fixtures(oracle_mod, tg, kernel):
    """Hand-derived relaxation cases (the 60/70/80 probe relaxed to 50 post-release victims and no
    harm, lowest priority first, only as many as needed, none when insufficient, decode growth,
    best-effort claims, relaxation before deferral) on both kernels."""
    fx = relax_cases.fixtures()
    trace = gf.to_trace(tg, fx)
    gpu, ora = _both_kernel(oracle_mod, trace, kernel)
    errs = gf.check(fx, trace, *gpu)
    assert not errs, "\n".join(errs)
    compare_pools(trace, gpu, ora)


@pytest.mark.parametrize("kernel", KERNELS)
@pytest.mark.parametrize("seed,defer", [(81, False), (82, True)])
def test_random_relaxation_tiny(oracle_mod, kernel, seed, defer):
    """Relaxing pools of <= 12 blocks with demotable and best-effort claims, with and without
    deferral, tight tables, malformed events."""
    trace = randtrace.random_batch(seed, 3000, U_range=(1, 13), n_events=(0, 40), n_chains=3,
                                   relax=True, defer=defer, hard_share=0.8)
    gpu, ora = _both_kernel(oracle_mod, trace, kernel)
    compare_pools(trace, gpu, ora)
    assert gpu[1][:, 36].sum() > 50


@pytest.mark.parametrize("kernel", KERNELS)
def test_random_relaxation_medium(oracle_mod, kernel):
    """Relaxing and deferring pools up to 300 blocks and 400 events, up to 64 live claims: the
    demotion order is a wave-wide minimum over many claim lanes."""
    trace = randtrace.random_batch(91, 400, U_range=(8, 300), n_events=(1, 400), n_chains=9,
                                   p_malformed=0.01, tight_every=7, caps=(256, 64), defer=True,
                                   relax=True, hard_share=0.8)
    gpu, ora = _both_kernel(oracle_mod, trace, kernel)
    compare_pools(trace, gpu, ora)
    assert gpu[1][:, 37].sum() > 50


# ---- offload to a second tier: both kernels --------------------------------------------------
@pytest.mark.parametrize("kernel", KERNELS)
def test_offload_fixtures(oracle_mod, tg, kernel):
    """Hand-derived offload cases (offload before demotion, a footprint larger than the free room
    falls back to demotion, restore accounting on a later prefill, expiry and release drop the
    copy, offloaded claims never harmed, peak second-tier use) on both kernels."""
    fx = relax_cases.offload_fixtures()
    trace = gf.to_trace(tg, fx)
    gpu, ora = _both_kernel(oracle_mod, trace, kernel)
    errs = gf.check(fx, trace, *gpu)
    assert not errs, "\n".join(errs)
    compare_pools(trace, gpu, ora)


@pytest.mark.parametrize("kernel", KERNELS)
@pytest.mark.parametrize("seed,defer", [(401, False), (402, True)])
def test_random_offload_tiny(oracle_mod, kernel, seed, defer):
    """Relaxing pools of <= 12 blocks with a second tier of random capacity, offloadable and
    demotable claims, with and without deferral."""
    trace = randtrace.random_batch(seed, 3000, U_range=(1, 13), n_events=(0, 40), n_chains=3,
                                   relax=True, offload=True, defer=defer, hard_share=0.8)
    gpu, ora = _both_kernel(oracle_mod, trace, kernel)
    compare_pools(trace, gpu, ora)
    assert gpu[1][:, 38].sum() > 50


@pytest.mark.parametrize("kernel", KERNELS)
def test_random_offload_medium(oracle_mod, kernel):
    """Offloading pools up to 300 blocks and 400 events, up to 64 live claims, deferral mixed in:
    the offload order is a wave-wide minimum over many claim lanes and the room runs out."""
    trace = randtrace.random_batch(411, 400, U_range=(8, 300), n_events=(1, 400), n_chains=9,
                                   p_malformed=0.01, tight_every=7, caps=(256, 64), defer=True,
                                   relax=True, offload=True, hard_share=0.8)
    gpu, ora = _both_kernel(oracle_mod, trace, kernel)
    compare_pools(trace, gpu, ora)
    pt = gpu[1]
    assert pt[:, 38].sum() > 50 and pt[:, 40].sum() > 0


def test_zipf_relax_full_sampled(oracle_mod, tg):
    """65,536 relaxing hard-protection pools x 2,048 blocks x 1,024 events, half the claims
    demotable, in the benchmark's launch configuration; sampled pools against the oracle."""
    trace = tg.generate("zipf_relax")
    pools = _sample(trace.n_pools, 96)
    gpu, ora = _both(oracle_mod, trace, pools=pools)
    compare_pools(trace, gpu, ora, pools=pools)
    _properties(trace, gpu)
    assert gpu[1][:, 36].sum() > trace.n_pools


@pytest.mark.parametrize("kernel", KERNELS)
def test_random_all_features(oracle_mod, kernel):
    """Every pool defers and carries the relaxation flag (ignored outside hard protection), claims
    are demotable, best-effort and offloadable at random, half the pools are hard, the rest cycle
    the policies; pools up to 400 blocks and 300 events, tight and overflowing tables, malformed
    events.  Every word of both kernels against the oracle."""
    trace = randtrace.random_batch(501, 2000, U_range=(1, 400), n_events=(0, 300), n_chains=12,
                                   p_malformed=0.02, tight_every=6, caps=(256, 64), defer=True,
                                   relax=True, offload=True, hard_share=0.5)
    gpu, ora = _both_kernel(oracle_mod, trace, kernel)
    compare_pools(trace, gpu, ora)
    pt = gpu[1]
    assert pt[:, 32].sum() > 100 and pt[:, 37].sum() > 100 and pt[:, 38].sum() > 100


def test_zipf_offload_full_sampled(oracle_mod, tg):
    """65,536 relaxing hard-protection pools x 2,048 blocks x 1,024 events with a 1,024-block second
    tier, half the claims offloadable and a quarter demotable, in the benchmark's launch
    configuration; sampled pools against the oracle."""
    trace = tg.generate("zipf_offload")
    pools = _sample(trace.n_pools, 96)
    gpu, ora = _both(oracle_mod, trace, pools=pools)
    compare_pools(trace, gpu, ora, pools=pools)
    _properties(trace, gpu)
    pt = gpu[1]
    assert pt[:, 38].sum() > trace.n_pools and pt[:, 40].sum() > 0
    assert (pt[:, 41] <= 1024).all()


def test_compact_kernel_at_its_limits(oracle_mod, tg):
    """One batch at the compact kernel's limits: 32,767-block pools, 256 chains, a pool of 65,533
    events (16-bit ids up to 65,532), live-claim and live-request tables filled to exactly 64 and
    256 and then overflowed, an empty pool, an all-malformed pool, and a deferring / relaxing pool
    and an offloading one at full size.  Every outcome, pool word and claim record against the oracle."""
    import bench
    rng = np.random.default_rng(2026)
    big = randtrace.random_pool(rng, 32767, 3, 3000, n_chains=256, p_malformed=0.01)
    big["max_live_requests"], big["max_live_claims"] = 256, 64
    long_pool = randtrace.random_pool(rng, 8, 0, 65533, n_chains=1, p_malformed=0.01)
    long_pool["max_live_requests"], long_pool["max_live_claims"] = 256, 64
    ext = randtrace.random_pool(rng, 32767, 3, 2000, n_chains=256, p_malformed=0.01, defer_limit=3,
                                relax=True)
    ext["mode"] = 3 | tg.MODE_RELAX
    ext["max_live_requests"], ext["max_live_claims"] = 256, 64
    off = randtrace.random_pool(rng, 32767, 3, 2000, n_chains=256, p_malformed=0.01, defer_limit=3,
                                relax=True, offload=True)
    off["mode"] = 3 | tg.MODE_RELAX
    off["max_live_requests"], off["max_live_claims"], off["offload_blocks"] = 256, 64, 16000
    tables = dict(usable_blocks=400, mode=1, n_chains=256, max_live_claims=64, max_live_requests=256,
                  events=[tg.claim(1, c, 1) for c in range(65)] + [tg.prefill(1)] * 257
                  + [tg.release(0), tg.claim(2, 70, 2), tg.finish(3), tg.prefill(2, 200, 2)])
    pools = [big, long_pool, ext, tables,
             dict(usable_blocks=1, mode=2, n_chains=0, events=[]),
             dict(usable_blocks=32767, mode=3, n_chains=256,
                  events=[tg.ev(11), tg.prefill(0), tg.claim(5, 256), tg.extend(-1), tg.ev(15)]),
             off]
    trace = tg.from_pools(pools, "compact-limits")
    lim = trace.limits()
    assert lim["max_usable_blocks"] == 32767 and lim["max_events"] == 65533
    assert lim["max_chains"] == 256 and bench.kernel_name(lim) == "rkc_lean"
    gpu, ora = _both(oracle_mod, trace)
    compare_pools(trace, gpu, ora)
    pt = gpu[1]
    assert pt[3, 31] == 3  # request and claim tables both overflowed (status bits 1 | 2)
    assert pt[3, 29] == 256 and pt[3, 30] == 64 and pt[3, 9] == 2
    assert pt[4, 27] == 1 and pt[4, :].sum() == 1  # the empty pool: one FREE block, nothing else
    assert (pt[5, 9] == 5) and (pt[5, :9] == 0).all()
    assert pt[6, 38] > 0 and pt[6, 41] <= 16000
