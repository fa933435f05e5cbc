"""GPU parity of the workgroup-per-pool replay (several waves per pool share the scans and moves of
long live lists) against the oracle, and against the one-wave-per-pool replay of the same inputs.

The workgroup path serves batches of at most 256 pools whose live lists live in global scratch; the
262,144-block workload is one (its every pool is checked in tests/test_gpu_full.py).  Here: random
pools with every feature, and pools built to hold thousands of live requests and claims, so that
list moves take several rounds of the workgroup and the claim scans span every wave.
"""
import numpy as np
import pytest

from tests import randtrace
from tests.gpu_util import compare_pools, gpu_replay, say

pytestmark = pytest.mark.gpu


def _global_list_limits(trace):
    lim = dict(trace.limits())
    lim["max_live_requests"] = max(lim["max_live_requests"], 20000)
    lim["max_live_claims"] = max(lim["max_live_claims"], 4096)
    return lim


def _run(trace, flags):
    import paper_2605_24259_amd as rkc
    db = rkc.DeviceBatch(trace.desc, trace.events, trace.n_claim_slots, _global_list_limits(trace),
                         flags=flags)
    return db.replay().results()


def _check(oracle_mod, trace):
    import paper_2605_24259_amd as rkc
    assert trace.n_pools <= 256
    say(f"case group {trace.name}: {trace.n_pools} pools, {trace.n_events} events")
    ora = oracle_mod.replay(trace.desc, trace.events, trace.n_claim_slots, threads=16)
    assert not ora[3].any()
    grp = _run(trace, 0)
    compare_pools(trace, grp, ora)
    one = _run(trace, rkc.FLAG_ONE_WAVE_PER_POOL)
    compare_pools(trace, one, ora)


@pytest.mark.parametrize("seed,defer,relax,offload", [(91, False, False, False), (92, True, False, False),
                                                      (93, True, True, False), (94, True, True, True)])
def test_group_random(oracle_mod, seed, defer, relax, offload):
    """256 random pools (every policy, malformed events, tight tables, several 64-event tiles)."""
    trace = randtrace.random_batch(seed, 256, U_range=(8, 300), n_events=(1, 400), n_chains=9,
                                   p_malformed=0.01, tight_every=7, caps=(256, 64), defer=defer,
                                   relax=relax, offload=offload, hard_share=0.6)
    _check(oracle_mod, trace)


def long_list_pools(tg, seed, n_pools=4):
    """Pools that grow thousands of live requests and claims on a few shared chains, then finish,
    release, extend and prefill at random: every list move spans several workgroup rounds."""
    rng = np.random.default_rng(seed)
    pools = []
    for i in range(n_pools):
        evs = []
        for t in range(5200):
            phase1 = t < 2600
            r = rng.random()
            sel = int(rng.integers(0, 1 << 31))
            if phase1 and r < 0.62:
                c = int(rng.integers(0, 8))
                evs.append(tg.prefill(int(rng.integers(1, 4)), c, 1))
            elif r < (0.95 if phase1 else 0.30):
                L = int(rng.integers(1, 60))
                dur = 0 if rng.random() < 0.5 else int(rng.integers(50, 2500))
                evs.append(tg.claim(L, int(rng.integers(0, 8)), int(rng.integers(0, L + 1)),
                                    hard=int(rng.integers(0, 2)), prio=int(rng.integers(0, 4)), dur=dur))
            elif phase1:
                evs.append(tg.extend(1, sel))
            elif r < 0.55:
                evs.append(tg.finish(sel))
            elif r < 0.68:
                evs.append(tg.release(sel))
            elif r < 0.80:
                evs.append(tg.extend(int(rng.integers(1, 40)), sel))
            elif r < 0.85:
                evs.append(tg.demote(sel))
            else:
                c = int(rng.integers(0, 8))
                S = int(rng.integers(1, 3000))
                evs.append(tg.prefill(S, c, int(rng.integers(0, min(S, 70) + 1))))
        pools.append(dict(usable_blocks=9000, mode=i % 4, n_chains=8, max_live_requests=4000,
                          max_live_claims=2000, events=evs))
    return tg.from_pools(pools, f"long-lists{seed}")


@pytest.mark.parametrize("seed", [101, 102])
def test_group_long_lists(oracle_mod, tg, seed):
    trace = long_list_pools(tg, seed)
    _check(oracle_mod, trace)
