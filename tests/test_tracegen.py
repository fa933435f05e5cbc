"""The seeded workload generator: determinism, slicing, and the recipe's shapes (no GPU needed)."""
import numpy as np
import pytest


def test_deterministic_and_sliceable(tg):
    a = tg.generate("small", n_pools=40)
    b = tg.generate("small", n_pools=40)
    assert a.sha256() == b.sha256()
    c = tg.generate("small", n_pools=10, first_pool=20)
    eo = a.field("event_offset")
    ne = a.field("n_events")
    assert np.array_equal(c.events, a.events[eo[20]: eo[30 - 1] + ne[29]])
    # descriptors describe the slice contiguously
    assert c.field("event_offset")[0] == 0
    assert np.array_equal(c.field("n_claim_slots"), a.field("n_claim_slots")[20:30])
    assert list(c.field("mode")) == [p % 4 for p in range(20, 30)]


@pytest.mark.parametrize("name", ["small", "zipf", "nested", "huge"])
def test_recipe_shapes(tg, name):
    n = 4 if name == "huge" else 64
    t = tg.generate(name, n_pools=n)
    p = tg.CONFIGS[name]
    ev = t.events
    typ = ev[:, 0] & 15
    frac = np.bincount(typ, minlength=6)[:6] / len(typ)
    mix = np.array(p["mix"]) / 1000.0
    tol = 0.02 if name != "huge" else 0.01
    if name == "huge":
        # claims drawn at the outstanding cap turn into releases
        assert abs(frac[0] - mix[0]) < tol and abs(frac[1] - mix[1]) < tol
    else:
        assert np.all(np.abs(frac - mix) < tol), (frac, mix)
    pre = ev[typ == 0]
    assert pre[:, 1].min() >= p["prefill_min"] and pre[:, 1].max() <= p["prefill_max"]
    assert (pre[:, 3] <= pre[:, 1]).all() and (pre[:, 3] >= 0).all()
    cl = ev[typ == 2]
    assert (cl[:, 3] <= cl[:, 1]).all()
    dur = cl[:, 0].view(np.uint32) >> 16
    assert dur.min() >= p["dur_min"] and dur.max() <= p["dur_max"]
    prio = (cl[:, 0] >> 5) & 3
    assert prio.max() <= 3
    hard_frac = ((cl[:, 0] >> 4) & 1).mean()
    assert abs(hard_frac - p["hard_permille"] / 1000.0) < 0.05
    assert t.n_claim_slots == int((typ == 2).sum())
    if p["chain_pick"] == 1:
        # Zipf(1.1): chain 0 is the most frequent
        counts = np.bincount(pre[:, 2], minlength=p["n_chains"])
        assert counts[0] == counts.max()
    if name == "huge":
        # outstanding claims never exceed the cap within a pool
        for i in range(t.n_pools):
            e = ev[i * p["n_events"]: (i + 1) * p["n_events"]]
            out = 0
            for x in e[:, 0] & 15:
                if x == 2:
                    out += 1
                elif x == 4 and out > 0:
                    out -= 1
                assert out <= p["claim_cap"]


def test_probe_layout(tg):
    t = tg.probe()
    assert t.n_pools == 4 and t.n_events == 8 and t.n_claim_slots == 4
    assert list(t.field("mode")) == [0, 1, 2, 3]
    assert list(t.field("usable_blocks")) == [80] * 4


def test_prefix_replay_is_the_leading_part_of_the_full_replay(oracle_mod, tg):
    """Trace.prefix keeps each pool's first events (and the CLAIM slots among them); replay is
    causal, so the oracle's outcomes on the prefix equal the leading outcomes of the full pool."""
    import numpy as np
    t = tg.generate("small", n_pools=6)
    full = oracle_mod.replay(t.desc, t.events, t.n_claim_slots)
    eo = t.field("event_offset")
    for k in (0, 1, 17, 100, 256):
        p = t.prefix([0, 2, 5], k)
        assert p.n_events == 3 * k
        assert p.n_claim_slots == int(sum(((t.events[eo[i]: eo[i] + k, 0] & 15) == 2).sum() for i in (0, 2, 5)))
        out = oracle_mod.replay(p.desc, p.events, p.n_claim_slots)
        assert not out[3].any()
        for j, i in enumerate((0, 2, 5)):
            assert np.array_equal(out[0][j * k:(j + 1) * k], full[0][eo[i]: eo[i] + k])


def test_nested_active_load_is_calibrated(oracle_mod, tg):
    """The nested workload's frozen extend size (tests/calibrate_nested.py) makes about 30 % of all
    steps active refusals; on the first 64 pools the share is within sampling noise of that."""
    import numpy as np
    t = tg.generate("nested", n_pools=64)
    assert t.meta["params"]["extend_k"] == 152
    out = oracle_mod.replay(t.desc, t.events, t.n_claim_slots, threads=8)
    assert not out[3].any()
    code = out[0][:, 0] & 255
    share = float(np.mean((code == 2) | (code == 3)))
    assert 0.28 <= share <= 0.32, share
