"""Capacity sweep (§5.3 capacity-sweep figure, generalized to a grid of resident footprint R,
active size A, usable blocks U and the four policies).

Pins: every cell's outcome follows from the feasibility inequality Pr + req <= U (§3.4) in closed
form -- the claim materializes iff R <= U; the active side alone fits iff A <= U; both coexist iff
R + A <= U; otherwise the hard-protection policy refuses the active request attributed to the
claim (a = R protected, b = A required, shortfall R + A - U) and the other policies serve it by
evicting R + A - U resident blocks.  The oracle is checked against that closed form on the CPU;
the GPU replay is checked bit-exactly against the oracle on every cell.
"""
import numpy as np
import pytest

from tests.gpu_util import compare_pools, gpu_replay, say

HARD = 3


def closed_form(mode, R, A, U):
    """(t0 code, t1 code, t1 id, t1 a, t1 b, class) for one cell."""
    from paper_2605_24259_amd import sweep as sw
    if R > U:
        t1 = (0, 0, 0) if A <= U else (3, -1, 0)
        code1 = t1[0]
        return 4, code1, (1 if code1 == 0 else -1), 0, (0 if code1 == 0 else A), sw.CLAIM_FAILED
    if A > U:
        return 0, 3, -1, (R if mode == HARD else 0), A, sw.REFUSED_CAPACITY
    if R + A <= U:
        return 0, 0, 1, 0, 0, sw.COEXIST
    if mode == HARD:
        return 0, 2, 0, R, A, sw.REFUSED_CLAIM
    return 0, 1, 1, R + A - U, 0, sw.RESIDENT_LOST


def _grid_cells(trace):
    g = trace.meta["grid"]
    m, r, a, u = np.meshgrid(np.asarray(g["modes"]), np.asarray(g["residents"]), np.asarray(g["actives"]),
                             np.asarray(g["usables"]), indexing="ij")
    return m.reshape(-1), r.reshape(-1), a.reshape(-1), u.reshape(-1)


def test_oracle_matches_closed_form_on_the_sweep(oracle_mod, tg):
    from paper_2605_24259_amd import sweep as sw
    trace = tg.sweep(residents=(1, 30, 60, 61, 100), actives=(1, 20, 70, 71, 129, 130),
                     usables=(1, 29, 30, 59, 60, 61, 69, 70, 71, 90, 129, 130, 131, 200))
    out, pt, ct, chk = oracle_mod.replay(trace.desc, trace.events, trace.n_claim_slots, threads=8)
    assert not chk.any()
    o = out.reshape(-1, 2, 4)
    cls = sw.heatmap(trace, out).reshape(-1)
    for j, (m, R, A, U) in enumerate(zip(*_grid_cells(trace))):
        c0, c1, id1, a1, b1, k = closed_form(int(m), int(R), int(A), int(U))
        got = (int(o[j, 0, 0] & 255), int(o[j, 1, 0] & 255), int(o[j, 1, 1]), int(o[j, 1, 2]))
        assert got == (c0, c1, id1, a1), (m, R, A, U, got)
        if c1 in (2, 3):
            assert int(o[j, 1, 3]) == b1 and int(o[j, 1, 2]) + int(o[j, 1, 3]) > U
        assert cls[j] == k, (m, R, A, U)
    # the boundary of the paper's figure: 60 resident + 70 active coexist from 130 blocks on
    g = trace.meta["grid"]
    hm = sw.heatmap(trace, out)
    ri, ai = g["residents"].index(60), g["actives"].index(70)
    for mi in range(4):
        row = hm[mi, ri, ai]
        for ui, U in enumerate(g["usables"]):
            assert (row[ui] == sw.COEXIST) == (U >= 130), (mi, U)


@pytest.mark.gpu
def test_sweep_gpu_bit_exact(oracle_mod, tg):
    """The full default sweep grid (131,072 cells) on the GPU equals the oracle on every cell, and
    its heatmap equals the closed form."""
    from paper_2605_24259_amd import sweep as sw
    trace = tg.sweep()
    say(f"case sweep: {trace.n_pools} pools")
    gpu = gpu_replay(trace)
    ora = oracle_mod.replay(trace.desc, trace.events, trace.n_claim_slots, threads=16)
    assert not ora[3].any()
    compare_pools(trace, gpu, ora)
    hm = sw.heatmap(trace, gpu[0]).reshape(-1)
    want = np.array([closed_form(int(m), int(R), int(A), int(U))[5] for m, R, A, U in zip(*_grid_cells(trace))])
    assert np.array_equal(hm, want)
