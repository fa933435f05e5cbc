"""Calibration of the nested workload's active load (test infrastructure; run by hand).

The nested workload asks that 30 % of all steps be infeasible for the active side.  With its event
mix (30 % prefill, 25 % extend, 20 % claim, 10 % demote, 10 % finish, 5 % release) a refusal can
only hit a prefill or an extend, and prefill sizes alone cannot get there: with prefill sizes
log-uniform in [16, S_max] the refused share stays between 15 % and 19 % for any S_max up to the
2^24 field limit, because a refused prefill leaves the pool free enough for the next extend.  The
knob is therefore the size of an extend (a chunk of a request's continued prefill or decode),
chosen by bisection on the oracle so that REFUSED_CLAIM + REFUSED_CAPACITY outcomes are 30 % +- 1 %
of all steps over the first 1,024 pools.  Result (frozen in tracegen.CONFIGS["nested"]):
extend = 152 blocks, 29.93 % refused.

    python tests/calibrate_nested.py [n_pools]
"""
import os
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)


def refused_share(extend_k: int, n_pools: int, threads: int = 8) -> float:
    import oracle
    from paper_2605_24259_amd import tracegen as tg
    t = tg.generate("nested", n_pools=n_pools, extend_k=extend_k)
    out = oracle.replay(t.desc, t.events, t.n_claim_slots, threads=threads)
    code = out[0][:, 0] & 255
    return float(np.mean((code == 2) | (code == 3)))


def calibrate(n_pools: int = 1024, lo: int = 1, hi: int = 512, target: float = 0.30) -> int:
    """Smallest extend size whose refused share reaches the target (the share grows with it)."""
    while lo < hi:
        mid = (lo + hi) // 2
        share = refused_share(mid, n_pools)
        print(f"extend {mid:4d}: refused {share:.4f}", flush=True)
        if share < target:
            lo = mid + 1
        else:
            hi = mid
    return lo


if __name__ == "__main__":
    n = int(sys.argv[1]) if len(sys.argv) > 1 else 1024
    k = calibrate(n)
    print(f"extend = {k} blocks: refused share {refused_share(k, n):.4f} over the first {n} pools")
