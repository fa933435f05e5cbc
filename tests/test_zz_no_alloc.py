"""The no-allocation entry point (rkc_replay_batch_noalloc, for callers that cannot allocate) gives
the same outputs as rkc_replay_batch with a caller scratch buffer, bit for bit, on two calls in a
row (the second smaller, so it runs on the first call's leftover scratch contents), on both kernels;
a batch beyond its built-in scratch is refused."""
import numpy as np
import pytest

from tests.gpu_util import say

pytestmark = pytest.mark.gpu


def _both(rkc, trace, flags=0):
    ref = rkc.DeviceBatch.from_trace(trace, flags=flags).replay().results()
    db = rkc.DeviceBatch.from_trace(trace, flags=flags, scratch=False)
    assert db.scratch is None and db.scratch_needed <= rkc.NOALLOC_SCRATCH_BYTES
    got = db.replay_noalloc().results()
    for g, r, what in zip(got, ref, ("outcomes", "pool telemetry", "claim telemetry")):
        assert np.array_equal(g, r), f"{trace.name}: {what} differ"


def test_noalloc_matches_replay_batch(tg):
    import paper_2605_24259_amd as rkc
    cases = [(tg.generate("zipf", n_pools=1024), 0),                  # compact kernel, ~31 MiB
             (tg.generate("zipf", n_pools=300, first_pool=5000), 0),  # smaller, stale scratch
             (tg.generate("nested", n_pools=16), 0),                  # general kernel
             (tg.generate("small", n_pools=200), rkc.FLAG_GENERAL_KERNEL)]
    for trace, flags in cases:
        say(f"case noalloc {trace.name} {trace.n_pools} pools flags {flags}")
        _both(rkc, trace, flags)


def test_noalloc_refuses_oversized_batch(tg):
    import paper_2605_24259_amd as rkc
    trace = tg.generate("zipf", n_pools=4096)
    db = rkc.DeviceBatch.from_trace(trace, scratch=False)
    assert db.scratch_needed > rkc.NOALLOC_SCRATCH_BYTES
    with pytest.raises(rkc.RkcError) as e:
        db.replay_noalloc()
    assert e.value.status == -8
