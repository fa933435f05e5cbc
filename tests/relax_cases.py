"""Hand-derived cases of runtime relaxation and best-effort claims, in the fixture format of
tests/golden_fixtures.py.

§3.1 protection modes: a demotable claim may be downgraded before loss, provided the demotion comes
before the predicate-breaking eviction; a best-effort claim is telemetry only.  §3.5 mechanism
table, "relax resident claim": the active side is served by demoting resident state.  §5.4 L4: when
demotion precedes the loss, the 60/70/80 probe loses 50 blocks after release and harms nothing.

Pools with mode flag `relax` demote, before refusing an active request on behalf of claims, the
demotable claims among the blocking ones, lowest priority first, then lowest id, until the request
fits; none when even all of them would not make it fit.  Expected values are worked out by hand from
the feasibility inequality Pr + req <= U (§3.4) and the eviction order (level, last use, position).
"""
from tests import golden_fixtures as gf

RELAX_CASES = """
# The 60/70/80 probe with a demotable hard claim in a relaxing pool: the runtime demotes the claim,
# then the prefill evicts 50 of its blocks as post-release loss; no harm (§5.4 L4 counts).
[pool probe_relaxed]
usable = 80
mode = hard
relax = 1
chains = 2
events:
  claim L=60 c=0 T=60 hard=1 prio=3 demotable=1
  prefill S=70 c=1 P=0
expect:
  t0 code=admit b=60 flags=
  t1 code=relaxed id=1 a=50 b=0 n16=1 flags=pred_fail|post_release_loss
  tel n_relaxed=1 runtime_demoted=1 resident=50 post_release=50 harm=0 cached=10 active=70
  tel demoted=0 n_refused_claim=0
  claim0 state=demoted demote=1 pred_fail=1 harm=-1 lead_end=10 demotable=1 relaxed=1 eff=2

# Without the pool flag the same claim protects as any hard claim: attributed refusal.
[pool probe_no_relax_flag]
usable = 80
mode = hard
chains = 2
events:
  claim L=60 c=0 T=60 hard=1 prio=3 demotable=1
  prefill S=70 c=1 P=0
expect:
  t1 code=refused_claim id=0 a=60 b=70 n16=1
  claim0 state=materialized demote=-1 relaxed=0 blocked=1

# A relaxing pool never demotes a claim that does not allow it.
[pool probe_not_demotable]
usable = 80
mode = hard
relax = 1
chains = 2
events:
  claim L=60 c=0 T=60 hard=1 prio=3
  prefill S=70 c=1 P=0
expect:
  t1 code=refused_claim id=0 a=60 b=70 n16=1
  tel n_relaxed=0 runtime_demoted=0

# Lowest priority first, and only as many as needed: 40 free + 30 from the priority-0 claim cover
# the 60 blocks; its top 20 positions go (level 1), the priority-1 claim keeps its protection.
[pool lowest_priority_first]
usable = 100
mode = hard
relax = 1
chains = 3
events:
  claim L=30 c=0 T=30 hard=1 prio=1 demotable=1
  claim L=30 c=1 T=30 hard=1 prio=0 demotable=1
  prefill S=60 c=2 P=0
expect:
  t2 code=relaxed id=2 a=20 b=0 n16=1 flags=pred_fail|post_release_loss
  claim0 state=materialized demote=-1 lead_end=30 relaxed=0
  claim1 state=demoted demote=2 pred_fail=2 lead_end=10 relaxed=1
  tel runtime_demoted=1 protected=30 cached=40

# Equal priorities: the older claim goes first.
[pool oldest_first]
usable = 100
mode = hard
relax = 1
chains = 3
events:
  claim L=30 c=0 T=30 hard=1 prio=2 demotable=1
  claim L=30 c=1 T=30 hard=1 prio=2 demotable=1
  prefill S=60 c=2 P=0
expect:
  t2 code=relaxed id=2 a=20 n16=1
  claim0 state=demoted demote=2 lead_end=10
  claim1 state=materialized demote=-1 lead_end=30

# Both demotable claims are needed: 40 free + 30 + 30 >= 90.
[pool both_needed]
usable = 100
mode = hard
relax = 1
chains = 3
events:
  claim L=30 c=0 T=30 hard=1 prio=1 demotable=1
  claim L=30 c=1 T=30 hard=1 prio=0 demotable=1
  prefill S=90 c=2 P=0
expect:
  t2 code=relaxed id=2 a=50 n16=2 flags=pred_fail|post_release_loss
  tel runtime_demoted=2 cached=10 active=90 harm=0
  claim0 state=demoted demote=2
  claim1 state=demoted demote=2

# Demoting every demotable blocker would still leave 40 + 30 < 80: nothing is demoted and the
# refusal names both blockers (Pr 60, required 80).
[pool insufficient]
usable = 100
mode = hard
relax = 1
chains = 3
events:
  claim L=30 c=0 T=30 hard=1 prio=1
  claim L=30 c=1 T=30 hard=1 prio=0 demotable=1
  prefill S=80 c=2 P=0
expect:
  t2 code=refused_claim id=0 a=60 b=80 n16=2
  tel runtime_demoted=0 protected=60
  claim0 state=materialized blocked=1
  claim1 state=materialized blocked=1 demote=-1

# Decode growth is relaxed like a prefill: b = active blocks after the extension.
[pool extend_relaxed]
usable = 80
mode = hard
relax = 1
chains = 2
events:
  claim L=60 c=0 T=60 hard=1 prio=0 demotable=1
  prefill S=20 c=1 P=0
  extend k=5 sel=0
expect:
  t1 code=admit id=1 b=0
  t2 code=relaxed id=1 a=5 b=25 n16=1 flags=pred_fail|post_release_loss
  claim0 state=demoted demote=2 pred_fail=2 lead_end=55

# A best-effort claim carries no obligation in any policy: observed (shadow), never protects, its
# loss is a predicate failure without harm.
[pool best_effort_in_hard_pool]
usable = 80
mode = hard
chains = 2
events:
  claim L=60 c=0 T=60 hard=1 prio=3 best_effort=1
  prefill S=70 c=1 P=0
expect:
  t0 code=admit b=60 flags=shadow
  t1 code=evict_resident id=1 a=50 flags=pred_fail
  tel shadow=1 accepted=0 harm=0 protected=0 resident=50 post_release=0
  claim0 decision=shadow state=observed eff=0 best_effort=1 pred_fail=1 harm=-1

# Relaxation comes first; a request that no relaxation can serve is still deferred.
[pool relax_then_defer]
usable = 68
mode = hard
relax = 1
defer_limit = 1
chains = 3
events:
  claim L=40 c=0 T=40 hard=1 prio=3
  claim L=10 c=1 T=10 hard=1 prio=0 demotable=1
  prefill S=46 c=2 P=0
  prefill S=10 c=2 P=0
  retry
expect:
  t2 code=deferred id=0 a=50 b=46 n16=2
  t3 code=admit id=3
  t4 code=refused_claim id=0 a=50 b=56 n16=2
  tel n_deferred=1 retry_refused=1 runtime_demoted=0
"""


# Offload to a second tier (§3.1 offloadable: the content may leave GPU memory only if the
# predicate stays restorable; §3.5 "offload resident": the resident survives and the active side is
# served, subject to restore cost).  Pools with a second tier of `offload` blocks offload a blocking
# claim that allows it when its footprint fits the free room; its predicate then never fails, its
# GPU blocks are ordinary cache (victims it covers are not resident loss), and a later prefill that
# reaches past its leading GPU hits into the claim's footprint counts those positions as restored.
OFFLOAD_CASES = """
# The 60/70/80 probe with an offloadable claim and a 60-block second tier: the claim is offloaded,
# 50 of its GPU blocks are taken without loss (unclaimed victims), no predicate failure, no harm.
[pool probe_offloaded]
usable = 80
mode = hard
relax = 1
offload = 60
chains = 2
events:
  claim L=60 c=0 T=60 hard=1 prio=3 offloadable=1
  prefill S=70 c=1 P=0
expect:
  t1 code=relaxed id=1 a=0 b=0 n16=1 flags=evict_unclaimed
  tel n_relaxed=1 off_claims=1 off_blocks=60 t2_peak=60 runtime_demoted=0 resident=0 victims=50
  tel pred_fail=0 harm=0 cached=10 protected=0
  claim0 state=materialized eff=3 relaxed=1 offloadable=1 pred_fail=-1 harm=-1 lead_end=10

# Too little room (50 < 60): an offloadable-only claim cannot be relaxed, the refusal stands; a
# claim that also allows demotion is demoted instead.
[pool no_room]
usable = 80
mode = hard
relax = 1
offload = 50
chains = 3
events:
  claim L=60 c=0 T=60 hard=1 prio=3 offloadable=1
  prefill S=70 c=1 P=0
expect:
  t1 code=refused_claim id=0 a=60 b=70 n16=1
  tel off_claims=0 t2_peak=0
  claim0 state=materialized eff=2 relaxed=0 blocked=1

[pool no_room_demoted]
usable = 80
mode = hard
relax = 1
offload = 50
chains = 3
events:
  claim L=60 c=0 T=60 hard=1 prio=3 offloadable=1 demotable=1
  prefill S=70 c=1 P=0
expect:
  t1 code=relaxed id=1 a=50 n16=1 flags=pred_fail|post_release_loss
  tel off_claims=0 runtime_demoted=1
  claim0 state=demoted eff=2 relaxed=1 demote=1 pred_fail=1 harm=-1

# Restore: after the offload, the request finishes and a prefill of 40 on the claim's chain hits the
# 10 GPU-resident positions and restores 30 from the second tier (it still takes 30 GPU blocks, the
# oldest cached ones of the finished request's private run).
[pool restore]
usable = 80
mode = hard
relax = 1
offload = 60
chains = 2
events:
  claim L=60 c=0 T=60 hard=1 prio=3 offloadable=1
  prefill S=70 c=1 P=0
  finish sel=0
  prefill S=40 c=0 P=40
expect:
  t3 code=admit id=3 a=0 b=10 flags=evict_unclaimed
  tel restored=30 off_claims=1 live_requests=1
  claim0 state=materialized eff=3 lead_end=40

# DEMOTE never selects an offloaded claim; RELEASE drops its copy, so the next offload fits.
[pool release_frees_room]
usable = 100
mode = hard
relax = 1
offload = 60
chains = 3
events:
  claim L=60 c=0 T=60 hard=1 offloadable=1
  prefill S=90 c=2 P=0
  demote sel=0
  finish sel=0
  release sel=0
  claim L=60 c=1 T=60 hard=1 offloadable=1
  prefill S=90 c=2 P=0
expect:
  t1 code=relaxed id=1 n16=1
  t2 code=noop
  t6 code=relaxed id=6 n16=1
  tel off_claims=2 off_blocks=120 t2_peak=60
  claim0 state=released eff=3
  claim1 state=materialized eff=3

# Expiry ends the runtime's responsibility: the copy is dropped and the claim, now expired, loses
# its protection class (effective protection none).  Its predicate held only through the copy: the
# chain keeps 10 < T = 60 leading blocks, so it fails at the expiry step, without harm (the claim is
# expired).  The next prefill of 75 takes the chain's 10 GPU blocks first (last used at step 0,
# before the finished run's step 4): resident, post-release loss.
[pool expiry_drops_copy]
usable = 80
mode = hard
relax = 1
offload = 60
chains = 3
events:
  claim L=60 c=0 T=60 hard=1 offloadable=1 dur=3
  prefill S=70 c=1 P=0
  nop
  nop
  finish sel=0
  prefill S=75 c=2 P=0
expect:
  t1 code=relaxed id=1 n16=1
  t3 code=noop n16=1 flags=expired|pred_fail
  t5 code=evict_resident id=5 a=10 flags=post_release_loss|evict_unclaimed
  tel expired=1 off_claims=1 t2_peak=60 harm=0 pred_fail=1
  claim0 state=expired eff=0 expire=3 pred_fail=3 harm=-1

# The same with T = 10: the 10 leading blocks left on the GPU still satisfy the predicate when the
# copy is dropped, so nothing fails.
[pool expiry_keeps_predicate]
usable = 80
mode = hard
relax = 1
offload = 60
chains = 3
events:
  claim L=60 c=0 T=10 hard=1 offloadable=1 dur=3
  prefill S=70 c=1 P=0
  nop
  nop
expect:
  t1 code=relaxed id=1 n16=1
  t3 code=noop n16=1 flags=expired
  tel expired=1 off_claims=1 pred_fail=0 harm=0
  claim0 state=expired eff=0 expire=3 pred_fail=-1 lead_end=10
"""


def fixtures():
    return gf.parse_text(RELAX_CASES, "relaxation closed forms")


def offload_fixtures():
    return gf.parse_text(OFFLOAD_CASES, "offload closed forms")
