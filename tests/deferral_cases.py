"""Active deferral (§3.5 mechanism table "active deferral"; §3.2 table: a hard claim that blocks
active admission yields an active refusal or deferral).  Expected values below are worked out by
hand from the feasibility inequality Pr + req <= U (§3.4) and the queue rules: only a refusal
attributed to claims is deferred, the oldest deferred request is retried first, a request is
deferred at most defer_limit times, and a served request keeps its PREFILL step as its id.
"""
from tests import golden_fixtures as gf

DEFERRAL_CASES = """
# Released claim: the retried request is served by evicting 18 of the 40 unclaimed blocks (the
# highest positions first), leaving a leading run of 22.
[pool served_after_release]
usable = 68
mode = hard
chains = 2
defer_limit = 1
events:
  claim L=40 c=0 T=40 hard=1 prio=3
  prefill S=46 c=1 P=0
  release sel=0
  retry
expect:
  t1 code=deferred id=0 a=40 b=46 n16=1
  t2 code=released id=0 a=40 b=40
  t3 code=admit id=1 a=0 b=0 flags=evict_unclaimed
  tel n_deferred=1 retry_served=1 retry_refused=0 queued=0 victims=18 resident=0 active=46
  tel cached=22 free=0 live_requests=1 live_claims=0
  claim0 state=released blocked=1 lead_end=22

# defer_limit 2: two DEFERRED outcomes, then the terminal refusal; a further RETRY finds no queue.
[pool deferred_twice]
usable = 68
mode = hard
chains = 2
defer_limit = 2
events:
  claim L=40 c=0 T=40 hard=1
  prefill S=46 c=1 P=0
  retry
  retry
  retry
expect:
  t1 code=deferred id=0 a=40 b=46
  t2 code=deferred id=0 a=40 b=46
  t3 code=refused_claim id=0 a=40 b=46 n16=1
  t4 code=noop id=-1 a=0 b=0
  tel n_deferred=2 n_refused_claim=1 retry_refused=1 queued=0
  claim0 blocked=3

# The queue holds at most max_live_requests requests: the second blocked prefill is refused.
[pool queue_full]
usable = 68
mode = hard
chains = 2
defer_limit = 3
max_requests = 1
events:
  claim L=40 c=0 T=40 hard=1
  prefill S=46 c=1 P=0
  prefill S=46 c=1 P=0
  retry
expect:
  t1 code=deferred
  t2 code=refused_claim id=0 a=40 b=46
  t3 code=deferred id=0 a=40 b=46
  tel n_deferred=2 n_refused_claim=1 retry_refused=0 retry_served=0 queued=1 status=0

# A full live-request table turns the RETRY into INVALID and keeps the request queued; the next
# RETRY, after the live request finished, refuses it for good (its 10 blocks are now cached and
# evictable, but 28 + 10 < 46 and the claim still protects 40).
[pool retry_table_full]
usable = 68
mode = hard
chains = 2
defer_limit = 1
max_requests = 1
events:
  claim L=40 c=0 T=40 hard=1
  prefill S=46 c=1 P=0
  prefill S=10
  retry
  finish sel=0
  retry
expect:
  t1 code=deferred
  t2 code=admit id=2 b=0
  t3 code=invalid id=-1 a=0 b=0
  t4 code=finished id=2 a=10 b=0
  t5 code=refused_claim id=0 a=40 b=46
  tel status=1 retry_refused=1 queued=0 n_deferred=1

# A capacity refusal (the active side alone exceeds U) is never deferred.
[pool capacity_not_deferred]
usable = 68
mode = hard
chains = 2
defer_limit = 3
events:
  claim L=40 c=0 T=40 hard=1
  prefill S=70 c=1 P=0
  retry
expect:
  t1 code=refused_capacity id=-1 a=40 b=70 n16=0
  t2 code=noop
  tel n_deferred=0 queued=0 n_refused_capacity=1

# Other policies never attribute a refusal to claims, so they never defer.
[pool soft_never_defers]
usable = 68
mode = soft
chains = 2
defer_limit = 3
events:
  claim L=40 c=0 T=40 hard=1
  prefill S=46 c=1 P=0
  retry
expect:
  t1 code=evict_resident id=1 a=18 flags=pred_fail|harm
  t2 code=noop
  tel n_deferred=0 queued=0

# FIFO retries; the request served late keeps id 1 and sits before request 3 in the live set, so
# FINISH selector 0 finishes it first.  The second deferred request (30 blocks) no longer fits
# next to 51 active blocks: capacity refusal, 51 + 30 = 81 > 68.
[pool fifo_and_id_order]
usable = 68
mode = hard
chains = 2
defer_limit = 1
events:
  claim L=40 c=0 T=40 hard=1
  prefill S=46 c=1 P=0
  prefill S=30 c=1 P=0
  prefill S=5
  release sel=0
  retry
  retry
  finish sel=0
  finish sel=0
expect:
  t1 code=deferred id=0 a=40 b=46
  t2 code=deferred id=0 a=40 b=30
  t3 code=admit id=3
  t5 code=admit id=1 a=0 b=0 flags=evict_unclaimed
  t6 code=refused_capacity id=-1 a=0 b=81
  t7 code=finished id=1 a=46
  t8 code=finished id=3 a=5
  tel n_deferred=2 retry_served=1 retry_refused=1 queued=0 live_requests=0
"""


def fixtures():
    return gf.parse_text(DEFERRAL_CASES, "deferral closed forms")
