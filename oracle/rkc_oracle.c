/*
 * rkc_oracle.c -- plain, slow, single-threaded reference replay of the resident-KV-claim contract.
 *
 * TEST INFRASTRUCTURE.  Only the test suite, the smoke check and the benchmark's CPU-baseline leg
 * load this library.  It shares no code, header, table or helper with the HIP library: the record
 * layouts below are this file's own copy of the documented ABI layouts.
 *
 * The pool is kept one block at a time, exactly as the contract is stated:
 *   - a block is FREE, ACTIVE (refcount > 0) or CACHED (refcount 0, content kept); it holds a
 *     content position (shared chain, pos) or a request-private position, a last-use step, and
 *     whether it sits in the prefix-reuse index (paged KV with prefix caching, §2.1; one block per
 *     (chain, pos) in the index, §4.1 ledger rule "block ids map one-to-one to prefix positions");
 *   - claims carry the §3.1 schema fields (id, chain, footprint L, predicate threshold T,
 *     protection mode, priority, optional duration) plus decision, state and step telemetry;
 *   - every step runs: expiry, validation, dispatch, predicate sweep, emission;
 *   - a pool that defers (active deferral, §3.5) queues a prefill refused on behalf of resident
 *     claims; RETRY events later serve it, defer it again or refuse it for good;
 *   - a pool that relaxes demotes demotable hard claims when that lets an active request be served.
 *
 * Nothing here relies on the prefix shape of what survives: hits are the leading registered run,
 * the predicate walks the reuse index from position 0, victims are chosen by sorting every
 * candidate block on its key.  Structural invariants are checked after every step and reported
 * through a separate check word (never through the replay outputs).
 *
 * Readings of the paper used where it is silent are listed in the design notes; each is marked
 * "reading" where it is applied.
 *
 * Parity unpinned (the paper fixes no value that could catch a mistake in these; the brute-force
 * model shares the reading, so agreement with it checks the code, not the reading):
 *   - the victim key order (level, last use, position descending): the paper prints only the
 *     counts of its probe (50 evicted, 10 remain);
 *   - the offload and restore accounting (pool words 38-41): the paper fixes only the precondition
 *     of offloading (§3.1 offloadable; §3.5 offload resident).
 */
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

/* ---- this file's copy of the record layouts -------------------------------------------------- */
enum { EV_PREFILL = 0, EV_EXTEND = 1, EV_CLAIM = 2, EV_FINISH = 3, EV_RELEASE = 4, EV_DEMOTE = 5,
       EV_NOP = 6, EV_RETRY = 7 };
enum { MODE_LRU = 0, MODE_SOFT = 1, MODE_NOADMIT = 2, MODE_HARD = 3, MODE_RELAX_FLAG = 16 };
enum { OC_ADMIT = 0, OC_EVICT_RESIDENT = 1, OC_REFUSED_CLAIM = 2, OC_REFUSED_CAPACITY = 3,
       OC_MATFAIL = 4, OC_DEMOTED = 5, OC_RELEASED = 6, OC_FINISHED = 7, OC_NOOP = 8,
       OC_INVALID = 9, OC_DEFERRED = 10, OC_RELAXED = 11 };
enum { FL_EXPIRED = 1, FL_PRED_FAIL = 2, FL_HARM = 4, FL_POST_RELEASE = 8, FL_UNCLAIMED = 16,
       FL_NOADMIT_DROP = 32, FL_LOWERED = 64, FL_SHADOW = 128 };
enum { DEC_NONE = 0, DEC_ACCEPTED = 1, DEC_APPROX = 2, DEC_SHADOW = 3, DEC_REJECTED = 4 };
enum { ST_SUBMITTED = 0, ST_OBSERVED = 1, ST_MATERIALIZED = 2, ST_DEMOTED = 3, ST_EXPIRED = 4,
       ST_RELEASED = 5, ST_HARMED = 6, ST_REJECTED = 7 };
enum { PROT_NONE = 0, PROT_SOFT = 1, PROT_HARD = 2, PROT_OFFLOADED = 3 };
enum { PS_REQ_TABLE = 1, PS_CLAIM_TABLE = 2, PS_SLOT_TABLE = 4 };
enum { BLK_FREE = 0, BLK_ACTIVE = 1, BLK_CACHED = 2 };

/* pool telemetry word indices */
enum { T_VICTIMS = 10, T_RESIDENT = 11, T_POSTREL = 12, T_DROPPED = 13, T_HITS = 14,
       T_ACCEPTED = 15, T_APPROX = 16, T_SHADOW = 17, T_REJECTED = 18, T_HARM = 19,
       T_PREDFAIL = 20, T_EXPIRED = 21, T_DEMOTED = 22, T_RELEASED = 23, T_PEAK_ACTIVE = 24,
       T_ACTIVE = 25, T_CACHED = 26, T_FREE = 27, T_PROTECTED = 28, T_LIVE_REQ = 29,
       T_LIVE_CLAIMS = 30, T_STATUS = 31, T_DEFERRED = 32, T_RETRY_SERVED = 33,
       T_RETRY_REFUSED = 34, T_QUEUED = 35, T_RELAXED = 36, T_RUNTIME_DEMOTED = 37, T_OFF_CLAIMS = 38,
       T_OFF_BLOCKS = 39, T_RESTORED = 40, T_T2_PEAK = 41, N_TEL = 64 };

/* invariant check bits (oracle-only diagnostics) */
enum {
  CHK_COUNTS = 1,        /* I1: ACTIVE + CACHED + FREE = U, counters agree with the blocks      */
  CHK_HARD_VICTIM = 2,   /* I2: a block covered by a materialized hard claim became a victim    */
  CHK_HARD_HARM = 4,     /* I3: a hard claim in a hard-protection pool was harmed               */
  CHK_SHADOW_POOL = 8,   /* I4: a claim was accepted or harmed in an LRU / no-admit pool         */
  CHK_REFUSAL = 16,      /* I6: refusal identity Pr + req > U, attribution preconditions        */
  CHK_INDEX = 32,        /* I7: two blocks registered for one (chain, pos)                       */
  CHK_TRANSITION = 64,   /* I8: a claim state change outside the lifecycle graph                */
  CHK_KEY_TIE = 128,     /* I9: two candidates with equal (level, last_use, pos)                */
  CHK_PREFIX = 256,      /* registered positions of a chain are not exactly [0, n)              */
  CHK_REFCOUNT = 512,    /* a block's refcount disagrees with the live requests holding it      */
  CHK_ALLOC = 1024       /* internal: allocation bookkeeping failed                             */
};

#define MAX_FIELD_BLOCKS (1 << 24)
#define N16_MAX 65535

typedef struct {
  int32_t state;      /* BLK_*                                                             */
  int32_t chain;      /* shared chain id, or -1 when the position is private to a request  */
  int32_t owner;      /* request owning a private position, else -1                         */
  int32_t pos;        /* content position                                                   */
  int32_t last_use;   /* step of the last touch                                             */
  int32_t refcount;   /* live requests holding the block                                    */
  int32_t registered; /* in the prefix-reuse index                                          */
  int32_t producer;   /* request that computed the block, or -1 for a claim                 */
  int32_t mark;       /* scratch: member of the current hit set                             */
} block_t;

typedef struct {
  int32_t live;
  int32_t chain, P, h, S, len; /* shared chain, shared prefix, leading hits, size, private end */
  int32_t nblk, cap;
  int32_t* blk;                /* blocks held (hits, new blocks, extensions)                     */
} request_t;

typedef struct {
  int32_t has_slot, valid;
  int32_t id, chain, L, T, hard, prio, dur;
  int32_t decision, state, eff;
  int32_t accept, demote, expire, release, pred_fail, harm;
  int32_t blocked;
  int32_t demotable;   /* the client lets the runtime demote it (§3.1 demotable)               */
  int32_t best_effort; /* telemetry only (§3.1 best_effort)                                    */
  int32_t relaxed;     /* demoted or offloaded by the runtime to serve an active request        */
  int32_t offloadable; /* its content may move to the second tier (§3.1 offloadable)           */
  int32_t offloaded;   /* holds a second-tier copy: effective protection OFFLOADED              */
} claim_t;

/* A deferred active request waiting in the scheduler queue (active deferral, §3.5 mechanism table;
 * §5.4 live scheduler run).  It holds no blocks while it waits. */
typedef struct {
  int32_t id, S, chain, P; /* its PREFILL step and request fields */
  int32_t deferrals;       /* DEFERRED outcomes it has received   */
} deferred_t;

typedef struct {
  int32_t U, mode, n_events, n_chains, max_claims, max_reqs, n_slots, defer_limit;
  int32_t relax;   /* the runtime relaxes demotable hard claims before refusing (mode flag 16) */
  int32_t U2;      /* second-tier capacity in blocks                                        */
  int64_t t2_used; /* second-tier blocks held by offloaded claims                           */
  block_t* b;
  request_t* req;  /* indexed by request id (= step)           */
  claim_t* cl;     /* indexed by slot                          */
  int32_t n_cl;    /* CLAIM events seen so far (= slots used)  */
  int32_t* idx;    /* reuse index: idx[idx_off[c] + p]         */
  int64_t* idx_off;
  int32_t* idx_len;
  int32_t* tmp;    /* U ints of scratch                        */
  int32_t* taken;  /* U ints: blocks handed to the current event */
  int32_t* bucket_head; /* per chain: first live claim slot      */
  int32_t* bucket_next; /* per slot                              */
  int32_t* keyidx;
  int64_t* keys;
  deferred_t* dq;  /* FIFO of deferred requests: dq[dq_head .. dq_tail) */
  int32_t dq_head, dq_tail;
  int32_t check;
  int32_t tel[N_TEL];
} pool_t;

/* ---- small helpers ---------------------------------------------------------------------------- */
static int32_t imin(int32_t a, int32_t b) { return a < b ? a : b; }

static int claim_live(const claim_t* q) {
  /* live: still tracked by the runtime (not rejected, not released) */
  return q->valid && (q->state == ST_OBSERVED || q->state == ST_MATERIALIZED ||
                      q->state == ST_DEMOTED || q->state == ST_EXPIRED || q->state == ST_HARMED);
}

/* Lifecycle graph (§3.1 state list, §3.2 harm table): submitted -> materialized / observed /
 * rejected; materialized -> demoted / expired / released / harmed; demoted -> expired / released;
 * expired, harmed, observed -> released. */
static void set_state(pool_t* p, claim_t* q, int32_t to) {
  int from = q->state, ok = 0;
  switch (from) {
    case ST_SUBMITTED: ok = (to == ST_MATERIALIZED || to == ST_OBSERVED || to == ST_REJECTED); break;
    case ST_MATERIALIZED: ok = (to == ST_DEMOTED || to == ST_EXPIRED || to == ST_RELEASED || to == ST_HARMED); break;
    case ST_DEMOTED: ok = (to == ST_EXPIRED || to == ST_RELEASED); break;
    case ST_EXPIRED: case ST_HARMED: case ST_OBSERVED: ok = (to == ST_RELEASED); break;
    default: ok = 0;
  }
  if (!ok) p->check |= CHK_TRANSITION;
  q->state = to;
}

static int32_t* idx_at(pool_t* p, int32_t c, int32_t pos) {
  if (c < 0 || c >= p->n_chains || pos < 0 || pos >= p->idx_len[c]) return NULL;
  return &p->idx[p->idx_off[c] + pos];
}

/* Leading registered length of chain c: the first position with no block in the reuse index
 * (§4.1: cached tokens = first missing block x 16). */
static int32_t lead(pool_t* p, int32_t c) {
  int32_t n = 0;
  int32_t* slot;
  while ((slot = idx_at(p, c, n)) != NULL && *slot >= 0) n++;
  return n;
}

/* Materialization predicate (§3.1 "useful resident value"; §4.1; §5.4 L6): the leading contiguous
 * registered run of the claim's chain, capped at its footprint L, reaches the threshold T.
 * Survivors after the first missing position do not count. */
static int pred_holds(pool_t* p, const claim_t* q) {
  return imin(lead(p, q->chain), q->L) >= q->T;
}

/* covers(q, b): q is live and b is the registered block of one of q's positions [0, L). */
static int covers(const claim_t* q, const block_t* b) {
  return claim_live(q) && b->registered && b->chain == q->chain && b->pos < q->L;
}

/* Per-chain lists of live claims, rebuilt before each use (keeps per-block questions cheap). */
static void build_buckets(pool_t* p) {
  for (int32_t c = 0; c < p->n_chains; c++) p->bucket_head[c] = -1;
  for (int32_t s = p->n_cl - 1; s >= 0; s--) {
    claim_t* q = &p->cl[s];
    p->bucket_next[s] = -1;
    if (!claim_live(q)) continue;
    p->bucket_next[s] = p->bucket_head[q->chain];
    p->bucket_head[q->chain] = s;
  }
}

/* Soft eviction level of a block: highest (prio + 1) over covering claims that rank victims --
 * accepted soft (or lowered) claims still materialized, and demoted claims (§3.1 soft_priority:
 * "may influence eviction order"; demotion turns hard into soft).  Zero in LRU / no-admit pools. */
static int32_t block_level(pool_t* p, const block_t* b) {
  if (p->mode != MODE_SOFT && p->mode != MODE_HARD) return 0;
  if (!b->registered || b->chain < 0) return 0;
  int32_t lv = 0;
  for (int32_t s = p->bucket_head[b->chain]; s >= 0; s = p->bucket_next[s]) {
    claim_t* q = &p->cl[s];
    if (!covers(q, b)) continue;
    if ((q->state == ST_MATERIALIZED && q->eff == PROT_SOFT) || q->state == ST_DEMOTED)
      if (q->prio + 1 > lv) lv = q->prio + 1;
  }
  return lv;
}

/* Hard protected-resident exclusion (§3.1 hard_protected; §5.3 "resident victim exclusion"):
 * a cached block covered by a materialized claim whose effective protection is hard. */
static int block_protected(pool_t* p, const block_t* b) {
  if (p->mode != MODE_HARD || b->state != BLK_CACHED) return 0;
  if (!b->registered || b->chain < 0) return 0;
  for (int32_t s = p->bucket_head[b->chain]; s >= 0; s = p->bucket_next[s]) {
    claim_t* q = &p->cl[s];
    if (covers(q, b) && q->state == ST_MATERIALIZED && q->eff == PROT_HARD) return 1;
  }
  return 0;
}

static void count_blocks(pool_t* p, int64_t* nfree, int64_t* nact, int64_t* ncached) {
  int64_t f = 0, a = 0, c = 0;
  for (int32_t i = 0; i < p->U; i++) {
    if (p->b[i].state == BLK_FREE) f++;
    else if (p->b[i].state == BLK_ACTIVE) a++;
    else c++;
  }
  *nfree = f; *nact = a; *ncached = c;
}

static void clear_block(block_t* b) {
  b->state = BLK_FREE; b->chain = -1; b->owner = -1; b->pos = -1; b->last_use = -1;
  b->refcount = 0; b->registered = 0; b->producer = -1; b->mark = 0;
}

static void unregister(pool_t* p, block_t* b, int32_t id) {
  if (!b->registered) return;
  int32_t* slot = idx_at(p, b->chain, b->pos);
  if (slot && *slot == id) *slot = -1; else p->check |= CHK_INDEX;
  b->registered = 0;
}

static void do_register(pool_t* p, int32_t id, int32_t c, int32_t pos) {
  int32_t* slot = idx_at(p, c, pos);
  if (!slot) { p->check |= CHK_INDEX; return; }
  if (*slot >= 0) { p->check |= CHK_INDEX; return; } /* I7: already registered */
  *slot = id;
  p->b[id].registered = 1;
}

static void req_push(request_t* r, int32_t blk) {
  if (r->nblk == r->cap) {
    r->cap = r->cap ? 2 * r->cap : 16;
    r->blk = (int32_t*)realloc(r->blk, (size_t)r->cap * sizeof(int32_t));
  }
  r->blk[r->nblk++] = blk;
}

/* ---- ALLOC --------------------------------------------------------------------------------------
 * Take `need` blocks: FREE blocks first; then the (need - F) candidates with the smallest key
 * (level asc, last_use asc, pos desc), where candidates are CACHED blocks that are neither in the
 * current hit set (marked) nor hard-protected.  Infeasible when need > F + |candidates|.
 * Victims are removed from the reuse index and classified by the claims covering them:
 * resident (some live claim covers it), post-release (every covering live claim was demoted or
 * expired first, §3.2), or unclaimed.  On success the chosen blocks are listed in p->taken.
 * ---------------------------------------------------------------------------------------------- */
typedef struct {
  int feasible;
  int64_t F, E;                 /* FREE blocks and evictable candidates before the event */
  int32_t victims, resident, post_release, unclaimed;
  int32_t unregistered;         /* victims that left the reuse index                      */
} alloc_t;

static int cmp_key(const void* x, const void* y) {
  const int64_t* a = (const int64_t*)x;
  const int64_t* b = (const int64_t*)y;
  for (int i = 0; i < 4; i++) {
    if (a[i] < b[i]) return -1;
    if (a[i] > b[i]) return 1;
  }
  return 0;
}

static alloc_t alloc_blocks(pool_t* p, int64_t need) {
  alloc_t r;
  memset(&r, 0, sizeof r);
  build_buckets(p);
  int64_t F = 0;
  for (int32_t i = 0; i < p->U; i++) if (p->b[i].state == BLK_FREE) F++;
  /* candidates with their keys: (level, last_use, -pos, block id) */
  int64_t* k = p->keys;
  int32_t nc = 0;
  for (int32_t i = 0; i < p->U; i++) {
    block_t* b = &p->b[i];
    if (b->state != BLK_CACHED || b->mark || block_protected(p, b)) continue;
    k[4 * nc + 0] = block_level(p, b);
    k[4 * nc + 1] = b->last_use;
    k[4 * nc + 2] = -(int64_t)b->pos;
    k[4 * nc + 3] = i;
    nc++;
  }
  r.F = F;
  r.E = nc;
  if (need > F + nc) { r.feasible = 0; return r; }
  r.feasible = 1;
  int32_t got = 0;
  for (int32_t i = 0; i < p->U && got < need; i++)
    if (p->b[i].state == BLK_FREE) p->taken[got++] = i;
  if (got < need) {
    qsort(k, (size_t)nc, 4 * sizeof(int64_t), cmp_key);
    for (int32_t j = 0; j + 1 < nc; j++)
      if (k[4 * j] == k[4 * j + 4] && k[4 * j + 1] == k[4 * j + 5] && k[4 * j + 2] == k[4 * j + 6])
        p->check |= CHK_KEY_TIE;
    int32_t nv = (int32_t)(need - got);
    for (int32_t j = 0; j < nv; j++) {
      int32_t id = (int32_t)k[4 * j + 3];
      block_t* b = &p->b[id];
      /* classify against the covering live claims */
      int covered = 0, covered_strict = 0, covered_hard = 0;
      if (b->registered && b->chain >= 0) {
        for (int32_t s = p->bucket_head[b->chain]; s >= 0; s = p->bucket_next[s]) {
          claim_t* q = &p->cl[s];
          if (!covers(q, b) || q->offloaded) continue;
          covered = 1;
          if (q->state != ST_DEMOTED && q->state != ST_EXPIRED) covered_strict = 1;
          if (p->mode == MODE_HARD && q->state == ST_MATERIALIZED && q->eff == PROT_HARD) covered_hard = 1;
        }
      }
      if (covered_hard) p->check |= CHK_HARD_VICTIM;
      r.victims++;
      if (covered) {
        r.resident++;
        if (!covered_strict) r.post_release++;
      } else {
        r.unclaimed++;
      }
      if (b->registered) r.unregistered++;
      unregister(p, b, id);
      p->taken[got++] = id;
    }
  }
  /* hand the blocks over as blank FREE blocks; the caller gives them their new content */
  for (int32_t j = 0; j < got; j++) clear_block(&p->b[p->taken[j]]);
  return r;
}

/* ---- event-level helpers --------------------------------------------------------------------- */

/* Leading hits of a request or claim on chain c over positions [0, upto): the registered run
 * starting at position 0 (vLLM-style prefix hit; §4.1 "survived positions form leading ranges"). */
static int32_t leading_hits(pool_t* p, int32_t c, int32_t upto) {
  int32_t h = 0;
  int32_t* slot;
  while (h < upto && (slot = idx_at(p, c, h)) != NULL && *slot >= 0) h++;
  return h;
}

static void mark_hits(pool_t* p, int32_t c, int32_t h, int32_t on) {
  for (int32_t pos = 0; pos < h; pos++) p->b[*idx_at(p, c, pos)].mark = on;
}

/* Refusal record for an active event that cannot be served (§3.4 boundary; §5.4 record):
 * A = ACTIVE blocks, Hc = hits that are CACHED, Pr = protected CACHED blocks outside the hits,
 * req = A + Hc + need (active live required).  Infeasible exactly when Pr + req > U.
 * Attributed to the protecting claims when Pr > 0 and the active side alone would fit (req <= U);
 * otherwise a plain capacity refusal. */
static void refusal(pool_t* p, int64_t need, int32_t t, int32_t* o) {
  build_buckets(p);
  int64_t A = 0, Hc = 0, Pr = 0;
  for (int32_t i = 0; i < p->U; i++) {
    block_t* b = &p->b[i];
    if (b->state == BLK_ACTIVE) A++;
    if (b->state == BLK_CACHED && b->mark) Hc++;
    if (b->state == BLK_CACHED && !b->mark && block_protected(p, b)) Pr++;
  }
  int64_t req = A + Hc + need;
  if (!(Pr + req > p->U)) p->check |= CHK_REFUSAL;
  int32_t code, id = -1, n16 = 0;
  if (Pr > 0 && req <= p->U) {
    code = OC_REFUSED_CLAIM;
    if (p->mode != MODE_HARD) p->check |= CHK_REFUSAL;
    /* B: materialized hard claims covering at least one protected block outside the hits */
    for (int32_t s = 0; s < p->n_cl; s++) {
      claim_t* q = &p->cl[s];
      if (!(claim_live(q) && q->state == ST_MATERIALIZED && q->eff == PROT_HARD)) continue;
      int blocking = 0;
      for (int32_t pos = 0; pos < q->L && !blocking; pos++) {
        int32_t* slot = idx_at(p, q->chain, pos);
        if (!slot || *slot < 0) continue;
        block_t* b = &p->b[*slot];
        if (b->state == BLK_CACHED && !b->mark) blocking = 1;
      }
      if (!blocking) continue;
      if (id < 0 || q->id < id) id = q->id;
      n16++;
      q->blocked++;
    }
    if (n16 == 0) p->check |= CHK_REFUSAL;
  } else {
    code = OC_REFUSED_CAPACITY;
  }
  (void)t;
  o[0] = code;
  o[1] = id;
  o[2] = (int32_t)Pr;
  o[3] = (int32_t)req;
  o[4] = n16 > N16_MAX ? N16_MAX : n16;
}

static int32_t live_requests(pool_t* p, int32_t t, int32_t* list) {
  int32_t n = 0;
  for (int32_t r = 0; r < t; r++) if (p->req[r].live) list[n++] = r;
  return n;
}

static int32_t count_active(pool_t* p) {
  int32_t a = 0;
  for (int32_t i = 0; i < p->U; i++) a += p->b[i].state == BLK_ACTIVE;
  return a;
}

/* FREE blocks plus eviction candidates (CACHED, outside the current hit set, not hard-protected). */
static int64_t available(pool_t* p) {
  build_buckets(p);
  int64_t n = 0;
  for (int32_t i = 0; i < p->U; i++) {
    block_t* b = &p->b[i];
    if (b->state == BLK_FREE) n++;
    else if (b->state == BLK_CACHED && !b->mark && !block_protected(p, b)) n++;
  }
  return n;
}

/* Runtime relaxation before an active allocation of `need` blocks (hits already marked): §3.1
 * demotable (the downgrade must come before the predicate-breaking eviction) and offloadable (the
 * content may leave GPU memory if the predicate stays restorable); §3.5 "relax resident claim" and
 * "offload resident" (the active side is served by demoting or offloading resident state, the
 * latter subject to restore cost).  When the pool relaxes and hard protection makes the allocation
 * infeasible, the claims blocking it (materialized hard claims covering a cached block outside the
 * hits, as for attribution) that allow demotion or offload are taken lowest priority first, then
 * lowest id: each is offloaded when it allows it and its footprint fits the second tier's free
 * capacity, else demoted when it allows it, else left alone, until the allocation fits.  If it never
 * fits, nothing changes.  Returns the number of claims relaxed. */
static int32_t relax(pool_t* p, int64_t need, int32_t t) {
  if (p->mode != MODE_HARD || !p->relax) return 0;
  if (need <= available(p)) return 0;
  int32_t* order = p->tmp;  /* max(events, U) entries: at least one per claim slot */
  int32_t n = 0;
  for (int32_t s = 0; s < p->n_cl; s++) {
    claim_t* q = &p->cl[s];
    if (!(claim_live(q) && q->state == ST_MATERIALIZED && q->eff == PROT_HARD &&
          (q->demotable || q->offloadable))) continue;
    int blocking = 0;
    for (int32_t pos = 0; pos < q->L && !blocking; pos++) {
      int32_t* slot = idx_at(p, q->chain, pos);
      if (!slot || *slot < 0) continue;
      block_t* b = &p->b[*slot];
      if (b->state == BLK_CACHED && !b->mark) blocking = 1;
    }
    if (blocking) order[n++] = s;
  }
  /* insertion sort by (priority, id) */
  for (int32_t i = 1; i < n; i++) {
    int32_t v = order[i], j = i;
    while (j > 0 && (p->cl[order[j - 1]].prio > p->cl[v].prio ||
                     (p->cl[order[j - 1]].prio == p->cl[v].prio && p->cl[order[j - 1]].id > p->cl[v].id))) {
      order[j] = order[j - 1];
      j--;
    }
    order[j] = v;
  }
  /* tentative picks: 1 offload, 2 demote, 0 left alone */
  int32_t* pick = (int32_t*)malloc((size_t)(n > 0 ? n : 1) * sizeof(int32_t));
  int64_t room = (int64_t)p->U2 - p->t2_used;
  int fits = 0;
  int32_t k = 0;
  for (; k < n && !fits; k++) {
    claim_t* q = &p->cl[order[k]];
    pick[k] = 0;
    if (q->offloadable && q->L <= room) {
      pick[k] = 1;
      q->eff = PROT_OFFLOADED;
      room -= q->L;
    } else if (q->demotable) {
      pick[k] = 2;
      q->state = ST_DEMOTED;
    } else {
      continue;
    }
    fits = need <= available(p);
  }
  int32_t relaxed = 0;
  for (int32_t j = 0; j < k; j++) {
    claim_t* q = &p->cl[order[j]];
    if (pick[j] == 1) {
      if (fits) {
        q->offloaded = 1; q->relaxed = 1;
        p->t2_used += q->L;
        p->tel[T_OFF_CLAIMS]++; p->tel[T_OFF_BLOCKS] += q->L;
        relaxed++;
      } else {
        q->eff = PROT_HARD;
      }
    } else if (pick[j] == 2) {
      q->state = ST_MATERIALIZED;
      if (fits) {
        set_state(p, q, ST_DEMOTED);
        q->demote = t; q->relaxed = 1;
        p->tel[T_RUNTIME_DEMOTED]++;
        relaxed++;
      }
    }
  }
  if (p->t2_used > p->tel[T_T2_PEAK]) p->tel[T_T2_PEAK] = (int32_t)p->t2_used;
  free(pick);
  return relaxed;
}

/* Positions [h, P) of chain c that a claim holding a second-tier copy covers: a served prefill
 * takes them from the second tier instead of recomputing them (the restore cost, §3.5 "offload
 * resident"); they still take new GPU blocks like any position past the hits. */
static int32_t restorable(pool_t* p, int32_t c, int32_t h, int32_t Pp) {
  int32_t e = 0;
  for (int32_t s = 0; s < p->n_cl; s++) {
    claim_t* q = &p->cl[s];
    if (claim_live(q) && q->offloaded && q->chain == c && q->L > e) e = q->L;
  }
  int32_t top = imin(Pp, e);
  return top > h ? top - h : 0;
}

/* Serve an active prefill of request rid (S blocks, shared chain c, shared prefix P) at step t: the
 * chain's leading registered run below P is hit and the rest allocated (§3.4 feasibility).  Served:
 * returns 1 with o = {code, id, a, b, n16 = -1}; the blocks turn ACTIVE, last used at t, produced by
 * rid, and shared positions below P enter the reuse index unless the pool is write no-admit (§1,
 * §5.2).  Not servable: returns 0 with the refusal record in o. */
static int serve_prefill(pool_t* p, int32_t t, int32_t rid, int32_t S, int32_t c, int32_t Pp,
                         int32_t* o, int32_t* flags, int* unregistered) {
  int32_t h = Pp > 0 ? leading_hits(p, c, Pp) : 0;
  int64_t need = (int64_t)S - h;
  if (h) mark_hits(p, c, h, 1);
  int32_t relaxed = relax(p, need, t);
  alloc_t r = alloc_blocks(p, need);
  if (!r.feasible) {
    refusal(p, need, t, o);
    if (h) mark_hits(p, c, h, 0);
    return 0;
  }
  if (h) mark_hits(p, c, h, 0);
  request_t* rq = &p->req[rid];
  rq->live = 1; rq->chain = Pp > 0 ? c : -1; rq->P = Pp; rq->h = h; rq->S = S; rq->len = S;
  for (int32_t pos = 0; pos < h; pos++) {
    int32_t bid = *idx_at(p, c, pos);
    block_t* b = &p->b[bid];
    b->refcount++; b->state = BLK_ACTIVE; b->last_use = t;
    req_push(rq, bid);
  }
  for (int64_t j = 0; j < need; j++) {
    int32_t bid = p->taken[j];
    block_t* b = &p->b[bid];
    int32_t pos = h + (int32_t)j;
    b->state = BLK_ACTIVE; b->refcount = 1; b->last_use = t; b->producer = rid; b->pos = pos;
    if (pos < Pp) {
      b->chain = c;
      if (p->mode != MODE_NOADMIT) do_register(p, bid, c, pos);
    } else {
      b->chain = -1; b->owner = rid;
    }
    req_push(rq, bid);
  }
  o[0] = relaxed ? OC_RELAXED : r.resident > 0 ? OC_EVICT_RESIDENT : OC_ADMIT;
  o[1] = rid; o[2] = r.resident; o[3] = h; o[4] = relaxed ? relaxed : -1;
  if (Pp > h) p->tel[T_RESTORED] += restorable(p, c, h, Pp);
  if (r.post_release) *flags |= FL_POST_RELEASE;
  if (r.unclaimed) *flags |= FL_UNCLAIMED;
  p->tel[T_VICTIMS] += r.victims; p->tel[T_RESIDENT] += r.resident;
  p->tel[T_POSTREL] += r.post_release; p->tel[T_HITS] += h;
  *unregistered += r.unregistered;
  return 1;
}

/* ---- one pool ---------------------------------------------------------------------------------- */

static void pool_free(pool_t* p) {
  if (p->req) for (int32_t r = 0; r < p->n_events; r++) free(p->req[r].blk);
  free(p->b); free(p->req); free(p->cl); free(p->idx); free(p->idx_off); free(p->idx_len);
  free(p->tmp); free(p->taken); free(p->bucket_head); free(p->bucket_next); free(p->keys);
  free(p->dq);
}

static int pool_init(pool_t* p, const int32_t* d, const int32_t* ev) {
  memset(p, 0, sizeof *p);
  p->U = d[0]; p->mode = d[1] & ~MODE_RELAX_FLAG; p->relax = (d[1] & MODE_RELAX_FLAG) != 0;
  p->U2 = d[8];
  if (p->U2 < 0 || d[9] != 0 || d[10] != 0 || d[11] != 0) return -1;
  p->n_events = d[2]; p->n_chains = d[3];
  p->max_claims = d[4]; p->max_reqs = d[5]; p->n_slots = d[6]; p->defer_limit = d[7];
  if (p->U < 1 || p->n_events < 0 || p->n_chains < 0 || p->n_slots < 0 || p->defer_limit < 0)
    return -1;
  size_t U = (size_t)p->U, E = (size_t)(p->n_events > 0 ? p->n_events : 1);
  size_t NC = (size_t)(p->n_chains > 0 ? p->n_chains : 1);
  p->b = (block_t*)malloc(U * sizeof(block_t));
  p->req = (request_t*)calloc(E, sizeof(request_t));
  p->cl = (claim_t*)calloc((size_t)(p->n_slots > 0 ? p->n_slots : 1), sizeof(claim_t));
  p->idx_off = (int64_t*)calloc(NC, sizeof(int64_t));
  p->idx_len = (int32_t*)calloc(NC, sizeof(int32_t));
  p->tmp = (int32_t*)malloc((E > U ? E : U) * sizeof(int32_t));
  p->taken = (int32_t*)malloc(U * sizeof(int32_t));
  p->bucket_head = (int32_t*)malloc(NC * sizeof(int32_t));
  p->bucket_next = (int32_t*)malloc((size_t)(p->n_slots > 0 ? p->n_slots : 1) * sizeof(int32_t));
  p->keys = (int64_t*)malloc(U * 4 * sizeof(int64_t));
  p->dq = (deferred_t*)malloc(E * sizeof(deferred_t)); /* each PREFILL is queued at most once */
  if (!p->b || !p->req || !p->cl || !p->idx_off || !p->idx_len || !p->tmp || !p->taken ||
      !p->bucket_head || !p->bucket_next || !p->keys || !p->dq) return -1;
  for (size_t i = 0; i < U; i++) clear_block(&p->b[i]);
  /* reuse-index extent per chain: the largest position any event could register */
  for (int32_t t = 0; t < p->n_events; t++) {
    const int32_t* e = ev + 4 * (size_t)t;
    int32_t type = e[0] & 15, c = e[2], ext = 0;
    if (type == EV_PREFILL) ext = e[3];
    else if (type == EV_CLAIM) ext = e[1];
    else continue;
    if (c < 0 || c >= p->n_chains || ext <= 0 || ext > MAX_FIELD_BLOCKS) continue;
    if (ext > p->idx_len[c]) p->idx_len[c] = ext;
  }
  int64_t total = 0;
  for (int32_t c = 0; c < p->n_chains; c++) { p->idx_off[c] = total; total += p->idx_len[c]; }
  p->idx = (int32_t*)malloc((size_t)(total > 0 ? total : 1) * sizeof(int32_t));
  if (!p->idx) return -1;
  for (int64_t i = 0; i < total; i++) p->idx[i] = -1;
  for (int i = 0; i < N_TEL; i++) p->tel[i] = 0;
  return 0;
}

/* Structural invariants after a step (oracle diagnostics only). */
static void check_step(pool_t* p, int32_t t) {
  int64_t f, a, c;
  count_blocks(p, &f, &a, &c);
  if (f + a + c != p->U) p->check |= CHK_COUNTS;
  /* refcounts = number of live requests holding the block */
  for (int32_t i = 0; i < p->U; i++) p->tmp[i] = 0;
  for (int32_t r = 0; r < t + 1 && r < p->n_events; r++)
    if (p->req[r].live)
      for (int32_t j = 0; j < p->req[r].nblk; j++) p->tmp[p->req[r].blk[j]]++;
  for (int32_t i = 0; i < p->U; i++) {
    block_t* b = &p->b[i];
    if (b->refcount != p->tmp[i]) p->check |= CHK_REFCOUNT;
    if ((b->state == BLK_ACTIVE) != (b->refcount > 0)) p->check |= CHK_REFCOUNT;
  }
  /* registered positions of every chain are exactly [0, lead) */
  for (int32_t ch = 0; ch < p->n_chains; ch++) {
    int32_t n = lead(p, ch);
    for (int32_t pos = n; pos < p->idx_len[ch]; pos++)
      if (p->idx[p->idx_off[ch] + pos] >= 0) { p->check |= CHK_PREFIX; break; }
  }
  for (int32_t s = 0; s < p->n_cl; s++) {
    claim_t* q = &p->cl[s];
    if (!q->valid) continue;
    if ((p->mode == MODE_LRU || p->mode == MODE_NOADMIT) &&
        (q->decision == DEC_ACCEPTED || q->decision == DEC_APPROX || q->state == ST_HARMED))
      p->check |= CHK_SHADOW_POOL;
    if (p->mode == MODE_HARD && q->eff == PROT_HARD && q->state == ST_HARMED && q->demote < 0)
      p->check |= CHK_HARD_HARM;
  }
}

static int replay_pool(const int32_t* d, const int32_t* ev, int32_t* out, int32_t* ptel,
                       int32_t* ctel, int32_t* check) {
  pool_t P;
  pool_t* p = &P;
  if (pool_init(p, d, ev) != 0) { pool_free(p); return -1; }
  int32_t* livebuf = (int32_t*)malloc((size_t)(p->n_events > 0 ? p->n_events : 1) * sizeof(int32_t));
  int32_t peak = 0;

  for (int32_t t = 0; t < p->n_events; t++) {
    const int32_t* e = ev + 4 * (size_t)t;
    uint32_t w0 = (uint32_t)e[0];
    int32_t type = (int32_t)(w0 & 15u), hard = (int32_t)((w0 >> 4) & 1u);
    int32_t prio = (int32_t)((w0 >> 5) & 3u), dur = (int32_t)(w0 >> 16);
    int32_t code = OC_NOOP, flags = 0, id = -1, a = 0, bb = 0, n16 = -1;
    int unregistered = 0;

    /* 1. expiry at the start of the step: responsibility ends at accept + duration (§3.1
     *    "expiring"; reading: a demoted claim can still expire, shadow claims never expire). */
    int32_t expired = 0;
    for (int32_t s = 0; s < p->n_cl; s++) {
      claim_t* q = &p->cl[s];
      if (!q->valid || q->dur <= 0) continue;
      if ((q->state == ST_MATERIALIZED || q->state == ST_DEMOTED) && q->accept + q->dur <= t) {
        set_state(p, q, ST_EXPIRED);
        q->expire = t;
        expired++;
        if (q->offloaded) {  /* responsibility ends: the second-tier copy is dropped */
          p->t2_used -= q->L; q->offloaded = 0; q->eff = PROT_NONE;
          /* its predicate held only through the copy: without it, a chain already shorter than
           * T fails the predicate now (§3.1 offloadable: only while it stays restorable) */
          if (q->pred_fail < 0 && !pred_holds(p, q)) {
            q->pred_fail = t;
            flags |= FL_PRED_FAIL;
            p->tel[T_PREDFAIL]++;
          }
        }
      }
    }
    if (expired) { flags |= FL_EXPIRED; p->tel[T_EXPIRED] += expired; }

    /* 2. validation */
    int invalid = 0;
    claim_t* slot = NULL;
    int32_t n_live_req = live_requests(p, t, livebuf);
    int32_t n_live_cl = 0;
    for (int32_t s = 0; s < p->n_cl; s++) n_live_cl += claim_live(&p->cl[s]);
    if (type == EV_PREFILL) {
      int32_t S = e[1], c = e[2], Pp = e[3];
      if (S < 1 || S > MAX_FIELD_BLOCKS || Pp < 0 || Pp > S || (Pp > 0 && (c < 0 || c >= p->n_chains)))
        invalid = 1;
      else if (n_live_req >= p->max_reqs) { invalid = 1; p->tel[T_STATUS] |= PS_REQ_TABLE; }
    } else if (type == EV_EXTEND) {
      if (e[1] < 1 || e[1] > MAX_FIELD_BLOCKS) invalid = 1;
    } else if (type == EV_CLAIM) {
      int32_t L = e[1], c = e[2], T = e[3];
      if (p->n_cl >= p->n_slots) { invalid = 1; p->tel[T_STATUS] |= PS_SLOT_TABLE; }
      else {
        slot = &p->cl[p->n_cl++];
        memset(slot, 0, sizeof *slot);
        slot->has_slot = 1;
        slot->id = t;
        slot->accept = slot->demote = slot->expire = slot->release = slot->pred_fail = slot->harm = -1;
        if (L < 1 || L > MAX_FIELD_BLOCKS || c < 0 || c >= p->n_chains || T < 0 || T > L) invalid = 1;
        else if (n_live_cl >= p->max_claims) { invalid = 1; p->tel[T_STATUS] |= PS_CLAIM_TABLE; }
      }
    } else if (type == EV_RETRY) {
      /* the retried request needs a live-request entry; without one it stays queued */
      if (p->dq_head < p->dq_tail && n_live_req >= p->max_reqs) {
        invalid = 1; p->tel[T_STATUS] |= PS_REQ_TABLE;
      }
    } else if (type > EV_RETRY) {
      invalid = 1;
    }

    if (invalid) {
      code = OC_INVALID;
    } else if (type == EV_PREFILL) {
      /* 3a. active prefill.  When the pool defers, a refusal attributed to resident claims queues
       *     the request instead (§3.5 mechanism table "active deferral"; §3.2 table: an accepted hard
       *     claim that blocks active admission yields an active refusal or deferral). */
      int32_t o[5];
      if (!serve_prefill(p, t, t, e[1], e[2], e[3], o, &flags, &unregistered) &&
          o[0] == OC_REFUSED_CLAIM && p->defer_limit > 0 && p->dq_tail - p->dq_head < p->max_reqs) {
        deferred_t* q = &p->dq[p->dq_tail++];
        q->id = t; q->S = e[1]; q->chain = e[2]; q->P = e[3]; q->deferrals = 1;
        o[0] = OC_DEFERRED;
      }
      code = o[0]; id = o[1]; a = o[2]; bb = o[3]; n16 = o[4];
    } else if (type == EV_RETRY) {
      /* 3e. the scheduler retries the oldest deferred request: it is served, deferred again while
       *     it has deferrals left, or refused for good (§5.4 live scheduler run: deferred once, then
       *     a terminal refusal). */
      if (p->dq_head == p->dq_tail) {
        code = OC_NOOP;
      } else {
        deferred_t* q = &p->dq[p->dq_head];
        int32_t o[5];
        if (serve_prefill(p, t, q->id, q->S, q->chain, q->P, o, &flags, &unregistered)) {
          p->dq_head++;
          p->tel[T_RETRY_SERVED]++;
        } else if (o[0] == OC_REFUSED_CLAIM && q->deferrals < p->defer_limit) {
          q->deferrals++;
          o[0] = OC_DEFERRED;
        } else {
          p->dq_head++;
          p->tel[T_RETRY_REFUSED]++;
        }
        code = o[0]; id = o[1]; a = o[2]; bb = o[3]; n16 = o[4];
      }
    } else if (type == EV_EXTEND) {
      /* 3b. decode / next chunk of a live request: new private blocks (§3.1 active live KV) */
      if (n_live_req == 0) {
        code = OC_NOOP;
      } else {
        int32_t rid = livebuf[(uint32_t)e[2] % (uint32_t)n_live_req];
        request_t* rq = &p->req[rid];
        int64_t need = e[1];
        int32_t relaxed = relax(p, need, t);
        alloc_t r = alloc_blocks(p, need);
        if (!r.feasible) {
          int32_t o[5];
          refusal(p, need, t, o);
          code = o[0]; id = o[1]; a = o[2]; bb = o[3]; n16 = o[4];
        } else {
          for (int64_t j = 0; j < need; j++) {
            int32_t bid = p->taken[j];
            block_t* b = &p->b[bid];
            b->state = BLK_ACTIVE; b->refcount = 1; b->last_use = t; b->producer = rid;
            b->chain = -1; b->owner = rid; b->pos = rq->len + (int32_t)j;
            req_push(rq, bid);
          }
          rq->len += (int32_t)need;
          code = relaxed ? OC_RELAXED : r.resident > 0 ? OC_EVICT_RESIDENT : OC_ADMIT;
          id = rid; a = r.resident; bb = count_active(p);
          if (relaxed) n16 = relaxed;
          if (r.post_release) flags |= FL_POST_RELEASE;
          if (r.unclaimed) flags |= FL_UNCLAIMED;
          p->tel[T_VICTIMS] += r.victims; p->tel[T_RESIDENT] += r.resident;
          p->tel[T_POSTREL] += r.post_release;
          unregistered += r.unregistered;
        }
      }
    } else if (type == EV_CLAIM) {
      /* 3c. resident claim: materialize [0, L) of chain c as reusable cache, then decide by the
       *     pool's policy (§3.1 decision; §5.4 C1 lowering; reading: all-or-nothing at once). */
      int32_t L = e[1], c = e[2], T = e[3];
      claim_t* q = slot;
      q->valid = 1; q->chain = c; q->L = L; q->T = T; q->hard = hard; q->prio = prio; q->dur = dur;
      q->demotable = (int32_t)((w0 >> 7) & 1u);
      q->offloadable = (int32_t)((w0 >> 9) & 1u);
      q->best_effort = (int32_t)((w0 >> 8) & 1u);
      /* a best-effort claim carries no preservation obligation: it is observed like a claim in a
       * pool that does not accept claims (§3.1 best_effort: telemetry only) */
      const int observe = p->mode == MODE_LRU || p->mode == MODE_NOADMIT || q->best_effort;
      q->eff = q->best_effort ? PROT_NONE
             : p->mode == MODE_HARD ? (hard ? PROT_HARD : PROT_SOFT)
             : p->mode == MODE_SOFT ? PROT_SOFT : PROT_NONE;
      int32_t h = leading_hits(p, c, L);
      int64_t need = (int64_t)L - h;
      if (h) mark_hits(p, c, h, 1);
      alloc_t r = alloc_blocks(p, need);
      if (h) mark_hits(p, c, h, 0);
      if (!r.feasible) {
        q->decision = observe ? DEC_SHADOW : DEC_REJECTED;
        set_state(p, q, ST_REJECTED);
        code = OC_MATFAIL; id = t; a = (int32_t)need; bb = (int32_t)(r.F + r.E);
      } else {
        for (int32_t pos = 0; pos < h; pos++) p->b[*idx_at(p, c, pos)].last_use = t;
        for (int64_t j = 0; j < need; j++) {
          int32_t bid = p->taken[j];
          block_t* b = &p->b[bid];
          b->state = BLK_CACHED; b->refcount = 0; b->last_use = t; b->producer = -1;
          b->chain = c; b->pos = h + (int32_t)j;
          do_register(p, bid, c, b->pos);
        }
        if (observe) {
          q->decision = DEC_SHADOW; set_state(p, q, ST_OBSERVED); flags |= FL_SHADOW;
        } else if (p->mode == MODE_SOFT && hard) {
          q->decision = DEC_APPROX; set_state(p, q, ST_MATERIALIZED); flags |= FL_LOWERED;
        } else {
          q->decision = DEC_ACCEPTED; set_state(p, q, ST_MATERIALIZED);
        }
        q->accept = t;
        code = r.resident > 0 ? OC_EVICT_RESIDENT : OC_ADMIT;
        id = t; a = r.resident; bb = (int32_t)need;
        if (r.post_release) flags |= FL_POST_RELEASE;
        if (r.unclaimed) flags |= FL_UNCLAIMED;
        p->tel[T_VICTIMS] += r.victims; p->tel[T_RESIDENT] += r.resident;
        p->tel[T_POSTREL] += r.post_release;
        unregistered += r.unregistered;
      }
      if (q->decision == DEC_ACCEPTED) p->tel[T_ACCEPTED]++;
      else if (q->decision == DEC_APPROX) p->tel[T_APPROX]++;
      else if (q->decision == DEC_SHADOW) p->tel[T_SHADOW]++;
      else if (q->decision == DEC_REJECTED) p->tel[T_REJECTED]++;
    } else if (type == EV_FINISH) {
      /* 3d. request finishes: its blocks lose one holder; a block nobody holds becomes reusable
       *     cache, except that write no-admit drops the blocks the request itself produced. */
      if (n_live_req == 0) {
        code = OC_NOOP;
      } else {
        int32_t rid = livebuf[(uint32_t)e[1] % (uint32_t)n_live_req];
        request_t* rq = &p->req[rid];
        int32_t turned = 0, dropped = 0;
        for (int32_t j = 0; j < rq->nblk; j++) {
          block_t* b = &p->b[rq->blk[j]];
          b->refcount--;
          b->last_use = t;
          if (b->refcount == 0) {
            if (p->mode == MODE_NOADMIT && b->producer == rid) {
              unregister(p, b, rq->blk[j]);
              clear_block(b);
              dropped++;
            } else {
              b->state = BLK_CACHED;
              turned++;
            }
          }
        }
        rq->live = 0;
        rq->nblk = 0;
        code = OC_FINISHED; id = rid; a = turned; bb = dropped;
        if (dropped) flags |= FL_NOADMIT_DROP;
        p->tel[T_DROPPED] += dropped;
      }
    } else if (type == EV_RELEASE) {
      int32_t n = 0;
      for (int32_t s = 0; s < p->n_cl; s++) if (claim_live(&p->cl[s])) livebuf[n++] = s;
      if (n == 0) {
        code = OC_NOOP;
      } else {
        claim_t* q = &p->cl[livebuf[(uint32_t)e[1] % (uint32_t)n]];
        set_state(p, q, ST_RELEASED);
        q->release = t;
        if (q->offloaded) { p->t2_used -= q->L; q->offloaded = 0; }
        code = OC_RELEASED; id = q->id; a = imin(lead(p, q->chain), q->L); bb = q->T;
        p->tel[T_RELEASED]++;
      }
    } else if (type == EV_DEMOTE) {
      /* hard -> soft (§3.1 demotable; §3.2: later loss is post-release, not harm) */
      int32_t n = 0;
      if (p->mode == MODE_SOFT || p->mode == MODE_HARD)
        for (int32_t s = 0; s < p->n_cl; s++) {
          claim_t* q = &p->cl[s];
          if (q->valid && q->state == ST_MATERIALIZED && q->hard && !q->offloaded) livebuf[n++] = s;
        }
      if (n == 0) {
        code = OC_NOOP;
      } else {
        claim_t* q = &p->cl[livebuf[(uint32_t)e[1] % (uint32_t)n]];
        set_state(p, q, ST_DEMOTED);
        q->demote = t;
        code = OC_DEMOTED; id = q->id; a = imin(lead(p, q->chain), q->L); bb = q->T;
        p->tel[T_DEMOTED]++;
      }
    } else {
      code = OC_NOOP;
    }

    /* 4. predicate sweep: a claim fails when its leading registered length drops below T;
     *    the first failure of a materialized (accepted) claim is harm (§3.2).  The predicate can
     *    only turn false when blocks leave the reuse index, so the sweep runs on those steps. */
    if (!invalid && unregistered > 0) {
      for (int32_t s = 0; s < p->n_cl; s++) {
        claim_t* q = &p->cl[s];
        if (!q->valid || q->pred_fail >= 0) continue;
        if (!(q->state == ST_OBSERVED || q->state == ST_MATERIALIZED || q->state == ST_DEMOTED ||
              q->state == ST_EXPIRED)) continue;
        if (q->offloaded || pred_holds(p, q)) continue;
        q->pred_fail = t;
        flags |= FL_PRED_FAIL;
        p->tel[T_PREDFAIL]++;
        if (q->state == ST_MATERIALIZED) {
          set_state(p, q, ST_HARMED);
          q->harm = t;
          flags |= FL_HARM;
          p->tel[T_HARM]++;
        }
      }
    }

    /* 5. emit */
    if (code == OC_INVALID || code == OC_NOOP) { id = -1; a = 0; bb = 0; }
    if (n16 < 0) n16 = expired > N16_MAX ? N16_MAX : expired;
    out[4 * (size_t)t + 0] = (int32_t)((uint32_t)code | ((uint32_t)flags << 8) | ((uint32_t)n16 << 16));
    out[4 * (size_t)t + 1] = id;
    out[4 * (size_t)t + 2] = a;
    out[4 * (size_t)t + 3] = bb;
    p->tel[code == OC_DEFERRED ? T_DEFERRED : code == OC_RELAXED ? T_RELAXED : code]++;
    int32_t act = count_active(p);
    if (act > peak) peak = act;
    check_step(p, t);
  }

  /* final pool telemetry */
  build_buckets(p);
  int64_t f, a, c;
  count_blocks(p, &f, &a, &c);
  int32_t prot = 0;
  for (int32_t i = 0; i < p->U; i++) prot += block_protected(p, &p->b[i]);
  int32_t nlr = live_requests(p, p->n_events, livebuf), nlc = 0;
  for (int32_t s = 0; s < p->n_cl; s++) nlc += claim_live(&p->cl[s]);
  p->tel[T_PEAK_ACTIVE] = peak; p->tel[T_ACTIVE] = (int32_t)a; p->tel[T_CACHED] = (int32_t)c;
  p->tel[T_FREE] = (int32_t)f; p->tel[T_PROTECTED] = prot; p->tel[T_LIVE_REQ] = nlr;
  p->tel[T_LIVE_CLAIMS] = nlc; p->tel[T_QUEUED] = p->dq_tail - p->dq_head;
  for (int i = 0; i < N_TEL; i++) ptel[i] = p->tel[i];

  /* claim telemetry, one slot per CLAIM event in step order; unused slots are blank */
  for (int32_t s = 0; s < p->n_slots; s++) {
    int32_t* w = ctel + 10 * (size_t)s;
    if (s >= p->n_cl) {
      w[0] = -1; w[1] = 0;
      for (int i = 2; i < 8; i++) w[i] = -1;
      w[8] = 0; w[9] = 0;
      continue;
    }
    claim_t* q = &p->cl[s];
    w[0] = q->id;
    w[1] = q->valid ? (q->decision | (q->state << 4) | (q->hard << 8) | (q->prio << 9) | (q->eff << 11) |
                       (q->demotable << 13) | (q->best_effort << 14) | (q->relaxed << 15) |
                       (q->offloadable << 16)) : 0;
    w[2] = q->accept; w[3] = q->demote; w[4] = q->expire; w[5] = q->release;
    w[6] = q->pred_fail; w[7] = q->harm; w[8] = q->blocked;
    w[9] = q->valid ? imin(lead(p, q->chain), q->L) : 0;
  }
  *check = p->check;
  free(livebuf);
  pool_free(p);
  return 0;
}

/* Batch entry: pools [first, first + count) of a batch laid out like the device ABI.
 * desc: 16 int32 per pool (64-byte records); events/outcomes: 4 int32 per event; pool_tel: 64 int32
 * per pool; claim_tel: 10 int32 per slot; check: one int32 per pool (invariant violation bits,
 * -1 when the pool could not be set up).  Returns the number of pools with a non-zero check. */
int rkc_oracle_replay(const int32_t* desc, int32_t first, int32_t count, const int32_t* events,
                      int32_t* outcomes, int32_t* pool_tel, int32_t* claim_tel, int32_t* check) {
  int bad = 0;
  for (int32_t i = first; i < first + count; i++) {
    const int32_t* d = desc + 16 * (size_t)i;
    int64_t ev_off = (int64_t)(uint32_t)d[12] | ((int64_t)d[13] << 32);
    int64_t cl_off = (int64_t)(uint32_t)d[14] | ((int64_t)d[15] << 32);
    int rc = replay_pool(d, events + 4 * ev_off, outcomes + 4 * ev_off, pool_tel + N_TEL * (size_t)i,
                         claim_tel + 10 * cl_off, &check[i]);
    if (rc != 0) check[i] = -1;
    if (check[i] != 0) bad++;
  }
  return bad;
}

/* Test hook: evaluate the materialization predicate of a claim (footprint L, threshold T) on a
 * chain whose registered positions are exactly those with registered[pos] != 0, pos < npos.
 * Lets the tests pin the predicate on survivor sets that replay can never produce (§5.4 L6). */
int rkc_oracle_predicate(const uint8_t* registered, int32_t npos, int32_t L, int32_t T) {
  pool_t P;
  memset(&P, 0, sizeof P);
  int32_t len = npos;
  int64_t off = 0;
  P.n_chains = 1;
  P.idx_len = &len;
  P.idx_off = &off;
  P.idx = (int32_t*)malloc((size_t)(npos > 0 ? npos : 1) * sizeof(int32_t));
  for (int32_t i = 0; i < npos; i++) P.idx[i] = registered[i] ? i : -1;
  claim_t q;
  memset(&q, 0, sizeof q);
  q.chain = 0; q.L = L; q.T = T;
  int r = pred_holds(&P, &q);
  free(P.idx);
  return r;
}
