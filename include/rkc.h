/*
 * rkc.h -- C ABI of the MI355X (gfx950) batched replay of resident-KV-claim arbitration.
 *
 * What is replayed.  Many independent paged-KV block pools, each driven by its own event trace,
 * through the resident-claim contract of "Resident KV Claims: A Conformance Contract for Future
 * Reuse under Active KV Pressure" (Stepanek, 2026):
 *   - the active/resident feasibility check  protected_resident + active_live <= usable  (§3.4);
 *   - ordinary (LRU) eviction, soft priority, write no-admit and hard protected claims as pool
 *     policies (§3.1 protection-mode table; §3.5 mechanism table; §5.2; §5.3);
 *   - the leading-prefix materialization predicate (§3.1 "useful resident value"; §4.1 ledger);
 *   - claim decisions, lifecycle, demotion, expiry and harm (§3.1 schema table; §3.2 harm table);
 *   - scheduler-visible active refusal with blocking-claim attribution and its capacity proof
 *     (§5.4 refusal record: protected 60, required 70, sum 130, usable 80, shortfall 50).
 *
 * Everything on this path is integer.  Conflicts are contract outcomes, not errors (§3.2, §7):
 * a refusal, a materialization failure or a harm is reported in the outcome stream; only bad calls
 * return a negative status.
 *
 * Ownership.  The caller owns every buffer (in practice torch tensors in device memory).  The
 * library allocates no device memory and is re-entrant for disjoint buffers on different streams;
 * its one piece of global state is the built-in scratch of rkc_replay_batch_noalloc (a fixed
 * per-device array, see there).  Every output buffer is fully overwritten by a replay, so callers
 * need not clear them.  Buffers must stay alive until the stream has finished the replay.
 *
 * All integers are little-endian.  Device pointers are HIP device addresses of the current device.
 */
#ifndef RKC_H
#define RKC_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define RKC_ABI_VERSION 5

/* Hard limits of this implementation (checked on the host and per pool on the device). */
#define RKC_MAX_USABLE_BLOCKS   (1 << 22) /* U per pool                                        */
#define RKC_MAX_EVENTS_PER_POOL (1 << 24) /* events per pool; request/claim ids are < this     */
#define RKC_MAX_FIELD_BLOCKS    (1 << 24) /* S, k, L, P, T above this make an event malformed  */
/* Size of the built-in device scratch that rkc_replay_batch_noalloc uses instead of a caller buffer. */
#define RKC_NOALLOC_SCRATCH_BYTES (64u << 20)

/* ----------------------------------------------------------------------------------------------
 * Event: 16 bytes = 4 x int32, pool-major (CSR by rkc_pool_desc.event_offset).
 *
 * w0 = type[0:4] | hard[4] | prio[5:7] | demotable[7] | best_effort[8] | offloadable[9]
 *      | reserved[10:16] | duration[16:32] (u16, 0 = no expiry); bits 4..9 and the duration matter
 *      for CLAIM only
 *
 *   PREFILL (0)  active request r = the event's step index.  w1 = S blocks, w2 = shared chain c
 *                (ignored when P = 0), w3 = shared prefix P (0 <= P <= S).  Positions [0,P) are
 *                content of shared chain c and can hit the prefix cache; positions [P,S) are
 *                private to r.  (§2.1 prefix caching; §4.1 leading-prefix ledger.)
 *   EXTEND  (1)  decode/chunk growth of a live request.  w1 = k blocks, w2 = selector (u32).  The
 *                request is the (selector mod #live)-th live request in ascending id order.
 *                (§3.1 "active live KV" grows across chunks; §5.2 chunked-prefill table.)
 *   CLAIM   (2)  resident claim q = the event's step index.  w1 = footprint L blocks, w2 = chain c,
 *                w3 = materialization threshold T (0 <= T <= L), hard/prio/duration from w0.
 *                (§3.1 ResidentClaimInput: footprint, protection mode, optional duration_steps,
 *                materialization predicate "leading contiguous survival >= T".)
 *                demotable (§3.1 protection modes): the runtime may demote the claim (hard -> soft)
 *                to serve an active request, in pools with RKC_MODE_RELAX, always before the
 *                eviction that breaks its predicate.  best_effort (§3.1: telemetry only): the claim
 *                is observed (decision SHADOW) in every policy, protects nothing, never expires and
 *                its loss is never harm.  offloadable (§3.1 protection modes): the runtime may move
 *                the claim's content to the pool's second tier (offload_blocks) to serve an active
 *                request, in pools with RKC_MODE_RELAX, as long as its predicate stays restorable;
 *                an offloaded claim keeps state MATERIALIZED with effective protection OFFLOADED.
 *   FINISH  (3)  w1 = selector: the request finishes and releases its live KV.
 *   RELEASE (4)  w1 = selector over live claims (ascending id): the claim is released.
 *   DEMOTE  (5)  w1 = selector over materialized hard-requested claims: hard -> soft (§3.1, §3.2).
 *   NOP     (6)  no operation.
 *   RETRY   (7)  the scheduler retries the oldest deferred request (active deferral, §3.5
 *                mechanism table "active deferral"; §5.4 live scheduler run: the active request is
 *                deferred by the scheduler gate, then refused).  w1..w3 unused.  Only pools with
 *                defer_limit > 0 ever hold deferred requests; with none queued RETRY is a NOOP.
 * Any other type, or out-of-range fields, makes the event malformed: outcome INVALID.
 * -------------------------------------------------------------------------------------------- */
typedef struct rkc_event {
  int32_t w[4];
} rkc_event;

enum rkc_event_type {
  RKC_EV_PREFILL = 0,
  RKC_EV_EXTEND = 1,
  RKC_EV_CLAIM = 2,
  RKC_EV_FINISH = 3,
  RKC_EV_RELEASE = 4,
  RKC_EV_DEMOTE = 5,
  RKC_EV_NOP = 6,
  RKC_EV_RETRY = 7
};

/* Pool policy: how the runtime lowers claims (§3.5 mechanism table rows "native eviction",
 * "write no-admit only", "resident victim exclusion"; §5.4 check C1 for soft lowering). */
enum rkc_pool_mode {
  RKC_MODE_LRU = 0,     /* native eviction: claims are only observed (shadow)                  */
  RKC_MODE_SOFT = 1,    /* soft priority: claims accepted, hard requests lowered (approximate)  */
  RKC_MODE_NOADMIT = 2, /* write no-admit: request KV never becomes reusable; claims observed   */
  RKC_MODE_HARD = 3,    /* hard protected-resident exclusion with scheduler-visible refusal     */
  /* flag OR'ed into rkc_pool_desc.mode: runtime relaxation (§3.5 mechanism table "relax resident
   * claim": the active side is served by demoting resident state).  In a hard-protection pool,
   * before an active PREFILL / EXTEND / RETRY is refused on behalf of claims, the blocking claims
   * that are offloadable or demotable are taken lowest priority first, then lowest id: each is
   * offloaded when it is offloadable and its footprint L fits the second tier's free room
   * (offload_blocks minus the blocks offloaded claims hold), else demoted when it is demotable,
   * else left alone, until the request fits; no claim changes when even all of them would not make
   * it fit (§3.5 mechanism table "relax resident claim", "offload resident").  An offloaded claim
   * protects nothing, ranks nothing, its victims count as unclaimed and its predicate never fails;
   * its copy (L blocks of the second tier) is dropped when it expires or is released, and DEMOTE
   * never selects it.  A served PREFILL / RETRY with shared prefix P past its hits h counts
   * min(P, largest footprint of an offloaded claim on its chain) - h blocks as restored from the
   * second tier (pool telemetry [40]); they still take new GPU blocks.  No effect under the other
   * policies (they never refuse on behalf of claims). */
  RKC_MODE_RELAX = 16
};

/* ----------------------------------------------------------------------------------------------
 * Pool descriptor: 64 bytes.
 * -------------------------------------------------------------------------------------------- */
typedef struct rkc_pool_desc {
  int32_t usable_blocks;     /* U, 1..RKC_MAX_USABLE_BLOCKS; block size is 16 tokens (§4.1)     */
  int32_t mode;              /* enum rkc_pool_mode, optionally | RKC_MODE_RELAX                  */
  int32_t n_events;          /* events of this pool                                              */
  int32_t n_chains;          /* valid shared chain ids are [0, n_chains)                         */
  int32_t max_live_claims;   /* live-claim table capacity; a CLAIM beyond it is INVALID          */
  int32_t max_live_requests; /* live-request table capacity; a PREFILL beyond it is INVALID      */
  int32_t n_claim_slots;     /* telemetry slots; the k-th CLAIM event uses slot k                */
  int32_t defer_limit;       /* active deferral (0 = off): a PREFILL that would be refused and
                                attributed to resident claims is DEFERRED instead and queued (FIFO,
                                at most max_live_requests deep); a queued request receives at most
                                defer_limit DEFERRED outcomes before a RETRY that still finds it
                                blocked refuses it                                               */
  int32_t offload_blocks;    /* second-tier capacity in blocks, >= 0 (0 = no second tier); used
                                by relaxing hard-protection pools only                           */
  int32_t reserved[3];       /* must be 0                                                        */
  int64_t event_offset;      /* index of the pool's first event in the event (and outcome) array */
  int64_t claim_slot_offset; /* index of the pool's first slot in the claim telemetry array      */
} rkc_pool_desc;

/* ----------------------------------------------------------------------------------------------
 * Outcome: 16 bytes, one per event, at the event's index.   (§3.1 ClaimEvent; §5.4 refusal record)
 *
 * w0 = code[0:8] | flags[8:16] | n16[16:32]
 *   n16 = number of blocking claims for REFUSED_CLAIM and DEFERRED, 0 for REFUSED_CAPACITY, the
 *         number of claims the runtime demoted or offloaded for RELAXED, otherwise the number of claims that
 *         expired at the start of this step; saturates at 65535.
 * w1 = id, w2 = a, w3 = b:
 *   ADMIT / EVICT_RESIDENT  after PREFILL: id = request, a = resident victims, b = leading hits h
 *                           after EXTEND : id = request, a = resident victims, b = active blocks after
 *                           after CLAIM  : id = claim,   a = resident victims, b = blocks allocated
 *   REFUSED_CLAIM/CAPACITY  id = smallest blocking claim id (or -1), a = protected resident Pr,
 *                           b = active live required (A + cached hits + need); shortfall = a + b - U
 *   MATFAIL                 id = claim, a = blocks needed, b = FREE + evictable blocks available
 *   DEMOTED / RELEASED      id = claim, a = min(leading registered length, L), b = T
 *   FINISHED                id = request, a = blocks turned cached, b = blocks dropped (no-admit)
 *   NOOP / INVALID          id = -1, a = 0, b = 0
 *   DEFERRED                the refusal record of REFUSED_CLAIM (id = smallest blocking claim id,
 *                           a = Pr, b = required, n16 = blocking claims): the request is queued
 *   RELAXED                 served after the runtime demoted or offloaded claims (RKC_MODE_RELAX):
 *                           id, a, b as ADMIT for the event (PREFILL, EXTEND or RETRY), n16 = claims
 *                           demoted + claims offloaded
 * RETRY reports the retried request: served -> ADMIT / EVICT_RESIDENT with id = the request (its
 * PREFILL step), a = resident victims, b = leading hits; still blocked -> DEFERRED; refused for good
 * -> REFUSED_CLAIM / REFUSED_CAPACITY; full live-request table -> INVALID (the request stays queued);
 * served after relaxation -> RELAXED.
 * -------------------------------------------------------------------------------------------- */
typedef struct rkc_outcome {
  int32_t w[4];
} rkc_outcome;

enum rkc_outcome_code {
  RKC_OC_ADMIT = 0,
  RKC_OC_EVICT_RESIDENT = 1,
  RKC_OC_REFUSED_CLAIM = 2,
  RKC_OC_REFUSED_CAPACITY = 3,
  RKC_OC_MATFAIL = 4,
  RKC_OC_DEMOTED = 5,
  RKC_OC_RELEASED = 6,
  RKC_OC_FINISHED = 7,
  RKC_OC_NOOP = 8,
  RKC_OC_INVALID = 9,
  RKC_OC_DEFERRED = 10,
  RKC_OC_RELAXED = 11
};

enum rkc_outcome_flag {
  RKC_FL_EXPIRED = 1,           /* >= 1 claim expired at the start of this step                  */
  RKC_FL_PRED_FAIL = 2,         /* >= 1 claim first failed its materialization predicate         */
  RKC_FL_HARM = 4,              /* >= 1 accepted claim was harmed (§3.2)                          */
  RKC_FL_POST_RELEASE_LOSS = 8, /* a victim was covered only by demoted/expired claims (§3.2)     */
  RKC_FL_EVICT_UNCLAIMED = 16,  /* a victim was covered by no live claim                          */
  RKC_FL_NOADMIT_DROP = 32,     /* FINISH dropped non-admitted blocks                              */
  RKC_FL_LOWERED = 64,          /* hard request lowered to soft priority (check C1, §5.4)          */
  RKC_FL_SHADOW = 128           /* claim materialized as ordinary cache, not accepted              */
};

/* ----------------------------------------------------------------------------------------------
 * Claim telemetry: 40 bytes = 10 x int32, one slot per CLAIM event in step order.
 *   [0] claim_id (step index; -1 for an unused slot)
 *   [1] packed = decision[0:4] | state[4:8] | hard_req[8] | prio[9:11] | eff_prot[11:13]
 *                | demotable[13] | best_effort[14] | relaxed_by_runtime[15] | offloadable[16]
 *       (eff_prot 3 = OFFLOADED: the claim holds a second-tier copy)
 *   [2] accept_step [3] demote_step [4] expire_step [5] release_step [6] pred_fail_step
 *   [7] harm_step   (every step field is -1 when the transition never happened)
 *   [8] blocked_count: active refusals this claim was attributed to
 *   [9] lead_end = min(leading registered length of the chain, L) at the end of the replay
 * A malformed or table-rejected CLAIM keeps its slot with packed = 0 and lead_end = 0.
 * -------------------------------------------------------------------------------------------- */
typedef struct rkc_claim_telemetry {
  int32_t w[10];
} rkc_claim_telemetry;

enum rkc_decision { /* §3.1 ResidentClaimDecision */
  RKC_DEC_NONE = 0,
  RKC_DEC_ACCEPTED = 1,
  RKC_DEC_ACCEPTED_APPROX = 2,
  RKC_DEC_SHADOW = 3,
  RKC_DEC_REJECTED = 4
};

enum rkc_claim_state { /* §3.1 ResidentClaimState */
  RKC_ST_SUBMITTED = 0,
  RKC_ST_OBSERVED = 1,
  RKC_ST_MATERIALIZED = 2,
  RKC_ST_DEMOTED = 3,
  RKC_ST_EXPIRED = 4,
  RKC_ST_RELEASED = 5,
  RKC_ST_HARMED = 6,
  RKC_ST_REJECTED = 7
};

enum rkc_protection { RKC_PROT_NONE = 0, RKC_PROT_SOFT = 1, RKC_PROT_HARD = 2, RKC_PROT_OFFLOADED = 3 };

/* ----------------------------------------------------------------------------------------------
 * Pool telemetry: 256 bytes = 64 x int32.
 *   [0..9]  outcomes per code          [10] victims  [11] resident victims  [12] post-release victims
 *   [13] blocks dropped by no-admit    [14] sum of leading hits of served prefills
 *   [15] accepted [16] accepted-approx [17] shadow [18] rejected                  (claim decisions)
 *   [19] harmed [20] predicate failures [21] expired [22] demoted [23] released   (lifecycle)
 *   [24] peak active blocks [25] final active blocks
 *   [26] final cached blocks [27] final free blocks [28] final protected blocks
 *   [29] final live requests [30] final live claims
 *   [31] status: 0, or RKC_PS_* bits
 *   [32] DEFERRED outcomes [33] deferred requests served by RETRY [34] deferred requests refused by
 *   RETRY [35] deferred requests still queued at the end
 *   [36] RELAXED outcomes [37] claims demoted by the runtime
 *   [38] claims offloaded [39] blocks offloaded [40] blocks restored from the second tier
 *   [41] peak second-tier blocks held                                  [42..63] 0 (reserved)
 * -------------------------------------------------------------------------------------------- */
typedef struct rkc_pool_telemetry {
  int32_t w[64];
} rkc_pool_telemetry;

enum rkc_pool_status {
  RKC_PS_REQUEST_TABLE = 1, /* a PREFILL found the live-request table full                   */
  RKC_PS_CLAIM_TABLE = 2,   /* a CLAIM found the live-claim table full                         */
  RKC_PS_SLOT_TABLE = 4,    /* more CLAIM events than n_claim_slots                            */
  RKC_PS_DESCRIPTOR = 256,  /* descriptor outside the batch limits; the pool was not replayed,
                               every outcome is INVALID (an ABI fault, not a contract outcome) */
  RKC_PS_INTERNAL = (int32_t)0x80000000u /* a kernel's own consistency guard fired (an allocation
                               that feasibility said must succeed found no block, a touch-stack
                               node beyond its bound, a runaway loop); the pool's outputs from
                               that step on are unreliable.  Never set on a correct build: the
                               parity tests require it to be clear on every pool */
};

/* ----------------------------------------------------------------------------------------------
 * Batch: host struct describing one replay launch.
 * -------------------------------------------------------------------------------------------- */
typedef struct rkc_batch {
  int32_t n_pools;           /* >= 0                                                             */
  int32_t max_usable_blocks; /* >= every pool's U                                                */
  int32_t max_events;        /* >= every pool's n_events                                         */
  int32_t max_chains;        /* >= every pool's n_chains                                         */
  int32_t max_live_requests; /* >= every pool's max_live_requests                                */
  int32_t max_live_claims;   /* >= every pool's max_live_claims                                  */
  int32_t max_claim_slots;   /* >= every pool's n_claim_slots                                    */
  int32_t flags;             /* RKC_FLAG_* bits (below); other bits are an error                  */
  int64_t n_events_total;    /* length of the event and outcome arrays                           */
  int64_t n_claim_slots_total; /* length of the claim telemetry array                            */
  const rkc_pool_desc* d_pools;     /* [n_pools], 16-byte aligned                               */
  const rkc_event* d_events;        /* [n_events_total], 16-byte aligned                        */
  rkc_outcome* d_outcomes;          /* [n_events_total], 16-byte aligned, written               */
  rkc_pool_telemetry* d_pool_tel;   /* [n_pools], 16-byte aligned, written                      */
  rkc_claim_telemetry* d_claim_tel; /* [n_claim_slots_total], 8-byte aligned, written           */
  void* d_scratch;                  /* >= rkc_scratch_bytes(b) bytes, 256-byte aligned          */
  size_t scratch_bytes;
} rkc_batch;

/* rkc_batch.flags: replay with the general kernel even when the batch fits the compact one (the
 * compact kernel is chosen for usable blocks <= 32,767, events <= 65,533, chains <= 256, live
 * claims <= 64 and live requests <= 256).  Both give identical outputs; the flag exists so the
 * general kernel can be checked on the same inputs. */
#define RKC_FLAG_GENERAL_KERNEL 1
/* rkc_batch.flags: one wavefront per pool everywhere.  Without it, a batch of at most 256 pools (one
 * per compute unit) whose live lists do not fit in LDS is replayed by a workgroup of 8 wavefronts
 * per pool (wave 0 runs the pool's event loop; the others share the scans and moves of its long
 * lists).  Both give identical outputs; the flag exists so both can be checked on the same inputs. */
#define RKC_FLAG_ONE_WAVE_PER_POOL 2

typedef enum rkc_status {
  RKC_OK = 0,
  RKC_E_NULL = -1,        /* a required pointer is NULL                                       */
  RKC_E_ALIGN = -2,       /* a pointer is misaligned                                           */
  RKC_E_RANGE = -3,       /* a count, index or limit is out of range                           */
  RKC_E_UNSUPPORTED = -4, /* a limit beyond what this implementation supports                  */
  RKC_E_SCRATCH = -5,     /* scratch buffer missing or too small                               */
  RKC_E_HIP = -6,         /* a HIP runtime call failed (launch, copy, synchronize)             */
  RKC_E_POOL_STATUS = -7, /* query succeeded, but the pool's status word is non-zero           */
  RKC_E_SCRATCH_LIMIT = -8 /* rkc_replay_batch_noalloc: the batch needs more scratch than
                              RKC_NOALLOC_SCRATCH_BYTES                                          */
} rkc_status;

/* ABI version (RKC_ABI_VERSION).  Implementation detail, no passage of the paper. */
int32_t rkc_abi_version(void);

/* Device scratch bytes rkc_replay_batch needs for this batch (an implementation detail: the paper
 * defines no storage, only the contract the replay follows): per pool, the pool state that does not
 * stay on chip (touch-stack nodes beyond the LDS part, the FIFO of finished requests' private runs,
 * one entry per claim slot, a deferral ring of max_live_requests entries, and the live lists when
 * they do not fit in LDS), plus 4 bytes per pool for the launch order of the compact kernel.  Reads
 * only the host-side limits of b; never fails (returns 0 for a NULL b or an empty batch). */
size_t rkc_scratch_bytes(const rkc_batch* b);

/* Replay every pool of the batch from empty pools (all U blocks FREE, no claims, no requests).
 * What each event does is the contract of the paper: the claim input schema and the ClaimEvent
 * surface (§3.1 minimal conformance schema; protection-mode table), decisions and the lifecycle
 * (§3.1 decision and state rows; §3.2 harm semantics; §3.3), the feasibility boundary
 * protected_resident + active_live <= usable (§3.4), the policies and runtime actions (§3.5
 * mechanism table) and scheduler-visible refusal with its record (§5.4 refusal record).
 * Arguments: b describes device buffers laid out as above (the host struct itself is read during
 * the call only); s is a hipStream_t of the current device (NULL = the default stream).
 * Asynchronous: validates the host struct, then only enqueues kernels on s.  Pool i is replayed by
 * its own wavefront or workgroup; pools are independent, so results do not depend on batch
 * composition or order.  Returns RKC_OK or a negative status; on a negative status nothing was
 * enqueued.  Outcomes, pool telemetry and claim telemetry are written in full; scratch contents are
 * undefined afterwards. */
rkc_status rkc_replay_batch(const rkc_batch* b, void* s /* hipStream_t */);

/* For callers that cannot allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc): rkc_replay_batch with the library's built-in scratch instead of
 * b->d_scratch (b->d_scratch and b->scratch_bytes are ignored and may be NULL / 0).  Same outputs,
 * same asynchrony, same statuses, plus RKC_E_SCRATCH_LIMIT when rkc_scratch_bytes(b) exceeds
 * RKC_NOALLOC_SCRATCH_BYTES (64 MiB: e.g. 4,096 pools of 80 blocks x 256 events, or 2,048 pools of
 * 2,048 blocks x 1,024 events).  It calls no hipMalloc / hipFree: the scratch is a static device array
 * of the library, one per device, looked up on the first call made with that device current and
 * held until the process ends.  Every call on one device shares that array, so calls that overlap
 * on one device (different streams, or threads) race and give undefined results: serialize them.
 * Nothing in the array needs clearing between calls. */
rkc_status rkc_replay_batch_noalloc(const rkc_batch* b, void* s /* hipStream_t */);

/* Copy outcomes [first, first + count) of pool `pool` into host_dst (caller-owned, count records)
 * after synchronizing s.  One outcome per input event: the ClaimEvent stream of §3.1 (event type,
 * claim or request id, step = index, predicate / capacity fields), with refusals carrying the §5.4
 * refusal record (blocking claim id, protected resident, active required; shortfall = a + b - U).
 * Also reads the pool descriptor back to locate the events.  Returns RKC_E_RANGE when the range
 * leaves the pool or the descriptor's event offset does not fit the batch (nothing copied),
 * RKC_E_POOL_STATUS (data still copied) when the pool's status is non-zero. */
rkc_status rkc_query_outcomes(const rkc_batch* b, int32_t pool, int32_t first, int32_t count,
                              rkc_outcome* host_dst, void* s);

/* Copy pool telemetry of `pool` (if host_pool != NULL) and up to max_claims of its claim
 * telemetry slots (if host_claims != NULL; *n_claims receives the pool's slot count) after
 * synchronizing s.  The claim records are the claim-level telemetry of the §7 runtime-surface table
 * (accepted, refused, demoted, evicted, offloaded or harmed) over the §3.1 decision and state rows
 * and the §3.2 harm table.  Returns RKC_E_RANGE when the descriptor's slot range does not fit the
 * batch (claim records not copied), RKC_E_POOL_STATUS (data still copied) for a non-zero pool
 * status. */
rkc_status rkc_query_telemetry(const rkc_batch* b, int32_t pool, rkc_pool_telemetry* host_pool,
                               rkc_claim_telemetry* host_claims, int32_t max_claims,
                               int32_t* n_claims, void* s);

/* Static, human-readable name of a status.  Implementation detail, no passage of the paper. */
const char* rkc_status_string(rkc_status st);

#ifdef __cplusplus
}
#endif

#endif /* RKC_H */
