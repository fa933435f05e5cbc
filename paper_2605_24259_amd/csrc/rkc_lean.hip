// rkc_lean.hip -- the compact replay kernel for pools whose whole state fits in 16-bit words.
//
// Same contract, same outputs, as the general kernel in rkc_replay.hip; this variant serves the
// batches whose limits allow a tighter encoding:
//   usable blocks <= 32,767, events per pool <= 65,533, live requests <= 256,
//   claim slots <= 65,534, and live claims <= 64 with shared chains <= 256 or live claims <= 256
//   (four 64-claim sets) with shared chains <= 64.
// One 64-lane wavefront replays one pool.  The per-event state machine runs on the scalar unit:
// every branch is on a wave-uniform value, so no exec-mask juggling happens on the event path.
//
// Representation (why it is exact is explained in rkc_replay.hip): the registered positions of
// every shared chain are a leading run [0, n), eviction takes chains from the top, and every
// touch, hold, protection and coverage is a leading range.  Per chain, one 16-byte LDS record
//   n | hold, prot | bt, nx | covA, stop | sbot       (16-bit halves)
// n registered length, hold leading positions held by live requests, prot protection extent of
// materialized hard claims (hard-protection pools), covA the largest footprint of a live claim on
// the chain, and a touch stack of (extent, step) nodes (top stop, bottom sbot; bt = bottom step,
// nx = extent of the node above the bottom).  Everything else a claim implies for its chain --
// soft levels, which victims are resident or post-release, which predicates can fail -- lies
// inside [0, covA) and is computed from the claim lanes only when a position below covA is
// involved.  Each chain's eviction key lives in LDS as one 32-bit word
//   key = level << 25 | last use << 9 | (chain + 1)
// so one wave min-reduction over the keys both orders candidates (level, last use) and names the
// chain; a finished request's private run has key level 0 | finish step << 9 | 0, which puts it
// ahead of a chain touched at the same step (it lies above that chain's touched prefix).  A run
// boundary taken above the true one only splits a run of equal keys into several iterations.
//
// Live claims sit one per lane in six VGPRs (16-bit halves), so expiry, attribution, predicate
// sweeps and claim maxima are single vector passes with DPP reductions.  Live requests are a
// compact id-ordered list (8 bytes each) in LDS, past its first 128 entries in global scratch
// (one claim set).  Touch-stack nodes use LDS first, then global scratch; finished requests'
// private runs form a FIFO in global scratch, and so do the deferred requests of
// hard-protection pools that defer (a ring of live-request-capacity entries).
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "rkc.h"
#include "rkc_lean.h"

namespace {

typedef uint32_t u32;
typedef int32_t i32;
typedef uint64_t u64;
typedef int64_t i64;

typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) u32 lds_u32;
typedef __attribute__((address_space(3))) u32x2 lds_u32x2;
typedef __attribute__((address_space(3))) u32x4 lds_u32x4;
typedef __attribute__((address_space(1))) u32x2 glb_u32x2;
typedef __attribute__((address_space(1))) u32x4 glb_u32x4;

constexpr u32 NIL = 0xFFFFu;       // 16-bit nil (positions, steps, indices are all below it)
constexpr u32 KINF = 0xFFFFFFFFu;  // key of a chain with no candidate
constexpr u32 NEVER = 0xFFFFFFFFu;

enum : u32 { ST_SUBMITTED = 0, ST_OBSERVED = 1, ST_MATERIALIZED = 2, ST_DEMOTED = 3, ST_EXPIRED = 4,
             ST_RELEASED = 5, ST_HARMED = 6, ST_REJECTED = 7 };
enum : u32 { DEC_ACCEPTED = 1, DEC_APPROX = 2, DEC_SHADOW = 3, DEC_REJECTED = 4 };
// pool telemetry words accumulated lane-distributed
enum : u32 { TW_VICTIMS = 10, TW_RESIDENT = 11, TW_POST = 12, TW_DROPPED = 13, TW_HITS = 14,
             TW_ACCEPTED = 15, TW_HARM = 19, TW_PREDFAIL = 20, TW_EXPIRED = 21, TW_DEMOTED = 22,
             TW_RELEASED = 23, TW_RETRY_SERVED = 33, TW_RETRY_REFUSED = 34, TW_RUNTIME_DEMOTED = 37,
             TW_OFF_CLAIMS = 38, TW_OFF_BLOCKS = 39, TW_RESTORED = 40 };

// live-claim meta (low half of qc): state[0:3) eff[3:5) hard[5] prio[6:8) pending[8] decision[9:12)
// demotable[12] best_effort[13] relaxed_by_runtime[14] offloadable[15]
constexpr u32 M_DEMQ = 1u << 12, M_BE = 1u << 13, M_RELAXED = 1u << 14, M_OFFQ = 1u << 15;
__device__ __forceinline__ u32 m_state(u32 m) { return m & 7u; }
__device__ __forceinline__ u32 m_eff(u32 m) { return (m >> 3) & 3u; }
__device__ __forceinline__ u32 m_hard(u32 m) { return (m >> 5) & 1u; }
__device__ __forceinline__ u32 m_prio(u32 m) { return (m >> 6) & 3u; }
__device__ __forceinline__ u32 m_pend(u32 m) { return (m >> 8) & 1u; }
__device__ __forceinline__ u32 m_dec(u32 m) { return (m >> 9) & 7u; }
__device__ __forceinline__ u32 packed_of(u32 m) {
  return m_dec(m) | (m_state(m) << 4) | (m_hard(m) << 8) | (m_prio(m) << 9) | (m_eff(m) << 11) |
         (((m >> 12) & 15u) << 13);
}

__device__ __forceinline__ u32 lo16(u32 v) { return v & 0xFFFFu; }
__device__ __forceinline__ u32 hi16(u32 v) { return v >> 16; }
// two 16-bit halves as one vector, so that uniform operands pack in one scalar instruction
typedef unsigned short u16x2 __attribute__((ext_vector_type(2)));
__device__ __forceinline__ u32 pk(u32 lo, u32 hi) {
  const u16x2 v = {(unsigned short)lo, (unsigned short)hi};
  return __builtin_bit_cast(u32, v);
}
__device__ __forceinline__ i32 st16(u32 v) { return v == NIL ? -1 : (i32)v; }  // step field

// ---- wave primitives (all 64 lanes active) ----------------------------------------------------
// A value every lane holds identically, moved to a scalar register.  Built with RKC_CHECK_UNIFORM
// (a checking build, never the product one), every call also verifies that the active lanes agree
// and counts the calls where they do not.
#ifdef RKC_CHECK_UNIFORM
__device__ unsigned int g_lean_uniform_violations;
__device__ __forceinline__ u32 ufl(u32 v) {
  const u32 f = (u32)__builtin_amdgcn_readfirstlane((int)v);
  if (__ballot(v != f) != 0 && __lane_id() == (u32)__builtin_ctzll(__ballot(true)))
    atomicAdd(&g_lean_uniform_violations, 1u);
  return f;
}
#else
__device__ __forceinline__ u32 ufl(u32 v) { return (u32)__builtin_amdgcn_readfirstlane((int)v); }
#endif
__device__ __forceinline__ u32 rdl(u32 v, u32 l) { return (u32)__builtin_amdgcn_readlane((int)v, (int)l); }
// x mod n for wave-uniform x and 1 <= n <= 1024, on the vector unit (the scalar unit is the busier
// one): x / n from a double-precision reciprocal refined by two Newton steps (relative error below
// 2^-48, so x / n is off by less than 2^-16 < 1 / n), whose floor is the quotient or, when x is a
// multiple of n, one less; a single comparison corrects that.
__device__ __forceinline__ u32 umod(u32 x, u32 n) {
  const double dn = (double)n;
  double r = __builtin_amdgcn_rcp(dn);
  r = __builtin_fma(r, __builtin_fma(-dn, r, 1.0), r);
  r = __builtin_fma(r, __builtin_fma(-dn, r, 1.0), r);
  const u32 q = (u32)__builtin_floor((double)x * r);
  const u32 m = x - q * n;
  return ufl(m >= n ? m - n : m);
}
// a - b, or 0 when b exceeds a
__device__ __forceinline__ u32 sub0(u32 a, u32 b) { return a > b ? a - b : 0u; }
// lane l of `old` replaced by the uniform value v
__device__ __forceinline__ u32 wrl(u32 old, u32 v, u32 l) { return __lane_id() == l ? v : old; }
__device__ __forceinline__ u64 ballot(bool p) { return __ballot(p); }
// A wave-uniform index moved to a vector register, so that the address arithmetic of an LDS or
// global access at that index runs on the vector unit: the scalar unit is the busier one, and a
// global address from a scalar index takes three scalar instructions (64-bit shift and add).
__device__ __forceinline__ u32 vx(u32 i) {
  u32 r;
  asm("v_mov_b32 %0, %1" : "=v"(r) : "s"(ufl(i)));
  return r;
}
// &base[i] for a wave-uniform i, the byte offset formed on the vector unit (a 32-bit offset to a
// scalar base, which the global instructions take as such)
template <class T>
__device__ __forceinline__ T* gat(T* base, u32 i) {
  return (T*)((__attribute__((address_space(1))) char*)base + (u64)(vx(i) * (u32)sizeof(T)));
}

// every source lane exists for the permutes used here, so the moved value never needs an old
// value and the move folds into the consuming min / max / add
template <int CTRL>
__device__ __forceinline__ u32 dpp(u32 v) {
  return (u32)__builtin_amdgcn_mov_dpp((int)v, CTRL, 0xF, 0xF, true);
}
struct OpMax { __device__ static u32 f(u32 a, u32 b) { return a > b ? a : b; } };
struct OpMin { __device__ static u32 f(u32 a, u32 b) { return a < b ? a : b; } };
struct OpAdd { __device__ static u32 f(u32 a, u32 b) { return a + b; } };
// Row-level butterflies (quad perms, half-row and row mirrors), then the four row results.
template <class Op>
__device__ __forceinline__ u32 wreduce(u32 v) {
  v = Op::f(v, dpp<0xB1>(v));   // quad_perm [1,0,3,2]
  v = Op::f(v, dpp<0x4E>(v));   // quad_perm [2,3,0,1]
  v = Op::f(v, dpp<0x141>(v));  // row_half_mirror
  v = Op::f(v, dpp<0x140>(v));  // row_mirror
  return Op::f(Op::f(rdl(v, 0), rdl(v, 16)), Op::f(rdl(v, 32), rdl(v, 48)));
}
__device__ __forceinline__ u32 wmax(u32 v) { return wreduce<OpMax>(v); }
__device__ __forceinline__ u32 wmin(u32 v) { return wreduce<OpMin>(v); }
__device__ __forceinline__ u32 wsum(u32 v) { return wreduce<OpAdd>(v); }
// lane l receives lane l + 1's value (lane 63 keeps its own)
__device__ __forceinline__ u32 shift_down(u32 v) {
  return (u32)__builtin_amdgcn_update_dpp((int)v, (int)v, 0x130 /* wave_shl:1 */, 0xF, 0xF, false);
}

// storage of NQ claim sets: one register per set (an array for one set, a vector for four)
template <int NQ> struct QSets;
template <> struct QSets<1> { typedef u32 type[1]; };
template <> struct QSets<4> { typedef u32 type __attribute__((ext_vector_type(4))); };

// chain record: n | hold, prot | bt, nx | covA, stop | sbot (16-bit halves, 16 bytes)
struct G0 { u32 n, hold, prot, bt, nx, covA, stop, sbot; };

struct AllocRes {
  u32 ok, E, resident, post, unclaimed;
  u32 hit;  // the allocation took blocks from the hit chain (its record changed)
};

// LDS of one pool (bytes), fixed per instantiation so that every region's address is a constant
// of the code (no registers hold LDS bases): status block, outcome counters, eviction keys, chain
// records, the LDS part of the live-request list and of the touch-stack node pool.  NS and NQ
// bound the chains (64 NS) and the live requests kept in LDS; with one claim set the LDS a pool
// takes sets how many pools share a CU (the CU allocates LDS in 1,280-byte units), with four the
// registers set it.
template <int NS, int NQ>
struct LdsMap {
  // live requests in LDS: a zipf pool that allows 256 live requests holds ~50 on average and 165 at
  // most, so with one claim set the first 128 (96 with 256 chains) stay in LDS and the rest go to
  // global scratch
  static constexpr u32 RQL = NQ == 4 ? 256u : NS == 4 ? 96u : 128u;
  // touch-stack nodes in LDS (a zipf pool of 256 chains peaks at ~80-115 live nodes, the 80-block
  // pools at ~35): with 256 chains 48, which brings a pool to 6,400 B, five allocation units, so 25
  // pools share a CU instead of 21 (more than paying for the slower node accesses); of those five
  // units, 96 requests and 48 nodes measured faster than 128 and 16 or 64 and 80
  static constexpr u32 NL = NS == 4 ? 48u : 64u;
  static constexpr u32 COLD = 0, HIST = 64, KEYS = 128, CH = KEYS + 256u * NS, RQ = CH + 1024u * NS,
                       ND = RQ + 8u * RQL, BYTES = ND + 8u * NL;
};

// ---- one pool ---------------------------------------------------------------------------------
// NS: 64-key groups (chains <= 64 NS); NQ: 64-claim sets (live claims <= 64 NQ; claim j sits in lane
// j mod 64 of set j / 64); MODE: the pool policy, fixed at compile time so that each policy's event
// loop carries only the logic that policy can reach; EXT: a hard-protection pool that defers or
// relaxes, whose loop carries the deferral ring and the runtime relaxation.
template <int NS, int NQ, int MODE, bool EXT>
struct Lean {
  static constexpr u32 KC = 64u * NS;  // key slots (chains padded to whole lanes)
  // descriptor: the rarely used limits one per lane of `cst`
  static constexpr u32 mode = MODE;
  u32 cst;  // lane 0 U, 1 chains, 2 live-claim cap, 3 live-request cap, 4 claim slots, 5 node cap,
            // 6 defer limit, 7 relaxation on, 8 second-tier capacity
  u32 lane;
  __device__ __forceinline__ u32 U() const { return rdl(cst, 0); }
  __device__ __forceinline__ u32 nch() const { return rdl(cst, 1); }
  __device__ __forceinline__ u32 maxq() const { return rdl(cst, 2); }
  __device__ __forceinline__ u32 maxr() const { return rdl(cst, 3); }
  __device__ __forceinline__ u32 nslots() const { return rdl(cst, 4); }
  __device__ __forceinline__ u32 ncap() const { return rdl(cst, 5); }
  __device__ __forceinline__ u32 dlim() const { return rdl(cst, 6); }
  __device__ __forceinline__ u32 relax_on() const { return rdl(cst, 7); }
  __device__ __forceinline__ u32 t2cap() const { return rdl(cst, 8); }
  // soft levels and acceptance (soft, hard pools: mode bit 0), hard protection, write no-admit
  __device__ __forceinline__ static constexpr bool softl() { return MODE & 1; }
  __device__ __forceinline__ static constexpr bool shadm() { return !(MODE & 1); }
  __device__ __forceinline__ static constexpr bool hardm() { return MODE == RKC_MODE_HARD; }
  __device__ __forceinline__ static constexpr bool noadm() { return MODE == RKC_MODE_NOADMIT; }
  // only hard protection refuses on behalf of claims, so only hard-protection pools can defer or
  // relax
  __device__ __forceinline__ static constexpr bool ext() { return MODE == RKC_MODE_HARD && EXT; }
  // meta m says offloaded to the second tier (only relaxing pools offload)
  __device__ __forceinline__ static bool offl(u32 m) { return ext() && m_eff(m) == RKC_PROT_OFFLOADED; }
  // memory
  lds_u32* kk;
  lds_u32* hist;  // outcomes per code (16 counters; entry 15 collects the lanes past the end)
  lds_u32x4* ch;
  // live requests: entries [0, RQL) in LDS, the rest in global scratch
  static constexpr u32 RQL = LdsMap<NS, NQ>::RQL;
  lds_u32x2* rq;
  glb_u32x2* rqg;
  // (per-lane j; L: the caller knows every index it uses lies in LDS, so no lane-dependent branch
  // between LDS and scratch is formed)
  template <bool L>
  __device__ __forceinline__ u32x2 rq_ld(u32 j) const {
    u32x2 v;
    if (L || RQL >= 256u || j < RQL) v = rq[j]; else v = rqg[j - RQL];
    return v;
  }
  template <bool L>
  __device__ __forceinline__ void rq_st(u32 j, u32x2 v) {
    if (L || RQL >= 256u || j < RQL) rq[j] = v; else rqg[j - RQL] = v;
  }
  // the same for a wave-uniform j (address arithmetic on the vector unit)
  __device__ __forceinline__ u32x2 rq_get(u32 j) const {
    u32x2 v;
    if (RQL >= 256u || j < RQL) v = rq[vx(j)]; else v = *gat(rqg, j - RQL);
    return u32x2{ufl(v.x), ufl(v.y)};
  }
  __device__ __forceinline__ void rq_put(u32 j, u32x2 v) {
    if (RQL >= 256u || j < RQL) rq[vx(j)] = v; else *gat(rqg, j - RQL) = v;
  }
  // entry j's length grows by k (a wave-uniform j); returns its first word
  __device__ __forceinline__ u32 rq_grow(u32 j, u32 k) {
    u32 x;
    if (RQL >= 256u || j < RQL) {
      const u32 a = vx(j);
      const u32x2 e = rq[a];
      x = ufl(e.x);
      const u32 y = ufl(e.y);
      rq[a] = u32x2{x, pk(lo16(y), hi16(y) + k)};
    } else {
      glb_u32x2* a = gat(rqg, j - RQL);
      const u32x2 e = *a;
      x = ufl(e.x);
      const u32 y = ufl(e.y);
      *a = u32x2{x, pk(lo16(y), hi16(y) + k)};
    }
    return x;
  }
  lds_u32x2* ndl;
  glb_u32x2* ndg;
  // nodes [0, NL) in LDS, the rest in global scratch
  static constexpr u32 NL = LdsMap<NS, NQ>::NL;
  glb_u32x2* fifo;  // finished requests' private runs: finish step | low end << 16, top (16-bit fields)
  glb_u32x4* dq;  // deferred requests: PREFILL step, S, chain, P
  // Claim records.  A live claim's words 0..8 are written by its own lane when it is released or at
  // the end; everything else by the final pass, from the slot table: per slot (x) L | chain << 16
  // (0 for a malformed claim), from which lead_end follows, and (y) NEVER for a claim that became
  // live, else the claim id | its packed word << 16 (a rejected or malformed claim, whose record the
  // final pass writes whole: those records, most of a pool's, then go out as full consecutive lines
  // instead of pieces).  The packed word of such a claim never has the relaxed-by-runtime bit (15),
  // so its bit 16 (offloadable) travels in bit 15.
  rkc_claim_telemetry* rec;
  glb_u32x2* slot2;
  __device__ __forceinline__ static u32 pack_rejected(u32 id, u32 packed) {
    return id | ((packed & 0x7FFFu) | ((packed >> 16) << 15)) << 16;
  }
  // live claims, one per lane of each set (a vector of NQ registers, so that the sets stay in
  // registers whatever the compiler does with the loops over them)
  typedef typename QSets<NQ>::type qv;
  qv qa;  // id | chain
  qv qb;  // L | T
  qv qc;  // meta | slot
  qv qd;  // duration | blocked count
  qv qe;  // demote step | expire step
  qv qf;  // predicate-failure step | harm step
  u32 tv;  // pool telemetry word `lane`
  // scalars
  // E: the evictable blocks, those of chains above their hold and protection plus the private runs
  // of finished requests (write no-admit pools never keep private runs)
  u32 F, A, PR, peak, E;
  u32 nreq, ncl, nexp;
  u32 sweep_due;  // a victim fell inside a claim whose predicate held: sweep at the end of the step
  u32 vic, post;  // victims, post-release losses (pool telemetry words 10 and 12)
  u32 nslot;      // claim slots used
  // Scalars that only a few paths touch live in LDS (`cold`), so that the registers carried around
  // the event loop are the hot counters only: node free-list head and bump allocator, the FIFO of
  // private runs (head, tail, the front run's eviction key, or KINF when there is none, and its
  // bounds), the status word, the deferral ring (head, length, DEFERRED outcomes of the head
  // entry; every entry behind the head has had exactly one), and the second tier's use and peak.
  lds_u32* cold;
  // (QH..FLO is one 16-byte group, DQH, DQL an 8-byte group: keep their word offsets aligned)
  enum : u32 { C_QH = 0, C_QT, C_FKEY, C_FLO, C_FTOP, C_FNODE, C_BUMP, C_STATUS,
               C_DQH, C_DQL, C_DQC, C_T2, C_T2PK, C_WORDS };
  static_assert(C_QH % 4 == 0 && C_DQH % 2 == 0 && C_DQL == C_DQH + 1 && C_WORDS <= 16, "cold block layout");
  u32 qh, qt, fk, flo, ftop;    // valid between cold_fifo_in() and cold_fifo_out()
  __device__ __forceinline__ void cold_fifo_in() {
    const u32x4 v = *(lds_u32x4*)(cold + C_QH);  // QH, QT, FKEY, FLO
    qh = ufl(v.x); qt = ufl(v.y); fk = ufl(v.z); flo = ufl(v.w); ftop = ufl(cold[C_FTOP]);
  }
  __device__ __forceinline__ void cold_fifo_out() {
    *(lds_u32x4*)(cold + C_QH) = u32x4{qh, qt, fk, flo};
    cold[C_FTOP] = ftop;
  }
  __device__ __forceinline__ void set_status(u32 bits) { cold[C_STATUS] = ufl(cold[C_STATUS]) | bits; }

  // -- telemetry: word w lives in lane w of tv.  The word index is made opaque here so that the
  //    lane comparison is done where it is used, instead of being hoisted out of the event loop as
  //    one 64-bit lane mask per word (which exhausts the scalar registers). --
  __device__ __forceinline__ void tadd(u32 w, u32 v) {
    asm volatile("" : "+s"(w));
    tv += lane == w ? v : 0u;
  }

  // -- chain records --
  __device__ __forceinline__ G0 rd0(u32 c) {
    const u32x4 v = ch[vx(c)];
    const u32 a = ufl(v.x), b = ufl(v.y), d = ufl(v.z), e = ufl(v.w);
    // (only hard-protection pools ever protect positions: elsewhere the field is 0, and saying so
    // here lets the compiler drop the protection terms from those pools' loops)
    return G0{lo16(a), hi16(a), hardm() ? lo16(b) : 0u, hi16(b), lo16(d), hi16(d), lo16(e), hi16(e)};
  }
  __device__ __forceinline__ void wr0(u32 c, const G0& g) {
    u32x4 v;
    v.x = pk(g.n, g.hold); v.y = pk(g.prot, g.bt); v.z = pk(g.nx, g.covA); v.w = pk(g.stop, g.sbot);
    ch[vx(c)] = v;
  }
  __device__ __forceinline__ u32 chain_n(u32 c) { return lo16(((lds_u32*)(ch + c))[0]); }
  __device__ __forceinline__ u32 chain_hold(u32 c) { return hi16(((lds_u32*)(ch + c))[0]); }

  // -- touch-stack nodes: x | t, up | down --
  __device__ __forceinline__ u32x2 nget(u32 i) {
    u32x2 v;
    if (i < NL) v = ndl[vx(i)]; else v = *gat(ndg, i - NL);
    v.x = ufl(v.x); v.y = ufl(v.y);
    return v;
  }
  __device__ __forceinline__ void nset(u32 i, u32x2 v) {
    if (i < NL) ndl[vx(i)] = v; else *gat(ndg, i - NL) = v;
  }
  __device__ __forceinline__ void nset_y(u32 i, u32 y) {
    if (i < NL) ((lds_u32*)(ndl + vx(i)))[1] = y; else ((__attribute__((address_space(1))) u32*)gat(ndg, i - NL))[1] = y;
  }
  // (the free list head and the bump pointer are read and written in the cold block where they
  // are needed: a touch that reuses a popped node needs neither)
  __device__ __forceinline__ u32 nalloc() {
    u32 i;
    const u32 fn = ufl(cold[C_FNODE]);
    if (fn != NIL) {
      i = fn;
      cold[C_FNODE] = hi16(nget(i).y);
    } else {
      const u32 b = ufl(cold[C_BUMP]);
      if (b < ncap()) {
        i = b;
        cold[C_BUMP] = b + 1;
      } else {
        set_status(0x80000000u);  // cannot happen: one node per touch, at most node cap - 2 touches
        i = 0;
      }
    }
    return i;
  }

  // -- chain counters: E (evictable blocks) and PR (protected cached blocks) --
  __device__ __forceinline__ static u32 evictable(u32 n, u32 hold, u32 prot) {
    const u32 lo = max(hold, prot);
    return n > lo ? n - lo : 0u;
  }
  __device__ __forceinline__ static u32 protd(u32 hold, u32 prot) { return prot > hold ? prot - hold : 0u; }

  // -- what the claims on a chain imply, computed from the claim lanes when it matters --
  // this lane's claim of set q is live (claim index 64 q + lane below the live count)
  __device__ __forceinline__ bool live(u32 q) const { return q * 64u + lane < ncl; }
  // ... and on chain c
  __device__ __forceinline__ bool on_chain(u32 c, u32 q) const { return live(q) && hi16(qa[q]) == c; }
  // ... and ranks victims at soft level prio + 1 (accepted soft or lowered claims still
  // materialized, and demoted claims; §3.1 soft priority, demotion to soft)
  __device__ __forceinline__ bool leveled(u32 c, u32 q) const {
    const u32 m = lo16(qc[q]), st = m_state(m);
    return on_chain(c, q) && ((st == ST_MATERIALIZED && m_eff(m) == RKC_PROT_SOFT) || st == ST_DEMOTED);
  }
  // this lane's claim of set q is a materialized hard claim (hard protection in effect)
  __device__ __forceinline__ bool hmat(u32 q) const {
    const u32 m = lo16(qc[q]);
    return live(q) && m_state(m) == ST_MATERIALIZED && m_eff(m) == RKC_PROT_HARD;
  }
  // relaxation order of this lane's claim of set q: priority, then id
  __device__ __forceinline__ u32 rkey(u32 q) const { return (m_prio(lo16(qc[q])) << 16) | lo16(qa[q]); }
  // soft level of position p of chain c
  __device__ __forceinline__ u32 level_of(u32 c, u32 p) const {
    u32 v = 0;
#pragma unroll
    for (u32 q = 0; q < NQ; q++) v = max(v, leveled(c, q) && lo16(qb[q]) > p ? m_prio(lo16(qc[q])) + 1u : 0u);
    return wmax(v);
  }
  // positions at or above the result have a level <= lvl: the largest footprint of the claims
  // ranking above lvl (they all end at or below the position where level lvl starts)
  __device__ __forceinline__ u32 level_floor(u32 c, u32 lvl) const {
    u32 v = 0;
#pragma unroll
    for (u32 q = 0; q < NQ; q++) v = max(v, leveled(c, q) && m_prio(lo16(qc[q])) + 1u > lvl ? lo16(qb[q]) : 0u);
    return wmax(v);
  }

  // Key of chain c's top run; advances a stale stack bottom (the node above it reaches n).
  // (Control flow on the event path is written without early exits: the compiler's structurizer
  // turns every break / early return into flow blocks with register copies paid by every event.)
  // (moved: set when the stack bottom advanced, i.e. the record's bottom fields changed)
  __device__ __forceinline__ u32 top_key(u32 c, G0& g, bool& moved) {
    u32 key = KINF;
    if (g.n > max(g.hold, g.prot)) {
      if (g.nx >= g.n) {
        moved = true;
        // (rare: the node free list is read and written here, not kept in registers around it)
        u32 fn = ufl(cold[C_FNODE]);
        u32 b = g.sbot;
        u32x2 nb = nget(b);
        u32 up = lo16(nb.y), nxv = 0;
        bool go = up != NIL;
        for (u32 guard = 0; go && guard < 0x10000u; guard++) {
          const u32x2 nu = nget(up);
          nxv = lo16(nu.x);
          if (nxv >= g.n) {
            // node b leaves the stack: free it; up becomes the bottom (its down link is cut)
            nset_y(b, pk(NIL, fn));
            fn = b;
            b = up;
            nb = nu;
            up = lo16(nb.y);
            nxv = 0;
            go = up != NIL;
          } else {
            go = false;
          }
        }
        nset_y(b, pk(up, NIL));
        cold[C_FNODE] = fn;
        g.sbot = b;
        g.bt = hi16(nb.x);
        g.nx = nxv;
      }
      // no claim reaches the top position unless covA >= n
      const u32 lvl = (softl() && g.covA >= g.n) ? level_of(c, g.n - 1) : 0u;
      // (formed on the vector unit, where the key is stored from)
      key = (lvl << 25) | (vx(g.bt) << 9) | (c + 1);
    }
    return key;
  }

  // Record a touch of positions [0, x) of chain c at step t (x > 0).
  __device__ __forceinline__ void touch(G0& g, u32 x, u32 t) {
    u32 tp = g.stop, tpd = NIL, reuse = NIL;
    bool go = tp != NIL;
    for (u32 guard = 0; go && guard < 0x10000u; guard++) {
      const u32x2 nt = nget(tp);
      tpd = hi16(nt.y);
      if (lo16(nt.x) <= x) {
        // the node leaves the stack; the last one to leave becomes the new node, the others go to
        // the free list
        if (reuse != NIL) {
          nset_y(reuse, pk(NIL, ufl(cold[C_FNODE])));
          cold[C_FNODE] = reuse;
        }
        reuse = tp;
        tp = tpd;
        go = tp != NIL;
      } else {
        go = false;
      }
    }
    const u32 nw = reuse != NIL ? reuse : nalloc();
    nset(nw, u32x2{pk(x, t), pk(NIL, tp)});
    if (tp != NIL) {
      nset_y(tp, pk(nw, tpd));
      if (tp == g.sbot) g.nx = x;  // the new node sits right above the bottom
    } else {
      g.sbot = nw;                 // the new node is the whole stack
      g.bt = t;
      g.nx = 0;
    }
    g.stop = nw;
  }

  // Apply new (n, hold, prot) to chain c (keeping E and PR exact), optionally touch [0, x)
  // at t, refresh the key and store the record.
  __device__ __forceinline__ void commit(u32 c, G0 g, u32 nn, u32 hh, u32 pp, u32 x, u32 t) {
    E += evictable(nn, hh, pp) - evictable(g.n, g.hold, g.prot);
    PR += protd(hh, pp) - protd(g.hold, g.prot);
    g.n = nn; g.hold = hh; g.prot = pp;
    if (x) touch(g, x, t);
    bool moved = false;
    kk[vx(c)] = top_key(c, g, moved);
    wr0(c, g);
  }

  // After a lifecycle change of claims on chain c: the extent of its live claims, its hard
  // protection extent (hard-protection pools), and its key (soft levels may have changed).
  __device__ __forceinline__ void recompute(u32 c) {
    u32 pv = 0, cv = 0;
#pragma unroll
    for (u32 q = 0; q < NQ; q++) {
      const u32 L = lo16(qb[q]), m = lo16(qc[q]);
      const bool on = on_chain(c, q);
      pv = max(pv, (on && hardm() && m_state(m) == ST_MATERIALIZED && m_eff(m) == RKC_PROT_HARD) ? L : 0u);
      cv = max(cv, on && !offl(m) ? L : 0u);
    }
    const u32 pp = hardm() ? wmax(pv) : 0u;  // (0 outside hard protection, known as such)
    G0 g = rd0(c);
    g.covA = wmax(cv);
    commit(c, g, g.n, g.hold, pp, 0, 0);
  }
  // recompute every chain named by a claim lane in `mask` (one lane mask per claim set)
  __device__ __forceinline__ void recompute_lanes(u64 (&mask)[NQ]) {
#pragma unroll
    for (u32 q = 0; q < NQ; q++) {
      for (u32 guard = 0; mask[q] && guard < 64; guard++) {
        const u32 l = (u32)__builtin_ctzll(mask[q]);
        const u32 c = rdl(hi16(qa[q]), l);
        recompute(c);
#pragma unroll
        for (u32 q2 = q; q2 < NQ; q2++) mask[q2] &= ~ballot(hi16(qa[q2]) == c);
      }
    }
  }

  // Record of the live claim in this lane of set q (the caller selects the lanes).
  __device__ __forceinline__ void write_own_record(u32 q, u32 state, i32 rel) {
    const u32 id = lo16(qa[q]), m = lo16(qc[q]);
    const u32 mm = (m & ~7u) | state;
    rkc_claim_telemetry* r = rec + hi16(qc[q]);
    r->w[0] = (i32)id; r->w[1] = (i32)packed_of(mm); r->w[2] = (i32)id;
    r->w[3] = st16(lo16(qe[q])); r->w[4] = st16(hi16(qe[q])); r->w[5] = rel;
    r->w[6] = st16(lo16(qf[q])); r->w[7] = st16(hi16(qf[q])); r->w[8] = (i32)hi16(qd[q]);
  }

  // Expiry at the start of step t (claims materialized or demoted with a duration).
  __device__ __forceinline__ void expire(u32 t, u32& flags, u32& expired) {
    u64 hm[NQ];
    u32 nx = NEVER;
    expired = 0;
#pragma unroll
    for (u32 q = 0; q < NQ; q++) {
      const u32 m = lo16(qc[q]), st = m_state(m), dur = lo16(qd[q]);
      const bool cand = live(q) && (st == ST_MATERIALIZED || st == ST_DEMOTED) && dur != 0;
      const u32 ex = lo16(qa[q]) + dur;
      const bool hit = cand && ex <= t;
      if (ext()) {
        // responsibility ends: an offloaded claim's second-tier copy is dropped
        const bool off = hit && m_eff(m) == RKC_PROT_OFFLOADED;
        if (__builtin_expect(ballot(off) != 0, 0)) {
          cold[C_T2] = ufl(cold[C_T2]) - wsum(off ? lo16(qb[q]) : 0u);
          // its predicate held only through the dropped copy: a chain already shorter than T
          // fails it now (no harm: the claim is expired)
          const bool fail = off && m_pend(m) && chain_n(hi16(qa[q])) < hi16(qb[q]);
          qc[q] = off ? pk(m & ~(3u << 3) & ~(fail ? 1u << 8 : 0u), hi16(qc[q])) : qc[q];
          qf[q] = fail ? pk(t, hi16(qf[q])) : qf[q];
          const u32 nf = (u32)__builtin_popcountll(ballot(fail));
          if (nf) {
            flags |= RKC_FL_PRED_FAIL;
            tadd(TW_PREDFAIL, nf);
          }
        }
      }
      qc[q] = hit ? pk((lo16(qc[q]) & ~7u) | ST_EXPIRED, hi16(qc[q])) : qc[q];
      qe[q] = hit ? pk(lo16(qe[q]), t) : qe[q];
      hm[q] = ballot(hit);
      nx = min(nx, cand && !hit ? ex : NEVER);
      expired += (u32)__builtin_popcountll(hm[q]);
    }
    nexp = wmin(nx);
    if (__builtin_expect(expired != 0, 0)) {
      recompute_lanes(hm);
      flags |= RKC_FL_EXPIRED;
      tadd(TW_EXPIRED, expired);
    }
  }

  // Predicate sweep after evictions: a claim whose chain now holds fewer than T leading blocks
  // fails for the first time; a materialized (accepted) claim is harmed (§3.2).
  __device__ __forceinline__ u32 sweep(u32 t) {
    u64 fm[NQ];
    u32 pf = 0, hc = 0;
#pragma unroll
    for (u32 q = 0; q < NQ; q++) {
      const u32 m = lo16(qc[q]), T = hi16(qb[q]), c = hi16(qa[q]);
      const u32 nc = chain_n(c);
      const bool fail = live(q) && m_pend(m) && nc < T && !offl(m);
      const bool harm = fail && m_state(m) == ST_MATERIALIZED;
      const u32 m2 = (m & ~(1u << 8) & ~(harm ? 7u : 0u)) | (harm ? ST_HARMED : 0u);
      qc[q] = fail ? pk(m2, hi16(qc[q])) : qc[q];
      qf[q] = fail ? pk(t, harm ? t : hi16(qf[q])) : qf[q];
      fm[q] = ballot(fail);
      pf += (u32)__builtin_popcountll(fm[q]);
      hc += (u32)__builtin_popcountll(ballot(harm));
    }
    u32 fl = 0;
    if (__builtin_expect(pf != 0, 0)) {
      tadd(TW_PREDFAIL, pf);
      tadd(TW_HARM, hc);
      recompute_lanes(fm);
      fl = RKC_FL_PRED_FAIL | (hc ? (u32)RKC_FL_HARM : 0u);
    }
    return fl;
  }

  __device__ __forceinline__ void fifo_pop() {
    qh++;
    fk = KINF;
    if (qh != qt) {
      const u32x2 e = *gat(fifo, qh);
      const u32 x = ufl(e.x);
      fk = lo16(x) << 9; flo = hi16(x); ftop = ufl(e.y);
    }
  }

  // ALLOC: FREE blocks first, then the (need - F) smallest-key candidates (§3.1 soft priority;
  // §5.3 ordinary eviction; hard-protected blocks are never candidates).  hc >= 0 names the chain
  // whose leading h blocks are the event's own hits (not candidates).
  __device__ __forceinline__ AllocRes alloc(u32 need, i32 hc, u32 h, const G0& ghc) {
    AllocRes r = {1, 0, 0, 0, 0, 0};
    if (need <= F) {
      F -= need;
    } else {
      u32 Ec = E;
      u32 hlo = 0;  // candidates of chain hc start at hlo
      if (hc >= 0) {
        const u32 lo = max(ghc.hold, ghc.prot);
        hlo = max(lo, h);
        Ec -= sub0(min(ghc.n, hlo), lo);  // = evictable(n, lo) - evictable(n, hlo), hlo >= lo
      }
      r.E = Ec;
      // (F + Ec is at most twice the usable blocks and need at most 2^24: every sum here fits 32 bits)
      if (need > F + Ec) {
        r.ok = 0;
      } else {
        u32 K = need - F;
        F = 0;
        // (every block taken below is a victim, so the victims are K; those inside no live claim
        // are the victims less the resident ones; a feasible allocation is always served)
        const u32 K0 = K;
        vic += K;
        // the front private run's key (the rest of the FIFO state is read when a run is taken)
        u32 kf = noadm() ? KINF : ufl(cold[C_FKEY]);
        // the hit chain stops being a candidate once only hits remain
        if (hc >= 0 && ghc.n <= hlo) kk[vx(hc)] = KINF;
        for (u32 guard = 0; K > 0; guard++) {
          u32 kmin;
          if (NS == 4) {
            const u32x4 k4 = ((lds_u32x4*)kk)[lane];
            kmin = min(min(k4.x, k4.y), min(k4.z, k4.w));
          } else if (NS == 2) {
            const u32x2 k2 = ((lds_u32x2*)kk)[lane];
            kmin = min(k2.x, k2.y);
          } else {
            kmin = kk[lane];
          }
          const u32 m1 = wmin(kmin);
          if (kf < m1) {
            // the oldest finished request's private run (level 0)
            cold_fifo_in();
            const u32 m = min(K, ftop - flo);
            ftop -= m;
            E -= m;
            K -= m;
            if (ftop == flo) fifo_pop();
            cold_fifo_out();
            kf = fk;
          } else if (m1 != KINF) {
            const u32 c = (m1 & 511u) - 1u;
            G0 g = rd0(c);
            const u32 nn = g.n;
            u32 lo = max(g.hold, g.prot);
            if ((i32)c == hc) { lo = max(lo, h); r.hit = 1; }
            // the top run shares (level, last use): positions below nx were touched later,
            // positions below a higher-level claim's footprint rank higher (only claims within
            // covA matter)
            u32 run_lo = max(lo, g.nx);
            if (softl() && g.covA > run_lo) run_lo = max(run_lo, level_floor(c, m1 >> 25));
            const u32 m = min(K, nn - run_lo);
            const u32 nw = nn - m;
            u32 rs = 0, sc = 0;
            if (g.covA > nw) {
              // victims inside live claims: resident; inside only demoted / expired ones: post-release
              u32 cv = 0, due = 0;
#pragma unroll
              for (u32 q = 0; q < NQ; q++) {
                // (the barrier keeps the per-lane claim tests here, where they are needed, instead of
                // ahead of the eviction loop, where every evicting allocation would pay for them;
                // the tests are 0/1 words combined bitwise, so that no lane-dependent branch forms)
                u32 mc = lo16(qc[q]);
                asm volatile("" : "+v"(mc));
                const u32 st = m_state(mc);
                const u32 on = (u32)live(q) & (u32)(hi16(qa[q]) == c) & (u32)!offl(mc);
                // observed (1), materialized (2) or harmed (6)
                const u32 res = (0x46u >> st) & 1u;
                static_assert(ST_OBSERVED == 1 && ST_MATERIALIZED == 2 && ST_HARMED == 6, "state codes");
                cv = max(cv, (on & res) ? lo16(qb[q]) : 0u);
                // a claim whose predicate still holds needs more than nw leading blocks
                due |= on & (u32)(m_pend(mc) != 0) & (u32)(hi16(qb[q]) > nw);
              }
              const u32 covS = wmax(cv);
              rs = min(nn, g.covA) - nw;
              sc = min(nn, covS) > nw ? min(nn, covS) - nw : 0u;
              if (ballot(due)) sweep_due = 1;
            }
            r.resident += rs;
            r.post += rs - sc;
            E -= m;
            g.n = nw;
            K -= m;
            bool moved = false;
            u32 key = top_key(c, g, moved);
            // (the hit chain stops being a candidate once only hits remain; any other chain's key
            // is already KINF when nw <= lo)
            if (nw <= lo) key = KINF;
            kk[vx(c)] = key;
            // (only n changed unless the stack bottom advanced)
            if (moved) wr0(c, g);
            else ((lds_u32*)(ch + vx(c)))[0] = pk(g.n, g.hold);
          } else {
            set_status(0x80000000u);  // cannot happen: feasibility was checked
            K = 0;
          }
          if (__builtin_expect(guard > 0x10000u, 0)) { set_status(0x80000000u); K = 0; }
        }
        r.unclaimed = K0 - r.resident;
      }
    }
    return r;
  }

  // Refusal record of an active event that cannot be served (§3.4; §5.4 refusal record).
  struct Out;
  __device__ __forceinline__ void refusal(u32 need, i32 hc, u32 h, u32 Hc, const G0& ghc, Out& o) {
    u32 Pr = PR;
    if (hardm() && hc >= 0) {
      const u32 p = min(ghc.prot, h);
      Pr -= p > ghc.hold ? p - ghc.hold : 0u;
    }
    const u32 req = A + Hc + need;
    if (Pr > 0 && req <= U()) {
      o.code = RKC_OC_REFUSED_CLAIM;
      u32 mn = NEVER, nb = 0;
#pragma unroll
      for (u32 q = 0; q < NQ; q++) {
        const u32 m = lo16(qc[q]), c = hi16(qa[q]);
        u32 cov = chain_hold(c);
        if ((i32)c == hc) cov = max(cov, h);
        const bool blk = live(q) && m_state(m) == ST_MATERIALIZED && m_eff(m) == RKC_PROT_HARD &&
                         lo16(qb[q]) > cov;
        qd[q] += blk ? (1u << 16) : 0u;
        nb += (u32)__builtin_popcountll(ballot(blk));
        mn = min(mn, blk ? lo16(qa[q]) : NEVER);
      }
      o.id = (i32)wmin(mn);
      o.n16 = min(nb, 65535u);
    } else {
      o.code = RKC_OC_REFUSED_CAPACITY;
      o.id = -1;
      o.n16 = 0;
    }
    o.a = (i32)Pr;
    o.b = (i32)req;
  }

  __device__ __forceinline__ void served(const AllocRes& r, Out& o) {
    o.code = r.resident ? RKC_OC_EVICT_RESIDENT : RKC_OC_ADMIT;
    o.a = (i32)r.resident;
    o.flags |= (r.post ? (u32)RKC_FL_POST_RELEASE_LOSS : 0u) | (r.unclaimed ? (u32)RKC_FL_EVICT_UNCLAIMED : 0u);
    post += r.post;
  }

  // Remove request entry i from the compact list of n entries (n <= 256).
  template <bool L>
  __device__ __forceinline__ void rq_remove_(u32 i, u32 n) {
    for (u32 base = i; base + 1 < n; base += 64) {
      const u32 j = base + lane;
      const u32 src = min(j + 1, n - 1);
      const u32x2 v = rq_ld<L>(src);
      __builtin_amdgcn_wave_barrier();
      if (j + 1 < n) rq_st<L>(j, v);
      __builtin_amdgcn_wave_barrier();
    }
  }
  __device__ __forceinline__ void rq_remove(u32 i, u32 n) {
    if (n <= RQL) rq_remove_<true>(i, n); else rq_remove_<false>(i, n);
  }
  // Insert entry e at its id-ordered place in the compact list of n entries (n below the
  // capacity): entries with larger ids move up one place, highest chunk first.
  template <bool L>
  __device__ __forceinline__ void rq_insert_(u32x2 e, u32 n) {
    const u32 id = lo16(e.x);
    u32 below = 0;
    for (u32 base = 0; base < n; base += 64) {
      const u32 j = base + lane;
      below += (u32)(j < n && lo16(rq_ld<L>(min(j, n - 1)).x) < id);
    }
    const u32 k = wsum(below);
    for (u32 top = n; top > k;) {
      const u32 base = top - k > 64 ? top - 64 : k;
      const u32 j = base + lane;
      const u32x2 v = rq_ld<L>(min(j, top - 1));
      __builtin_amdgcn_wave_barrier();
      if (j < top) rq_st<L>(j + 1, v);
      __builtin_amdgcn_wave_barrier();
      top = base;
    }
    rq_put(k, e);
  }
  __device__ __forceinline__ void rq_insert(u32x2 e, u32 n) {
    if (n + 1 <= RQL) rq_insert_<true>(e, n); else rq_insert_<false>(e, n);
  }
  // largest R of the live requests on chain c
  template <bool L>
  __device__ __forceinline__ u32 rq_hold_(u32 c, u32 n) {
    u32 hv = 0;
    for (u32 base = 0; base < n; base += 64) {
      const u32 j = base + lane;
      const u32x2 v = rq_ld<L>(min(j, n - 1));
      hv = max(hv, (j < n && hi16(v.x) == c) ? lo16(v.y) : 0u);
    }
    return wmax(hv);
  }
  __device__ __forceinline__ u32 rq_hold(u32 c, u32 n) {
    return n <= RQL ? rq_hold_<true>(c, n) : rq_hold_<false>(c, n);
  }

  // ---- event handlers: each fills the outcome fields; no early exits (see top_key) ----
  struct Out {
    u32 code, flags, n16;
    i32 id, a, b;
  };

  __device__ __forceinline__ void dq_pop(u32 dh, u32 dl) {
    *(lds_u32x2*)(cold + C_DQH) = u32x2{dh + 1 == maxr() ? 0u : dh + 1, dl - 1};
    cold[C_DQC] = 1;
  }

  // Runtime relaxation (§3.1 demotable: the downgrade comes before the predicate-breaking
  // eviction; offloadable: the content may leave GPU memory if the predicate stays restorable; §3.5
  // "relax resident claim" and "offload resident").  Before an active allocation of `need` blocks
  // that hard protection makes infeasible, the blocking claims (materialized hard claims reaching a
  // cached position outside the hits) that allow demotion or offload are taken lowest priority
  // first, then lowest id: each is offloaded when it allows it and its footprint fits the second
  // tier's free room, else demoted when it allows it, else left alone, until the allocation would
  // fit; only then do the picked claims change.  Nothing changes when it never fits.  Returns the
  // number of claims relaxed; ghc (the hit chain's record) is re-read when claims changed.
  __device__ __forceinline__ u32 relax(u32 t, u32 need, i32 hc, u32 h, G0& ghc) {
    u32 k = 0;
    if (relax_on() && need > F) {
      u32 Ec = E;
      if (hc >= 0) {
        const u32 lo = max(ghc.hold, ghc.prot);
        Ec -= sub0(min(ghc.n, max(lo, h)), lo);
      }
      u32 avail = F + Ec;
      if (need > avail) {
        // Per lane and claim set q, three bits of `sel`: bit q the claim is a candidate not yet
        // visited, bit 4 + q picked, bit 8 + q picked for offload (the rest of the picks are
        // demoted).  The claim fields are read from the claim registers, which stay unchanged
        // until the picks are applied.
        u32 sel = 0, nleft = 0;
#pragma unroll
        for (u32 q = 0; q < NQ; q++) {
          const u32 m = lo16(qc[q]), c = hi16(qa[q]);
          u32 cov = chain_hold(c);
          if ((i32)c == hc) cov = max(cov, h);
          const bool cand = hmat(q) && (m & (M_DEMQ | M_OFFQ)) && lo16(qb[q]) > cov;
          sel |= cand ? 1u << q : 0u;
          nleft += (u32)__builtin_popcountll(ballot(cand));
        }
        u32 room = sub0(t2cap(), ufl(cold[C_T2])), moved = 0;
        for (u32 guard = 0; nleft > 0 && need > avail && guard < 64u * NQ; guard++) {
          u32 kv = NEVER;
#pragma unroll
          for (u32 q = 0; q < NQ; q++) kv = min(kv, ((sel >> q) & 1u) ? rkey(q) : NEVER);
          const u32 kmin = wmin(kv);
          // the claim with the smallest (priority, id): set lq, lane l (keys are distinct)
          u32 lq = 0, l = 0, ml = 0, Ll = 0, cq = 0;
#pragma unroll
          for (u32 q = 0; q < NQ; q++) {
            const u64 b = ballot(((sel >> q) & 1u) && rkey(q) == kmin);
            if (b) {
              lq = q;
              l = (u32)__builtin_ctzll(b);
              ml = lo16(rdl(qc[q], l)); Ll = lo16(rdl(qb[q], l)); cq = hi16(rdl(qa[q], l));
            }
          }
          sel &= lane == l ? ~(1u << lq) : ~0u;
          nleft--;
          const bool off = (ml & M_OFFQ) && Ll <= room;
          if (off || (ml & M_DEMQ)) {
            if (off) { room -= Ll; moved += Ll; }
            const G0 g = rd0(cq);
            const u32 base = (i32)cq == hc ? max(g.hold, h) : g.hold;
            u32 bv = 0;
#pragma unroll
            for (u32 q = 0; q < NQ; q++) {
              const bool on = hmat(q) && hi16(qa[q]) == cq;
              bv = max(bv, on && !((sel >> (4 + q)) & 1u) ? lo16(qb[q]) : 0u);
            }
            sel |= lane == l ? (1u << (4 + lq)) | (off ? 1u << (8 + lq) : 0u) : 0u;
            u32 av = 0;
#pragma unroll
            for (u32 q = 0; q < NQ; q++) {
              const bool on = hmat(q) && hi16(qa[q]) == cq;
              av = max(av, on && !((sel >> (4 + q)) & 1u) ? lo16(qb[q]) : 0u);
            }
            const u32 before = wmax(bv), after = wmax(av);
            avail += evictable(g.n, base, after) - evictable(g.n, base, before);
          }
        }
        if (need <= avail) {
          u32 no = 0;
          u64 S[NQ];
#pragma unroll
          for (u32 q = 0; q < NQ; q++) {
            const u32 m = lo16(qc[q]);
            const bool o = (sel >> (8 + q)) & 1u, d = ((sel >> (4 + q)) & 1u) && !o;
            qc[q] = d ? pk((m & ~7u) | ST_DEMOTED | M_RELAXED, hi16(qc[q])) : qc[q];
            qc[q] = o ? pk((m & ~(3u << 3)) | (RKC_PROT_OFFLOADED << 3) | M_RELAXED, hi16(qc[q])) : qc[q];
            qe[q] = d ? pk(t, hi16(qe[q])) : qe[q];
            S[q] = ballot((sel >> (4 + q)) & 1u);
            k += (u32)__builtin_popcountll(S[q]);
            no += (u32)__builtin_popcountll(ballot(o));
          }
          recompute_lanes(S);
          tadd(TW_RUNTIME_DEMOTED, k - no);
          if (no) {
            const u32 used = ufl(cold[C_T2]) + moved;
            cold[C_T2] = used;
            cold[C_T2PK] = max(ufl(cold[C_T2PK]), used);
            tadd(TW_OFF_CLAIMS, no);
            tadd(TW_OFF_BLOCKS, moved);
          }
          if (hc >= 0) ghc = rd0((u32)hc);
        }
      }
    }
    return k;
  }

  // Serve request rid (S blocks, shared chain cc when P > 0, shared prefix P) at step t; late: a
  // retried request, inserted into the live list by id and taken off the deferral ring (dh, dl).
  // In relaxing pools, demotable blocking claims are demoted first when that lets it fit.  A
  // refusal on behalf of resident claims defers the request in deferring pools (§3.5 active
  // deferral): a new one enters the ring, a retried one is deferred again while its deferrals
  // last, else refused for good (§5.4 live scheduler run).
  __device__ __forceinline__ void admit(u32 t, u32 rid, u32 S, u32 cc, u32 P, bool late, u32 dh, u32 dl,
                                        Out& o) {
    i32 hc = -1;
    u32 h = 0, Hc = 0;
    G0 g = {0, 0, 0, 0, 0, 0, 0, 0};
    if (P > 0) {
      hc = (i32)cc;
      g = rd0(cc);
      h = min(P, g.n);
      Hc = h > g.hold ? h - g.hold : 0u;
    }
    const u32 need = S - h;
    u32 relaxed = 0;
    if (ext()) relaxed = relax(t, need, hc, h, g);
    const AllocRes r = alloc(need, hc, h, g);
    if (!r.ok) {
      refusal(need, hc, h, Hc, g, o);
      if (ext()) {
        const bool by_claim = o.code == RKC_OC_REFUSED_CLAIM;
        if (late) {
          const u32 cnt = ufl(cold[C_DQC]);
          if (by_claim && cnt < dlim()) {
            cold[C_DQC] = cnt + 1;
            o.code = RKC_OC_DEFERRED;
          } else {
            dq_pop(dh, dl);
            tadd(TW_RETRY_REFUSED, 1);
          }
        } else if (by_claim && dlim() > 0) {
          const u32x2 hl = *(lds_u32x2*)(cold + C_DQH);
          const u32 h0 = ufl(hl.x), l0 = ufl(hl.y);
          if (l0 < maxr()) {
            const u32 slot = h0 + l0 >= maxr() ? h0 + l0 - maxr() : h0 + l0;
            *gat(dq, slot) = u32x4{t, S, cc, P};  // every lane, one value
            cold[C_DQL] = l0 + 1;
            o.code = RKC_OC_DEFERRED;
          }
        }
      }
    } else {
      A += Hc + need;
      u32 R = 0;
      if (hc >= 0) {
        const G0 g2 = r.hit ? rd0(cc) : g;  // victims may have shortened this chain above the hits
        R = noadm() ? h : P;
        const u32 nn = (!noadm() && P > g2.n) ? P : g2.n;
        commit(cc, g2, nn, max(g2.hold, R), g2.prot, R, t);
      }
      const u32x2 e = u32x2{pk(rid, hc >= 0 ? cc : NIL), pk(R, S)};
      if (late) {
        // the live list stays in id order: the retried request goes before later ids
        rq_insert(e, nreq);
        dq_pop(dh, dl);
        tadd(TW_RETRY_SERVED, 1);
      } else {
        rq_put(nreq, e);
      }
      nreq++;
      o.id = (i32)rid;
      o.b = (i32)h;
      served(r, o);
      if (relaxed) { o.code = RKC_OC_RELAXED; o.n16 = min(relaxed, 65535u); }
      if (ext() && P > h && t2cap() > 0) {
        // positions past the hits that a claim holding a second-tier copy covers are restored
        // from the second tier (restore cost), still on new GPU blocks
        u32 ev = 0;
#pragma unroll
        for (u32 q = 0; q < NQ; q++)
          ev = max(ev, on_chain(cc, q) && m_eff(lo16(qc[q])) == RKC_PROT_OFFLOADED ? lo16(qb[q]) : 0u);
        const u32 e = wmax(ev);
        tadd(TW_RESTORED, sub0(min(P, e), h));
      }
    }
  }

  // (bad: the event's fields are out of range, decided for the whole tile by malformed())
  __device__ __forceinline__ void ev_prefill(u32 t, u32 w1, u32 w2, u32 w3, u32 bad, Out& o) {
    if (bad) {
      o.code = RKC_OC_INVALID;
    } else if (nreq >= maxr()) {
      o.code = RKC_OC_INVALID;
      set_status(RKC_PS_REQUEST_TABLE);
    } else {
      admit(t, t, w1, w2, w3, false, 0, 0, o);
    }
  }

  // RETRY (hard-protection pools that defer or relax): the oldest deferred request is served,
  // deferred again or refused.
  __device__ __forceinline__ void ev_retry(u32 t, Out& o) {
    const u32x2 hl = *(lds_u32x2*)(cold + C_DQH);
    const u32 dh = ufl(hl.x), dl = ufl(hl.y);
    if (dl > 0) {
      if (nreq >= maxr()) {
        o.code = RKC_OC_INVALID;  // the request stays queued
        set_status(RKC_PS_REQUEST_TABLE);
      } else {
        const u32x4 q = *gat(dq, dh);
        admit(t, ufl(q.x), ufl(q.y), ufl(q.z), ufl(q.w), true, dh, dl, o);
      }
    }
  }

  __device__ __forceinline__ void ev_extend(u32 t, u32 w1, u32 w2, u32 bad, Out& o) {
    if (bad) {
      o.code = RKC_OC_INVALID;
    } else if (nreq > 0) {
      const u32 i = umod(w2, nreq), need = w1;
      G0 g = {0, 0, 0, 0, 0, 0, 0, 0};
      u32 relaxed = 0;
      if (ext()) relaxed = relax(t, need, -1, 0, g);
      const AllocRes r = alloc(need, -1, 0, g);
      if (!r.ok) {
        refusal(need, -1, 0, 0, g, o);
      } else {
        A += need;
        o.id = (i32)lo16(rq_grow(i, need));
        o.b = (i32)A;
        served(r, o);
        if (relaxed) { o.code = RKC_OC_RELAXED; o.n16 = min(relaxed, 65535u); }
      }
    }
  }

  __device__ __forceinline__ void ev_claim(u32 t, u32 w0, u32 w1, u32 w2, u32 w3, u32 bad, Out& o) {
    if (nslot >= nslots()) {
      o.code = RKC_OC_INVALID;
      set_status(RKC_PS_SLOT_TABLE);
    } else {
      const u32 s = nslot++;
      bool ok = !bad;
      if (ok && ncl >= maxq()) { set_status(RKC_PS_CLAIM_TABLE); ok = false; }
      if (!ok) {
        *gat(slot2, s) = u32x2{0u, pack_rejected(t, 0)};  // every lane, one value
        o.code = RKC_OC_INVALID;
      } else {
        const u32 L = w1, c = w2, T = w3;
        const u32 hardq = (w0 >> 4) & 1u, prio = (w0 >> 5) & 3u, dur = w0 >> 16;
        // a best-effort claim is observed in every policy (§3.1 best_effort: telemetry only)
        const u32 beq = (w0 >> 8) & 1u;
        const u32 req_bits = (w0 & (1u << 7) ? M_DEMQ : 0u) | (beq ? M_BE : 0u) | (w0 & (1u << 9) ? M_OFFQ : 0u);
        const bool obs = shadm() || beq;
        const G0 g = rd0(c);
        const u32 h = min(L, g.n), need = L - h;
        const AllocRes r = alloc(need, (i32)c, h, g);
        const u32 eff = beq ? RKC_PROT_NONE : hardm() ? (hardq ? RKC_PROT_HARD : RKC_PROT_SOFT)
                      : (mode == RKC_MODE_SOFT ? RKC_PROT_SOFT : RKC_PROT_NONE);
        if (!r.ok) {
          const u32 dec = obs ? DEC_SHADOW : DEC_REJECTED;
          const u32 m = ST_REJECTED | (eff << 3) | (hardq << 5) | (prio << 6) | (dec << 9) | req_bits;
          *gat(slot2, s) = u32x2{pk(L, c), pack_rejected(t, packed_of(m))};
          o.code = RKC_OC_MATFAIL;
          o.id = (i32)t;
          o.a = (i32)need;
          o.b = (i32)(F + r.E);
          tadd(TW_ACCEPTED + dec - DEC_ACCEPTED, 1);
        } else {
          *gat(slot2, s) = u32x2{pk(L, c), NEVER};  // every lane, one value
          const u32 lowered = (mode == RKC_MODE_SOFT) && hardq;
          const u32 dec = obs ? DEC_SHADOW : lowered ? DEC_APPROX : DEC_ACCEPTED;
          const u32 st = obs ? ST_OBSERVED : ST_MATERIALIZED;
          o.flags |= obs ? (u32)RKC_FL_SHADOW : lowered ? (u32)RKC_FL_LOWERED : 0u;
          const u32 m = st | (eff << 3) | (hardq << 5) | (prio << 6) | (1u << 8) | (dec << 9) | req_bits;
          const u32 dur_eff = obs ? 0u : dur;  // shadow claims never expire
          const u32 k = ncl++, kq = k >> 6, kl = k & 63u;
#pragma unroll
          for (u32 q = 0; q < NQ; q++) {
            if (NQ == 1 || q == kq) {
              qa[q] = wrl(qa[q], pk(t, c), kl);
              qb[q] = wrl(qb[q], pk(L, T), kl);
              qc[q] = wrl(qc[q], pk(m, s), kl);
              qd[q] = wrl(qd[q], dur_eff, kl);
              qe[q] = wrl(qe[q], 0xFFFFFFFFu, kl);
              qf[q] = wrl(qf[q], 0xFFFFFFFFu, kl);
            }
          }
          if (dur_eff > 0) nexp = min(nexp, t + dur_eff);
          G0 g2 = r.hit ? rd0(c) : g;
          g2.covA = max(g2.covA, L);
          // a materialized hard claim in a hard-protection pool protects [0, L)
          const u32 pp = eff == RKC_PROT_HARD ? max(g2.prot, L) : g2.prot;
          commit(c, g2, max(g2.n, L), g2.hold, pp, L, t);
          o.id = (i32)t;
          o.b = (i32)need;
          served(r, o);
          tadd(TW_ACCEPTED + dec - DEC_ACCEPTED, 1);
        }
      }
    }
  }

  __device__ __forceinline__ void ev_finish(u32 t, u32 w1, Out& o) {
    if (nreq > 0) {
      const u32 i = umod(w1, nreq);
      const u32x2 e = rq_get(i);
      const u32 rid = lo16(e.x), c = hi16(e.x), R = lo16(e.y), len = hi16(e.y);
      rq_remove(i, nreq);
      nreq--;
      u32 turned = 0;
      if (c != NIL) {
        const G0 g = rd0(c);
        // the chain's hold is the largest R of its live requests: it can change only when this
        // request held it (R == hold), and only then are the others scanned
        const u32 hn = R < g.hold ? g.hold : rq_hold(c, nreq);
        turned += R > hn ? R - hn : 0u;
        commit(c, g, g.n, hn, g.prot, R, t);
      }
      // write no-admit drops the request's own blocks; otherwise they become a private run
      const u32 own = len - R;
      const u32 dropped = noadm() ? own : 0u;
      const u32 kept = own - dropped;
      turned += kept;
      F += dropped;
      E += kept;
      if (kept > 0) {
        cold_fifo_in();
        if (qh == qt) { fk = t << 9; flo = R; ftop = len; }
        *gat(fifo, qt) = u32x2{pk(t, R), len};  // every lane, one value
        qt++;
        cold_fifo_out();
      }
      // (A only falls here: its peak is taken before each fall and once at the end)
      peak = max(peak, A);
      A -= turned + dropped;
      o.code = RKC_OC_FINISHED;
      o.id = (i32)rid;
      o.a = (i32)turned;
      o.b = (i32)dropped;
      if (dropped) o.flags |= RKC_FL_NOADMIT_DROP;
      tadd(TW_DROPPED, dropped);
    }
  }

  // RELEASE (the selected live claim) or DEMOTE (the selected materialized hard-requested claim,
  // hard -> soft; soft and hard pools only)
  __device__ __forceinline__ void ev_lifecycle(u32 t, u32 type, u32 w1, Out& o) {
    u32 i = NEVER;
    if (type == RKC_EV_RELEASE) {
      if (ncl > 0) i = umod(w1, ncl);
    } else if (softl()) {
      // the (w1 mod count)-th demotable claim in id order (claims sit in id order, set by set)
      u64 cm[NQ];
      u32 cnt = 0;
#pragma unroll
      for (u32 q = 0; q < NQ; q++) {
        const u32 m = lo16(qc[q]);
        cm[q] = ballot(live(q) && m_state(m) == ST_MATERIALIZED && m_hard(m) && !offl(m));
        cnt += (u32)__builtin_popcountll(cm[q]);
      }
      if (cnt > 0) {
        u32 k = umod(w1, cnt);
#pragma unroll
        for (u32 q = 0; q < NQ; q++) {
          const u32 pc = (u32)__builtin_popcountll(cm[q]);
          if (i == NEVER && k < pc) {
            const u32 rank = __builtin_amdgcn_mbcnt_hi((u32)(cm[q] >> 32), __builtin_amdgcn_mbcnt_lo((u32)cm[q], 0u));
            i = 64u * q + (u32)__builtin_ctzll(ballot(((cm[q] >> lane) & 1ull) && rank == k));
          } else if (i == NEVER) {
            k -= pc;
          }
        }
      }
    }
    if (i != NEVER) {
      const u32 iq = i >> 6, il = i & 63u;
      u32 qav = 0, qbv = 0, qcv = 0;
#pragma unroll
      for (u32 q = 0; q < NQ; q++) {
        if (NQ == 1 || q == iq) { qav = rdl(qa[q], il); qbv = rdl(qb[q], il); qcv = rdl(qc[q], il); }
      }
      const u32 qid = lo16(qav), c = hi16(qav);
      if (type == RKC_EV_RELEASE) {
#pragma unroll
        for (u32 q = 0; q < NQ; q++)
          if ((NQ == 1 || q == iq) && lane == il) write_own_record(q, ST_RELEASED, (i32)t);
        if (ext() && m_eff(lo16(qcv)) == RKC_PROT_OFFLOADED) cold[C_T2] = ufl(cold[C_T2]) - lo16(qbv);
        // close the gap: claims above i move down one place (lane 63 of a set takes lane 0 of the
        // next set, read before that set moves)
#pragma unroll
        for (u32 q = 0; q < NQ; q++) {
          if (q >= iq) {
            const bool up = q > iq || lane >= il;
            qa[q] = up ? shift_down(qa[q]) : qa[q]; qb[q] = up ? shift_down(qb[q]) : qb[q];
            qc[q] = up ? shift_down(qc[q]) : qc[q]; qd[q] = up ? shift_down(qd[q]) : qd[q];
            qe[q] = up ? shift_down(qe[q]) : qe[q]; qf[q] = up ? shift_down(qf[q]) : qf[q];
            if (q + 1 < NQ) {
              qa[q] = wrl(qa[q], rdl(qa[q + 1], 0), 63); qb[q] = wrl(qb[q], rdl(qb[q + 1], 0), 63);
              qc[q] = wrl(qc[q], rdl(qc[q + 1], 0), 63); qd[q] = wrl(qd[q], rdl(qd[q + 1], 0), 63);
              qe[q] = wrl(qe[q], rdl(qe[q + 1], 0), 63); qf[q] = wrl(qf[q], rdl(qf[q + 1], 0), 63);
            }
          }
        }
        ncl--;
        o.code = RKC_OC_RELEASED;
        tadd(TW_RELEASED, 1);
      } else {
#pragma unroll
        for (u32 q = 0; q < NQ; q++) {
          const bool me = (NQ == 1 || q == iq) && lane == il;
          qc[q] = me ? pk((lo16(qc[q]) & ~7u) | ST_DEMOTED, hi16(qc[q])) : qc[q];
          qe[q] = me ? pk(t, hi16(qe[q])) : qe[q];
        }
        o.code = RKC_OC_DEMOTED;
        tadd(TW_DEMOTED, 1);
      }
      recompute(c);
      const u32 nc = ufl(chain_n(c));
      o.id = (i32)qid;
      o.a = (i32)min(nc, lo16(qbv));
      o.b = (i32)hi16(qbv);
    }
  }

  // Malformed events of a tile (lane k holds event k, and its flag): field ranges of PREFILL,
  // EXTEND and CLAIM, decided for all 64 events at once (the table limits are checked per event,
  // in order).
  __device__ __forceinline__ u32 malformed(u32 e0, u32 e1, u32 e2, u32 e3) const {
    const u32 ty = e0 & 15u;
    const i32 s1 = (i32)e1, s2 = (i32)e2, s3 = (i32)e3;
    const bool fb = s1 < 1 || s1 > RKC_MAX_FIELD_BLOCKS;
    const bool cb = s2 < 0 || e2 >= nch();
    const bool bad = (ty == RKC_EV_PREFILL && (fb || s3 < 0 || s3 > s1 || (s3 > 0 && cb))) ||
                     (ty == RKC_EV_EXTEND && fb) ||
                     (ty == RKC_EV_CLAIM && (fb || cb || s3 < 0 || s3 > s1));
    return (u32)bad;
  }

  // One event: its outcome fields in o (the caller assembles the outcome words of a whole tile at
  // once).  Dispatch is an if / else chain in order of how often the event types occur in the
  // benchmark mixes.
  __device__ __forceinline__ void step(u32 t, u32 w0, u32 w1, u32 w2, u32 w3, u32 bad, Out& o) {
    const u32 type = w0 & 15u;
    // (every outcome that is not quiet sets id, a and b; a quiet one gets id -1 and a = b = 0 when
    // the tile's outcome words are assembled, so they start unspecified here and no path pays for
    // materializing them)
    const i32 any = __builtin_nondeterministic_value(0);
    o = Out{RKC_OC_NOOP, 0, 0, any, any, any};
    // (claims in native and write no-admit pools are only observed, and observed claims never
    // expire: those loops carry no expiry)
    if (!shadm() && __builtin_expect(t >= nexp, 0)) {
      u32 expired;
      expire(t, o.flags, expired);
      // n16 is the claims expired at the start of the step unless the event sets it
      o.n16 = min(expired, 65535u);
    }
    if (type == RKC_EV_PREFILL) ev_prefill(t, w1, w2, w3, bad, o);
    else if (type == RKC_EV_EXTEND) ev_extend(t, w1, w2, bad, o);
    else if (type == RKC_EV_CLAIM) ev_claim(t, w0, w1, w2, w3, bad, o);
    else if (type == RKC_EV_FINISH) ev_finish(t, w1, o);
    else if (type == RKC_EV_RELEASE || type == RKC_EV_DEMOTE) ev_lifecycle(t, type, w1, o);
    else if (ext() && type == RKC_EV_RETRY) ev_retry(t, o);
    else if ((type & ~1u) != RKC_EV_NOP) o.code = RKC_OC_INVALID;  // NOP, or RETRY with no ring
    static_assert(RKC_EV_NOP == 6 && RKC_EV_RETRY == 7, "NOP and RETRY differ in bit 0 only");
    if (__builtin_expect(sweep_due != 0, 0)) {
      sweep_due = 0;
      o.flags |= sweep(t);
    }
  }
};

// Replay of one pool with policy MODE (the descriptor has been checked by the caller).
template <int NS, int NQ, int MODE, bool EXT>
__device__ __forceinline__ void replay_pool(const rkc_lean_args& g, const rkc_pool_desc& d, u32 pool,
                                            unsigned char* lds_raw, const rkc_event* __restrict__ evs) {
  typedef Lean<NS, NQ, MODE, EXT> LP;
  LP P;
  P.lane = __lane_id();
  const i64 ev_off = d.event_offset, slot_off = d.claim_slot_offset;
  rkc_pool_telemetry* ptel = g.pool_tel + pool;
  {
    const u32 l = P.lane;
    P.cst = l == 0 ? (u32)d.usable_blocks : l == 1 ? (u32)d.n_chains : l == 2 ? (u32)d.max_live_claims
          : l == 3 ? (u32)d.max_live_requests : l == 4 ? (u32)d.n_claim_slots : l == 5 ? g.node_cap
          : l == 6 ? (u32)d.defer_limit : l == 7 ? (u32)((d.mode & RKC_MODE_RELAX) != 0)
          : (u32)d.offload_blocks;
  }
  const u32 U = (u32)d.usable_blocks, nch = (u32)d.n_chains, nslots = (u32)d.n_claim_slots;

  lds_u32* lds = (lds_u32*)lds_raw;
  typedef LdsMap<NS, NQ> M;
  P.kk = lds + M::KEYS / 4;
  P.ch = (lds_u32x4*)(lds + M::CH / 4);
  P.rq = (lds_u32x2*)(lds + M::RQ / 4);
  P.ndl = (lds_u32x2*)(lds + M::ND / 4);
  unsigned char* scr = (unsigned char*)g.scratch + (u64)pool * g.scr_pool_bytes;
  P.ndg = (glb_u32x2*)(scr + g.scr_off_nodes);
  P.fifo = (glb_u32x2*)(scr + g.scr_off_fifo);
  P.slot2 = (glb_u32x2*)(scr + g.scr_off_slots);
  P.dq = (glb_u32x4*)(scr + g.scr_off_defer);
  P.rqg = (glb_u32x2*)(scr + g.scr_off_reqs);
  P.rec = g.claim_tel + slot_off;

  for (u32 c = P.lane; c < LP::KC; c += 64) P.kk[c] = KINF;
  P.hist = lds + M::HIST / 4;
  if (P.lane < 16) P.hist[P.lane] = 0;
  const u32 nrec = nch > 0 ? nch : 1u;
  for (u32 c = P.lane; c < nrec; c += 64) {
    P.ch[c] = u32x4{0, 0, 0, pk(NIL, NIL)};
  }
#pragma unroll
  for (u32 q = 0; q < NQ; q++) P.qa[q] = P.qb[q] = P.qc[q] = P.qd[q] = P.qe[q] = P.qf[q] = 0;
  P.tv = 0;
  P.F = U; P.A = 0; P.PR = 0; P.peak = 0; P.E = 0;
  P.nreq = 0; P.ncl = 0; P.nexp = NEVER; P.sweep_due = 0; P.vic = 0; P.post = 0; P.nslot = 0;
  P.cold = lds + M::COLD / 4;
  if (P.lane < LP::C_WORDS)
    P.cold[P.lane] = P.lane == LP::C_FNODE ? NIL : P.lane == LP::C_DQC ? 1u : P.lane == LP::C_FKEY ? KINF : 0u;
  __syncthreads();

  const rkc_event* __restrict__ ev = evs + ev_off;
  rkc_outcome* out = g.outcomes + ev_off;
  const u32 ne = (u32)d.n_events;
  for (u32 base = 0; base < ne; base += 64) {
    const u32 cnt = min(64u, ne - base);
    u32 e0 = 0, e1 = 0, e2 = 0, e3 = 0;
    if (P.lane < cnt) {
      const int4 x = *(const int4*)(ev + base + P.lane);
      e0 = (u32)x.x; e1 = (u32)x.y; e2 = (u32)x.z; e3 = (u32)x.w;
    }
    const u32 badv = P.malformed(e0, e1, e2, e3);
    // outcome fields of event k go to lane k; the words are assembled for the tile at once
    u32 vcode = 0, vflags = 0, vn16 = 0, vid = 0, va = 0, vb = 0;
    for (u32 k = 0; k < cnt; k++) {
      typename LP::Out o;
      // (the event's words straight into scalar registers: a scalar load from the read-only event
      // array instead of four lane reads of the tile's vector load, which serves the tile-wide
      // checks; a 32-bit byte offset to the tile's base keeps the address a single shift; the
      // event's malformed flag is read from its lane, one vector instruction in place of a 64-bit
      // scalar shift and a mask)
      const int4 xe = *(const int4*)((const char*)(ev + base) + (k << 4));
      P.step(base + k, (u32)xe.x, (u32)xe.y, (u32)xe.z, (u32)xe.w, rdl(badv, k), o);
      vcode = wrl(vcode, o.code, k); vflags = wrl(vflags, o.flags, k); vn16 = wrl(vn16, o.n16, k);
      vid = wrl(vid, (u32)o.id, k); va = wrl(va, (u32)o.a, k); vb = wrl(vb, (u32)o.b, k);
    }
    // no-op and invalid outcomes carry id -1, a = b = 0
    const bool quiet = vcode == RKC_OC_NOOP || vcode == RKC_OC_INVALID;
    const u32 o0 = vcode | (vflags << 8) | (vn16 << 16);
    const u32 o1 = quiet ? 0xFFFFFFFFu : vid, o2 = quiet ? 0u : va, o3 = quiet ? 0u : vb;
    if (P.lane < cnt) *(int4*)(out + base + P.lane) = make_int4((i32)o0, (i32)o1, (i32)o2, (i32)o3);
    // outcomes per code; resident victims (a) and leading hits (b of a served prefill)
    const u32 oc = o0 & 255u;
    __hip_atomic_fetch_add(P.hist + (P.lane < cnt ? oc : 15u), 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
    const bool srv = P.lane < cnt && (oc <= RKC_OC_EVICT_RESIDENT || (LP::ext() && oc == RKC_OC_RELAXED));
    P.tadd(TW_RESIDENT, wsum(srv ? o2 : 0u));
    const u32 ty = e0 & 15u;
    P.tadd(TW_HITS, wsum(srv && (ty == RKC_EV_PREFILL || (LP::ext() && ty == RKC_EV_RETRY)) ? o3 : 0u));
  }

  const u32 nslot_used = P.nslot;
  const u32 vic = P.vic, post = P.post;
  const u32 status = ufl(P.cold[LP::C_STATUS]), queued = ufl(P.cold[LP::C_DQL]);
  const u32 t2peak = ufl(P.cold[LP::C_T2PK]);
  // Final records of the claims still live (each lane writes its own) ...
#pragma unroll
  for (u32 q = 0; q < NQ; q++)
    if (P.live(q)) P.write_own_record(q, m_state(lo16(P.qc[q])), -1);
  __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "workgroup");
  // ... then lead_end = min(final leading registered length, L) of every used slot, and blank
  // records for unused slots.
  for (u32 s = P.lane; s < nslots; s += 64) {
    if (s < nslot_used) {
      const u32x2 v = P.slot2[s];
      const i32 le = (i32)min(P.chain_n(hi16(v.x)), lo16(v.x));
      if (v.y == NEVER) {
        P.rec[s].w[9] = le;
      } else {
        const u32 pw = hi16(v.y);
        const i32 packed = (i32)((pw & 0x7FFFu) | ((pw >> 15) << 16));
        P.rec[s] = rkc_claim_telemetry{{(i32)lo16(v.y), packed, -1, -1, -1, -1, -1, -1, 0, le}};
      }
    } else {
      P.rec[s] = rkc_claim_telemetry{{-1, 0, -1, -1, -1, -1, -1, -1, 0, 0}};
    }
  }
  __syncthreads();
  {
    const u32 w = P.lane;
    i32 v = (i32)P.tv;
    if (w < 10) v += (i32)P.hist[w];
    if (w == 32) v += (i32)P.hist[RKC_OC_DEFERRED];
    if (w == 36) v += (i32)P.hist[RKC_OC_RELAXED];
    if (w == 41) v = (i32)t2peak;
    if (w == TW_VICTIMS) v = (i32)vic;
    else if (w == TW_POST) v = (i32)post;
    else if (w == 24) v = (i32)max(P.peak, P.A);
    else if (w == 25) v = (i32)P.A;
    else if (w == 26) v = (i32)(U - P.F - P.A);
    else if (w == 27) v = (i32)P.F;
    else if (w == 28) v = (i32)P.PR;
    else if (w == 29) v = (i32)P.nreq;
    else if (w == 30) v = (i32)P.ncl;
    else if (w == 31) v = (i32)status;
    else if (w == 35) v = (i32)queued;
    ptel->w[w] = v;
  }
}

// Event loop a pool runs: 0 hard protection with deferral or relaxation, 1 hard, 2 soft, 3 native,
// 4 no-admit, 5 a descriptor the replay rejects (heaviest loops first).
__device__ __forceinline__ u32 loop_class(const rkc_pool_desc& d) {
  const i32 m = d.mode & ~RKC_MODE_RELAX;
  if (m < 0 || m > 3) return 5u;
  if (m == RKC_MODE_HARD) return (d.defer_limit > 0 || (d.mode & RKC_MODE_RELAX)) ? 0u : 1u;
  return m == RKC_MODE_SOFT ? 2u : m == RKC_MODE_LRU ? 3u : 4u;
}

// Launch order: the pools grouped by the event loop they run, so that the workgroups resident on a
// CU execute one loop and share its instructions in the instruction cache (pools of mixed policies
// side by side thrash it: ~9 % of the replay time on a batch cycling through the four policies).
// Two short passes over 1,024-pool tiles: count each tile's pools per loop class, then scatter
// every pool to its class's range (tiles in order, pools within a tile in wave-arrival order).
// Every pool index appears exactly once; the replay does not depend on the order.
constexpr u32 kOrderTile = 1024, kClasses = 6;

__global__ __launch_bounds__(1024) void rkc_lean_order_count(const rkc_pool_desc* pools, i32 n_pools,
                                                              unsigned char* cls, u32* tile_count) {
  __shared__ u32 cnt[kClasses];
  const u32 tid = threadIdx.x, lane = __lane_id();
  if (tid < kClasses) cnt[tid] = 0;
  __syncthreads();
  const i32 p = (i32)(blockIdx.x * kOrderTile + tid);
  const u32 k = p < n_pools ? loop_class(pools[p]) : 7u;
  if (p < n_pools) cls[p] = (unsigned char)k;
  for (u32 c = 0; c < kClasses; c++) {
    const u64 m = __ballot(k == c);
    if (m && lane == (u32)__builtin_ctzll(m)) atomicAdd(&cnt[c], (u32)__builtin_popcountll(m));
  }
  __syncthreads();
  if (tid < kClasses) tile_count[blockIdx.x * kClasses + tid] = cnt[tid];
}

__global__ __launch_bounds__(1024) void rkc_lean_order_scatter(i32 n_pools, const unsigned char* cls,
                                                                const u32* tile_count, u32* order) {
  __shared__ u32 cur[kClasses];
  const u32 tid = threadIdx.x, lane = __lane_id(), tiles = gridDim.x;
  if (tid < kClasses) {
    // start of this tile's share of class tid: every pool of lower classes, then this class's
    // pools in lower tiles
    u32 start = 0;
    for (u32 t = 0; t < tiles; t++) {
      for (u32 c = 0; c < tid; c++) start += tile_count[t * kClasses + c];
      if (t < blockIdx.x) start += tile_count[t * kClasses + tid];
    }
    cur[tid] = start;
  }
  __syncthreads();
  const i32 p = (i32)(blockIdx.x * kOrderTile + tid);
  const u32 k = p < n_pools ? (u32)cls[p] : 7u;
  for (u32 c = 0; c < kClasses; c++) {
    const u64 m = __ballot(k == c);
    if (m) {
      const u32 first = (u32)__builtin_ctzll(m);
      u32 at = 0;
      if (lane == first) at = atomicAdd(&cur[c], (u32)__builtin_popcountll(m));
      at = (u32)__shfl((int)at, (int)first);
      const u32 rank = __builtin_amdgcn_mbcnt_hi((u32)(m >> 32), __builtin_amdgcn_mbcnt_lo((u32)m, 0u));
      if (k == c) order[at + rank] = (u32)p;
    }
  }
}

// Batch order (pools of a few events: grouping them by event loop does not pay for its passes).
__global__ __launch_bounds__(1024) void rkc_lean_order_identity(i32 n_pools, u32* order) {
  const i32 p = (i32)(blockIdx.x * kOrderTile + threadIdx.x);
  if (p < n_pools) order[p] = (u32)p;
}

// One wavefront per pool, in the launch order above; the pool's policy selects its specialized
// event loop once.  With four claim sets the registers, not LDS, bound residency: the kernel is
// held to 6 waves per SIMD (80 vector registers, a few values spilled to scratch; 5 waves and 93
// registers otherwise, measured slower: nested 9.9 vs 9.3 ms).
template <int NS, int NQ>
// (the events come as a separate restrict-qualified argument as well, so that the compiler knows no
// store of the replay reaches them and may read them through the scalar cache)
__global__ __launch_bounds__(64, NQ > 1 ? 6 : 1) void rkc_lean(rkc_lean_args g, const rkc_event* __restrict__ evs) {
  extern __shared__ __align__(16) unsigned char lds_raw[];
  if ((i32)blockIdx.x >= g.n_pools) return;
  const u32 pool = ((const u32*)((const unsigned char*)g.scratch + g.scr_off_order))[blockIdx.x];
  const u32 lane = __lane_id();
  const rkc_pool_desc d = g.pools[pool];
  const i64 ev_off = d.event_offset, slot_off = d.claim_slot_offset;
  rkc_pool_telemetry* ptel = g.pool_tel + pool;
  const bool ev_ok = d.n_events >= 0 && ev_off >= 0 && ev_off + d.n_events <= g.n_events_total;
  const bool sl_ok = d.n_claim_slots >= 0 && slot_off >= 0 && slot_off + d.n_claim_slots <= g.n_slots_total;
  const bool ok = ev_ok && sl_ok && d.usable_blocks >= 1 && d.usable_blocks <= g.max_usable &&
                  (d.mode & ~RKC_MODE_RELAX) >= 0 && (d.mode & ~RKC_MODE_RELAX) <= 3 &&
                  d.n_events <= g.max_events && d.n_chains >= 0 &&
                  d.n_chains <= g.max_chains && d.max_live_claims >= 0 && d.max_live_claims <= g.max_claims &&
                  d.max_live_requests >= 0 && d.max_live_requests <= g.max_reqs &&
                  d.n_claim_slots <= g.max_slots && d.defer_limit >= 0 && d.offload_blocks >= 0 &&
                  d.reserved[0] == 0 && d.reserved[1] == 0 && d.reserved[2] == 0;
  if (!ok) {
    if (ev_ok)
      for (i32 i = (i32)lane; i < d.n_events; i += 64) g.outcomes[ev_off + i] = rkc_outcome{{RKC_OC_INVALID, -1, 0, 0}};
    if (sl_ok)
      for (i32 i = (i32)lane; i < d.n_claim_slots; i += 64)
        g.claim_tel[slot_off + i] = rkc_claim_telemetry{{-1, 0, -1, -1, -1, -1, -1, -1, 0, 0}};
    ptel->w[lane] = lane == 31 ? RKC_PS_DESCRIPTOR : (lane == RKC_OC_INVALID && ev_ok) ? d.n_events : 0;
    return;
  }
  const u32 mode = (u32)__builtin_amdgcn_readfirstlane(d.mode & ~RKC_MODE_RELAX);
  const u32 ext = (u32)__builtin_amdgcn_readfirstlane(d.defer_limit) > 0 || (d.mode & RKC_MODE_RELAX);
  if (mode == RKC_MODE_LRU) replay_pool<NS, NQ, RKC_MODE_LRU, false>(g, d, pool, lds_raw, evs);
  else if (mode == RKC_MODE_SOFT) replay_pool<NS, NQ, RKC_MODE_SOFT, false>(g, d, pool, lds_raw, evs);
  else if (mode == RKC_MODE_NOADMIT) replay_pool<NS, NQ, RKC_MODE_NOADMIT, false>(g, d, pool, lds_raw, evs);
  else if (!ext) replay_pool<NS, NQ, RKC_MODE_HARD, false>(g, d, pool, lds_raw, evs);
  else replay_pool<NS, NQ, RKC_MODE_HARD, true>(g, d, pool, lds_raw, evs);
}

u64 align_up(u64 v, u64 a) { return (v + a - 1) / a * a; }

}  // namespace

// Layout of the compact kernel for batch b, or false when the batch is outside its limits.
bool rkc_lean_layout(const rkc_batch* b, rkc_lean_args* g) {
  // up to 64 live claims with up to 256 chains, or up to 256 live claims (four claim sets) with up
  // to 64 chains
  const bool many_claims = b->max_live_claims > 64;
  if (b->max_usable_blocks > 32767 || b->max_events > 65533 || b->max_chains > (many_claims ? 64 : 256) ||
      b->max_live_claims > 256 || b->max_live_requests > 256 || b->max_claim_slots > 65534)
    return false;
  const u32 chains = b->max_chains > 0 ? (u32)b->max_chains : 1u;
  const u32 ns = chains <= 64 ? 1u : chains <= 128 ? 2u : 4u;
  g->nq = many_claims ? 4u : 1u;
  const u32 reqs = b->max_live_requests > 0 ? (u32)b->max_live_requests : 1u;
  g->ns = ns;
  g->node_cap = (u32)b->max_events + 2;
  u32 rql;
  if (g->nq == 4) {
    g->lds_bytes = LdsMap<1, 4>::BYTES; g->nodes_lds = LdsMap<1, 4>::NL; rql = LdsMap<1, 4>::RQL;
  } else if (ns == 1) {
    g->lds_bytes = LdsMap<1, 1>::BYTES; g->nodes_lds = LdsMap<1, 1>::NL; rql = LdsMap<1, 1>::RQL;
  } else if (ns == 2) {
    g->lds_bytes = LdsMap<2, 1>::BYTES; g->nodes_lds = LdsMap<2, 1>::NL; rql = LdsMap<2, 1>::RQL;
  } else {
    g->lds_bytes = LdsMap<4, 1>::BYTES; g->nodes_lds = LdsMap<4, 1>::NL; rql = LdsMap<4, 1>::RQL;
  }
  u64 s = 0;
  g->scr_off_nodes = s;
  s += 8ull * (g->node_cap > g->nodes_lds ? g->node_cap - g->nodes_lds : 0u);
  s = align_up(s, 256);
  g->scr_off_fifo = s; s += 8ull * ((u64)b->max_events + 1); s = align_up(s, 256);
  g->scr_off_slots = s; s += 8ull * (u64)(b->max_claim_slots > 0 ? b->max_claim_slots : 1);
  s = align_up(s, 256);
  g->scr_off_defer = s; s += 16ull * reqs;
  s = align_up(s, 256);
  g->scr_off_reqs = s; s += 8ull * (reqs > rql ? reqs - rql : 0u);
  g->scr_pool_bytes = align_up(s, 256);
  const u64 np = b->n_pools > 0 ? (u64)b->n_pools : 0u;
  const u64 tiles = (np + kOrderTile - 1) / kOrderTile;
  g->scr_off_order = g->scr_pool_bytes * np;
  g->scr_off_cls = g->scr_off_order + align_up(4ull * np, 256);
  g->scr_off_tiles = g->scr_off_cls + align_up(np, 256);
  g->scr_total = g->scr_off_tiles + align_up(4ull * kClasses * tiles, 256);
  return true;
}

#ifdef RKC_CHECK_UNIFORM
unsigned rkc_lean_uniform_violations(void) {
  unsigned v = 0;
  if (hipMemcpyFromSymbol(&v, HIP_SYMBOL(g_lean_uniform_violations), sizeof v) != hipSuccess) return ~0u;
  return v;
}
#endif

template <int NS, int NQ>
rkc_status launch_ns(const rkc_lean_args* g, hipStream_t s) {
  if (g->lds_bytes > 64 * 1024 &&
      hipFuncSetAttribute((const void*)rkc_lean<NS, NQ>, hipFuncAttributeMaxDynamicSharedMemorySize,
                          (int)g->lds_bytes) != hipSuccess)
    return RKC_E_HIP;
  unsigned char* scr = (unsigned char*)g->scratch;
  const unsigned tiles = (unsigned)(((u64)g->n_pools + kOrderTile - 1) / kOrderTile);
  if (g->max_events >= 64) {
    // long event loops: group the pools by loop so that a CU's resident pools share one loop
    hipLaunchKernelGGL(rkc_lean_order_count, dim3(tiles), dim3(kOrderTile), 0, s, g->pools, (i32)g->n_pools,
                       scr + g->scr_off_cls, (u32*)(scr + g->scr_off_tiles));
    hipLaunchKernelGGL(rkc_lean_order_scatter, dim3(tiles), dim3(kOrderTile), 0, s, (i32)g->n_pools,
                       (const unsigned char*)(scr + g->scr_off_cls), (const u32*)(scr + g->scr_off_tiles),
                       (u32*)(scr + g->scr_off_order));
  } else {
    hipLaunchKernelGGL(rkc_lean_order_identity, dim3(tiles), dim3(kOrderTile), 0, s, (i32)g->n_pools,
                       (u32*)(scr + g->scr_off_order));
  }
  if (hipGetLastError() != hipSuccess) return RKC_E_HIP;
  hipLaunchKernelGGL((rkc_lean<NS, NQ>), dim3((unsigned)g->n_pools), dim3(64), g->lds_bytes, s, *g, g->events);
  return hipGetLastError() == hipSuccess ? RKC_OK : RKC_E_HIP;
}

rkc_status rkc_lean_launch(const rkc_lean_args* g, hipStream_t s) {
  if (g->nq == 4) return launch_ns<1, 4>(g, s);
  if (g->ns == 1) return launch_ns<1, 1>(g, s);
  if (g->ns == 2) return launch_ns<2, 1>(g, s);
  return launch_ns<4, 1>(g, s);
}
