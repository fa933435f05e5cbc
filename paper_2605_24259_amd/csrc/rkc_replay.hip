// rkc_replay.hip -- batched replay of resident-KV-claim arbitration on MI355X (gfx950).
//
// One wavefront replays one pool.  Pools are independent (the contract is per pool), so the grid is
// one 64-lane workgroup per pool and the hardware dispatcher balances them over the 256 CUs.
//
// The pool is not kept one block at a time.  Because every touch, hit, hold, protection and claim
// coverage is a leading range [0, x) of a chain, the registered positions of every shared chain are
// always a leading run [0, n_c) and eviction always takes a chain from its top.  The kernel therefore
// keeps one 64-byte record per shared chain in LDS:
//   n      registered length              hold   leading positions held ACTIVE by live requests
//   prot   max L of materialized hard claims (hard-protection pools)
//   lv[v]  max L of claims that rank victims at soft level v (priority + 1)
//   covA   max L of live claims           covS   max L of live claims not demoted / expired
//   tpend  max T of claims whose predicate has not failed yet
//   a touch stack: (x, t) pairs, x strictly decreasing, t increasing; position p was last touched
//          at the t of the newest pair with x > p; its bottom pair's step (bt) and the extent of
//          the pair above it (nx) are cached in the record
// and the eviction key (level, last use) of each chain's top candidate (in registers for the first
// 256 chains).  Finished requests' private blocks form runs (finish step, [lo, top)); runs
// finish in step order, so they sit in a FIFO and the front run is always the oldest.
//
// Victim selection takes the (need - F) smallest keys (level asc, last use asc, pos desc) over all
// candidates (§3.1 soft priority; §5.3 ordinary eviction after free blocks; hard-protected blocks
// excluded).  It merges chain tops: a wave min-reduction finds the chain with the smallest top key,
// then a whole run of equal (level, last use) is evicted at once.  Every event touches at most one
// chain, so (level, last use) already identifies a chain's top run: no two chains ever share it.
// The only possible tie is between a chain and the private run of the request that finished at the
// step that touched it; that run lies above every position of the chain that the finish touched
// (the request's shared prefix ends where its own blocks begin), so the private run goes first.
//
// Everything the pool's logic reads with a uniform address is moved into scalar registers
// (readfirstlane), so the per-event state machine runs on the scalar unit; lanes are used for scans
// over claims and requests, for DPP reductions, and to hold the pool's counters (lane k = word k).
//
// LDS holds the chain records, the live-request and live-claim lists and the first touch-stack
// nodes; global scratch holds the remaining nodes, the FIFO ring and the per-slot (chain, L) table.
// Scratch is only read back by the lane(s) that wrote it, or after a workgroup fence.
#include <hip/hip_runtime.h>
#include <stdint.h>
#include <string.h>

#include <mutex>

#include "rkc.h"
#include "rkc_lean.h"

// Built-in device scratch of rkc_replay_batch_noalloc, for callers that cannot allocate.  Each device
// the library runs on holds its own copy until the process ends.  Host code never passes this name to
// a kernel or a copy: it is a host-side stand-in; the device address comes from hipGetSymbolAddress.
static __device__ __align__(256) unsigned char scratch[RKC_NOALLOC_SCRATCH_BYTES];

namespace {

typedef uint32_t u32;
typedef int32_t i32;
typedef uint64_t u64;
typedef int64_t i64;

// Explicit address spaces, so every access compiles to a ds_ or global_ instruction, never a flat one.
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) u32 lds_u32;
typedef __attribute__((address_space(3))) u32x4 lds_u32x4;
typedef __attribute__((address_space(3))) uint4 lds_uint4;
typedef __attribute__((address_space(3))) u64 lds_u64;
typedef __attribute__((address_space(1))) u32 glb_u32;
typedef __attribute__((address_space(1))) uint4 glb_uint4;

// Storage width of LDS-resident pool state: 16-bit words when every stored position, step, index
// and count is below 0xFFFF (usable blocks <= 32,767, events <= 65,533), else 32-bit words.  All
// arithmetic is 32-bit; the all-ones word of either width stands for NIL.
template <typename W> struct Store;
template <> struct Store<uint16_t> {
  typedef __attribute__((address_space(3))) uint16_t lds_w;
  typedef unsigned short w4 __attribute__((ext_vector_type(4)));
  typedef __attribute__((address_space(3))) w4 lds_w4;
  static constexpr u32 wnil = 0xFFFFu;
};
template <> struct Store<u32> {
  typedef lds_u32 lds_w;
  typedef u32x4 w4;
  typedef lds_u32x4 lds_w4;
  static constexpr u32 wnil = 0xFFFFFFFFu;
};
// lists in LDS with the pool's word width, or in global scratch as 32-bit words
template <typename W, bool kGL> struct ListMem { typedef typename Store<W>::lds_w word; };
template <typename W> struct ListMem<W, true> { typedef glb_u32 word; };

constexpr u32 NIL = 0xFFFFFFFFu;
constexpr u32 KEY_INF = 0xFFFFFFFFu;
constexpr u32 EXP_NEVER = 0xFFFFFFFFu;

// claim states (ResidentClaimState, §3.1) and decisions
enum : u32 { ST_SUBMITTED = 0, ST_OBSERVED = 1, ST_MATERIALIZED = 2, ST_DEMOTED = 3, ST_EXPIRED = 4,
             ST_RELEASED = 5, ST_HARMED = 6, ST_REJECTED = 7 };
enum : u32 { DEC_ACCEPTED = 1, DEC_APPROX = 2, DEC_SHADOW = 3, DEC_REJECTED = 4 };

// chain record words (four 16-byte groups)
enum : u32 { CF_N = 0, CF_HOLD = 1, CF_PROT = 2, CF_BT = 3,          // group 0
             CF_NX = 4, CF_COVA = 5, CF_COVS = 6, CF_TPEND = 7,      // group 1
             CF_LV = 8,                                              // group 2: lv[0..3]
             CF_STOP = 12, CF_SBOT = 13, CF_HCNT = 14,               // group 3
             CF_WORDS = 16 };

// live-claim list arrays (struct of arrays, capacity cl_cap each)
// (the demotion, expiry, predicate-failure and harm steps go straight into the claim's record in
// the caller's telemetry buffer when they happen: they are never read on the event path)
enum : u32 { CL_ID = 0, CL_C, CL_L, CL_T, CL_META, CL_EXP, CL_SLOT, CL_BLK, CL_ARRAYS };
// words of a claim record written when the step happens
enum : u32 { RW_DEM = 3, RW_EXST = 4, RW_PF = 6, RW_HARM = 7 };
// live-request list arrays
enum : u32 { RQ_ID = 0, RQ_C, RQ_R, RQ_LEN, RQ_ARRAYS };

// pool telemetry words kept in lane k of one register
enum : u32 { TW_VICTIMS = 10, TW_RESIDENT = 11, TW_POST = 12, TW_DROPPED = 13, TW_HITS = 14,
             TW_ACCEPTED = 15, TW_HARM = 19, TW_PREDFAIL = 20, TW_EXPIRED = 21, TW_DEMOTED = 22,
             TW_RELEASED = 23, TW_DEFERRED = 32, TW_RETRY_SERVED = 33, TW_RETRY_REFUSED = 34,
             TW_QUEUED = 35, TW_RELAXED = 36, TW_RUNTIME_DEMOTED = 37, TW_OFF_CLAIMS = 38,
             TW_OFF_BLOCKS = 39, TW_RESTORED = 40, TW_T2_PEAK = 41 };

// live-claim meta word: state[0:3) eff[3:5) hard[5] prio[6:8) pending[8] decision[9:12)
// demotable[12] best_effort[13] relaxed_by_runtime[14] offloadable[15] (16 bits)
constexpr u32 M_DEMQ = 1u << 12, M_BE = 1u << 13, M_RELAXED = 1u << 14, M_OFFQ = 1u << 15;
__device__ __forceinline__ u32 m_with_eff(u32 m, u32 e) { return (m & ~(3u << 3)) | (e << 3); }
__device__ __forceinline__ u32 m_state(u32 m) { return m & 7u; }
__device__ __forceinline__ u32 m_eff(u32 m) { return (m >> 3) & 3u; }
__device__ __forceinline__ u32 m_hard(u32 m) { return (m >> 5) & 1u; }
__device__ __forceinline__ u32 m_prio(u32 m) { return (m >> 6) & 3u; }
__device__ __forceinline__ u32 m_pending(u32 m) { return (m >> 8) & 1u; }
__device__ __forceinline__ u32 m_dec(u32 m) { return (m >> 9) & 7u; }
__device__ __forceinline__ u32 m_with_state(u32 m, u32 s) { return (m & ~7u) | s; }

__device__ __forceinline__ u32 packed_of(u32 m) {
  return m_dec(m) | (m_state(m) << 4) | (m_hard(m) << 8) | (m_prio(m) << 9) | (m_eff(m) << 11) |
         (((m >> 12) & 15u) << 13);
}

// eviction key of a run of candidates with one (level, last use); steps are below 2^24
__device__ __forceinline__ u32 make_key(u32 level, u32 lu) { return (level << 28) | lu; }

// ---- wave primitives ------------------------------------------------------------------------
__device__ __forceinline__ u32 lane_id() { return __lane_id(); }
__device__ __forceinline__ u64 ballot(bool p) { return __ballot(p); }
__device__ __forceinline__ i32 rdlane(i32 v, u32 l) { return __builtin_amdgcn_readlane(v, (int)l); }
// A value every lane holds identically, moved to a scalar register.  Built with RKC_CHECK_UNIFORM
// (a checking build, never the product one), every call also verifies that the active lanes agree
// and counts the calls where they do not.
#ifdef RKC_CHECK_UNIFORM
__device__ unsigned int g_wave_uniform_violations;
__device__ __forceinline__ u32 ufl(u32 v) {
  const u32 f = (u32)__builtin_amdgcn_readfirstlane((int)v);
  if (__ballot(v != f) != 0 && __lane_id() == (u32)__builtin_ctzll(__ballot(true)))
    atomicAdd(&g_wave_uniform_violations, 1u);
  return f;
}
#else
__device__ __forceinline__ u32 ufl(u32 v) { return (u32)__builtin_amdgcn_readfirstlane((int)v); }
#endif
__device__ __forceinline__ uint4 ufl4(uint4 v) { return make_uint4(ufl(v.x), ufl(v.y), ufl(v.z), ufl(v.w)); }

// Cross-lane reductions with DPP row permutes (no LDS round trip): within each 16-lane row,
// combine lanes i^1, i^2, the mirrored half-row and the mirrored row, so every lane of a row holds
// the row's result; then combine the four rows through readlane.  All 64 lanes must be active.
template <int CTRL>
__device__ __forceinline__ u32 dpp(u32 v) {
  return (u32)__builtin_amdgcn_update_dpp((int)v, (int)v, CTRL, 0xF, 0xF, false);
}
constexpr int kDppXor1 = 0xB1;       // quad_perm [1,0,3,2]
constexpr int kDppXor2 = 0x4E;       // quad_perm [2,3,0,1]
constexpr int kDppHalfMirror = 0x141;
constexpr int kDppMirror = 0x140;

struct OpMax { __device__ static u32 f(u32 a, u32 b) { return a > b ? a : b; } };
struct OpMin { __device__ static u32 f(u32 a, u32 b) { return a < b ? a : b; } };
struct OpAdd { __device__ static u32 f(u32 a, u32 b) { return a + b; } };

template <class Op>
__device__ __forceinline__ u32 wave_reduce(u32 v) {
  v = Op::f(v, dpp<kDppXor1>(v));
  v = Op::f(v, dpp<kDppXor2>(v));
  v = Op::f(v, dpp<kDppHalfMirror>(v));
  v = Op::f(v, dpp<kDppMirror>(v));
  const u32 r0 = (u32)rdlane((i32)v, 0), r1 = (u32)rdlane((i32)v, 16);
  const u32 r2 = (u32)rdlane((i32)v, 32), r3 = (u32)rdlane((i32)v, 48);
  return Op::f(Op::f(r0, r1), Op::f(r2, r3));
}
__device__ __forceinline__ u32 wave_max(u32 v) { return wave_reduce<OpMax>(v); }
__device__ __forceinline__ u32 wave_min(u32 v) { return wave_reduce<OpMin>(v); }
__device__ __forceinline__ u32 wave_sum(u32 v) { return wave_reduce<OpAdd>(v); }


// ---- launch geometry (computed on the host) ---------------------------------------------------
struct Layout {
  u32 chains, reqs, claims, nodes_lds;
  u32 off_chain, off_mark, off_key, off_rq, off_cl, off_node, off_job;
  u32 lds_bytes;
  u64 scr_pool_bytes, scr_off_node, scr_off_fifo, scr_off_slot, scr_off_dq, scr_off_rq, scr_off_cl;
  u32 fifo_cap, node_cap;
  u32 global_lists, narrow;
  u32 waves;  // waves per pool (1, or kGroupWaves for the workgroup-per-pool kernel)
};

struct Args {
  const rkc_pool_desc* pools;
  const rkc_event* events;
  rkc_outcome* outcomes;
  rkc_pool_telemetry* pool_tel;
  rkc_claim_telemetry* claim_tel;
  unsigned char* scratch;
  i64 n_events_total, n_slots_total;
  i32 n_pools, max_usable, max_events, max_chains, max_reqs, max_claims, max_slots;
  Layout L;
};

enum : u32 { MK_SWEEP = 1, MK_RECOMP = 2 };

// Workgroup per pool (NW > 1 waves): wave 0 runs the per-event state machine; the other waves wait
// on the workgroup barrier and join the scans that cover a pool's live lists.  Wave 0 posts a job
// (a word and its arguments on the LDS job board) and passes a barrier; every wave then takes its
// share of the scan (entries wave * 64 + lane, stepping 64 * NW), reduces it across its lanes and
// leaves up to 8 partial results on the board; a second barrier, and wave 0 combines them.
enum : u32 { J_EXIT = 0, J_MAXIMA, J_EXPIRE, J_SWEEP, J_ATTRIB, J_HOLD, J_MOVE };
constexpr u32 JB_ARGS = 16;   // board words before the partials (job word + arguments)
constexpr u32 kGroupWaves = 8; // waves per pool in the workgroup-per-pool kernel
// internal-consistency fault bit in the pool status word: set only if a structural bound that
// the algorithm guarantees is ever violated; loops stop instead of running on.
constexpr u32 kFault = 0x80000000u;
// chains whose top keys live in registers (four per lane)
constexpr u32 kRegChains = 256;

struct AllocRes {
  u32 ok;
  i32 E;  // evictable candidates before the event (valid when need > F)
  i32 victims, resident, post, unclaimed;
};

// ---- the per-pool replay ----------------------------------------------------------------------
// kGL: the live-request and live-claim lists live in global scratch instead of LDS (pools whose
// lists do not fit on chip).  Lane-parallel writes to them are then followed by a workgroup fence
// before any other lane reads them.
template <typename W, bool kGL, int NW>
struct Pool {
  static_assert(NW >= 1 && 8 * NW <= 64, "at most 8 waves per pool");
  static constexpr u32 kSpan = 64u * NW;  // entries one pass of the workgroup covers
  typedef typename ListMem<W, kGL>::word lword;
  typedef typename Store<W>::lds_w lds_w;
  typedef typename Store<W>::w4 w4;
  typedef typename Store<W>::lds_w4 lds_w4;
  static constexpr u32 kListNil = kGL ? 0xFFFFFFFFu : Store<W>::wnil;
  static constexpr u32 kWordNil = Store<W>::wnil;
  // descriptor
  i32 U, mode, n_events, n_chains, max_claims, max_reqs, n_slots, defer_limit;
  u32 relax_on;  // the pool relaxes demotable hard claims (mode flag RKC_MODE_RELAX)
  u32 t2cap, t2used, t2peak;  // second tier: capacity, blocks held by offloaded claims, peak
  u32 lane;
  u32 wave;           // wave index in the workgroup (wave 0 runs the state machine)
  lds_u32* jb;        // job board (NW > 1)
  // memory
  lds_w* ch;          // chain records, CF_WORDS words each
  lds_u32* mk;        // per-chain mark bits
  lds_u32* tk;        // top keys of chains >= kRegChains
  lword* rq;          // live requests, RQ_ARRAYS arrays of rq_cap (stride)
  lword* cl;          // live claims, CL_ARRAYS arrays of cl_cap
  u32 rq_cap, cl_cap;
  // Lists in global scratch: entry 0 of the live-request list sits at rq_head, with twice the
  // table's capacity allocated, so a finish can close its gap from whichever side is shorter.
  u32 rq_head;
  lds_w4* node_lds;   // nodes [0, nl)
  glb_uint4* node_glb;  // nodes [nl, node_cap), 32-bit words
  u32 nl, node_cap;
  uint4* fifo;  // private runs in finish order; one push per event at most, so it never wraps
  uint2* slot_cl;
  // deferred requests (active deferral): a ring of max_reqs entries (PREFILL step, S, chain, P);
  // dq_cnt counts the DEFERRED outcomes of the head entry (every entry behind it has had one)
  uint4* dq;
  u32 dq_head, dq_len, dq_cnt;
  rkc_claim_telemetry* rec;
  // registers
  u32 kr0, kr1, kr2, kr3;  // top key of chain 64 * k + lane, k = 0..3
  u32 tv;                  // pool telemetry word `lane`
  // scalar state (wave-uniform)
  i32 F, A, PR, peak;
  i32 Eall;       // sum over chains of max(0, n - max(hold, prot)): evictable shared blocks
  u32 nreq, ncl, nslot;
  u32 next_exp;
  u32 free_head, bump;
  u32 fhead, ftail, ft, flo, ftop;
  i32 fblocks;
  u32 status;

  // -- telemetry words held lane-distributed --
  __device__ __forceinline__ void tadd(u32 w, u32 v) { tv += lane == w ? v : 0u; }

  // -- chain records --
  __device__ __forceinline__ static u32 widen(u32 v, u32 wnil) { return v == wnil ? NIL : v; }
  __device__ __forceinline__ u32 cf(u32 c, u32 f) { return ufl(ch[c * CF_WORDS + f]); }
  __device__ __forceinline__ u32 cfn(u32 c, u32 f) { return widen(cf(c, f), kWordNil); }  // NIL-able field
  __device__ __forceinline__ void cs(u32 c, u32 f, u32 v) { ch[c * CF_WORDS + f] = (W)v; }
  __device__ __forceinline__ uint4 cg(u32 c, u32 g) {
    const w4 v = ((lds_w4*)(ch + c * CF_WORDS))[g];
    return ufl4(make_uint4(v.x, v.y, v.z, v.w));
  }
  __device__ __forceinline__ void cgs(u32 c, u32 g, uint4 v) {
    w4 w;
    w.x = (W)v.x; w.y = (W)v.y; w.z = (W)v.z; w.w = (W)v.w;
    ((lds_w4*)(ch + c * CF_WORDS))[g] = w;
  }

  // -- lists --
  __device__ __forceinline__ lword* cla(u32 k) { return cl + k * cl_cap; }
  __device__ __forceinline__ lword* rqa(u32 k) { return rq + k * rq_cap + (kGL ? rq_head : 0u); }
  __device__ __forceinline__ static u32 lnil(u32 v) { return v == kListNil ? NIL : v; }
  __device__ __forceinline__ void lists_fence() {
    if (kGL) __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "workgroup");
  }

  // -- cooperative scans --
  __device__ __forceinline__ u32 first() const { return wave * 64u + lane; }
  // wave 0: post a job and its arguments, and release the other waves into it
  __device__ __forceinline__ void post(u32 job, u32 a0 = 0, u32 a1 = 0, u32 a2 = 0, u32 a3 = 0, u32 a4 = 0) {
    if (NW > 1) {
      if (lane < 6)
        jb[lane] = lane == 0 ? job : lane == 1 ? a0 : lane == 2 ? a1 : lane == 3 ? a2 : lane == 4 ? a3 : a4;
      __syncthreads();
    }
  }
  __device__ __forceinline__ u32 arg(u32 k) { return ufl(jb[1 + k]); }
  // Publish this wave's partial results p[0..NP) and, on wave 0, combine the waves' partials: slot k
  // takes the maximum where bit k of maxs is set, the minimum where bit k of mins is set, else the sum.
  template <u32 NP>
  __device__ __forceinline__ void exchange(u32 (&p)[NP], u32 maxs, u32 mins) {
    if (NW > 1) {
      u32 v = 0;
#pragma unroll
      for (u32 k = 0; k < NP; k++) v = lane == k ? p[k] : v;
      if (lane < NP) jb[JB_ARGS + 8 * wave + lane] = v;
      __syncthreads();
      if (wave == 0) {
        const u32 x = lane < 8 * NW ? (u32)jb[JB_ARGS + lane] : 0u;
#pragma unroll
        for (u32 k = 0; k < NP; k++) {
          u32 r = (u32)rdlane((i32)x, k);
#pragma unroll
          for (u32 w = 1; w < (u32)NW; w++) {
            const u32 y = (u32)rdlane((i32)x, 8 * w + k);
            r = ((maxs >> k) & 1u) ? max(r, y) : ((mins >> k) & 1u) ? min(r, y) : r + y;
          }
          p[k] = r;
        }
      }
    }
  }
  __device__ __forceinline__ void mark_or(u32 c, u32 bit) {
    if (NW > 1) __hip_atomic_fetch_or(mk + c, bit, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
    else mk[c] |= bit;
  }

  // -- nodes (x = extent, y = step, z = up (newer), w = down (older)); the first nl live in LDS,
  //    the rest in global scratch (read and written by every lane with uniform addresses) --
  __device__ __forceinline__ uint4 nget(u32 i) {
    uint4 v;
    if (i < nl) {
      const w4 r = node_lds[i];
      v = make_uint4(r.x, r.y, widen(r.z, kWordNil), widen(r.w, kWordNil));
    } else {
      const glb_uint4& r = node_glb[i - nl];
      v = make_uint4(r.x, r.y, r.z, r.w);
    }
    return ufl4(v);
  }
  __device__ __forceinline__ u32 nget_x(u32 i) { u32 v; if (i < nl) v = node_lds[i].x; else v = node_glb[i - nl].x; return ufl(v); }
  __device__ __forceinline__ u32 nget_z(u32 i) { u32 v; if (i < nl) v = widen(node_lds[i].z, kWordNil); else v = node_glb[i - nl].z; return ufl(v); }
  __device__ __forceinline__ u32 nget_w(u32 i) { u32 v; if (i < nl) v = widen(node_lds[i].w, kWordNil); else v = node_glb[i - nl].w; return ufl(v); }
  __device__ __forceinline__ void nset(u32 i, uint4 v) {
    if (i < nl) {
      w4 w;
      w.x = (W)v.x; w.y = (W)v.y; w.z = (W)v.z; w.w = (W)v.w;
      node_lds[i] = w;
    } else {
      node_glb[i - nl].x = v.x; node_glb[i - nl].y = v.y; node_glb[i - nl].z = v.z; node_glb[i - nl].w = v.w;
    }
  }
  __device__ __forceinline__ void nset_z(u32 i, u32 v) { if (i < nl) node_lds[i].z = (W)v; else node_glb[i - nl].z = v; }
  __device__ __forceinline__ void nset_w(u32 i, u32 v) { if (i < nl) node_lds[i].w = (W)v; else node_glb[i - nl].w = v; }
  __device__ __forceinline__ u32 node_alloc() {
    u32 i;
    if (free_head != NIL) {
      i = free_head;
      free_head = nget_w(i);
    } else if (bump < node_cap) {
      i = bump++;
    } else {
      // cannot happen: every touch allocates one node and a pool has at most node_cap - 2 events
      status |= kFault;
      i = 0;
    }
    return i;
  }
  __device__ __forceinline__ void node_free(u32 i) {
    nset_w(i, free_head);
    free_head = i;
  }

  // -- top keys: registers for chains < kRegChains, LDS above --
  __device__ __forceinline__ void set_key(u32 c, u32 k) {
    if (c < kRegChains) {
      const u32 l = c & 63u, s = c >> 6;
      if (lane == l) {
        if (s == 0) kr0 = k;
        else if (s == 1) kr1 = k;
        else if (s == 2) kr2 = k;
        else kr3 = k;
      }
    } else {
      tk[c] = k;
    }
  }

  // -- chain counters: every change of n, hold or prot keeps Eall and PR (protected cached
  //    blocks, hard-protection pools) exact --
  __device__ __forceinline__ static i32 evictable(u32 nn, u32 hh, u32 pp) { return max(0, (i32)nn - (i32)max(hh, pp)); }
  __device__ __forceinline__ void chain_update(u32 c, uint4 g0, u32 nn, u32 hh, u32 pp) {
    Eall += evictable(nn, hh, pp) - evictable(g0.x, g0.y, g0.z);
    PR += max(0, (i32)pp - (i32)hh) - max(0, (i32)g0.z - (i32)g0.y);
    cgs(c, 0, make_uint4(nn, hh, pp, g0.w));
  }

  __device__ __forceinline__ bool soft_levels() const { return mode == RKC_MODE_SOFT || mode == RKC_MODE_HARD; }

  // soft level of position p and the lowest position sharing it
  __device__ __forceinline__ u32 level_at(uint4 lv, u32 p, u32& lvb) {
    u32 lvl = 0;
    lvb = 0;
    if (soft_levels()) {
      if (lv.x > p) lvl = 1;
      if (lv.y > p) lvl = 2;
      if (lv.z > p) lvl = 3;
      if (lv.w > p) lvl = 4;
      if (lvl < 1) lvb = max(lvb, lv.x);
      if (lvl < 2) lvb = max(lvb, lv.y);
      if (lvl < 3) lvb = max(lvb, lv.z);
      if (lvl < 4) lvb = max(lvb, lv.w);
    }
    return lvl;
  }

  // Key of chain c's top run.  The stack bottom is the newest pair covering position n-1
  // exactly when the pair above it (extent nx) does not reach n-1; otherwise advance the bottom.
  __device__ __forceinline__ u32 top_key(u32 c) {
    const uint4 g0 = cg(c, 0);
    const u32 nn = g0.x;
    if (nn <= max(g0.y, g0.z)) return KEY_INF;
    u32 t_bot = g0.w;
    if (cf(c, CF_NX) >= nn) {
      u32 b = cfn(c, CF_SBOT);
      if (b == NIL) { status |= kFault; return KEY_INF; }
      u32 up = nget_z(b);
      for (u32 guard = 0; guard < node_cap && up != NIL && nget_x(up) >= nn; guard++) {
        nset_w(up, NIL);
        node_free(b);
        b = up;
        up = nget_z(b);
      }
      cs(c, CF_SBOT, b);
      t_bot = nget(b).y;
      cs(c, CF_BT, t_bot);
      cs(c, CF_NX, up != NIL ? nget_x(up) : 0u);
    }
    u32 lvb;
    const u32 lvl = level_at(cg(c, 2), nn - 1, lvb);
    return make_key(lvl, t_bot);
  }
  __device__ __forceinline__ void refresh(u32 c) { set_key(c, top_key(c)); }

  // Record a touch of positions [0, x) of chain c at step t.
  __device__ __forceinline__ void touch(u32 c, u32 x, u32 t) {
    if (x == 0) return;
    u32 tp = cfn(c, CF_STOP), reuse = NIL;
    const u32 sb = cfn(c, CF_SBOT);
    for (u32 guard = 0; guard < node_cap && tp != NIL && nget_x(tp) <= x; guard++) {
      const u32 d = nget_w(tp);
      // the last node to leave the stack becomes the new one, the others go to the free list
      if (reuse != NIL) node_free(reuse);
      reuse = tp;
      tp = d;
    }
    const u32 nw = reuse != NIL ? reuse : node_alloc();
    nset(nw, make_uint4(x, t, NIL, tp));
    if (tp != NIL) {
      nset_z(tp, nw);
      if (tp == sb) cs(c, CF_NX, x);   // the new pair sits right above the bottom
    } else {
      cs(c, CF_SBOT, nw);              // the new pair is the whole stack
      cs(c, CF_BT, t);
      cs(c, CF_NX, 0);
    }
    cs(c, CF_STOP, nw);
  }

  // Recompute chain c's claim maxima from the live-claim list; returns the new hard protection
  // (the caller applies it through chain_update).
  __device__ __forceinline__ u32 claim_maxima(u32 c) {
    post(J_MAXIMA, c, ncl);
    u32 q[8];
    maxima_slice(c, ncl, q);
    cgs(c, 2, make_uint4(q[1], q[2], q[3], q[4]));
    cs(c, CF_COVA, q[5]); cs(c, CF_COVS, q[6]); cs(c, CF_TPEND, q[7]);
    return q[0];
  }
  // This wave's share of the claim maxima of chain c over the n live claims (all waves: the
  // combined maxima in q on wave 0): hard protection, soft levels 1..4, coverage of live claims,
  // of live claims not demoted / expired, and the largest pending threshold.
  __device__ __forceinline__ void maxima_slice(u32 c, u32 ncl, u32 (&q)[8]) {
    u32 pr = 0, l1 = 0, l2 = 0, l3 = 0, l4 = 0, ca = 0, cso = 0, tp = 0;
    const bool hardm = mode == RKC_MODE_HARD, softl = soft_levels();
    // uniform chunks, every lane reading a valid entry and selecting, so that no lane mask is
    // saved and restored per condition
    for (u32 base = wave * 64u; base < ncl; base += kSpan) {
      const u32 i = base + lane, j = i < ncl ? i : base;
      const u32 m = cla(CL_META)[j], L = cla(CL_L)[j], T = cla(CL_T)[j], st = m_state(m);
      // an offloaded claim's victims are not resident and its predicate never fails
      const bool on = i < ncl && (u32)cla(CL_C)[j] == c && m_eff(m) != RKC_PROT_OFFLOADED;
      const u32 x = on ? L : 0u;
      ca = max(ca, x);
      cso = max(cso, (st == ST_OBSERVED || st == ST_MATERIALIZED || st == ST_HARMED) ? x : 0u);
      pr = max(pr, (hardm && st == ST_MATERIALIZED && m_eff(m) == RKC_PROT_HARD) ? x : 0u);
      const u32 p = m_prio(m);
      const u32 sx = (softl && ((st == ST_MATERIALIZED && m_eff(m) == RKC_PROT_SOFT) || st == ST_DEMOTED)) ? x : 0u;
      l1 = max(l1, p == 0 ? sx : 0u); l2 = max(l2, p == 1 ? sx : 0u);
      l3 = max(l3, p == 2 ? sx : 0u); l4 = max(l4, p == 3 ? sx : 0u);
      tp = max(tp, on && m_pending(m) ? T : 0u);
    }
    // (the soft levels are zero in every lane outside soft levels, the hard extent outside hard
    // protection: those reductions are skipped)
    if (hardm) pr = wave_max(pr);
    if (softl) { l1 = wave_max(l1); l2 = wave_max(l2); l3 = wave_max(l3); l4 = wave_max(l4); }
    ca = wave_max(ca); cso = wave_max(cso); tp = wave_max(tp);
    q[0] = pr; q[1] = l1; q[2] = l2; q[3] = l3; q[4] = l4; q[5] = ca; q[6] = cso; q[7] = tp;
    exchange(q, 0xFFu, 0u);
  }
  __device__ __forceinline__ void recompute(u32 c) {
    const u32 pr = claim_maxima(c);
    const uint4 g0 = cg(c, 0);
    chain_update(c, g0, g0.x, g0.y, pr);
    refresh(c);
  }

  // Recompute every chain whose mark has bit `bit`, and clear the marks.
  __device__ __forceinline__ void recompute_marked(u32 bit) {
    for (u32 base = 0; base < (u32)n_chains; base += 64) {
      const u32 c = base + lane;
      const bool m = c < (u32)n_chains && (mk[c] & bit);
      u64 b = ballot(m);
      while (b) {
        const u32 l = (u32)__builtin_ctzll(b);
        b &= b - 1;
        const u32 cc = base + l;
        recompute(cc);
        mk[cc] &= ~bit;
      }
    }
  }

  // Candidates: shared-chain tops above max(hold, prot) (and above the hits on chain hc), plus the
  // private FIFO runs.
  __device__ __forceinline__ i32 candidates(i32 hc, u32 h) {
    i32 e = Eall + fblocks;
    if (hc >= 0) {
      const uint4 g0 = cg((u32)hc, 0);
      const u32 lo = max(g0.y, g0.z);
      e -= evictable(g0.x, lo, 0) - evictable(g0.x, max(lo, h), 0);
    }
    return e;
  }

  __device__ __forceinline__ void fifo_pop_front() {
    fhead++;
    if (fhead != ftail) {
      const uint4 e = ufl4(fifo[fhead]);
      ft = e.x; flo = e.y; ftop = e.z;
    }
  }

  // ALLOC: FREE blocks first, then the (need - F) smallest-key candidates.
  __device__ __forceinline__ AllocRes alloc(i32 need, i32 hc, u32 h, u32& sweep_due) {
    AllocRes r = {1, 0, 0, 0, 0, 0};
    if (need <= F) {
      F -= need;
      return r;
    }
    const i32 E = candidates(hc, h);
    r.E = E;
    // (usable blocks are at most 2^22 and a request at most 2^24: these sums fit 32 bits)
    if (need > F + E) {
      r.ok = 0;
      return r;
    }
    i32 K = need - F;
    F = 0;
    for (u32 guard = 0; K > 0; guard++) {
      if (guard > (u32)U + 1) { status |= kFault; break; }
      // every remaining candidate of the hit chain is a hit (evictions may have reached the hits)
      const bool hc_empty = hc >= 0 && cf((u32)hc, CF_N) <= h;
      u32 k1 = KEY_INF, i1 = NIL;
      const u32 krs[4] = {kr0, kr1, kr2, kr3};
#pragma unroll
      for (u32 q = 0; q < 4; q++) {
        const u32 c = 64 * q + lane;
        const u32 k = (hc_empty && (i32)c == hc) ? KEY_INF : krs[q];
        if (k < k1) { k1 = k; i1 = c; }
      }
      for (u32 c = kRegChains + lane; c < (u32)n_chains; c += 64) {
        const u32 k = (hc_empty && (i32)c == hc) ? KEY_INF : (u32)tk[c];
        if (k < k1) { k1 = k; i1 = c; }
      }
      const u32 m1 = wave_min(k1);
      const u32 kf = (fhead != ftail) ? make_key(0, ft) : KEY_INF;
      if (kf == KEY_INF && m1 == KEY_INF) { status |= kFault; break; }
      if (kf <= m1) {
        // the FIFO front run (on a tie it lies above the tied chain's run)
        const u32 m = min((u32)K, ftop - flo);
        if (m == 0) { status |= kFault; break; }
        ftop -= m;
        fblocks -= (i32)m;
        r.victims += (i32)m;
        r.unclaimed += (i32)m;
        K -= (i32)m;
        if (ftop == flo) fifo_pop_front();
      } else {
        const u32 c = (u32)rdlane((i32)i1, (u32)__builtin_ctzll(ballot(k1 == m1)));
        const uint4 g0 = cg(c, 0), g1 = cg(c, 1);
        const u32 nn = g0.x;
        u32 lo = max(g0.y, g0.z);
        if ((i32)c == hc) lo = max(lo, h);
        u32 lvb;
        level_at(cg(c, 2), nn - 1, lvb);
        const u32 run_lo = max(lo, max(lvb, g1.x));  // positions below nx were touched later
        const u32 m = min((u32)K, nn - run_lo);
        if (m == 0 || m > nn) { status |= kFault; break; }
        const u32 nw = nn - m;
        const i32 res = max(0, (i32)min(nn, g1.y) - (i32)nw);
        const i32 strict = max(0, (i32)min(nn, g1.z) - (i32)nw);
        r.victims += (i32)m;
        r.resident += res;
        r.post += res - strict;
        r.unclaimed += (i32)m - res;
        chain_update(c, g0, nw, g0.y, g0.z);
        refresh(c);
        if (nw < g1.w) {
          mk[c] |= MK_SWEEP;
          sweep_due = 1;
        }
        K -= (i32)m;
      }
    }
    return r;
  }

  // Predicate sweep over claims on chains that shrank below a pending threshold (§3.2 harm).
  __device__ __forceinline__ u32 sweep(u32 t) {
    post(J_SWEEP, t, ncl);
    u32 q[2];
    sweep_slice(t, ncl, q);
    const u32 pf = q[0], hm = q[1];
    tadd(TW_PREDFAIL, pf);
    tadd(TW_HARM, hm);
    recompute_marked(MK_SWEEP);
    return (pf ? (u32)RKC_FL_PRED_FAIL : 0u) | (hm ? (u32)RKC_FL_HARM : 0u);
  }
  // this wave's share of the sweep (q: predicate failures, harms; combined on wave 0)
  __device__ __forceinline__ void sweep_slice(u32 t, u32 ncl, u32 (&q)[2]) {
    u32 pf = 0, hm = 0;
    for (u32 i = first(); i < ncl; i += kSpan) {
      const u32 c = cla(CL_C)[i];
      if (!(mk[c] & MK_SWEEP)) continue;
      u32 m = cla(CL_META)[i];
      const u32 st = m_state(m);
      if (!m_pending(m) || m_eff(m) == RKC_PROT_OFFLOADED) continue;
      if (ch[c * CF_WORDS + CF_N] >= cla(CL_T)[i]) continue;
      m &= ~(1u << 8);
      pf++;
      rkc_claim_telemetry* r = rec + (u32)cla(CL_SLOT)[i];
      r->w[RW_PF] = (i32)t;
      if (st == ST_MATERIALIZED) {
        m = m_with_state(m, ST_HARMED);
        hm++;
        r->w[RW_HARM] = (i32)t;
      }
      cla(CL_META)[i] = m;
    }
    lists_fence();
    q[0] = wave_sum(pf);
    q[1] = wave_sum(hm);
    exchange(q, 0u, 0u);
  }

  // Refusal record of an active event that cannot be served (§3.4; §5.4 refusal record).
  __device__ __forceinline__ void refusal(i32 need, i32 hc, u32 h, i32 Hc, i32& code, i32& id,
                                          i32& a, i32& b, u32& n16) {
    i32 Pr = PR;
    if (mode == RKC_MODE_HARD && hc >= 0) {
      const uint4 g0 = cg((u32)hc, 0);
      Pr -= max(0, (i32)min(g0.z, h) - (i32)g0.y);
    }
    const i32 req = A + Hc + need;
    if (Pr > 0 && req <= U) {
      code = RKC_OC_REFUSED_CLAIM;
      post(J_ATTRIB, (u32)hc, h, ncl);
      u32 q[2];
      attrib_slice(hc, h, ncl, q);
      id = (i32)q[0];
      n16 = min(q[1], 65535u);
    } else {
      code = RKC_OC_REFUSED_CAPACITY;
      id = -1;
      n16 = 0;
    }
    a = Pr;
    b = (i32)req;
  }

  // This wave's share of the attribution of a refusal (§5.4 blocking_claim_ids): every
  // materialized hard claim reaching a cached position outside the hits (h leading positions of
  // chain hc) counts it; q = smallest blocking id, number of blocking claims (combined on wave 0).
  __device__ __forceinline__ void attrib_slice(i32 hc, u32 h, u32 ncl, u32 (&q)[2]) {
    u32 mn = NIL, cnt = 0;
    for (u32 i = first(); i < ncl; i += kSpan) {
      const u32 m = cla(CL_META)[i];
      if (m_state(m) != ST_MATERIALIZED || m_eff(m) != RKC_PROT_HARD) continue;
      const u32 c = cla(CL_C)[i];
      u32 cov = ch[c * CF_WORDS + CF_HOLD];
      if ((i32)c == hc) cov = max(cov, h);
      if (cla(CL_L)[i] <= cov) continue;
      cla(CL_BLK)[i] += 1;
      cnt++;
      mn = min(mn, (u32)cla(CL_ID)[i]);
    }
    lists_fence();
    q[0] = wave_min(mn);
    q[1] = wave_sum(cnt);
    exchange(q, 0u, 1u);
  }

  // Claim records: a rejected claim's words 0..8 are written at birth (lane k writes word k); a
  // live claim's step words 3, 4, 6, 7 start at -1 at birth and take their step when it happens,
  // and its words 0, 1, 2, 5, 8 are written once, when it is released or at the end; word 9
  // (lead_end) is written by the final pass.
  __device__ __forceinline__ void write_record(u32 slot, i32 id, u32 packed, i32 accept, i32 dem,
                                               i32 exst, i32 rel, i32 pf, i32 harm, i32 blk) {
    if (lane < 9) {
      const i32 v = lane == 0 ? id : lane == 1 ? (i32)packed : lane == 2 ? accept : lane == 3 ? dem
                  : lane == 4 ? exst : lane == 5 ? rel : lane == 6 ? pf : lane == 7 ? harm : blk;
      rec[slot].w[lane] = v;
    }
  }
  __device__ __forceinline__ void write_birth_record(u32 slot) {
    if (lane == RW_DEM || lane == RW_EXST || lane == RW_PF || lane == RW_HARM) rec[slot].w[lane] = -1;
  }
  __device__ __forceinline__ void write_live_record(u32 i, u32 state, i32 rel) {
    const u32 id = ufl(cla(CL_ID)[i]), slot = ufl(cla(CL_SLOT)[i]);
    const u32 packed = packed_of(m_with_state(ufl(cla(CL_META)[i]), state)), blk = ufl(cla(CL_BLK)[i]);
    if (lane == 0 || lane == 1 || lane == 2 || lane == 5 || lane == 8) {
      const i32 v = lane == 0 || lane == 2 ? (i32)id : lane == 1 ? (i32)packed : lane == 5 ? rel : (i32)blk;
      rec[slot].w[lane] = v;
    }
  }
  // the step word w of live claim i's record (every lane, one value)
  __device__ __forceinline__ void record_step(u32 i, u32 w, i32 v) { rec[ufl(cla(CL_SLOT)[i])].w[w] = v; }

  // Remove entry i of a struct-of-arrays list (NARR arrays of capacity cap) by shifting the tail
  // down one place.  Each round loads KU chunks of 64 entries of every array before it stores any,
  // so KU * NARR loads are in flight together (the lists of large pools live in global scratch,
  // where one dependent round trip per chunk and array would dominate).  A round's stores land
  // below the entries its later chunks and the next rounds read, and every load a store could
  // overwrite has completed before that store issues.
  template <u32 NARR, u32 KU>
  __device__ __forceinline__ void list_remove(lword* base0, u32 cap, u32 len, u32 i) {
    for (u32 base = i; base + 1 < len; base += 64 * KU) {
      u32 v[KU][NARR];
#pragma unroll
      for (u32 u = 0; u < KU; u++) {
        const u32 j = base + 64 * u + lane;
#pragma unroll
        for (u32 k = 0; k < NARR; k++) v[u][k] = j + 1 < len ? (u32)base0[k * cap + j + 1] : 0u;
      }
      __builtin_amdgcn_wave_barrier();
#pragma unroll
      for (u32 u = 0; u < KU; u++) {
        const u32 j = base + 64 * u + lane;
        if (j + 1 < len) {
#pragma unroll
          for (u32 k = 0; k < NARR; k++) base0[k * cap + j] = (lword)v[u][k];
        }
      }
      __builtin_amdgcn_wave_barrier();
    }
    lists_fence();
  }

  // Open a gap at entry i of a struct-of-arrays list of len entries (len < cap) by shifting
  // [i, len) up one place, highest chunks first, KU chunks of every array loaded per round before
  // any store (the mirror image of list_remove).
  template <u32 NARR, u32 KU>
  __device__ __forceinline__ void list_open(lword* base0, u32 cap, u32 len, u32 i) {
    for (u32 top = len; top > i;) {
      u32 v[KU][NARR];
      u32 lo = top;
#pragma unroll
      for (u32 u = 0; u < KU; u++) {
        const u32 hi = lo;
        lo = hi > i + 64 ? hi - 64 : i;
        const u32 j = lo + lane;
#pragma unroll
        for (u32 k = 0; k < NARR; k++) v[u][k] = j < hi ? (u32)base0[k * cap + j] : 0u;
      }
      __builtin_amdgcn_wave_barrier();
      u32 lo2 = top;
#pragma unroll
      for (u32 u = 0; u < KU; u++) {
        const u32 hi = lo2;
        lo2 = hi > i + 64 ? hi - 64 : i;
        const u32 j = lo2 + lane;
        if (j < hi) {
#pragma unroll
          for (u32 k = 0; k < NARR; k++) base0[k * cap + j + 1] = (lword)v[u][k];
        }
      }
      __builtin_amdgcn_wave_barrier();
      top = lo;
    }
    lists_fence();
  }

  // Move entries [d, d + len) of every array down to [0, len), KU chunks of every array loaded per
  // round before any store (ascending rounds: a round stores below what later rounds read).
  template <u32 NARR, u32 KU>
  __device__ __forceinline__ void list_compact(lword* base0, u32 cap, u32 len, u32 d) {
    for (u32 base = 0; base < len; base += 64 * KU) {
      u32 v[KU][NARR];
#pragma unroll
      for (u32 u = 0; u < KU; u++) {
        const u32 j = base + 64 * u + lane;
#pragma unroll
        for (u32 k = 0; k < NARR; k++) v[u][k] = j < len ? (u32)base0[k * cap + j + d] : 0u;
      }
      __builtin_amdgcn_wave_barrier();
#pragma unroll
      for (u32 u = 0; u < KU; u++) {
        const u32 j = base + 64 * u + lane;
        if (j < len) {
#pragma unroll
          for (u32 k = 0; k < NARR; k++) base0[k * cap + j] = (lword)v[u][k];
        }
      }
      __builtin_amdgcn_wave_barrier();
    }
    lists_fence();
  }

  // Workgroup version of the list moves (NW > 1): entries [src, src + len) of every array move to
  // [dst, dst + len), in rounds of KU chunks of 64 entries per wave; each round loads its share,
  // passes a workgroup barrier and only then stores, and the rounds run away from the destination
  // (ascending when moving down, descending when moving up), so no store of a round lands on an
  // entry a later round still has to load.
  template <u32 NARR, u32 KU>
  __device__ __forceinline__ void move_slice(lword* base0, u32 cap, u32 src, u32 dst, u32 len) {
    constexpr u32 S = kSpan * KU;
    const bool down = dst < src;
    const u32 rounds = (len + S - 1) / S;
    for (u32 r = 0; r < rounds; r++) {
      const u32 r0 = down ? r * S : (len > (r + 1) * S ? len - (r + 1) * S : 0u);
      const u32 r1 = down ? min(len, r0 + S) : len - r * S;
      u32 v[KU][NARR];
#pragma unroll
      for (u32 u = 0; u < KU; u++) {
        const u32 j = r0 + (wave * KU + u) * 64u + lane;
#pragma unroll
        for (u32 k = 0; k < NARR; k++) v[u][k] = j < r1 ? (u32)base0[k * cap + src + j] : 0u;
      }
      __syncthreads();
#pragma unroll
      for (u32 u = 0; u < KU; u++) {
        const u32 j = r0 + (wave * KU + u) * 64u + lane;
        if (j < r1) {
#pragma unroll
          for (u32 k = 0; k < NARR; k++) base0[k * cap + dst + j] = (lword)v[u][k];
        }
      }
    }
    __syncthreads();
  }
  // list 0: the live requests (indices relative to the arrays' start), 1: the live claims
  __device__ __forceinline__ void list_move(u32 list, u32 src, u32 dst, u32 len) {
    post(J_MOVE, list, src, dst, len);
    move_any(list, src, dst, len);
  }
  __device__ __forceinline__ void move_any(u32 list, u32 src, u32 dst, u32 len) {
    if (list == 0) move_slice<RQ_ARRAYS, 4>(rq, rq_cap, src, dst, len);
    else move_slice<CL_ARRAYS, 2>(cl, cl_cap, src, dst, len);
  }

  // This wave's share of the hold rescan of chain c over the n live requests: the largest R on
  // the chain and how many requests hold it (wave 0 receives the combination).
  __device__ __forceinline__ void hold_slice(u32 c, u32 n, u32& hm, u32& hk) {
    constexpr u32 KU = kGL ? 2 : 1;
    u32 m = 0, k = 0;
    for (u32 base = wave * 64u * KU; base < n; base += kSpan * KU) {
      u32 cc[KU], rr[KU];
#pragma unroll
      for (u32 u = 0; u < KU; u++) {
        const u32 j = base + 64 * u + lane;
        cc[u] = j < n ? (u32)rqa(RQ_C)[j] : kListNil;
        rr[u] = j < n ? (u32)rqa(RQ_R)[j] : 0u;
      }
#pragma unroll
      for (u32 u = 0; u < KU; u++) {
        if (cc[u] == c && rr[u] >= m) {
          k = rr[u] > m ? 1u : k + 1u;
          m = rr[u];
        }
      }
    }
    u32 q[2];
    q[0] = wave_max(m);
    q[1] = wave_sum(m == q[0] ? k : 0u);
    hm = q[0];
    hk = q[1];
    if (NW > 1) {
      if (lane < 2) jb[JB_ARGS + 8 * wave + lane] = lane == 0 ? q[0] : q[1];
      __syncthreads();
      if (wave == 0) {
        hm = 0;
        for (u32 w = 0; w < (u32)NW; w++) hm = max(hm, ufl(jb[JB_ARGS + 8 * w]));
        hk = 0;
        for (u32 w = 0; w < (u32)NW; w++)
          hk += ufl(jb[JB_ARGS + 8 * w]) == hm ? ufl(jb[JB_ARGS + 8 * w + 1]) : 0u;
      }
    }
  }

  // Waves 1..NW-1: run the jobs wave 0 posts until it posts J_EXIT.
  __device__ __forceinline__ void serve() {
    for (;;) {
      __syncthreads();
      const u32 job = ufl(jb[0]);
      if (job == J_EXIT) break;
      if (job == J_MAXIMA) {
        u32 q[8];
        maxima_slice(arg(0), arg(1), q);
      } else if (job == J_EXPIRE) {
        u32 q[4];
        expire_slice(arg(0), arg(1), q);
      } else if (job == J_SWEEP) {
        u32 q[2];
        sweep_slice(arg(0), arg(1), q);
      } else if (job == J_ATTRIB) {
        u32 q[2];
        attrib_slice((i32)arg(0), arg(1), arg(2), q);
      } else if (job == J_HOLD) {
        rq_head = arg(2);
        u32 hm, hk;
        hold_slice(arg(0), arg(1), hm, hk);
      } else {
        move_any(arg(0), arg(1), arg(2), arg(3));
      }
    }
  }

  __device__ __forceinline__ void expire(u32 t, u32& flags, u32& expired) {
    post(J_EXPIRE, t, ncl);
    u32 q[4];
    expire_slice(t, ncl, q);
    const u32 cnt = q[0], pf = q[3];
    t2used -= q[2];
    if (pf) {
      flags |= RKC_FL_PRED_FAIL;
      tadd(TW_PREDFAIL, pf);
    }
    next_exp = q[1];
    if (cnt) {
      recompute_marked(MK_RECOMP);
      flags |= RKC_FL_EXPIRED;
      tadd(TW_EXPIRED, cnt);
    }
    expired = cnt;
  }
  // This wave's share of the expiry at the start of step t (q: claims expired, next expiry step,
  // second-tier blocks dropped, predicate failures; combined on wave 0).
  __device__ __forceinline__ void expire_slice(u32 t, u32 ncl, u32 (&q)[4]) {
    u32 cnt = 0, nx = EXP_NEVER, drop = 0, pf = 0;
    for (u32 i = first(); i < ncl; i += kSpan) {
      const u32 m = cla(CL_META)[i], st = m_state(m), dur = cla(CL_EXP)[i];
      if ((st != ST_MATERIALIZED && st != ST_DEMOTED) || dur == 0) continue;
      const u32 ex = (u32)cla(CL_ID)[i] + dur;
      if (ex <= t) {
        // responsibility ends: an offloaded claim's second-tier copy is dropped
        const bool off = m_eff(m) == RKC_PROT_OFFLOADED;
        u32 m2 = m;
        if (off) {
          drop += cla(CL_L)[i];
          m2 = m_with_eff(m2, RKC_PROT_NONE);
          // its predicate held only through the dropped copy: a chain already shorter than T
          // fails it now (no harm: the claim is expired)
          if (m_pending(m) && (u32)ch[(u32)cla(CL_C)[i] * CF_WORDS + CF_N] < (u32)cla(CL_T)[i]) {
            m2 &= ~(1u << 8);
            rec[(u32)cla(CL_SLOT)[i]].w[RW_PF] = (i32)t;
            pf++;
          }
        }
        cla(CL_META)[i] = m_with_state(m2, ST_EXPIRED);
        rec[(u32)cla(CL_SLOT)[i]].w[RW_EXST] = (i32)t;
        mark_or(cla(CL_C)[i], MK_RECOMP);
        cnt++;
      } else {
        nx = min(nx, ex);
      }
    }
    lists_fence();
    q[0] = wave_sum(cnt);
    q[1] = wave_min(nx);
    q[2] = wave_sum(drop);
    q[3] = wave_sum(pf);
    __builtin_amdgcn_wave_barrier();
    exchange(q, 0u, 2u);
  }

  __device__ __forceinline__ void count_victims(const AllocRes& r, u32 hits) {
    tv += lane == TW_VICTIMS ? (u32)r.victims : lane == TW_RESIDENT ? (u32)r.resident
        : lane == TW_POST ? (u32)r.post : lane == TW_HITS ? hits : 0u;
  }

  // Largest footprint of the materialized hard claims on chain c (tentative picks of the
  // relaxation have left that state already).
  __device__ __forceinline__ u32 hard_extent(u32 c) {
    u32 pr = 0;
    for (u32 i = lane; i < ncl; i += 64) {
      const u32 m = cla(CL_META)[i];
      if ((u32)cla(CL_C)[i] == c && m_state(m) == ST_MATERIALIZED && m_eff(m) == RKC_PROT_HARD)
        pr = max(pr, (u32)cla(CL_L)[i]);
    }
    return wave_max(pr);
  }

  // Runtime relaxation (§3.1 demotable: the downgrade comes before the predicate-breaking
  // eviction; offloadable: the content may leave GPU memory if the predicate stays restorable; §3.5
  // "relax resident claim" and "offload resident").  Before an active allocation of `need` blocks
  // that hard protection makes infeasible, the blocking claims (materialized hard claims reaching a
  // cached position outside the hits) that allow demotion or offload are visited lowest priority
  // first, then lowest id: each is offloaded when it allows it and its footprint fits the second
  // tier's free room, else demoted when it allows it, else left alone, until the allocation would
  // fit.  The picks change the claims tentatively (offload: effective protection OFFLOADED; demote:
  // state DEMOTED), marked by the demotion step t in the claim's record, which no other claim can
  // carry at t; they are kept when the allocation fits and undone otherwise.  Returns the number of claims relaxed.
  __device__ __forceinline__ u32 relax(u32 t, i32 need, i32 hc, u32 h) {
    u32 k = 0;
    if (relax_on && need > F) {
      i32 avail = F + candidates(hc, h);
      if (need > avail) {
        u32 room = t2cap > t2used ? t2cap - t2used : 0u, moved = 0, no = 0, lo = 0;
        for (u32 guard = 0; need > avail && guard <= ncl; guard++) {
          u32 best = 0xFFFFFFFFu, bi = 0;
          for (u32 i = lane; i < ncl; i += 64) {
            const u32 m = cla(CL_META)[i];
            if (m_state(m) != ST_MATERIALIZED || m_eff(m) != RKC_PROT_HARD || !(m & (M_DEMQ | M_OFFQ))) continue;
            const u32 c = cla(CL_C)[i];
            u32 cov = (u32)ch[c * CF_WORDS + CF_HOLD];
            if ((i32)c == hc) cov = max(cov, h);
            if ((u32)cla(CL_L)[i] <= cov) continue;  // not blocking: no cached position outside the hits
            const u32 key = (m_prio(m) << 24) | (u32)cla(CL_ID)[i];
            if (key >= lo && key < best) { best = key; bi = i; }
          }
          const u32 wb = wave_min(best);
          if (wb == 0xFFFFFFFFu) break;
          lo = wb + 1;  // visited: a claim left alone is not visited again
          const u64 at = ballot(best == wb);
          const u32 i = (u32)rdlane((i32)bi, (u32)__builtin_ctzll(at));
          const u32 m = ufl(cla(CL_META)[i]), L = ufl(cla(CL_L)[i]);
          const bool off = (m & M_OFFQ) && L <= room;
          if (!off && !(m & M_DEMQ)) continue;
          const u32 c = ufl(cla(CL_C)[i]);
          const u32 before = hard_extent(c);
          // every lane, one value
          cla(CL_META)[i] = off ? m_with_eff(m, RKC_PROT_OFFLOADED) : m_with_state(m, ST_DEMOTED);
          record_step(i, RW_DEM, (i32)t);
          lists_fence();
          const u32 after = hard_extent(c);
          const uint4 g0 = cg(c, 0);
          const u32 base = (i32)c == hc ? max(g0.y, h) : g0.y;
          avail += evictable(g0.x, base, after) - evictable(g0.x, base, before);
          if (off) { room -= L; moved += L; no++; }
          k++;
        }
        const bool fits = need <= avail;
        if (k) {
          __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "workgroup");  // the marks reach the scan
          for (u32 i = lane; i < ncl; i += 64) {
            i32* dem = &rec[(u32)cla(CL_SLOT)[i]].w[RW_DEM];
            if (*dem != (i32)t) continue;
            const u32 m = cla(CL_META)[i];
            const bool off = m_eff(m) == RKC_PROT_OFFLOADED;
            if (fits) {
              cla(CL_META)[i] = m | M_RELAXED;
              if (off) *dem = -1;  // an offloaded claim records no demotion
              mk[cla(CL_C)[i]] |= MK_RECOMP;
            } else {
              cla(CL_META)[i] = off ? m_with_eff(m, RKC_PROT_HARD) : m_with_state(m, ST_MATERIALIZED);
              *dem = -1;
            }
          }
          lists_fence();
        }
        if (fits) {
          __builtin_amdgcn_wave_barrier();
          recompute_marked(MK_RECOMP);
          tadd(TW_RUNTIME_DEMOTED, k - no);
          if (no) {
            t2used += moved;
            t2peak = max(t2peak, t2used);
            tadd(TW_OFF_CLAIMS, no);
            tadd(TW_OFF_BLOCKS, moved);
          }
        } else {
          k = 0;
        }
      }
    }
    return k;
  }

  // One event.  Returns the outcome words.
  //
  // Control flow is kept to two switches over a small integer: uniform conditions held in u32
  // words (not bools) compile to scalar compares and branches instead of lane-mask selects.
  enum : u32 { K_NOOP = 0, K_INVALID, K_PREFILL, K_EXTEND, K_CLAIM, K_FINISH, K_RELEASE, K_DEMOTE,
              K_REFUSED };
  __device__ __forceinline__ int4 step(u32 t, u32 uw0, i32 w1, i32 w2, i32 w3) {
    const u32 type = uw0 & 15u, hardq = (uw0 >> 4) & 1u, prio = (uw0 >> 5) & 3u, dur = uw0 >> 16;
    u32 flags = 0, expired = 0, n16 = NIL, sweep_due = 0;
    i32 code = RKC_OC_NOOP, id = -1, a = 0, b = 0;

    if (t >= next_exp) expire(t, flags, expired);

    // Decode: validity (malformed events and table limits) and the allocation request.  A RETRY
    // turns into the prefill of the oldest deferred request (id rid, its own S, chain and P).
    u32 kind = K_NOOP, sel = 0, h = 0, s = 0, rid = t, retry = 0;
    i32 need = 0, hc = -1, Hc = 0;
    const u32 fieldbad = (u32)(w1 < 1) | (u32)(w1 > RKC_MAX_FIELD_BLOCKS);
    const u32 chainbad = (u32)(w2 < 0) | (u32)(w2 >= n_chains);
    const u32 thrbad = (u32)(w3 < 0) | (u32)(w3 > w1);
    switch (type) {
      case RKC_EV_PREFILL:
        if (fieldbad | thrbad | ((u32)(w3 > 0) & chainbad)) {
          kind = K_INVALID;
        } else if (nreq >= (u32)max_reqs) {
          kind = K_INVALID;
          status |= RKC_PS_REQUEST_TABLE;
        } else {
          kind = K_PREFILL;
        }
        break;
      case RKC_EV_RETRY:
        if (dq_len == 0) {
          kind = K_NOOP;
        } else if (nreq >= (u32)max_reqs) {
          kind = K_INVALID;  // the request stays queued
          status |= RKC_PS_REQUEST_TABLE;
        } else {
          const uint4 q = dq[dq_head];
          rid = ufl(q.x); w1 = (i32)ufl(q.y); w2 = (i32)ufl(q.z); w3 = (i32)ufl(q.w);
          retry = 1;
          kind = K_PREFILL;
        }
        break;
      case RKC_EV_EXTEND:
        if (fieldbad) {
          kind = K_INVALID;
        } else if (nreq > 0) {
          kind = K_EXTEND;
          sel = (u32)w2 % nreq;
          need = w1;
        }
        break;
      case RKC_EV_CLAIM:
        if (nslot >= (u32)n_slots) {
          kind = K_INVALID;
          status |= RKC_PS_SLOT_TABLE;
        } else {
          s = nslot++;
          u32 ok = 0;
          if (fieldbad | chainbad | thrbad) {
          } else if (ncl >= (u32)max_claims) {
            status |= RKC_PS_CLAIM_TABLE;
          } else {
            ok = 1;
          }
          // (chain, L) of a valid claim for its final lead_end; invalid claims report 0
          slot_cl[s] = ok ? make_uint2((u32)w2, (u32)w1) : make_uint2(NIL, 0);
          if (ok) {
            kind = K_CLAIM;
            hc = w2;
            h = min((u32)w1, cf((u32)w2, CF_N));
            need = w1 - (i32)h;
          } else {
            kind = K_INVALID;
            write_record(s, (i32)t, 0, -1, -1, -1, -1, -1, -1, 0);
          }
        }
        break;
      case RKC_EV_FINISH: kind = nreq > 0 ? K_FINISH : K_NOOP; break;
      case RKC_EV_RELEASE: kind = ncl > 0 ? K_RELEASE : K_NOOP; break;
      case RKC_EV_DEMOTE: kind = K_DEMOTE; break;
      case RKC_EV_NOP: break;
      default: kind = K_INVALID; break;
    }
    if (kind == K_PREFILL) {
      if (w3 > 0) {
        hc = w2;
        const uint4 g0 = cg((u32)hc, 0);
        h = min((u32)w3, g0.x);
        Hc = max(0, (i32)h - (i32)g0.y);
      }
      need = w1 - (i32)h;
    }

    // One allocation site for prefill, extend and claim; active requests may first relax claims.
    u32 relaxed = 0;
    if (mode == RKC_MODE_HARD && (kind == K_PREFILL || kind == K_EXTEND)) relaxed = relax(t, need, hc, h);
    AllocRes r = {1, 0, 0, 0, 0, 0};
    if (kind == K_PREFILL || kind == K_EXTEND || kind == K_CLAIM) r = alloc(need, hc, h, sweep_due);
    if (!r.ok && kind != K_CLAIM) {
      refusal(need, hc, h, Hc, code, id, a, b, n16);
      // active deferral: a prefill refused on behalf of claims waits in the queue; a retried one
      // is deferred again while its deferrals last, else refused for good
      const u32 by_claim = (u32)(code == RKC_OC_REFUSED_CLAIM);
      if (kind == K_PREFILL && retry) {
        if (by_claim && dq_cnt < (u32)defer_limit) {
          dq_cnt++;
          code = RKC_OC_DEFERRED;
        } else {
          dq_head = dq_head + 1 == (u32)max_reqs ? 0u : dq_head + 1;
          dq_len--;
          dq_cnt = 1;
          tadd(TW_RETRY_REFUSED, 1);
        }
      } else if (kind == K_PREFILL && by_claim && defer_limit > 0 && dq_len < (u32)max_reqs) {
        u32 slot = dq_head + dq_len;
        slot = slot >= (u32)max_reqs ? slot - (u32)max_reqs : slot;
        dq[slot] = make_uint4(t, (u32)w1, (u32)w2, (u32)w3);  // every lane, one value
        dq_len++;
        code = RKC_OC_DEFERRED;
      }
      kind = K_REFUSED;  // no further effect
    }

    // Effects; the chain the event touches gets its new (n, hold, prot), its touch of [0, tx)
    // and its new top key once, after the switch.
    u32 tc = NIL, tn = 0, th = 0, tpr = 0, tx = 0;
    switch (kind) {
      case K_INVALID:
        code = RKC_OC_INVALID;
        break;
      case K_PREFILL: {
        A += Hc + need;
        u32 R = 0;
        if (hc >= 0) {
          const uint4 g0 = cg((u32)hc, 0);  // victims may have shortened this chain above the hits
          R = mode == RKC_MODE_NOADMIT ? h : (u32)w3;
          tc = (u32)hc;
          tn = (mode != RKC_MODE_NOADMIT && (u32)w3 > g0.x) ? (u32)w3 : g0.x;
          th = max(g0.y, R);
          tpr = g0.z;
          tx = R;
          // the chain's hold is the largest R of its live requests; CF_HCNT counts the requests
          // holding exactly that much, so a finish rarely has to look for the next largest
          if (R > 0 && R >= g0.y) cs((u32)hc, CF_HCNT, R > g0.y ? 1u : cf((u32)hc, CF_HCNT) + 1u);
        }
        // the live list stays in id order: a retried request goes before the later ids
        if (kGL && rq_head + nreq >= rq_cap) {
          // no room above the list: move it back to the start of its arrays
          if (NW > 1) list_move(0, rq_head, 0, nreq);
          else list_compact<RQ_ARRAYS, 8>(rq, rq_cap, nreq, rq_head);
          rq_head = 0;
        }
        u32 k = nreq;
        if (retry) {
          u32 below = 0;
          for (u32 j = lane; j < nreq; j += 64) below += (u32)((u32)rqa(RQ_ID)[j] < rid);
          k = wave_sum(below);
          if (NW > 1) list_move(0, rq_head + k, rq_head + k + 1, nreq - k);
          else list_open<RQ_ARRAYS, kGL ? 8 : 1>(rqa(0), rq_cap, nreq, k);
          dq_head = dq_head + 1 == (u32)max_reqs ? 0u : dq_head + 1;
          dq_len--;
          dq_cnt = 1;
          tadd(TW_RETRY_SERVED, 1);
        }
        nreq++;
        rqa(RQ_ID)[k] = rid; rqa(RQ_C)[k] = hc >= 0 ? (u32)hc : kListNil; rqa(RQ_R)[k] = R;
        rqa(RQ_LEN)[k] = (u32)w1;
        lists_fence();
        id = (i32)rid; b = (i32)h;
        count_victims(r, h);
        if (hc >= 0 && (u32)w3 > h && t2cap > 0) {
          // positions past the hits that a claim holding a second-tier copy covers are restored
          // from the second tier (restore cost), still on new GPU blocks
          u32 e = 0;
          for (u32 i = lane; i < ncl; i += 64)
            if ((u32)cla(CL_C)[i] == (u32)hc && m_eff(cla(CL_META)[i]) == RKC_PROT_OFFLOADED) e = max(e, (u32)cla(CL_L)[i]);
          const u32 top = min((u32)w3, wave_max(e));
          if (top > h) tadd(TW_RESTORED, top - h);
        }
        break;
      }
      case K_EXTEND:
        A += need;
        rqa(RQ_LEN)[sel] = ufl(rqa(RQ_LEN)[sel]) + (u32)need;
        id = (i32)ufl(rqa(RQ_ID)[sel]); b = A;
        count_victims(r, 0);
        break;
      case K_CLAIM: {
        const i32 L = w1, T = w3;
        const u32 c = (u32)w2;
        // a best-effort claim is observed in every policy (§3.1 best_effort: telemetry only)
        const u32 demq = (uw0 >> 7) & 1u, beq = (uw0 >> 8) & 1u;
        const u32 eff = beq ? RKC_PROT_NONE : mode == RKC_MODE_HARD ? (hardq ? RKC_PROT_HARD : RKC_PROT_SOFT)
                      : mode == RKC_MODE_SOFT ? RKC_PROT_SOFT : RKC_PROT_NONE;
        const u32 shadow = (u32)(mode == RKC_MODE_LRU) | (u32)(mode == RKC_MODE_NOADMIT) | beq;
        const u32 req_bits = (demq ? M_DEMQ : 0u) | (beq ? M_BE : 0u) | ((uw0 >> 9) & 1u ? M_OFFQ : 0u);
        u32 dec;
        if (!r.ok) {
          dec = shadow ? DEC_SHADOW : DEC_REJECTED;
          const u32 m = ST_REJECTED | (eff << 3) | (hardq << 5) | (prio << 6) | (dec << 9) | req_bits;
          write_record(s, (i32)t, packed_of(m), -1, -1, -1, -1, -1, -1, 0);
          code = RKC_OC_MATFAIL; id = (i32)t; a = need; b = F + r.E;
        } else {
          const u32 lowered = (u32)(mode == RKC_MODE_SOFT) & hardq;
          dec = shadow ? DEC_SHADOW : lowered ? DEC_APPROX : DEC_ACCEPTED;
          const u32 st = shadow ? ST_OBSERVED : ST_MATERIALIZED;
          flags |= shadow ? (u32)RKC_FL_SHADOW : lowered ? (u32)RKC_FL_LOWERED : 0u;
          const u32 m = st | (eff << 3) | (hardq << 5) | (prio << 6) | (1u << 8) | (dec << 9) | req_bits;
          const u32 k = ncl++;
          // only a materialized claim with a duration expires (shadow claims never do)
          const u32 dur_eff = shadow ? 0u : dur;
          cla(CL_ID)[k] = t; cla(CL_C)[k] = c; cla(CL_L)[k] = (u32)L; cla(CL_T)[k] = (u32)T;
          cla(CL_META)[k] = m; cla(CL_EXP)[k] = dur_eff; cla(CL_SLOT)[k] = s; cla(CL_BLK)[k] = 0;
          write_birth_record(s);
          // a new live claim only raises the chain's maxima
          const uint4 g1 = cg(c, 1);
          cgs(c, 1, make_uint4(g1.x, max(g1.y, (u32)L), max(g1.z, (u32)L), max(g1.w, (u32)T)));
          if (soft_levels() && !shadow && eff == RKC_PROT_SOFT)
            cs(c, CF_LV + prio, max(cf(c, CF_LV + prio), (u32)L));
          if (dur_eff > 0) next_exp = min(next_exp, t + dur_eff);
          const uint4 g0 = cg(c, 0);
          tc = c;
          tn = max(g0.x, (u32)L);
          th = g0.y;
          // a materialized hard claim in a hard-protection pool protects [0, L)
          tpr = eff == RKC_PROT_HARD ? max(g0.z, (u32)L) : g0.z;
          tx = (u32)L;
          id = (i32)t; b = need;
          count_victims(r, 0);
        }
        tadd(TW_ACCEPTED + dec - DEC_ACCEPTED, 1);
        break;
      }
      case K_FINISH: {
        const u32 i = (u32)w1 % nreq;
        const u32 rid = ufl(rqa(RQ_ID)[i]), c = lnil(ufl(rqa(RQ_C)[i])), R = ufl(rqa(RQ_R)[i]);
        const u32 len = ufl(rqa(RQ_LEN)[i]);
        if (kGL && 2 * i + 1 < nreq) {
          // fewer entries below the gap than above it: move those up one place
          if (NW > 1) list_move(0, rq_head, rq_head + 1, i);
          else list_open<RQ_ARRAYS, 8>(rqa(0), rq_cap, i, 0);
          rq_head++;
        } else if (NW > 1) {
          list_move(0, rq_head + i + 1, rq_head + i, nreq - i - 1);
        } else {
          list_remove<RQ_ARRAYS, kGL ? 8 : 1>(rqa(0), rq_cap, nreq, i);
        }
        nreq--;
        i32 turned = 0;
        if (c != NIL) {
          // the new hold of the chain is the largest R of the requests still on it: unchanged
          // unless this request was the only one holding the current hold
          const uint4 g0 = cg(c, 0);
          u32 hn = g0.y;
          if (R > 0 && R == g0.y) {
            const u32 hk = cf(c, CF_HCNT);
            if (hk > 1) {
              cs(c, CF_HCNT, hk - 1);
            } else {
              // scan the live list for the largest R on the chain and how many requests hold it
              if (NW > 1) {
                post(J_HOLD, c, nreq, rq_head);
                u32 hk2;
                hold_slice(c, nreq, hn, hk2);
                cs(c, CF_HCNT, hk2);
              } else {
                // (in global scratch: 8 chunks per round, their loads in flight together)
                constexpr u32 KU = kGL ? 8 : 1;
                u32 m = 0, k = 0;
                for (u32 base = 0; base < nreq; base += 64 * KU) {
                  u32 cc[KU], rr[KU];
#pragma unroll
                  for (u32 u = 0; u < KU; u++) {
                    const u32 j = base + 64 * u + lane;
                    cc[u] = j < nreq ? (u32)rqa(RQ_C)[j] : kListNil;
                    rr[u] = j < nreq ? (u32)rqa(RQ_R)[j] : 0u;
                  }
#pragma unroll
                  for (u32 u = 0; u < KU; u++) {
                    if (cc[u] == c && rr[u] >= m) {
                      k = rr[u] > m ? 1u : k + 1u;
                      m = rr[u];
                    }
                  }
                }
                hn = wave_max(m);
                cs(c, CF_HCNT, wave_sum(m == hn ? k : 0u));
              }
            }
          }
          turned += max(0, (i32)R - (i32)hn);
          tc = c; tn = g0.x; th = hn; tpr = g0.z; tx = R;
        }
        // write no-admit drops the request's own blocks; otherwise they become a private run
        const i32 own = (i32)(len - R);
        const i32 dropped = mode == RKC_MODE_NOADMIT ? own : 0;
        const i32 kept = own - dropped;
        turned += kept;
        F += dropped;
        fblocks += kept;
        if (kept > 0) {
          if (fhead == ftail) { ft = t; flo = R; ftop = len; }
          fifo[ftail] = make_uint4(t, R, len, 0);
          ftail++;
        }
        A -= turned + dropped;
        code = RKC_OC_FINISHED; id = (i32)rid; a = turned; b = dropped;
        if (dropped) flags |= RKC_FL_NOADMIT_DROP;
        tadd(TW_DROPPED, (u32)dropped);
        break;
      }
      case K_RELEASE:
      case K_DEMOTE: {
        // the selected live claim: release removes it, demotion turns hard into soft (§3.1)
        u32 i = NIL;
        if (kind == K_RELEASE) {
          i = (u32)w1 % ncl;
        } else if (soft_levels()) {
          u32 cnt = 0;
          for (u32 base = 0; base < ncl; base += 64) {
            const u32 j = base + lane;
            const u32 m = j < ncl ? (u32)cla(CL_META)[j] : 0u;
            const bool cand = j < ncl && m_state(m) == ST_MATERIALIZED && m_hard(m) && m_eff(m) != RKC_PROT_OFFLOADED;
            cnt += (u32)__builtin_popcountll(ballot(cand));
          }
          if (cnt > 0) {
            u32 k = (u32)w1 % cnt;
            for (u32 base = 0; base < ncl && i == NIL; base += 64) {
              const u32 j = base + lane;
              const u32 m = j < ncl ? (u32)cla(CL_META)[j] : 0u;
              const bool cand = j < ncl && m_state(m) == ST_MATERIALIZED && m_hard(m) && m_eff(m) != RKC_PROT_OFFLOADED;
              const u64 bl = ballot(cand);
              const u32 pc = (u32)__builtin_popcountll(bl);
              if (k < pc) {
                u64 x = bl;
                for (u32 q = 0; q < k; q++) x &= x - 1;
                i = base + (u32)__builtin_ctzll(x);
              } else {
                k -= pc;
              }
            }
          }
        }
        if (i != NIL) {
          const u32 qid = ufl(cla(CL_ID)[i]), c = ufl(cla(CL_C)[i]), L = ufl(cla(CL_L)[i]);
          const u32 T = ufl(cla(CL_T)[i]);
          if (kind == K_RELEASE) {
            write_live_record(i, ST_RELEASED, (i32)t);
            if (m_eff(ufl(cla(CL_META)[i])) == RKC_PROT_OFFLOADED) t2used -= L;  // the copy is dropped
            __builtin_amdgcn_wave_barrier();
            if (NW > 1) list_move(1, i + 1, i, ncl - i - 1);
            else list_remove<CL_ARRAYS, kGL ? 4 : 1>(cl, cl_cap, ncl, i);
            ncl--;
            code = RKC_OC_RELEASED;
            tadd(TW_RELEASED, 1);
          } else {
            cla(CL_META)[i] = m_with_state(ufl(cla(CL_META)[i]), ST_DEMOTED);
            record_step(i, RW_DEM, (i32)t);
            __builtin_amdgcn_wave_barrier();
            code = RKC_OC_DEMOTED;
            tadd(TW_DEMOTED, 1);
          }
          const u32 pr = claim_maxima(c);
          const uint4 g0 = cg(c, 0);
          tc = c; tn = g0.x; th = g0.y; tpr = pr; tx = 0;
          id = (i32)qid; a = (i32)min(g0.x, L); b = (i32)T;
        }
        break;
      }
      default:
        break;
    }
    if (kind == K_PREFILL || kind == K_EXTEND || (kind == K_CLAIM && r.ok)) {
      code = relaxed ? RKC_OC_RELAXED : r.resident > 0 ? RKC_OC_EVICT_RESIDENT : RKC_OC_ADMIT;
      if (relaxed) n16 = min(relaxed, 65535u);
      a = r.resident;
      flags |= (r.post ? (u32)RKC_FL_POST_RELEASE_LOSS : 0u) | (r.unclaimed ? (u32)RKC_FL_EVICT_UNCLAIMED : 0u);
    }

    if (tc != NIL) {
      const uint4 g0 = cg(tc, 0);
      chain_update(tc, g0, tn, th, tpr);
      if (tx) touch(tc, tx, t);
      refresh(tc);
    }

    if (sweep_due) {
      __builtin_amdgcn_wave_barrier();
      flags |= sweep(t);
    }
    const u32 quiet = (u32)(code == RKC_OC_NOOP) | (u32)(code == RKC_OC_INVALID);
    id = quiet ? -1 : id;
    a = quiet ? 0 : a;
    b = quiet ? 0 : b;
    n16 = n16 == NIL ? min(expired, 65535u) : n16;
    tadd(code == RKC_OC_DEFERRED ? (u32)TW_DEFERRED : code == RKC_OC_RELAXED ? (u32)TW_RELAXED : (u32)code, 1);
    peak = max(peak, A);
    return make_int4((i32)((u32)code | (flags << 8) | (n16 << 16)), id, a, b);
  }
};

template <typename W, bool kGL, int NW>
__global__ __launch_bounds__(64 * NW) void rkc_replay_wave(Args g) {
  extern __shared__ __align__(16) unsigned char lds_raw[];
  const u32 pool = blockIdx.x;
  if ((i32)pool >= g.n_pools) return;
  const Layout& L = g.L;
  Pool<W, kGL, NW> P;
  P.lane = lane_id();
  P.wave = NW > 1 ? (u32)__builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6)) : 0u;
  const rkc_pool_desc d = g.pools[pool];
  P.U = d.usable_blocks; P.mode = d.mode & ~RKC_MODE_RELAX; P.n_events = d.n_events; P.n_chains = d.n_chains;
  P.relax_on = (d.mode & RKC_MODE_RELAX) != 0;
  P.t2cap = (u32)d.offload_blocks; P.t2used = 0; P.t2peak = 0;
  P.max_claims = d.max_live_claims; P.max_reqs = d.max_live_requests; P.n_slots = d.n_claim_slots;
  const i64 ev_off = d.event_offset, slot_off = d.claim_slot_offset;
  rkc_pool_telemetry* ptel = g.pool_tel + pool;

  // Descriptor checks against the batch limits the launch was sized for.
  const bool ev_ok = P.n_events >= 0 && ev_off >= 0 && ev_off + P.n_events <= g.n_events_total;
  const bool sl_ok = P.n_slots >= 0 && slot_off >= 0 && slot_off + P.n_slots <= g.n_slots_total;
  const bool ok = ev_ok && sl_ok && P.U >= 1 && P.U <= g.max_usable && P.U <= RKC_MAX_USABLE_BLOCKS &&
                  P.mode >= 0 && P.mode <= 3 && P.n_events <= g.max_events && P.n_chains >= 0 &&
                  P.n_chains <= g.max_chains && P.max_claims >= 0 && P.max_claims <= g.max_claims &&
                  P.max_reqs >= 0 && P.max_reqs <= g.max_reqs && P.n_slots <= g.max_slots &&
                  d.defer_limit >= 0 && d.offload_blocks >= 0 && d.reserved[0] == 0 &&
                  d.reserved[1] == 0 && d.reserved[2] == 0;
  if (!ok) {
    // (every wave of the workgroup returns here; wave 0 writes)
    if (P.wave == 0) {
      if (ev_ok)
        for (i32 i = (i32)P.lane; i < P.n_events; i += 64)
          g.outcomes[ev_off + i] = rkc_outcome{{RKC_OC_INVALID, -1, 0, 0}};
      if (sl_ok)
        for (i32 i = (i32)P.lane; i < P.n_slots; i += 64)
          g.claim_tel[slot_off + i] = rkc_claim_telemetry{{-1, 0, -1, -1, -1, -1, -1, -1, 0, 0}};
      ptel->w[P.lane] = P.lane == 31 ? RKC_PS_DESCRIPTOR : (P.lane == RKC_OC_INVALID && ev_ok) ? P.n_events : 0;
    }
    return;
  }

  // memory carve-up
  typedef typename Pool<W, kGL, NW>::lword lword;
  typedef typename Pool<W, kGL, NW>::lds_w lds_w;
  typedef typename Pool<W, kGL, NW>::lds_w4 lds_w4;
  lds_u32* lds = (lds_u32*)lds_raw;
  P.ch = (lds_w*)(lds + L.off_chain / 4);
  P.mk = lds + L.off_mark / 4;
  P.tk = lds + L.off_key / 4;
  P.jb = lds + L.off_job / 4;
  unsigned char* scr = g.scratch + (u64)pool * L.scr_pool_bytes;
  if (kGL) {
    P.rq = (lword*)(scr + L.scr_off_rq);
    P.cl = (lword*)(scr + L.scr_off_cl);
  } else {
    P.rq = (lword*)(lds + L.off_rq / 4);
    P.cl = (lword*)(lds + L.off_cl / 4);
  }
  P.rq_cap = L.global_lists ? 2 * L.reqs : L.reqs;
  P.rq_head = 0;
  P.cl_cap = L.claims;
  P.node_lds = (lds_w4*)(lds + L.off_node / 4);
  P.node_glb = (glb_uint4*)(scr + L.scr_off_node);
  P.nl = L.nodes_lds;
  P.node_cap = L.node_cap;
  P.fifo = (uint4*)(scr + L.scr_off_fifo);
  P.slot_cl = (uint2*)(scr + L.scr_off_slot);
  P.dq = (uint4*)(scr + L.scr_off_dq);
  P.defer_limit = d.defer_limit;
  P.rec = g.claim_tel + slot_off;

  for (i32 c = (i32)P.first(); c < P.n_chains; c += (i32)P.kSpan) {
    P.cgs((u32)c, 0, make_uint4(0, 0, 0, 0));
    P.cgs((u32)c, 1, make_uint4(0, 0, 0, 0));
    P.cgs((u32)c, 2, make_uint4(0, 0, 0, 0));
    P.cgs((u32)c, 3, make_uint4(NIL, NIL, 0, 0));
    P.mk[c] = 0;
    if ((u32)c >= kRegChains) P.tk[c] = KEY_INF;
  }
  P.kr0 = P.kr1 = P.kr2 = P.kr3 = KEY_INF;
  P.tv = 0;
  P.F = P.U; P.A = 0; P.PR = 0; P.peak = 0; P.Eall = 0;
  P.nreq = 0; P.ncl = 0; P.nslot = 0; P.next_exp = EXP_NEVER;
  P.free_head = NIL; P.bump = 0;
  P.fhead = 0; P.ftail = 0; P.ft = 0; P.flo = 0; P.ftop = 0; P.fblocks = 0;
  P.status = 0;
  P.dq_head = 0; P.dq_len = 0; P.dq_cnt = 1;
  __syncthreads();
  if (NW > 1 && P.wave != 0) {
    P.serve();
    return;
  }

  const rkc_event* ev = g.events + ev_off;
  rkc_outcome* out = g.outcomes + ev_off;
  for (i32 base = 0; base < P.n_events; base += 64) {
    const i32 cnt = min(64, P.n_events - base);
    int4 e = make_int4(0, 0, 0, 0);
    if ((i32)P.lane < cnt) {
      const rkc_event x = ev[base + P.lane];
      e = make_int4(x.w[0], x.w[1], x.w[2], x.w[3]);
    }
    int4 mine = make_int4(0, 0, 0, 0);
    for (i32 k = 0; k < cnt; k++) {
      const int4 o = P.step((u32)(base + k), (u32)rdlane(e.x, (u32)k), rdlane(e.y, (u32)k),
                            rdlane(e.z, (u32)k), rdlane(e.w, (u32)k));
      if ((i32)P.lane == k) mine = o;
    }
    if ((i32)P.lane < cnt) out[base + P.lane] = rkc_outcome{{mine.x, mine.y, mine.z, mine.w}};
  }
  P.post(J_EXIT);  // the other waves leave

  // Final claim records of the claims still live ...
  for (u32 i = 0; i < P.ncl; i++) P.write_live_record(i, m_state(ufl((u32)P.cla(CL_META)[i])), -1);
  // ... then lead_end = min(final leading registered length, L) for every used slot, and blank
  // records for unused slots.
  __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "workgroup");
  for (i32 s = (i32)P.lane; s < P.n_slots; s += 64) {
    if (s < (i32)P.nslot) {
      const uint2 cl2 = P.slot_cl[s];
      P.rec[s].w[9] = cl2.x == NIL ? 0 : (i32)min((u32)P.ch[cl2.x * CF_WORDS + CF_N], cl2.y);
    } else {
      P.rec[s] = rkc_claim_telemetry{{-1, 0, -1, -1, -1, -1, -1, -1, 0, 0}};
    }
  }
  __builtin_amdgcn_wave_barrier();
  {
    const u32 w = P.lane;
    i32 v = (i32)P.tv;
    if (w == 24) v = P.peak;
    else if (w == 25) v = P.A;
    else if (w == 26) v = P.U - P.F - P.A;
    else if (w == 27) v = P.F;
    else if (w == 28) v = P.PR;
    else if (w == 29) v = (i32)P.nreq;
    else if (w == 30) v = (i32)P.ncl;
    else if (w == 31) v = (i32)P.status;
    else if (w == TW_QUEUED) v = (i32)P.dq_len;
    else if (w == TW_T2_PEAK) v = (i32)P.t2peak;
    ptel->w[w] = v;
  }
}

// ---- host side -----------------------------------------------------------------------------
u64 align_up(u64 v, u64 a) { return (v + a - 1) / a * a; }

constexpr u32 kNodesLdsNarrow = 128, kNodesLdsWide = 64;

constexpr u64 kLdsBudget = 160 * 1024;
constexpr u32 kCUs = 256;  // compute units of one MI355X

// 16-bit storage holds every stored value of the batch below 0xFFFF
bool narrow_ok(const rkc_batch* b) {
  return b->max_usable_blocks <= 32767 && b->max_events <= 65533 && b->max_chains <= 65534 &&
         b->max_claim_slots <= 65534;
}

bool make_layout(const rkc_batch* b, Layout* L, bool narrow, bool global_lists) {
  memset(L, 0, sizeof *L);
  L->narrow = narrow;
  L->global_lists = global_lists;
  // Batches of at most one pool per CU whose lists live in global scratch get a workgroup of
  // several waves per pool: the other waves share the scans of the long lists.
  L->waves = (global_lists && b->n_pools <= (i32)kCUs && !(b->flags & RKC_FLAG_ONE_WAVE_PER_POOL)) ? kGroupWaves : 1;
  const u64 ws = narrow ? 2 : 4;
  L->chains = (u32)(b->max_chains > 0 ? b->max_chains : 1);
  L->reqs = (u32)(b->max_live_requests > 0 ? b->max_live_requests : 1);
  L->claims = (u32)(b->max_live_claims > 0 ? b->max_live_claims : 1);
  L->node_cap = (u32)b->max_events + 2;
  const u32 nlds = narrow ? kNodesLdsNarrow : kNodesLdsWide;
  L->nodes_lds = L->node_cap < nlds ? L->node_cap : nlds;
  u64 o = 0;
  auto take = [&](u64 bytes, u64 al) { o = align_up(o, al); u64 r = o; o += bytes; return (u32)r; };
  const u64 C = L->chains;
  L->off_chain = take(ws * CF_WORDS * C, 16);
  L->off_key = take(4 * (C > kRegChains ? C : 1), 16);
  L->off_mark = take(4 * C, 16);
  L->off_job = take(L->waves > 1 ? 4ull * (JB_ARGS + 8 * L->waves) : 0, 16);
  if (!global_lists) {
    L->off_rq = take(ws * RQ_ARRAYS * L->reqs, 16);
    L->off_cl = take(ws * CL_ARRAYS * L->claims, 16);
  }
  if (b->n_pools <= (i32)kCUs) {
    // at most one pool per CU: the node pool takes the LDS the other regions leave
    const u64 left = align_up(o, 16) < kLdsBudget ? kLdsBudget - align_up(o, 16) : 0;
    const u64 fit = left / (4 * ws);
    L->nodes_lds = (u32)(fit < L->node_cap ? fit : L->node_cap);
    if (L->nodes_lds < nlds && L->nodes_lds < L->node_cap) L->nodes_lds = L->node_cap < nlds ? L->node_cap : nlds;
  }
  L->off_node = take(4 * ws * L->nodes_lds, 16);
  o = align_up(o, 16);
  if (o > kLdsBudget) return false;
  L->lds_bytes = (u32)o;
  // scratch per pool: spilled nodes, FIFO ring, slot table, and the lists when they are global
  L->fifo_cap = (u32)b->max_events + 1;  // one entry per event at most
  u64 s = 0;
  L->scr_off_node = s; s += 16ull * (L->node_cap - L->nodes_lds); s = align_up(s, 256);
  L->scr_off_fifo = s; s += 16ull * L->fifo_cap; s = align_up(s, 256);
  L->scr_off_slot = s; s += 8ull * (u64)(b->max_claim_slots > 0 ? b->max_claim_slots : 1);
  s = align_up(s, 256);
  L->scr_off_dq = s; s += 16ull * L->reqs; s = align_up(s, 256);  // deferred requests (ring)
  if (global_lists) {
    L->scr_off_rq = s; s += 4ull * RQ_ARRAYS * 2 * L->reqs; s = align_up(s, 256);  // two-sided
    L->scr_off_cl = s; s += 4ull * CL_ARRAYS * L->claims;
  }
  L->scr_pool_bytes = align_up(s, 256);
  return true;
}

// Narrowest storage that fits: 16-bit words in LDS, else 32-bit words in LDS, else 32-bit words
// with the lists in global scratch.
bool choose_layout(const rkc_batch* b, Layout* L) {
  return (narrow_ok(b) && make_layout(b, L, true, false)) || make_layout(b, L, false, false) ||
         make_layout(b, L, false, true);
}

rkc_status check_batch(const rkc_batch* b) {
  if (!b) return RKC_E_NULL;
  if (b->n_pools < 0 || b->max_usable_blocks < 0 || b->max_events < 0 || b->max_chains < 0 ||
      b->max_live_requests < 0 || b->max_live_claims < 0 || b->max_claim_slots < 0 ||
      b->n_events_total < 0 || b->n_claim_slots_total < 0 ||
      (b->flags & ~(RKC_FLAG_GENERAL_KERNEL | RKC_FLAG_ONE_WAVE_PER_POOL)) != 0)
    return RKC_E_RANGE;
  if (b->max_usable_blocks > RKC_MAX_USABLE_BLOCKS || b->max_events > RKC_MAX_EVENTS_PER_POOL)
    return RKC_E_UNSUPPORTED;
  if (b->n_pools == 0) return RKC_OK;
  if (!b->d_pools || !b->d_pool_tel || (b->n_events_total > 0 && (!b->d_events || !b->d_outcomes)) ||
      (b->n_claim_slots_total > 0 && !b->d_claim_tel))
    return RKC_E_NULL;
  if (((uintptr_t)b->d_pools & 15) || ((uintptr_t)b->d_events & 15) || ((uintptr_t)b->d_outcomes & 15) ||
      ((uintptr_t)b->d_pool_tel & 15) || ((uintptr_t)b->d_claim_tel & 7) || ((uintptr_t)b->d_scratch & 255))
    return RKC_E_ALIGN;
  return RKC_OK;
}

template <typename W, bool kGL, int NW>
rkc_status launch(const Args& g, unsigned n_pools, hipStream_t s) {
  const void* fn = (const void*)rkc_replay_wave<W, kGL, NW>;
  if (g.L.lds_bytes > 64 * 1024 &&
      hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)g.L.lds_bytes) != hipSuccess)
    return RKC_E_HIP;
  hipLaunchKernelGGL((rkc_replay_wave<W, kGL, NW>), dim3(n_pools), dim3(64 * NW), g.L.lds_bytes, s, g);
  return hipGetLastError() == hipSuccess ? RKC_OK : RKC_E_HIP;
}

// The compact kernel serves every batch within its limits unless the caller asks for the
// general one.
bool use_lean(const rkc_batch* b, rkc_lean_args* g) {
  memset(g, 0, sizeof *g);
  return !(b->flags & RKC_FLAG_GENERAL_KERNEL) && rkc_lean_layout(b, g);
}

}  // namespace

extern "C" {

int32_t rkc_abi_version(void) { return RKC_ABI_VERSION; }

size_t rkc_scratch_bytes(const rkc_batch* b) {
  if (!b || b->n_pools <= 0) return 0;
  rkc_lean_args lg;
  if (use_lean(b, &lg)) return (size_t)lg.scr_total;
  Layout L;
  if (!choose_layout(b, &L)) return 0;
  return (size_t)(L.scr_pool_bytes * (u64)b->n_pools);
}

static rkc_status replay(const rkc_batch* b, void* s) {
  rkc_status st = check_batch(b);
  if (st != RKC_OK) return st;
  if (b->n_pools == 0) return RKC_OK;
  rkc_lean_args lg;
  if (use_lean(b, &lg)) {
    const u64 need = lg.scr_total;
    if (!b->d_scratch || b->scratch_bytes < need) return RKC_E_SCRATCH;
    lg.pools = b->d_pools; lg.events = b->d_events; lg.outcomes = b->d_outcomes;
    lg.pool_tel = b->d_pool_tel; lg.claim_tel = b->d_claim_tel; lg.scratch = b->d_scratch;
    lg.n_events_total = b->n_events_total; lg.n_slots_total = b->n_claim_slots_total;
    lg.n_pools = b->n_pools; lg.max_usable = b->max_usable_blocks; lg.max_events = b->max_events;
    lg.max_chains = b->max_chains; lg.max_reqs = b->max_live_requests; lg.max_claims = b->max_live_claims;
    lg.max_slots = b->max_claim_slots;
    return rkc_lean_launch(&lg, (hipStream_t)s);
  }
  Args g;
  memset(&g, 0, sizeof g);
  if (!choose_layout(b, &g.L)) return RKC_E_UNSUPPORTED;
  const u64 need = g.L.scr_pool_bytes * (u64)b->n_pools;
  if (!b->d_scratch || b->scratch_bytes < need) return RKC_E_SCRATCH;
  g.pools = b->d_pools; g.events = b->d_events; g.outcomes = b->d_outcomes;
  g.pool_tel = b->d_pool_tel; g.claim_tel = b->d_claim_tel; g.scratch = (unsigned char*)b->d_scratch;
  g.n_events_total = b->n_events_total; g.n_slots_total = b->n_claim_slots_total;
  g.n_pools = b->n_pools; g.max_usable = b->max_usable_blocks; g.max_events = b->max_events;
  g.max_chains = b->max_chains; g.max_reqs = b->max_live_requests; g.max_claims = b->max_live_claims;
  g.max_slots = b->max_claim_slots;
  if (g.L.narrow) return launch<uint16_t, false, 1>(g, (unsigned)b->n_pools, (hipStream_t)s);
  if (g.L.global_lists && g.L.waves > 1)
    return launch<u32, true, kGroupWaves>(g, (unsigned)b->n_pools, (hipStream_t)s);
  if (g.L.global_lists) return launch<u32, true, 1>(g, (unsigned)b->n_pools, (hipStream_t)s);
  return launch<u32, false, 1>(g, (unsigned)b->n_pools, (hipStream_t)s);
}

rkc_status rkc_replay_batch(const rkc_batch* b, void* s) { return replay(b, s); }

// Device address of the built-in scratch on the current device, looked up once per device.
static void* noalloc_scratch(void) {
  enum { kMaxDevices = 64 };
  static std::mutex mu;
  static void* addr[kMaxDevices];
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
  std::lock_guard<std::mutex> lock(mu);
  if (!addr[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return nullptr;
    addr[dev] = p;
  }
  return addr[dev];
}

rkc_status rkc_replay_batch_noalloc(const rkc_batch* b, void* s) {
  if (!b) return RKC_E_NULL;
  rkc_batch nb = *b;
  nb.d_scratch = nullptr;
  nb.scratch_bytes = 0;
  rkc_status st = check_batch(&nb);
  if (st != RKC_OK) return st;
  if (nb.n_pools == 0) return RKC_OK;
  if (rkc_scratch_bytes(&nb) > (size_t)RKC_NOALLOC_SCRATCH_BYTES) return RKC_E_SCRATCH_LIMIT;
  void* p = noalloc_scratch();
  if (!p) return RKC_E_HIP;
  nb.d_scratch = p;
  nb.scratch_bytes = (size_t)RKC_NOALLOC_SCRATCH_BYTES;
  return replay(&nb, s);
}

static rkc_status read_desc(const rkc_batch* b, int32_t pool, rkc_pool_desc* d, void* s) {
  if (!b) return RKC_E_NULL;
  if (pool < 0 || pool >= b->n_pools) return RKC_E_RANGE;
  if (hipStreamSynchronize((hipStream_t)s) != hipSuccess) return RKC_E_HIP;
  if (hipMemcpy(d, b->d_pools + pool, sizeof *d, hipMemcpyDeviceToHost) != hipSuccess) return RKC_E_HIP;
  return RKC_OK;
}

static rkc_status pool_status(const rkc_batch* b, int32_t pool, rkc_status ok) {
  int32_t w = 0;
  if (hipMemcpy(&w, &b->d_pool_tel[pool].w[31], 4, hipMemcpyDeviceToHost) != hipSuccess) return RKC_E_HIP;
  return w != 0 ? RKC_E_POOL_STATUS : ok;
}

rkc_status rkc_query_outcomes(const rkc_batch* b, int32_t pool, int32_t first, int32_t count,
                              rkc_outcome* host_dst, void* s) {
  if (!host_dst && count > 0) return RKC_E_NULL;
  rkc_pool_desc d;
  rkc_status st = read_desc(b, pool, &d, s);
  if (st != RKC_OK) return st;
  if (first < 0 || count < 0 || (int64_t)first + count > d.n_events) return RKC_E_RANGE;
  // the descriptor is caller data: never copy from outside the batch's outcome array
  if (d.event_offset < 0 || d.event_offset > b->n_events_total ||
      (int64_t)first + count > b->n_events_total - d.event_offset)
    return RKC_E_RANGE;
  if (count > 0 && hipMemcpy(host_dst, b->d_outcomes + d.event_offset + first,
                             (size_t)count * sizeof(rkc_outcome), hipMemcpyDeviceToHost) != hipSuccess)
    return RKC_E_HIP;
  return pool_status(b, pool, RKC_OK);
}

rkc_status rkc_query_telemetry(const rkc_batch* b, int32_t pool, rkc_pool_telemetry* host_pool,
                               rkc_claim_telemetry* host_claims, int32_t max_claims,
                               int32_t* n_claims, void* s) {
  rkc_pool_desc d;
  rkc_status st = read_desc(b, pool, &d, s);
  if (st != RKC_OK) return st;
  if (n_claims) *n_claims = d.n_claim_slots;
  if (host_pool && hipMemcpy(host_pool, b->d_pool_tel + pool, sizeof *host_pool,
                             hipMemcpyDeviceToHost) != hipSuccess)
    return RKC_E_HIP;
  if (host_claims && max_claims > 0) {
    int32_t k = d.n_claim_slots < max_claims ? d.n_claim_slots : max_claims;
    // the descriptor is caller data: never copy from outside the batch's claim telemetry array
    if (k > 0 && (d.claim_slot_offset < 0 || d.claim_slot_offset > b->n_claim_slots_total ||
                  k > b->n_claim_slots_total - d.claim_slot_offset))
      return RKC_E_RANGE;
    if (k > 0 && hipMemcpy(host_claims, b->d_claim_tel + d.claim_slot_offset,
                           (size_t)k * sizeof(rkc_claim_telemetry), hipMemcpyDeviceToHost) != hipSuccess)
      return RKC_E_HIP;
  }
  return pool_status(b, pool, RKC_OK);
}

#ifdef RKC_CHECK_UNIFORM
// Checking build only (not part of the ABI): readfirstlane calls of either kernel whose active lanes
// held different values, since the library was loaded.
uint32_t rkc_debug_uniform_violations(void) {
  unsigned v = 0;
  if (hipMemcpyFromSymbol(&v, HIP_SYMBOL(g_wave_uniform_violations), sizeof v) != hipSuccess) return ~0u;
  const unsigned w = rkc_lean_uniform_violations();
  return w == ~0u ? ~0u : v + w;
}
#endif

const char* rkc_status_string(rkc_status st) {
  switch (st) {
    case RKC_OK: return "ok";
    case RKC_E_NULL: return "null pointer";
    case RKC_E_ALIGN: return "misaligned pointer";
    case RKC_E_RANGE: return "argument out of range";
    case RKC_E_UNSUPPORTED: return "unsupported size or mode";
    case RKC_E_SCRATCH: return "scratch buffer missing or too small";
    case RKC_E_HIP: return "HIP runtime error";
    case RKC_E_POOL_STATUS: return "pool status is non-zero";
    case RKC_E_SCRATCH_LIMIT: return "batch needs more scratch than the built-in buffer holds";
  }
  return "unknown status";
}

}  // extern "C"
