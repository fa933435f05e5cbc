// rkc_replay.hip -- batched replay of resident-KV-claim arbitration on MI355X (gfx950).
//
// One wavefront replays one pool.  Pools are independent (the contract is per pool), so the grid is
// one 64-lane workgroup per pool and the hardware dispatcher balances them over the 256 CUs.
//
// The pool is not kept one block at a time.  Because every touch, hit, hold, protection and claim
// coverage is a leading range [0, x) of a chain, the registered positions of every shared chain are
// always a leading run [0, n_c) and eviction always takes a chain from its top.  The kernel therefore
// keeps, per shared chain:
//   n      registered length              hold   leading positions held ACTIVE by live requests
//   prot   max L of materialized hard claims (hard-protection pools)
//   lv[v]  max L of claims that rank victims at soft level v (priority + 1)
//   covA   max L of live claims           covS   max L of live claims not demoted / expired
//   tpend  max T of claims whose predicate has not failed yet
//   a touch stack: (x, t) pairs, x strictly decreasing, t increasing; position p was last touched
//          at the t of the newest pair with x > p
//   topkey the eviction key (level, last use, -pos) of the chain's top candidate
// Finished requests' private blocks form runs (finish step, [lo, top)); runs finish in step order,
// so they sit in a FIFO and the front run is always the oldest.
//
// Victim selection takes the (need - F) smallest keys (level asc, last use asc, pos desc) over all
// candidates (§3.1 soft priority; §5.3 ordinary eviction after free blocks; hard-protected blocks
// excluded).  It merges chain tops: a wave min-reduction finds the chain with the smallest top key
// and the runner-up key, then whole runs of equal (level, last use) are evicted at once.
//
// LDS holds the per-chain arrays, the live-request and live-claim lists and the first touch-stack
// nodes; global scratch holds the remaining nodes, the FIFO ring and the per-slot (chain, L) table.
// Scratch is only read back by the lane(s) that wrote it, or after a workgroup fence.
#include <hip/hip_runtime.h>
#include <stdint.h>
#include <string.h>

#include "rkc.h"

namespace {

typedef uint32_t u32;
typedef int32_t i32;
typedef uint64_t u64;
typedef int64_t i64;

// Explicit address spaces for arrays reached through a run-time choice (LDS part or global part
// of the node arena), so each access compiles to a ds_ or global_ instruction, never a flat one.
typedef __attribute__((address_space(3))) uint4 lds_uint4;
typedef __attribute__((address_space(1))) uint4 glb_uint4;

constexpr u32 NIL = 0xFFFFFFFFu;
constexpr u64 KEY_INF = ~0ull;
constexpr u32 EXP_NEVER = 0xFFFFFFFFu;

// claim states (ResidentClaimState, §3.1) and decisions
enum : u32 { ST_SUBMITTED = 0, ST_OBSERVED = 1, ST_MATERIALIZED = 2, ST_DEMOTED = 3, ST_EXPIRED = 4,
             ST_RELEASED = 5, ST_HARMED = 6, ST_REJECTED = 7 };
enum : u32 { DEC_ACCEPTED = 1, DEC_APPROX = 2, DEC_SHADOW = 3, DEC_REJECTED = 4 };

// live-claim meta word: state[0:3) eff[3:5) hard[5] prio[6:8) pending[8] decision[9:12)
__device__ __forceinline__ u32 m_state(u32 m) { return m & 7u; }
__device__ __forceinline__ u32 m_eff(u32 m) { return (m >> 3) & 3u; }
__device__ __forceinline__ u32 m_hard(u32 m) { return (m >> 5) & 1u; }
__device__ __forceinline__ u32 m_prio(u32 m) { return (m >> 6) & 3u; }
__device__ __forceinline__ u32 m_pending(u32 m) { return (m >> 8) & 1u; }
__device__ __forceinline__ u32 m_dec(u32 m) { return (m >> 9) & 7u; }
__device__ __forceinline__ u32 m_with_state(u32 m, u32 s) { return (m & ~7u) | s; }

__device__ __forceinline__ u32 packed_of(u32 m) {
  return m_dec(m) | (m_state(m) << 4) | (m_hard(m) << 8) | (m_prio(m) << 9) | (m_eff(m) << 11);
}

__device__ __forceinline__ u64 make_key(u32 level, u32 lu, u32 pos) {
  return ((u64)level << 60) | ((u64)(lu & 0x0FFFFFFFu) << 32) | (u64)(0xFFFFFFFFu - pos);
}

// ---- wave primitives ------------------------------------------------------------------------
__device__ __forceinline__ u32 lane_id() { return __lane_id(); }

__device__ __forceinline__ u64 ballot(bool p) { return __ballot(p); }
__device__ __forceinline__ i32 rdlane(i32 v, u32 l) { return __builtin_amdgcn_readlane(v, (int)l); }

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

template <int CTRL>
__device__ __forceinline__ u64 dpp64(u64 v) {
  return ((u64)dpp<CTRL>((u32)(v >> 32)) << 32) | dpp<CTRL>((u32)v);
}
__device__ __forceinline__ u64 min64(u64 a, u64 b) { return a < b ? a : b; }
__device__ __forceinline__ u64 rdlane64(u64 v, u32 l) {
  return ((u64)(u32)rdlane((i32)(u32)(v >> 32), l) << 32) | (u32)rdlane((i32)(u32)v, l);
}
__device__ __forceinline__ u64 wave_min64(u64 v) {
  v = min64(v, dpp64<kDppXor1>(v));
  v = min64(v, dpp64<kDppXor2>(v));
  v = min64(v, dpp64<kDppHalfMirror>(v));
  v = min64(v, dpp64<kDppMirror>(v));
  return min64(min64(rdlane64(v, 0), rdlane64(v, 16)), min64(rdlane64(v, 32), rdlane64(v, 48)));
}

// ---- launch geometry (computed on the host) ---------------------------------------------------
struct Layout {
  u32 chains, reqs, claims, nodes_lds;
  u32 off_n, off_hold, off_prot, off_covA, off_covS, off_tpend, off_lv, off_stop, off_sbot,
      off_mark, off_key, off_tel, off_rq, off_cl, off_node, off_bt, off_nx;
  u32 lds_bytes;
  u64 scr_pool_bytes, scr_off_node, scr_off_fifo, scr_off_slot, scr_off_rq, scr_off_cl;
  u32 fifo_cap, node_cap;
  u32 global_lists;
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
// internal-consistency fault bit in the pool status word: set only if a structural bound that
// the algorithm guarantees is ever violated; loops stop instead of running on.
constexpr u32 kFault = 0x80000000u;
// chains whose top keys live in registers (four per lane)
constexpr u32 kRegChains = 256;

struct AllocRes {
  bool ok;
  i32 E;  // evictable candidates before the event (valid when need > F)
  i32 victims, resident, post, unclaimed;
};

// ---- the per-pool replay ----------------------------------------------------------------------
// kGL: the live-request and live-claim lists live in global scratch instead of LDS (pools whose
// lists do not fit on chip).  Lane-parallel writes to them are then followed by a workgroup fence
// before any other lane reads them.
template <bool kGL>
struct Pool {
  // descriptor
  i32 U, mode, n_events, n_chains, max_claims, max_reqs, n_slots;
  i64 ev_off, slot_off;
  u32 lane;
  // LDS arrays
  u32 *n, *hold, *prot, *covA, *covS, *tpend, *lv, *stop, *sbot, *mark, *tel;
  u32 *bt, *nx;   // cached bottom of each touch stack: its step, and the extent of the pair above
  u64* topkey;    // chains >= kRegChains; lower chains keep their top key in registers (kr)
  u64 kr0, kr1, kr2, kr3;  // top key of chain 64 * k + lane, k = 0..3
  u32 *rq_id, *rq_c, *rq_R, *rq_len;
  u32 *cl_id, *cl_c, *cl_L, *cl_T, *cl_meta, *cl_exp, *cl_slot, *cl_blk;
  u32 *cl_dem, *cl_exst, *cl_pf, *cl_harm;  // demote / expire / predicate-failure / harm steps
  u32 cl_cap, rq_cap;
  lds_uint4* node_lds;
  glb_uint4* node_glb;
  u32 nl;
  uint4* fifo;
  u32 fifo_cap;
  uint2* slot_cl;
  rkc_claim_telemetry* rec;
  // scalar state (wave-uniform)
  i32 F, A, PR, peak;
  i32 Eall;       // sum over chains of max(0, n - max(hold, prot)): evictable shared blocks
  u32 nreq, ncl, nslot;
  u32 next_exp;
  u32 free_head, bump;
  u32 fhead, ftail, ft, flo, ftop;
  i32 fblocks;
  u32 status;
  u32 node_cap;

  // -- nodes (x = extent, y = step, z = up (newer), w = down (older)); the first nl live in LDS,
  //    the rest in global scratch (both read and written by every lane with uniform addresses) --
  __device__ __forceinline__ uint4 nget(u32 i) {
    uint4 v;
    if (i < nl) { const lds_uint4& r = node_lds[i]; v = make_uint4(r.x, r.y, r.z, r.w); }
    else { const glb_uint4& r = node_glb[i - nl]; v = make_uint4(r.x, r.y, r.z, r.w); }
    return v;
  }
  __device__ __forceinline__ u32 nget_x(u32 i) { u32 v; if (i < nl) v = node_lds[i].x; else v = node_glb[i - nl].x; return v; }
  __device__ __forceinline__ u32 nget_z(u32 i) { u32 v; if (i < nl) v = node_lds[i].z; else v = node_glb[i - nl].z; return v; }
  __device__ __forceinline__ u32 nget_w(u32 i) { u32 v; if (i < nl) v = node_lds[i].w; else v = node_glb[i - nl].w; return v; }
  __device__ __forceinline__ void nset(u32 i, uint4 v) {
    if (i < nl) { node_lds[i].x = v.x; node_lds[i].y = v.y; node_lds[i].z = v.z; node_lds[i].w = v.w; }
    else { node_glb[i - nl].x = v.x; node_glb[i - nl].y = v.y; node_glb[i - nl].z = v.z; node_glb[i - nl].w = v.w; }
  }
  __device__ __forceinline__ void nset_z(u32 i, u32 v) { if (i < nl) node_lds[i].z = v; else node_glb[i - nl].z = v; }
  __device__ __forceinline__ void nset_w(u32 i, u32 v) { if (i < nl) node_lds[i].w = v; else node_glb[i - nl].w = v; }
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
  __device__ __forceinline__ void set_key(u32 c, u64 k) {
    if (c < kRegChains) {
      const u32 l = c & 63u, s = c >> 6;
      if (lane == l) {
        if (s == 0) kr0 = k;
        else if (s == 1) kr1 = k;
        else if (s == 2) kr2 = k;
        else kr3 = k;
      }
    } else {
      topkey[c] = k;
    }
  }

  // -- chain counters: every change of n, hold or prot keeps Eall and PR (protected cached
  //    blocks, hard-protection pools) exact --
  __device__ __forceinline__ i32 evictable(u32 nn, u32 hh, u32 pp) { return max(0, (i32)nn - (i32)max(hh, pp)); }
  __device__ __forceinline__ void chain_update(u32 c, u32 nn, u32 hh, u32 pp) {
    const u32 n0 = n[c], h0 = hold[c], p0 = prot[c];
    Eall += evictable(nn, hh, pp) - evictable(n0, h0, p0);
    PR += max(0, (i32)pp - (i32)hh) - max(0, (i32)p0 - (i32)h0);
    n[c] = nn; hold[c] = hh; prot[c] = pp;
  }

  __device__ __forceinline__ void lists_fence() {
    if (kGL) __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "workgroup");
  }

  __device__ __forceinline__ bool soft_levels() const { return mode == RKC_MODE_SOFT || mode == RKC_MODE_HARD; }

  __device__ __forceinline__ u32 level_at(u32 c, u32 p) {
    if (!soft_levels()) return 0;
    u32 lvl = 0;
#pragma unroll
    for (u32 v = 1; v <= 4; v++)
      if (lv[4 * c + v - 1] > p) lvl = v;
    return lvl;
  }

  // Key of chain c's top candidate.  The stack bottom is the newest pair covering position n-1
  // exactly when the pair above it (extent nx) does not reach n-1; otherwise advance the bottom.
  __device__ __forceinline__ u64 top_key(u32 c) {
    const u32 nn = n[c];
    const u32 lo = max(hold[c], prot[c]);
    if (nn <= lo) return KEY_INF;
    u32 t_bot = bt[c];
    if (nx[c] >= nn) {
      u32 b = sbot[c];
      if (b == NIL) { status |= kFault; return KEY_INF; }
      u32 up = nget_z(b);
      for (u32 guard = 0; guard < node_cap && up != NIL && nget_x(up) >= nn; guard++) {
        nset_w(up, NIL);
        node_free(b);
        b = up;
        up = nget_z(b);
      }
      sbot[c] = b;
      t_bot = nget(b).y;
      bt[c] = t_bot;
      nx[c] = up != NIL ? nget_x(up) : 0u;
    }
    return make_key(level_at(c, nn - 1), t_bot, nn - 1);
  }
  __device__ __forceinline__ void refresh(u32 c) { set_key(c, top_key(c)); }

  // Record a touch of positions [0, x) of chain c at step t.
  __device__ __forceinline__ void touch(u32 c, u32 x, u32 t) {
    if (x == 0) return;
    u32 tp = stop[c];
    for (u32 guard = 0; guard < node_cap && tp != NIL && nget_x(tp) <= x; guard++) {
      const u32 d = nget_w(tp);
      node_free(tp);
      tp = d;
    }
    const u32 nw = node_alloc();
    nset(nw, make_uint4(x, t, NIL, tp));
    if (tp != NIL) {
      nset_z(tp, nw);
      if (tp == sbot[c]) nx[c] = x;   // the new pair sits right above the bottom
    } else {
      sbot[c] = nw;                   // the new pair is the whole stack
      bt[c] = t;
      nx[c] = 0;
    }
    stop[c] = nw;
  }


  // Recompute chain c's claim maxima from the live-claim list.
  __device__ __forceinline__ void recompute(u32 c) {
    u32 pr = 0, l1 = 0, l2 = 0, l3 = 0, l4 = 0, ca = 0, cs = 0, tp = 0;
    const bool hardm = mode == RKC_MODE_HARD, softl = soft_levels();
    for (u32 i = lane; i < ncl; i += 64) {
      if (cl_c[i] != c) continue;
      u32 m = cl_meta[i], L = cl_L[i], st = m_state(m);
      ca = max(ca, L);
      if (st == ST_OBSERVED || st == ST_MATERIALIZED || st == ST_HARMED) cs = max(cs, L);
      if (hardm && st == ST_MATERIALIZED && m_eff(m) == RKC_PROT_HARD) pr = max(pr, L);
      if (softl && ((st == ST_MATERIALIZED && m_eff(m) == RKC_PROT_SOFT) || st == ST_DEMOTED)) {
        u32 p = m_prio(m);
        if (p == 0) l1 = max(l1, L); else if (p == 1) l2 = max(l2, L);
        else if (p == 2) l3 = max(l3, L); else l4 = max(l4, L);
      }
      if (m_pending(m) && st != ST_HARMED) tp = max(tp, cl_T[i]);
    }
    pr = wave_max(pr); l1 = wave_max(l1); l2 = wave_max(l2); l3 = wave_max(l3); l4 = wave_max(l4);
    ca = wave_max(ca); cs = wave_max(cs); tp = wave_max(tp);
    chain_update(c, n[c], hold[c], pr);
    lv[4 * c + 0] = l1; lv[4 * c + 1] = l2; lv[4 * c + 2] = l3; lv[4 * c + 3] = l4;
    covA[c] = ca; covS[c] = cs; tpend[c] = tp;
    refresh(c);
  }

  // Recompute every chain whose mark has bit `bit`, and clear the marks.
  __device__ __forceinline__ void recompute_marked(u32 bit) {
    for (u32 base = 0; base < (u32)n_chains; base += 64) {
      u32 c = base + lane;
      bool mk = c < (u32)n_chains && (mark[c] & bit);
      u64 b = ballot(mk);
      while (b) {
        u32 l = (u32)__builtin_ctzll(b);
        b &= b - 1;
        u32 cc = base + l;
        recompute(cc);
        mark[cc] &= ~bit;
      }
    }
  }

  // Candidates: shared-chain tops above max(hold, prot) (and above the hits on chain hc), plus the
  // private FIFO runs.
  __device__ __forceinline__ i32 candidates(i32 hc, u32 h) {
    i32 e = Eall + fblocks;
    if (hc >= 0) {
      const u32 nn = n[hc], lo = max(hold[hc], prot[hc]);
      e -= evictable(nn, lo, 0) - evictable(nn, max(lo, h), 0);
    }
    return e;
  }

  __device__ __forceinline__ void fifo_pop_front() {
    fhead++;
    if (fhead != ftail) {
      uint4 e = fifo[fhead % fifo_cap];
      ft = e.x; flo = e.y; ftop = e.z;
    }
  }

  // ALLOC: FREE blocks first, then the (need - F) smallest-key candidates.
  __device__ __forceinline__ AllocRes alloc(i32 need, i32 hc, u32 h, bool& any_sweep) {
    AllocRes r = {true, 0, 0, 0, 0, 0};
    if (need <= F) {
      F -= need;
      return r;
    }
    i32 E = candidates(hc, h);
    r.E = E;
    if ((i64)need > (i64)F + E) {
      r.ok = false;
      return r;
    }
    i32 K = need - F;
    F = 0;
    for (u32 guard = 0; K > 0; guard++) {
      if (guard > (u32)U + 1) { status |= kFault; break; }
      u64 k1 = KEY_INF, k2 = KEY_INF;
      u32 i1 = NIL;
      const bool hc_empty = hc >= 0 && n[hc] <= h;  // every candidate of the hit chain is a hit
      const u64 krs[4] = {kr0, kr1, kr2, kr3};
#pragma unroll
      for (u32 q = 0; q < 4; q++) {
        const u32 c = 64 * q + lane;
        u64 k = krs[q];
        if (hc_empty && (i32)c == hc) k = KEY_INF;
        if (k < k1) { k2 = k1; k1 = k; i1 = c; }
        else if (k < k2) k2 = k;
      }
      for (u32 c = kRegChains + lane; c < (u32)n_chains; c += 64) {
        u64 k = topkey[c];
        if (hc_empty && (i32)c == hc) k = KEY_INF;
        if (k < k1) { k2 = k1; k1 = k; i1 = c; }
        else if (k < k2) k2 = k;
      }
      u64 m1 = wave_min64(k1);
      u64 kf = (fhead != ftail) ? make_key(0, ft, ftop - 1) : KEY_INF;
      u64 best, second;
      u32 src;
      if (kf < m1) {
        best = kf; second = m1; src = NIL;
      } else {
        u64 bl = ballot(k1 == m1);
        u32 l = (u32)__builtin_ctzll(bl);
        src = (u32)rdlane((i32)i1, l);
        u64 mine = (lane == l) ? k2 : k1;
        u64 m2 = wave_min64(mine);
        best = m1;
        second = m2 < kf ? m2 : kf;
      }
      if (best == KEY_INF) { status |= kFault; break; }
      const bool tie = second != KEY_INF && (second >> 32) == (best >> 32);
      const u32 p2 = 0xFFFFFFFFu - (u32)second;
      if (src == NIL) {
        u32 m_run = ftop - flo;
        if (tie) m_run = ftop - max(flo, p2 + 1);
        u32 m = min((u32)K, m_run);
        if (m == 0 || m > ftop - flo) { status |= kFault; break; }
        ftop -= m;
        fblocks -= (i32)m;
        r.victims += (i32)m;
        r.unclaimed += (i32)m;
        K -= (i32)m;
        if (ftop == flo) fifo_pop_front();
      } else {
        u32 c = src, nn = n[c], p = nn - 1;
        u32 lo = max(hold[c], prot[c]);
        if ((i32)c == hc) lo = max(lo, h);
        u32 lvl = level_at(c, p);
        u32 lvb = 0;
        if (soft_levels())
          for (u32 v = lvl + 1; v <= 4; v++) lvb = max(lvb, lv[4 * c + v - 1]);
        const u32 lub = nx[c];  // positions below it were touched later
        u32 run_lo = max(lo, max(lvb, lub));
        u32 m_run = nn - run_lo;
        if (tie) m_run = nn - max(run_lo, p2 + 1);
        u32 m = min((u32)K, m_run);
        if (m == 0 || m > nn) { status |= kFault; break; }
        u32 nw = nn - m;
        i32 res = max(0, (i32)min(nn, covA[c]) - (i32)nw);
        i32 strict = max(0, (i32)min(nn, covS[c]) - (i32)nw);
        r.victims += (i32)m;
        r.resident += res;
        r.post += res - strict;
        r.unclaimed += (i32)m - res;
        chain_update(c, nw, hold[c], prot[c]);
        refresh(c);
        if (nw < tpend[c]) {
          mark[c] |= MK_SWEEP;
          any_sweep = true;
        }
        K -= (i32)m;
      }
    }
    return r;
  }

  // Predicate sweep over claims on chains that shrank below a pending threshold (§3.2 harm).
  __device__ __forceinline__ u32 sweep(u32 t) {
    u32 pf = 0, hm = 0;
    for (u32 i = lane; i < ncl; i += 64) {
      u32 c = cl_c[i];
      if (!(mark[c] & MK_SWEEP)) continue;
      u32 m = cl_meta[i], st = m_state(m);
      if (!m_pending(m) || st == ST_HARMED) continue;
      if (n[c] >= cl_T[i]) continue;
      m &= ~(1u << 8);
      pf++;
      cl_pf[i] = t;
      if (st == ST_MATERIALIZED) {
        m = m_with_state(m, ST_HARMED);
        hm++;
        cl_harm[i] = t;
      }
      cl_meta[i] = m;
    }
    lists_fence();
    pf = wave_sum(pf);
    hm = wave_sum(hm);
    tel[20] += pf;
    tel[19] += hm;
    recompute_marked(MK_SWEEP);
    return (pf ? (u32)RKC_FL_PRED_FAIL : 0u) | (hm ? (u32)RKC_FL_HARM : 0u);
  }

  // Refusal record of an active event that cannot be served (§3.4; §5.4 refusal record).
  __device__ __forceinline__ void refusal(i32 need, i32 hc, u32 h, i32 Hc, i32& code, i32& id, i32& a, i32& b,
                          u32& n16) {
    i32 Pr = PR;
    if (mode == RKC_MODE_HARD && hc >= 0)
      Pr -= max(0, (i32)min(prot[hc], h) - (i32)hold[hc]);
    i64 req = (i64)A + Hc + need;
    if (Pr > 0 && req <= U) {
      code = RKC_OC_REFUSED_CLAIM;
      u32 mn = NIL, cnt = 0;
      for (u32 i = lane; i < ncl; i += 64) {
        u32 m = cl_meta[i];
        if (m_state(m) != ST_MATERIALIZED || m_eff(m) != RKC_PROT_HARD) continue;
        u32 c = cl_c[i];
        u32 cov = hold[c];
        if ((i32)c == hc) cov = max(cov, h);
        if (cl_L[i] <= cov) continue;
        cl_blk[i] += 1;
        cnt++;
        mn = min(mn, cl_id[i]);
      }
      lists_fence();
      id = (i32)wave_min(mn);
      n16 = min(wave_sum(cnt), 65535u);
    } else {
      code = RKC_OC_REFUSED_CAPACITY;
      id = -1;
      n16 = 0;
    }
    a = Pr;
    b = (i32)req;
  }

  // Claim records: words 0..8 are written exactly once (lane k writes word k), when the claim is
  // final (rejected at birth, released, or live at the end); word 9 (lead_end) is written by the
  // final pass.
  __device__ __forceinline__ void write_record(u32 slot, i32 id, u32 packed, i32 accept, i32 dem, i32 exst, i32 rel,
                               i32 pf, i32 harm, i32 blk) {
    if (lane < 9) {
      i32 v = lane == 0 ? id : lane == 1 ? (i32)packed : lane == 2 ? accept : lane == 3 ? dem
            : lane == 4 ? exst : lane == 5 ? rel : lane == 6 ? pf : lane == 7 ? harm : blk;
      rec[slot].w[lane] = v;
    }
  }
  __device__ __forceinline__ i32 step_or_none(u32 v) { return v == NIL ? -1 : (i32)v; }
  __device__ __forceinline__ void write_live_record(u32 i, u32 state, i32 rel) {
    write_record(cl_slot[i], (i32)cl_id[i], packed_of(m_with_state(cl_meta[i], state)), (i32)cl_id[i],
                 step_or_none(cl_dem[i]), step_or_none(cl_exst[i]), rel, step_or_none(cl_pf[i]),
                 step_or_none(cl_harm[i]), (i32)cl_blk[i]);
  }

  // Remove entry i of a struct-of-arrays list (narr arrays of capacity cap) by shifting the tail
  // down one place; lanes read their source entries before any lane writes.
  __device__ __forceinline__ void list_remove(u32* base0, u32 cap, u32 narr, u32 len, u32 i) {
    for (u32 base = i; base + 1 < len; base += 64) {
      const u32 j = base + lane;
      const bool act = j + 1 < len;
      for (u32 k = 0; k < narr; k++) {
        u32* a = base0 + k * cap;
        u32 v = act ? a[j + 1] : 0;
        __builtin_amdgcn_wave_barrier();
        if (act) a[j] = v;
        __builtin_amdgcn_wave_barrier();
      }
    }
    lists_fence();
  }
  __device__ __forceinline__ void claim_remove(u32 i) {
    list_remove(cl_id, cl_cap, 12, ncl, i);
    ncl--;
  }

  __device__ __forceinline__ void expire(u32 t, u32& flags, u32& expired) {
    u32 cnt = 0, nx = EXP_NEVER;
    for (u32 i = lane; i < ncl; i += 64) {
      u32 m = cl_meta[i], st = m_state(m), ex = cl_exp[i];
      if ((st != ST_MATERIALIZED && st != ST_DEMOTED) || ex == EXP_NEVER) continue;
      if (ex <= t) {
        cl_meta[i] = m_with_state(m, ST_EXPIRED);
        cl_exst[i] = t;
        mark[cl_c[i]] |= MK_RECOMP;
        cnt++;
      } else {
        nx = min(nx, ex);
      }
    }
    lists_fence();
    cnt = wave_sum(cnt);
    next_exp = wave_min(nx);
    if (cnt) {
      __builtin_amdgcn_wave_barrier();
      recompute_marked(MK_RECOMP);
      flags |= RKC_FL_EXPIRED;
      tel[21] += cnt;
    }
    expired = cnt;
  }

  // One event.  Returns the outcome words.
  __device__ __forceinline__ int4 step(u32 t, i32 w0, i32 w1, i32 w2, i32 w3) {
    const u32 uw0 = (u32)w0;
    const u32 type = uw0 & 15u, hardq = (uw0 >> 4) & 1u, prio = (uw0 >> 5) & 3u, dur = uw0 >> 16;
    u32 flags = 0, expired = 0, n16 = NIL;
    i32 code = RKC_OC_NOOP, id = -1, a = 0, b = 0;
    bool any_sweep = false;

    if (t >= next_exp) expire(t, flags, expired);

    // validation (malformed events and table limits)
    bool invalid = false;
    if (type == RKC_EV_PREFILL) {
      if (w1 < 1 || w1 > RKC_MAX_FIELD_BLOCKS || w3 < 0 || w3 > w1 ||
          (w3 > 0 && (w2 < 0 || w2 >= n_chains)))
        invalid = true;
      else if (nreq >= (u32)max_reqs) { invalid = true; status |= RKC_PS_REQUEST_TABLE; }
    } else if (type == RKC_EV_EXTEND) {
      invalid = w1 < 1 || w1 > RKC_MAX_FIELD_BLOCKS;
    } else if (type == RKC_EV_CLAIM) {
      if (nslot >= (u32)n_slots) {
        invalid = true;
        status |= RKC_PS_SLOT_TABLE;
      } else {
        u32 s = nslot++;
        bool bad = w1 < 1 || w1 > RKC_MAX_FIELD_BLOCKS || w2 < 0 || w2 >= n_chains || w3 < 0 || w3 > w1;
        if (bad) invalid = true;
        else if (ncl >= (u32)max_claims) { invalid = true; status |= RKC_PS_CLAIM_TABLE; }
        // (chain, L) of a valid claim for its final lead_end; invalid claims report 0
        slot_cl[s] = invalid ? make_uint2(NIL, 0) : make_uint2((u32)w2, (u32)w1);
        if (invalid) write_record(s, (i32)t, 0, -1, -1, -1, -1, -1, -1, 0);
      }
    } else if (type > RKC_EV_NOP) {
      invalid = true;
    }

    if (invalid) {
      code = RKC_OC_INVALID;
    } else if (type == RKC_EV_PREFILL) {
      const i32 S = w1, P = w3;
      const i32 hc = P > 0 ? w2 : -1;
      const u32 h = hc >= 0 ? min((u32)P, n[hc]) : 0u;
      const i32 need = S - (i32)h;
      const i32 Hc = hc >= 0 ? max(0, (i32)h - (i32)hold[hc]) : 0;
      AllocRes r = alloc(need, hc, h, any_sweep);
      if (!r.ok) {
        refusal(need, hc, h, Hc, code, id, a, b, n16);
      } else {
        A += Hc + need;
        u32 R = 0;
        if (hc >= 0) {
          const u32 c = (u32)hc;
          R = mode == RKC_MODE_NOADMIT ? h : (u32)P;
          const u32 nn = (mode != RKC_MODE_NOADMIT && (u32)P > n[c]) ? (u32)P : n[c];
          chain_update(c, nn, max(hold[c], R), prot[c]);
          touch(c, R, t);
          refresh(c);
        }
        const u32 k = nreq++;
        rq_id[k] = t; rq_c[k] = hc >= 0 ? (u32)hc : NIL; rq_R[k] = R; rq_len[k] = (u32)S;
        code = r.resident > 0 ? RKC_OC_EVICT_RESIDENT : RKC_OC_ADMIT;
        id = (i32)t; a = r.resident; b = (i32)h;
        if (r.post) flags |= RKC_FL_POST_RELEASE_LOSS;
        if (r.unclaimed) flags |= RKC_FL_EVICT_UNCLAIMED;
        tel[10] += r.victims; tel[11] += r.resident; tel[12] += r.post; tel[14] += h;
      }
    } else if (type == RKC_EV_EXTEND) {
      if (nreq == 0) {
        code = RKC_OC_NOOP;
      } else {
        const u32 i = (u32)w2 % nreq;
        const i32 need = w1;
        AllocRes r = alloc(need, -1, 0, any_sweep);
        if (!r.ok) {
          refusal(need, -1, 0, 0, code, id, a, b, n16);
        } else {
          A += need;
          rq_len[i] += (u32)need;
          code = r.resident > 0 ? RKC_OC_EVICT_RESIDENT : RKC_OC_ADMIT;
          id = (i32)rq_id[i]; a = r.resident; b = A;
          if (r.post) flags |= RKC_FL_POST_RELEASE_LOSS;
          if (r.unclaimed) flags |= RKC_FL_EVICT_UNCLAIMED;
          tel[10] += r.victims; tel[11] += r.resident; tel[12] += r.post;
        }
      }
    } else if (type == RKC_EV_CLAIM) {
      const i32 L = w1, T = w3;
      const u32 c = (u32)w2, s = nslot - 1;
      const u32 eff = mode == RKC_MODE_HARD ? (hardq ? RKC_PROT_HARD : RKC_PROT_SOFT)
                    : mode == RKC_MODE_SOFT ? RKC_PROT_SOFT : RKC_PROT_NONE;
      const u32 h = min((u32)L, n[c]);
      const i32 need = L - (i32)h;
      AllocRes r = alloc(need, (i32)c, h, any_sweep);
      u32 dec;
      if (!r.ok) {
        dec = (mode == RKC_MODE_LRU || mode == RKC_MODE_NOADMIT) ? DEC_SHADOW : DEC_REJECTED;
        u32 m = ST_REJECTED | (eff << 3) | (hardq << 5) | (prio << 6) | (dec << 9);
        write_record(s, (i32)t, packed_of(m), -1, -1, -1, -1, -1, -1, 0);
        code = RKC_OC_MATFAIL; id = (i32)t; a = need; b = F + r.E;
      } else {
        if ((u32)L > n[c]) chain_update(c, (u32)L, hold[c], prot[c]);
        touch(c, (u32)L, t);
        u32 st;
        if (mode == RKC_MODE_LRU || mode == RKC_MODE_NOADMIT) {
          dec = DEC_SHADOW; st = ST_OBSERVED; flags |= RKC_FL_SHADOW;
        } else if (mode == RKC_MODE_SOFT && hardq) {
          dec = DEC_APPROX; st = ST_MATERIALIZED; flags |= RKC_FL_LOWERED;
        } else {
          dec = DEC_ACCEPTED; st = ST_MATERIALIZED;
        }
        const u32 m = st | (eff << 3) | (hardq << 5) | (prio << 6) | (1u << 8) | (dec << 9);
        const u32 k = ncl++;
        const u32 ex = (dur > 0 && st == ST_MATERIALIZED) ? t + dur : EXP_NEVER;
        cl_id[k] = t; cl_c[k] = c; cl_L[k] = (u32)L; cl_T[k] = (u32)T; cl_meta[k] = m;
        cl_exp[k] = ex; cl_slot[k] = s; cl_blk[k] = 0;
        cl_dem[k] = NIL; cl_exst[k] = NIL; cl_pf[k] = NIL; cl_harm[k] = NIL;
        // a new live claim only raises the chain's maxima
        covA[c] = max(covA[c], (u32)L);
        covS[c] = max(covS[c], (u32)L);
        tpend[c] = max(tpend[c], (u32)T);
        if (mode == RKC_MODE_HARD && st == ST_MATERIALIZED && eff == RKC_PROT_HARD)
          chain_update(c, n[c], hold[c], max(prot[c], (u32)L));
        if (soft_levels() && st == ST_MATERIALIZED && eff == RKC_PROT_SOFT)
          lv[4 * c + prio] = max(lv[4 * c + prio], (u32)L);
        refresh(c);
        next_exp = min(next_exp, ex);
        code = r.resident > 0 ? RKC_OC_EVICT_RESIDENT : RKC_OC_ADMIT;
        id = (i32)t; a = r.resident; b = need;
        if (r.post) flags |= RKC_FL_POST_RELEASE_LOSS;
        if (r.unclaimed) flags |= RKC_FL_EVICT_UNCLAIMED;
        tel[10] += r.victims; tel[11] += r.resident; tel[12] += r.post;
      }
      tel[dec == DEC_ACCEPTED ? 15 : dec == DEC_APPROX ? 16 : dec == DEC_SHADOW ? 17 : 18] += 1;
    } else if (type == RKC_EV_FINISH) {
      if (nreq == 0) {
        code = RKC_OC_NOOP;
      } else {
        const u32 i = (u32)w1 % nreq;
        const u32 rid = rq_id[i], c = rq_c[i], R = rq_R[i], len = rq_len[i];
        list_remove(rq_id, rq_cap, 4, nreq, i);
        nreq--;
        i32 turned = 0, dropped = 0;
        if (c != NIL) {
          u32 hn = 0;
          for (u32 j = lane; j < nreq; j += 64)
            if (rq_c[j] == c) hn = max(hn, rq_R[j]);
          hn = wave_max(hn);
          turned += max(0, (i32)R - (i32)hn);
          chain_update(c, n[c], hn, prot[c]);
          touch(c, R, t);
          refresh(c);
        }
        // write no-admit drops the request's own blocks; otherwise they become a private run
        const i32 own = (i32)(len - R);
        const bool drop = mode == RKC_MODE_NOADMIT;
        dropped = drop ? own : 0;
        turned += drop ? 0 : own;
        F += dropped;
        fblocks += drop ? 0 : own;
        if (!drop && own > 0) {
          if (fhead == ftail) { ft = t; flo = R; ftop = len; }
          fifo[ftail % fifo_cap] = make_uint4(t, R, len, 0);
          ftail++;
        }
        A -= turned + dropped;
        code = RKC_OC_FINISHED; id = (i32)rid; a = turned; b = dropped;
        if (dropped) flags |= RKC_FL_NOADMIT_DROP;
        tel[13] += dropped;
      }
    } else if (type == RKC_EV_RELEASE) {
      if (ncl == 0) {
        code = RKC_OC_NOOP;
      } else {
        const u32 i = (u32)w1 % ncl;
        const u32 qid = cl_id[i], c = cl_c[i], L = cl_L[i], T = cl_T[i];
        write_live_record(i, ST_RELEASED, (i32)t);
        __builtin_amdgcn_wave_barrier();
        claim_remove(i);
        recompute(c);
        code = RKC_OC_RELEASED; id = (i32)qid; a = (i32)min(n[c], L); b = (i32)T;
        tel[23] += 1;
      }
    } else if (type == RKC_EV_DEMOTE) {
      u32 cnt = 0;
      const bool ok_mode = soft_levels();
      if (ok_mode)
        for (u32 base = 0; base < ncl; base += 64) {
          u32 j = base + lane;
          bool cand = j < ncl && m_state(cl_meta[j]) == ST_MATERIALIZED && m_hard(cl_meta[j]);
          cnt += (u32)__builtin_popcountll(ballot(cand));
        }
      if (cnt == 0) {
        code = RKC_OC_NOOP;
      } else {
        u32 k = (u32)w1 % cnt, pick = NIL;
        for (u32 base = 0; base < ncl && pick == NIL; base += 64) {
          u32 j = base + lane;
          bool cand = j < ncl && m_state(cl_meta[j]) == ST_MATERIALIZED && m_hard(cl_meta[j]);
          u64 bl = ballot(cand);
          u32 pc = (u32)__builtin_popcountll(bl);
          if (k < pc) {
            u64 x = bl;
            for (u32 q = 0; q < k; q++) x &= x - 1;
            pick = base + (u32)__builtin_ctzll(x);
          } else {
            k -= pc;
          }
        }
        const u32 i = pick, c = cl_c[i];
        cl_meta[i] = m_with_state(cl_meta[i], ST_DEMOTED);
        cl_dem[i] = t;
        __builtin_amdgcn_wave_barrier();
        recompute(c);
        code = RKC_OC_DEMOTED; id = (i32)cl_id[i]; a = (i32)min(n[c], cl_L[i]); b = (i32)cl_T[i];
        tel[22] += 1;
      }
    } else {
      code = RKC_OC_NOOP;
    }

    if (!invalid && any_sweep) {
      __builtin_amdgcn_wave_barrier();
      flags |= sweep(t);
    }
    if (code == RKC_OC_NOOP || code == RKC_OC_INVALID) { id = -1; a = 0; b = 0; }
    if (n16 == NIL) n16 = min(expired, 65535u);
    tel[code] += 1;
    peak = max(peak, A);
    return make_int4((i32)((u32)code | (flags << 8) | (n16 << 16)), id, a, b);
  }
};

template <bool kGL>
__global__ __launch_bounds__(64) void rkc_replay_wave(Args g) {
  extern __shared__ __align__(16) unsigned char lds[];
  const u32 pool = blockIdx.x;
  if ((i32)pool >= g.n_pools) return;
  const Layout& L = g.L;
  Pool<kGL> P;
  P.lane = lane_id();
  const rkc_pool_desc d = g.pools[pool];
  P.U = d.usable_blocks; P.mode = d.mode; P.n_events = d.n_events; P.n_chains = d.n_chains;
  P.max_claims = d.max_live_claims; P.max_reqs = d.max_live_requests; P.n_slots = d.n_claim_slots;
  P.ev_off = d.event_offset; P.slot_off = d.claim_slot_offset;
  rkc_pool_telemetry* ptel = g.pool_tel + pool;

  // Descriptor checks against the batch limits the launch was sized for.
  const bool ev_ok = P.n_events >= 0 && P.ev_off >= 0 && P.ev_off + P.n_events <= g.n_events_total;
  const bool sl_ok = P.n_slots >= 0 && P.slot_off >= 0 && P.slot_off + P.n_slots <= g.n_slots_total;
  const bool ok = ev_ok && sl_ok && P.U >= 1 && P.U <= g.max_usable && P.U <= RKC_MAX_USABLE_BLOCKS &&
                  P.mode >= 0 && P.mode <= 3 && P.n_events <= g.max_events && P.n_chains >= 0 &&
                  P.n_chains <= g.max_chains && P.max_claims >= 0 && P.max_claims <= g.max_claims &&
                  P.max_reqs >= 0 && P.max_reqs <= g.max_reqs && P.n_slots <= g.max_slots &&
                  d.reserved == 0;
  if (!ok) {
    if (ev_ok)
      for (i32 i = (i32)P.lane; i < P.n_events; i += 64)
        g.outcomes[P.ev_off + i] = rkc_outcome{{RKC_OC_INVALID, -1, 0, 0}};
    if (sl_ok)
      for (i32 i = (i32)P.lane; i < P.n_slots; i += 64)
        g.claim_tel[P.slot_off + i] = rkc_claim_telemetry{{-1, 0, -1, -1, -1, -1, -1, -1, 0, 0}};
    if (P.lane < 32)
      ptel->w[P.lane] = P.lane == 31 ? RKC_PS_DESCRIPTOR : (P.lane == RKC_OC_INVALID && ev_ok) ? P.n_events : 0;
    return;
  }

  // LDS carve-up
  P.n = (u32*)(lds + L.off_n); P.hold = (u32*)(lds + L.off_hold); P.prot = (u32*)(lds + L.off_prot);
  P.covA = (u32*)(lds + L.off_covA); P.covS = (u32*)(lds + L.off_covS);
  P.tpend = (u32*)(lds + L.off_tpend); P.lv = (u32*)(lds + L.off_lv);
  P.stop = (u32*)(lds + L.off_stop); P.sbot = (u32*)(lds + L.off_sbot);
  P.mark = (u32*)(lds + L.off_mark); P.topkey = (u64*)(lds + L.off_key);
  P.bt = (u32*)(lds + L.off_bt); P.nx = (u32*)(lds + L.off_nx);
  P.tel = (u32*)(lds + L.off_tel);
  unsigned char* scr = g.scratch + (u64)pool * L.scr_pool_bytes;
  u32* rq = kGL ? (u32*)(scr + L.scr_off_rq) : (u32*)(lds + L.off_rq);
  P.rq_cap = L.reqs;
  P.rq_id = rq; P.rq_c = rq + L.reqs; P.rq_R = rq + 2 * L.reqs; P.rq_len = rq + 3 * L.reqs;
  u32* cl = kGL ? (u32*)(scr + L.scr_off_cl) : (u32*)(lds + L.off_cl);
  P.cl_cap = L.claims;
  P.cl_id = cl; P.cl_c = cl + L.claims; P.cl_L = cl + 2 * L.claims; P.cl_T = cl + 3 * L.claims;
  P.cl_meta = cl + 4 * L.claims; P.cl_exp = cl + 5 * L.claims; P.cl_slot = cl + 6 * L.claims;
  P.cl_blk = cl + 7 * L.claims; P.cl_dem = cl + 8 * L.claims; P.cl_exst = cl + 9 * L.claims;
  P.cl_pf = cl + 10 * L.claims; P.cl_harm = cl + 11 * L.claims;
  P.node_cap = L.node_cap;
  P.node_lds = (lds_uint4*)(lds + L.off_node);
  P.nl = L.nodes_lds;
  P.node_glb = (glb_uint4*)(scr + L.scr_off_node);
  P.fifo = (uint4*)(scr + L.scr_off_fifo);
  P.fifo_cap = L.fifo_cap;
  P.slot_cl = (uint2*)(scr + L.scr_off_slot);
  P.rec = g.claim_tel + P.slot_off;

  for (i32 c = (i32)P.lane; c < P.n_chains; c += 64) {
    P.n[c] = 0; P.hold[c] = 0; P.prot[c] = 0; P.covA[c] = 0; P.covS[c] = 0; P.tpend[c] = 0;
    P.lv[4 * c] = 0; P.lv[4 * c + 1] = 0; P.lv[4 * c + 2] = 0; P.lv[4 * c + 3] = 0;
    P.stop[c] = NIL; P.sbot[c] = NIL; P.mark[c] = 0; P.bt[c] = 0; P.nx[c] = 0;
    if ((u32)c >= kRegChains) P.topkey[c] = KEY_INF;
  }
  P.kr0 = P.kr1 = P.kr2 = P.kr3 = KEY_INF;
  if (P.lane < 32) P.tel[P.lane] = 0;
  P.F = P.U; P.A = 0; P.PR = 0; P.peak = 0; P.Eall = 0;
  P.nreq = 0; P.ncl = 0; P.nslot = 0; P.next_exp = EXP_NEVER;
  P.free_head = NIL; P.bump = 0;
  P.fhead = 0; P.ftail = 0; P.ft = 0; P.flo = 0; P.ftop = 0; P.fblocks = 0;
  P.status = 0;
  __syncthreads();

  const rkc_event* ev = g.events + P.ev_off;
  rkc_outcome* out = g.outcomes + P.ev_off;
  for (i32 base = 0; base < P.n_events; base += 64) {
    const i32 cnt = min(64, P.n_events - base);
    int4 e = make_int4(0, 0, 0, 0);
    if ((i32)P.lane < cnt) {
      const rkc_event x = ev[base + P.lane];
      e = make_int4(x.w[0], x.w[1], x.w[2], x.w[3]);
    }
    int4 mine = make_int4(0, 0, 0, 0);
    for (i32 k = 0; k < cnt; k++) {
      const int4 o = P.step((u32)(base + k), rdlane(e.x, (u32)k), rdlane(e.y, (u32)k),
                            rdlane(e.z, (u32)k), rdlane(e.w, (u32)k));
      if ((i32)P.lane == k) mine = o;
    }
    if ((i32)P.lane < cnt) out[base + P.lane] = rkc_outcome{{mine.x, mine.y, mine.z, mine.w}};
  }

  // Final claim records of the claims still live ...
  for (u32 i = 0; i < P.ncl; i++) P.write_live_record(i, m_state(P.cl_meta[i]), -1);
  // ... then lead_end = min(final leading registered length, L) for every used slot, and blank
  // records for unused slots.
  __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "workgroup");
  for (i32 s = (i32)P.lane; s < P.n_slots; s += 64) {
    if (s < (i32)P.nslot) {
      const uint2 cl2 = P.slot_cl[s];
      P.rec[s].w[9] = cl2.x == NIL ? 0 : (i32)min(P.n[cl2.x], cl2.y);
    } else {
      P.rec[s] = rkc_claim_telemetry{{-1, 0, -1, -1, -1, -1, -1, -1, 0, 0}};
    }
  }
  __builtin_amdgcn_wave_barrier();
  if (P.lane < 32) {
    const u32 w = P.lane;
    i32 v = (i32)P.tel[w];
    if (w == 24) v = P.peak;
    else if (w == 25) v = P.A;
    else if (w == 26) v = P.U - P.F - P.A;
    else if (w == 27) v = P.F;
    else if (w == 28) v = P.PR;
    else if (w == 29) v = (i32)P.nreq;
    else if (w == 30) v = (i32)P.ncl;
    else if (w == 31) v = (i32)P.status;
    ptel->w[w] = v;
  }
}

// ---- host side -----------------------------------------------------------------------------
u64 align_up(u64 v, u64 a) { return (v + a - 1) / a * a; }

constexpr u32 kNodesLds = 64;

constexpr u64 kLdsBudget = 160 * 1024;

bool make_layout(const rkc_batch* b, Layout* L, bool global_lists) {
  memset(L, 0, sizeof *L);
  L->global_lists = global_lists;
  L->chains = (u32)(b->max_chains > 0 ? b->max_chains : 1);
  L->reqs = (u32)(b->max_live_requests > 0 ? b->max_live_requests : 1);
  L->claims = (u32)(b->max_live_claims > 0 ? b->max_live_claims : 1);
  L->node_cap = (u32)b->max_events + 2;
  L->nodes_lds = L->node_cap < kNodesLds ? L->node_cap : kNodesLds;
  u64 o = 0;
  auto take = [&](u64 bytes, u64 al) { o = align_up(o, al); u64 r = o; o += bytes; return (u32)r; };
  const u64 C = L->chains;
  L->off_key = take(8 * (C > kRegChains ? C - 0 : 1), 16);
  L->off_n = take(4 * C, 4); L->off_hold = take(4 * C, 4); L->off_prot = take(4 * C, 4);
  L->off_covA = take(4 * C, 4); L->off_covS = take(4 * C, 4); L->off_tpend = take(4 * C, 4);
  L->off_lv = take(16 * C, 16); L->off_stop = take(4 * C, 4); L->off_sbot = take(4 * C, 4);
  L->off_mark = take(4 * C, 4); L->off_tel = take(128, 16);
  L->off_bt = take(4 * C, 4); L->off_nx = take(4 * C, 4);
  if (!global_lists) {
    L->off_rq = take(16ull * L->reqs, 16);
    L->off_cl = take(48ull * L->claims, 16);
  }
  L->off_node = take(16ull * L->nodes_lds, 16);
  o = align_up(o, 16);
  if (o > kLdsBudget) return false;
  L->lds_bytes = (u32)o;
  // scratch per pool: spilled nodes, FIFO ring, slot table
  L->fifo_cap = (u32)b->max_events + 1;
  u64 s = 0;
  L->scr_off_node = s; s += 16ull * (L->node_cap - L->nodes_lds); s = align_up(s, 256);
  L->scr_off_fifo = s; s += 16ull * L->fifo_cap; s = align_up(s, 256);
  L->scr_off_slot = s; s += 8ull * (u64)(b->max_claim_slots > 0 ? b->max_claim_slots : 1);
  s = align_up(s, 256);
  if (global_lists) {
    L->scr_off_rq = s; s += 16ull * L->reqs; s = align_up(s, 256);
    L->scr_off_cl = s; s += 48ull * L->claims;
  }
  L->scr_pool_bytes = align_up(s, 256);
  return true;
}

// Lists in LDS when the whole pool state fits, else in global scratch.
bool choose_layout(const rkc_batch* b, Layout* L) {
  return make_layout(b, L, false) || make_layout(b, L, true);
}

rkc_status check_batch(const rkc_batch* b) {
  if (!b) return RKC_E_NULL;
  if (b->n_pools < 0 || b->max_usable_blocks < 0 || b->max_events < 0 || b->max_chains < 0 ||
      b->max_live_requests < 0 || b->max_live_claims < 0 || b->max_claim_slots < 0 ||
      b->n_events_total < 0 || b->n_claim_slots_total < 0 || b->flags != 0)
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

}  // namespace

extern "C" {

int32_t rkc_abi_version(void) { return RKC_ABI_VERSION; }

size_t rkc_scratch_bytes(const rkc_batch* b) {
  if (!b || b->n_pools <= 0) return 0;
  Layout L;
  if (!choose_layout(b, &L)) return 0;
  return (size_t)(L.scr_pool_bytes * (u64)b->n_pools);
}

rkc_status rkc_replay_batch(const rkc_batch* b, void* s) {
  rkc_status st = check_batch(b);
  if (st != RKC_OK) return st;
  if (b->n_pools == 0) return RKC_OK;
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
  const void* fn = g.L.global_lists ? (const void*)rkc_replay_wave<true> : (const void*)rkc_replay_wave<false>;
  if (g.L.lds_bytes > 64 * 1024) {
    if (hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)g.L.lds_bytes) != hipSuccess)
      return RKC_E_HIP;
  }
  if (g.L.global_lists)
    hipLaunchKernelGGL(rkc_replay_wave<true>, dim3((unsigned)b->n_pools), dim3(64), g.L.lds_bytes,
                       (hipStream_t)s, g);
  else
    hipLaunchKernelGGL(rkc_replay_wave<false>, dim3((unsigned)b->n_pools), dim3(64), g.L.lds_bytes,
                       (hipStream_t)s, g);
  if (hipGetLastError() != hipSuccess) return RKC_E_HIP;
  return RKC_OK;
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
    if (k > 0 && hipMemcpy(host_claims, b->d_claim_tel + d.claim_slot_offset,
                           (size_t)k * sizeof(rkc_claim_telemetry), hipMemcpyDeviceToHost) != hipSuccess)
      return RKC_E_HIP;
  }
  return pool_status(b, pool, RKC_OK);
}

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
  }
  return "unknown status";
}

}  // extern "C"
