// rkc_lean.h -- internal interface between the C ABI (rkc_replay.hip) and the compact replay
// kernel (rkc_lean.hip).  Not part of the public ABI.
#ifndef RKC_LEAN_H
#define RKC_LEAN_H

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "rkc.h"

struct rkc_lean_args {
  const rkc_pool_desc* pools;
  const rkc_event* events;
  rkc_outcome* outcomes;
  rkc_pool_telemetry* pool_tel;
  rkc_claim_telemetry* claim_tel;
  void* scratch;
  int64_t n_events_total, n_slots_total;
  int32_t n_pools, max_usable, max_events, max_chains, max_reqs, max_claims, max_slots;
  // layout: LDS byte offsets, node split, per-pool scratch regions
  uint32_t ns, nq, node_cap, nodes_lds;  // 64-chain key groups, 64-claim sets, node split
  uint32_t lds_bytes;  // LDS per pool (its regions sit at offsets fixed per kernel instantiation)
  uint64_t scr_pool_bytes, scr_off_nodes, scr_off_fifo, scr_off_slots, scr_off_defer, scr_off_reqs;
  // after the per-pool regions: the launch order (one u32 pool index per workgroup), each pool's
  // loop class (one byte) and per-tile class counts of the ordering passes
  uint64_t scr_off_order, scr_off_cls, scr_off_tiles, scr_total;
};

// Fill the layout part of g for batch b; false when b is outside the compact kernel's limits
// (usable blocks <= 32,767, events <= 65,533, live requests <= 256, and live claims <= 64 with
// chains <= 256 or live claims <= 256 with chains <= 64).
bool rkc_lean_layout(const rkc_batch* b, rkc_lean_args* g);

// Launch the compact kernel (one 64-lane workgroup per pool) on stream s.
rkc_status rkc_lean_launch(const rkc_lean_args* g, hipStream_t s);

#ifdef RKC_CHECK_UNIFORM
// checking build only: calls of the compact kernel's readfirstlane whose active lanes disagreed
unsigned rkc_lean_uniform_violations(void);
#endif

#endif
