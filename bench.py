"""Benchmark: replayed allocator events/s of the batched resident-claim replay on one MI355X.

A step is one launch that replays every pool of the workload from empty pools through every event
(expiry, validation, feasibility, victim selection, commit, lifecycle, predicate sweep, outcome and
telemetry emission).  Inputs are resident in HBM before timing starts; outputs are fully
overwritten by every launch, so repeated steps are identical.

Default workload: 65,536 pools x 2,048 usable blocks x 1,024 events (prefixes shared through 256
Zipf(1.1) chains per pool), i.e. 67,108,864 events per step.

Prints one JSON line (rank 0).  Also:
  --mode copy   runs only a plain device copy of known size (calibrates rocprofv3 byte counters and
                gives the measured copy ceiling).
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0  # MI355X HBM3E, AMD published peak
# Algorithmic bytes of the hot-path scope: 16 B per event read, 16 B per outcome written, 40 B per
# claim record written, 128 B of pool telemetry written and a 48 B descriptor read per pool.  (The
# ABI's pool telemetry record is 256 B and its descriptor 64 B; those are reported beside, never
# credited.)
BYTES_EVENT, BYTES_OUTCOME, BYTES_CLAIM_SLOT, BYTES_POOL_TEL, BYTES_DESC = 16, 16, 40, 128, 48
ABI_POOL_TEL, ABI_DESC = 256, 64
COPY_BYTES = 1 << 30
METRIC = "replayed allocator events/sec (1 GPU) + % of HBM peak; bit-exact vs oracle"


def credited_bytes(trace, pool_tel=BYTES_POOL_TEL, desc=BYTES_DESC) -> int:
    """Algorithmic bytes of one replay launch: events in, outcomes out, claim slots out, pool
    telemetry out, descriptors in.  Scratch, LDS traffic and re-reads are not credited."""
    return (trace.n_events * (BYTES_EVENT + BYTES_OUTCOME) + trace.n_claim_slots * BYTES_CLAIM_SLOT
            + trace.n_pools * (pool_tel + desc))


def copy_ceiling(torch, reps=20):
    n = COPY_BYTES // 4
    a = torch.empty(n, dtype=torch.int32, device="cuda").fill_(1)
    b = torch.empty_like(a)
    for _ in range(3):
        b.copy_(a)
    s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    s.record()
    for _ in range(reps):
        b.copy_(a)
    e.record()
    torch.cuda.synchronize()
    ms = s.elapsed_time(e) / reps
    return 2.0 * COPY_BYTES / (ms * 1e-3) / 1e9


# The per-block oracle spends O(usable blocks) per event; pools bigger than this many
# (blocks x events) are sampled by their leading events (replay is causal).
ORACLE_POOL_WORK = 2e8


def oracle_prefix(trace):
    """Events per pool the oracle replays in a bounded sample (all of them for small pools)."""
    lim = trace.limits()
    per_event = max(1, lim["max_usable_blocks"])
    if lim["max_events"] * per_event <= ORACLE_POOL_WORK:
        return lim["max_events"]
    return max(256, int(ORACLE_POOL_WORK // per_event))


def _oracle_rate(trace, threads, seconds_budget):
    """Events/s of the oracle over the leading pools of the workload (for very large pools, their
    leading events), in chunks until the wall budget is spent."""
    import oracle
    pre = oracle_prefix(trace)
    done_pools, done_events = 0, 0
    t0 = time.perf_counter()
    chunk = threads * 8 if pre >= trace.limits()["max_events"] else threads
    while done_pools < trace.n_pools and time.perf_counter() - t0 < seconds_budget:
        pools = list(range(done_pools, min(trace.n_pools, done_pools + chunk)))
        sub = trace.prefix(pools, pre)
        oracle.replay(sub.desc, sub.events, sub.n_claim_slots, threads=threads)
        done_pools += len(pools)
        done_events += sub.n_events
    wall = time.perf_counter() - t0
    what = "" if pre >= trace.limits()["max_events"] else f" (first {pre} events of each)"
    return done_events / wall, (f"first {done_pools} pools of the workload{what}, {done_events} events, "
                                f"{threads} thread{'s' if threads > 1 else ''}, {wall:.1f} s wall")


def cpu_model() -> str:
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(trace, seconds_budget=12.0, single_budget=4.0):
    """The oracle as it stands, on the host's cores, over a bounded sample of the same workload
    (up to 16 worker threads, each pool single-threaded), and the same oracle on one core."""
    threads = max(1, min(16, os.cpu_count() or 1))
    rate, sample = _oracle_rate(trace, threads, seconds_budget)
    rate1, sample1 = _oracle_rate(trace, 1, single_budget)
    return dict(value=rate, unit="events/s", cores=threads, kind="oracle", sample=sample,
                host_cpus=os.cpu_count(), cpu_model=cpu_model(),
                single_core=dict(value=rate1, unit="events/s", cores=1, sample=sample1))


def profile_record(kernel, workload, kernel_sha):
    """The committed rocprofv3 counter summary of this kernel and workload (HBM bytes and scalar
    instructions per launch), if it was taken on the current kernel sources; else {}."""
    path = os.path.join(ROOT, "profiles", f"{kernel}_{workload}_traffic.json")
    if not os.path.exists(path):
        return {}
    d = json.load(open(path))
    if d.get("kernel_source_sha256") != kernel_sha:
        return {}
    return d


# Scalar issue ceiling: one scalar instruction per CU per cycle, 256 CUs at the 2.4 GHz peak
# engine clock, in G instructions/s.
SCALAR_ISSUE_PEAK = 256 * 2.4


def kernel_name(lim):
    """Which replay kernel the library picks for these batch limits (the compact one when every
    limit fits its 16-bit encoding: up to 64 live claims on up to 256 chains, or up to 256 live
    claims on up to 64 chains)."""
    claims_ok = (lim["max_live_claims"] <= 64 and lim["max_chains"] <= 256) or \
                (lim["max_live_claims"] <= 256 and lim["max_chains"] <= 64)
    fits = (lim["max_usable_blocks"] <= 32767 and lim["max_events"] <= 65533 and claims_ok
            and lim["max_live_requests"] <= 256 and lim["max_claim_slots"] <= 65534)
    return "rkc_lean" if fits else "rkc_replay_wave"


def parallelism(trace, kernel):
    """How pools map to the GPU for this batch (mirrors the library's launch choice)."""
    if kernel == "rkc_lean":
        return "one wavefront per pool"
    lim = trace.limits()
    # the general kernel keeps the live lists in LDS when they fit beside the chain records
    lists_on_chip = (lim["max_live_requests"] * 16 + lim["max_live_claims"] * 32
                     + max(1, lim["max_chains"]) * 72) <= 159 * 1024
    if not lists_on_chip and trace.n_pools <= 256:
        return "one workgroup of 8 wavefronts per pool"
    return "one wavefront per pool"


KERNEL_SOURCES = {
    "rkc_lean": ("paper_2605_24259_amd/csrc/rkc_lean.hip", "paper_2605_24259_amd/csrc/rkc_lean.h",
                 "include/rkc.h", "paper_2605_24259_amd/build.py"),
    "rkc_replay_wave": ("paper_2605_24259_amd/csrc/rkc_replay.hip", "include/rkc.h",
                        "paper_2605_24259_amd/build.py"),
}


def kernel_source_sha(kernel="rkc_lean"):
    """SHA-256 over the sources that define one replay kernel and its launch, and the build script
    that holds its compiler flags (the counters describe the build of those sources)."""
    import hashlib
    h = hashlib.sha256()
    for f in KERNEL_SOURCES[kernel]:
        h.update(open(os.path.join(ROOT, f), "rb").read())
    return h.hexdigest()


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--workload", default="zipf", choices=["small", "zipf", "nested", "huge", "sweep", "zipf_defer", "zipf_relax", "zipf_offload"])
    ap.add_argument("--mode", default="replay", choices=["replay", "copy"])
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-parity", action="store_true")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py: the replay runs on one GPU only (pools are independent; a multi-GPU "
              "run would split the pool range across ranks, which is not implemented)", flush=True)
        sys.exit(2)

    import numpy as np
    import torch

    if args.mode == "copy":
        gbps = copy_ceiling(torch, reps=args.steps)
        print(json.dumps(dict(mode="copy", bytes_per_copy=2 * COPY_BYTES, gbps=round(gbps, 1))), flush=True)
        return

    import paper_2605_24259_amd as rkc
    from paper_2605_24259_amd import tracegen as tg

    trace = tg.generate(args.workload)
    db = rkc.DeviceBatch.from_trace(trace)
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    for _ in range(args.warmup):
        db.replay(stream)
    torch.cuda.synchronize()
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    start.record(stream)
    for _ in range(args.steps):
        db.replay(stream)
    end.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms_per_step = start.elapsed_time(end) / args.steps
    events = trace.n_events
    value = events / (ms_per_step * 1e-3)
    cbytes = credited_bytes(trace)
    cbytes_abi = credited_bytes(trace, ABI_POOL_TEL, ABI_DESC)
    achieved = cbytes / (ms_per_step * 1e-3) / 1e9

    parity = None
    if not args.no_parity:
        import oracle
        out, ptel, ctel = db.results()
        pools = sorted(set(int(i) for i in np.linspace(0, trace.n_pools - 1, 16).astype(int)))
        pre = oracle_prefix(trace)
        whole = pre >= trace.limits()["max_events"]
        sub = trace.prefix(pools, pre)
        o_out, o_pt, o_ct, chk = oracle.replay(sub.desc, sub.events, sub.n_claim_slots, threads=16)
        eo, ne, so, ns = (trace.field(k) for k in ("event_offset", "n_events", "claim_slot_offset",
                                                    "n_claim_slots"))
        eo2, ne2, so2 = sub.field("event_offset"), sub.field("n_events"), sub.field("claim_slot_offset")
        ok = not chk.any()
        for j, p in enumerate(pools):
            k = int(ne2[j])
            ok &= np.array_equal(out[eo[p]: eo[p] + k], o_out[eo2[j]: eo2[j] + k])
            if whole:
                ok &= np.array_equal(ptel[p], o_pt[j])
                ok &= np.array_equal(ctel[so[p]: so[p] + ns[p]], o_ct[so2[j]: so2[j] + ns[p]])
        what = "" if whole else f" (their first {pre} outcomes)"
        parity = f"{'bit-exact' if ok else 'MISMATCH'} vs oracle on {len(pools)} sampled pools{what}"

    ceiling = copy_ceiling(torch)
    base = None if args.no_cpu_baseline else cpu_baseline(trace)
    lim = trace.limits()
    prof = profile_record(kernel_name(lim), args.workload, kernel_source_sha(kernel_name(lim)))
    salu = prof.get("sq_insts_salu_per_launch")
    line = {
        "metric": METRIC,
        "value": round(value, 1),
        "unit": "events/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "int32",
        "data": "synthetic",
        "config": {
            "workload": f"{args.workload}: {trace.n_pools} pools x {lim['max_usable_blocks']} usable "
                        f"blocks x {lim['max_events']} events",
            "pools": trace.n_pools, "usable_blocks": lim["max_usable_blocks"],
            "events_per_pool": lim["max_events"], "events_per_step": events,
            "claim_slots": trace.n_claim_slots, "parallelism": parallelism(trace, kernel_name(lim)),
            "kernel": kernel_name(lim),
        },
        "roofline": {
            "bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBPS, "unit": "GB/s",
            "frac": round(achieved / HBM_PEAK_GBPS, 4),
            "traffic": prof.get("traffic_bytes_per_launch"),
            "credited_bytes_per_launch": cbytes,
            # the same count with the ABI's 256-B telemetry record and 64-B descriptor per pool
            "abi_record_bytes_per_launch": cbytes_abi,
            "copy_ceiling_gbps": round(ceiling, 1),
            "frac_of_copy_ceiling": round(achieved / ceiling, 4),
            # what actually bounds the replay: the scalar instructions the counters saw per launch
            # over this launch time, against the scalar issue ceiling
            "scalar_issue": None if salu is None else {
                "achieved": round(salu / (ms_per_step * 1e-3) / 1e9, 1), "peak": SCALAR_ISSUE_PEAK,
                "unit": "G scalar instr/s", "frac": round(salu / (ms_per_step * 1e-3) / 1e9 / SCALAR_ISSUE_PEAK, 4)},
        },
        "cpu_baseline": base,
        "parity": parity,
        "wall_s": round(wall, 3),
    }
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
