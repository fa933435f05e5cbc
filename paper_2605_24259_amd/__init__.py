"""Batched replay of resident-KV-claim arbitration on MI355X -- Python binding.

Thin ctypes marshalling over the C ABI in ``include/rkc.h`` (librkc.so, built for gfx950 by
``paper_2605_24259_amd.build``).  Every step of the replay runs in the HIP kernels; PyTorch only
provides device buffers and the current stream.  There is no CPU fallback: the functions here raise
when the library is not built or no GPU is present.
"""
from __future__ import annotations

import ctypes
import os

_PKG = os.path.dirname(os.path.abspath(__file__))
# RKC_LIBRARY may name another build of the same sources (the uniformity-checking build)
LIB_PATH = os.environ.get("RKC_LIBRARY") or os.path.join(_PKG, "librkc.so")
_lib = None

# layouts and codes of this binding (rkc.h RKC_ABI_VERSION)
ABI_VERSION = 5
POOL_TEL_WORDS = 64

# rkc_batch.flags: replay with the general kernel even where the compact one applies
FLAG_GENERAL_KERNEL = 1
# rkc_batch.flags: one wavefront per pool even where a workgroup per pool applies
FLAG_ONE_WAVE_PER_POOL = 2

# status codes (rkc_status)
STATUS = {0: "ok", -1: "null pointer", -2: "misaligned pointer", -3: "argument out of range",
          -4: "unsupported size or mode", -5: "scratch buffer missing or too small",
          -6: "HIP runtime error", -7: "pool status is non-zero",
          -8: "batch needs more scratch than the built-in buffer holds"}

# size of the built-in scratch of rkc_replay_batch_noalloc (RKC_NOALLOC_SCRATCH_BYTES)
NOALLOC_SCRATCH_BYTES = 64 << 20


class RkcError(RuntimeError):
    def __init__(self, status: int, what: str):
        super().__init__(f"{what}: {STATUS.get(status, status)} ({status})")
        self.status = status


class Batch(ctypes.Structure):
    """rkc_batch (include/rkc.h)."""
    _fields_ = [
        ("n_pools", ctypes.c_int32),
        ("max_usable_blocks", ctypes.c_int32),
        ("max_events", ctypes.c_int32),
        ("max_chains", ctypes.c_int32),
        ("max_live_requests", ctypes.c_int32),
        ("max_live_claims", ctypes.c_int32),
        ("max_claim_slots", ctypes.c_int32),
        ("flags", ctypes.c_int32),
        ("n_events_total", ctypes.c_int64),
        ("n_claim_slots_total", ctypes.c_int64),
        ("d_pools", ctypes.c_void_p),
        ("d_events", ctypes.c_void_p),
        ("d_outcomes", ctypes.c_void_p),
        ("d_pool_tel", ctypes.c_void_p),
        ("d_claim_tel", ctypes.c_void_p),
        ("d_scratch", ctypes.c_void_p),
        ("scratch_bytes", ctypes.c_size_t),
    ]


def load():
    """Load librkc.so (raises when it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is not built; run paper_2605_24259_amd.build.build()")
        lib = ctypes.CDLL(LIB_PATH)
        vp, i32 = ctypes.c_void_p, ctypes.c_int32
        bp = ctypes.POINTER(Batch)
        lib.rkc_abi_version.restype = i32
        lib.rkc_scratch_bytes.argtypes = [bp]
        lib.rkc_scratch_bytes.restype = ctypes.c_size_t
        lib.rkc_replay_batch.argtypes = [bp, vp]
        lib.rkc_replay_batch.restype = ctypes.c_int
        lib.rkc_replay_batch_noalloc.argtypes = [bp, vp]
        lib.rkc_replay_batch_noalloc.restype = ctypes.c_int
        lib.rkc_query_outcomes.argtypes = [bp, i32, i32, i32, vp, vp]
        lib.rkc_query_outcomes.restype = ctypes.c_int
        lib.rkc_query_telemetry.argtypes = [bp, i32, vp, vp, i32, ctypes.POINTER(i32), vp]
        lib.rkc_query_telemetry.restype = ctypes.c_int
        lib.rkc_status_string.argtypes = [ctypes.c_int]
        lib.rkc_status_string.restype = ctypes.c_char_p
        if lib.rkc_abi_version() != ABI_VERSION:
            raise RuntimeError(f"{LIB_PATH} implements ABI {lib.rkc_abi_version()}, this binding "
                               f"ABI {ABI_VERSION}; rebuild the library")
        _lib = lib
    return _lib


EXPORTS = ("rkc_abi_version", "rkc_scratch_bytes", "rkc_replay_batch", "rkc_replay_batch_noalloc",
           "rkc_query_outcomes", "rkc_query_telemetry", "rkc_status_string")


def _stream_ptr(stream):
    import torch
    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


class DeviceBatch:
    """Device-resident inputs, outputs and scratch of one replay launch (torch tensors)."""

    def __init__(self, desc, events, n_claim_slots: int, limits: dict, device="cuda", flags: int = 0,
                 scratch: bool = True):
        import torch
        if not torch.cuda.is_available():
            raise RuntimeError("no GPU: the replay runs only in the HIP kernels")
        lib = load()
        self.device = torch.device(device)
        self.desc = torch.as_tensor(desc, dtype=torch.int32).reshape(-1, 16).to(self.device).contiguous()
        self.events = torch.as_tensor(events, dtype=torch.int32).reshape(-1, 4).to(self.device).contiguous()
        n_pools = int(self.desc.shape[0])
        n_ev = int(self.events.shape[0])
        self.n_claim_slots = int(n_claim_slots)
        self.outcomes = torch.empty((max(n_ev, 1), 4), dtype=torch.int32, device=self.device)
        self.pool_tel = torch.empty((max(n_pools, 1), POOL_TEL_WORDS), dtype=torch.int32, device=self.device)
        self.claim_tel = torch.empty((max(self.n_claim_slots, 1), 10), dtype=torch.int32,
                                     device=self.device)
        b = Batch()
        b.n_pools = n_pools
        for k in ("max_usable_blocks", "max_events", "max_chains", "max_live_requests",
                  "max_live_claims", "max_claim_slots"):
            setattr(b, k, int(limits[k]))
        b.flags = int(flags)
        b.n_events_total = n_ev
        b.n_claim_slots_total = self.n_claim_slots
        b.d_pools = self.desc.data_ptr()
        b.d_events = self.events.data_ptr()
        b.d_outcomes = self.outcomes.data_ptr()
        b.d_pool_tel = self.pool_tel.data_ptr()
        b.d_claim_tel = self.claim_tel.data_ptr()
        self.scratch_needed = int(lib.rkc_scratch_bytes(ctypes.byref(b)))
        if scratch:
            self.scratch = torch.empty(max(self.scratch_needed, 256), dtype=torch.uint8, device=self.device)
            b.d_scratch = self.scratch.data_ptr()
            b.scratch_bytes = int(self.scratch.numel())
        else:  # only for replay_noalloc, which brings its own
            self.scratch = None
            b.d_scratch = None
            b.scratch_bytes = 0
        self.batch = b
        self.n_pools = n_pools
        self.n_events = n_ev

    @classmethod
    def from_trace(cls, trace, device="cuda", flags: int = 0, scratch: bool = True):
        return cls(trace.desc, trace.events, trace.n_claim_slots, trace.limits(), device, flags, scratch)

    def replay(self, stream=None):
        """Enqueue the replay on `stream` (default: torch's current stream)."""
        st = load().rkc_replay_batch(ctypes.byref(self.batch), _stream_ptr(stream))
        if st != 0:
            raise RkcError(st, "rkc_replay_batch")
        return self

    def replay_noalloc(self, stream=None):
        """Enqueue the replay through rkc_replay_batch_noalloc (the library's built-in scratch; no
        device allocation in the call)."""
        st = load().rkc_replay_batch_noalloc(ctypes.byref(self.batch), _stream_ptr(stream))
        if st != 0:
            raise RkcError(st, "rkc_replay_batch_noalloc")
        return self

    def results(self):
        """(outcomes [E,4], pool telemetry [P,64], claim telemetry [C,10]) as host numpy arrays."""
        import torch
        torch.cuda.synchronize(self.device)
        return (self.outcomes[: self.n_events].cpu().numpy(), self.pool_tel[: self.n_pools].cpu().numpy(),
                self.claim_tel[: self.n_claim_slots].cpu().numpy())

    def query_outcomes(self, pool: int, first: int, count: int, stream=None):
        import numpy as np
        out = np.zeros((max(count, 1), 4), np.int32)
        st = load().rkc_query_outcomes(ctypes.byref(self.batch), pool, first, count,
                                       ctypes.c_void_p(out.ctypes.data), _stream_ptr(stream))
        return st, out[:count]

    def query_telemetry(self, pool: int, max_claims: int, stream=None):
        import numpy as np
        ptel = np.zeros(POOL_TEL_WORDS, np.int32)
        ctel = np.zeros((max(max_claims, 1), 10), np.int32)
        n = ctypes.c_int32(0)
        st = load().rkc_query_telemetry(ctypes.byref(self.batch), pool, ctypes.c_void_p(ptel.ctypes.data),
                                        ctypes.c_void_p(ctel.ctypes.data), max_claims, ctypes.byref(n),
                                        _stream_ptr(stream))
        return st, ptel, ctel[: min(max_claims, n.value)], n.value


def replay(trace, stream=None):
    """Replay a trace (tracegen.Trace) on the GPU; returns host (outcomes, pool_tel, claim_tel)."""
    return DeviceBatch.from_trace(trace).replay(stream).results()
