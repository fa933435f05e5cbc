"""The C-ABI library on the CPU: it loads, exports every function include/rkc.h declares, its
record layouts match the documented sizes, and the host-side argument checks return the documented
status codes (these paths return before any HIP call, so no GPU is needed)."""
import ctypes
import os
import re
import subprocess
import tempfile

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "rkc.h")


@pytest.fixture(scope="module")
def lib():
    import paper_2605_24259_amd as rkc
    if not os.path.exists(rkc.LIB_PATH):
        from paper_2605_24259_amd import build
        build.build()
    return rkc.load()


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(rkc_[a-z_]+)\s*\(", text)))


def test_exports_every_declared_function(lib):
    import paper_2605_24259_amd as rkc
    decl = declared_functions()
    assert set(decl) == set(rkc.EXPORTS)
    out = subprocess.check_output(["nm", "-D", "--defined-only", rkc.LIB_PATH], text=True)
    exported = set(re.findall(r"\bT (rkc_\w+)", out))
    assert set(decl) <= exported, set(decl) - exported
    for name in decl:
        assert hasattr(lib, name)


def test_layouts_match_header():
    src = r"""
#include <stddef.h>
#include <stdio.h>
#include "rkc.h"
int main(void) {
  printf("%zu %zu %zu %zu %zu %zu\n", sizeof(rkc_event), sizeof(rkc_pool_desc), sizeof(rkc_outcome),
         sizeof(rkc_claim_telemetry), sizeof(rkc_pool_telemetry), sizeof(rkc_batch));
  printf("%zu %zu %zu %zu\n", offsetof(rkc_pool_desc, event_offset), offsetof(rkc_pool_desc, claim_slot_offset),
         offsetof(rkc_batch, d_pools), offsetof(rkc_batch, scratch_bytes));
  return 0;
}
"""
    import paper_2605_24259_amd as rkc
    with tempfile.TemporaryDirectory() as d:
        c = os.path.join(d, "t.c")
        exe = os.path.join(d, "t")
        open(c, "w").write(src)
        subprocess.check_call(["gcc", "-std=c11", "-I", os.path.join(ROOT, "include"), c, "-o", exe])
        lines = subprocess.check_output([exe], text=True).split("\n")
    sizes = [int(x) for x in lines[0].split()]
    offs = [int(x) for x in lines[1].split()]
    assert sizes == [16, 64, 16, 40, 256, ctypes.sizeof(rkc.Batch)]
    assert offs == [48, 56, rkc.Batch.d_pools.offset, rkc.Batch.scratch_bytes.offset]


def _batch(**kw):
    import paper_2605_24259_amd as rkc
    b = rkc.Batch()
    b.n_pools = 2
    b.max_usable_blocks = 80
    b.max_events = 4
    b.max_chains = 2
    b.max_live_requests = 4
    b.max_live_claims = 4
    b.max_claim_slots = 2
    b.n_events_total = 8
    b.n_claim_slots_total = 4
    # plausible, aligned device addresses; none is dereferenced by the host-side checks
    b.d_pools = 0x10000
    b.d_events = 0x20000
    b.d_outcomes = 0x30000
    b.d_pool_tel = 0x40000
    b.d_claim_tel = 0x50000
    b.d_scratch = 0x60000
    b.scratch_bytes = 0
    for k, v in kw.items():
        setattr(b, k, v)
    return b


def test_version_and_strings(lib):
    assert lib.rkc_abi_version() == 5
    assert lib.rkc_status_string(0) == b"ok"
    assert lib.rkc_status_string(-5).startswith(b"scratch")
    assert b"built-in" in lib.rkc_status_string(-8)
    assert lib.rkc_status_string(-99) == b"unknown status"


def test_host_argument_checks(lib):
    null = ctypes.POINTER(type(_batch()))()
    assert lib.rkc_replay_batch(null, None) == -1
    assert lib.rkc_replay_batch(ctypes.byref(_batch(d_events=0)), None) == -1
    assert lib.rkc_replay_batch(ctypes.byref(_batch(d_outcomes=0x30008)), None) == -2
    assert lib.rkc_replay_batch(ctypes.byref(_batch(d_scratch=0x60010)), None) == -2
    assert lib.rkc_replay_batch(ctypes.byref(_batch(n_pools=-1)), None) == -3
    assert lib.rkc_replay_batch(ctypes.byref(_batch(flags=4)), None) == -3
    assert lib.rkc_replay_batch(ctypes.byref(_batch(max_usable_blocks=(1 << 22) + 1)), None) == -4
    # scratch too small (the batch needs > 0 bytes)
    b = _batch()
    need = lib.rkc_scratch_bytes(ctypes.byref(b))
    assert need > 0
    b.scratch_bytes = need - 1
    assert lib.rkc_replay_batch(ctypes.byref(b), None) == -5
    b.d_scratch = 0
    b.scratch_bytes = need
    assert lib.rkc_replay_batch(ctypes.byref(b), None) == -5
    # an empty batch is a valid no-op
    assert lib.rkc_replay_batch(ctypes.byref(_batch(n_pools=0)), None) == 0
    assert lib.rkc_scratch_bytes(null) == 0


def test_noalloc_host_checks(lib):
    """The no-allocation entry point checks the batch like rkc_replay_batch (it ignores the scratch
    fields) and refuses, before any HIP call, a batch whose scratch exceeds its built-in 64 MiB."""
    import paper_2605_24259_amd as rkc
    null = ctypes.POINTER(type(_batch()))()
    assert lib.rkc_replay_batch_noalloc(null, None) == -1
    assert lib.rkc_replay_batch_noalloc(ctypes.byref(_batch(d_events=0)), None) == -1
    assert lib.rkc_replay_batch_noalloc(ctypes.byref(_batch(d_outcomes=0x30008)), None) == -2
    assert lib.rkc_replay_batch_noalloc(ctypes.byref(_batch(n_pools=-1)), None) == -3
    assert lib.rkc_replay_batch_noalloc(ctypes.byref(_batch(n_pools=0, d_scratch=0)), None) == 0
    big = _batch(n_pools=4096, max_events=4096, d_scratch=0)
    assert lib.rkc_scratch_bytes(ctypes.byref(big)) > rkc.NOALLOC_SCRATCH_BYTES
    assert lib.rkc_replay_batch_noalloc(ctypes.byref(big), None) == -8


def test_scratch_grows_with_limits(lib):
    small = lib.rkc_scratch_bytes(ctypes.byref(_batch()))
    big = lib.rkc_scratch_bytes(ctypes.byref(_batch(max_events=4096)))
    many = lib.rkc_scratch_bytes(ctypes.byref(_batch(n_pools=20)))
    # per-pool regions, plus the launch order, class bytes and tile counts (256 bytes each here)
    assert big > small and many - 768 == 10 * (small - 768)


@pytest.mark.parametrize("max_events", [0, 1, 13, 63, 64, 65, 1024])
def test_scratch_is_proportional_to_the_limits(lib, max_events):
    """Scratch per pool stays within a few bytes per event and claim slot for both kernels (the
    compact one is chosen for these limits, the general one when the batch flag forces it)."""
    for flags in (0, 1):
        b = _batch(n_pools=1, max_events=max_events, flags=flags)
        n = lib.rkc_scratch_bytes(ctypes.byref(b))
        bound = 64 * (max_events + 2) + 16 * (b.max_claim_slots + 1) + 4096
        if flags:
            bound += 64 * (b.max_live_requests + b.max_live_claims)
        assert 0 < n <= bound, (flags, max_events, n, bound)
