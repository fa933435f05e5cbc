"""The C oracle and the trace generator under AddressSanitizer and UndefinedBehaviorSanitizer.

Both are rebuilt with gcc's sanitizers into a temporary directory and driven, in a child process
with the sanitizer runtimes preloaded, through random pools with every feature and through the
benchmark workloads' generators; any sanitizer report fails the test.
"""
import os
import subprocess
import sys
import textwrap

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

CHILD = textwrap.dedent("""
    import sys
    sys.path.insert(0, {root!r})
    import oracle
    oracle._LIB = {olib!r}
    from paper_2605_24259_amd import tracegen as tg
    tg._LIB = {tlib!r}
    tg._lib = None
    from tests import randtrace
    for name in tg.CONFIGS:
        tg.generate(name, n_pools=2)
    cases = [(501, dict(U_range=(1, 200), n_events=(0, 200), n_chains=9, p_malformed=0.03,
                        tight_every=4, caps=(64, 16), defer=True, relax=True, offload=True,
                        hard_share=0.5)),
             (41, dict(U_range=(2, 120), n_events=(1, 150), n_chains=5, tight_every=3))]
    for seed, kw in cases:
        tr = randtrace.random_batch(seed, 120, **kw)
        out = oracle.replay(tr.desc, tr.events, tr.n_claim_slots, threads=1)
        assert not out[3].any()
    for name in ("zipf", "zipf_offload"):
        tr = tg.generate(name, n_pools=2)
        out = oracle.replay(tr.desc, tr.events, tr.n_claim_slots, threads=1)
        assert not out[3].any()
    print("sanitized run ok")
""")


def _runtime(name):
    path = subprocess.run(["gcc", f"-print-file-name={name}"], capture_output=True, text=True).stdout.strip()
    return path if os.path.isabs(path) and os.path.exists(path) else None


def test_oracle_and_generator_under_sanitizers(tmp_path):
    asan, ubsan = _runtime("libasan.so"), _runtime("libubsan.so")
    if not asan or not ubsan:
        pytest.skip("gcc sanitizer runtimes not installed")
    flags = ["gcc", "-O1", "-g", "-std=c11", "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
             "-fno-omit-frame-pointer", "-shared", "-fPIC"]
    olib, tlib = str(tmp_path / "liboracle.so"), str(tmp_path / "libtracegen.so")
    subprocess.check_call(flags + [os.path.join(ROOT, "oracle", "rkc_oracle.c"), "-o", olib])
    subprocess.check_call(flags + [os.path.join(ROOT, "paper_2605_24259_amd", "tracegen", "tracegen.c"),
                                   "-o", tlib, "-lm"])
    env = dict(os.environ, LD_PRELOAD=f"{asan}:{ubsan}", ASAN_OPTIONS="detect_leaks=0",
               UBSAN_OPTIONS="halt_on_error=1")
    child = CHILD.format(root=ROOT, olib=olib, tlib=tlib)
    r = subprocess.run([sys.executable, "-c", child], env=env, capture_output=True, text=True, timeout=600)
    report = [line for line in (r.stdout + r.stderr).splitlines()
              if "runtime error" in line or "ERROR: AddressSanitizer" in line]
    assert r.returncode == 0 and not report, (r.stdout[-2000:], r.stderr[-4000:])
    assert "sanitized run ok" in r.stdout
