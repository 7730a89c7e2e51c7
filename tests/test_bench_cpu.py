"""Host logic of bench.py that needs no GPU: the kernel code hash that ties the stored HBM
counters (profiles/traffic_full*.json) to the code they were taken on."""
import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import bench


def test_code_hash_ignores_comments_and_layout():
    a = "int f(int x) {\n  return x + 1;  // one more\n}\n"
    b = "/* f */ int f(int x)\n{ return x + 1; }"
    assert bench.code_hash(a) == bench.code_hash(b)


def test_code_hash_sees_code_and_literals():
    base = bench.code_hash('int a = 1; const char *s = "x";')
    assert bench.code_hash('int a = 2; const char *s = "x";') != base
    # text that looks like a comment inside a string or char literal is code
    assert bench.code_hash('const char *s = "// x";') != bench.code_hash('const char *s = "// y";')
    assert bench.code_hash("char c = '/'; int d;") != bench.code_hash("char c = '/'; int e;")


def test_stored_counters_match_the_kernel_code():
    """The committed counters were taken on the current kernel code (else bench.py reports
    traffic as null)."""
    import json
    for name in ("traffic_full.json", "traffic_full_tiers.json"):
        tr = json.load(open(os.path.join(ROOT, "profiles", name)))
        assert tr["kernel_src_sha"] == bench.kernel_sha(), name


def test_bench_refuses_step_counts_it_cannot_time():
    """No per-kernel timing pass (or no timed step) would leave the roofline without a
    duration: the arguments are refused before any device work."""
    import subprocess
    for bad in (["--kernel-steps", "0"], ["--steps", "0"], ["--warmup", "-1"]):
        r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py")] + bad, capture_output=True, text=True,
                           timeout=120)
        assert r.returncode == 2 and "at least" in r.stderr, (bad, r.stderr[-300:])
