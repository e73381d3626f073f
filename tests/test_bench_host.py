"""Host-side checks of the benchmark: its FLOP count against the oracle's
(App. A), the scheduled workloads' segments, the one-GPU guard and the key
of the traffic figure."""
import json
import os
import subprocess
import sys

import pytest

import bench
from lact_synth import CONFIGS, make_schedule
from oracle import lact_oracle as O

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.mark.parametrize("name", [n for n, c in CONFIGS.items() if not c.schedule])
def test_bench_flops_match_the_oracle_count(name):
    c = CONFIGS[name]
    if c.linear:
        ref = O.linear_flops(c.BH, c.d, c.n_kv, c.n_q, c.n_chunks, bool(c.use_muon), c.ns_steps)
    else:
        ref = O.layer_flops(c.BH, c.d, c.h, c.n_kv, c.n_q, c.n_chunks, bool(c.use_muon), c.ns_steps)
    assert bench.workload_flops(c) == pytest.approx(ref, rel=1e-12)


def test_video_teacher_forcing_schedule_and_flops():
    c = CONFIGS["video_tf"]
    sched = make_schedule(c)
    assert len(sched) == 37 and sched[0][1] == 0 and sched[-1][2] == c.n_kv
    assert all(a[2] == b[1] for a, b in zip(sched, sched[1:]))          # contiguous
    modes = [m for m, _, _ in sched]
    assert modes[0] == modes[-1] == "apply_only" and modes.count("update_then_apply") == 18
    assert all(modes[i] != modes[i + 1] for i in range(len(modes) - 1))  # alternating
    # every segment counted as a one-chunk layer of its own length
    ref = 0.0
    for m, b, e in sched:
        n = e - b
        ref += O.layer_flops(c.BH, c.d, c.h, 0 if m == "apply_only" else n, n, 0 if m == "apply_only" else 1,
                             bool(c.use_muon), c.ns_steps)
    assert bench.workload_flops(c) == pytest.approx(ref, rel=1e-12)


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2 and "one GPU" in json.loads(r.stdout.strip().splitlines()[-1])["error"]


def test_source_hash_ignores_comments_and_whitespace_only():
    # the traffic figure is keyed to the kernel sources as the compiler sees them
    a = 'int x = 1; // rate\n/* tile */ const char* s = "a // b";  float y;'
    b = 'int x = 1;\n\n   const char* s = "a // b"; /* other words */ float y; // end'
    c = 'int x = 2; const char* s = "a // b"; float y;'
    assert bench._code_only(a) == bench._code_only(b)
    assert bench._code_only(a) != bench._code_only(c)
    assert bench._code_only('char q = \'"\'; // "') == "char q = '\"';"
