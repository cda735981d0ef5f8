"""The benchmark's command-line contract on the CPU: more than one GPU is
refused with a message (the benchmark measures one GPU), and the traffic
record is keyed to the tile kernel's code, not its comments."""
import json
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    rec = json.loads(r.stdout.strip().splitlines()[-1])
    assert rec["n_gpus"] == 2 and "one GPU" in rec["error"]


def test_kernel_hash_ignores_comments_only():
    src = "int f(int x) {\n  // add one\n  return x + 1; /* done */\n}\n"
    same = "int f(int x) {\n\n  return x + 1;\n}\n// trailing note\n"
    other = "int f(int x) {\n  return x + 2;\n}\n"
    assert bench.code_text(src) == bench.code_text(same)
    assert bench.code_text(src) != bench.code_text(other)
    assert bench.kernel_source_hash([src, ""]) == bench.kernel_source_hash([same, ""])
