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
    assert bench.kernel_source_hash([src, "", ""]) == bench.kernel_source_hash([same, "", ""])


def test_element_exact_flops_count_the_kept_pairs():
    # brute force over the Triangle mask (j <= i and (j < S or i - j < W),
    # or i in the last L rows) on a small packed batch, against the closed
    # form the benchmark uses
    from paper_2507_21526_amd import binding
    from paper_2507_21526_amd.inputs import WORKLOADS
    import numpy as np

    class W:
        sink, window, last, hq = 5, 17, 9, 3

    cu = [0, 40, 40, 101]
    pairs = 0
    for b in range(len(cu) - 1):
        n = cu[b + 1] - cu[b]
        i = np.arange(n)[:, None]
        j = np.arange(n)[None, :]
        keep = (j <= i) & ((j < W.sink) | (i - j < W.window) | (i >= n - min(W.last, n)))
        pairs += int(keep.sum())
    rec = bench.element_exact(binding, cu, W, 64, 1.0)
    assert rec["pairs_per_head"] == pairs
    assert rec["flops"] == 4.0 * 64 * W.hq * pairs
    # the 128K Llama workload: 4.904e12 FLOPs of kept pairs
    w = WORKLOADS["llama8b_n128k"]
    big = bench.element_exact(binding, list(w.cu_seqlens), w, w.d, 1.0)
    assert abs(big["flops"] - 4.9043e12) < 1e9
