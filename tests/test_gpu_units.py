"""GPU tests of the multi-unit tile kernel: workgroups of five to eight waves
that run several (item, row block) units of a Triangle pass as one pipeline.

The kernel computes every row with the same 64-key steps, in the same order,
as the single-unit kernel, so its outputs must be bit-identical to it;
TRIATTN_UNITS_PER_WG (read by the library at each launch) forces the unit
count, so small shapes run through unit boundaries of every kind: ragged
q-tiles whose second row block is empty, Last-row splits without a step for
some rows (written as zero partials), units of different sequences of a
packed batch, sinks that are not tile aligned, one- or two-key windows, and
bf16 and fp32 outputs.  One configuration is also checked against the fp64
oracle."""
import math
import os

import numpy as np
import pytest
import torch

from paper_2507_21526_amd.inputs import draw_qkv
from tests.parity import compare, log, run_pass

pytestmark = pytest.mark.gpu

ENV = "TRIATTN_UNITS_PER_WG"

CASES = [
    # cu, hq, hkv, d, S, W, L, T, splits
    ([0, 1500], 16, 2, 128, 1, 1, 1, 128, 0),                      # G 8, 2-key rows
    ([0, 0, 100, 100, 357, 1000], 8, 2, 64, 3, 50, 77, 64, 0),     # G 4, packed, empty
    ([0, 640], 8, 2, 128, 130, 65, 129, 128, 3),                   # sink not aligned
    ([0, 2000], 28, 4, 128, 16, 100, 40, 128, 0),                  # G 7 (Qwen group)
    ([0, 700, 1300], 6, 2, 128, 8, 64, 200, 64, 5),                # G 3, six waves
    ([0, 1000], 5, 1, 64, 4, 128, 300, 128, 7),                    # G 5, five waves
    ([0, 1000], 8, 2, 128, 16, 128, 200, 128, 8),                  # splits without steps
]


def _run(kind, q, k, v, cu, S, W, L, T, splits, upw, out_dtype):
    os.environ[ENV] = str(upw)
    try:
        o, lse, _ = run_pass(kind, q, k, v, cu, S, W, L, T, splits, out_dtype=out_dtype,
                             poison=True)
        torch.cuda.synchronize()
    finally:
        del os.environ[ENV]
    return o, lse


@pytest.mark.parametrize("cu,hq,hkv,d,S,W,L,T,splits", CASES)
def test_units_bit_identical_to_single_unit(cu, hq, hkv, d, S, W, L, T, splits):
    log(f"case units cu={cu} hq={hq} hkv={hkv} d={d} S={S} W={W} L={L} T={T} splits={splits}")
    q, k, v = (t.cuda() for t in draw_qkv(cu, hq, hkv, d, seed=len(cu) + hq + S))
    for out_dtype in (torch.float32, torch.bfloat16):
        ref_o, ref_l = _run("triangle", q, k, v, cu, S, W, L, T, splits, 1, out_dtype)
        assert not torch.isnan(ref_o).any()
        for upw in (2, 3, 7, 128):
            o, lse = _run("triangle", q, k, v, cu, S, W, L, T, splits, upw, out_dtype)
            assert not torch.isnan(o).any(), (upw, out_dtype)
            assert torch.equal(o, ref_o), (upw, out_dtype)
            assert torch.equal(lse, ref_l), (upw, out_dtype)
    log(f"units cu={cu}: bit-identical for 2, 3, 7 and 128 units per workgroup")


def test_units_against_oracle():
    cu, hq, hkv, d, S, W, L, T = [0, 900, 2100], 8, 2, 128, 20, 300, 150, 128
    q, k, v = draw_qkv(cu, hq, hkv, d, seed=77)
    qg, kg, vg = q.cuda(), k.cuda(), v.cuda()
    o, lse = _run("triangle", qg, kg, vg, cu, S, W, L, T, 0, 5, torch.float32)
    compare("triangle", q, k, v, cu, S, W, L, 1.0 / math.sqrt(d), o, lse,
            np.arange(cu[-1]), range(hq), label="units=5 vs oracle")


def test_units_noalloc_and_graph_replay():
    """The no-allocation entry point and HIP graph replays run the same
    multi-unit launches: the library's own unit rule picks the multi-unit
    kernel for this shape (sink 8, window 128 and 32 explicit Last splits:
    items of at most 4 k-tiles, 8 steps at d = 128), which the single-unit
    kernel (one unit per workgroup forced) must match bit for bit."""
    from paper_2507_21526_amd import binding
    cu, hq, hkv, d = [0, 16384], 32, 8, 128
    q, k, v = (t.cuda() for t in draw_qkv(cu, hq, hkv, d, seed=78))
    plan = binding.Plan("triangle", cu, 8, 128, 128, 128, hq, d, splits=32)
    assert plan.info.max_item_tiles * 2 <= 8
    ref = torch.empty(q.shape, dtype=torch.bfloat16, device=q.device)
    plan.run(q, k, v, ref, None, d ** -0.5)
    os.environ[ENV] = "1"
    try:
        single = torch.empty_like(ref)
        plan.run(q, k, v, single, None, d ** -0.5)
        torch.cuda.synchronize()
    finally:
        del os.environ[ENV]
    assert torch.equal(ref, single)
    na = torch.empty_like(ref)
    binding.triangle_attn_fwd_noalloc(q, k, v, na, None, plan.sched, plan.info, d ** -0.5)
    torch.cuda.synchronize()
    assert torch.equal(na, ref)
    graph = torch.cuda.CUDAGraph()
    out = torch.zeros_like(ref)
    with torch.cuda.graph(graph):
        plan.run(q, k, v, out, None, d ** -0.5)
    for _ in range(3):
        out.fill_(float("nan"))
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(out, ref)
