"""GPU test of triangle_attn_fwd_noalloc, the entry point that allocates
nothing (its split partials live in the library's per-GPU scratch array):
through the C interface, its output equals triangle_attn_fwd's bit for bit
on two calls in a row, the second with a smaller input (the array keeps the
first call's contents, which the second must overwrite where it reads)."""
import math

import pytest
import torch

from paper_2507_21526_amd import binding
from paper_2507_21526_amd.inputs import draw_qkv
from tests.parity import log

pytestmark = pytest.mark.gpu


def _pair(cu, hq, hkv, d, S, W, L, T, splits, seed, out_dtype):
    q, k, v = (t.to("cuda:0") for t in draw_qkv(cu, hq, hkv, d, seed))
    scale = 1.0 / math.sqrt(d)
    plan = binding.Plan("triangle", cu, S, W, L, T, hq, d, splits, device=q.device)
    assert plan.info.n_merge_items > 0
    need = binding.ta_workspace_bytes(plan.info, hq, d)
    ref = torch.full(q.shape, float("nan"), dtype=out_dtype, device=q.device)
    ref_lse = torch.full((hq, cu[-1]), float("nan"), device=q.device)
    plan.run(q, k, v, ref, ref_lse, scale)
    got = torch.full_like(ref, float("nan"))
    got_lse = torch.full_like(ref_lse, float("nan"))
    binding.triangle_attn_fwd_noalloc(q, k, v, got, got_lse, plan.sched, plan.info, scale)
    torch.cuda.synchronize()
    log(f"noalloc cu={cu} hq={hq} d={d} splits={plan.info.max_splits}: "
        f"{need} bytes of partials")
    assert not torch.isnan(got).any()
    assert torch.equal(got, ref)
    assert torch.equal(got_lse, ref_lse)
    return need


def test_noalloc_matches_workspace_entry_point():
    # first call: two sequences, many splits (tens of MB of partials)
    big = _pair([0, 9000, 16384], 32, 8, 128, 128, 2048, 512, 128, 0, 31,
                torch.bfloat16)
    # second call: a smaller input; its partials reuse the start of the array
    small = _pair([0, 1500], 8, 2, 64, 16, 256, 300, 64, 7, 32, torch.float32)
    assert 0 < small < big


def test_noalloc_without_partials():
    # L = 0: no Last rows, no split partials, the scratch array is not used
    q, k, v = (t.to("cuda:0") for t in draw_qkv([0, 700], 4, 1, 128, 33))
    plan = binding.Plan("triangle", [0, 700], 8, 128, 0, 128, 4, 128, device=q.device)
    assert binding.ta_workspace_bytes(plan.info, 4, 128) == 0
    ref = torch.empty(q.shape, dtype=torch.float32, device=q.device)
    plan.run(q, k, v, ref, None, 0.1)
    got = torch.empty_like(ref)
    binding.triangle_attn_fwd_noalloc(q, k, v, got, None, plan.sched, plan.info, 0.1)
    torch.cuda.synchronize()
    assert torch.equal(got, ref)
