"""GPU parity of the region-contribution probe (Sec. 2.2, Grad(M-hat, l) over
the sections of Appendix A.3) through the C interface, against the fp64
oracle on the same seeded Q, K, V, dO and the same fp32 row normalisers
(taken from the oracle's causal LSE, rounded to fp32)."""
import math
import os

import numpy as np
import pytest
import torch

import oracle
from paper_2507_21526_amd import binding as B
from paper_2507_21526_amd.inputs import draw_dout, draw_qkv
from tests.parity import log

pytestmark = pytest.mark.gpu

# |GPU - oracle| <= REL_ABS * (sum of |A_ij <dO_i, V_j>| over the section):
# the kernel rounds each product to fp32 (logits from exact bf16 inputs with
# fp32 accumulation, exp2 within an ulp or two) and sums 32 of them in fp32
# per step before an fp64 accumulate, so each term carries a relative error
# of a few 1e-6.
REL_ABS = 5e-5


def _probe(q, k, v, dout, lse, cu, tile, S, W, L, scale, plan=None):
    if plan is None:
        plan = B.Plan("causal", cu, 0, 1, 0, tile, q.shape[1], q.shape[2], device=q.device)
    nbytes = B.ta_probe_workspace_bytes(plan.info, q.shape[1])
    ws = torch.full((max(nbytes, 1),), 0xFF, dtype=torch.uint8, device=q.device)
    sums = torch.full((q.shape[1], 3), float("nan"), dtype=torch.float64, device=q.device)
    B.region_grad_probe(q, k, v, dout, lse, plan.sched, plan.info, scale, S, W, L, sums,
                        ws if nbytes else None)
    torch.cuda.synchronize()
    return sums.cpu().numpy(), plan


def _check(cu, hq, hkv, d, tile, S, W, L, seed):
    log(f"case probe cu={cu} hq={hq} hkv={hkv} d={d} T={tile} S={S} W={W} L={L}")
    q, k, v = draw_qkv(cu, hq, hkv, d, seed)
    dout = draw_dout(cu, hq, d, seed + 1)
    scale = 1.0 / math.sqrt(d)
    _, lse64 = oracle.attn_full(q, k, v, cu, "causal", 0, 1, 0, scale)
    lse32 = lse64.astype(np.float32)
    want, absw = oracle.region_grad(q, k, v, dout, lse32, cu, S, W, L, scale)
    got, _ = _probe(q.cuda(), k.cuda(), v.cuda(), dout.cuda(),
                    torch.from_numpy(lse32).cuda(), cu, tile, S, W, L, scale)
    err = np.abs(got - want)
    bound = REL_ABS * absw + 1e-12
    worst = float((err / np.maximum(absw, 1e-300)).max())
    log(f"  worst |err| / sum|term| = {worst:.2e}")
    assert np.all(np.isfinite(got))
    assert np.all(err <= bound), f"err {err.max():.3e}; rel {worst:.2e}"
    return got, want


CASES = [
    # cu, hq, hkv, d, tile, S, W, L
    ([0, 1024], 4, 1, 64, 64, 64, 256, 64),
    ([0, 700], 8, 2, 128, 128, 16, 100, 50),           # ragged q-tile
    ([0, 0, 333, 900, 901], 28, 4, 128, 64, 4, 40, 30),  # varlen, G = 7
    ([0, 513], 6, 2, 64, 128, 0, 1, 0),                 # no sink, W = 1, no Last
    ([0, 300], 5, 1, 128, 64, 300, 10, 300),            # all sink, all Last
    ([0, 200], 3, 1, 64, 64, 5, 0, 10),                 # empty window
    ([0, 777], 16, 2, 128, 64, 8, 512, 128),            # paper's S and W, G = 8
]


@pytest.mark.parametrize("cu,hq,hkv,d,tile,S,W,L", CASES)
def test_probe_parity(cu, hq, hkv, d, tile, S, W, L):
    _check(cu, hq, hkv, d, tile, S, W, L, len(cu) + hq + d + S)


@pytest.mark.parametrize("cu,hq,hkv,d,tile,S,W,L", [
    ([0, 0, 333, 900, 901], 28, 4, 128, 64, 4, 40, 30),
    ([0, 2048], 32, 8, 128, 128, 64, 128, 128),
])
def test_probe_shares(cu, hq, hkv, d, tile, S, W, L):
    """Any number of equal shares (one slot: each workgroup walks every item;
    more slots than k-tiles: most shares empty) gives the oracle's sums; the
    shares cut items at 64-key step boundaries, so the sums differ only in fp64
    summation order between slot counts."""
    runs = {}
    try:
        for slots in (1, 3, 16, 512):
            os.environ["TRIATTN_PROBE_SLOTS"] = str(slots)
            log(f"  slots {slots}")
            runs[slots], _ = _check(cu, hq, hkv, d, tile, S, W, L, 77)
    finally:
        os.environ.pop("TRIATTN_PROBE_SLOTS", None)
    ref = runs[1]
    for slots, got in runs.items():
        assert np.allclose(got, ref, rtol=1e-12, atol=1e-15), slots


def test_probe_corrupt_schedule_gives_nan():
    cu, hq, hkv, d = [0, 900], 8, 2, 128
    q, k, v = (t.cuda() for t in draw_qkv(cu, hq, hkv, d, 9))
    dout = draw_dout(cu, hq, d, 10).cuda()
    lse = torch.zeros((hq, cu[-1]), dtype=torch.float32, device="cuda")
    plan = B.Plan("causal", cu, 0, 1, 0, 128, hq, d, device="cuda")
    good = plan.sched.clone()
    got, _ = _probe(q, k, v, dout, lse, cu, 128, 16, 64, 32, 0.1, plan)
    assert np.all(np.isfinite(got))
    item = B.HDR_WORDS + B.ITEM_WORDS * (plan.info.n_items - 1)
    for word, value, what in ((0, int(good[0]) ^ 1, "magic"),
                              (item + 10, int(good[item + 10]) + 1, "cost"),
                              (item + 5, 1 << 20, "ka1 past the sequence"),
                              (item + 3, 1 << 20, "r1 past the sequence")):
        plan.sched.copy_(good)
        plan.sched[word] = value
        got, _ = _probe(q, k, v, dout, lse, cu, 128, 16, 64, 32, 0.1, plan)
        assert np.isnan(got).any(), what
        log(f"corrupt probe schedule ({what}): NaN sums")


def test_probe_per_item_negative_cost_gives_nan():
    """The per-item launch rejects a negative item cost, which would skip the
    item's checks.  32K tokens, 8 heads of group 1: 256 q-tiles of at most
    256 k-tiles against 64 slots of four-wave workgroups (2 per CU, 8 kv
    heads), and 256 * 64 * 2 <= 256 * 257 / 2 kept k-tiles, so one workgroup
    runs each item."""
    cu, hq, hkv, d = [0, 32768], 8, 8, 128
    q, k, v = (t.cuda() for t in draw_qkv(cu, hq, hkv, d, 9))
    dout = draw_dout(cu, hq, d, 10).cuda()
    lse = torch.zeros((hq, cu[-1]), dtype=torch.float32, device="cuda")
    plan = B.Plan("causal", cu, 0, 1, 0, 128, hq, d, device="cuda")
    assert plan.info.max_item_tiles * 64 * 2 <= plan.info.kept_tiles_per_qhead
    got, _ = _probe(q, k, v, dout, lse, cu, 128, 16, 64, 32, 0.1, plan)
    assert np.all(np.isfinite(got))
    item = B.HDR_WORDS + B.ITEM_WORDS * (plan.info.n_items - 1)
    plan.sched[item + 10] = -1
    got, _ = _probe(q, k, v, dout, lse, cu, 128, 16, 64, 32, 0.1, plan)
    assert np.isnan(got).any()


def test_probe_paper_shape():
    # one Llama-3.1-8B layer on a 2K-token prompt with the probe's sections
    # (si 64, sl 128, last 128)
    got, want = _check([0, 2048], 32, 8, 128, 128, 64, 128, 128, 1006)
    counts = B.ta_region_counts([0, 2048], 64, 128, 128)
    g_got = B.ta_region_grad_mean(got, counts)
    g_want = oracle_mean = want.sum(axis=0) / (32 * counts)
    assert np.allclose(g_got, oracle_mean, rtol=1e-3, atol=1e-12), (g_got, g_want)


def test_probe_deterministic_and_zero_dout():
    cu, hq, hkv, d = [0, 1000], 8, 2, 128
    q, k, v = (t.cuda() for t in draw_qkv(cu, hq, hkv, d, 3))
    dout = draw_dout(cu, hq, d, 4).cuda()
    lse = torch.zeros((hq, 1000), dtype=torch.float32, device="cuda")
    a, _ = _probe(q, k, v, dout, lse, cu, 128, 16, 64, 32, 0.1)
    b, _ = _probe(q, k, v, dout, lse, cu, 128, 16, 64, 32, 0.1)
    assert np.array_equal(a, b)
    z, _ = _probe(q, k, v, torch.zeros_like(dout), lse, cu, 128, 16, 64, 32, 0.1)
    assert np.all(z == 0)


def test_probe_empty_batch_writes_zeros():
    cu = [0, 0]
    e = torch.empty((0, 4, 64), dtype=torch.bfloat16, device="cuda")
    ek = torch.empty((0, 1, 64), dtype=torch.bfloat16, device="cuda")
    lse = torch.empty((4, 0), dtype=torch.float32, device="cuda")
    got, plan = _probe(e, ek, ek, e, lse, cu, 64, 1, 1, 1, 0.1)
    assert plan.info.n_items == 0 and np.all(got == 0)


def test_probe_total_equals_dout_dot_output_32k():
    # at full size: the sections partition the causal pairs, so their sums
    # add up to sum_i <dO_i, O_i> with O the causal attention output (the
    # kernel's own fp32 output and LSE here; O carries bf16 probabilities,
    # hence the looser bound)
    cu, hq, hkv, d = [0, 32768], 32, 8, 128
    log("case probe 32K identity")
    q, k, v = (t.cuda() for t in draw_qkv(cu, hq, hkv, d, 1002, head_scale=(0.5, 2.0)))
    dout = draw_dout(cu, hq, d, 1003).cuda()
    plan = B.Plan("causal", cu, 0, 1, 0, 128, hq, d, device="cuda")
    o = torch.empty(q.shape, dtype=torch.float32, device="cuda")
    lse = torch.empty((hq, cu[-1]), dtype=torch.float32, device="cuda")
    plan.run(q, k, v, o, lse, 1.0 / math.sqrt(d))
    sums, _ = _probe(q, k, v, dout, lse, cu, 128, 64, 128, 128, 1.0 / math.sqrt(d))
    terms = (dout.double() * o.double()).sum(dim=2)  # [T, hq]
    want = terms.sum(dim=0).cpu().numpy()
    scale_ref = terms.abs().sum(dim=0).cpu().numpy()
    err = np.abs(sums.sum(axis=1) - want)
    log(f"  worst |err| / sum|<dO, O>| = {float((err / scale_ref).max()):.2e}")
    assert np.all(err <= 2e-3 * scale_ref)


def test_region_grad_helper_matches_oracle_means():
    # the one-call helper (causal pass for the LSE, probe, counts, means)
    # against the oracle's sums over its own fp64 causal LSE
    cu, hq, hkv, d, S, W, L = [0, 600, 1500], 8, 2, 128, 32, 256, 100
    log("case probe helper")
    q, k, v = draw_qkv(cu, hq, hkv, d, 51)
    dout = draw_dout(cu, hq, d, 52)
    scale = 1.0 / math.sqrt(d)
    grad, sums = B.region_grad(q.cuda(), k.cuda(), v.cuda(), dout.cuda(), cu, S, W, L,
                               tile=128)
    _, lse64 = oracle.attn_full(q, k, v, cu, "causal", 0, 1, 0, scale)
    want, absw = oracle.region_grad(q, k, v, dout, lse64, cu, S, W, L, scale)
    # the GPU LSE differs from the fp64 one by ~1e-6 (fp32), which moves
    # every A_ij by that relative amount
    assert np.all(np.abs(sums - want) <= 1e-4 * absw + 1e-12)
    counts = oracle.region_counts(cu, S, W, L)
    want_grad = want.sum(axis=0) / (hq * counts)
    assert np.allclose(grad, want_grad, rtol=0,
                       atol=1e-4 * float(absw.sum(axis=0).max()) / (hq * counts.min()))
    layers = B.ta_select_triangle_layers([grad[1], 10 * grad[1], 0.1 * grad[1]], 2)
    assert layers == [0, 2]
