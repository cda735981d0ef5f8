"""GPU parity of block-sparse causal attention (the dense layers handed to a
dynamic sparse method, Sec. 2.4 and Sec. 3.1) through the C interface,
against the fp64 oracle on the same seeded inputs and k-tile lists."""
import math

import numpy as np
import pytest
import torch

import oracle
from paper_2507_21526_amd import binding as B
from paper_2507_21526_amd.inputs import WORKLOADS, blocksparse_lists, draw_qkv, workload_qkv
from tests.parity import LSE_ABS, MAX_ABS, REL_L2, log, run_pass
from tests.test_blocksparse import random_lists

pytestmark = pytest.mark.gpu


def _run_bs(q, k, v, cu, tile, ptr, idx, max_tiles, out_dtype=torch.float32):
    d = q.shape[2]
    plan = B.Plan("blocksparse", cu, 0, 1, 0, tile, q.shape[1], d, max_tiles,
                  device=q.device, blocks=(ptr, idx))
    o = torch.full(q.shape, float("nan"), dtype=out_dtype, device=q.device)
    lse = torch.full((q.shape[1], q.shape[0]), float("nan"), dtype=torch.float32,
                     device=q.device)
    if plan.workspace is not None:
        plan.workspace.view(torch.uint8).fill_(0xFF)
    plan.run(q, k, v, o, lse, 1.0 / math.sqrt(d))
    torch.cuda.synchronize()
    return o, lse, plan


def _compare(q, k, v, cu, tile, ptr, idx, o, lse, toks, label):
    hq, d = q.shape[1], q.shape[2]
    rt = np.repeat(np.asarray(toks, dtype=np.int64), hq)
    rh = np.tile(np.arange(hq, dtype=np.int32), len(toks))
    ref_o, ref_l = oracle.attn_rows_bs(q, k, v, cu, tile, ptr, idx, 1.0 / math.sqrt(d),
                                       rt, rh)
    it, ih = torch.from_numpy(rt).cuda(), torch.from_numpy(rh.astype(np.int64)).cuda()
    got_o = o[it, ih].double().cpu().numpy()
    got_l = lse[ih, it].double().cpu().numpy()
    worst = 0.0
    for h in range(hq):
        sel = rh == h
        err = got_o[sel] - ref_o[sel]
        mx = float(np.abs(err).max()) if err.size else 0.0
        rel = float(np.linalg.norm(err) / max(np.linalg.norm(ref_o[sel]), 1e-30))
        assert mx <= MAX_ABS and rel <= REL_L2, f"{label} head {h}: {mx:.3e} {rel:.3e}"
        fin = np.isfinite(ref_l[sel])
        assert np.array_equal(np.isfinite(got_l[sel]), fin), f"{label}: lse finiteness"
        if fin.any():
            assert float(np.abs(got_l[sel][fin] - ref_l[sel][fin]).max()) <= LSE_ABS
        worst = max(worst, mx)
    log(f"{label}: {len(toks)} rows x {hq} heads, worst max-abs {worst:.2e}")


CASES = [
    # cu, hq, hkv, d, tile, density, diag, max_tiles
    ([0, 700], 8, 2, 128, 128, 0.5, True, 0),
    ([0, 700], 8, 2, 128, 128, 0.5, None, 1),       # many splits per q-tile
    ([0, 1000], 4, 1, 64, 64, 0.3, False, 2),       # no diagonal tile
    ([0, 0, 333, 900, 901], 28, 4, 128, 64, 0.6, None, 3),  # varlen, G = 7
    ([0, 1500], 16, 2, 128, 128, 0.1, None, 0),     # sparse, some empty rows
    ([0, 520], 3, 1, 64, 128, 1.0, None, 2),        # full lists cut in splits
    ([0, 1200], 4, 4, 128, 128, 0.4, None, 0),      # G = 1: Q tiles in a K/V stage
    ([0, 900], 2, 2, 64, 64, 0.5, True, 1),         # G = 1, T = 64: two waves
]


@pytest.mark.parametrize("cu,hq,hkv,d,tile,density,diag,max_tiles", CASES)
def test_blocksparse_full_parity(cu, hq, hkv, d, tile, density, diag, max_tiles):
    log(f"case blocksparse cu={cu} hq={hq} hkv={hkv} d={d} T={tile} "
        f"density={density} diag={diag} bound={max_tiles}")
    q, k, v = draw_qkv(cu, hq, hkv, d, len(cu) + hq + d)
    ptr, idx = random_lists(cu, tile, density, hq + d, diag=diag)
    o, lse, plan = _run_bs(q.cuda(), k.cuda(), v.cuda(), cu, tile, ptr, idx, max_tiles)
    assert not torch.isnan(o).any(), "an output row was not written"
    assert not torch.isnan(lse).any(), "an lse entry was not written"
    _compare(q, k, v, cu, tile, ptr, idx, o, lse, np.arange(cu[-1]),
             f"blocksparse cu={cu} bound={max_tiles} splits={plan.info.n_merge_items}")


def test_skewed_lists_split_by_the_automatic_bound():
    # one q-tile lists every k-tile, the others only the diagonal: the
    # automatic bound cuts that list alone into a split and a merge
    cu, tile = [0, 40 * 64 - 17], 64
    ptr, idx = [0], []
    for t in range(40):
        idx.extend(range(40) if t == 39 else [t])
        ptr.append(len(idx))
    log(f"case blocksparse skewed lists cu={cu} T={tile} bound=auto")
    q, k, v = draw_qkv(cu, 8, 2, 128, 41)
    o, lse, plan = _run_bs(q.cuda(), k.cuda(), v.cuda(), cu, tile, ptr, idx, 0)
    assert plan.info.n_merge_items == 1
    assert not torch.isnan(o).any() and not torch.isnan(lse).any()
    _compare(q, k, v, cu, tile, ptr, idx, o, lse, np.arange(cu[-1]), "blocksparse skewed")


def test_full_lists_equal_the_causal_kernel():
    # every q-tile lists every k-tile up to the diagonal and the bound keeps
    # them in one item: the same work items as the dense causal pass
    cu, tile = [0, 1000, 1777], 128
    q, k, v = (t.cuda() for t in draw_qkv(cu, 8, 2, 128, 9))
    ptr, idx = random_lists(cu, tile, 1.0, 0)
    o_bs, l_bs, _ = _run_bs(q, k, v, cu, tile, ptr, idx, 1000)
    o_c, l_c, _ = run_pass("causal", q, k, v, cu, 0, 1, 0, tile)
    torch.cuda.synchronize()
    assert torch.equal(o_bs, o_c) and torch.equal(l_bs, l_c)


def test_empty_lists_write_zero_rows():
    cu, tile = [0, 300], 64
    q, k, v = (t.cuda() for t in draw_qkv(cu, 4, 1, 64, 3))
    o, lse, _ = _run_bs(q, k, v, cu, tile, [0] * 6, [], 0, out_dtype=torch.bfloat16)
    assert torch.all(o == 0) and torch.all(torch.isneginf(lse))


def test_blocksparse_32k_sampled():
    # a Llama-shaped 32K layer with about a tenth of the causal tiles kept
    # (always the diagonal tile, as block estimators do), sampled rows
    cu, tile = [0, 32768], 128
    q, k, v = draw_qkv(cu, 32, 8, 128, 77)
    ptr, idx = random_lists(cu, tile, 0.1, 78, diag=True)
    o, lse, plan = _run_bs(q.cuda(), k.cuda(), v.cuda(), cu, tile, ptr, idx, 0)
    rng = np.random.default_rng(79)
    toks = np.unique(np.concatenate([rng.integers(0, 32768, 160),
                                     np.arange(0, 32768, 4096), [32767]]))
    _compare(q, k, v, cu, tile, ptr, idx, o, lse, toks,
             f"blocksparse 32K kept tiles {plan.info.kept_tiles_per_qhead}")


def test_blocksparse_128k_bench_config():
    # the benchmark's configuration: the 128K Llama layer with about a tenth
    # of each q-tile's causal k-tiles plus its diagonal (the same seeded
    # lists), automatic work bound; sampled rows, including rows of the
    # q-tiles the bound split (merged rows) and q-tile edges
    w = WORKLOADS["llama8b_n128k"]
    cu, tile = list(w.cu_seqlens), w.tile
    nq = -(-cu[-1] // tile)
    ptr, idx = blocksparse_lists(nq, 0.1, w.seed)
    log(f"case blocksparse 128K bench config, {len(idx)} listed tiles")
    q, k, v = workload_qkv(w)
    o, lse, plan = _run_bs(q.cuda(), k.cuda(), v.cuda(), cu, tile, ptr, idx, 0)
    words = plan.words
    m0 = 16 + 12 * plan.info.n_items
    merges = words[m0:m0 + 8 * plan.info.n_merge_items].reshape(-1, 8)
    assert len(merges) > 0
    rng = np.random.default_rng(80)
    split_rows = [int(m[1]) + r for m in merges[:: max(1, len(merges) // 4)] for r in (0, 77, 127)]
    toks = np.unique(np.concatenate([rng.integers(0, cu[-1], 128), split_rows,
                                     [0, 127, 128, 65535, 65536, cu[-1] - 1]]))
    _compare(q, k, v, cu, tile, ptr, idx, o, lse, toks,
             f"blocksparse 128K, {len(merges)} split q-tiles")


def test_list_longer_than_the_key_table():
    # one q-tile lists 2050 k-tiles (T = 64, one item, no split): more steps
    # than the kernel's LDS key table holds, so that item reads its list in
    # global memory at every step; the other q-tiles list their diagonal
    cu, tile = [0, 2049 * 64 + 5], 64
    nq = -(-cu[-1] // tile)
    ptr, idx = [0], []
    for t in range(nq):
        idx.extend(range(t + 1) if t == nq - 1 else [t])
        ptr.append(len(idx))
    log(f"case blocksparse long list: {nq} q-tiles, last lists {nq} tiles")
    q, k, v = draw_qkv(cu, 2, 1, 64, 91)
    o, lse, plan = _run_bs(q.cuda(), k.cuda(), v.cuda(), cu, tile, ptr, idx, 100000)
    assert plan.info.n_merge_items == 0
    toks = np.concatenate([np.arange((nq - 1) * tile, cu[-1]), [0, 63, 64, 100000]])
    _compare(q, k, v, cu, tile, ptr, idx, o, lse, toks, "blocksparse long list")
