"""Block-sparse causal attention on the CPU: the oracle pinned against numpy
brute force and the causal mask, its schedule against the packing rule
written in the interface, and the library's schedule builder word for word
against the oracle (Sec. 2.4 and Sec. 3.1: the dense layers handed to a
dynamic sparse method that lists the kept k-tiles of every q-tile)."""
import ctypes
import math

import numpy as np
import pytest
import torch

import oracle
from paper_2507_21526_amd import binding as B
from paper_2507_21526_amd.inputs import draw_qkv


def random_lists(cu, tile, density, seed, diag=None):
    """CSR lists of kept k-tiles (sorted, <= the q-tile index).  diag: force
    (True) or drop (False) the diagonal tile; None = random like the rest."""
    rng = np.random.default_rng(seed)
    ptr, idx = [0], []
    for b in range(len(cu) - 1):
        n = cu[b + 1] - cu[b]
        for t in range(-(-n // tile)):
            keep = [kt for kt in range(t + 1) if rng.random() < density]
            if diag is True and t not in keep:
                keep.append(t)
            if diag is False and t in keep:
                keep.remove(t)
            idx.extend(sorted(keep))
            ptr.append(len(idx))
    return ptr, idx


def lists_of_seq(cu, tile, ptr, idx, b):
    """The k-tile lists of the q-tiles of sequence b."""
    base = sum(-(-(cu[s + 1] - cu[s]) // tile) for s in range(b))
    nq = -(-(cu[b + 1] - cu[b]) // tile)
    return [idx[ptr[base + t]:ptr[base + t + 1]] for t in range(nq)]


def numpy_attention(q, k, v, cu, tile, ptr, idx, scale):
    """Masked softmax attention written out with numpy in fp64 (the plain
    definition, Sec. 2.1), mask built from the lists directly."""
    qf = q.double().numpy()
    kf = k.double().numpy()
    vf = v.double().numpy()
    total, hq, d = qf.shape
    hkv = kf.shape[1]
    g = hq // hkv
    out = np.zeros((total, hq, d))
    lse = np.full((hq, total), -np.inf)
    for b in range(len(cu) - 1):
        off, n = cu[b], cu[b + 1] - cu[b]
        lists = lists_of_seq(cu, tile, ptr, idx, b)
        for i in range(n):
            keys = [j for j in range(i + 1) if (j // tile) in lists[i // tile]]
            if not keys:
                continue
            for h in range(hq):
                z = scale * (kf[off + np.array(keys), h // g] @ qf[off + i, h])
                m = z.max()
                p = np.exp(z - m)
                out[off + i, h] = p @ vf[off + np.array(keys), h // g] / p.sum()
                lse[h, off + i] = m + math.log(p.sum())
    return out, lse


# ---- oracle pins -----------------------------------------------------------

def test_full_lists_give_the_causal_mask():
    n, tile = 150, 16
    lists = [list(range(t + 1)) for t in range(-(-n // tile))]
    bs = oracle.bs_mask_matrix(n, tile, lists)
    causal = oracle.mask_matrix("causal", n, 0, 1, 0)
    assert np.array_equal(bs, causal)


def test_diagonal_lists_give_block_local_causal_mask():
    n, tile = 70, 8
    lists = [[t] for t in range(-(-n // tile))]
    bs = oracle.bs_mask_matrix(n, tile, lists)
    i, j = np.meshgrid(np.arange(n), np.arange(n), indexing="ij")
    want = (j <= i) & (j // tile == i // tile)
    assert np.array_equal(bs.astype(bool), want)


@pytest.mark.parametrize("density,seed", [(0.3, 1), (0.7, 2), (1.0, 3)])
def test_oracle_matches_numpy_brute_force(density, seed):
    cu, tile = [0, 45, 45, 83], 8
    q, k, v = draw_qkv(cu, 4, 2, 16, seed)
    ptr, idx = random_lists(cu, tile, density, seed)
    scale = 0.25
    want_o, want_l = numpy_attention(q, k, v, cu, tile, ptr, idx, scale)
    total, hq = cu[-1], 4
    tok = np.repeat(np.arange(total), hq)
    head = np.tile(np.arange(hq), total)
    got_o, got_l = oracle.attn_rows_bs(q, k, v, cu, tile, ptr, idx, scale, tok, head)
    got_o = got_o.reshape(total, hq, 16)
    got_l = got_l.reshape(total, hq).T
    assert np.allclose(got_o, want_o, atol=1e-12, rtol=0)
    fin = np.isfinite(want_l)
    assert np.array_equal(np.isfinite(got_l), fin)
    assert np.allclose(got_l[fin], want_l[fin], atol=1e-12, rtol=0)


def test_oracle_empty_lists_give_zero_rows():
    cu, tile = [0, 40], 8
    q, k, v = draw_qkv(cu, 2, 1, 16, 4)
    ptr = [0] * (5 + 1)
    out, lse = oracle.attn_rows_bs(q, k, v, cu, tile, ptr, [], 0.25,
                                   np.arange(40), np.zeros(40, dtype=np.int32))
    assert np.all(out == 0) and np.all(np.isneginf(lse))


def test_oracle_full_lists_equal_causal_attention():
    cu, tile = [0, 100, 230], 16
    q, k, v = draw_qkv(cu, 4, 1, 32, 5)
    ptr, idx = random_lists(cu, tile, 1.0, 5)
    tok = np.arange(cu[-1])
    head = np.arange(cu[-1]) % 4
    a, la = oracle.attn_rows_bs(q, k, v, cu, tile, ptr, idx, 0.2, tok, head)
    b, lb = oracle.attn_rows(q, k, v, cu, "causal", 0, 1, 0, 0.2, tok, head)
    assert np.array_equal(a, b) and np.array_equal(la, lb)


# ---- schedule --------------------------------------------------------------

def _items(words):
    n_items, n_merges, n_lists = words[11], words[12], words[6]
    items = words[16:16 + 12 * n_items].reshape(-1, 12)
    m0 = 16 + 12 * n_items
    merges = words[m0:m0 + 8 * n_merges].reshape(-1, 8)
    lists = words[m0 + 8 * n_merges:]
    assert lists.size == n_lists
    return items, merges, lists


@pytest.mark.parametrize("max_tiles", [0, 1, 2, 5])
def test_oracle_schedule_follows_the_packing_rule(max_tiles):
    cu, tile = [0, 1000, 1000, 1700], 64
    ptr, idx = random_lists(cu, tile, 0.5, 7, diag=True)
    words = oracle.schedule_bs(cu, tile, ptr, idx, max_tiles)
    nq = sum(-(-(cu[b + 1] - cu[b]) // tile) for b in range(len(cu) - 1))
    bound = max_tiles or max(16, -(-2 * len(idx) // nq))
    items, merges, lists = _items(words)
    # every listed tile meets the mask (all lie on or below the diagonal), so
    # the appended lists are the caller's lists in q-tile order
    assert words[2] == 2 and words[14] == len(idx) and np.array_equal(lists, idx)
    # every q-tile's items are balanced chunks that cover its list in order
    chunks = {}
    for it in items:
        off, n, r0, r1, ka0, ka1, kb0, kb1, mode, pb, cost, _ = (int(x) for x in it)
        assert mode == 2 and kb0 == kb1 == 0 and cost == ka1 <= bound
        chunks.setdefault((off, r0), []).append((ka0, ka1))
    g = 0
    for b in range(len(cu) - 1):
        for t, lst in enumerate(lists_of_seq(cu, tile, ptr, idx, b)):
            mine = sorted(chunks.pop((cu[b], t * tile)))
            assert mine[0][0] == ptr[g + t]
            assert sum(c for _, c in mine) == len(lst)
            for (a0, c0), (a1, _) in zip(mine, mine[1:]):
                assert a1 == a0 + c0
            sizes = [c for _, c in mine]
            assert len(sizes) == max(1, -(-len(lst) // bound))
            assert max(sizes) - min(sizes) <= 1
        g += -(-(cu[b + 1] - cu[b]) // tile)
    assert not chunks
    # split items: contiguous partial slots per q-tile, one merge each
    split = items[items[:, 9] >= 0]
    assert words[13] == sum(int(m[3]) * (int(m[2]) - int(m[1])) for m in merges)
    for m in merges:
        off, r0, r1, ns, pb = (int(x) for x in m[:5])
        mine = split[(split[:, 0] == off) & (split[:, 2] == r0)]
        assert len(mine) == ns >= 2
        assert sorted(int(x) for x in mine[:, 9]) == [pb + c * (r1 - r0) for c in range(ns)]
    # order: split items first, each group by decreasing cost
    nsplit = len(split)
    assert np.all(items[:nsplit, 9] >= 0) and np.all(items[nsplit:, 9] < 0)
    for grp in (items[:nsplit], items[nsplit:]):
        assert np.all(np.diff(grp[:, 10]) <= 0)


def test_automatic_bound_cuts_only_long_lists():
    # 40 q-tiles of 64: the last lists all 40 k-tiles, the others only the
    # diagonal, so the mean is 79 / 40 and the automatic bound is 16
    cu, tile = [0, 40 * 64], 64
    ptr, idx = [0], []
    for t in range(40):
        idx.extend(range(40) if t == 39 else [t])
        ptr.append(len(idx))
    words = oracle.schedule_bs(cu, tile, ptr, idx, 0)
    assert np.array_equal(words, B.ta_build_blocksparse_schedule(cu, tile, ptr, idx, 0)[0])
    items, merges, _ = _items(words)
    assert len(merges) == 1 and int(merges[0][1]) == 39 * 64 and int(merges[0][3]) == 3
    assert sorted(int(x) for x in items[:, 10]) == [1] * 39 + [13, 13, 14]
    # uniform lists (every q-tile lists everything up to the diagonal): the
    # longest is about twice the mean, so nothing is cut
    ptr, idx = random_lists(cu, tile, 1.0, 0)
    words = oracle.schedule_bs(cu, tile, ptr, idx, 0)
    assert words[12] == 0 and words[11] == 40


@pytest.mark.parametrize("seed", range(6))
@pytest.mark.parametrize("tile", [64, 128])
@pytest.mark.parametrize("max_tiles", [0, 1, 3, 100])
def test_builder_matches_oracle_schedule(seed, tile, max_tiles):
    rng = np.random.default_rng(seed)
    lens = [int(x) for x in rng.integers(0, 1500, size=3)] + [0, 1]
    cu = [0]
    for n in lens:
        cu.append(cu[-1] + n)
    density = [0.05, 0.3, 0.9][seed % 3]
    ptr, idx = random_lists(cu, tile, density, seed + 100,
                            diag=[None, True, False][seed % 3])
    words, info = B.ta_build_blocksparse_schedule(cu, tile, ptr, idx, max_tiles)
    want = oracle.schedule_bs(cu, tile, ptr, idx, max_tiles)
    assert np.array_equal(words, want)
    assert info.kind == B.BLOCKSPARSE and info.kept_tiles_per_qhead == len(idx)
    assert info.n_items == words[11] and info.n_merge_items == words[12]


def test_builder_empty_and_full_lists():
    cu, tile = [0, 300], 64
    words, info = B.ta_build_blocksparse_schedule(cu, tile, [0] * 6, [])
    items, merges, lists = _items(words)
    assert info.n_items == 5 and info.n_merge_items == 0 and info.kept_tiles_per_qhead == 0
    assert lists.size == 0 and np.all(items[:, 5:8] == 0) and np.all(items[:, 8] == 2)
    # full lists with a large bound: one item per q-tile over its whole list
    ptr, idx = random_lists(cu, tile, 1.0, 0)
    words, info = B.ta_build_blocksparse_schedule(cu, tile, ptr, idx, 100)
    items, _, lists = _items(words)
    assert info.n_merge_items == 0 and np.array_equal(lists, idx)
    for it in items:
        qt = it[2] // tile
        assert it[4] == ptr[qt] and it[5] == qt + 1 and it[6] == it[7] == 0


def _status(cu, tile, ptr, idx, max_tiles=0):
    cu = np.asarray(cu, dtype=np.int32)
    ptr = np.asarray(ptr, dtype=np.int32)
    idx = np.asarray(idx, dtype=np.int32)
    info = B.ScheduleInfo()
    return B.lib().ta_build_blocksparse_schedule(
        cu.ctypes.data, cu.size - 1, tile, ptr.ctypes.data,
        idx.ctypes.data if idx.size else None, max_tiles, None, 0, ctypes.byref(info))


def test_builder_rejects_bad_lists():
    cu = [0, 200]  # 4 q-tiles of 64
    ok = ([0, 1, 2, 4, 5], [0, 0, 1, 2, 3])  # q-tiles: [0] [0] [1 2] [3]
    assert _status(cu, 64, *ok) == B.TA_OK
    bad = B.TA_ERR_INVALID_ARG
    assert _status(cu, 64, [0, 1, 2, 4, 5], [1, 0, 1, 2, 3]) == bad  # above the diagonal
    assert _status(cu, 64, [0, 1, 2, 4, 5], [0, 0, 1, 1, 3]) == bad  # repeated
    assert _status(cu, 64, [0, 1, 2, 4, 5], [0, 0, 2, 1, 3]) == bad  # descending
    assert _status(cu, 64, [0, 1, 2, 4, 5], [0, -1, 1, 2, 3]) == bad  # negative
    assert _status(cu, 64, [0, 1, 0, 4, 5], [0, 0, 1, 2, 3]) == bad  # ptr decreases
    assert _status(cu, 64, [1, 1, 2, 4, 5], [0, 0, 1, 2, 3]) == bad  # ptr[0] != 0
    assert _status(cu, 64, [0, 1, 2, 4, 5], []) == bad  # NULL idx
    assert _status(cu, 32, *ok) == B.TA_ERR_UNSUPPORTED
    assert _status(cu, 64, *ok, max_tiles=-1) == B.TA_ERR_INVALID_ARG
    with pytest.raises(ValueError):
        oracle.schedule_bs(cu, 64, [0, 1, 2, 4, 5], [1, 0, 1, 2, 3])
