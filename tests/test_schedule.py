"""Host tile-schedule builder of the library vs the brute-force oracle schedule,
word for word (no GPU needed: the builder is host code)."""
import numpy as np
import pytest

import oracle
from paper_2507_21526_amd import binding
from paper_2507_21526_amd.inputs import WORKLOADS


def _both(kind, cu, S, W, L, T, splits=0):
    got, info = binding.ta_build_schedule(kind, cu, S, W, L, T, splits)
    want = oracle.schedule(kind, cu, S, W, L, T, splits)
    return got, info, want


GRID = [
    # cu_seqlens, sink, window, last, tile
    ([0, 1024], 64, 256, 64, 64),
    ([0, 1], 0, 1, 0, 64),
    ([0, 1], 5, 1, 3, 128),
    ([0, 100], 0, 1, 0, 64),
    ([0, 1000], 8, 512, 50, 64),
    ([0, 1000], 8, 512, 50, 128),
    ([0, 777], 130, 70, 129, 64),
    ([0, 5000], 0, 200, 0, 128),
    ([0, 2048], 64, 128, 128, 64),          # the paper's probing shape
    ([0, 0, 300, 300, 301, 1500], 3, 100, 64, 64),
    ([0, 640, 1280], 128, 1, 1, 128),
    ([0, 4096], 4096, 1, 0, 128),
    ([0, 3000], 10, 10000, 10, 64),
    ([0, 129, 258], 1, 127, 300, 128),
]


@pytest.mark.parametrize("kind", ["triangle", "causal"])
@pytest.mark.parametrize("cu,S,W,L,T", GRID)
def test_schedule_matches_oracle(kind, cu, S, W, L, T):
    got, info, want = _both(kind, cu, S, W, L, T)
    np.testing.assert_array_equal(got, want)
    assert info.words == got.size
    assert info.n_items == got[11] and info.n_merge_items == got[12]
    assert info.n_partial_rows == got[13]
    assert info.kept_tiles_per_qhead == got[14]
    assert info.n_last_rows == got[15]


@pytest.mark.parametrize("splits", [1, 2, 3, 7, 1000])
def test_schedule_explicit_splits(splits):
    for T in (64, 128):
        got, _, want = _both("triangle", [0, 3333, 9000], 16, 300, 200, T,
                             splits)
        np.testing.assert_array_equal(got, want)


@pytest.mark.parametrize("name", ["tiny_n1024_d64", "llama8b_n32k",
                                  "llama8b_varlen4"])
def test_schedule_workloads(name):
    w = WORKLOADS[name]
    for kind in ("triangle", "causal"):
        got, info, want = _both(kind, w.cu_seqlens, w.sink, w.window, w.last,
                                w.tile)
        np.testing.assert_array_equal(got, want)


def test_schedule_workload_counts():
    """Kept k-tiles per query head and item counts of the large workloads,
    from the closed-form counts of the pattern (streaming + Last)."""
    expect = {
        "tiny_n1024_d64": (91, 136),
        "llama8b_n32k": (4693, 32896),
        "llama8b_n128k": (19285, 524800),
        "llama8b_varlen4": (21204, 225856),
        "qwen7b_n128k_stack28": (36234, 524800),
    }
    for name, (tri, cau) in expect.items():
        w = WORKLOADS[name]
        _, ti = binding.ta_build_schedule("triangle", w.cu_seqlens, w.sink,
                                          w.window, w.last, w.tile)
        _, ci = binding.ta_build_schedule("causal", w.cu_seqlens, w.sink,
                                          w.window, w.last, w.tile)
        assert ti.kept_tiles_per_qhead == tri, name
        assert ci.kept_tiles_per_qhead == cau, name
    _, info = binding.ta_build_schedule("triangle", [0, 131072], 128, 2048,
                                        128, 128)
    assert info.n_items == 57 + 1023 and info.max_splits == 57
    assert info.n_partial_rows == 57 * 128 and info.n_last_rows == 128


def test_automatic_split_counts():
    """Reading of the split count (Algorithm 1 leaves it open): a Last q-tile
    with nk kept k-tiles gets ceil(nk / t) splits, t = max(ceil(S/T) +
    ceil(W/T) + 1, ceil(2048/T)); the values below are that arithmetic done
    by hand for the 128K Last q-tile (nk = 1024 at T = 128, 2048 at T = 64)."""
    cases = [
        # S, W, T, expected splits
        (128, 2048, 128, 57),   # t = 1 + 16 + 1 = 18: ceil(1024 / 18)
        (128, 4096, 128, 31),   # t = 1 + 32 + 1 = 34: ceil(1024 / 34)
        (8, 512, 128, 64),      # t = max(1 + 4 + 1, 16) = 16
        (64, 128, 128, 64),     # t = max(1 + 1 + 1, 16) = 16
        (8, 512, 64, 64),       # t = max(1 + 8 + 1, 32) = 32: ceil(2048 / 32)
    ]
    for S, W, T, want in cases:
        _, info = binding.ta_build_schedule("triangle", [0, 131072], S, W, 128, T)
        assert info.max_splits == want, (S, W, T, info.max_splits)
    # a short sequence: the Last q-tile of 1024 tokens has 8 k-tiles, fewer
    # than t = 16, so it is not split (one partial item and its merge)
    _, info = binding.ta_build_schedule("triangle", [0, 1024], 8, 512, 128, 128)
    assert info.max_splits == 1 and info.n_last_items == 1


def test_schedule_llama_128k_matches_oracle():
    w = WORKLOADS["llama8b_n128k"]
    got, _, want = _both("triangle", w.cu_seqlens, w.sink, w.window, w.last,
                         w.tile)
    np.testing.assert_array_equal(got, want)
