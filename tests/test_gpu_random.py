"""GPU parity of Triangle and dense causal attention against the fp64 oracle
on seeded random configurations (full outputs): packed batches with empty
and length-1 sequences, GQA group 1 to 8, d 64 and 128, tiles of 64 and 128,
random sink, window and Last-row counts (Appendix A.3 sections) and split
counts.  Complements the hand-picked edge shapes."""
import numpy as np
import pytest

from tests.test_gpu_kernels import _full_check

pytestmark = pytest.mark.gpu


def _config(seed):
    rng = np.random.default_rng(7000 + seed)
    nseq = int(rng.integers(1, 4))
    lens = [int(x) for x in rng.integers(0, 1400, size=nseq)]
    if seed % 4 == 0:
        lens.append(1)
    if seed % 5 == 0:
        lens.insert(0, 0)
    cu = [0]
    for n in lens:
        cu.append(cu[-1] + n)
    group = int(rng.integers(1, 9))
    hkv = int(rng.integers(1, 3))
    d = int(rng.choice([64, 128]))
    tile = int(rng.choice([64, 128]))
    sink = int(rng.integers(0, 300))
    window = int(rng.integers(1, 1200))
    last = int(rng.integers(0, 400))
    splits = int(rng.choice([0, 0, 1, 3]))
    return cu, group * hkv, hkv, d, sink, window, last, tile, splits


@pytest.mark.parametrize("seed", range(12))
def test_random_triangle(seed):
    cu, hq, hkv, d, S, W, L, T, splits = _config(seed)
    _full_check("triangle", cu, hq, hkv, d, S, W, L, T, splits, seed=seed,
                label=f"random {seed}: cu={cu} hq={hq} hkv={hkv} d={d} S={S} W={W} "
                      f"L={L} T={T} splits={splits}")


@pytest.mark.parametrize("seed", range(4))
def test_random_causal(seed):
    cu, hq, hkv, d, _, _, _, T, _ = _config(100 + seed)
    _full_check("causal", cu, hq, hkv, d, 0, 1, 0, T, 0, seed=seed,
                label=f"random causal {seed}: cu={cu} hq={hq} hkv={hkv} d={d} T={T}")
