"""Seeded synthetic inputs and the workload table.

This module holds no attention arithmetic: it draws the Q/K/V tensors that
both the HIP path and the CPU oracle consume, so that the two sides read the
same bf16 bytes.  Values are drawn in fp32 from a seeded numpy PCG64
generator (i.i.d. N(0, 1), optionally scaled per head or with a boosted
key 0) and rounded once to bf16 (round to nearest even).

The workloads stand in for the attention-kernel latency measurements of the
paper (Sec. 3.4, table of attention kernel latency: Llama-3.1-8B and
Qwen2.5-7B attention layers at 32K to 128K tokens); the shapes are those
models' attention shapes, the values are synthetic.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field

import numpy as np
import torch


@dataclass(frozen=True)
class Workload:
    name: str
    cu_seqlens: tuple
    hq: int
    hkv: int
    d: int
    tile: int
    sink: int
    window: int
    last: int
    seed: int
    head_scale: tuple | None = None      # (lo, hi): per-(tensor, head) U[lo, hi]
    key0_boost: float | None = None      # multiply K[0, :, :] by this factor
    layers: int = 1
    triangle_layers: int = 1             # how many of the layers use Triangle
    note: str = ""

    @property
    def total(self) -> int:
        return int(self.cu_seqlens[-1])

    @property
    def scale(self) -> float:
        return 1.0 / math.sqrt(self.d)


WORKLOADS = {
    "tiny_n1024_d64": Workload(
        "tiny_n1024_d64", (0, 1024), hq=4, hkv=1, d=64, tile=64, sink=64,
        window=256, last=64, seed=1001,
        note="one layer, GQA 4:1, N=1024, d=64"),
    "llama8b_n32k": Workload(
        "llama8b_n32k", (0, 32768), hq=32, hkv=8, d=128, tile=128, sink=128,
        window=2048, last=128, seed=1002, head_scale=(0.5, 2.0),
        note="Llama-3.1-8B attention shape, N=32768, per-head RMS scale"),
    "llama8b_n128k": Workload(
        "llama8b_n128k", (0, 131072), hq=32, hkv=8, d=128, tile=128, sink=128,
        window=2048, last=128, seed=1003, key0_boost=8.0,
        note="Llama-3.1-8B attention shape, N=131072, key 0 with 8x norm"),
    "llama8b_varlen4": Workload(
        "llama8b_varlen4", (0, 8192, 32768, 81920, 147456), hq=32, hkv=8,
        d=128, tile=128, sink=128, window=2048, last=128, seed=1004,
        note="4 packed sequences of 8K, 24K, 48K, 64K tokens"),
    "qwen7b_n128k_stack28": Workload(
        "qwen7b_n128k_stack28", (0, 131072), hq=28, hkv=4, d=128, tile=128,
        sink=128, window=4096, last=256, seed=1005, layers=28,
        triangle_layers=20,
        note="Qwen2.5-7B attention shape, 28 layers: 20 Triangle, 8 dense"),
    "qwen7b_n128k_layer": Workload(
        "qwen7b_n128k_layer", (0, 131072), hq=28, hkv=4, d=128, tile=128,
        sink=128, window=4096, last=256, seed=1005,
        note="one Triangle layer of the Qwen2.5-7B stack (GQA 7:1), for "
             "per-layer timing and counters"),
    "triangle_n1m_g8": Workload(
        "triangle_n1m_g8", (0, 1048576), hq=8, hkv=1, d=128, tile=128,
        sink=128, window=2048, last=128, seed=1007,
        note="maximum-size check: one 1M-token sequence, 8 query heads on one "
             "kv head (64-bit addressing, Last rows split 456 ways)"),
    "mha_n32k": Workload(
        "mha_n32k", (0, 32768), hq=32, hkv=32, d=128, tile=128, sink=128,
        window=2048, last=128, seed=1008,
        note="multi-head attention (GQA group 1, the Llama-2-7B attention "
             "shape), N=32768: four-wave workgroups, two per CU"),
    "llama8b_probe_n2048": Workload(
        "llama8b_probe_n2048", (0, 2048), hq=32, hkv=8, d=128, tile=128,
        sink=64, window=128, last=128, seed=1006,
        note="region-contribution probe: a ~2K-token prompt of one Llama-3.1-8B "
             "layer, sections with si 64, sl 128, last 128 (App. A.3)"),
}


def draw_qkv(cu_seqlens, hq: int, hkv: int, d: int, seed: int,
             head_scale=None, key0_boost=None):
    """Seeded bf16 Q [T, Hq, d], K and V [T, Hkv, d] on the CPU.

    Draw order from one numpy PCG64 generator: Q, K, V (N(0, 1) fp32), then,
    if ``head_scale`` is given, per-head factors U[lo, hi] for Q (Hq values),
    K and V (Hkv values each).  ``key0_boost`` multiplies the key of token 0
    of every kv head.  A single rounding to bf16 ends the draw.
    """
    total = int(cu_seqlens[-1])
    rng = np.random.default_rng(int(seed))
    q = rng.standard_normal((total, hq, d), dtype=np.float32)
    k = rng.standard_normal((total, hkv, d), dtype=np.float32)
    v = rng.standard_normal((total, hkv, d), dtype=np.float32)
    if head_scale is not None:
        lo, hi = head_scale
        sq = rng.uniform(lo, hi, hq).astype(np.float32)
        sk = rng.uniform(lo, hi, hkv).astype(np.float32)
        sv = rng.uniform(lo, hi, hkv).astype(np.float32)
        q *= sq.reshape(1, hq, 1)
        k *= sk.reshape(1, hkv, 1)
        v *= sv.reshape(1, hkv, 1)
    if key0_boost is not None and total > 0:
        k[0] *= np.float32(key0_boost)
    return tuple(torch.from_numpy(x).to(torch.bfloat16) for x in (q, k, v))


def draw_dout(cu_seqlens, hq: int, d: int, seed: int):
    """Seeded bf16 upstream gradient dO [T, Hq, d] of an attention output
    (i.i.d. N(0, 1) fp32 from numpy PCG64, rounded once to bf16)."""
    total = int(cu_seqlens[-1])
    rng = np.random.default_rng(int(seed))
    g = rng.standard_normal((total, hq, d), dtype=np.float32)
    return torch.from_numpy(g).to(torch.bfloat16)


def blocksparse_lists(n_qtiles: int, density: float, seed: int):
    """Seeded per-q-tile k-tile lists in CSR form (qtile_ptr, ktile_idx) for
    one sequence, standing in for a dynamic sparse method's block estimate:
    q-tile t keeps each earlier k-tile with probability ``density`` (one
    uniform draw per (t, k-tile), numpy PCG64) and always its diagonal tile,
    as block estimators do."""
    rng = np.random.default_rng(int(seed))
    ptr, idx = [0], []
    for t in range(n_qtiles):
        keep = np.flatnonzero(rng.random(t) < density).tolist() + [t]
        idx.extend(keep)
        ptr.append(len(idx))
    return ptr, idx


def workload_qkv(w: Workload, layer: int = 0):
    """Inputs of one layer of a workload (layer l of a stack: seed*1000 + l)."""
    seed = w.seed if w.layers == 1 else w.seed * 1000 + layer
    return draw_qkv(w.cu_seqlens, w.hq, w.hkv, w.d, seed, w.head_scale,
                    w.key0_boost)


def triangle_layer_set(w: Workload, count: int | None = None) -> list:
    """Seeded choice of which layers of a stack use Triangle attention (the
    first ``count`` of one seeded permutation, default the workload's
    number, so a smaller set is a subset of a larger one)."""
    if w.layers == 1:
        return [0]
    gen = torch.Generator(device="cpu").manual_seed(int(w.seed))
    perm = torch.randperm(w.layers, generator=gen)
    count = w.triangle_layers if count is None else count
    return sorted(int(x) for x in perm[:count])
