"""fp64 CPU oracle for Triangle attention and dense causal attention.

TEST INFRASTRUCTURE ONLY.  Only the tests, the smoke check and the CPU
baseline leg of the benchmark may import this package; the product path
(`paper_2507_21526_amd`) never does.  The arithmetic lives in ``oracle.c``
(plain C, double precision, OpenMP over rows) and follows the paper:

* masks: the Streaming, Last Q-K and Middle Q-K sections of Appendix A.3,
  Triangle = Streaming + Last Q-K (Sec. 2.4);
* attention: the masked softmax of Sec. 2.1, row by row, masked logits
  removed exactly;
* tile schedule: brute force over every (q-tile, k-tile) block, emitted in
  the documented packed int32 format;
* block-sparse causal attention (the dense layers handed to a dynamic sparse
  method, Sec. 2.4 and Sec. 3.1): a row keeps key j iff j <= i and the
  k-tile of j is listed for the row's q-tile;
* the region-contribution probe of Sec. 2.2: per head and section, the sum
  of A_ij <dO_i, V_j> (the derivative of y with respect to the probing
  variable theta_ij at theta = 1).

This module only marshals arguments through ctypes and compiles the C file
with gcc when no built library is present.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
_LIB_PATH = os.path.join(_HERE, "liboracle.so")

TRIANGLE = 0
CAUSAL = 1

_lib = None


def build(force: bool = True) -> str:
    """Compile oracle.c into liboracle.so next to it (gcc, -O2, OpenMP)."""
    if force or not os.path.exists(_LIB_PATH):
        tmp = _LIB_PATH + ".tmp"
        cmd = ["gcc", "-O3", "-std=c11", "-fopenmp", "-fPIC", "-shared",
               "-Wall", "-Wextra", "-o", tmp, _SRC, "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        build(force=True)
    lib = ctypes.CDLL(_LIB_PATH)
    i64, i32, dbl = ctypes.c_int64, ctypes.c_int32, ctypes.c_double
    vp = ctypes.c_void_p
    lib.oracle_in_streaming.argtypes = [i64, i64, i64, i64]
    lib.oracle_in_last.argtypes = [i64, i64, i64, i64, i64, i64]
    lib.oracle_in_middle.argtypes = [i64, i64, i64, i64, i64, i64]
    lib.oracle_mask.argtypes = [ctypes.c_int, i64, i64, i64, i64, i64, i64]
    lib.oracle_mask_row.argtypes = [ctypes.c_int, i64, i64, i64, i64, i64, vp]
    lib.oracle_mask_row.restype = None
    lib.oracle_mask_nnz.argtypes = [ctypes.c_int, i64, i64, i64, i64]
    lib.oracle_mask_nnz.restype = i64
    lib.oracle_attn_rows.argtypes = [vp, vp, vp, vp, i32, i32, i32, i32,
                                     ctypes.c_int, i64, i64, i64, dbl,
                                     vp, vp, i64, vp, vp]
    lib.oracle_attn_rows.restype = ctypes.c_int
    lib.oracle_attn_rows_absw.argtypes = list(lib.oracle_attn_rows.argtypes) + [vp]
    lib.oracle_attn_rows_absw.restype = ctypes.c_int
    lib.oracle_schedule.argtypes = [ctypes.c_int, vp, i32, i32, i32, i32, i32,
                                    i32, vp, i64]
    lib.oracle_schedule.restype = i64
    lib.oracle_bs_mask.argtypes = [i64, i64, i64, vp, i64]
    lib.oracle_bs_mask.restype = ctypes.c_int
    lib.oracle_attn_rows_bs.argtypes = [vp, vp, vp, vp, i32, i32, i32, i32, i32,
                                        vp, vp, dbl, vp, vp, i64, vp, vp]
    lib.oracle_attn_rows_bs.restype = ctypes.c_int
    lib.oracle_bs_schedule.argtypes = [vp, i32, i32, vp, vp, i32, vp, i64]
    lib.oracle_bs_schedule.restype = i64
    lib.oracle_region_grad.argtypes = [vp, vp, vp, vp, vp, vp, i32, i32, i32, i32,
                                       i64, i64, i64, dbl, vp, vp]
    lib.oracle_region_grad.restype = ctypes.c_int
    lib.oracle_region_counts.argtypes = [vp, i32, i64, i64, i64, vp]
    lib.oracle_region_counts.restype = ctypes.c_int
    lib.oracle_num_threads.restype = ctypes.c_int
    _lib = lib
    return lib


def _kind(kind) -> int:
    if kind in (TRIANGLE, "triangle"):
        return TRIANGLE
    if kind in (CAUSAL, "causal"):
        return CAUSAL
    raise ValueError(f"unknown kind {kind!r}")


def _bf16_bits(t) -> np.ndarray:
    """Raw bf16 bit patterns of a torch bf16 tensor (or a uint16 array)."""
    if isinstance(t, np.ndarray):
        assert t.dtype == np.uint16
        return np.ascontiguousarray(t)
    import torch
    assert t.dtype == torch.bfloat16, t.dtype
    return t.detach().cpu().contiguous().view(torch.int16).numpy().view(np.uint16)


def num_threads() -> int:
    return int(load().oracle_num_threads())


def in_streaming(i, j, sink, window) -> bool:
    return bool(load().oracle_in_streaming(i, j, sink, window))


def in_last(i, j, n, sink, window, last) -> bool:
    return bool(load().oracle_in_last(i, j, n, sink, window, last))


def in_middle(i, j, n, sink, window, last) -> bool:
    return bool(load().oracle_in_middle(i, j, n, sink, window, last))


def mask_row(kind, n, sink, window, last, i) -> np.ndarray:
    row = np.zeros(n, dtype=np.uint8)
    load().oracle_mask_row(_kind(kind), n, sink, window, last, i,
                           row.ctypes.data)
    return row


def mask_matrix(kind, n, sink, window, last) -> np.ndarray:
    """Full n x n mask (small n only)."""
    return np.stack([mask_row(kind, n, sink, window, last, i) for i in range(n)]) \
        if n > 0 else np.zeros((0, 0), np.uint8)


def mask_nnz(kind, n, sink, window, last) -> int:
    return int(load().oracle_mask_nnz(_kind(kind), n, sink, window, last))


def attn_rows(q, k, v, cu_seqlens, kind, sink, window, last, scale,
              row_tok, row_head, with_absw=False):
    """fp64 output rows and natural-log LSE for (token, query head) pairs.

    q: [total, Hq, d], k/v: [total, Hkv, d] as torch bf16 (or uint16 bits).
    Returns (out [nrows, d] float64, lse [nrows] float64), and with
    ``with_absw`` also absw [nrows, d]: sum_j p_j |v_j| per element (the
    probability-weighted mean of |v|, which bounds the effect of relative
    rounding errors in the probabilities on the output).
    """
    qb, kb, vb = _bf16_bits(q), _bf16_bits(k), _bf16_bits(v)
    total, hq, d = qb.shape
    hkv = kb.shape[1]
    cu = np.ascontiguousarray(np.asarray(cu_seqlens, dtype=np.int32))
    assert cu[-1] == total and kb.shape == (total, hkv, d) and vb.shape == kb.shape
    rt = np.ascontiguousarray(np.asarray(row_tok, dtype=np.int64))
    rh = np.ascontiguousarray(np.asarray(row_head, dtype=np.int32))
    assert rt.shape == rh.shape
    out = np.zeros((rt.size, d), dtype=np.float64)
    lse = np.zeros(rt.size, dtype=np.float64)
    args = (qb.ctypes.data, kb.ctypes.data, vb.ctypes.data, cu.ctypes.data,
            cu.size - 1, hq, hkv, d, _kind(kind), sink, window, last,
            float(scale), rt.ctypes.data, rh.ctypes.data, rt.size,
            out.ctypes.data, lse.ctypes.data)
    if with_absw:
        absw = np.zeros((rt.size, d), dtype=np.float64)
        rc = load().oracle_attn_rows_absw(*args, absw.ctypes.data)
    else:
        rc = load().oracle_attn_rows(*args)
    if rc != 0:
        raise ValueError("oracle_attn_rows rejected the request")
    return (out, lse, absw) if with_absw else (out, lse)


def attn_full(q, k, v, cu_seqlens, kind, sink, window, last, scale):
    """Every (token, head) row: returns out [total, Hq, d], lse [Hq, total]."""
    total, hq, d = tuple(q.shape)
    tok = np.repeat(np.arange(total, dtype=np.int64), hq)
    head = np.tile(np.arange(hq, dtype=np.int32), total)
    out, lse = attn_rows(q, k, v, cu_seqlens, kind, sink, window, last, scale,
                         tok, head)
    return out.reshape(total, hq, d), lse.reshape(total, hq).T.copy()


def schedule(kind, cu_seqlens, sink, window, last, tile, splits=0) -> np.ndarray:
    """Brute-force tile schedule in the packed int32 format."""
    cu = np.ascontiguousarray(np.asarray(cu_seqlens, dtype=np.int32))
    lib = load()
    words = lib.oracle_schedule(_kind(kind), cu.ctypes.data, cu.size - 1, sink,
                                window, last, tile, splits, None, 0)
    if words < 0:
        raise ValueError("oracle_schedule rejected the parameters")
    out = np.zeros(words, dtype=np.int32)
    got = lib.oracle_schedule(_kind(kind), cu.ctypes.data, cu.size - 1, sink,
                              window, last, tile, splits, out.ctypes.data, words)
    assert got == words
    return out


# ---- block-sparse causal attention ----------------------------------------

def _csr(qtile_ptr, ktile_idx):
    ptr = np.ascontiguousarray(np.asarray(qtile_ptr, dtype=np.int32))
    idx = np.ascontiguousarray(np.asarray(ktile_idx, dtype=np.int32))
    if idx.size == 0:
        idx = np.zeros(1, dtype=np.int32)  # valid pointer, never read
    return ptr, idx


def bs_mask_row(i, n, tile, kept_tiles) -> np.ndarray:
    """Mask row i (sequence-relative) given the k-tile list of its q-tile."""
    lst = np.ascontiguousarray(np.asarray(kept_tiles, dtype=np.int32))
    if lst.size == 0:
        lst = np.zeros(1, dtype=np.int32)
        ln = 0
    else:
        ln = lst.size
    lib = load()
    return np.array([lib.oracle_bs_mask(i, j, tile, lst.ctypes.data, ln)
                     for j in range(n)], dtype=np.uint8)


def bs_mask_matrix(n, tile, lists) -> np.ndarray:
    """Full n x n block-sparse mask of one sequence; lists[t] = k-tiles of
    q-tile t (small n only)."""
    return np.stack([bs_mask_row(i, n, tile, lists[i // tile]) for i in range(n)]) \
        if n > 0 else np.zeros((0, 0), np.uint8)


def attn_rows_bs(q, k, v, cu_seqlens, tile, qtile_ptr, ktile_idx, scale,
                 row_tok, row_head):
    """Block-sparse causal attention rows: (out [nrows, d], lse [nrows])."""
    qb, kb, vb = _bf16_bits(q), _bf16_bits(k), _bf16_bits(v)
    total, hq, d = qb.shape
    hkv = kb.shape[1]
    cu = np.ascontiguousarray(np.asarray(cu_seqlens, dtype=np.int32))
    ptr, idx = _csr(qtile_ptr, ktile_idx)
    rt = np.ascontiguousarray(np.asarray(row_tok, dtype=np.int64))
    rh = np.ascontiguousarray(np.asarray(row_head, dtype=np.int32))
    out = np.zeros((rt.size, d), dtype=np.float64)
    lse = np.zeros(rt.size, dtype=np.float64)
    rc = load().oracle_attn_rows_bs(qb.ctypes.data, kb.ctypes.data, vb.ctypes.data,
                                    cu.ctypes.data, cu.size - 1, hq, hkv, d, tile,
                                    ptr.ctypes.data, idx.ctypes.data, float(scale),
                                    rt.ctypes.data, rh.ctypes.data, rt.size,
                                    out.ctypes.data, lse.ctypes.data)
    if rc != 0:
        raise ValueError("oracle_attn_rows_bs rejected the request")
    return out, lse


def schedule_bs(cu_seqlens, tile, qtile_ptr, ktile_idx, max_tiles=0) -> np.ndarray:
    """Block-sparse schedule in the packed int32 format."""
    cu = np.ascontiguousarray(np.asarray(cu_seqlens, dtype=np.int32))
    ptr, idx = _csr(qtile_ptr, ktile_idx)
    lib = load()
    words = lib.oracle_bs_schedule(cu.ctypes.data, cu.size - 1, tile, ptr.ctypes.data,
                                   idx.ctypes.data, max_tiles, None, 0)
    if words < 0:
        raise ValueError("oracle_bs_schedule rejected the lists")
    out = np.zeros(words, dtype=np.int32)
    got = lib.oracle_bs_schedule(cu.ctypes.data, cu.size - 1, tile, ptr.ctypes.data,
                                 idx.ctypes.data, max_tiles, out.ctypes.data, words)
    assert got == words
    return out


REGIONS = ("streaming", "middle", "last")


def region_grad(q, k, v, dout, lse, cu_seqlens, sink, window, last, scale):
    """Per query head and section (streaming, middle, last): the sum of
    A_ij <dO_i, V_j> and the sum of its absolute values, fp64.

    q, dout: [total, Hq, d]; k, v: [total, Hkv, d] (torch bf16 or uint16
    bits); lse: [Hq, total] natural log (any float array; used as float64).
    Returns (sums [Hq, 3], abs_sums [Hq, 3]).
    """
    qb, kb, vb, db = _bf16_bits(q), _bf16_bits(k), _bf16_bits(v), _bf16_bits(dout)
    total, hq, d = qb.shape
    hkv = kb.shape[1]
    cu = np.ascontiguousarray(np.asarray(cu_seqlens, dtype=np.int32))
    assert cu[-1] == total and db.shape == qb.shape and vb.shape == kb.shape
    ls = np.ascontiguousarray(np.asarray(lse, dtype=np.float64))
    assert ls.shape == (hq, total)
    sums = np.zeros((hq, 3), dtype=np.float64)
    abs_sums = np.zeros((hq, 3), dtype=np.float64)
    rc = load().oracle_region_grad(qb.ctypes.data, kb.ctypes.data, vb.ctypes.data,
                                   db.ctypes.data, ls.ctypes.data, cu.ctypes.data,
                                   cu.size - 1, hq, hkv, d, sink, window, last,
                                   float(scale), sums.ctypes.data, abs_sums.ctypes.data)
    if rc != 0:
        raise ValueError("oracle_region_grad rejected the request")
    return sums, abs_sums


def region_counts(cu_seqlens, sink, window, last) -> np.ndarray:
    """Pairs per head in each section (streaming, middle, last), brute force."""
    cu = np.ascontiguousarray(np.asarray(cu_seqlens, dtype=np.int32))
    out = np.zeros(3, dtype=np.int64)
    if load().oracle_region_counts(cu.ctypes.data, cu.size - 1, sink, window, last,
                                   out.ctypes.data) != 0:
        raise ValueError("oracle_region_counts rejected the request")
    return out
