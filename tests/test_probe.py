"""The region-contribution probe (Sec. 2.2, Grad(M-hat, l) over the sections
of Appendix A.3) on the CPU: the oracle pinned against torch autograd of the
paper's own construction (a probing variable theta multiplying the attention
probabilities), against the identity sum_j A_ij <dO_i, V_j> = <dO_i, O_i>, and
its section counts against the pinned mask counts."""
import math

import numpy as np
import pytest
import torch

import oracle
from paper_2507_21526_amd.inputs import draw_dout, draw_qkv


def _sections(n, S, W, L):
    """Boolean [3, n, n] masks of the sections (streaming, middle, last),
    written from Appendix A.3 with 0-indexed rows and keys."""
    i, j = np.meshgrid(np.arange(n), np.arange(n), indexing="ij")
    causal = j <= i
    stream = causal & ((j < S) | (i - j < W))
    last_row = i >= n - min(L, n)
    return np.stack([stream, causal & ~stream & ~last_row, causal & ~stream & last_row])


def _autograd_probe(q, k, v, dout, cu, S, W, L, scale):
    """theta = 1 multiplies the causal softmax probabilities; y = <O, dO>
    makes dO the upstream gradient; theta.grad summed per section."""
    total, hq, d = q.shape
    g = hq // k.shape[1]
    sums = np.zeros((hq, 3))
    lse = np.zeros((hq, total))
    for b in range(len(cu) - 1):
        off, n = cu[b], cu[b + 1] - cu[b]
        if n == 0:
            continue
        sec = _sections(n, S, W, L)
        for h in range(hq):
            Q = q[off:off + n, h].double()
            K = k[off:off + n, h // g].double()
            V = v[off:off + n, h // g].double()
            dO = dout[off:off + n, h].double()
            z = scale * Q @ K.T
            z = z.masked_fill(~torch.ones(n, n, dtype=torch.bool).tril(), -math.inf)
            A = torch.softmax(z, dim=-1)
            lse[h, off:off + n] = torch.logsumexp(z, dim=-1).numpy()
            theta = torch.ones(n, n, dtype=torch.float64, requires_grad=True)
            O = (theta * A) @ V
            (O * dO).sum().backward()
            grad = theta.grad.numpy()
            for r in range(3):
                sums[h, r] += grad[sec[r]].sum()
    return sums, lse


@pytest.mark.parametrize("cu,hq,hkv,d,S,W,L", [
    ([0, 29, 29, 61], 4, 2, 16, 3, 5, 4),
    ([0, 40], 2, 1, 32, 0, 1, 0),       # no sink, window 1, no Last rows
    ([0, 17, 50], 3, 3, 16, 4, 64, 9),  # window covers the sequence
    ([0, 6], 2, 1, 16, 2, 2, 10),       # every row is a Last row
])
def test_probe_matches_autograd(cu, hq, hkv, d, S, W, L):
    q, k, v = draw_qkv(cu, hq, hkv, d, 11)
    dout = draw_dout(cu, hq, d, 12)
    scale = 1.0 / math.sqrt(d)
    want, lse = _autograd_probe(q, k, v, dout, cu, S, W, L, scale)
    got, got_abs = oracle.region_grad(q, k, v, dout, lse, cu, S, W, L, scale)
    assert np.all(got_abs >= np.abs(got))
    assert np.allclose(got, want, rtol=0, atol=1e-12 * max(1.0, got_abs.max()))


def test_probe_rows_sum_to_dout_dot_output():
    # sum_j A_ij <dO_i, V_j> = <dO_i, O_i>: the three sections partition the
    # causal pairs, so their sums add up to sum_i <dO_i, O_i> per head
    cu, hq, hkv, d, scale = [0, 300, 555], 4, 1, 32, 0.2
    q, k, v = draw_qkv(cu, hq, hkv, d, 21)
    dout = draw_dout(cu, hq, d, 22)
    out, lse = oracle.attn_full(q, k, v, cu, "causal", 0, 1, 0, scale)
    sums, abs_sums = oracle.region_grad(q, k, v, dout, lse, cu, 16, 40, 30, scale)
    want = np.einsum("thd,thd->h", dout.double().numpy(), out)
    assert np.allclose(sums.sum(axis=1), want, rtol=0, atol=1e-10 * abs_sums.sum())
    assert np.all(sums[:, 1] != 0) and np.all(sums[:, 2] != 0)


def test_probe_zero_upstream_gradient():
    cu, hq, d = [0, 50], 2, 16
    q, k, v = draw_qkv(cu, hq, 1, d, 31)
    _, lse = oracle.attn_full(q, k, v, cu, "causal", 0, 1, 0, 0.25)
    zero = torch.zeros(50, hq, d, dtype=torch.bfloat16)
    sums, abs_sums = oracle.region_grad(q, k, v, zero, lse, cu, 4, 8, 8, 0.25)
    assert np.all(sums == 0) and np.all(abs_sums == 0)


@pytest.mark.parametrize("n,S,W,L", [(1, 0, 1, 0), (100, 3, 7, 11), (100, 0, 1, 100),
                                     (257, 64, 128, 128), (64, 80, 8, 3), (90, 5, 200, 0)])
def test_region_counts_match_mask_counts(n, S, W, L):
    # streaming = the Triangle mask with no Last rows; last = what the Last
    # rows add to it; middle = causal minus Triangle
    stream = oracle.mask_nnz("triangle", n, S, W, 0)
    tri = oracle.mask_nnz("triangle", n, S, W, L)
    causal = oracle.mask_nnz("causal", n, S, W, L)
    assert list(oracle.region_counts([0, n], S, W, L)) == [stream, causal - tri, tri - stream]


def test_region_counts_of_packed_sequences_add():
    parts = [oracle.region_counts([0, n], 64, 128, 128) for n in (2048, 0, 700)]
    assert np.array_equal(oracle.region_counts([0, 2048, 2048, 2748], 64, 128, 128),
                          sum(parts))


# ---- library host functions (no GPU) ---------------------------------------

from paper_2507_21526_amd import binding as B  # noqa: E402


@pytest.mark.parametrize("cu,S,W,L", [
    ([0, 2048], 64, 128, 128), ([0, 0, 1, 100, 357], 3, 7, 11), ([0, 64], 80, 8, 3),
    ([0, 90, 200], 5, 200, 0), ([0, 300], 0, 0, 10), ([0], 1, 1, 1),
])
def test_library_region_counts_match_oracle(cu, S, W, L):
    assert np.array_equal(B.ta_region_counts(cu, S, W, L), oracle.region_counts(cu, S, W, L))


def test_library_region_counts_at_128k():
    # the 128K layer with the probe's sections, against the mask counts
    n, S, W, L = 131072, 64, 128, 128
    stream = oracle.mask_nnz("triangle", n, S, W, 0)
    tri = oracle.mask_nnz("triangle", n, S, W, L)
    causal = n * (n + 1) // 2
    assert list(B.ta_region_counts([0, n], S, W, L)) == [stream, causal - tri, tri - stream]


def test_region_grad_mean():
    rng = np.random.default_rng(5)
    sums = rng.standard_normal((8, 3))
    counts = np.array([100, 0, 7])
    got = B.ta_region_grad_mean(sums, counts)
    assert got[1] == 0.0
    assert np.allclose(got[[0, 2]], sums.sum(axis=0)[[0, 2]] / (8 * counts[[0, 2]]),
                       rtol=1e-15, atol=0)


@pytest.mark.parametrize("seed", range(5))
def test_select_triangle_layers_brute_force(seed):
    rng = np.random.default_rng(seed)
    n = int(rng.integers(1, 40))
    g = np.round(rng.standard_normal(n), 1)  # rounding makes ties
    for k in (0, 1, n // 2, n):
        want = sorted(sorted(range(n), key=lambda l: (abs(g[l]), l))[:k])
        assert B.ta_select_triangle_layers(g, k) == want


def test_select_triangle_layers_rejects_bad_input():
    with pytest.raises(B.TriAttnError):
        B.ta_select_triangle_layers([0.1, float("nan")], 1)
    with pytest.raises(B.TriAttnError):
        B.ta_select_triangle_layers([0.1, 0.2], 3)


def test_probe_rejects_bad_arguments_without_launching():
    import ctypes
    FAKE = 0x10000  # never dereferenced: every call below fails its checks first
    _, cau = B.ta_build_schedule("causal", [0, 100], 0, 1, 0, 64)
    _, tri = B.ta_build_schedule("triangle", [0, 100], 4, 8, 2, 64)
    ws = B.ta_probe_workspace_bytes(cau, 8)
    # one fp64 partial per (slot, 32-row block, head, section), at most 512
    # slots per (kv head, row block)
    assert ws == 512 * 2 * 8 * 3 * 8

    def call(info=cau, total=100, hq=8, hkv=2, d=128, scale=0.1, S=4, W=8, L=2,
             sums=FAKE, ws_ptr=FAKE, ws_bytes=ws, ptr=FAKE):
        p = ctypes.c_void_p(ptr)
        return B.lib().region_grad_probe(
            p, p, p, p, p, p, ctypes.byref(info) if info is not None else None,
            total, hq, hkv, d, scale, S, W, L, ctypes.c_void_p(sums),
            ctypes.c_void_p(ws_ptr), ws_bytes, None)

    assert call(info=None) == B.TA_ERR_INVALID_ARG
    assert call(info=tri) == B.TA_ERR_SCHEDULE_MISMATCH
    assert call(total=99) == B.TA_ERR_SCHEDULE_MISMATCH
    assert call(hq=7) == B.TA_ERR_INVALID_ARG
    assert call(hq=18) == B.TA_ERR_UNSUPPORTED
    assert call(d=96) == B.TA_ERR_UNSUPPORTED
    assert call(scale=0.0) == B.TA_ERR_INVALID_ARG
    assert call(W=-1) == B.TA_ERR_INVALID_ARG
    assert call(sums=0) == B.TA_ERR_INVALID_ARG
    assert call(sums=FAKE + 4) == B.TA_ERR_INVALID_ARG
    assert call(ptr=0) == B.TA_ERR_INVALID_ARG
    assert call(ptr=FAKE + 8) == B.TA_ERR_INVALID_ARG
    assert call(ws_ptr=0) == B.TA_ERR_WORKSPACE
    assert call(ws_bytes=ws - 1) == B.TA_ERR_WORKSPACE
    bad = B.ScheduleInfo.from_buffer_copy(cau)
    bad.words += 1
    assert call(info=bad) == B.TA_ERR_SCHEDULE_MISMATCH
