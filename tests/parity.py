"""Shared helpers of the GPU parity tests: run a pass through the C interface
and compare sampled (row, head) outputs with the fp64 oracle."""
from __future__ import annotations

import math
import sys

import numpy as np
import torch

import oracle
from paper_2507_21526_amd import binding

# Parity bar: per head, max-abs <= 1e-2 and relative L2 <= 5e-3 on fp32 output;
# LSE within 1e-3 absolute.
MAX_ABS = 1e-2
REL_L2 = 5e-3
LSE_ABS = 1e-3


def log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def run_pass(kind, q, k, v, cu, sink, window, last, tile, splits=0,
             out_dtype=torch.float32, scale=None, poison=False):
    """q, k, v: cuda bf16.  Returns (o, lse, plan)."""
    d = q.shape[2]
    scale = scale if scale is not None else 1.0 / math.sqrt(d)
    plan = binding.Plan(kind, cu, sink, window, last, tile, q.shape[1], d,
                        splits, device=q.device)
    o = torch.empty(q.shape, dtype=out_dtype, device=q.device)
    lse = torch.empty((q.shape[1], q.shape[0]), dtype=torch.float32,
                      device=q.device)
    if poison:
        o.fill_(float("nan"))
        lse.fill_(float("nan"))
        if plan.workspace is not None:
            plan.workspace.view(torch.uint8).fill_(0xFF)  # NaN bit patterns
    plan.run(q, k, v, o, lse, scale)
    return o, lse, plan


def boundary_rows(n, sink, window, last, tile):
    lr = min(last, n)
    cand = {0, 1, sink - 1, sink, sink + 1, sink + window - 1, sink + window,
            window - 1, window, n - lr - 1, n - lr, n - 1, n - 2}
    for b in (sink, window, sink + window, n - lr):
        for t in (b // tile * tile, b // tile * tile + tile - 1):
            cand.update((t - 1, t, t + 1))
    return sorted(r for r in cand if 0 <= r < n)


def sample_rows(cu, sink, window, last, tile, n_random, seed, all_last=True):
    rng = np.random.default_rng(seed)
    toks = set()
    for b in range(len(cu) - 1):
        off, n = cu[b], cu[b + 1] - cu[b]
        if n == 0:
            continue
        toks.update(off + r for r in boundary_rows(n, sink, window, last, tile))
        if all_last:
            toks.update(off + r for r in range(max(0, n - last), n))
        toks.update(int(off + r) for r in rng.integers(0, n, size=n_random))
    return np.array(sorted(toks), dtype=np.int64)


# Rounding the probabilities to bf16 for the PV product (round to nearest
# even, 8 significant bits) changes each p_j by a relative error of at most
# u = 2^-8, while the normaliser l sums the unrounded fp32 values.  The
# output error of element (i, c) is then sum_j (p'_j - p_j) v_jc / l, at most
# u * sum_j p_j |v_jc| / l = u * absw_ic, a weighted mean of |v| that the
# oracle computes.  Spread-out rows average the rounding errors away (max-abs
# a few 1e-3); rows dominated by one key of large |v| can approach u |v|.
# The factor 1 + 2^-6 covers the fp32 logits, exp2 and accumulation.
P_ROUND_U = 2.0 ** -8
P_BOUND_FACTOR = P_ROUND_U * (1.0 + 2.0 ** -6)
P_BOUND_ABS = 1e-5


def compare(kind, q_cpu, k_cpu, v_cpu, cu, sink, window, last, scale, o, lse,
            toks, heads, label="", max_abs=MAX_ABS, p_bound=False):
    """Check GPU rows o[toks, h] (fp32/bf16 cuda) against the oracle.

    With ``p_bound`` an element may exceed ``max_abs`` only up to the bf16
    probability-rounding bound of that element (P_BOUND_FACTOR * absw +
    P_BOUND_ABS); relative L2 and LSE keep the flat bar."""
    toks = np.asarray(toks, dtype=np.int64)
    heads = list(heads)
    rt = np.repeat(toks, len(heads))
    rh = np.tile(np.array(heads, dtype=np.int32), toks.size)
    if p_bound:
        ref_o, ref_lse, absw = oracle.attn_rows(q_cpu, k_cpu, v_cpu, cu, kind, sink,
                                                window, last, scale, rt, rh,
                                                with_absw=True)
        tol = np.maximum(max_abs, P_BOUND_FACTOR * absw + P_BOUND_ABS)
    else:
        ref_o, ref_lse = oracle.attn_rows(q_cpu, k_cpu, v_cpu, cu, kind, sink,
                                          window, last, scale, rt, rh)
        tol = np.full(ref_o.shape, max_abs)
    idx_t = torch.from_numpy(rt).to(o.device)
    idx_h = torch.from_numpy(rh.astype(np.int64)).to(o.device)
    got_o = o[idx_t, idx_h].double().cpu().numpy()
    got_lse = lse[idx_h, idx_t].double().cpu().numpy()
    worst = {}
    over_flat = 0
    for h in heads:
        sel = rh == h
        err = got_o[sel] - ref_o[sel]
        max_err = float(np.abs(err).max()) if err.size else 0.0
        rel = float(np.linalg.norm(err) / max(np.linalg.norm(ref_o[sel]), 1e-30))
        lse_err = float(np.abs(got_lse[sel] - ref_lse[sel]).max())
        worst[h] = (max_err, rel, lse_err)
        elem_ok = bool((np.abs(err) <= tol[sel]).all())
        over_flat += int((np.abs(err) > MAX_ABS).sum())
        if not (elem_ok and rel <= REL_L2 and lse_err <= LSE_ABS):
            bad = np.argwhere(np.abs(err) > tol[sel])
            rows = sorted(set(int(rt[sel][i]) for i, _ in bad[:20]))
            raise AssertionError(
                f"{label} head {h}: max-abs {max_err:.3e}, rel-L2 {rel:.3e}, "
                f"lse {lse_err:.3e}; first bad tokens {rows[:10]}")
    log(f"{label}: {len(toks)} rows x {len(heads)} heads, worst max-abs "
        f"{max(w[0] for w in worst.values()):.2e} rel-L2 "
        f"{max(w[1] for w in worst.values()):.2e} lse "
        f"{max(w[2] for w in worst.values()):.2e}"
        + (f"; {over_flat} elements above {MAX_ABS:g}, within the bf16-P bound"
           if over_flat else ""))
    return worst
