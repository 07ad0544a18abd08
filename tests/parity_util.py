"""Shared checks of the GPU parity tests (bars documented in test_gpu_parity)."""

import numpy as np
import torch

from oracle import wise_oracle as O

ATOL_MAX, ATOL_MEAN, LSE_TOL, ACC_TOL, TIE = 1e-2, 1e-3, 1e-3, 1e-5, 1e-5


def f64(t):
    return t.detach().float().cpu().numpy().astype(np.float64)


def say(*a):
    print(*a, flush=True)


def attn_errors(gpu, ref):
    g = f64(gpu) if isinstance(gpu, torch.Tensor) else gpu
    err = np.abs(g - ref)
    big = np.abs(ref) >= 4.0
    small_max = err[~big].max() if (~big).any() else 0.0
    big_ratio = (err[big] / (2.0 ** -7 * np.abs(ref[big]))).max() if big.any() else 0.0
    return err, small_max, big_ratio, int(big.sum())


def assert_attn(gpu, ref, what=""):
    err, small_max, big_ratio, nbig = attn_errors(gpu, ref)
    say(f"  {what}: max-abs {err.max():.3g} (|ref|<4: {small_max:.3g}; {nbig} outputs |ref|>=4 "
        f"at {big_ratio:.2f} spacing) mean-abs {err.mean():.3g}")
    assert small_max <= ATOL_MAX and big_ratio <= 1.0 and err.mean() <= ATOL_MEAN, \
        f"{what}: max {err.max():.3g} (small {small_max:.3g}, big {big_ratio:.2f}) mean {err.mean():.3g}"


def assert_lse(gpu, ref, what=""):
    g = f64(gpu) if isinstance(gpu, torch.Tensor) else gpu
    both_inf = np.isneginf(g) & np.isneginf(ref)
    err = np.abs(np.where(both_inf, 0.0, g - ref))
    assert err.max() <= LSE_TOL, f"{what}: lse max {err.max():.3g}"


def rows_of(rp, ci):
    rp = rp.cpu().numpy() if isinstance(rp, torch.Tensor) else rp
    ci = ci.cpu().numpy() if isinstance(ci, torch.Tensor) else ci
    return [list(ci[rp[r]:rp[r + 1]]) for r in range(len(rp) - 1)]


def near_tie(v, qb, tau):
    m = O.support_margins(v, qb, tau)
    return min(m["delta_minus"], m["delta_plus"], m["delta_rank"]) < TIE


def compare_support(gpu_rows, acc_ref, tau, flags, row_ids=None):
    """End-to-end CSR rows vs the oracle's selection on its own accumulator."""
    bt, h, nb, _ = acc_ref.shape
    flat = acc_ref.reshape(bt * h * nb, nb)
    reported = []
    ids = range(bt * h * nb) if row_ids is None else row_ids
    for i, r in enumerate(ids):
        qb = r % nb
        want = O.select_row(flat[r], qb, tau, flags)
        got = [int(x) for x in gpu_rows[i]]
        if got != want:
            assert near_tie(flat[r], qb, tau), f"row {r}: gpu {got} oracle {want}"
            reported.append(r)
    if reported:
        say(f"near-tie CSR rows reported (not failed): {reported[:20]} ({len(reported)})")
    return reported


