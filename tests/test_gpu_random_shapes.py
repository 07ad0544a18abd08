"""Seeded random geometries through the whole path on the GPU: dense
attention with mass pooling, selection, and the late step on the selected
support, each against the oracle on the same bf16 inputs (the grouped late
step bit for bit against the one-row kernel).  Every draw stays
inside the documented limits (head_dim 64/96/128, block 16/32/64/128,
seq_len a multiple of the block and of 64, heads a multiple of kv_heads)."""

import numpy as np
import pytest
import torch

from oracle import wise_oracle as O
from parity_util import ACC_TOL, assert_attn, assert_lse, check_row_vs_oracle, f64, say

pytestmark = pytest.mark.gpu


def draw(seed):
    if seed >= 16:    # seeds 16..: every block size, up to 4 query heads per key-value head
        rng = np.random.default_rng(seed + 7919)
        d = int(rng.choice([64, 96, 128]))
        B = int(rng.choice([16, 32, 64, 128]))
        nb = int(rng.integers(1, 14))
        n = nb * B if B >= 64 else 64 * int(rng.integers(1, 8))
        kvh = int(rng.choice([1, 2, 4]))
        h = kvh * int(rng.choice([1, 2, 3]))
        bt = int(rng.integers(1, 3))
        tau = float(np.float32(rng.choice([0.3, 0.5, 0.8, 0.95, 0.99, 1.0])))
        return bt, h, kvh, n, d, B, tau
    rng = np.random.default_rng(seed)
    d = int(rng.choice([64, 96, 128]))
    B = int(rng.choice([32, 64, 128]))
    if seed >= 12:    # seeds 12..15 draw 16-key blocks
        B = 16
    nb = int(rng.integers(1, 12))
    n = nb * B if B >= 64 else 64 * int(rng.integers(1, 7))
    kvh = int(rng.choice([1, 2]))
    h = kvh * int(rng.choice([1, 2, 3]))
    bt = int(rng.integers(1, 3))
    tau = float(np.float32(rng.choice([0.5, 0.8, 0.95, 1.0])))
    return bt, h, kvh, n, d, B, tau


@pytest.mark.parametrize("seed", range(64))
def test_random_geometry_end_to_end(gpu_lib, seed):
    w = gpu_lib
    bt, h, kvh, n, d, B, tau = draw(seed)
    nb = n // B
    say(f"random geometry seed {seed}: bt={bt} heads={h} kv_heads={kvh} n={n} d={d} B={B} tau={tau}")
    g = torch.Generator().manual_seed(1000 + seed)
    q = (torch.randn((bt, h, n, d), generator=g) * 2.0).to(torch.bfloat16)
    k = torch.randn((bt, kvh, n, d), generator=g).to(torch.bfloat16)
    v = torch.randn((bt, kvh, n, d), generator=g).to(torch.bfloat16)
    qe, ke, ve = f64(q), O.expand_kv(f64(k), h), O.expand_kv(f64(v), h)
    s = w.make_shape(bt, h, n, d, B, kv_heads=kvh)
    qd, kd, vd = q.cuda(), k.cuda(), v.cuda()
    o = torch.empty_like(qd)
    lse = torch.empty((bt, h, n), device="cuda")
    acc = torch.zeros((bt, h, nb, nb), device="cuda")
    w.wise_dense_attn_accum(s, qd, kd, vd, o, lse, acc, w.mass_workspace(s))
    sched = w.Schedule(s).select(acc, tau)
    torch.cuda.synchronize()
    o_ref, l_ref = O.dense_attention(qe, ke, ve)
    assert_attn(o, o_ref, "dense O")
    assert_lse(lse, l_ref, "dense lse")
    r_ref = O.block_mass(qe, ke, B)
    assert np.abs(f64(acc) - r_ref).max() <= ACC_TOL
    # selection: the oracle's own choice on its own masses, near ties reported
    rp_ref, ci_ref = O.select_support(r_ref, tau)
    rp = sched.row_ptr.cpu().numpy()
    ci = sched.col_idx[: int(rp[-1])].cpu().numpy()
    flat = r_ref.reshape(-1, nb)
    agree = np.zeros((bt * h, n), bool)
    for r in range(bt * h * nb):
        if check_row_vs_oracle(ci[rp[r]:rp[r + 1]], flat[r], r % nb, tau, 3, f"row {r}"):
            agree[r // nb, (r % nb) * B:(r % nb + 1) * B] = True
        else:
            say(f"  near-tie row {r} reported")
    o_ref2, l_ref2 = O.sparse_attention(qe, ke, ve, rp_ref, ci_ref, B)
    # the late step on the oracle's support (with its row order), every row
    o2 = torch.empty_like(qd)
    l2 = torch.empty((bt, h, n), device="cuda")
    w.wise_sparse_attn(s, qd, kd, vd, torch.from_numpy(rp_ref).cuda(),
                       torch.from_numpy(ci_ref).cuda(),
                       torch.from_numpy(O.schedule_order(rp_ref, nb)).cuda(), o2, l2)
    torch.cuda.synchronize()
    assert_attn(o2, o_ref2, "sparse O (oracle CSR)")
    assert_lse(l2, l_ref2, "sparse lse (oracle CSR)")
    # the grouped late step on the same support: the same bits (it runs the
    # one-row kernel where the shape has no group)
    o3 = torch.empty_like(qd)
    l3 = torch.empty((bt, h, n), device="cuda")
    w.wise_sparse_attn_grouped(s, qd, kd, vd, torch.from_numpy(rp_ref).cuda(),
                               torch.from_numpy(ci_ref).cuda(), o3, l3)
    torch.cuda.synchronize()
    assert torch.equal(o2, o3) and torch.equal(l2, l3), "grouped late step"
    # and on the GPU's own support, on the rows whose supports agree
    w.wise_sparse_attn(s, qd, kd, vd, sched.row_ptr, sched.col_idx, sched.row_order, o2, l2)
    torch.cuda.synchronize()
    keep = agree.reshape(bt, h, n)
    if not keep.any():
        return
    assert_attn(f64(o2)[keep], o_ref2[keep], "sparse O (own CSR)")
    assert_lse(f64(l2)[keep], l_ref2[keep], "sparse lse (own CSR)")
