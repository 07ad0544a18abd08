"""The whole path at the widest supported rows: 1024 key blocks (seq_len
65536 with 64-key blocks, one head, d 64), the limit of the selection kernel
and of the grouped late step.  Every row is checked by properties that hold
at any size (accumulator rows sum to one, CSR rows well formed, row order a
longest-first permutation, the grouped late step equal to the one-row kernel
bit for bit); sampled rows, the first, a middle one and the last, against the
oracle on the same bf16 inputs: dense O and LSE, block masses, the selected
row, and the late step on the oracle's own row."""

import numpy as np
import pytest
import torch

from oracle import wise_oracle as O
from parity_util import (ACC_TOL, assert_attn, assert_lse, check_csr, check_row_order,
                         check_row_vs_oracle, f64, say)

pytestmark = pytest.mark.gpu


def test_whole_path_at_1024_key_blocks(gpu_lib):
    w = gpu_lib
    n, d, B, tau, flags = 65536, 64, 64, float(np.float32(0.9)), 3
    nb = n // B
    say(f"whole path at {nb} key blocks: n={n} d={d} B={B} tau={tau}")
    g = torch.Generator().manual_seed(77)
    q = (torch.randn((1, 1, n, d), generator=g) * 3.0).to(torch.bfloat16)
    k = torch.randn((1, 1, n, d), generator=g).to(torch.bfloat16)
    v = torch.randn((1, 1, n, d), generator=g).to(torch.bfloat16)
    s = w.make_shape(1, 1, n, d, B)
    qd, kd, vd = q.cuda(), k.cuda(), v.cuda()
    o = torch.empty_like(qd)
    lse = torch.empty((1, 1, n), device="cuda")
    acc = torch.zeros((1, 1, nb, nb), device="cuda")
    w.wise_dense_attn_accum(s, qd, kd, vd, o, lse, acc, w.mass_workspace(s))
    sched = w.Schedule(s).select(acc, tau)
    o_r, o_g = torch.empty_like(qd), torch.empty_like(qd)
    l_r, l_g = (torch.empty((1, 1, n), device="cuda") for _ in range(2))
    w.wise_sparse_attn(s, qd, kd, vd, sched.row_ptr, sched.col_idx, sched.row_order, o_r, l_r)
    w.wise_sparse_attn_grouped(s, qd, kd, vd, sched.row_ptr, sched.col_idx, o_g, l_g)
    torch.cuda.synchronize()

    # every row: properties of the GPU's own outputs
    a = f64(acc)[0, 0]
    assert np.all(np.triu(a, 1) == 0.0)
    assert np.abs(a.sum(axis=1) - 1.0).max() <= ACC_TOL
    rp = sched.row_ptr.cpu().numpy()
    ci = sched.col_idx[: int(rp[-1])].cpu().numpy()
    check_csr(rp, ci, nb, flags)
    check_row_order(sched.row_order.cpu().numpy(), rp, nb)
    assert torch.equal(o_r, o_g) and torch.equal(l_r, l_g)
    say(f"  {nb} rows: accumulator rows sum to 1, CSR and row order well formed (nnz {rp[-1]}, "
        f"density {rp[-1] / (nb * (nb + 1) / 2):.3f}), grouped late step = one-row kernel")

    # sampled rows against the oracle
    qh, kh, vh = (f64(x[0, 0]) for x in (q, k, v))
    scale = O.default_scale(d)
    for qb in (0, nb // 2, nb - 1):
        rows = np.arange(qb * B, (qb + 1) * B)
        _, o_ref, l_ref = O.causal_attention_rows(qh, kh, vh, rows, scale)
        assert_attn(o[0, 0, qb * B:(qb + 1) * B], o_ref, f"row {qb}: dense O")
        assert_lse(lse[0, 0, qb * B:(qb + 1) * B], l_ref, f"row {qb}: dense lse")
        r_ref = O.block_mass_row(qh, kh, qb, B, scale)
        assert np.abs(a[qb] - r_ref).max() <= ACC_TOL, f"row {qb}: block mass"
        got = ci[rp[qb]:rp[qb + 1]]
        check_row_vs_oracle(got, r_ref, qb, tau, flags, f"row {qb}")
        want = O.select_row(r_ref, qb, tau, flags)
        so, sl = O.sparse_attention_row(qh, kh, vh, qb, want, B, scale)
        if list(got) == list(want):
            assert_attn(o_g[0, 0, qb * B:(qb + 1) * B], so, f"row {qb}: late step ({len(want)} blocks)")
            assert_lse(l_g[0, 0, qb * B:(qb + 1) * B], sl, f"row {qb}: late lse")
