"""GPU parity of grouped-query attention (query heads sharing key-value
heads; the paper's second backbone, Appendix B) through the C ABI against
the oracle on the expanded key-value heads.  Masses, supports and outputs
stay per query head."""

import numpy as np
import pytest
import torch

from oracle import wise_oracle as O
from parity_util import ACC_TOL, assert_attn, assert_lse, f64, say

pytestmark = pytest.mark.gpu

CASES = [  # bt, heads, kv_heads, n, d, B
    (2, 4, 2, 384, 64, 32), (1, 6, 3, 512, 96, 64), (1, 4, 1, 512, 128, 128),
    (2, 8, 2, 640, 64, 64), (1, 16, 4, 256, 96, 32),
]


def make(bt, h, kvh, n, d, seed):
    g = torch.Generator().manual_seed(seed)
    q = (torch.randn((bt, h, n, d), generator=g) * 1.5).to(torch.bfloat16)
    k = torch.randn((bt, kvh, n, d), generator=g).to(torch.bfloat16)
    v = torch.randn((bt, kvh, n, d), generator=g).to(torch.bfloat16)
    return q, k, v


@pytest.mark.parametrize("bt,h,kvh,n,d,B", CASES)
def test_gqa_dense_mass_sparse(gpu_lib, bt, h, kvh, n, d, B):
    w = gpu_lib
    say(f"gqa bt={bt} heads={h} kv_heads={kvh} n={n} d={d} B={B}")
    q, k, v = make(bt, h, kvh, n, d, seed=h * 100 + n + B)
    qe, ke, ve = f64(q), O.expand_kv(f64(k), h), O.expand_kv(f64(v), h)
    s = w.make_shape(bt, h, n, d, B, kv_heads=kvh)
    nb = n // B
    o = torch.empty_like(q, device="cuda")
    lse = torch.empty((bt, h, n), device="cuda")
    acc = torch.zeros((bt, h, nb, nb), device="cuda")
    qd, kd, vd = q.cuda(), k.cuda(), v.cuda()
    w.wise_dense_attn_accum(s, qd, kd, vd, o, lse, acc, w.mass_workspace(s))
    torch.cuda.synchronize()
    o_ref, l_ref = O.dense_attention(qe, ke, ve)
    assert_attn(o, o_ref, "gqa dense O")
    assert_lse(lse, l_ref, "gqa dense lse")
    r_ref = O.block_mass(qe, ke, B)
    assert np.abs(f64(acc) - r_ref).max() <= ACC_TOL
    # sparse on a per-query-head random support
    rng = np.random.default_rng(n + h)
    rp, ci = [0], []
    for _ in range(bt * h):
        for qb in range(nb):
            ci.extend(sorted(set(rng.integers(0, qb + 1, size=3).tolist()) | {qb}))
            rp.append(len(ci))
    rp, ci = np.array(rp, np.int32), np.array(ci, np.int32)
    w.wise_sparse_attn(s, qd, kd, vd, torch.from_numpy(rp).cuda(), torch.from_numpy(ci).cuda(),
                       torch.from_numpy(O.schedule_order(rp, nb)).cuda(), o, lse)
    torch.cuda.synchronize()
    o_ref, l_ref = O.sparse_attention(qe, ke, ve, rp, ci, B)
    assert_attn(o, o_ref, "gqa sparse O")
    assert_lse(lse, l_ref, "gqa sparse lse")


def test_explicit_kv_heads_equal_heads_is_plain_attention(gpu_lib):
    """kv_heads = heads and kv_heads = 0 run the same computation bit for bit."""
    w = gpu_lib
    bt, h, n, d, B = 1, 4, 512, 64, 64
    q, k, v = (x.cuda() for x in make(bt, h, h, n, d, seed=5))
    outs = []
    for kvh in (0, h):
        s = w.make_shape(bt, h, n, d, B, kv_heads=kvh)
        o = torch.empty_like(q)
        lse = torch.empty((bt, h, n), device="cuda")
        acc = torch.zeros((bt, h, n // B, n // B), device="cuda")
        w.wise_dense_attn_accum(s, q, k, v, o, lse, acc, w.mass_workspace(s))
        outs.append((o, lse, acc))
    torch.cuda.synchronize()
    for a, b in zip(*outs):
        assert torch.equal(a, b)
