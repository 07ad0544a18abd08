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
    (2, 8, 2, 640, 64, 64), (1, 16, 4, 256, 96, 32), (2, 4, 2, 256, 96, 16),
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


@pytest.mark.parametrize("gq,d,B", [(2, 64, 32), (4, 96, 32), (8, 128, 32), (4, 64, 32),
                                    (4, 96, 16)])
def test_shared_kv_heads_match_repeated_kv(gpu_lib, gq, d, B):
    """32- and 16-key blocks, kv_heads < heads: every query head comes out bit for bit
    as with its key-value head repeated explicitly (kv_heads = heads), and a
    sampled head per batch matches the oracle.  Supports: random per query
    head, with empty rows, local bands, ids past the diagonal after the
    diagonal block, and 4160 keys (130 or 260 query blocks)."""
    w = gpu_lib
    bt, kvh, n = 2, 2, 32 * 130
    h = gq * kvh
    nb = n // B
    say(f"shared kv heads gq={gq} d={d} B={B} heads={h} n={n}")
    q, k, v = (x.cuda() for x in make(bt, h, kvh, n, d, seed=7 * gq + d))
    rng = np.random.default_rng(gq * 1000 + d)
    rp, ci = [0], []
    for bh in range(bt * h):
        for qb in range(nb):
            u = rng.random()
            if u < 0.05:
                ids = []                                          # empty row
            elif u < 0.15:
                ids = sorted({0, qb} | set(range(max(0, qb - 5), qb)))   # local band
            else:
                ids = sorted(set(np.nonzero(rng.random(qb + 1) < 0.3)[0].tolist()) | {qb})
                if u > 0.95:
                    ids = ids + [qb + 1 + int(rng.integers(3))]    # past the diagonal
            ci.extend(ids)
            rp.append(len(ci))
    rp_t = torch.tensor(rp, dtype=torch.int32, device="cuda")
    ci_t = torch.tensor(ci, dtype=torch.int32, device="cuda")
    s_g = w.make_shape(bt, h, n, d, B, kv_heads=kvh)
    o_g = torch.empty_like(q)
    l_g = torch.empty((bt, h, n), device="cuda")
    w.wise_sparse_attn(s_g, q, k, v, rp_t, ci_t, None, o_g, l_g)
    ke = k.repeat_interleave(gq, dim=1).contiguous()
    ve = v.repeat_interleave(gq, dim=1).contiguous()
    s_r = w.make_shape(bt, h, n, d, B)
    o_r = torch.empty_like(q)
    l_r = torch.empty((bt, h, n), device="cuda")
    w.wise_sparse_attn(s_r, q, ke, ve, rp_t, ci_t, None, o_r, l_r)
    torch.cuda.synchronize()
    assert torch.equal(o_g, o_r)
    assert torch.equal(l_g, l_r)
    # and one sampled head per batch against the oracle
    rows = np.array(rp, np.int32)
    for bh in (0, h + gq):
        b, hh = divmod(bh, h)
        sl = slice(bh * nb, (bh + 1) * nb + 1)
        rph = rows[sl] - rows[bh * nb]
        cih = np.array(ci[rows[bh * nb]:rows[(bh + 1) * nb]], np.int32)
        valid = np.concatenate([[x for x in cih[rph[i]:rph[i + 1]] if x <= i] for i in range(nb)]
                               + [np.zeros(0)]).astype(np.int32)
        cnt = [sum(1 for x in cih[rph[i]:rph[i + 1]] if x <= i) for i in range(nb)]
        rpv = np.concatenate([[0], np.cumsum(cnt)]).astype(np.int32)
        qh = f64(q[b, hh])[None, None]
        kh = f64(k[b, hh // gq])[None, None]
        vh = f64(v[b, hh // gq])[None, None]
        o_ref, l_ref = O.sparse_attention(qh, kh, vh, rpv, valid, B)
        assert_attn(o_g[b, hh], o_ref[0, 0], f"head {bh} O")
        assert_lse(l_g[b, hh], l_ref[0, 0], f"head {bh} lse")


@pytest.mark.parametrize("B", [32, 16])
def test_mass_workspace_smaller_than_all_heads(gpu_lib, B):
    """A mass workspace smaller than wise_mass_workspace_bytes runs the heads
    in consecutive launches of whole key-value groups; O, LSE and the
    accumulator come out bit for bit as with one launch, chunks crossing
    batch boundaries included, and the accumulator matches the oracle."""
    w = gpu_lib
    bt, h, kvh, n, d = 3, 8, 2, 384, 96
    nb = n // B
    q, k, v = (x.cuda() for x in make(bt, h, kvh, n, d, seed=77 + B))
    s = w.make_shape(bt, h, n, d, B, kv_heads=kvh)
    full, least = w.wise_mass_workspace_bytes(s), w.wise_mass_workspace_min_bytes(s)
    say(f"workspace full {full} B, one group {least} B")
    outs = []
    for size in (full, least, 2 * least + least // 2):      # 1, 6 and 3 launches
        o = torch.empty_like(q)
        lse = torch.empty((bt, h, n), device="cuda")
        acc = torch.zeros((bt, h, nb, nb), device="cuda")
        ws = torch.empty(size, dtype=torch.uint8, device="cuda")
        w.wise_dense_attn_accum(s, q, k, v, o, lse, acc, ws)
        torch.cuda.synchronize()
        outs.append((o, lse, acc))
    for o, lse, acc in outs[1:]:
        assert torch.equal(o, outs[0][0]) and torch.equal(lse, outs[0][1])
        assert torch.equal(acc, outs[0][2])
    ref = O.block_mass(f64(q), O.expand_kv(f64(k), h), B)
    assert np.abs(f64(outs[1][2]) - ref).max() <= ACC_TOL
    with pytest.raises(w.WiseError):
        w.wise_dense_attn_accum(s, q, k, v, torch.empty_like(q), None,
                                torch.zeros((bt, h, nb, nb), device="cuda"),
                                torch.empty(least - 256, dtype=torch.uint8, device="cuda"))
