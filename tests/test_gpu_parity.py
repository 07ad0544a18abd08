"""GPU parity: the HIP path (through the C ABI) against the CPU oracle on the
same seeded, bf16-rounded inputs.

Bars (from the task's targets):
  attention outputs  max-abs <= 1e-2 and mean-abs <= 1e-3 vs the oracle.
                     The outputs are bf16: rounding them alone costs up to
                     half a bf16 spacing, 2^-8 for |O| in [1, 2), 2^-7 in
                     [2, 4) (leaving the kernel about 0.002 of the 1e-2 bar)
                     and 2^-6 in [4, 8) (beyond the bar by itself).  So the
                     max-abs bar applies where |ref| < 2, and where |ref| >= 2
                     (rows concentrated on a few value rows) the error must
                     stay within one bf16 spacing, 2^-7 |ref|.
  LSE                max-abs <= 1e-3 (natural log)
  accumulator        max-abs <= 1e-5 per window step (masses lie in [0, 1])
  CSR / row order    bit-exact; an end-to-end CSR row may differ only when
                     the oracle's own cut is within 1e-5 of a boundary (the
                     margins delta^-, delta^+, delta^rank of Appendix A),
                     and such rows are reported, not failed.
"""

import numpy as np
import pytest
import torch

from oracle import wise_oracle as O
from paper_2609_27373_amd.workloads import CONFIGS, Trajectory

pytestmark = pytest.mark.gpu

from parity_util import (ACC_TOL, ATOL_MAX, ATOL_MEAN, assert_attn, assert_lse, compare_support,
                         f64, rows_of, say)

def random_support(nb_rows, nb, rng, bh, with_diag=0.7):
    rp, ci = [0], []
    for _ in range(bh):
        for qb in range(nb):
            k = int(rng.integers(1, qb + 2))
            s = set(rng.choice(qb + 1, size=k, replace=False).tolist())
            if rng.random() < with_diag:
                s.add(qb)
            ci.extend(sorted(s))
            rp.append(len(ci))
    return np.array(rp, np.int32), np.array(ci, np.int32)


def inputs(bt, h, n, d, seed, scale=1.0, planted=False):
    g = torch.Generator().manual_seed(seed)
    q = torch.randn((bt, h, n, d), generator=g) * scale
    k = torch.randn((bt, h, n, d), generator=g)
    v = torch.randn((bt, h, n, d), generator=g)
    if planted:   # make some rows peaky so the O rescale path triggers
        q[..., ::7, :] *= 4
    return [x.to(torch.bfloat16) for x in (q, k, v)]


SHAPES = [  # bt, h, n, d, B  (ragged: n not a multiple of 128, single block, ...)
    (1, 1, 64, 64, 64), (2, 3, 384, 64, 64), (1, 2, 320, 96, 64), (1, 2, 640, 128, 64),
    (2, 2, 512, 128, 128), (1, 3, 384, 96, 128), (1, 1, 128, 64, 128), (1, 2, 1024, 128, 64),
    (1, 1, 64, 96, 32), (2, 2, 384, 96, 32), (1, 2, 320, 64, 32), (1, 3, 640, 128, 32),
    (1, 2, 256, 128, 64), (1, 1, 768, 128, 32),   # one and three 256-query dense tiles
    (1, 1, 64, 96, 16), (1, 2, 256, 64, 16), (2, 1, 384, 128, 16), (1, 3, 320, 96, 16),
]


@pytest.mark.parametrize("bt,h,n,d,B", SHAPES)
def test_dense_and_mass(gpu_lib, bt, h, n, d, B):
    w = gpu_lib
    say(f"dense+mass bt={bt} h={h} n={n} d={d} B={B}")
    q, k, v = inputs(bt, h, n, d, seed=n + d + B, scale=1.5)
    s = w.make_shape(bt, h, n, d, B)
    o = torch.empty_like(q, device="cuda")
    lse = torch.empty((bt, h, n), device="cuda")
    nb = n // B
    acc = torch.full((bt, h, nb, nb), 0.25, device="cuda")   # RMW onto a non-zero start
    w.wise_dense_attn_accum(s, q.cuda(), k.cuda(), v.cuda(), o, lse, acc, w.mass_workspace(s))
    torch.cuda.synchronize()
    o_ref, l_ref = O.dense_attention(f64(q), f64(k), f64(v))
    assert_attn(o, o_ref, "dense O")
    assert_lse(lse, l_ref, "dense lse")
    r_ref = O.block_mass(f64(q), f64(k), B)
    a = f64(acc) - 0.25
    upper = np.triu(np.ones((nb, nb), bool), 1)
    assert np.all(a[..., upper] == 0), "entries past the diagonal must stay untouched"
    assert np.abs(a - r_ref).max() <= ACC_TOL, np.abs(a - r_ref).max()


@pytest.mark.parametrize("bt,h,n,d,B", SHAPES)
def test_sparse_random_support(gpu_lib, bt, h, n, d, B):
    w = gpu_lib
    say(f"sparse bt={bt} h={h} n={n} d={d} B={B}")
    q, k, v = inputs(bt, h, n, d, seed=7 * n + d, scale=1.5)
    nb = n // B
    rng = np.random.default_rng(n * d)
    rp, ci = random_support(None, nb, rng, bt * h)
    order = O.schedule_order(rp, nb)
    s = w.make_shape(bt, h, n, d, B)
    o = torch.empty_like(q, device="cuda")
    lse = torch.empty((bt, h, n), device="cuda")
    for ord_t in (None, torch.from_numpy(order).cuda()):
        w.wise_sparse_attn(s, q.cuda(), k.cuda(), v.cuda(), torch.from_numpy(rp).cuda(),
                           torch.from_numpy(ci).cuda(), ord_t, o, lse)
        torch.cuda.synchronize()
        o_ref, l_ref = O.sparse_attention(f64(q), f64(k), f64(v), rp, ci, B)
        assert_attn(o, o_ref, "sparse O")
        assert_lse(lse, l_ref, "sparse lse")


@pytest.mark.parametrize("d,B", [(64, 64), (128, 64), (96, 128), (96, 32)])
def test_peaky_rows(gpu_lib, d, B):
    """Near one-hot rows (queries scaled x6): the running max jumps by large
    amounts between tiles, so the O rescale path runs often, and O is close to
    single value rows, some beyond 4 in magnitude."""
    w = gpu_lib
    bt, h, n = 1, 2, 512
    q, k, v = inputs(bt, h, n, d, seed=99 + d, scale=1.0)
    q = (q.float() * 6).to(torch.bfloat16)
    s = w.make_shape(bt, h, n, d, B)
    o = torch.empty_like(q, device="cuda")
    lse = torch.empty((bt, h, n), device="cuda")
    w.wise_dense_attn_accum(s, q.cuda(), k.cuda(), v.cuda(), o, lse, None)
    torch.cuda.synchronize()
    o_ref, l_ref = O.dense_attention(f64(q), f64(k), f64(v))
    assert_attn(o, o_ref, "peaky O")
    assert_lse(lse, l_ref, "peaky lse")


@pytest.mark.parametrize("d,B", [(64, 64), (96, 64), (128, 64), (128, 128), (96, 128), (64, 32),
                                 (96, 32), (128, 32), (64, 16), (96, 16), (128, 16)])
def test_full_support_sparse_equals_dense(gpu_lib, d, B):
    """With every causal block in the support, R = 0 and the sparse kernel
    computes the dense result.  For blocks of 64 and 128 keys both kernels
    walk the same 64-key tiles in the same order with the same arithmetic,
    so the outputs agree bit for bit; 32- and 16-key blocks are walked in
    32-key tiles (a different online-softmax grouping), so there both are
    held to the oracle instead."""
    w = gpu_lib
    bt, h, n = 1, 2, 768
    q, k, v = (x.cuda() for x in inputs(bt, h, n, d, seed=d + B, scale=1.5, planted=True))
    nb = n // B
    rp, ci = [0], []
    for _ in range(bt * h):
        for qb in range(nb):
            ci.extend(range(qb + 1))
            rp.append(len(ci))
    s = w.make_shape(bt, h, n, d, B)
    od, os_ = torch.empty_like(q), torch.empty_like(q)
    ld, ls = torch.empty((bt, h, n), device="cuda"), torch.empty((bt, h, n), device="cuda")
    w.wise_dense_attn_accum(s, q, k, v, od, ld, None)
    w.wise_sparse_attn(s, q, k, v, torch.tensor(rp, dtype=torch.int32, device="cuda"),
                       torch.tensor(ci, dtype=torch.int32, device="cuda"), None, os_, ls)
    torch.cuda.synchronize()
    if B >= 64:
        assert torch.equal(od, os_)
        assert torch.equal(ld, ls)
    else:
        o_ref, l_ref = O.dense_attention(f64(q), f64(k), f64(v))
        assert_attn(od, o_ref, "dense O")
        assert_attn(os_, o_ref, "full-support sparse O")
        assert_lse(ls, l_ref, "full-support sparse lse")


@pytest.mark.parametrize("bt,h,kvh,n,d,B", [
    (1, 2, 2, 1024, 128, 64), (2, 3, 3, 640, 128, 64), (1, 4, 2, 512, 96, 64), (2, 2, 1, 384, 64, 64),
    (1, 2, 2, 512, 96, 32), (1, 2, 2, 512, 128, 128), (1, 2, 2, 320, 64, 64),
    (2, 3, 3, 1280, 128, 128), (1, 4, 2, 1024, 128, 128), (1, 2, 2, 640, 128, 128),
    (1, 2, 2, 512, 96, 128),
])
def test_grouped_equals_rows(gpu_lib, bt, h, kvh, n, d, B):
    """wise_sparse_attn_grouped (block 64: 4 or 2 consecutive rows per group,
    block 128 at d 128: 2, over the union of their supports) gives
    wise_sparse_attn's outputs bit for bit, and both match the oracle: random
    rows, empty rows, local bands, full rows, rows without their diagonal
    block and ids past the diagonal.  Block 32, block 128 below d 128 and
    lengths the group's queries do not divide (n = 320 at d 64, 640 at d 128
    with block 128) run the one-row kernel."""
    w = gpu_lib
    nb = n // B
    s = w.make_shape(bt, h, n, d, B, kv_heads=kvh)
    say(f"grouped vs rows bt={bt} h={h} kvh={kvh} n={n} d={d} B={B}: "
        f"{w.wise_sparse_group_rows(s)} rows per group")
    g = torch.Generator().manual_seed(n + d + B)
    q = (torch.randn((bt, h, n, d), generator=g) * 1.5).to(torch.bfloat16)
    k = torch.randn((bt, kvh, n, d), generator=g).to(torch.bfloat16)
    v = torch.randn((bt, kvh, n, d), generator=g).to(torch.bfloat16)
    rng = np.random.default_rng(n * d + B)
    rp, ci, keep = [0], [], []
    for _ in range(bt * h):
        for qb in range(nb):
            u = rng.random()
            if u < 0.1:
                ids = []
            elif u < 0.25:
                ids = list(range(max(0, qb - 3), qb + 1))
            elif u < 0.45:
                ids = list(range(qb + 1))
            elif u < 0.55:
                ids = sorted(set(np.nonzero(rng.random(qb + 1) < 0.5)[0].tolist()) - {qb})
            else:
                ids = sorted(set(np.nonzero(rng.random(qb + 1) < 0.6)[0].tolist()) | {qb})
            keep.append(list(ids))
            if u > 0.9:
                ids = ids + [qb + 1 + int(rng.integers(3))]     # past the diagonal
            ci.extend(ids)
            rp.append(len(ci))
    rp_t = torch.tensor(rp, dtype=torch.int32, device="cuda")
    ci_t = torch.tensor(ci, dtype=torch.int32, device="cuda")
    qd, kd, vd = q.cuda(), k.cuda(), v.cuda()
    o_r, o_g = torch.empty_like(qd), torch.empty_like(qd)
    l_r, l_g = (torch.empty((bt, h, n), device="cuda") for _ in range(2))
    w.wise_sparse_attn(s, qd, kd, vd, rp_t, ci_t, None, o_r, l_r)
    w.wise_sparse_attn_grouped(s, qd, kd, vd, rp_t, ci_t, o_g, l_g)
    torch.cuda.synchronize()
    assert torch.equal(o_r, o_g) and torch.equal(l_r, l_g)
    rp_k = np.array([0] + list(np.cumsum([len(r) for r in keep])), np.int32)
    ci_k = np.array([b for r in keep for b in r], np.int32)
    o_ref, l_ref = O.sparse_attention(f64(q), O.expand_kv(f64(k), h), O.expand_kv(f64(v), h),
                                      rp_k, ci_k, B)
    assert_attn(o_g, o_ref, "grouped O")
    assert_lse(l_g, l_ref, "grouped lse")


@pytest.mark.parametrize("n,B", [(65536, 64), (131072, 128)])
def test_grouped_at_most_key_blocks(gpu_lib, n, B):
    """1024 key blocks, the grouped kernel's largest support (16 mask words
    per row): sparse random rows with the sink, a block in every 64-block word
    and the diagonal give the one-row kernel's bits, and the oracle's values."""
    w = gpu_lib
    d, nb = 128, n // B
    s = w.make_shape(1, 1, n, d, B)
    assert w.wise_sparse_group_rows(s) > 0
    say(f"grouped at {nb} key blocks: n={n} B={B}, {w.wise_sparse_group_rows(s)} rows per group")
    g = torch.Generator().manual_seed(n + B)
    q = (torch.randn((1, 1, n, d), generator=g) * 1.5).to(torch.bfloat16).cuda()
    k = torch.randn((1, 1, n, d), generator=g).to(torch.bfloat16).cuda()
    v = torch.randn((1, 1, n, d), generator=g).to(torch.bfloat16).cuda()
    rng = np.random.default_rng(n)
    rp, ci = [0], []
    for qb in range(nb):
        ids = {0, qb} | {int(x) for x in rng.integers(0, qb + 1, size=3)}
        ids |= {int(wd * 64 + rng.integers(64)) for wd in range(qb // 64 + 1) if wd * 64 <= qb}
        ids = sorted(x for x in ids if x <= qb)
        ci.extend(ids)
        rp.append(len(ci))
    rp_t = torch.tensor(rp, dtype=torch.int32, device="cuda")
    ci_t = torch.tensor(ci, dtype=torch.int32, device="cuda")
    o_r, o_g = torch.empty_like(q), torch.empty_like(q)
    l_r, l_g = (torch.empty((1, 1, n), device="cuda") for _ in range(2))
    w.wise_sparse_attn(s, q, k, v, rp_t, ci_t, None, o_r, l_r)
    w.wise_sparse_attn_grouped(s, q, k, v, rp_t, ci_t, o_g, l_g)
    torch.cuda.synchronize()
    assert torch.equal(o_r, o_g) and torch.equal(l_r, l_g)
    # against the oracle, every row
    o_ref, l_ref = O.sparse_attention(f64(q), f64(k), f64(v), np.array(rp, np.int32),
                                      np.array(ci, np.int32), B)
    assert_attn(o_g, o_ref, f"grouped O, {nb} rows")
    assert_lse(l_g, l_ref, "grouped lse")


def test_grouped_past_1024_key_blocks_runs_the_one_row_kernel(gpu_lib):
    """1032 key blocks: no group shape (the masks hold 1024), so the grouped
    call runs the one-row kernel in natural row order: the same bits as
    wise_sparse_attn without a row order."""
    w = gpu_lib
    n, d, B = 1032 * 64, 128, 64
    s = w.make_shape(1, 1, n, d, B)
    assert w.wise_sparse_group_rows(s) == 0
    g = torch.Generator().manual_seed(5)
    q, k, v = ((torch.randn((1, 1, n, d), generator=g)).to(torch.bfloat16).cuda() for _ in range(3))
    nb = n // B
    rp, ci = [0], []
    for qb in range(nb):
        ci.extend(sorted({0, qb, qb // 2}))
        rp.append(len(ci))
    rp_t = torch.tensor(rp, dtype=torch.int32, device="cuda")
    ci_t = torch.tensor(ci, dtype=torch.int32, device="cuda")
    o_r, o_g = torch.empty_like(q), torch.empty_like(q)
    w.wise_sparse_attn(s, q, k, v, rp_t, ci_t, None, o_r, None)
    w.wise_sparse_attn_grouped(s, q, k, v, rp_t, ci_t, o_g, None)
    torch.cuda.synchronize()
    assert torch.equal(o_r, o_g)


def test_sparse_edge_rows(gpu_lib):
    """Empty rows give O = 0 and lse = -inf; ids past the diagonal are skipped."""
    w = gpu_lib
    bt, h, n, d, B = 1, 1, 256, 64, 64
    q, k, v = inputs(bt, h, n, d, seed=3)
    rp = np.array([0, 1, 1, 3, 6], np.int32)         # row 1 empty
    ci = np.array([0, 1, 2, 0, 2, 3], np.int32)      # rows: [0], [], [1, 2], [0, 2, 3]
    ci_bad = ci.copy()
    ci_bad[2] = 3                                     # row 2 now names block 3 > qb = 2
    s = w.make_shape(bt, h, n, d, B)
    o = torch.empty_like(q, device="cuda")
    lse = torch.empty((bt, h, n), device="cuda")
    w.wise_sparse_attn(s, q.cuda(), k.cuda(), v.cuda(), torch.from_numpy(rp).cuda(),
                       torch.from_numpy(ci_bad).cuda(), None, o, lse)
    torch.cuda.synchronize()
    ci_eff = np.array([0, 1, 0, 2, 3], np.int32)
    rp_eff = np.array([0, 1, 1, 2, 5], np.int32)
    o_ref, l_ref = O.sparse_attention(f64(q), f64(k), f64(v), rp_eff, ci_eff, B)
    assert torch.all(o[0, 0, 64:128] == 0)
    assert torch.all(torch.isneginf(lse[0, 0, 64:128]))
    assert_attn(o, o_ref, "edge sparse O")
    assert_lse(lse, l_ref, "edge lse")


def test_sparse_block16_rows(gpu_lib):
    """16-key blocks run two blocks of a row per 32-key tile, the row's 16
    queries duplicated over the wave's 32 columns: empty rows next to full
    ones, odd block counts (a last tile with one block), consecutive and
    distant block pairs, the diagonal in either half of the last tile, and
    ids past a row's diagonal must leave each row exactly its own attention
    (and the next row's outputs untouched)."""
    w = gpu_lib
    bt, h, n, d, B = 1, 2, 192, 64, 16
    q, k, v = inputs(bt, h, n, d, seed=16, scale=1.5)
    per_head = [[], [0, 1],            # an empty row next to a full one
                [0, 2], [],
                [], [],
                [1, 3, 6, 7], [0, 5, 7],   # row 6 names 7 (past its diagonal)
                [8], [0, 1, 2, 3, 4, 5, 6, 7, 8, 9],
                [10], [11]]            # diagonal blocks only
    rows = per_head + [[b for b in r if b % 3 != 1] for r in per_head]
    keep = [[b for b in r if b <= i % 12] for i, r in enumerate(rows)]
    rp = np.array([0] + list(np.cumsum([len(r) for r in rows])), np.int32)
    ci = np.array([b for r in rows for b in r], np.int32)
    rp_k = np.array([0] + list(np.cumsum([len(r) for r in keep])), np.int32)
    ci_k = np.array([b for r in keep for b in r], np.int32)
    s = w.make_shape(bt, h, n, d, B)
    o = torch.empty_like(q, device="cuda")
    lse = torch.empty((bt, h, n), device="cuda")
    w.wise_sparse_attn(s, q.cuda(), k.cuda(), v.cuda(), torch.from_numpy(rp).cuda(),
                       torch.from_numpy(ci).cuda(), None, o, lse)
    torch.cuda.synchronize()
    o_ref, l_ref = O.sparse_attention(f64(q), f64(k), f64(v), rp_k, ci_k, B)
    for r in (0, 3, 4, 5):             # empty rows: zeros and -inf
        assert torch.all(o[0, 0, 16 * r:16 * r + 16] == 0)
        assert torch.all(torch.isneginf(lse[0, 0, 16 * r:16 * r + 16]))
    assert_attn(o, o_ref, "B16 rows O")
    assert_lse(lse, l_ref, "B16 rows lse")


@pytest.mark.parametrize("nb,seed", [(1, 0), (8, 1), (63, 2), (64, 3), (65, 4), (128, 5),
                                     (200, 6), (256, 7), (513, 8), (1024, 9)])
def test_select_only_parity(gpu_lib, nb, seed):
    """Selection on identical fp32 masses: CSR and row order are bit-exact."""
    w = gpu_lib
    rng = np.random.default_rng(seed)
    h = 3 if nb <= 256 else 1
    acc = rng.gamma(0.25, size=(1, h, nb, nb)).astype(np.float32)
    acc[rng.random(acc.shape) < 0.15] = 0.0
    acc[..., 1::3] = np.round(acc[..., 1::3], 1)        # exact ties between blocks
    if nb >= 8:
        acc[0, 0, 5, :] = 0.0                           # an all-zero row
    s = w.make_shape(1, h, nb * 64, 64, 64)
    sched = w.Schedule(s)
    for tau in (0.5, 0.9, 0.95, 1.0):
        for flags in (0, 1, 2, 3):
            t32 = float(np.float32(tau))
            sched.select(torch.from_numpy(acc).cuda(), t32, flags)
            torch.cuda.synchronize()
            rp_ref, ci_ref = O.select_support(acc.astype(np.float64), t32, flags)
            nnz = sched.nnz()
            assert np.array_equal(sched.row_ptr.cpu().numpy(), rp_ref), (tau, flags)
            assert np.array_equal(sched.col_idx[:nnz].cpu().numpy(), ci_ref), (tau, flags)
            assert np.array_equal(sched.row_order.cpu().numpy(), O.schedule_order(rp_ref, nb))


@pytest.mark.parametrize("block", [64, 16])
def test_tiny_trajectory(gpu_lib, block):
    """The whole path on the tiny workload: 4 discovery steps (all in the
    window), selection, 4 late steps; everything against the oracle."""
    from paper_2609_27373_amd.pipeline import WisePipeline
    cfg = CONFIGS["tiny"].with_(block=block)
    tr = Trajectory(cfg)
    pipe = WisePipeline.for_config(cfg)
    masses = []
    for t in range(1, cfg.steps + 1):
        q, k, v = (x.to(torch.bfloat16) for x in tr.next())
        qg, kg, vg = q.cuda(), k.cuda(), v.cuda()
        out = torch.empty_like(qg)
        qd, kd, vd = f64(q), f64(k), f64(v)
        if t <= cfg.discovery_steps:
            pipe.discovery_step(qg, kg, vg, out, accumulate=t in cfg.window)
            torch.cuda.synchronize()
            o_ref, l_ref = O.dense_attention(qd, kd, vd)
            assert_attn(out, o_ref, f"step {t} dense")
            assert_lse(pipe.lse, l_ref, f"step {t} lse")
            if t in cfg.window:
                masses.append(O.block_mass(qd, kd, cfg.block))
                acc_ref = O.accumulate(masses)
                assert np.abs(f64(pipe.acc) - acc_ref).max() <= ACC_TOL * len(masses)
            if t == cfg.discovery_steps:
                sched = pipe.select()
                torch.cuda.synchronize()
                tau = float(np.float32(cfg.tau))
                reported = compare_support(rows_of(sched.row_ptr, sched.col_idx[: sched.nnz()]),
                                           acc_ref, tau, pipe.flags)
                # late steps are compared over the oracle's own support
                rp, ci = O.select_support(acc_ref, tau, pipe.flags)
                if reported:   # near ties: run the late steps on the oracle's CSR
                    sched.row_ptr.copy_(torch.from_numpy(rp))
                    sched.col_idx[: ci.size].copy_(torch.from_numpy(ci))
                    sched.row_order.copy_(torch.from_numpy(O.schedule_order(rp, cfg.nb)))
        else:
            lse = torch.empty_like(pipe.lse)
            pipe.late_step(qg, kg, vg, out, lse)
            torch.cuda.synchronize()
            o_ref, l_ref = O.sparse_attention(qd, kd, vd, rp, ci, cfg.block)
            assert_attn(out, o_ref, f"step {t} sparse")
            assert_lse(lse, l_ref, f"step {t} sparse lse")
            om, _ = O.sparse_attention_masked(qd, kd, vd, rp, ci, cfg.block)
            assert_attn(out, om, f"step {t} sparse vs masked-dense form")


def test_determinism(gpu_lib):
    from paper_2609_27373_amd.pipeline import WisePipeline
    cfg = CONFIGS["tiny"].with_(heads=4, seq_len=1024)
    outs = []
    for _ in range(2):
        tr = Trajectory(cfg, device="cuda")
        pipe = WisePipeline.for_config(cfg)
        o = None
        for t in range(1, 6):
            q, k, v = tr.next(torch.bfloat16)
            o = torch.empty_like(q)
            if t <= 4:
                pipe.discovery_step(q, k, v, o, accumulate=True)
                if t == 4:
                    pipe.select()
            else:
                pipe.late_step(q, k, v, o)
        torch.cuda.synchronize()
        s = pipe.schedule
        outs.append((o.clone(), pipe.acc.clone(), s.row_ptr.clone(),
                     s.col_idx[: s.nnz()].clone(), s.row_order.clone()))
    for a, b in zip(*outs):
        assert torch.equal(a, b)


@pytest.mark.parametrize("B", [16, 32, 64, 128])
def test_sparse_ids_past_diagonal_after_the_diagonal(gpu_lib, B):
    """Ids past the diagonal that follow the diagonal block are skipped and
    the diagonal block is still attended (with its causal mask)."""
    w = gpu_lib
    bt, h, d = 1, 2, 64
    nb = 4
    n = nb * B
    q, k, v = inputs(bt, h, n, d, seed=11 + B)
    rows = [[0, 1], [0, 1, 2], [1, 2, 5], [3, 4, 7]]        # the (qb, id) pairs past qb are skipped
    keep = [[x for x in r if x <= qb] for qb, r in enumerate(rows)]
    rp = np.array([0] + list(np.cumsum([len(r) for r in rows * h])), np.int32)
    ci = np.array([x for r in rows * h for x in r], np.int32)
    rp_k = np.array([0] + list(np.cumsum([len(r) for r in keep * h])), np.int32)
    ci_k = np.array([x for r in keep * h for x in r], np.int32)
    s = w.make_shape(bt, h, n, d, B)
    o = torch.empty_like(q, device="cuda")
    lse = torch.empty((bt, h, n), device="cuda")
    w.wise_sparse_attn(s, q.cuda(), k.cuda(), v.cuda(), torch.from_numpy(rp).cuda(),
                       torch.from_numpy(ci).cuda(), None, o, lse)
    torch.cuda.synchronize()
    o_ref, l_ref = O.sparse_attention(f64(q), f64(k), f64(v), rp_k, ci_k, B)
    assert_attn(o, o_ref, f"B{B} O")
    assert_lse(lse, l_ref, f"B{B} lse")


@pytest.mark.parametrize("d,B,scale", [(64, 64, 0.05), (128, 32, 0.2), (96, 128, 0.08)])
def test_explicit_scale(gpu_lib, d, B, scale):
    """wise_shape.scale > 0 replaces 1/sqrt(d) in dense attention, the pooled
    masses and the late step alike."""
    w = gpu_lib
    bt, h, n = 1, 2, 512
    say(f"explicit scale {scale} d={d} B={B}")
    q, k, v = inputs(bt, h, n, d, seed=int(scale * 1000) + d, scale=2.0)
    s = w.make_shape(bt, h, n, d, B, scale=scale)
    nb = n // B
    o = torch.empty_like(q, device="cuda")
    lse = torch.empty((bt, h, n), device="cuda")
    acc = torch.zeros((bt, h, nb, nb), device="cuda")
    qd, kd, vd = q.cuda(), k.cuda(), v.cuda()
    w.wise_dense_attn_accum(s, qd, kd, vd, o, lse, acc, w.mass_workspace(s))
    torch.cuda.synchronize()
    o_ref, l_ref = O.dense_attention(f64(q), f64(k), f64(v), scale=scale)
    assert_attn(o, o_ref, "scaled dense O")
    assert_lse(lse, l_ref, "scaled dense lse")
    assert np.abs(f64(acc) - O.block_mass(f64(q), f64(k), B, scale=scale)).max() <= ACC_TOL
    rng = np.random.default_rng(d + B)
    rp, ci = [0], []
    for _ in range(bt * h):
        for qb in range(nb):
            ci.extend(sorted(set(rng.integers(0, qb + 1, size=2).tolist()) | {0, qb}))
            rp.append(len(ci))
    rp, ci = np.array(rp, np.int32), np.array(ci, np.int32)
    w.wise_sparse_attn(s, qd, kd, vd, torch.from_numpy(rp).cuda(), torch.from_numpy(ci).cuda(),
                       None, o, lse)
    torch.cuda.synchronize()
    o_ref, l_ref = O.sparse_attention(f64(q), f64(k), f64(v), rp, ci, B, scale=scale)
    assert_attn(o, o_ref, "scaled sparse O")
    assert_lse(lse, l_ref, "scaled sparse lse")
