"""GPU parity of the paper's temporal-union working set and of the routing
diagnostics, through the C ABI, against the CPU oracle.

  wise_select_step          per-step sets B_q^(t, eta): bit-exact against the
                            oracle's selection on the same fp32 masses
  wise_support_from_masks   union CSR + row order: bit-exact against the
                            oracle's union of the same masses
  wise_mask_union / overlap rolling sets and their (intersection, union)
                            sizes: exact integers
  wise_support_mass         per-row retained mass: fp64 sums of the same fp32
                            values, agreeing to 1e-12 relative; the fraction
                            also checked against the oracle's probabilities
                            (to the block-mass tolerance)
"""

import itertools

import numpy as np
import pytest
import torch

from oracle import wise_oracle as O
from paper_2609_27373_amd import diagnostics
from paper_2609_27373_amd.pipeline import WisePipeline
from paper_2609_27373_amd.workloads import CONFIGS, Trajectory
from parity_util import (ACC_TOL, assert_attn, check_csr, check_row_order, f64, say,
                         tie_alternatives)
from whole_heads import HeadOracle

pytestmark = pytest.mark.gpu


def mask_rows(mask, nb):
    """Device bitmask [rows][words] (int64) -> list over rows of block ids."""
    m = mask.cpu().numpy().view(np.uint64).reshape(-1, mask.shape[-1])
    bits = np.unpackbits(m.view(np.uint8).reshape(m.shape[0], -1), axis=1, bitorder="little")
    return [list(np.nonzero(b[:nb])[0]) for b in bits]


def rows_to_mask(rows, nb, words):
    m = np.zeros((len(rows), words), dtype=np.uint64)
    for i, r in enumerate(rows):
        for kb in r:
            m[i, kb >> 6] |= np.uint64(1) << np.uint64(kb & 63)
    return torch.from_numpy(m.view(np.int64)).cuda()


def random_masses(bt, h, nb, seed, steps=1, ties=False):
    """Positive causal rows summing to 1 (fp32); `ties` repeats values so
    the (mass desc, block asc) tie rule decides."""
    rng = np.random.default_rng(seed)
    out = []
    for _ in range(steps):
        r = rng.gamma(0.3, size=(bt, h, nb, nb))
        if ties:
            r = np.round(r * 4) / 4 + 1e-3
        r = r * np.tril(np.ones((nb, nb)))
        out.append((r / r.sum(-1, keepdims=True)).astype(np.float32))
    return out


def shape_of(w, bt, h, nb, B=64, d=64):
    return w.make_shape(bt, h, nb * B, d, B)


@pytest.mark.parametrize("nb,seed,ties", [(1, 0, False), (9, 1, True), (64, 2, False),
                                          (65, 3, True), (130, 4, False), (300, 5, False)])
def test_select_step_parity(gpu_lib, nb, seed, ties):
    w = gpu_lib
    say(f"select_step nb={nb} seed={seed} ties={ties}")
    bt, h = 1, 2
    (r,) = random_masses(bt, h, nb, seed, ties=ties)
    s = shape_of(w, bt, h, nb)
    words = w.wise_mask_words(s)
    mask = torch.full((bt * h * nb, words), -1, dtype=torch.int64, device="cuda")  # stale bits
    for tau in (0.5, 0.9, 0.95, 1.0):
        t32 = float(np.float32(tau))
        w.wise_select_step(s, torch.from_numpy(r).cuda(), t32, mask)
        torch.cuda.synchronize()
        assert mask_rows(mask, 64 * words) == O.step_supports(r, t32), f"tau {tau}"


@pytest.mark.parametrize("nb,steps,seed", [(1, 1, 0), (12, 4, 1), (64, 4, 2), (100, 3, 3),
                                           (257, 4, 4)])
def test_union_csr_parity(gpu_lib, nb, steps, seed):
    w = gpu_lib
    say(f"union CSR nb={nb} steps={steps} seed={seed}")
    bt, h = 2, 2
    ms = random_masses(bt, h, nb, seed, steps=steps)
    s = shape_of(w, bt, h, nb)
    rows, words = bt * h * nb, w.wise_mask_words(s)
    masks = torch.empty((steps, rows, words), dtype=torch.int64, device="cuda")
    tau = float(np.float32(0.9))
    for i, m in enumerate(ms):
        w.wise_select_step(s, torch.from_numpy(m).cuda(), tau, masks[i])
    sched = w.Schedule(s)
    for flags in (0, w.WISE_FORCE_SINK, w.WISE_FORCE_DIAG, w.WISE_DEFAULT_FLAGS):
        sched.from_masks(masks, steps, flags)
        torch.cuda.synchronize()
        rp = sched.row_ptr.cpu().numpy()
        ci = sched.col_idx[: int(rp[-1])].cpu().numpy()
        rp_o, ci_o = O.select_support_union(ms, tau, flags)
        assert np.array_equal(rp, rp_o) and np.array_equal(ci, ci_o), f"flags {flags}"
        assert np.array_equal(sched.row_order.cpu().numpy(), O.schedule_order(rp_o, nb))


def test_union_ignores_bits_past_the_diagonal(gpu_lib):
    w = gpu_lib
    bt, h, nb = 1, 1, 70
    s = shape_of(w, bt, h, nb)
    words = w.wise_mask_words(s)
    rng = np.random.default_rng(7)
    rows = [sorted(set(rng.integers(0, 128, size=5).tolist())) for _ in range(nb)]
    say("union with stray bits past the diagonal (and past nb)")
    masks = rows_to_mask(rows, nb, words)
    sched = w.Schedule(s)
    sched.from_masks(masks, 1, 0)
    torch.cuda.synchronize()
    rp = sched.row_ptr.cpu().numpy()
    got = [list(sched.col_idx[rp[i]:rp[i + 1]].cpu().numpy()) for i in range(nb)]
    want = [[kb for kb in r if kb <= qb] or [qb] for qb, r in enumerate(rows)]
    assert got == want


@pytest.mark.parametrize("nb,seed", [(5, 0), (64, 1), (190, 2)])
def test_mask_union_and_overlap(gpu_lib, nb, seed):
    w = gpu_lib
    say(f"mask union / overlap nb={nb}")
    bt, h = 1, 3
    s = shape_of(w, bt, h, nb)
    rows, words = bt * h * nb, w.wise_mask_words(s)
    rng = np.random.default_rng(seed)
    per_step = [[sorted(set(rng.integers(0, qb + 1, size=3).tolist())) for qb in
                 [i % nb for i in range(rows)]] for _ in range(6)]
    slab = torch.stack([rows_to_mask(p, nb, words) for p in per_step])
    out = torch.empty((rows, words), dtype=torch.int64, device="cuda")
    counts = torch.empty(2, dtype=torch.int64, device="cuda")
    prev = None
    for t in range(1, 7):
        lo = max(1, t - 3)
        w.wise_mask_union(s, slab[lo - 1:t].contiguous(), t - lo + 1, out)
        torch.cuda.synchronize()
        want = O.rolling_working_set(per_step, t)
        assert mask_rows(out, 64 * words) == want, f"W^({t})"
        if prev is not None:
            w.wise_mask_overlap(s, prev, out, counts)
            torch.cuda.synchronize()
            assert tuple(counts.cpu().tolist()) == O.overlap_counts(
                O.rolling_working_set(per_step, t - 1), want)
        prev = out.clone()
    # in place: out coincides with the first mask
    buf = slab[:3].clone()
    w.wise_mask_union(s, buf, 3, buf[0])
    torch.cuda.synchronize()
    assert torch.equal(buf[0], slab[0] | slab[1] | slab[2])


@pytest.mark.parametrize("nb,seed", [(1, 0), (33, 1), (128, 2), (260, 3)])
def test_support_mass_parity(gpu_lib, nb, seed):
    w = gpu_lib
    say(f"support mass nb={nb}")
    bt, h = 2, 2
    (r,) = random_masses(bt, h, nb, seed)
    s = shape_of(w, bt, h, nb)
    rng = np.random.default_rng(seed)
    rp, ci = [0], []
    for _ in range(bt * h):
        for qb in range(nb):
            k = int(rng.integers(1, qb + 2))
            ci.extend(sorted(rng.choice(qb + 1, size=k, replace=False).tolist()))
            rp.append(len(ci))
    rp, ci = np.array(rp, np.int32), np.array(ci, np.int32)
    row_mass = torch.empty((bt * h * nb, 2), dtype=torch.float64, device="cuda")
    totals = torch.empty(2, dtype=torch.float64, device="cuda")
    w.wise_support_mass(s, torch.from_numpy(r).cuda(), torch.from_numpy(rp).cuda(),
                        torch.from_numpy(ci).cuda(), row_mass, totals)
    torch.cuda.synchronize()
    want = O.support_block_mass(r, rp, ci)
    got = row_mass.cpu().numpy()
    np.testing.assert_allclose(got, want, rtol=1e-12, atol=1e-15)
    t = totals.cpu().numpy()
    np.testing.assert_allclose(t, want.sum(0), rtol=1e-12)


def test_retained_mass_against_probabilities(gpu_lib):
    """The GPU's fraction (block masses of its own dense pass) against the
    oracle's from the attention probabilities of the same bf16 inputs."""
    w = gpu_lib
    bt, h, n, d, B = 1, 2, 512, 64, 64
    say(f"retained mass vs probabilities bt={bt} h={h} n={n} d={d} B={B}")
    g = torch.Generator().manual_seed(11)
    q, k, v = [(torch.randn((bt, h, n, d), generator=g) * sc).to(torch.bfloat16)
               for sc in (2.0, 1.0, 1.0)]
    s = w.make_shape(bt, h, n, d, B)
    nb = n // B
    rng = np.random.default_rng(3)
    rp, ci = [0], []
    for _ in range(bt * h):
        for qb in range(nb):
            ci.extend(sorted({0, qb} | set(rng.integers(0, qb + 1, size=2).tolist())))
            rp.append(len(ci))
    rp, ci = np.array(rp, np.int32), np.array(ci, np.int32)
    sched = w.Schedule(s)
    sched.row_ptr.copy_(torch.from_numpy(rp))
    sched.col_idx[: ci.size].copy_(torch.from_numpy(ci))
    frac, row_mass = diagnostics.retained_mass(s, q.cuda(), k.cuda(), v.cuda(), sched)
    per_head, want = O.retained_mass(f64(q), f64(k), rp, ci, B)
    say(f"  retained {frac:.6f} oracle {want:.6f}")
    assert abs(frac - want) <= ACC_TOL
    rm = row_mass.cpu().numpy()
    np.testing.assert_allclose(rm[:, 1], 1.0, atol=ACC_TOL)


@pytest.mark.parametrize("block", [64, 16])
def test_union_trajectory_tiny(gpu_lib, block):
    """Union mode end to end on the tiny workload: per-step masses on the
    GPU, union CSR bit-exact on those masses, end to end against the
    oracle's own masses (near-ties reported), and late-step attention."""
    cfg = CONFIGS["tiny"].with_(block=block)
    say(f"union trajectory {cfg.name}")
    tr = Trajectory(cfg, device="cpu")
    steps = [tr.next(torch.bfloat16) for _ in range(cfg.steps)]
    pipe = WisePipeline.for_config(cfg, mode="union")
    out = torch.empty(steps[0][0].shape, dtype=torch.bfloat16, device="cuda")
    gpu_r = []
    pipe.reset()
    for t in range(1, cfg.discovery_steps + 1):
        q, k, v = (x.cuda() for x in steps[t - 1])
        pipe.discovery_step(q, k, v, out, accumulate=t in cfg.window)
        if t in cfg.window:
            gpu_r.append(pipe.acc.cpu().numpy().copy())
    pipe.select()
    torch.cuda.synchronize()
    tau = float(np.float32(cfg.tau))
    nb = cfg.nb
    rp = pipe.schedule.row_ptr.cpu().numpy()
    ci = pipe.schedule.col_idx[: int(rp[-1])].cpu().numpy()
    # the oracle's per-step masses and union from the same inputs
    ref_r = [O.block_mass(f64(steps[t - 1][0]), f64(steps[t - 1][1]), cfg.block)
             for t in cfg.window]
    for a, b in zip(gpu_r, ref_r):
        assert np.abs(a - b).max() <= ACC_TOL
    rp_o, ci_o = O.select_support_union(ref_r, tau, pipe.flags)
    rows_o, rows_g = O.csr_rows(rp_o, ci_o), O.csr_rows(rp, ci)
    near = False
    for i, (g_, o_) in enumerate(zip(rows_g, rows_o)):
        if g_ != o_:
            assert g_ in union_options([r.reshape(-1, nb)[i] for r in ref_r], i % nb, tau,
                                       pipe.flags), i
            say(f"  near-tie row {i} reported")
            near = True
    q, k, v = steps[cfg.discovery_steps]
    if near:   # run the late step over the oracle's union instead
        s = pipe.schedule
        s.row_ptr.copy_(torch.from_numpy(rp_o))
        s.col_idx[: ci_o.size].copy_(torch.from_numpy(ci_o))
        s.row_order.copy_(torch.from_numpy(O.schedule_order(rp_o, nb)))
    pipe.late_step(q.cuda(), k.cuda(), v.cuda(), out)
    torch.cuda.synchronize()
    o_ref, _ = O.sparse_attention(f64(q), f64(k), f64(v), rp_o, ci_o, cfg.block)
    assert_attn(out, o_ref, "union late step")


def union_options(refs, qb, tau, flags):
    """Every union a near tie admits: each step's own set, or one of the
    alternatives its cut admits (tie_alternatives), unioned with the forced
    blocks."""
    per_step = [[O.select_row(r, qb, tau, flags=0)] + tie_alternatives(r, qb, tau, 0)
                for r in refs]
    forced = ({0} if flags & 1 else set()) | ({qb} if flags & 2 else set())
    out = []
    for combo in itertools.product(*per_step):
        u = set(forced)
        for c in combo:
            u.update(c)
        out.append(sorted(u or {qb}))
    return out


# Whole query heads checked: one in a short last XCD group at 55 and 220
# heads (see test_gpu_fullsize), two on different key-value heads for 4k-gqa.
UNION_WHOLE = {"4k-pr": (3, 30), "8k": (5, 54), "4k-b32": (26, 219), "4k-b16": (26, 219),
               "4k-gqa": (0, 101)}


@pytest.mark.timeout(600)
@pytest.mark.parametrize("name", ["4k-pr", "8k", "4k-b32", "4k-b16", "4k-gqa"])
def test_union_fullsize(gpu_lib, name):
    """Full-size union mode on whole heads: every row's per-step masses
    against the oracle's, every CSR row against the oracle's union of its own
    per-step sets (a differing row passes only as a union a near tie admits),
    the late-step kernel on the oracle's union CSR against the oracle, every
    row of the GPU's CSR well formed with a valid row order, and the
    retained-mass diagnostic at that size."""
    w = gpu_lib
    cfg = CONFIGS[name]
    n, d, nb, B = cfg.seq_len, cfg.head_dim, cfg.nb, cfg.block
    bh = cfg.batch * cfg.heads
    sel = list(UNION_WHOLE[name])
    say(f"union full-size {name}: whole heads {sel}")
    tr = Trajectory(cfg, device="cuda")
    pipe = WisePipeline.for_config(cfg, mode="union")
    tau = float(np.float32(cfg.tau))
    out = None
    gpu_r, host = [], {}
    idx = torch.tensor(sel, device="cuda")

    def kv_of(s):
        b, h = divmod(s, cfg.heads)
        return b * cfg.kvh + O.kv_head(h, cfg.heads, cfg.kvh)

    kidx = torch.tensor([kv_of(s) for s in sel], device="cuda")
    td = cfg.discovery_steps
    for t in range(1, td + 2):
        q, k, v = tr.next(torch.bfloat16)
        if out is None:
            out = torch.empty_like(q)
        if t in cfg.window or t == td + 1:
            fq, fk, fv = (x.view(-1, n, d) for x in (q, k, v))
            hq, hk, hv = (f64(x.index_select(0, i)) for x, i in ((fq, idx), (fk, kidx), (fv, kidx)))
            host[t] = {s: (hq[j], hk[j], hv[j]) for j, s in enumerate(sel)}
        if t <= td:
            pipe.discovery_step(q, k, v, out, accumulate=t in cfg.window)
            if t in cfg.window:
                gpu_r.append(f64(pipe.acc.view(-1, nb, nb).index_select(0, idx)))
        else:
            pipe.select()
            frac, _ = diagnostics.retained_mass(pipe.shape, q, k, v, pipe.schedule)
            step_in = (q, k, v)
    torch.cuda.synchronize()
    rp = pipe.schedule.row_ptr.cpu().numpy()
    ci = pipe.schedule.col_idx[: int(rp[-1])].cpu().numpy()
    check_csr(rp, ci, nb, pipe.flags)
    check_row_order(pipe.schedule.row_order.cpu().numpy(), rp, nb)
    orc = HeadOracle(host, B, 1.0 / np.sqrt(d), chunk=max(1, 8 * 4096 // n))
    refs = [orc.block_masses(t) for t in cfg.window]
    for j, r in enumerate(refs):
        err = max(np.abs(gpu_r[j][i] - r[s])[np.tril_indices(nb)].max() for i, s in enumerate(sel))
        assert err <= ACC_TOL, f"step {cfg.window[j]} masses: {err:.3g}"
    rows = [[int(x) for x in ci[rp[r]:rp[r + 1]]] for r in range(bh * nb)]
    oracle_rows = {s: [] for s in sel}
    reported = 0
    for s in sel:
        for qb in range(nb):
            rr = [r[s][qb] for r in refs]
            want = set()
            for r in rr:
                want.update(O.select_row(r, qb, tau, flags=0))
            want = sorted(want | {0, qb})
            got = rows[s * nb + qb]
            if got != want:
                assert got in union_options(rr, qb, tau, pipe.flags), \
                    f"head {s} row {qb}: {got} vs {want}"
                reported += 1
            oracle_rows[s].append(want)
            rows[s * nb + qb] = want
    say(f"  {len(sel) * nb} union rows checked, near-tie rows reported {reported}")
    rp_o = np.zeros(len(rows) + 1, np.int32)
    rp_o[1:] = np.cumsum([len(r) for r in rows])
    ci_o = np.array([b for r in rows for b in r], np.int32)
    o2 = torch.empty_like(out)
    q, k, v = step_in
    w.wise_sparse_attn(pipe.shape, q, k, v, torch.from_numpy(rp_o).cuda(),
                       torch.from_numpy(ci_o).cuda(),
                       torch.from_numpy(O.schedule_order(rp_o, nb)).cuda(), o2, None)
    torch.cuda.synchronize()
    ref = orc.sparse(td + 1, oracle_rows)
    assert_attn(f64(o2.view(-1, n, d).index_select(0, idx)),
                np.stack([ref[s][0] for s in sel]), "union late step O (oracle CSR)")
    if w.wise_sparse_group_rows(pipe.shape) > 0:
        o3 = torch.empty_like(out)
        w.wise_sparse_attn_grouped(pipe.shape, q, k, v, torch.from_numpy(rp_o).cuda(),
                                   torch.from_numpy(ci_o).cuda(), o3, None)
        torch.cuda.synchronize()
        assert torch.equal(o2, o3)
        say(f"  grouped late step on the union CSR bitwise equal to the one-row kernel")
    dens = rp[-1] / (bh * nb * (nb + 1) / 2)
    say(f"  union density {dens:.4f}, retained future mass (step t_d+1) {frac:.4f}")
    assert 0.0 < frac <= 1.0 + 1e-9 and frac >= 0.9 * cfg.tau
