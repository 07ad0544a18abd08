"""Seeded input generator: determinism, shapes, head-subset reproduction and
the planted structure the workloads promise."""

import numpy as np
import torch

from paper_2609_27373_amd.workloads import CONFIGS, Trajectory, planted_base, relevant_blocks


def test_configs_divide():
    for c in CONFIGS.values():
        assert c.seq_len % c.block == 0 and c.head_dim in (64, 96, 128) and c.block in (16, 32, 64, 128)
        assert c.heads % c.kvh == 0
        assert 1 <= len(c.window) <= 4 and c.window[-1] == c.discovery_steps


def test_relevant_blocks_structure():
    c = CONFIGS["4k"]
    rel = relevant_blocks(c)
    assert len(rel) == c.heads and len(rel[0]) == c.nb
    for per_q in rel[:3]:
        for q, r in enumerate(per_q):
            assert r.max() <= q and (q == 0 or 0 in r)
            assert len(r) == (1 if q <= 1 else min(5, q))
    c4 = CONFIGS["32k"]
    sizes = [len(r) for r in relevant_blocks(c4)[0][40:]]
    assert min(sizes) == 1 and max(sizes) == 32


def test_deterministic_and_subset_reproduces():
    c = CONFIGS["tiny"]
    a = Trajectory(c)
    b = Trajectory(c)
    for _ in range(3):
        xa, xb = a.next(), b.next()
    for u, w in zip(xa, xb):
        assert torch.equal(u, w)
    sub = Trajectory(c, heads=[1])
    for _ in range(3):
        xs = sub.next()
    for u, w in zip(xa, xs):
        assert torch.equal(u[:, 1], w[:, 0])


def test_random_walk_and_dtype():
    c = CONFIGS["4k"]
    tr = Trajectory(c, heads=[0])
    q1, _, _ = tr.next()
    q2, _, _ = tr.next()
    assert q1.dtype == torch.bfloat16
    diff = (q2.float() - q1.float()).std().item()
    assert 0.01 < diff < 0.04
    Q0, K0, V0 = planted_base(c, heads=[0])
    assert abs(K0.std().item() - 1) < 0.01 and abs(V0.mean().item()) < 0.01


def test_flop_accounting():
    from paper_2609_27373_amd import metrics
    nb, B, d = 4, 8, 16
    # full support == dense causal count
    rp, ci = [0], []
    for qb in range(nb):
        ci.extend(range(qb + 1))
        rp.append(len(ci))
    n = nb * B
    assert metrics.effective_flops(rp, ci, nb, B, d) == metrics.dense_flops(1, 1, n, d)
    # brute-force pair count on a random support
    rng = np.random.default_rng(0)
    rp, ci, want = [0], [], 0
    for qb in range(nb):
        s = sorted(set(rng.choice(qb + 1, size=2).tolist()))
        ci.extend(s)
        rp.append(len(ci))
        for i in range(qb * B, (qb + 1) * B):
            want += sum(1 for b in s for j in range(b * B, (b + 1) * B) if j <= i)
    assert metrics.support_pairs(rp, ci, nb, B) == want
    assert abs(metrics.density(rp, nb, 1) - len(ci) / 10) < 1e-12


def test_grouped_query_workload():
    """Key-value heads are shared: every query head of a group is planted on
    its group's K0, with its own relevant blocks; the walk moves K/V once per
    key-value head."""
    c = CONFIGS["tiny"].with_(batch=2, heads=4, kv_heads=2, seq_len=256)
    q0, k0, v0 = planted_base(c)
    assert q0.shape == (2, 4, 256, 64) and k0.shape == (2, 2, 256, 64) == v0.shape
    rel = relevant_blocks(c)
    B, nb = c.block, c.nb
    for b in range(2):
        for h in range(4):
            kt = k0[b, h // 2].reshape(nb, B, -1)
            for q in range(1, nb):
                # the query tile minus its planted mean is the 0.5-std noise
                resid = q0[b, h, q * B:(q + 1) * B] - c.gain * kt[rel[b * 4 + h][q]].mean(0)
                assert abs(resid.std().item() - c.noise) < 0.05
    tr, tr2 = Trajectory(c), Trajectory(c)
    for _ in range(2):
        a, a2 = tr.next(), tr2.next()
    for x, y in zip(a, a2):
        assert torch.equal(x, y)
    assert a[1].shape == (2, 2, 256, 64)
    import pytest
    with pytest.raises(ValueError):
        planted_base(c, heads=[0])
