"""Seeded input generator: determinism, shapes, head-subset reproduction and
the planted structure the workloads promise."""

import numpy as np
import torch

from paper_2609_27373_amd.workloads import CONFIGS, Trajectory, planted_base, relevant_blocks


def test_configs_divide():
    for c in CONFIGS.values():
        assert c.seq_len % c.block == 0 and c.head_dim in (64, 96, 128) and c.block in (64, 128)
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
