"""Oracle evaluation over whole heads, spread over threads (test
infrastructure).

numpy releases the GIL inside its array operations, so the oracle's per
query-block functions run in parallel from a thread pool (BLAS held to one
thread per worker).  Nothing here computes anything itself: every value comes
from an `oracle.wise_oracle` function called on host arrays that are the
same bf16-rounded inputs the GPU saw.
"""

from __future__ import annotations

import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np
from threadpoolctl import threadpool_limits

from oracle import wise_oracle as O


def workers() -> int:
    return max(1, min(16, int(os.environ.get("WISE_TEST_THREADS", os.cpu_count() or 1))))


def pmap(fn, items):
    items = list(items)
    with threadpool_limits(1), ThreadPoolExecutor(workers()) as ex:
        return list(ex.map(fn, items))


def _chunks(nb, size):
    return [list(range(a, min(nb, a + size))) for a in range(0, nb, size)]


class HeadOracle:
    """Per-head oracle results of one trajectory.

    inputs[t][s] = (q, k, v): float64 [n][d] of query head s at step t, with
    k, v the key-value head that query head reads.
    """

    def __init__(self, inputs, block, scale, chunk=8):
        self.inputs = inputs
        self.B = block
        self.scale = scale
        self.chunk = chunk

    def _heads(self, t):
        return sorted(self.inputs[t])

    def block_masses(self, t):
        """{s: [nb][nb]} block masses of step t (Section 5.1, eq. block_attention_mass)."""
        q0 = next(iter(self.inputs[t].values()))[0]
        nb = q0.shape[0] // self.B
        tasks = [(s, qbs) for s in self._heads(t) for qbs in _chunks(nb, self.chunk)]

        def run(task):
            s, qbs = task
            q, k, _ = self.inputs[t][s]
            return s, qbs, [O.block_mass_row(q, k, qb, self.B, self.scale) for qb in qbs]

        out = {s: np.zeros((nb, nb)) for s in self._heads(t)}
        for s, qbs, rows in pmap(run, tasks):
            for qb, r in zip(qbs, rows):
                out[s][qb] = r
        return out

    def dense(self, t):
        """{s: (O [n][d], lse [n])} of full causal attention at step t."""
        q0 = next(iter(self.inputs[t].values()))[0]
        n, d = q0.shape
        nb = n // self.B
        tasks = [(s, qbs) for s in self._heads(t) for qbs in _chunks(nb, self.chunk)]

        def run(task):
            s, qbs = task
            q, k, v = self.inputs[t][s]
            rows = np.arange(qbs[0] * self.B, (qbs[-1] + 1) * self.B)
            _, o, l = O.causal_attention_rows(q, k, v, rows, self.scale)
            return s, rows, o, l

        out = {s: (np.zeros((n, d)), np.zeros(n)) for s in self._heads(t)}
        for s, rows, o, l in pmap(run, tasks):
            out[s][0][rows] = o
            out[s][1][rows] = l
        return out

    def sparse(self, t, supports):
        """{s: (O, lse)} of attention restricted to supports[s][qb] at step t
        (Section 5.2, eq. wise_attention, gather form)."""
        q0 = next(iter(self.inputs[t].values()))[0]
        n, d = q0.shape
        nb = n // self.B
        tasks = [(s, qbs) for s in self._heads(t) for qbs in _chunks(nb, 4 * self.chunk)]

        def run(task):
            s, qbs = task
            q, k, v = self.inputs[t][s]
            return s, qbs, [O.sparse_attention_row(q, k, v, qb, supports[s][qb], self.B,
                                                   self.scale) for qb in qbs]

        out = {s: (np.zeros((n, d)), np.zeros(n)) for s in self._heads(t)}
        for s, qbs, res in pmap(run, tasks):
            for qb, (o, l) in zip(qbs, res):
                sl = slice(qb * self.B, (qb + 1) * self.B)
                out[s][0][sl] = o
                out[s][1][sl] = l
        return out
