"""Pure-Python element loops for tiny shapes — TEST INFRASTRUCTURE ONLY.

A second, deliberately naive reading of the same definitions the numpy oracle
implements, used to pin it: scalar loops over positions with math.exp, no
vectorisation, no numpy.  Inputs are nested lists (or anything indexable) of
floats for ONE (batch, head): q[i][c], k[j][c], v[j][c].

  attention        Section 3, eq. (recurrent_attention)
  block_mass       Section 5.1, eq. (block_attention_mass)
  min_support      Section 5.1, eq. (block_working_set) by exhaustive search
                   over all subsets of the admissible blocks
  masked_attention Section 5.2, eq. (wise_attention)
"""

from __future__ import annotations

import itertools
import math


def attention(q, k, v, scale):
    """Causal softmax attention; returns (A as list of rows, O, lse)."""
    n = len(q)
    dv = len(v[0])
    A, O, L = [], [], []
    for i in range(n):
        scores = []
        for j in range(i + 1):                     # admissible keys j <= i
            s = 0.0
            for c in range(len(q[i])):
                s += q[i][c] * k[j][c]
            scores.append(s * scale)
        m = max(scores)
        ex = [math.exp(s - m) for s in scores]
        z = sum(ex)
        row = [e / z for e in ex] + [0.0] * (n - i - 1)
        A.append(row)
        O.append([sum(row[j] * v[j][c] for j in range(n)) for c in range(dv)])
        L.append(m + math.log(z))
    return A, O, L


def block_mass(A, block):
    """r[qb][kb] = (1/B) sum_{i in I_qb} sum_{j in I_kb} A[i][j]."""
    n = len(A)
    nb = n // block
    r = [[0.0] * nb for _ in range(nb)]
    for qb in range(nb):
        for kb in range(nb):
            tot = 0.0
            for i in range(qb * block, (qb + 1) * block):
                for j in range(kb * block, (kb + 1) * block):
                    tot += A[i][j]
            r[qb][kb] = tot / block
    return r


def min_support(v, qb, tau):
    """All minimum-cardinality subsets S of {0..qb} with sum_S v >= tau*sum(v).

    Exhaustive: tries k = 0, 1, 2, ... and returns (k, list of every k-subset
    that reaches the threshold).  Exponential; only for qb <= ~10.
    """
    cand = list(range(qb + 1))
    total = sum(v[b] for b in cand)
    thr = tau * total
    for kk in range(0, qb + 2):
        hits = [set(c) for c in itertools.combinations(cand, kk)
                if sum(v[b] for b in c) >= thr]
        if hits:
            return kk, hits
    raise AssertionError("unreachable for tau <= 1")


def masked_attention(q, k, v, scale, block, support):
    """Attention where key j is visible to query i iff j <= i and
    j // block is in support[i // block] (a dict or list of sets)."""
    n = len(q)
    dv = len(v[0])
    O, L = [], []
    for i in range(n):
        vis = [j for j in range(i + 1) if (j // block) in support[i // block]]
        if not vis:
            O.append([0.0] * dv)
            L.append(-math.inf)
            continue
        scores = {}
        for j in vis:
            scores[j] = scale * sum(q[i][c] * k[j][c] for c in range(len(q[i])))
        m = max(scores.values())
        ex = {j: math.exp(s - m) for j, s in scores.items()}
        z = sum(ex.values())
        O.append([sum(ex[j] / z * v[j][c] for j in vis) for c in range(dv)])
        L.append(m + math.log(z))
    return O, L
