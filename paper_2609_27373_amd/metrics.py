"""Work accounting for the benchmark (host-side integer arithmetic only).

Effective FLOPs of attention restricted to a block support count 4*d FLOPs per
admitted (query, key) pair — 2*d for the score, 2*d for the value product —
with an off-diagonal block contributing block^2 pairs and the diagonal block
its block*(block+1)/2 causal pairs (Section 4's O(nmd) late-routing cost with
m the admitted keys per query).  Dense causal attention under the same
convention is 4*d*batch*heads*n*(n+1)/2.
"""

from __future__ import annotations

import numpy as np


def support_pairs(row_ptr, col_idx, nb: int, block: int) -> int:
    """Admitted (query, key) pairs of a CSR support (causal within the diagonal)."""
    rp = np.asarray(row_ptr, dtype=np.int64)
    ci = np.asarray(col_idx[: int(rp[-1])], dtype=np.int64)
    rows = np.repeat(np.arange(rp.size - 1, dtype=np.int64), np.diff(rp))
    qb = rows % nb
    diag = ci == qb
    off = (ci < qb)
    return int(off.sum()) * block * block + int(diag.sum()) * block * (block + 1) // 2


def effective_flops(row_ptr, col_idx, nb: int, block: int, head_dim: int) -> int:
    return 4 * head_dim * support_pairs(row_ptr, col_idx, nb, block)


def dense_flops(batch: int, heads: int, n: int, head_dim: int) -> int:
    return 4 * head_dim * batch * heads * n * (n + 1) // 2


def density(row_ptr, nb: int, bh: int) -> float:
    """Fraction of causally admissible blocks kept: nnz / (bh * nb(nb+1)/2)."""
    return float(np.asarray(row_ptr)[-1]) / (bh * nb * (nb + 1) / 2)
