"""Plain CPU oracle for the WISE hot path — TEST INFRASTRUCTURE ONLY.

Only the test suite, the smoke check and the benchmark's CPU-baseline leg may
import this module.  The product path (the HIP library and its binding) never
calls it, and it shares no code with that path.

Everything here is numpy float64 on whatever values it is handed (callers pass
the same bf16-rounded inputs the GPU sees, converted exactly to float64).  Each
function is the plain definition from the paper, written out without blocking,
fusion or reordering beyond what the definition states:

  dense_attention         Section 3, eq. (recurrent_attention)
  block_mass              Section 5.1, eq. (block_attention_mass)
  accumulate              sum of per-step block masses over a discovery window
  select_support          Section 5.1, eq. (block_working_set), per-step arg-min
                          set, plus forced sink / diagonal blocks
  select_support_union    Section 5.1, eq. (block_working_set), the paper's
                          temporal union of per-step supports
  step_supports           the per-step sets B_q^(t, eta) inside that union
  rolling_working_set     Appendix C, "Stability of the Deployed Working Set":
                          W_q^(t), the union over steps max(1, t-3)..t
  overlap_counts, jaccard the adjacent rolling-set Jaccard J_roll of the same
                          subsection, as |A & B| and |A | B| over all
                          (batch, head, query block, key block) memberships
  retained_mass           Section 7.1 and Appendix B (evaluation metrics):
                          the fraction of unrestricted full-attention mass of
                          a step that falls inside a support, from the
                          attention probabilities themselves
  support_block_mass      the same quantity from block masses, per row
  expand_kv               grouped-query attention (Appendix B: the second
                          backbone has 32 query heads sharing 8 key-value
                          heads): query head h reads key-value head
                          h // (heads / kv_heads); expanding K, V to one copy
                          per query head turns every function above into its
                          grouped form
  schedule_order          per-head longest-support-first ordering of CSR rows
  sparse_attention        Section 5.2, eq. (wise_attention), gather form
  sparse_attention_masked Section 5.2, eq. (wise_attention) with the mask R
  support_margins         the nondegeneracy margins delta^-, delta^+,
                          delta^rank of Appendix A (proof of Theorem 1)

Shapes: q, k, v are [batch][heads][n][d]; block masses / accumulators are
[batch][heads][nb][nb] with nb = n // block; CSR row r = (b*heads + h)*nb + qb.
"""

from __future__ import annotations

import numpy as np

FORCE_SINK = 1
FORCE_DIAG = 2


def _f64(x):
    return np.asarray(x, dtype=np.float64)


def default_scale(d: int) -> float:
    """1/sqrt(d_h), the temperature of Section 3, eq. (recurrent_attention)."""
    return 1.0 / np.sqrt(float(d))


def kv_head(h, heads, kv_heads):
    """Key-value head read by query head h under grouped-query attention."""
    if heads % kv_heads:
        raise ValueError("heads must be a multiple of kv_heads")
    return h // (heads // kv_heads)


def expand_kv(x, heads):
    """[bt][kv_heads][n][d] -> [bt][heads][n][d]: query head h gets a copy
    of key-value head kv_head(h, heads, kv_heads)."""
    x = _f64(x)
    kvh = x.shape[1]
    return x[:, [kv_head(h, heads, kvh) for h in range(heads)]]


# ---------------------------------------------------------------------------
# Section 3, eq. (recurrent_attention): A = softmax(QK^T/sqrt(d_h) + M), O = AV
# ---------------------------------------------------------------------------

def causal_attention_rows(qh, kh, vh, rows, scale):
    """Attention of one (batch, head) for the query positions `rows`.

    qh, kh, vh: [n][d] float64.  Returns (A, O, lse) where A is
    [len(rows)][n] (zero where the causal mask M forbids j > i), O is
    [len(rows)][d] and lse is the natural-log normaliser of each row.
    """
    rows = np.asarray(rows)
    s = (qh[rows] @ kh.T) * scale                      # scores QK^T / sqrt(d)
    n = kh.shape[0]
    allowed = np.arange(n)[None, :] <= rows[:, None]   # causal mask M
    s = np.where(allowed, s, -np.inf)
    m = s.max(axis=1, keepdims=True)
    e = np.exp(s - m)
    l = e.sum(axis=1, keepdims=True)
    a = e / l                                          # softmax rows
    o = a @ vh
    lse = (m + np.log(l))[:, 0]
    return a, o, lse


def dense_attention(q, k, v, scale=None, chunk=256):
    """O and natural-log LSE of full causal attention, for every head.

    Rows are processed in independent chunks only to bound memory; each row
    is the plain softmax of its own scores.
    """
    q, k, v = _f64(q), _f64(k), _f64(v)
    bt, h, n, d = q.shape
    scale = default_scale(d) if scale is None else float(scale)
    o = np.zeros_like(q)
    lse = np.zeros((bt, h, n))
    for b in range(bt):
        for hh in range(h):
            for r0 in range(0, n, chunk):
                rows = np.arange(r0, min(n, r0 + chunk))
                _, o_r, l_r = causal_attention_rows(q[b, hh], k[b, hh], v[b, hh], rows, scale)
                o[b, hh, rows] = o_r
                lse[b, hh, rows] = l_r
    return o, lse


# ---------------------------------------------------------------------------
# Section 5.1, eq. (block_attention_mass):
#   r_qb = (1/|I_q|) sum_{i in I_q} sum_{j in I_b} A_ij
# ---------------------------------------------------------------------------

def block_mass_row(qh, kh, qb, block, scale):
    """r_{qb, .} for one (batch, head) and one query block: vector of length nb."""
    n = kh.shape[0]
    rows = np.arange(qb * block, (qb + 1) * block)
    a, _, _ = causal_attention_rows(qh, kh, np.zeros((n, 1)), rows, scale)
    per_key = a.sum(axis=0)                            # sum over i in I_q
    per_block = per_key.reshape(n // block, block).sum(axis=1)   # sum over j in I_b
    return per_block / block                           # 1/|I_q|


def block_mass(q, k, block, scale=None):
    """Block masses of one step for every head: [batch][heads][nb][nb]."""
    q, k = _f64(q), _f64(k)
    bt, h, n, d = q.shape
    scale = default_scale(d) if scale is None else float(scale)
    nb = n // block
    r = np.zeros((bt, h, nb, nb))
    for b in range(bt):
        for hh in range(h):
            for qb in range(nb):
                r[b, hh, qb] = block_mass_row(q[b, hh], k[b, hh], qb, block, scale)
    return r


def accumulate(step_masses):
    """acc = sum over the discovery-window steps of r^(t)."""
    acc = None
    for r in step_masses:
        acc = _f64(r).copy() if acc is None else acc + _f64(r)
    return acc


# ---------------------------------------------------------------------------
# Section 5.1, eq. (block_working_set): smallest set of admissible key blocks
# whose cumulative mass reaches eta.  The smallest such set is the top-k*
# blocks by mass (any k-set has at most the mass of the k heaviest), with
# k* the first prefix of the descending order that reaches the threshold.
# ---------------------------------------------------------------------------

def select_row(v, qb, tau, flags=FORCE_SINK | FORCE_DIAG):
    """Support of one row from masses v[0..qb] (entries past qb ignored).

    Order: mass descending, block index ascending on ties.  Prefix sums are
    sequential in that order, in float64; the threshold is tau times the
    row's own total.  Forced blocks are added after the cut.  Returns the
    sorted list of block ids.
    """
    v = _f64(v)[: qb + 1]
    tau = float(tau)
    idx = np.arange(qb + 1)
    order = np.lexsort((idx, -v))                      # primary: -v, secondary: idx
    c = np.concatenate(([0.0], np.cumsum(v[order])))   # c_0 .. c_{qb+1}
    total = c[-1]
    thr = tau * total
    kstar = int(np.argmax(c >= thr))                   # first k with c_k >= thr
    if not (c >= thr).any():                           # cannot happen for tau <= 1
        kstar = qb + 1
    chosen = set(int(b) for b in order[:kstar])
    if flags & FORCE_SINK:
        chosen.add(0)
    if flags & FORCE_DIAG:
        chosen.add(qb)
    if not chosen:
        chosen.add(qb)
    return sorted(chosen)


def select_support(acc, tau, flags=FORCE_SINK | FORCE_DIAG):
    """CSR (row_ptr int32[rows+1], col_idx int32[nnz]) for every row."""
    acc = _f64(acc)
    bt, h, nb, _ = acc.shape
    row_ptr = [0]
    col_idx = []
    for b in range(bt):
        for hh in range(h):
            for qb in range(nb):
                s = select_row(acc[b, hh, qb], qb, tau, flags)
                col_idx.extend(s)
                row_ptr.append(len(col_idx))
    return np.asarray(row_ptr, dtype=np.int32), np.asarray(col_idx, dtype=np.int32)


def select_support_union(step_masses, tau, flags=FORCE_SINK | FORCE_DIAG):
    """The paper's working set: union over the window of per-step supports
    B_q^(t, eta), each selected without forced blocks, then the forced blocks."""
    masses = [_f64(r) for r in step_masses]
    bt, h, nb, _ = masses[0].shape
    row_ptr = [0]
    col_idx = []
    for b in range(bt):
        for hh in range(h):
            for qb in range(nb):
                u = set()
                for r in masses:
                    u.update(select_row(r[b, hh, qb], qb, tau, flags=0))
                if flags & FORCE_SINK:
                    u.add(0)
                if flags & FORCE_DIAG:
                    u.add(qb)
                if not u:
                    u.add(qb)
                col_idx.extend(sorted(u))
                row_ptr.append(len(col_idx))
    return np.asarray(row_ptr, dtype=np.int32), np.asarray(col_idx, dtype=np.int32)


def step_supports(step_mass, tau):
    """B_q^(t, eta) of one step for every row (no forced blocks): list over
    rows r = (b*heads + h)*nb + qb of sorted block-id lists."""
    r = _f64(step_mass)
    bt, h, nb, _ = r.shape
    flat = r.reshape(bt * h * nb, nb)
    return [select_row(flat[i], i % nb, tau, flags=0) for i in range(bt * h * nb)]


def csr_rows(row_ptr, col_idx):
    """CSR -> list over rows of block-id lists."""
    return [[int(x) for x in col_idx[row_ptr[i]:row_ptr[i + 1]]] for i in range(len(row_ptr) - 1)]


def rolling_working_set(per_step, t, width=4):
    """W_q^(t) = union of B_q^(s) for s = max(1, t - width + 1) .. t.

    per_step[s - 1] is step s's support (list over rows of block-id lists,
    as from step_supports); returns a list over rows of sorted lists."""
    lo = max(1, t - width + 1)
    rows = len(per_step[0])
    out = []
    for i in range(rows):
        u = set()
        for s in range(lo, t + 1):
            u.update(per_step[s - 1][i])
        out.append(sorted(u))
    return out


def overlap_counts(a_rows, b_rows):
    """(|A & B|, |A | B|) of two supports read as sets of (row, key block)."""
    inter = union = 0
    for x, y in zip(a_rows, b_rows):
        x, y = set(x), set(y)
        inter += len(x & y)
        union += len(x | y)
    return inter, union


def jaccard(a_rows, b_rows):
    """|A & B| / |A | B| over (row, key block) memberships (1 for two empty sets)."""
    i, u = overlap_counts(a_rows, b_rows)
    return 1.0 if u == 0 else i / u


def retained_mass(q, k, row_ptr, col_idx, block, scale=None):
    """Fraction of the unrestricted causal attention mass of one step that
    lies inside a block support: sum of A_ij over causal (i, j) with
    b(j) in B_{q(i)}, over the sum of A_ij over all causal (i, j) (= n per
    head).  Returns (per-head fractions [bt][h], overall fraction)."""
    q, k = _f64(q), _f64(k)
    bt, h, n, d = q.shape
    scale = default_scale(d) if scale is None else float(scale)
    allowed = working_set_mask(row_ptr, col_idx, n, block, bt, h)
    causal = np.tril(np.ones((n, n), dtype=bool))
    inside = np.zeros((bt, h))
    total = np.zeros((bt, h))
    for b in range(bt):
        for hh in range(h):
            s = np.where(causal, (q[b, hh] @ k[b, hh].T) * scale, -np.inf)
            a = np.exp(s - s.max(axis=1, keepdims=True))
            a /= a.sum(axis=1, keepdims=True)
            inside[b, hh] = a[allowed[b, hh] & causal].sum()
            total[b, hh] = a.sum()
    return inside / total, inside.sum() / total.sum()


def support_block_mass(step_mass, row_ptr, col_idx):
    """Per row (b, h, qb): (sum of r_{qb,kb} over kb in the row's support,
    sum of r_{qb,kb} over kb <= qb), from one step's block masses."""
    r = _f64(step_mass)
    bt, h, nb, _ = r.shape
    flat = r.reshape(bt * h * nb, nb)
    out = np.zeros((bt * h * nb, 2))
    for i in range(bt * h * nb):
        qb = i % nb
        blocks = [int(x) for x in col_idx[row_ptr[i]:row_ptr[i + 1]] if 0 <= x <= qb]
        out[i, 0] = flat[i, blocks].sum()
        out[i, 1] = flat[i, :qb + 1].sum()
    return out


def schedule_order(row_ptr, nb):
    """Rows grouped by (batch, head) = row // nb ascending; within a head by
    support size descending, ties by row id ascending."""
    row_ptr = np.asarray(row_ptr, dtype=np.int64)
    nnz = np.diff(row_ptr)
    rid = np.arange(nnz.size)
    return np.lexsort((rid, -nnz, rid // nb)).astype(np.int32)


def support_margins(v, qb, tau):
    """Nondegeneracy margins of one row's cut, normalised by the row total.

    With the row sorted descending (r_(1) >= r_(2) >= ...) and k* the cut:
      delta^-    = tau - c_{k*-1}        (how far the shorter prefix falls short)
      delta^+    = c_{k*} - tau          (how far the chosen prefix overshoots)
      delta^rank = (r_(k*) - r_(k*+1))/2 (gap between last kept and first dropped)
    as defined in Appendix A (proof of Theorem 1).  Missing neighbours give +inf.
    """
    v = _f64(v)[: qb + 1]
    total = v.sum()
    if total <= 0:
        return dict(delta_minus=np.inf, delta_plus=np.inf, delta_rank=np.inf, kstar=0)
    w = v / total
    idx = np.arange(qb + 1)
    order = np.lexsort((idx, -w))
    ws = w[order]
    c = np.concatenate(([0.0], np.cumsum(ws)))
    kstar = int(np.argmax(c >= tau))
    if not (c >= tau).any():
        kstar = qb + 1
    dm = tau - c[kstar - 1] if kstar >= 1 else np.inf
    dp = c[kstar] - tau
    dr = (ws[kstar - 1] - ws[kstar]) / 2 if 1 <= kstar < ws.size else np.inf
    return dict(delta_minus=dm, delta_plus=dp, delta_rank=dr, kstar=kstar)


# ---------------------------------------------------------------------------
# Section 5.2, eq. (wise_attention):
#   softmax(QK^T/sqrt(d_h) + M + R) V,  R_ij = 0 iff b(j) in B_{q(i)}
# ---------------------------------------------------------------------------

def sparse_attention_row(qh, kh, vh, qb, blocks, block, scale):
    """Gather form for one query block: keys = concatenation of the support's
    blocks; causal mask applied by absolute position.  Returns (O, lse) of the
    block's rows; a row with no admissible key gives O = 0, lse = -inf."""
    rows = np.arange(qb * block, (qb + 1) * block)
    if len(blocks) == 0:
        return np.zeros((block, vh.shape[1])), np.full(block, -np.inf)
    keys = np.concatenate([np.arange(b * block, (b + 1) * block) for b in blocks])
    s = (qh[rows] @ kh[keys].T) * scale
    s = np.where(keys[None, :] <= rows[:, None], s, -np.inf)
    m = s.max(axis=1, keepdims=True)
    dead = ~np.isfinite(m[:, 0])
    m = np.where(np.isfinite(m), m, 0.0)
    e = np.exp(s - m)
    l = e.sum(axis=1, keepdims=True)
    with np.errstate(invalid="ignore", divide="ignore"):
        a = e / l
        o = a @ vh[keys]
        lse = (m + np.log(l))[:, 0]
    o[dead] = 0.0
    lse[dead] = -np.inf
    return o, lse


def sparse_attention(q, k, v, row_ptr, col_idx, block, scale=None):
    """Late-step attention restricted to a CSR block support (gather form)."""
    q, k, v = _f64(q), _f64(k), _f64(v)
    bt, h, n, d = q.shape
    scale = default_scale(d) if scale is None else float(scale)
    nb = n // block
    o = np.zeros_like(q)
    lse = np.zeros((bt, h, n))
    r = 0
    for b in range(bt):
        for hh in range(h):
            for qb in range(nb):
                blocks = [int(x) for x in col_idx[row_ptr[r]:row_ptr[r + 1]]]
                rows = slice(qb * block, (qb + 1) * block)
                o[b, hh, rows], lse[b, hh, rows] = sparse_attention_row(
                    q[b, hh], k[b, hh], v[b, hh], qb, blocks, block, scale)
                r += 1
    return o, lse


def working_set_mask(row_ptr, col_idx, n, block, bt, h):
    """The additive mask R of Section 5.2 as a boolean 'allowed' tensor
    [bt][h][n][n] (True where R_ij = 0)."""
    nb = n // block
    allowed = np.zeros((bt, h, n, n), dtype=bool)
    r = 0
    for b in range(bt):
        for hh in range(h):
            for qb in range(nb):
                for kb in col_idx[row_ptr[r]:row_ptr[r + 1]]:
                    allowed[b, hh, qb * block:(qb + 1) * block, kb * block:(kb + 1) * block] = True
                r += 1
    return allowed


def sparse_attention_masked(q, k, v, row_ptr, col_idx, block, scale=None):
    """Masked-dense form: full scores with M and R added as -inf, then softmax."""
    q, k, v = _f64(q), _f64(k), _f64(v)
    bt, h, n, d = q.shape
    scale = default_scale(d) if scale is None else float(scale)
    allowed = working_set_mask(row_ptr, col_idx, n, block, bt, h)
    causal = np.tril(np.ones((n, n), dtype=bool))
    o = np.zeros_like(q)
    lse = np.zeros((bt, h, n))
    for b in range(bt):
        for hh in range(h):
            s = (q[b, hh] @ k[b, hh].T) * scale
            ok = allowed[b, hh] & causal
            s = np.where(ok, s, -np.inf)
            m = s.max(axis=1, keepdims=True)
            dead = ~np.isfinite(m[:, 0])
            m = np.where(np.isfinite(m), m, 0.0)
            e = np.exp(s - m)
            l = e.sum(axis=1, keepdims=True)
            with np.errstate(invalid="ignore", divide="ignore"):
                o[b, hh] = (e / l) @ v[b, hh]
                lse[b, hh] = (m + np.log(l))[:, 0]
            o[b, hh][dead] = 0.0
            lse[b, hh][dead] = -np.inf
    return o, lse
