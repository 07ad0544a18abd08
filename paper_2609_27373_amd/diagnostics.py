"""Routing diagnostics of a WISE trajectory, on the device over the C ABI.

  retained future mass  Section 7.1 and Appendix B (evaluation metrics): the
                        fraction of one late step's unrestricted causal
                        attention mass that falls inside the frozen support.
                        Runs the dense kernel with block-mass pooling on that
                        step (a diagnostic pass, never part of reuse) and sums
                        the pooled masses over the support.
  rolling stability     Appendix C, "Stability of the Deployed Working Set":
                        W^(t) = union of the per-step sets B^(s, eta) over
                        s = max(1, t-3)..t, and the adjacent Jaccard
                        J_roll^(t) = |W^(t-1) & W^(t)| / |W^(t-1) | W^(t)|,
                        reconstructed from unrestricted attention at every
                        step, plus J(W^(t_d), W^(T)).

Every number comes from the library's kernels; this module only allocates
buffers and reads back the few scalars it reports.
"""

from __future__ import annotations

import torch

from . import wise


def retained_mass(shape, q, k, v, schedule, scratch=None):
    """(fraction, row_mass) of one step's full-attention mass inside the
    support held by `schedule`.  `scratch` may supply (o, lse, r, workspace)
    buffers."""
    bh = shape.batch * shape.heads
    nb = shape.seq_len // shape.block
    dev = q.device
    if scratch is None:
        scratch = (torch.empty_like(q),
                   torch.empty((shape.batch, shape.heads, shape.seq_len), dtype=torch.float32,
                               device=dev),
                   torch.empty((shape.batch, shape.heads, nb, nb), dtype=torch.float32,
                               device=dev),
                   wise.mass_workspace(shape, dev))
    o, lse, r, ws = scratch
    r.zero_()
    wise.wise_dense_attn_accum(shape, q, k, v, o, lse, r, ws)
    row_mass = torch.empty((bh * nb, 2), dtype=torch.float64, device=dev)
    totals = torch.empty(2, dtype=torch.float64, device=dev)
    wise.wise_support_mass(shape, r, schedule.row_ptr, schedule.col_idx, row_mass, totals)
    t = totals.cpu()
    return float(t[0] / t[1]), row_mass


class RollingSets:
    """Per-step supports B^(t, eta) of unrestricted attention and the rolling
    working sets W^(t) over the last `width` steps, kept as device bitmasks."""

    def __init__(self, shape, tau, width=4, device="cuda"):
        self.shape = shape
        self.tau = float(tau)
        self.width = int(width)
        nb = shape.seq_len // shape.block
        rows = shape.batch * shape.heads * nb
        words = wise.wise_mask_words(shape)
        self.ring = torch.zeros((self.width, rows, words), dtype=torch.int64, device=device)
        self.cur = torch.zeros((rows, words), dtype=torch.int64, device=device)
        self.prev = torch.zeros_like(self.cur)
        self.counts = torch.zeros(2, dtype=torch.int64, device=device)
        self.r = torch.empty((shape.batch, shape.heads, nb, nb), dtype=torch.float32,
                             device=device)
        self.lse = torch.empty((shape.batch, shape.heads, shape.seq_len), dtype=torch.float32,
                               device=device)
        self.ws = wise.mass_workspace(shape, device)
        self.t = 0

    def step(self, q, k, v, o):
        """Advance by one step of full attention; returns (|W^(t-1) & W^(t)|,
        |W^(t-1) | W^(t)|) for t >= 2, None for t = 1."""
        self.t += 1
        self.r.zero_()
        wise.wise_dense_attn_accum(self.shape, q, k, v, o, self.lse, self.r, self.ws)
        wise.wise_select_step(self.shape, self.r, self.tau, self.ring[(self.t - 1) % self.width])
        self.prev.copy_(self.cur)
        wise.wise_mask_union(self.shape, self.ring, min(self.t, self.width), self.cur)
        if self.t == 1:
            return None
        wise.wise_mask_overlap(self.shape, self.prev, self.cur, self.counts)
        c = self.counts.cpu()
        return int(c[0]), int(c[1])


def rolling_stability(shape, steps, tau, discovery_steps, width=4):
    """J_roll^(t) for t = 2..T over the trajectory `steps` (list of (q, k, v)),
    and J(W^(t_d), W^(T)).  Returns a dict of plain Python numbers."""
    rs = RollingSets(shape, tau, width, device=steps[0][0].device)
    o = torch.empty_like(steps[0][0])
    jroll = {}
    w_td = None
    for t, (q, k, v) in enumerate(steps, start=1):
        c = rs.step(q, k, v, o)
        if c is not None:
            jroll[t] = c[0] / c[1] if c[1] else 1.0
        if t == discovery_steps:
            w_td = rs.cur.clone()
    counts = torch.zeros(2, dtype=torch.int64, device=o.device)
    wise.wise_mask_overlap(shape, w_td, rs.cur, counts)
    c = counts.cpu()
    return {"j_roll": jroll, "j_td_T": float(c[0]) / float(c[1]) if int(c[1]) else 1.0}
