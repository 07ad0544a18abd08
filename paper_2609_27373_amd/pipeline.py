"""Host driver of one WISE trajectory over the libwise C ABI.

Section 5 of the paper in three phases, all on the device:
  discovery  steps 1..t_d: full causal attention; steps in the window also
             pool their attention mass into the fp32 accumulator
  selection  once after step t_d: per-row support + CSR + row order
  reuse      steps t_d+1..T: attention restricted to the fixed support, with
             this step's Q/K/V

Buffers are allocated once per trajectory (torch device memory); every call
enqueues on the current stream and returns.
"""

from __future__ import annotations

import torch

from . import wise


class WisePipeline:
    def __init__(self, batch, heads, seq_len, head_dim, block, tau, flags=wise.WISE_DEFAULT_FLAGS,
                 scale=0.0, device="cuda"):
        self.shape = wise.make_shape(batch, heads, seq_len, head_dim, block, scale)
        self.tau = float(tau)
        self.flags = int(flags)
        nb = seq_len // block
        self.acc = torch.zeros((batch, heads, nb, nb), dtype=torch.float32, device=device)
        self.lse = torch.empty((batch, heads, seq_len), dtype=torch.float32, device=device)
        self.schedule = wise.Schedule(self.shape, device)

    @classmethod
    def for_config(cls, cfg, tau=None, **kw):
        return cls(cfg.batch, cfg.heads, cfg.seq_len, cfg.head_dim, cfg.block,
                   cfg.tau if tau is None else tau, **kw)

    def reset(self):
        self.acc.zero_()

    def discovery_step(self, q, k, v, out, accumulate: bool):
        wise.wise_dense_attn_accum(self.shape, q, k, v, out, self.lse,
                                   self.acc if accumulate else None)
        return out

    def dense_step(self, q, k, v, out, lse=None):
        wise.wise_dense_attn_accum(self.shape, q, k, v, out, lse, None)
        return out

    def select(self):
        self.schedule.select(self.acc, self.tau, self.flags)
        return self.schedule

    def late_step(self, q, k, v, out, lse=None, ordered=True):
        s = self.schedule
        wise.wise_sparse_attn(self.shape, q, k, v, s.row_ptr, s.col_idx,
                              s.row_order if ordered else None, out, lse)
        return out
