"""Host driver of one WISE trajectory over the libwise C ABI.

Section 5 of the paper in three phases, all on the device:
  discovery  steps 1..t_d: full causal attention; steps in the window also
             pool their attention mass
  selection  once after step t_d: per-row support + CSR + row order
  reuse      steps t_d+1..T: attention restricted to the fixed support, with
             this step's Q/K/V

Two selection rules (mode):
  "accumulate"  the window steps' block masses are summed into one fp32
                accumulator and selected once
  "union"       the paper's eq. (block_working_set): each window step's
                masses are selected on their own (B_q^(t, eta)) into a
                bitmask, and the support is the union of those sets

Two late-step kernels compute the same outputs (late_kernel):
  "rows"     wise_sparse_attn, one work-group per support row
  "grouped"  wise_sparse_attn_grouped, work-groups of consecutive rows over
             the union of their supports (faster where supports are dense)
  "auto"     grouped where the library offers it and the selected support's
             density (nnz over the causal block pairs) is at least
             group_density (by default the measured break-even of the
             library's group shape and head_dim, GROUP_DENSITY; some shapes
             never), rows otherwise.  The
             first select() reads nnz back (one synchronisation); later ones
             copy it to pinned host memory asynchronously, and the choice
             follows when the copy has landed (checked without waiting at
             each select() and late step), so the host never waits on the
             device again.  Both kernels give the same outputs, so when the
             switch happens does not change any result.  A select() under
             graph capture keeps the current choice.

Buffers are allocated once per trajectory (torch device memory); every call
enqueues on the current stream and returns (except the first select() in
"auto" mode, which waits for the selection to read its size).
"""

from __future__ import annotations

import torch

from . import wise


class WisePipeline:
    MODES = ("accumulate", "union")
    LATE_KERNELS = ("auto", "rows", "grouped")
    # Density from which "auto" picks the grouped kernel, by (block, rows per
    # group, head_dim); None: never (slower at every density measured).  The
    # union of consecutive rows' supports grows as the density falls, and the
    # break-even is where it costs what the shared staging saves.  Late step,
    # grouped over one-row time on the same supports:
    #   block 64, 4 rows, d 128: 1.36 at density 0.39, 1.18 at 0.58, 1.08 at
    #     0.69, 1.04 at 0.74, 0.95 at 0.80, 0.94 at 0.88, 0.88 at 0.91
    #   block 64, 2 rows, d 128 (lengths 256 does not divide): 1.05 at 0.80,
    #     about 1.03 at 0.91
    #   block 64, 2 rows, d 96: 1.01 at 0.30, 0.98 at 0.42 and 0.54, 1.00 at
    #     0.55, 0.97 at 0.66, 0.94 at 0.78, 0.90 at 0.89-0.95
    #   block 64, 2 rows, d 64: 1.07 at 0.23, 1.02 at 0.58, 0.92 at 0.89
    #   block 128, 2 rows, d 128: 1.01 at 0.70, 1.00 at 0.80, 0.97 at 0.91,
    #     0.97 at 0.96
    GROUP_DENSITY = {(64, 4, 128): 0.78, (64, 2, 128): None, (64, 2, 96): 0.40,
                     (64, 2, 64): 0.70, (128, 2, 128): 0.80}

    def __init__(self, batch, heads, seq_len, head_dim, block, tau, flags=wise.WISE_DEFAULT_FLAGS,
                 scale=0.0, device="cuda", mode="accumulate", window=4, kv_heads=0,
                 late_kernel="auto", group_density=None):
        if mode not in self.MODES:
            raise ValueError(f"mode must be one of {self.MODES}")
        if late_kernel not in self.LATE_KERNELS:
            raise ValueError(f"late_kernel must be one of {self.LATE_KERNELS}")
        self.shape = wise.make_shape(batch, heads, seq_len, head_dim, block, scale, kv_heads)
        self.tau = float(tau)
        self.flags = int(flags)
        self.mode = mode
        nb = seq_len // block
        # accumulate mode: the running sum; union mode: one step's masses
        self.acc = torch.zeros((batch, heads, nb, nb), dtype=torch.float32, device=device)
        self.lse = torch.empty((batch, heads, seq_len), dtype=torch.float32, device=device)
        self.schedule = wise.Schedule(self.shape, device)
        self.mass_ws = wise.mass_workspace(self.shape, device)
        self.window = int(window)
        self.masks = None
        if mode == "union":
            words = wise.wise_mask_words(self.shape)
            self.masks = torch.zeros((self.window, batch * heads * nb, words), dtype=torch.int64,
                                     device=device)
        self.filled = 0
        self.late_kernel = late_kernel
        group_rows = wise.wise_sparse_group_rows(self.shape)
        if group_density is None:
            group_density = self.GROUP_DENSITY.get((block, group_rows, head_dim))
        self.group_density = None if group_density is None else float(group_density)
        self.grouped = late_kernel == "grouped"
        self._auto = late_kernel == "auto" and group_rows > 0 and self.group_density is not None
        self._decided = False
        self._nnz_host = torch.empty(1, dtype=torch.int32, pin_memory=True) if self._auto else None
        self._nnz_event = None

    @classmethod
    def for_config(cls, cfg, tau=None, **kw):
        return cls(cfg.batch, cfg.heads, cfg.seq_len, cfg.head_dim, cfg.block,
                   cfg.tau if tau is None else tau, kv_heads=cfg.kv_heads, **kw)

    def reset(self):
        self.acc.zero_()
        self.filled = 0

    def discovery_step(self, q, k, v, out, accumulate: bool):
        """One discovery step; `accumulate` marks a step of the window."""
        if accumulate and self.mode == "union":
            if self.filled >= self.window:
                raise RuntimeError("more window steps than the union window holds")
            self.acc.zero_()
            wise.wise_dense_attn_accum(self.shape, q, k, v, out, self.lse, self.acc, self.mass_ws)
            wise.wise_select_step(self.shape, self.acc, self.tau, self.masks[self.filled])
            self.filled += 1
        else:
            wise.wise_dense_attn_accum(self.shape, q, k, v, out, self.lse,
                                       self.acc if accumulate else None,
                                       self.mass_ws if accumulate else None)
        return out

    def dense_step(self, q, k, v, out, lse=None):
        wise.wise_dense_attn_accum(self.shape, q, k, v, out, lse, None)
        return out

    def select(self):
        if self.mode == "union":
            if self.filled == 0:
                raise RuntimeError("union mode: no window step was run before select()")
            self.schedule.from_masks(self.masks, self.filled, self.flags)
        else:
            self.schedule.select(self.acc, self.tau, self.flags)
        if self._auto and not torch.cuda.is_current_stream_capturing():
            if not self._decided:
                self._decide(self.schedule.nnz())
                self._decided = True
            else:
                self._poll()
                self._nnz_host.copy_(self.schedule.row_ptr[-1:], non_blocking=True)
                self._nnz_event = torch.cuda.Event()
                self._nnz_event.record()
        return self.schedule

    def _decide(self, nnz: int):
        self.grouped = nnz / wise.wise_support_capacity(self.shape) >= self.group_density

    def _poll(self):
        """Take up the last asynchronously copied support size if it has landed."""
        if self._nnz_event is not None and self._nnz_event.query():
            self._decide(int(self._nnz_host[0]))
            self._nnz_event = None

    def late_step(self, q, k, v, out, lse=None, ordered=True):
        s = self.schedule
        if self._nnz_event is not None and not torch.cuda.is_current_stream_capturing():
            self._poll()
        if self.grouped:
            wise.wise_sparse_attn_grouped(self.shape, q, k, v, s.row_ptr, s.col_idx, out, lse)
        else:
            wise.wise_sparse_attn(self.shape, q, k, v, s.row_ptr, s.col_idx,
                                  s.row_order if ordered else None, out, lse)
        return out

    def capture_late_step(self, q, k, v, out, lse=None) -> "LateStepGraph":
        """The late step on these fixed buffers as a HIP graph (see LateStepGraph)."""
        return LateStepGraph(self, q, k, v, out, lse)


class LateStepGraph:
    """One late step captured in a HIP graph over fixed q/k/v/out (and lse)
    buffers.  A serving loop writes each step's Q/K/V into those buffers and
    calls replay(): one launch of the recorded sparse kernel, which reads the
    support held in the pipeline's schedule buffers at replay time (so a new
    select() needs no re-capture; the kernel chosen at capture stays, and
    both late-step kernels give the same outputs).  The library allocates and clears nothing,
    so the graph holds only the kernel node."""

    def __init__(self, pipe: WisePipeline, q, k, v, out, lse=None):
        self.buffers = (q, k, v, out, lse)
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):              # warm-up launch outside the capture
            pipe.late_step(q, k, v, out, lse)
        torch.cuda.current_stream().wait_stream(side)
        self.graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(self.graph):
            pipe.late_step(q, k, v, out, lse)

    def replay(self):
        self.graph.replay()
        return self.buffers[3]

