"""Stream and graph behaviour of the C ABI on the GPU: calls on two streams
with disjoint outputs may run concurrently and give the same bits as in
sequence; the late step and the selection can be captured in a HIP graph
(no allocation, synchronisation or memset inside) and every replay, with
eager work and synchronisations between replays, gives the eager bits."""

import numpy as np
import pytest
import torch

from paper_2609_27373_amd.pipeline import WisePipeline
from paper_2609_27373_amd.workloads import CONFIGS, Trajectory
from parity_util import say

pytestmark = pytest.mark.gpu


def _trajectory_inputs(cfg, steps):
    tr = Trajectory(cfg, device="cuda")
    return [tr.next(torch.bfloat16) for _ in range(steps)]


def test_two_streams_match_sequential(gpu_lib):
    cfg = CONFIGS["tiny"].with_(heads=8, seq_len=2048)
    say(f"two streams: heads {cfg.heads} n {cfg.seq_len}")
    steps = _trajectory_inputs(cfg, cfg.discovery_steps + 2)
    pipe = WisePipeline.for_config(cfg)
    out = torch.empty_like(steps[0][0])
    pipe.reset()
    for t in range(1, cfg.discovery_steps + 1):
        pipe.discovery_step(*steps[t - 1], out, accumulate=t in cfg.window)
    pipe.select()
    a, b = steps[cfg.discovery_steps], steps[cfg.discovery_steps + 1]
    seq = [torch.empty_like(out), torch.empty_like(out)]
    pipe.late_step(*a, seq[0])
    pipe.late_step(*b, seq[1])
    torch.cuda.synchronize()
    par = [torch.empty_like(out), torch.empty_like(out)]
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    s1.wait_stream(torch.cuda.current_stream())
    s2.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s1):
        pipe.late_step(*a, par[0])
    with torch.cuda.stream(s2):
        pipe.late_step(*b, par[1])
    torch.cuda.synchronize()
    assert torch.equal(seq[0], par[0]) and torch.equal(seq[1], par[1])


@pytest.mark.parametrize("late_kernel", ["rows", "grouped"])
def test_graph_replays_match_eager(gpu_lib, late_kernel):
    cfg = CONFIGS["tiny"].with_(heads=4, seq_len=1024)
    say(f"graph capture: heads {cfg.heads} n {cfg.seq_len}, late kernel {late_kernel}")
    steps = _trajectory_inputs(cfg, cfg.discovery_steps + 1)
    pipe = WisePipeline.for_config(cfg, late_kernel=late_kernel)
    out = torch.empty_like(steps[0][0])
    pipe.reset()
    for t in range(1, cfg.discovery_steps + 1):
        pipe.discovery_step(*steps[t - 1], out, accumulate=t in cfg.window)
    torch.cuda.synchronize()
    acc_eager = pipe.acc.clone()
    q, k, v = steps[cfg.discovery_steps]
    # eager reference: selection, then the late step
    pipe.select()
    eager = torch.empty_like(out)
    pipe.late_step(q, k, v, eager)
    torch.cuda.synchronize()
    rp_eager = pipe.schedule.row_ptr.clone()
    # capture selection + late step (side stream, as torch requires)
    graph = torch.cuda.CUDAGraph()
    gout = torch.empty_like(out)
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        pipe.select()
        pipe.late_step(q, k, v, gout)
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    with torch.cuda.graph(graph):
        pipe.select()
        pipe.late_step(q, k, v, gout)
    for rep in range(3):
        gout.zero_()
        pipe.schedule.row_ptr.fill_(-1)
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(pipe.schedule.row_ptr, rp_eager), f"replay {rep}: row_ptr"
        assert torch.equal(gout, eager), f"replay {rep}: late-step output"
        # eager work between replays
        scratch = torch.empty_like(out)
        pipe.late_step(q, k, v, scratch)
        torch.cuda.synchronize()
        assert torch.equal(scratch, eager)
    assert torch.equal(pipe.acc, acc_eager)


@pytest.mark.parametrize("late_kernel", ["rows", "grouped"])
def test_captured_late_step_follows_new_inputs_and_supports(gpu_lib, late_kernel):
    """LateStepGraph: replays after writing new Q/K/V into the captured
    buffers, and after a new selection, give the eager late step's bits."""
    cfg = CONFIGS["tiny"].with_(heads=4, seq_len=1024)
    say(f"late-step graph: heads {cfg.heads} n {cfg.seq_len}, late kernel {late_kernel}")
    steps = _trajectory_inputs(cfg, cfg.discovery_steps + 3)
    pipe = WisePipeline.for_config(cfg, late_kernel=late_kernel)
    out = torch.empty_like(steps[0][0])
    pipe.reset()
    for t in range(1, cfg.discovery_steps + 1):
        pipe.discovery_step(*steps[t - 1], out, accumulate=t in cfg.window)
    pipe.select()
    qb, kb, vb = (torch.empty_like(x) for x in steps[0])
    ob = torch.empty_like(out)
    g = pipe.capture_late_step(qb, kb, vb, ob)
    eager = torch.empty_like(out)
    for rep, (q, k, v) in enumerate(steps[cfg.discovery_steps:]):
        qb.copy_(q); kb.copy_(k); vb.copy_(v)
        ob.zero_()
        g.replay()
        pipe.late_step(q, k, v, eager)
        torch.cuda.synchronize()
        assert torch.equal(ob, eager), f"replay {rep}"
    # a different support (tau lowered): the graph reads the new CSR
    pipe.tau = 0.5
    pipe.select()
    q, k, v = steps[-1]
    qb.copy_(q); kb.copy_(k); vb.copy_(v)
    g.replay()
    pipe.late_step(q, k, v, eager)
    torch.cuda.synchronize()
    assert torch.equal(ob, eager), "replay after a new selection"
