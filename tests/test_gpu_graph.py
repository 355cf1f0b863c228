"""A captured upr_rank_candidates call (HIP graph) replays to the eager
result bit for bit.  The call enqueues only kernel launches on the caller's
stream (no allocation, copy, memset or synchronization), so it can be
captured; each replay is checked after the scores were overwritten, with
eager work and synchronizations between replays."""
import numpy as np
import pytest
import torch

from paper_2606_00422_amd import upr
from synth import make_inputs
from tests.gpu_util import GpuRun, say

pytestmark = pytest.mark.gpu


def test_graph_replay_matches_eager():
    inp = make_inputs([300, 5, 1000, 0], [257, 64, 700, 9], 128, 2, 2, 256, dtype="bf16", seed=11)
    say(f"[gpu] graph replay: U={inp.U} Kc={inp.cand_offsets[-1]}")
    run = GpuRun(inp)
    run.encode()
    hs = upr.segments(run.hoff, run.hoff_d)
    cs = upr.segments(run.coff, run.coff_d)
    ws = run.model.workspace(upr.upr_rank_workspace_bytes(run.model.handle, hs, cs))

    def rank(out):
        run.model.rank(run.cache, run.hoff, run.hoff_d, run.C, run.coff, run.coff_d, out, ws=ws)

    rank(run.scores)
    torch.cuda.synchronize()
    ref = run.scores.clone()
    assert bool(torch.isfinite(ref).all())
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        rank(run.scores)
    other = torch.empty_like(run.scores)
    for rep in range(3):
        run.scores.fill_(float("nan"))
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(run.scores, ref), f"replay {rep} differs from the eager call"
        other.fill_(0.0)
        rank(other)                       # eager work between replays
        torch.cuda.synchronize()
        assert torch.equal(other, ref)
    del g
