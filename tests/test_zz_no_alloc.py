"""upr_rank_candidates_noalloc (the entry point for callers that cannot
allocate) against upr_rank_candidates on the same inputs, through the C ABI.

Both run the same kernels with the same launch plan, so the scores must agree
bit for bit; two calls in a row, the second on a smaller input (one user, a
sub-range of the packed buffers), show that the shared scratch array carries
nothing from one call into the next.  A call whose workspace exceeds the
scratch array fails with UPR_ERR_LIMIT and writes nothing.
"""
import numpy as np
import pytest
import torch

from paper_2606_00422_amd import upr
from synth import make_inputs
from tests.gpu_util import GpuRun, assert_scores_match, say

pytestmark = pytest.mark.gpu


def _noalloc(run, hoff, coff, out):
    hd = torch.from_numpy(hoff).cuda()
    cd = torch.from_numpy(coff).cuda()
    kv = upr.upr_kv_cache(run.cache.data_ptr(), run.cache.shape[3])
    upr.upr_rank_candidates_noalloc(run.model.handle, kv, upr.segments(hoff, hd), run.C.data_ptr(),
                                    upr.segments(coff, cd), out.data_ptr(), upr.current_stream())
    torch.cuda.synchronize()
    return out


def test_noalloc_matches_workspace_entry_point():
    # headline model shape; 3,500 candidate rows (about 39 MB of workspace)
    inp = make_inputs([1024, 700], [2000, 1500], 512, 8, 4, 2048, dtype="bf16", seed=77,
                      variant="perturbed")
    say(f"[gpu] noalloc: U={inp.U} Kc={inp.cand_offsets[-1]} d={inp.d} L={inp.L}")
    run = GpuRun(inp)
    run.encode()
    ref = run.rank().clone()
    torch.cuda.synchronize()
    hoff, coff = run.hoff, run.coff
    rows = int(coff[-1])
    out = torch.full_like(run.scores, float("nan"))
    # first call: both users
    _noalloc(run, hoff, coff, out)
    assert torch.equal(out[:rows], ref[:rows]), "no-alloc scores differ from the workspace call"
    # second call, smaller: user 1 alone (offsets[0] > 0), other rows untouched
    out2 = torch.full_like(run.scores, float("nan"))
    h1, c1 = np.ascontiguousarray(hoff[1:3]), np.ascontiguousarray(coff[1:3])
    _noalloc(run, h1, c1, out2)
    sl = slice(int(coff[1]), int(coff[2]))
    ref1 = torch.full_like(run.scores, float("nan"))
    run.rank(h1, c1, ref1)
    torch.cuda.synchronize()
    assert torch.equal(out2[sl], ref1[sl]), "second (smaller) no-alloc call differs"
    assert torch.isnan(out2[: int(coff[1])]).all(), "rows outside the call were written"
    # a user's scores from the one-user call equal the batched ones (same kernels)
    assert torch.equal(out2[sl], ref[sl])
    g = out[:rows].cpu().numpy().astype(np.float64)
    assert_scores_match(g, ref[:rows].cpu().numpy().astype(np.float64), "noalloc vs workspace")
    say(f"[gpu] noalloc: {rows} + {sl.stop - sl.start} scores bit-identical")


def test_noalloc_rejects_oversized_calls():
    # 8,000 rows of the headline shape need ~90 MB of workspace (> 64 MiB)
    inp = make_inputs([16], [8000], 512, 8, 1, 2048, dtype="bf16", seed=78)
    run = GpuRun(inp)
    hd = torch.from_numpy(run.hoff).cuda()
    cd = torch.from_numpy(run.coff).cuda()
    need = upr.upr_rank_workspace_bytes(run.model.handle, upr.segments(run.hoff, hd),
                                        upr.segments(run.coff, cd))
    assert need > upr.UPR_NOALLOC_SCRATCH_BYTES
    out = torch.full_like(run.scores, float("nan"))
    with pytest.raises(upr.UprError) as ei:
        _noalloc(run, run.hoff, run.coff, out)
    assert ei.value.status == upr.UPR_ERR_LIMIT
    assert torch.isnan(out).all(), "a rejected call wrote scores"
