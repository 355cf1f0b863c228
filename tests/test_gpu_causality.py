"""Cache causality and candidate independence on the GPU, through the C ABI
(paper Eq. 2: history position i attends to positions <= i only; Sec. 3,
KV-cache sharing: the history keys and values a later stage reads do not
depend on the candidates).

* Changing history token t of one user leaves every cache row of that user
  before t, and every row of the other users, bit-identical at every layer
  and in both planes; row t itself changes.
* Ranking reads the cache and never writes it, whatever the candidates.
* A GPU subset of the oracle's property tests: random small shapes drawn by
  hypothesis (derandomized), scores under the stated bound.
"""
import numpy as np
import pytest
from hypothesis import HealthCheck, given, settings
from hypothesis import strategies as st

import oracle
from synth import make_inputs, round_bf16
from tests.gpu_util import GpuRun, assert_order_kept, assert_scores_match, say

pytestmark = pytest.mark.gpu


def _inp():
    return make_inputs([300, 77, 513, 0], [40, 9, 130, 5], 256, 4, 3, 512, dtype="bf16", seed=31,
                       variant="perturbed")


@pytest.mark.parametrize("u,t", [(0, 0), (0, 150), (0, 299), (1, 76), (2, 257), (2, 511)])
def test_history_change_leaves_earlier_rows_bit_identical(u, t):
    inp = _inp()
    say(f"[gpu] causality: user {u} position {t}")
    base = GpuRun(inp)
    base.encode()
    c0 = base.cache_np()
    ho = inp.hist_offsets
    row = int(ho[u]) + t
    inp2 = _inp()
    bump = np.random.default_rng(row).standard_normal(inp.d) / np.sqrt(inp.d)
    inp2.hist_emb = inp.hist_emb.copy()
    inp2.hist_emb[row] = round_bf16((inp.hist_emb[row] + bump).astype(np.float32))
    assert not np.array_equal(inp2.hist_emb[row], inp.hist_emb[row])
    run = GpuRun(inp2)
    run.encode()
    c1 = run.cache_np()
    keep = np.ones(c0.shape[3], bool)
    keep[row:int(ho[u + 1])] = False
    assert np.array_equal(c1[:, :, :, keep, :], c0[:, :, :, keep, :])
    assert not np.array_equal(c1[0, :, :, row, :], c0[0, :, :, row, :])


def test_ranking_never_writes_the_cache():
    import torch
    inp = _inp()
    say("[gpu] ranking leaves the cache untouched")
    run = GpuRun(inp)
    run.encode()
    torch.cuda.synchronize()
    c0 = run.cache.clone()
    run.rank()
    torch.cuda.synchronize()
    assert torch.equal(run.cache, c0)
    run.C = (run.C.float() * -3.0 + 0.5).to(run.C.dtype)
    run.rank()
    torch.cuda.synchronize()
    assert torch.equal(run.cache, c0)


@st.composite
def gpu_problems(draw):
    U = draw(st.integers(1, 3))
    hist = draw(st.lists(st.integers(0, 400), min_size=U, max_size=U))
    cand = draw(st.lists(st.integers(0, 200), min_size=U, max_size=U))
    H = draw(st.sampled_from([2, 4, 8]))
    L = draw(st.integers(1, 2))
    F = draw(st.sampled_from([256, 512]))
    variant = draw(st.sampled_from(["base", "perturbed"]))
    seed = draw(st.integers(0, 2 ** 16))
    return make_inputs(hist, cand, d=64 * H, H=H, L=L, F=F, dtype="bf16", seed=seed, variant=variant)


@settings(max_examples=8, deadline=None, derandomize=True,
          suppress_health_check=[HealthCheck.too_slow, HealthCheck.data_too_large])
@given(gpu_problems())
def test_random_shapes_match_oracle(inp):
    say(f"[gpu] property: hist {np.diff(inp.hist_offsets).tolist()} cand "
        f"{np.diff(inp.cand_offsets).tolist()} d={inp.d} L={inp.L} F={inp.F}")
    run = GpuRun(inp)
    run.encode()
    run.rank()
    g = run.scores_np()
    cache = oracle.encode(inp.weights, inp.d, inp.H, inp.L, inp.F, inp.hist_emb, inp.hist_offsets)
    ref = oracle.rank(inp.weights, inp.d, inp.H, inp.L, inp.F, cache, inp.hist_offsets,
                      inp.cand_emb, inp.cand_offsets)
    n = len(ref)
    assert_scores_match(g[:n], ref, "property")
    co = inp.cand_offsets
    assert_order_kept(g[:n], ref, [np.arange(co[u], co[u + 1]) for u in range(inp.U)], "property")
