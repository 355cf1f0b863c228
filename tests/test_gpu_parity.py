"""GPU path vs the CPU oracle, through the C ABI.

Scores: |gpu - oracle| <= 2e-2 + 1e-2 |oracle| elementwise, and for every
user every candidate pair whose oracle scores differ by more than 5e-2 keeps
its order.  Cache: the same tolerance elementwise at identical indices, so a
mis-indexed row fails loudly.  Offsets are checked bit-exactly.
"""
import numpy as np
import pytest

import oracle
from synth import make_inputs, make_workload
from tests.gpu_util import (GpuRun, assert_cache_match, assert_order_kept, assert_scores_match,
                            say)

pytestmark = pytest.mark.gpu


def _oracle_full(inp, users=None, cand_rows=None):
    cache = oracle.encode(inp.weights, inp.d, inp.H, inp.L, inp.F, inp.hist_emb,
                          inp.hist_offsets, users=users)
    scores = oracle.rank(inp.weights, inp.d, inp.H, inp.L, inp.F, cache, inp.hist_offsets,
                         inp.cand_emb, inp.cand_offsets, users=users, cand_rows=cand_rows)
    return cache, scores


def _groups(offsets, rows=None):
    out = []
    for u in range(len(offsets) - 1):
        r = np.arange(offsets[u], offsets[u + 1])
        if rows is not None:
            r = r[np.isin(r, rows)]
        out.append(r)
    return out


def _check_all(inp, label, score_scale=1.0):
    say(f"[gpu] {label}: U={inp.U} T={inp.hist_offsets[-1]} Kc={inp.cand_offsets[-1]} "
        f"d={inp.d} H={inp.H} L={inp.L} F={inp.F} {inp.dtype}")
    run = GpuRun(inp)
    run.encode()
    run.rank()
    g_scores, g_cache = run.scores_np(), run.cache_np()
    o_cache, o_scores = _oracle_full(inp)
    rows = np.arange(int(inp.hist_offsets[-1]))
    assert_cache_match(g_cache, o_cache, rows, label)
    err = assert_scores_match(g_scores[: len(o_scores)], o_scores, label, scale=score_scale)
    if score_scale == 1.0:
        assert_order_kept(g_scores, o_scores, _groups(inp.cand_offsets), label)
    say(f"[gpu] {label}: max |score err| {err:.3e}")
    return run, g_scores


SMALL = [
    # (hist lens, cand lens, d, H, L, F, dtype): several tiles, ragged tails,
    # empty users on either side, one-row users
    ([64], [128], 64, 2, 1, 256, "f32"),
    ([0, 1, 63, 65, 130, 300], [1, 129, 0, 257, 64, 3], 128, 2, 2, 256, "bf16"),
    ([200, 0, 17], [300, 40, 1], 64, 2, 2, 128, "f32"),
    ([511, 5, 1000], [7, 513, 250], 256, 4, 1, 512, "bf16"),
    # rows that fill no tile width: q|k|v 1152 and FFN 768 columns, and the
    # fused LayerNorm tile with two of its eight column blocks empty
    ([100, 7, 600], [300, 65, 20], 384, 6, 2, 768, "bf16"),
    # rows wider than the fused residual+LayerNorm tile (512): separate
    # LayerNorm launches
    ([40, 300], [70, 129], 1024, 16, 2, 1024, "bf16"),
]


@pytest.mark.parametrize("case", range(len(SMALL)))
@pytest.mark.parametrize("variant", ["base", "perturbed", "sharp"])
def test_small_shapes_match_oracle(case, variant):
    n, k, d, H, L, F, dt = SMALL[case]
    scale = 1.0
    if variant == "sharp":
        # Query weights x4 multiply the logits, and the logit error of bf16
        # queries and keys, by 4: the tolerance scales by the same factor.
        # One layer exercises the peaked-softmax path without compounding it
        # through depth.
        L = 1
        scale = 4.0 if dt == "bf16" else 1.0
    inp = make_inputs(n, k, d, H, L, F, dtype=dt, seed=100 + case, variant=variant)
    _check_all(inp, f"small{case}/{variant}", score_scale=scale)


@pytest.mark.parametrize("variant", ["perturbed", "sharp"])
def test_exact_redo_path_matches_oracle(variant, monkeypatch):
    """The ranking attention keeps each query's own logit as the softmax
    reference; work items whose sums overflow are redone exactly (maximum
    logit first, then probabilities <= 1).  UPR_ATTN_EXACT=1 sends every
    work item through that redo, which must meet the same bar."""
    monkeypatch.setenv("UPR_ATTN_EXACT", "1")
    n, k, d, H, L, F, dt = SMALL[3]
    scale = 1.0
    if variant == "sharp":
        L, scale = 1, 4.0
    inp = make_inputs(n, k, d, H, L, F, dtype=dt, seed=321, variant=variant)
    _check_all(inp, f"redo/{variant}", score_scale=scale)


@pytest.mark.parametrize("name", ["tiny_f32", "u16_n256_k1000"])
def test_named_workload_full_oracle(name):
    _check_all(make_workload(name, seed=0), name)


@pytest.mark.parametrize("name,n_users,per_user", [
    ("u64_n1024_k2000", 6, 48),
    ("ragged_u64", 6, 48),
    ("u8_n8192_k4096", 1, 64),
])
def test_named_workload_sampled(name, n_users, per_user):
    """Full-size batch on the GPU (the benchmark's launch configuration);
    the oracle recomputes sampled users and candidates one by one."""
    inp = make_workload(name, seed=0)
    say(f"[gpu] {name}: full-size run U={inp.U} T={inp.hist_offsets[-1]} Kc={inp.cand_offsets[-1]}")
    run = GpuRun(inp)
    run.encode()
    run.rank()
    g_scores, g_cache = run.scores_np(), run.cache_np()
    assert np.all(np.isfinite(g_scores[: inp.cand_offsets[-1]]))
    rng = np.random.default_rng(1234)
    ho, co = inp.hist_offsets, inp.cand_offsets
    # heaviest and lightest users plus random ones
    lens = np.diff(ho)
    pick = {int(np.argmax(lens)), int(np.argmin(lens))}
    while len(pick) < min(n_users, inp.U):
        pick.add(int(rng.integers(inp.U)))
    users = sorted(pick)
    rows = []
    for u in users:
        k = co[u + 1] - co[u]
        sel = rng.choice(k, size=min(per_user, k), replace=False)
        rows.extend((co[u] + np.sort(np.concatenate([sel, [0, k - 1]]))).tolist())
    rows = np.unique(np.array(rows, dtype=np.int64))
    say(f"[gpu] {name}: oracle on users {users}, {rows.size} candidates")
    o_cache, o_scores = _oracle_full(inp, users=users, cand_rows=rows)
    hrows = np.concatenate([np.arange(ho[u], ho[u + 1]) for u in users])
    assert_cache_match(g_cache, o_cache, hrows, name)
    err = assert_scores_match(g_scores[rows], o_scores[rows], name)
    assert_order_kept(g_scores, o_scores, _groups(co, rows), name)
    say(f"[gpu] {name}: max |score err| {err:.3e} over {rows.size} sampled candidates")


def test_offsets_are_not_modified():
    inp = make_inputs([40, 0, 70], [33, 5, 0], 128, 2, 1, 256, dtype="bf16", seed=5)
    run = GpuRun(inp)
    run.encode()
    run.rank()
    run.scores_np()
    assert np.array_equal(run.hoff_d.cpu().numpy(), inp.hist_offsets)
    assert np.array_equal(run.coff_d.cpu().numpy(), inp.cand_offsets)
    assert np.array_equal(run.hoff, inp.hist_offsets)
