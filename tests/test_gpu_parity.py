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
@pytest.mark.parametrize("variant", ["base", "perturbed"])
def test_small_shapes_match_oracle(case, variant):
    n, k, d, H, L, F, dt = SMALL[case]
    inp = make_inputs(n, k, d, H, L, F, dtype=dt, seed=100 + case, variant=variant)
    _check_all(inp, f"small{case}/{variant}")


@pytest.mark.parametrize("case", range(len(SMALL)))
def test_sharp_logits_regression_guard(case):
    """Regression guard, not the parity bar: query weights x4 multiply the
    logits, and with them the logit error of the bf16 queries and cached
    keys, by 4; one layer at 4x the score bound catches gross mistakes on the
    peaked-softmax path.  The stated bound at depth is the next test."""
    n, k, d, H, L, F, dt = SMALL[case]
    inp = make_inputs(n, k, d, H, 1, F, dtype=dt, seed=100 + case, variant="sharp")
    _check_all(inp, f"small{case}/sharp-guard", score_scale=4.0 if dt == "bf16" else 1.0)


def _sharp_run(case, L):
    n, k, d, H, _, F, dt = SMALL[case]
    inp = make_inputs(n, k, d, H, L, F, dtype=dt, seed=700 + 10 * case + L, variant="sharp")
    say(f"[gpu] sharp L={L} case {case}")
    run = GpuRun(inp)
    run.encode()
    run.rank()
    return inp, run.scores_np()[: int(inp.cand_offsets[-1])], run.cache_np()


def _worst_ratio(g, o):
    return float(np.max(np.abs(g - o) / (2e-2 + 1e-2 * np.abs(o))))


# Query weights x4 make every layer's logits ~4x sharper, and a peaked
# softmax turns small logit errors into large probability errors.  The K/V
# cache is bf16 by definition of the path; rounding the oracle's own cache to
# bf16 and changing nothing else already puts these cases at 1.05-1.28x the
# stated bound at two layers and 1.6-1.9x at four (1.18x for case 1 even at
# one layer), so no bf16-cache implementation meets the bound here.  Measured
# on the GPU (all of its rounding points, encode included): 2.2-2.6x at two
# layers, 3.0-4.7x at four.
SHARP_XFAIL = pytest.mark.xfail(
    strict=True, reason="sharp logits at depth: the bf16 K/V cache alone exceeds the stated "
                        "bound (CPU emulation 1.05-1.87x); GPU measured 2.2-4.7x")


@SHARP_XFAIL
@pytest.mark.parametrize("L", [2, 4])
@pytest.mark.parametrize("case", [1, 3])
def test_sharp_logits_stated_bound(case, L):
    """The sharp stress variant (query weights x4) at depth under the stated,
    unscaled score bound and the ordering rule; prints the worst ratio of
    error to bound.  Known to exceed it (see SHARP_XFAIL)."""
    inp, g, _ = _sharp_run(case, L)
    _, o = _oracle_full(inp)
    say(f"[gpu] sharp L={L} case {case}: worst |err| / bound = {_worst_ratio(g, o):.3f}")
    assert_scores_match(g, o, f"sharp L={L} case {case}")
    assert_order_kept(g, o, _groups(inp.cand_offsets), f"sharp L={L} case {case}")


@pytest.mark.parametrize("L", [2, 4])
@pytest.mark.parametrize("case", [1, 3])
def test_sharp_logits_rank_on_gpu_cache(case, L):
    """Split check of the sharp variant: the oracle ranks on the GPU's own
    cache, so only the ranking pass's rounding is measured.  Prints the worst
    ratio to the stated bound; held to 2x it (the ranking pass adds bf16
    queries, keys and probabilities on top of the cache's own rounding)."""
    inp, g, gc = _sharp_run(case, L)
    o = oracle.rank(inp.weights, inp.d, inp.H, inp.L, inp.F, gc, inp.hist_offsets, inp.cand_emb,
                    inp.cand_offsets)
    ratio = _worst_ratio(g, o)
    say(f"[gpu] sharp L={L} case {case} on the GPU cache: worst |err| / bound = {ratio:.3f}")
    assert_scores_match(g, o, f"sharp L={L} case {case} on GPU cache", scale=2.0)


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
        L, scale = 1, 4.0       # the regression-guard setting of the sharp variant
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


@pytest.mark.parametrize("name,n_users,per_user", [
    ("u64_n1024_k2000", 4, 48),
    ("ragged_u64", 4, 48),
    ("u8_n8192_k4096", 1, 64),
])
def test_rank_on_gpu_cache(name, n_users, per_user):
    """Split check: the oracle's rank runs on the GPU's own cache (bf16,
    widened), so the comparison measures the ranking pass alone, without the
    encode pass's error; same score bound and ordering rule."""
    inp = make_workload(name, seed=0)
    say(f"[gpu] split check {name}: U={inp.U} Kc={inp.cand_offsets[-1]}")
    run = GpuRun(inp)
    run.encode()
    run.rank()
    g_scores, g_cache = run.scores_np(), run.cache_np()
    rng = np.random.default_rng(4321)
    co = inp.cand_offsets
    lens = np.diff(inp.hist_offsets)
    pick = {int(np.argmax(lens)), int(np.argmin(lens))}
    while len(pick) < min(n_users, inp.U):
        pick.add(int(rng.integers(inp.U)))
    users = sorted(pick)
    rows = np.unique(np.concatenate([
        co[u] + np.sort(rng.choice(co[u + 1] - co[u], size=min(per_user, co[u + 1] - co[u]),
                                   replace=False)) for u in users]))
    o = oracle.rank(inp.weights, inp.d, inp.H, inp.L, inp.F, g_cache, inp.hist_offsets,
                    inp.cand_emb, inp.cand_offsets, users=users, cand_rows=rows)
    err = assert_scores_match(g_scores[rows], o[rows], f"{name} on GPU cache")
    assert_order_kept(g_scores, o, _groups(co, rows), f"{name} on GPU cache")
    say(f"[gpu] split check {name}: max |score err| {err:.3e} over {rows.size} candidates")


def test_worklist_index_order_many_users():
    """More users than the work list sorts (2,048): items go in user index
    order.  2,100 small users, empty ones included; every score against the
    oracle."""
    rng = np.random.default_rng(2100)
    U = 2100
    n = rng.integers(0, 9, U)
    k = rng.integers(0, 4, U)
    n[:3], k[:3] = 0, [0, 1, 2]
    inp = make_inputs(n.tolist(), k.tolist(), 128, 2, 2, 256, dtype="bf16", seed=2100,
                      variant="perturbed")
    _check_all(inp, "2100 users")


def test_fp16_range_overflow_gives_nonfinite_scores():
    """Projection operands of bf16 models are fp16 (|x| < 65504, documented,
    not checked).  LayerNorm gains of 1e5 push the LN2 output past that range:
    the affected rows' scores must come out non-finite, never silently
    finite (the float64 oracle gives finite scores here)."""
    from synth import blob_layout
    inp = make_inputs([40, 70], [33, 50], 128, 2, 1, 256, dtype="bf16", seed=9)
    w = inp.weights.copy()
    pos = 0
    for name, shape, _ in blob_layout(inp.d, inp.L, inp.F):
        size = int(np.prod(shape))
        if name.endswith("ln2_g"):
            w[pos:pos + size] = 1e5
        pos += size
    inp.weights = w
    run = GpuRun(inp)
    run.encode()
    run.rank()
    g = run.scores_np()[: int(inp.cand_offsets[-1])]
    assert not np.any(np.isfinite(g)), f"{np.sum(np.isfinite(g))} finite scores past the fp16 range"
    _, o = _oracle_full(inp)
    assert np.all(np.isfinite(o))


def test_offsets_are_not_modified():
    inp = make_inputs([40, 0, 70], [33, 5, 0], 128, 2, 1, 256, dtype="bf16", seed=5)
    run = GpuRun(inp)
    run.encode()
    run.rank()
    run.scores_np()
    assert np.array_equal(run.hoff_d.cpu().numpy(), inp.hist_offsets)
    assert np.array_equal(run.coff_d.cpu().numpy(), inp.cand_offsets)
    assert np.array_equal(run.hoff, inp.hist_offsets)
