"""GPU-side invariants of the method, through the C ABI.

Candidates never see each other (Sec. 3, attention pattern; KV-cache
section: scores independent of batch composition), so on the GPU:
permuting candidates permutes scores bit-exactly, a single-user call on a
sub-range of the packed buffers reproduces the batched scores bit-exactly,
and repeated runs are bit-identical.  Validation errors leave outputs
untouched.
"""
import ctypes

import numpy as np
import pytest

from paper_2606_00422_amd import upr
from synth import make_inputs, make_workload
from tests.gpu_util import GpuRun, assert_scores_match, say
import oracle

pytestmark = pytest.mark.gpu


def _inp():
    return make_inputs([130, 0, 257, 64], [300, 17, 129, 1], 256, 4, 2, 512, dtype="bf16",
                       seed=21, variant="perturbed")


def test_candidate_permutation_is_bit_exact():
    import torch
    inp = _inp()
    say("[gpu] permutation")
    base = GpuRun(inp)
    base.encode()
    base.rank()
    s0 = base.scores_np()
    rng = np.random.default_rng(0)
    co = inp.cand_offsets
    perm = np.concatenate([co[u] + rng.permutation(co[u + 1] - co[u]) for u in range(inp.U)])
    inp2 = _inp()
    inp2.cand_emb = inp.cand_emb[perm]
    run = GpuRun(inp2)
    run.encode()
    run.rank()
    s1 = run.scores_np()
    assert np.array_equal(s1[: co[-1]], s0[perm])


def test_sub_range_single_user_calls_match_batch_bit_exactly():
    inp = _inp()
    say("[gpu] single-user sub-range calls")
    run = GpuRun(inp)
    run.encode()
    run.rank()
    batch = run.scores_np().copy()
    import torch
    ho, co = inp.hist_offsets, inp.cand_offsets
    for u in range(inp.U):
        run.scores.fill_(float("nan"))
        hoff = np.array([ho[u], ho[u + 1]], np.int32)
        coff = np.array([co[u], co[u + 1]], np.int32)
        run.rank(hoff=hoff, coff=coff)
        s = run.scores_np()
        assert np.array_equal(s[co[u]:co[u + 1]], batch[co[u]:co[u + 1]]), f"user {u}"
        others = np.ones(s.shape[0], bool)
        others[co[u]:co[u + 1]] = False
        assert np.all(np.isnan(s[others])), "rows outside the call were written"


def test_tile_height_does_not_change_scores():
    """A batch large enough that every projection GEMM takes its tall tiles
    (32768+ candidate rows at d = 256) against single-user calls, which take
    the short tiles: each output is the same MFMA chain over K and each
    LayerNorm row the same reduction, so the scores agree bit for bit."""
    U, k = 16, 2100
    inp = make_inputs([64] * U, [k] * U, 256, 4, 2, 1024, dtype="bf16", seed=33, variant="perturbed")
    say(f"[gpu] tall vs short tiles: {U * k} candidate rows, then single users")
    run = GpuRun(inp)
    run.encode()
    run.rank()
    batch = run.scores_np().copy()
    ho, co = inp.hist_offsets, inp.cand_offsets
    for u in [0, 7, U - 1]:
        run.scores.fill_(float("nan"))
        run.rank(hoff=np.array([ho[u], ho[u + 1]], np.int32), coff=np.array([co[u], co[u + 1]], np.int32))
        s = run.scores_np()
        assert np.array_equal(s[co[u]:co[u + 1]], batch[co[u]:co[u + 1]]), f"user {u}"


@pytest.mark.parametrize("model_dtype", ["bf16", "bf16_mxfp8"])
def test_long_history_items_do_not_change_scores(model_dtype):
    """Candidates that see 4,096+ history rows on average take 256-candidate
    attention items (eight waves per workgroup); single users of the same
    batch take 64-candidate items.  Every query's softmax and P.V run over
    the same keys in the same order either way, so the scores agree bit for
    bit (also in the fp8 variant, whose attention writes MXFP8), and for
    bf16 a sample of them agrees with the oracle."""
    hl, k = [4608, 4100, 5000, 4700], 4096
    inp = make_inputs(hl, [k] * len(hl), 512, 8, 1, 2048, dtype="bf16", seed=37, variant="perturbed")
    say(f"[gpu] long-history items ({model_dtype}): {len(hl)} users x {k} candidates, histories {hl}")
    run = GpuRun(inp, model_dtype=model_dtype)
    run.encode()
    run.rank()
    batch = run.scores_np().copy()
    assert np.all(np.isfinite(batch))
    ho, co = inp.hist_offsets, inp.cand_offsets
    for u in [0, 2]:
        run.scores.fill_(float("nan"))
        run.rank(hoff=np.array([ho[u], ho[u + 1]], np.int32), coff=np.array([co[u], co[u + 1]], np.int32))
        s = run.scores_np()
        assert np.array_equal(s[co[u]:co[u + 1]], batch[co[u]:co[u + 1]]), f"user {u}"
    if model_dtype != "bf16":
        return
    # a sample of user 1's candidates against the oracle
    rows = co[1] + np.arange(0, k, 257)
    cache = oracle.encode(inp.weights, inp.d, inp.H, inp.L, inp.F, inp.hist_emb, inp.hist_offsets,
                          users=[1])
    o = oracle.rank(inp.weights, inp.d, inp.H, inp.L, inp.F, cache, inp.hist_offsets, inp.cand_emb,
                    inp.cand_offsets, users=[1], cand_rows=rows)
    err = assert_scores_match(batch[rows], o[rows], "long-history sample")
    say(f"[gpu] long-history items: max |score err| {err:.3e} over {rows.size} sampled candidates")


def test_fused_ffn_matches_unfused_pair_bit_exactly():
    """The headline workload (128,000 candidate rows, 65,536 history rows:
    the fused FFN in rank and encode) against single-user calls (the unfused
    FFN-up / FFN-down pair on short tiles): the hidden values are written in
    the order the fused kernel feeds them to the FFN-down MFMAs and W2 is
    stored in that order, so both paths multiply the same pairs in the same
    order and the scores and caches agree bit for bit."""
    import torch
    inp = make_workload("u64_n1024_k2000", seed=6)
    say(f"[gpu] fused vs unfused FFN: {int(inp.cand_offsets[-1])} candidate rows, then single users")
    run = GpuRun(inp)
    run.encode()
    run.rank()
    batch = run.scores_np().copy()
    cache = run.cache.clone()
    ho, co = inp.hist_offsets, inp.cand_offsets
    for u in [0, 29, inp.U - 1]:
        run.scores.fill_(float("nan"))
        h1, c1 = np.array([ho[u], ho[u + 1]], np.int32), np.array([co[u], co[u + 1]], np.int32)
        run.cache.zero_()
        run.encode(hoff=h1)
        rows = slice(int(ho[u]), int(ho[u + 1]))
        assert torch.equal(run.cache[:, :, :, rows], cache[:, :, :, rows]), f"cache of user {u}"
        run.rank(hoff=h1, coff=c1)
        s = run.scores_np()
        assert np.array_equal(s[co[u]:co[u + 1]], batch[co[u]:co[u + 1]]), f"scores of user {u}"


def test_tile_height_does_not_change_scores_mxfp8():
    """The same for the MXFP8 projection variant on the headline workload
    (128,000 candidate rows: tall tiles in every projection, 64-row tiles for
    the O projection with its fused LN2) against single-user calls (short
    tiles, 64-candidate attention items)."""
    inp = make_workload("u64_n1024_k2000", seed=5)
    say(f"[gpu] mxfp8 tall vs short tiles: {int(inp.cand_offsets[-1])} candidate rows, then single users")
    run = GpuRun(inp, model_dtype="bf16_mxfp8")
    run.encode()
    run.rank()
    batch = run.scores_np().copy()
    assert np.all(np.isfinite(batch))
    ho, co = inp.hist_offsets, inp.cand_offsets
    for u in [0, 37, inp.U - 1]:
        run.scores.fill_(float("nan"))
        run.rank(hoff=np.array([ho[u], ho[u + 1]], np.int32), coff=np.array([co[u], co[u + 1]], np.int32))
        s = run.scores_np()
        assert np.array_equal(s[co[u]:co[u + 1]], batch[co[u]:co[u + 1]]), f"user {u}"


def test_sub_range_encode_matches_batch_encode():
    inp = _inp()
    say("[gpu] per-user encode")
    a = GpuRun(inp)
    a.encode()
    ca = a.cache_np()
    b = GpuRun(inp)
    ho = inp.hist_offsets
    for u in range(inp.U):
        b.encode(hoff=np.array([ho[u], ho[u + 1]], np.int32))
    cb = b.cache_np()
    assert np.array_equal(ca, cb)


def test_repeated_runs_are_bit_identical():
    inp = make_workload("u16_n256_k1000", seed=3)
    say("[gpu] determinism")
    run = GpuRun(inp)
    run.encode()
    c0 = run.cache_np()
    run.rank()
    s0 = run.scores_np().copy()
    for _ in range(2):
        run.encode()
        run.rank()
        assert np.array_equal(run.scores_np(), s0)
        assert np.array_equal(run.cache_np(), c0)


def test_empty_history_user_scores_match_oracle():
    inp = make_inputs([0, 0], [40, 3], 128, 2, 2, 256, dtype="bf16", seed=4, variant="perturbed")
    say("[gpu] empty histories")
    run = GpuRun(inp, capacity_rows=1)
    run.encode()
    run.rank()
    s = run.scores_np()
    cache = np.zeros((2, 2, 2, 1, 64))
    ref = oracle.rank(inp.weights, inp.d, inp.H, inp.L, inp.F, cache, inp.hist_offsets,
                      inp.cand_emb, inp.cand_offsets)
    assert_scores_match(s[:43], ref, "empty histories")


@pytest.mark.parametrize("what", ["decreasing", "capacity", "workspace", "users", "null_scores"])
def test_validation_errors_leave_outputs_untouched(what):
    import torch
    inp = make_inputs([20, 30], [10, 12], 128, 2, 1, 256, dtype="bf16", seed=6)
    run = GpuRun(inp)
    run.encode()
    run.scores.fill_(123.0)
    cache_before = run.cache.clone()
    hs = upr.segments(run.hoff, run.hoff_d)
    cs = upr.segments(run.coff, run.coff_d)
    need = upr.upr_rank_workspace_bytes(run.model.handle, hs, cs)
    ws = torch.empty(need, dtype=torch.uint8, device="cuda")
    kv = upr.upr_kv_cache(run.cache.data_ptr(), run.cap)
    scores_ptr = run.scores.data_ptr()
    ws_bytes = need
    if what == "decreasing":
        bad = np.array([0, 12, 10], np.int32)
        cs = upr.segments(bad, run.coff_d)
        code = upr.UPR_ERR_OFFSETS
    elif what == "capacity":
        kv = upr.upr_kv_cache(run.cache.data_ptr(), 49)
        code = upr.UPR_ERR_CAPACITY
    elif what == "workspace":
        ws_bytes = need - 1
        code = upr.UPR_ERR_WORKSPACE
    elif what == "users":
        one = np.array([0, 22], np.int32)
        cs = upr.segments(one, run.coff_d)
        code = upr.UPR_ERR_OFFSETS
    else:
        scores_ptr = 0
        code = upr.UPR_ERR_NULL
    with pytest.raises(upr.UprError) as ei:
        upr.upr_rank_candidates(run.model.handle, kv, hs, run.C.data_ptr(), cs, scores_ptr,
                                ws.data_ptr(), ws_bytes, upr.current_stream())
    assert ei.value.status == code
    torch.cuda.synchronize()
    assert torch.all(run.scores == 123.0)
    assert torch.equal(run.cache, cache_before)


@pytest.mark.parametrize("d,H,F", [(128, 2, 128), (256, 4, 384), (384, 6, 256)])
def test_fused_tail_other_widths(d, H, F):
    """The fused layer tail at the model widths it takes besides 512 (its
    weight ring is sized per width) and with a single hidden chunk (F = 128):
    36,000 candidate rows make 282 tiles of 128 rows, so the batched call
    runs the fused tail; single-user calls run the unfused pair on short
    tiles and must agree bit for bit, and sampled candidates match the
    oracle."""
    rng = np.random.default_rng(d + F)
    U = 36
    hist = rng.integers(1, 96, size=U).tolist()
    inp = make_inputs(hist, [1000] * U, d, H, 2, F, dtype="bf16", seed=d + F)
    say(f"[gpu] fused tail d={d} H={H} F={F}: {int(inp.cand_offsets[-1])} candidate rows")
    run = GpuRun(inp)
    run.encode()
    upr.upr_profile_enable(True)
    run.rank()
    batch = run.scores_np().copy()
    prof = upr.upr_profile_read()
    upr.upr_profile_enable(False)
    assert "rank.oproj_ffn" in prof, f"the batched call did not run the fused tail: {sorted(prof)}"
    assert np.all(np.isfinite(batch[: inp.cand_offsets[-1]]))
    ho, co = inp.hist_offsets, inp.cand_offsets
    for u in [0, U // 2, U - 1]:
        run.scores.fill_(float("nan"))
        run.rank(hoff=np.array([ho[u], ho[u + 1]], np.int32), coff=np.array([co[u], co[u + 1]], np.int32))
        s = run.scores_np()
        assert np.array_equal(s[co[u]:co[u + 1]], batch[co[u]:co[u + 1]]), f"scores of user {u}"
    users = [0, U - 1]
    rows = np.unique(np.concatenate([co[u] + np.sort(rng.choice(1000, size=40, replace=False))
                                     for u in users]))
    cache = oracle.encode(inp.weights, inp.d, inp.H, inp.L, inp.F, inp.hist_emb, ho, users=users)
    o = oracle.rank(inp.weights, inp.d, inp.H, inp.L, inp.F, cache, ho, inp.cand_emb, co,
                    users=users, cand_rows=rows)
    err = assert_scores_match(batch[rows], o[rows], f"fused tail d={d} F={F}")
    say(f"[gpu] fused tail d={d} F={F}: max |score err| {err:.3e} over {rows.size} candidates")


def test_device_offsets_that_disagree_are_skipped():
    """The device copy of the candidate offsets disagrees with the host array
    (a caller error the contract rules out).  The values are chosen so that
    every access would stay inside the buffers even if they were used as
    given (the device split has more tiles than the host one, and the work
    list holds at most the host count), so the case is safe either way; the
    work list's check must reject them and leave every item empty.  The
    attention then writes nothing, so the scores follow whatever the
    workspace held, while with a consistent device copy they do not depend
    on it."""
    import torch
    inp = make_inputs([50, 30], [300, 0], 256, 4, 1, 512, dtype="bf16", seed=5)
    say("[gpu] device offsets that disagree with the host ones")
    run = GpuRun(inp)
    run.encode()
    stale = torch.from_numpy(np.array([0, 1, 300], np.int32)).to("cuda")
    ws = run.model.rank(run.cache, run.hoff, run.hoff_d, run.C, run.coff, run.coff_d, run.scores)

    def scores_with(fill, cand_dev):
        ws.fill_(fill)
        run.scores.fill_(float("nan"))
        run.model.rank(run.cache, run.hoff, run.hoff_d, run.C, run.coff, cand_dev, run.scores, ws=ws)
        return run.scores_np()[:300].copy()

    good0, good1 = scores_with(0, run.coff_d), scores_with(0x3C, run.coff_d)
    assert np.array_equal(good0, good1), "a consistent call read workspace bytes it did not write"
    bad0, bad1 = scores_with(0, stale), scores_with(0x3C, stale)
    assert np.all(np.isfinite(bad0)) and np.all(np.isfinite(bad1))
    assert not np.array_equal(bad0, bad1), "the attention ran on offsets the check should reject"
