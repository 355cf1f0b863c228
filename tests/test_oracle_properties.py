"""Property tests of the oracle over random small shapes and values
(hypothesis, derandomized so every run draws the same examples).

Each property is one the paper fixes (Sec. 3): the cached path equals the
plain masked forward over [history || candidates]; candidates never see one
another (a candidate's score does not depend on which other candidates share
the call, and permuting them permutes the scores); the history cache is
causal (changing history position t leaves positions before t unchanged at
every layer) and does not depend on the candidates.
"""
import numpy as np
from hypothesis import HealthCheck, given, settings
from hypothesis import strategies as st

import oracle
from synth import make_inputs

SETTINGS = settings(max_examples=25, deadline=None, derandomize=True,
                    suppress_health_check=[HealthCheck.too_slow])


@st.composite
def problems(draw):
    U = draw(st.integers(1, 3))
    hist = draw(st.lists(st.integers(0, 12), min_size=U, max_size=U))
    cand = draw(st.lists(st.integers(0, 6), min_size=U, max_size=U))
    H = draw(st.sampled_from([1, 2, 4]))
    D = draw(st.sampled_from([4, 8]))
    L = draw(st.integers(1, 3))
    F = draw(st.sampled_from([8, 16, 32]))
    variant = draw(st.sampled_from(["base", "perturbed", "sharp"]))
    seed = draw(st.integers(0, 2 ** 16))
    return make_inputs(hist, cand, d=H * D, H=H, L=L, F=F, dtype="f32", seed=seed, variant=variant)


def _encode(inp, X=None):
    return oracle.encode(inp.weights, inp.d, inp.H, inp.L, inp.F,
                         inp.hist_emb if X is None else X, inp.hist_offsets)


def _rank(inp, cache, C=None, coff=None):
    return oracle.rank(inp.weights, inp.d, inp.H, inp.L, inp.F, cache, inp.hist_offsets,
                       inp.cand_emb if C is None else C, inp.cand_offsets if coff is None else coff)


@SETTINGS
@given(problems())
def test_cached_path_equals_full_sequence(inp):
    cache = _encode(inp)
    scores = _rank(inp, cache)
    ho, co = inp.hist_offsets, inp.cand_offsets
    for u in range(inp.U):
        ref, kv = oracle.full_sequence(inp.weights, inp.d, inp.H, inp.L, inp.F,
                                       inp.hist_emb[ho[u]:ho[u + 1]], inp.cand_emb[co[u]:co[u + 1]])
        np.testing.assert_allclose(scores[co[u]:co[u + 1]], ref, rtol=1e-10, atol=1e-10)
        for l, (K, V) in enumerate(kv):
            np.testing.assert_allclose(cache[l, 0, :, ho[u]:ho[u + 1], :], K, rtol=1e-10, atol=1e-10)
            np.testing.assert_allclose(cache[l, 1, :, ho[u]:ho[u + 1], :], V, rtol=1e-10, atol=1e-10)


@SETTINGS
@given(problems(), st.integers(0, 2 ** 16))
def test_candidates_are_independent(inp, seed):
    cache = _encode(inp)
    base = _rank(inp, cache)
    rng = np.random.default_rng(seed)
    co = inp.cand_offsets
    perm = np.concatenate([co[u] + rng.permutation(co[u + 1] - co[u]) for u in range(inp.U)]).astype(np.int64)
    np.testing.assert_allclose(_rank(inp, cache, C=inp.cand_emb[perm]), base[perm], rtol=1e-12, atol=1e-12)
    # every candidate alone in its user's list scores what it scored in the batch
    for u in range(inp.U):
        for c in range(co[u], co[u + 1]):
            coff = np.full(inp.U + 1, 0, np.int32)
            coff[u + 1:] = 1
            alone = _rank(inp, cache, C=inp.cand_emb[c:c + 1], coff=coff)
            np.testing.assert_allclose(alone[0], base[c], rtol=1e-12, atol=1e-12)


@SETTINGS
@given(problems(), st.data())
def test_cache_is_causal(inp, data):
    ho = inp.hist_offsets
    users = [u for u in range(inp.U) if ho[u + 1] > ho[u]]
    if not users:
        return
    u = data.draw(st.sampled_from(users))
    t = data.draw(st.integers(0, int(ho[u + 1] - ho[u]) - 1))
    c0 = _encode(inp)
    X = inp.hist_emb.copy()
    X[ho[u] + t] += np.random.default_rng(t).standard_normal(inp.d).astype(np.float32)
    c1 = _encode(inp, X)
    keep = np.ones(c0.shape[3], bool)
    keep[ho[u] + t:ho[u + 1]] = False
    np.testing.assert_allclose(c1[:, :, :, keep, :], c0[:, :, :, keep, :], rtol=1e-13, atol=1e-13)
    assert np.abs(c1[0, :, :, ho[u] + t, :] - c0[0, :, :, ho[u] + t, :]).max() > 0
