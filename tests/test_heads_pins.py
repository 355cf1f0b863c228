"""Pins of the per-action heads and utility top-K oracle (CPU only).

Each pin checks the oracle against something other than its own code:
torch's Linear / GELU(tanh) / Linear stack in float64 as the textbook MLP,
closed forms for zero weights, sigmoid identities, hand-worked top-K cases
with ties and NaNs, and an independent ordering (numpy lexsort) on random
cases.
"""
import math

import numpy as np
import pytest
import torch

import oracle
import oracle.upr_heads as heads_oracle
from synth import make_heads, make_inputs


def _final_and_hidden(d=48, rows=37, seed=3):
    inp = make_inputs([5], [rows], d=d, H=4, L=1, F=96, dtype="f32", seed=seed, variant="perturbed")
    _, final = oracle.unpack_weights(inp.weights, d, 1, 96)
    rng = np.random.default_rng(seed)
    hidden = rng.normal(size=(rows, d)) * 2.0 + 0.3
    return final, hidden


@pytest.mark.parametrize("variant", ["base", "perturbed"])
def test_action_logits_match_torch_mlp(variant):
    d, C, Fh = 48, 3, 20
    final, hidden = _final_and_hidden(d)
    blob = make_heads(d, C, Fh, dtype="f32", seed=5, variant=variant)
    got = heads_oracle.action_logits(hidden, final, blob, d, C, Fh)
    z = torch.nn.functional.layer_norm(torch.tensor(hidden, dtype=torch.float64), (d,),
                                       torch.tensor(final["lnf_g"]), torch.tensor(final["lnf_b"]),
                                       eps=1e-5)
    pos = 0
    b = torch.tensor(np.asarray(blob, dtype=np.float64))
    for c in range(C):
        mlp = torch.nn.Sequential(torch.nn.Linear(d, Fh), torch.nn.GELU(approximate="tanh"),
                                  torch.nn.Linear(Fh, 1)).double()
        with torch.no_grad():
            mlp[0].weight.copy_(b[pos:pos + Fh * d].reshape(Fh, d)); pos += Fh * d
            mlp[0].bias.copy_(b[pos:pos + Fh]); pos += Fh
            mlp[2].weight.copy_(b[pos:pos + Fh].reshape(1, Fh)); pos += Fh
            mlp[2].bias.copy_(b[pos:pos + 1]); pos += 1
            ref = mlp(z)[:, 0].numpy()
        np.testing.assert_allclose(got[:, c], ref, rtol=1e-12, atol=1e-12)
    assert pos == blob.size


def test_zero_first_layer_gives_constant_logits():
    d, C, Fh = 32, 2, 8
    final, hidden = _final_and_hidden(d, rows=9)
    blob = make_heads(d, C, Fh, dtype="f32", seed=2, variant="perturbed").astype(np.float64)
    per = Fh * d + 2 * Fh + 1
    expect = []
    for c in range(C):
        blob[c * per: c * per + Fh * d] = 0.0
        b1 = blob[c * per + Fh * d: c * per + Fh * d + Fh]
        w2 = blob[c * per + Fh * d + Fh: c * per + Fh * d + 2 * Fh]
        b2 = blob[c * per + Fh * d + 2 * Fh]
        # GELU(tanh) of each bias, written out from its definition
        g = np.array([0.5 * x * (1 + math.tanh(math.sqrt(2 / math.pi) * (x + 0.044715 * x ** 3))) for x in b1])
        expect.append(float(g @ w2 + b2))
    got = heads_oracle.action_logits(hidden, final, blob, d, C, Fh)
    for c in range(C):
        np.testing.assert_allclose(got[:, c], expect[c], rtol=0, atol=1e-12)


def test_sigmoid_identities():
    x = np.array([-1000.0, -30.0, -2.5, -1e-3, 0.0, 1e-3, 2.5, 30.0, 1000.0])
    p = heads_oracle.sigmoid(x)
    assert np.all(np.isfinite(p)) and p[4] == 0.5
    np.testing.assert_allclose(p + heads_oracle.sigmoid(-x), 1.0, rtol=0, atol=1e-15)
    mid = np.abs(x) < 50
    np.testing.assert_allclose(p[mid], 1.0 / (1.0 + np.exp(-x[mid])), rtol=1e-14)
    assert p[0] == 0.0 or p[0] < 1e-300
    assert p[-1] == 1.0


def test_utility_is_the_weighted_sum():
    probs = np.array([[0.1, 0.2, 0.3], [1.0, 0.0, 0.5]])
    np.testing.assert_allclose(heads_oracle.utility(probs, [1.0, 0.5, -2.0]),
                               [0.1 + 0.1 - 0.6, 1.0 + 0.0 - 1.0], rtol=0, atol=1e-15)


def test_topk_hand_worked_with_ties_and_nan():
    # user 0: rows 0..5, user 1: rows 6..7, user 2: empty
    util = np.array([0.5, 0.7, 0.5, np.nan, 0.7, -1.0, 2.0, 2.0])
    rows, vals = heads_oracle.topk_by_utility(util, [0, 6, 8, 8], K=4)
    assert rows[0].tolist() == [1, 4, 0, 2]        # 0.7 (row 1 before 4), then 0.5 (0 before 2)
    assert rows[1].tolist() == [6, 7, -1, -1]      # tie: lower row first; padding
    assert rows[2].tolist() == [-1, -1, -1, -1]
    np.testing.assert_array_equal(vals[0], [0.7, 0.7, 0.5, 0.5])
    assert np.isnan(vals[1, 2:]).all()
    rows, _ = heads_oracle.topk_by_utility(util, [0, 6, 8, 8], K=6)
    assert rows[0].tolist() == [1, 4, 0, 2, 5, 3]  # NaN after every number


def test_topk_matches_lexsort_on_random_cases():
    rng = np.random.default_rng(11)
    for trial in range(20):
        U = int(rng.integers(1, 6))
        lens = rng.integers(0, 40, size=U)
        offs = np.concatenate([[0], np.cumsum(lens)])
        util = rng.integers(-3, 4, size=offs[-1]).astype(np.float64) / 2.0   # many ties
        util[rng.random(offs[-1]) < 0.05] = np.nan
        K = int(rng.integers(1, 30))
        rows, vals = heads_oracle.topk_by_utility(util, offs, K)
        for u in range(U):
            r = np.arange(offs[u], offs[u + 1])
            v = util[r]
            key_nan = np.isnan(v).astype(np.int64)
            key_val = np.where(np.isnan(v), 0.0, -v)
            order = np.lexsort((r, key_val, key_nan))      # last key is primary
            want = r[order][:K]
            assert rows[u, :want.size].tolist() == want.tolist()
            assert (rows[u, want.size:] == -1).all()


def test_heads_blob_size_and_layout():
    d, C, Fh = 40, 4, 12
    blob = make_heads(d, C, Fh, dtype="f32", seed=1)
    assert blob.size == heads_oracle.heads_blob_size(d, C, Fh)
    hs = heads_oracle.unpack_heads(blob, d, C, Fh)
    per = Fh * d + 2 * Fh + 1
    assert len(hs) == C
    np.testing.assert_array_equal(hs[2]["W1"].reshape(-1), blob[2 * per: 2 * per + Fh * d])
    assert hs[3]["b2"] == blob[4 * per - 1]
    with pytest.raises(ValueError):
        heads_oracle.unpack_heads(blob[:-1], d, C, Fh)


def test_rank_hidden_feeds_the_score_head():
    """rank() is score_head(rank_hidden()): the heads see the same hidden
    states the single score uses."""
    inp = make_inputs([7, 0], [5, 3], d=32, H=2, L=2, F=64, dtype="f32", seed=4, variant="perturbed")
    cache = oracle.encode(inp.weights, inp.d, inp.H, inp.L, inp.F, inp.hist_emb, inp.hist_offsets)
    args = (inp.weights, inp.d, inp.H, inp.L, inp.F, cache, inp.hist_offsets, inp.cand_emb, inp.cand_offsets)
    hid = oracle.rank_hidden(*args)
    _, final = oracle.unpack_weights(inp.weights, inp.d, inp.L, inp.F)
    np.testing.assert_allclose(oracle.rank(*args), oracle.score_head(hid, final), rtol=0, atol=0)
    # and full_sequence's scores (the plain definition) agree
    for u in range(inp.U):
        h0, h1 = inp.hist_offsets[u], inp.hist_offsets[u + 1]
        c0, c1 = inp.cand_offsets[u], inp.cand_offsets[u + 1]
        s, _ = oracle.full_sequence(inp.weights, inp.d, inp.H, inp.L, inp.F,
                                    inp.hist_emb[h0:h1], inp.cand_emb[c0:c1])
        np.testing.assert_allclose(oracle.score_head(hid[c0:c1], final), s, rtol=1e-10, atol=1e-10)
