"""Pins of the CPU oracle against things other than itself.

* brute force: the cached path (encode + rank) equals one masked forward over
  [history || candidates] (the paper's definition, Sec. 3);
* textbook routines: torch's TransformerEncoderLayer (pre-LN) and
  scaled_dot_product_attention on the CPU, in float64, with the boolean mask;
* closed forms: one key returns V, zero query weights give the mean of the
  allowed values, an empty history reduces a layer to a per-token MLP;
* invariants: candidate and user permutations, batch composition,
  causality of the cache.
"""
import math

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle
from synth import make_inputs, round_bf16

torch.set_default_dtype(torch.float64)


def _full_vs_cached(inp):
    cache = oracle.encode(inp.weights, inp.d, inp.H, inp.L, inp.F, inp.hist_emb, inp.hist_offsets)
    scores = oracle.rank(inp.weights, inp.d, inp.H, inp.L, inp.F, cache, inp.hist_offsets,
                         inp.cand_emb, inp.cand_offsets)
    ho, co = inp.hist_offsets, inp.cand_offsets
    for u in range(inp.U):
        X = inp.hist_emb[ho[u]:ho[u + 1]]
        C = inp.cand_emb[co[u]:co[u + 1]]
        ref, kv = oracle.full_sequence(inp.weights, inp.d, inp.H, inp.L, inp.F, X, C)
        np.testing.assert_allclose(scores[co[u]:co[u + 1]], ref, rtol=1e-10, atol=1e-10)
        for l, (K, V) in enumerate(kv):
            np.testing.assert_allclose(cache[l, 0, :, ho[u]:ho[u + 1], :], K, rtol=1e-10, atol=1e-10)
            np.testing.assert_allclose(cache[l, 1, :, ho[u]:ho[u + 1], :], V, rtol=1e-10, atol=1e-10)
    return cache, scores


@pytest.mark.parametrize("variant", ["base", "perturbed", "sharp"])
def test_cached_equals_full_sequence(variant):
    inp = make_inputs([7, 0, 19, 1], [5, 3, 0, 9], d=32, H=4, L=3, F=64,
                      dtype="f32", seed=3, variant=variant)
    _full_vs_cached(inp)


def test_cached_equals_full_sequence_bf16_inputs():
    inp = make_inputs([33, 12], [17, 40], d=64, H=2, L=2, F=128, dtype="bf16", seed=11,
                      variant="perturbed")
    assert np.array_equal(inp.weights, round_bf16(inp.weights))
    _full_vs_cached(inp)


# ---------------------------------------------------------------------------
# Library cross-check: torch's pre-LN encoder layer with the same mask
# ---------------------------------------------------------------------------

def _torch_scores(inp, u, use_sdpa=False):
    d, H, L, Fd = inp.d, inp.H, inp.L, inp.F
    blob = torch.tensor(inp.weights, dtype=torch.float64)
    ho, co = inp.hist_offsets, inp.cand_offsets
    X = torch.tensor(inp.hist_emb[ho[u]:ho[u + 1]], dtype=torch.float64)
    C = torch.tensor(inp.cand_emb[co[u]:co[u + 1]], dtype=torch.float64)
    n, k = X.shape[0], C.shape[0]
    z = torch.cat([X, C], 0)[None]                    # [1, n+k, d]
    # allowed[i, j]: history rows causal (diagonal included), candidate rows
    # see all history and themselves.  Built here independently of the oracle.
    allowed = torch.zeros(n + k, n + k, dtype=torch.bool)
    for i in range(n + k):
        if i < n:
            allowed[i, :i + 1] = True
        else:
            allowed[i, :n] = True
            allowed[i, i] = True
    pos = 0

    def take(*shape):
        nonlocal pos
        size = int(np.prod(shape))
        t = blob[pos:pos + size].reshape(shape)
        pos += size
        return t

    for _ in range(L):
        layer = torch.nn.TransformerEncoderLayer(
            d_model=d, nhead=H, dim_feedforward=Fd, dropout=0.0,
            activation=lambda x: F.gelu(x, approximate="tanh"),
            layer_norm_eps=1e-5, batch_first=True, norm_first=True, dtype=torch.float64)
        layer.eval()
        with torch.no_grad():
            layer.norm1.weight.copy_(take(d)); layer.norm1.bias.copy_(take(d))
            Wq, bq, Wk, bk, Wv, bv = take(d, d), take(d), take(d, d), take(d), take(d, d), take(d)
            layer.self_attn.in_proj_weight.copy_(torch.cat([Wq, Wk, Wv], 0))
            layer.self_attn.in_proj_bias.copy_(torch.cat([bq, bk, bv], 0))
            layer.self_attn.out_proj.weight.copy_(take(d, d)); layer.self_attn.out_proj.bias.copy_(take(d))
            layer.norm2.weight.copy_(take(d)); layer.norm2.bias.copy_(take(d))
            layer.linear1.weight.copy_(take(Fd, d)); layer.linear1.bias.copy_(take(Fd))
            layer.linear2.weight.copy_(take(d, Fd)); layer.linear2.bias.copy_(take(d))
        with torch.no_grad():
            if use_sdpa:
                a = layer.norm1(z)
                qkv = F.linear(a, layer.self_attn.in_proj_weight, layer.self_attn.in_proj_bias)
                q, kk, vv = qkv.split(d, dim=-1)
                sh = lambda t: t.reshape(1, n + k, H, d // H).transpose(1, 2)
                o = F.scaled_dot_product_attention(sh(q), sh(kk), sh(vv), attn_mask=allowed)
                o = o.transpose(1, 2).reshape(1, n + k, d)
                z = z + layer.self_attn.out_proj(o)
                z = z + layer.linear2(F.gelu(layer.linear1(layer.norm2(z)), approximate="tanh"))
            else:
                z = layer(z, src_mask=~allowed)
    lnf_g, lnf_b, w, b = take(d), take(d), take(1, d), take(1)
    out = F.linear(F.layer_norm(z[0, n:], (d,), lnf_g, lnf_b, eps=1e-5), w, b)[:, 0]
    assert pos == blob.numel()
    return out.numpy()


@pytest.mark.parametrize("use_sdpa", [False, True])
@pytest.mark.parametrize("variant", ["base", "sharp"])
def test_oracle_matches_torch_encoder_layer(use_sdpa, variant):
    inp = make_inputs([13, 6], [9, 4], d=48, H=3, L=2, F=96, dtype="f32", seed=5, variant=variant)
    cache = oracle.encode(inp.weights, inp.d, inp.H, inp.L, inp.F, inp.hist_emb, inp.hist_offsets)
    scores = oracle.rank(inp.weights, inp.d, inp.H, inp.L, inp.F, cache, inp.hist_offsets,
                         inp.cand_emb, inp.cand_offsets)
    co = inp.cand_offsets
    for u in range(inp.U):
        ref = _torch_scores(inp, u, use_sdpa=use_sdpa)
        np.testing.assert_allclose(scores[co[u]:co[u + 1]], ref, rtol=1e-9, atol=1e-9)


def test_building_blocks_match_torch():
    rng = np.random.default_rng(0)
    x = rng.standard_normal((7, 40)) * 3 + 1
    g, b = rng.standard_normal(40), rng.standard_normal(40)
    ref = F.layer_norm(torch.tensor(x), (40,), torch.tensor(g), torch.tensor(b), eps=1e-5).numpy()
    np.testing.assert_allclose(oracle.layer_norm(x, g, b), ref, rtol=1e-12, atol=1e-12)
    y = rng.standard_normal(1000) * 4
    np.testing.assert_allclose(oracle.gelu_tanh(y), F.gelu(torch.tensor(y), approximate="tanh").numpy(),
                               rtol=1e-12, atol=1e-14)
    W, bb = rng.standard_normal((5, 40)), rng.standard_normal(5)
    np.testing.assert_allclose(oracle.linear(x, W, bb),
                               F.linear(torch.tensor(x), torch.tensor(W), torch.tensor(bb)).numpy(),
                               rtol=1e-12, atol=1e-12)


# ---------------------------------------------------------------------------
# Closed forms
# ---------------------------------------------------------------------------

def test_single_key_attention_returns_value_exactly():
    rng = np.random.default_rng(1)
    q = rng.standard_normal((4, 16)) * 10
    k = rng.standard_normal((1, 16))
    v = rng.standard_normal((1, 16))
    out = oracle.masked_softmax_attention(q, k, v, np.ones((4, 1), dtype=bool))
    assert np.array_equal(out, np.repeat(v, 4, axis=0))


def test_zero_logits_give_mean_of_allowed_values():
    rng = np.random.default_rng(2)
    k, v = rng.standard_normal((9, 8)), rng.standard_normal((9, 8))
    allowed = rng.random((5, 9)) < 0.5
    allowed[:, 0] = True
    out = oracle.masked_softmax_attention(np.zeros((5, 8)), k, v, allowed)
    for i in range(5):
        np.testing.assert_allclose(out[i], v[allowed[i]].mean(axis=0), rtol=1e-13, atol=1e-13)


def _torch_token_mlp(inp, x, attn_out_fn):
    """Per-token transformer with the attention output supplied by attn_out_fn."""
    d, L, Fd = inp.d, inp.L, inp.F
    layers, final = oracle.unpack_weights(inp.weights, d, L, Fd)
    g = torch.tensor(x)
    T = lambda a: torch.tensor(np.ascontiguousarray(a))
    for l, lw in enumerate(layers):
        a = F.layer_norm(g, (d,), T(lw["ln1_g"]), T(lw["ln1_b"]), eps=1e-5)
        o = attn_out_fn(l, a, lw)
        g = g + F.linear(o, T(lw["Wo"]), T(lw["bo"]))
        a2 = F.layer_norm(g, (d,), T(lw["ln2_g"]), T(lw["ln2_b"]), eps=1e-5)
        g = g + F.linear(F.gelu(F.linear(a2, T(lw["W1"]), T(lw["b1"])), approximate="tanh"),
                         T(lw["W2"]), T(lw["b2"]))
    hf = F.layer_norm(g, (d,), T(final["lnf_g"]), T(final["lnf_b"]), eps=1e-5)
    return (hf @ T(final["w_score"]) + float(final["b_score"])).numpy()


def test_empty_history_is_a_per_token_mlp():
    # n_u = 0: softmax over the single self logit is 1, so each layer's
    # attention output is the candidate's own value projection.
    inp = make_inputs([0, 4], [6, 2], d=32, H=2, L=2, F=64, dtype="f32", seed=7, variant="perturbed")
    cache = oracle.encode(inp.weights, inp.d, inp.H, inp.L, inp.F, inp.hist_emb, inp.hist_offsets)
    s = oracle.rank(inp.weights, inp.d, inp.H, inp.L, inp.F, cache, inp.hist_offsets,
                    inp.cand_emb, inp.cand_offsets)
    T = lambda a: torch.tensor(np.ascontiguousarray(a))
    ref = _torch_token_mlp(inp, inp.cand_emb[0:6].astype(np.float64),
                           lambda l, a, lw: F.linear(a, T(lw["Wv"]), T(lw["bv"])))
    np.testing.assert_allclose(s[0:6], ref, rtol=1e-11, atol=1e-11)


def test_zero_query_weights_average_history_and_self():
    # Wq = bq = 0 makes every logit 0, so one layer's attention output is the
    # plain mean of the user's cached values and the candidate's own value.
    inp = make_inputs([5], [3], d=16, H=2, L=1, F=32, dtype="f32", seed=8, variant="perturbed")
    d = inp.d
    w = inp.weights.astype(np.float64).copy()
    off = 2 * d                 # ln1_g, ln1_b, then Wq and bq
    w[off:off + d * d + d] = 0.0
    inp.weights = w
    cache = oracle.encode(w, d, inp.H, inp.L, inp.F, inp.hist_emb, inp.hist_offsets)
    s = oracle.rank(w, d, inp.H, inp.L, inp.F, cache, inp.hist_offsets, inp.cand_emb, inp.cand_offsets)
    layers, _ = oracle.unpack_weights(w, d, inp.L, inp.F)
    lw = layers[0]
    T = lambda a: torch.tensor(np.ascontiguousarray(a))
    Xh = T(inp.hist_emb.astype(np.float64))
    a_hist = F.layer_norm(Xh, (d,), T(lw["ln1_g"]), T(lw["ln1_b"]), eps=1e-5)
    v_hist = F.linear(a_hist, T(lw["Wv"]), T(lw["bv"]))            # [5, d]

    def mean_attn(l, a, lw_):
        v_self = F.linear(a, T(lw_["Wv"]), T(lw_["bv"]))          # [3, d]
        return (v_hist.sum(0, keepdim=True) + v_self) / (v_hist.shape[0] + 1)

    ref = _torch_token_mlp(inp, inp.cand_emb.astype(np.float64), mean_attn)
    np.testing.assert_allclose(s, ref, rtol=1e-11, atol=1e-11)


# ---------------------------------------------------------------------------
# Invariants
# ---------------------------------------------------------------------------

def _scores(inp, cand_emb=None, cand_offsets=None):
    cache = oracle.encode(inp.weights, inp.d, inp.H, inp.L, inp.F, inp.hist_emb, inp.hist_offsets)
    return oracle.rank(inp.weights, inp.d, inp.H, inp.L, inp.F, cache, inp.hist_offsets,
                       inp.cand_emb if cand_emb is None else cand_emb,
                       inp.cand_offsets if cand_offsets is None else cand_offsets)


def test_candidate_permutation_equivariance():
    inp = make_inputs([11, 8], [12, 7], d=32, H=4, L=2, F=64, dtype="f32", seed=9, variant="sharp")
    base = _scores(inp)
    perm = np.concatenate([np.random.default_rng(0).permutation(12),
                           12 + np.random.default_rng(1).permutation(7)])
    permuted = _scores(inp, cand_emb=inp.cand_emb[perm])
    np.testing.assert_allclose(permuted, base[perm], rtol=1e-12, atol=1e-12)


def test_user_permutation_equivariance():
    inp = make_inputs([11, 3, 8], [5, 7, 2], d=32, H=4, L=2, F=64, dtype="f32", seed=10)
    base = _scores(inp)
    order = [2, 0, 1]
    ho, co = inp.hist_offsets, inp.cand_offsets
    X = np.concatenate([inp.hist_emb[ho[u]:ho[u + 1]] for u in order])
    C = np.concatenate([inp.cand_emb[co[u]:co[u + 1]] for u in order])
    nh = np.concatenate([[0], np.cumsum([ho[u + 1] - ho[u] for u in order])]).astype(np.int32)
    nc = np.concatenate([[0], np.cumsum([co[u + 1] - co[u] for u in order])]).astype(np.int32)
    cache = oracle.encode(inp.weights, inp.d, inp.H, inp.L, inp.F, X, nh)
    s = oracle.rank(inp.weights, inp.d, inp.H, inp.L, inp.F, cache, nh, C, nc)
    expect = np.concatenate([base[co[u]:co[u + 1]] for u in order])
    np.testing.assert_allclose(s, expect, rtol=1e-12, atol=1e-12)


def test_batch_composition_independence():
    inp = make_inputs([9], [10], d=32, H=2, L=2, F=64, dtype="f32", seed=12)
    base = _scores(inp)
    for c in [0, 4, 9]:
        alone = _scores(inp, cand_emb=inp.cand_emb[c:c + 1], cand_offsets=np.array([0, 1], np.int32))
        np.testing.assert_allclose(alone[0], base[c], rtol=1e-12, atol=1e-12)


def test_cache_is_causal_and_candidate_independent():
    inp = make_inputs([10], [4], d=32, H=2, L=3, F=64, dtype="f32", seed=13, variant="perturbed")
    c0 = oracle.encode(inp.weights, inp.d, inp.H, inp.L, inp.F, inp.hist_emb, inp.hist_offsets)
    t = 6
    X2 = inp.hist_emb.copy()
    # a random (not constant) change: LayerNorm removes constant shifts
    X2[t] += np.random.default_rng(0).standard_normal(inp.d).astype(np.float32)
    c1 = oracle.encode(inp.weights, inp.d, inp.H, inp.L, inp.F, X2, inp.hist_offsets)
    np.testing.assert_allclose(c1[:, :, :, :t, :], c0[:, :, :, :t, :], rtol=1e-13, atol=1e-13)
    assert np.abs(c1[:, :, :, t:, :] - c0[:, :, :, t:, :]).max() > 1e-3
    # In the plain definition, changing candidates leaves history K/V untouched.
    _, kv0 = oracle.full_sequence(inp.weights, inp.d, inp.H, inp.L, inp.F, inp.hist_emb, inp.cand_emb)
    _, kv1 = oracle.full_sequence(inp.weights, inp.d, inp.H, inp.L, inp.F, inp.hist_emb,
                                  inp.cand_emb * -3.0 + 0.5)
    for (K0, V0), (K1, V1) in zip(kv0, kv1):
        np.testing.assert_allclose(K1, K0, rtol=1e-13, atol=1e-13)
        np.testing.assert_allclose(V1, V0, rtol=1e-13, atol=1e-13)


def test_cache_index_matches_row_major_shape():
    L, H, D, cap = 3, 4, 8, 37
    shape = oracle.cache_shape(L, H, D, cap)
    rng = np.random.default_rng(4)
    for _ in range(200):
        idx = tuple(int(rng.integers(0, s)) for s in shape)
        assert oracle.cache_index(H, D, cap, *idx) == np.ravel_multi_index(idx, shape)


def test_mask_shape_counts():
    n, k = 6, 4
    m = oracle.mfalcon_mask(n, k)
    # history row i sees i+1 keys; each candidate sees n history keys + itself.
    assert [int(m[i].sum()) for i in range(n)] == list(range(1, n + 1))
    assert all(int(m[n + j].sum()) == n + 1 for j in range(k))
    assert not m[:n, n:].any()
