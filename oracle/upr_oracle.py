"""CPU oracle for cross-stage KV-cache candidate ranking (UniPinRec).

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import, call or
link this module; only the tests, the smoke check and the benchmark's CPU
baseline leg use it.  It shares no code with the GPU library: it unpacks the
weight blob, indexes the cache and does every step of the arithmetic itself.

Everything is plain numpy in float64, on inputs that are given (bf16-rounded
for bf16 workloads, then widened).  No intermediate is rounded.

What is computed (paper, Sec. 3):

* One shared transformer processes the concatenated sequence
  [history tokens || candidate tokens].  History positions use ordinary
  causal attention; candidate position n+j attends to every history position
  and never to another candidate ("Masked Action Modeling", attention-pattern
  item).  Candidates also attend to themselves: the KV-cache section describes
  the candidate block as an identity mask, so each candidate score depends on
  nothing but the history and the candidate itself.
* Because history rows never attend to candidates, the history keys/values
  of every layer are candidate-independent (Eq. 2, the no-leakage property),
  so they can be produced once (retrieval) and reused (ranking): the
  "KV-cache sharing across stages" section.  ``encode`` produces that cache,
  ``rank`` consumes it, and ``full_sequence`` is the plain definition (one
  masked forward over the concatenated sequence) that the two must reproduce.

Readings where the paper is silent (each is listed in the design notes):
pre-LN blocks with a final LayerNorm, LayerNorm eps 1e-5 with biased variance
and affine gain/shift, tanh-form GELU in the FFN, a bias on every linear map,
attention scale 1/sqrt(D), H key/value heads (no grouping), no positional term
inside the model (all candidates share one position, so the caller folds any
position embedding into the tokens), and one linear(d -> 1) score head on the
final LayerNorm of the candidate's hidden state, returned as a raw logit.

Parity status: every function here is pinned by tests that do not reuse its
own code: brute force (``full_sequence`` vs ``encode`` + ``rank``), torch's
``TransformerEncoderLayer`` / ``scaled_dot_product_attention`` on CPU as a
textbook routine, closed forms (single key, zero query weights, empty
history), and permutation / batch-composition invariants.  The paper itself
prints no worked numerical example, so absolute values are pinned only by
those routes.
"""
from __future__ import annotations

import math

import numpy as np


# ----------------------------------------------------------------------------
# Weight blob
# ----------------------------------------------------------------------------

_LAYER_ENTRIES = ("ln1_g", "ln1_b", "Wq", "bq", "Wk", "bk", "Wv", "bv",
                  "Wo", "bo", "ln2_g", "ln2_b", "W1", "b1", "W2", "b2")


def unpack_weights(blob, d, L, F):
    """Split the flat weight blob into named float64 arrays.

    Blob order, per layer: ln1_g[d] ln1_b[d] Wq[d,d] bq[d] Wk[d,d] bk[d]
    Wv[d,d] bv[d] Wo[d,d] bo[d] ln2_g[d] ln2_b[d] W1[F,d] b1[F] W2[d,F] b2[d];
    then lnf_g[d] lnf_b[d] w_score[d] b_score[1].  Linear weights are
    [out, in].  Returns (list of per-layer dicts, dict of final weights).
    """
    blob = np.asarray(blob, dtype=np.float64).reshape(-1)
    shapes = {"ln1_g": (d,), "ln1_b": (d,), "Wq": (d, d), "bq": (d,),
              "Wk": (d, d), "bk": (d,), "Wv": (d, d), "bv": (d,),
              "Wo": (d, d), "bo": (d,), "ln2_g": (d,), "ln2_b": (d,),
              "W1": (F, d), "b1": (F,), "W2": (d, F), "b2": (d,)}
    pos = 0

    def take(shape):
        nonlocal pos
        size = int(np.prod(shape))
        out = blob[pos:pos + size].reshape(shape)
        pos += size
        return out

    layers = []
    for _ in range(L):
        layers.append({name: take(shapes[name]) for name in _LAYER_ENTRIES})
    final = {"lnf_g": take((d,)), "lnf_b": take((d,)),
             "w_score": take((d,)), "b_score": take((1,))[0]}
    if pos != blob.size:
        raise ValueError(f"weight blob has {blob.size} values, layout needs {pos}")
    return layers, final


# ----------------------------------------------------------------------------
# Building blocks (textbook definitions)
# ----------------------------------------------------------------------------

def layer_norm(x, gain, shift, eps=1e-5):
    """(x - mean) / sqrt(var + eps) * gain + shift over the last axis, with the
    population (biased) variance."""
    mu = x.mean(axis=-1, keepdims=True)
    var = ((x - mu) ** 2).mean(axis=-1, keepdims=True)
    return (x - mu) / np.sqrt(var + eps) * gain + shift


def gelu_tanh(x):
    """GELU, tanh form: 0.5 x (1 + tanh(sqrt(2/pi) (x + 0.044715 x^3)))."""
    return 0.5 * x * (1.0 + np.tanh(math.sqrt(2.0 / math.pi) * (x + 0.044715 * x ** 3)))


def linear(x, W, b):
    """x W^T + b with W stored [out, in]."""
    return x @ W.T + b


def masked_softmax_attention(q, k, v, allowed):
    """softmax(q k^T / sqrt(D) restricted to ``allowed``) v for one head.

    q [nq, D], k and v [nk, D], allowed bool [nq, nk] (every row allows at
    least one key).  Disallowed logits are -inf; the row maximum is
    subtracted before exponentiating.  No queries: no output rows.
    """
    D = q.shape[-1]
    if q.shape[0] == 0:
        return np.zeros((0, v.shape[-1]))
    s = (q @ k.T) / math.sqrt(D)
    s = np.where(allowed, s, -np.inf)
    m = s.max(axis=-1, keepdims=True)
    p = np.exp(s - m)
    p = p / p.sum(axis=-1, keepdims=True)
    return p @ v


def ffn(x, lw, lin=None):
    """Feed-forward sub-block input -> LN2 -> W1 -> GELU -> W2 (no residual)."""
    a = layer_norm(x, lw["ln2_g"], lw["ln2_b"])
    lin = linear if lin is None else lin
    return lin(gelu_tanh(lin(a, lw["W1"], lw["b1"])), lw["W2"], lw["b2"])


def score_head(h, final):
    """Raw logit w . LN_f(h) + b for each row of h."""
    return layer_norm(h, final["lnf_g"], final["lnf_b"]) @ final["w_score"] + final["b_score"]


def mfalcon_mask(n, k):
    """Boolean [n+k, n+k] mask of the concatenated sequence (True = may attend).

    Row i < n (history): causal, keys 0..i (the position itself included, as
    in Eq. 2).  Row n+j (candidate j): every history key 0..n-1 and itself,
    never another candidate.
    """
    N = n + k
    i = np.arange(N)[:, None]
    j = np.arange(N)[None, :]
    hist_row = (i < n) & (j <= i)
    cand_row = (i >= n) & ((j < n) | (j == i))
    return hist_row | cand_row


# ----------------------------------------------------------------------------
# Packed KV cache
# ----------------------------------------------------------------------------

def cache_index(H, D, capacity_rows, layer, kv, head, row, e):
    """Flat element index of (layer, kv, head, row, e) in the packed cache.

    Layout [L][2][H][capacity_rows][D]: per layer a K plane (kv=0) then a V
    plane (kv=1); inside a plane heads are outermost, then history rows (one
    per packed history token, user u owning rows hist_offsets[u] ..
    hist_offsets[u+1]-1), then the head's D features.
    """
    return (((layer * 2 + kv) * H + head) * capacity_rows + row) * D + e


def cache_shape(L, H, D, capacity_rows):
    return (L, 2, H, capacity_rows, D)


# ----------------------------------------------------------------------------
# The three entry points
# ----------------------------------------------------------------------------

def _split_heads(x, H):
    rows, d = x.shape
    return x.reshape(rows, H, d // H).transpose(1, 0, 2)      # [H, rows, D]


def encode(blob, d, H, L, F, hist_emb, hist_offsets, capacity_rows=None, users=None):
    """History encoding: fills the per-layer K/V cache (Sec. 3, KV-cache sharing).

    For each user, h = that user's history tokens; for every layer,
    a = LN1(h); q, k, v = a Wq^T + bq, a Wk^T + bk, a Wv^T + bv; k and v are
    stored in the cache rows of the user; each head attends causally (keys
    0..t for position t); h += O-projection of the concatenated heads; then
    h += FFN(h).  Returns the float64 cache [L][2][H][capacity][D] (rows of
    users not encoded stay 0).  ``users`` limits the work to a subset.
    """
    layers, _ = unpack_weights(blob, d, L, F)
    D = d // H
    offs = np.asarray(hist_offsets, dtype=np.int64)
    cap = int(offs[-1]) if capacity_rows is None else int(capacity_rows)
    cache = np.zeros(cache_shape(L, H, D, cap), dtype=np.float64)
    X = np.asarray(hist_emb, dtype=np.float64)
    U = len(offs) - 1
    for u in (range(U) if users is None else users):
        lo, hi = int(offs[u]), int(offs[u + 1])
        n = hi - lo
        if n == 0:
            continue
        h = X[lo:hi].copy()
        causal = np.tril(np.ones((n, n), dtype=bool))
        for l, lw in enumerate(layers):
            a = layer_norm(h, lw["ln1_g"], lw["ln1_b"])
            q = _split_heads(linear(a, lw["Wq"], lw["bq"]), H)
            k = _split_heads(linear(a, lw["Wk"], lw["bk"]), H)
            v = _split_heads(linear(a, lw["Wv"], lw["bv"]), H)
            cache[l, 0, :, lo:hi, :] = k
            cache[l, 1, :, lo:hi, :] = v
            if l == L - 1:
                break            # the last layer's output does not reach the cache
            o = np.stack([masked_softmax_attention(q[j], k[j], v[j], causal) for j in range(H)])
            h = h + linear(o.transpose(1, 0, 2).reshape(n, d), lw["Wo"], lw["bo"])
            h = h + ffn(h, lw)
    return cache


def _projection_rule(proj):
    """Linear map of the four projections of a ranking layer: the exact
    model's, or the MXFP8 projection variant's (oracle/upr_mx.py).  The paper
    runs the forward pass in FP8 with E4M3, quantizing the inputs of its fused
    LayerNorm/linear/activation modules (Sec. 3, "FP8 quantization"): here
    every projection input (LN1 output, attention output, LN2 output, GELU
    output) and every projection weight is MXFP8-encoded from its exact value
    along the contraction axis, and nothing else is rounded."""
    if proj == "exact":
        return linear
    if proj == "mxfp8":
        from .upr_mx import linear_mx
        return linear_mx
    raise ValueError(f"unknown projection rule {proj!r}")


def rank_hidden(blob, d, H, L, F, cache, hist_offsets, cand_emb, cand_offsets,
                users=None, cand_rows=None, proj="exact"):
    """Candidate forward pass against the cached history (Sec. 3, serving
    design and KV-cache sharing): only candidate tokens are processed.

    For candidate c of user u and every layer: a = LN1(g); q, k_c, v_c from a;
    per head, the logits are q . K_t / sqrt(D) over the user's cached history
    keys t plus q . k_c / sqrt(D) for the candidate's own key; the softmax of
    those n_u + 1 logits weights the cached values plus v_c; then
    g += O-projection and g += FFN(g).

    Returns the float64 final hidden states g [rows, d] of every packed
    candidate row (NaN for rows not requested).  ``users`` and ``cand_rows``
    (absolute packed row indices) restrict the work; candidates are
    independent, so a subset is exact.  ``proj="mxfp8"`` runs the four
    projections of every layer in MXFP8 (see ``_projection_rule``).
    """
    lin = _projection_rule(proj)
    layers, final = unpack_weights(blob, d, L, F)
    D = d // H
    hoffs = np.asarray(hist_offsets, dtype=np.int64)
    coffs = np.asarray(cand_offsets, dtype=np.int64)
    C = np.asarray(cand_emb, dtype=np.float64)
    cache = np.asarray(cache, dtype=np.float64)
    U = len(coffs) - 1
    hidden = np.full((C.shape[0], d), np.nan)
    wanted = None if cand_rows is None else np.asarray(cand_rows, dtype=np.int64)
    for u in (range(U) if users is None else users):
        rows = np.arange(coffs[u], coffs[u + 1])
        if wanted is not None:
            rows = rows[np.isin(rows, wanted)]
        if rows.size == 0:
            continue
        lo, hi = int(hoffs[u]), int(hoffs[u + 1])
        g = C[rows].copy()
        kc_rows = rows.size
        for l, lw in enumerate(layers):
            a = layer_norm(g, lw["ln1_g"], lw["ln1_b"])
            q = _split_heads(lin(a, lw["Wq"], lw["bq"]), H)
            ks = _split_heads(lin(a, lw["Wk"], lw["bk"]), H)
            vs = _split_heads(lin(a, lw["Wv"], lw["bv"]), H)
            o = np.empty((H, kc_rows, D))
            for j in range(H):
                Kh = cache[l, 0, j, lo:hi, :]          # [n_u, D]
                Vh = cache[l, 1, j, lo:hi, :]
                s_hist = (q[j] @ Kh.T) / math.sqrt(D)               # [k, n_u]
                s_self = np.sum(q[j] * ks[j], axis=-1) / math.sqrt(D)  # [k]
                s = np.concatenate([s_hist, s_self[:, None]], axis=1)
                m = s.max(axis=1, keepdims=True)
                p = np.exp(s - m)
                p = p / p.sum(axis=1, keepdims=True)
                o[j] = p[:, :-1] @ Vh + p[:, -1:] * vs[j]
            g = g + lin(o.transpose(1, 0, 2).reshape(kc_rows, d), lw["Wo"], lw["bo"])
            g = g + ffn(g, lw, lin)
        hidden[rows] = g
    return hidden


def rank(blob, d, H, L, F, cache, hist_offsets, cand_emb, cand_offsets,
         users=None, cand_rows=None, proj="exact"):
    """Candidate scores w . LN_f(g) + b of the final hidden states
    (``rank_hidden``); float64, NaN for rows not requested."""
    _, final = unpack_weights(blob, d, L, F)
    g = rank_hidden(blob, d, H, L, F, cache, hist_offsets, cand_emb, cand_offsets,
                    users=users, cand_rows=cand_rows, proj=proj)
    scores = np.full(g.shape[0], np.nan)
    ok = ~np.isnan(g[:, 0]) if g.shape[0] else np.zeros(0, dtype=bool)
    scores[ok] = score_head(g[ok], final)
    return scores


def full_sequence(blob, d, H, L, F, hist_tokens, cand_tokens):
    """The plain definition for one user: one masked transformer forward over
    [history || candidates] with the mask of ``mfalcon_mask``.

    Returns (scores [k], kv) where kv[l] = (K [H, n, D], V [H, n, D]) are the
    history rows' keys and values at layer l.
    """
    layers, final = unpack_weights(blob, d, L, F)
    X = np.asarray(hist_tokens, dtype=np.float64)
    Cc = np.asarray(cand_tokens, dtype=np.float64)
    n, k = X.shape[0], Cc.shape[0]
    z = np.concatenate([X, Cc], axis=0)
    mask = mfalcon_mask(n, k)
    kv = []
    for lw in layers:
        a = layer_norm(z, lw["ln1_g"], lw["ln1_b"])
        q = _split_heads(linear(a, lw["Wq"], lw["bq"]), H)
        kk = _split_heads(linear(a, lw["Wk"], lw["bk"]), H)
        vv = _split_heads(linear(a, lw["Wv"], lw["bv"]), H)
        kv.append((kk[:, :n, :].copy(), vv[:, :n, :].copy()))
        o = np.stack([masked_softmax_attention(q[j], kk[j], vv[j], mask) for j in range(H)])
        z = z + linear(o.transpose(1, 0, 2).reshape(n + k, d), lw["Wo"], lw["bo"])
        z = z + ffn(z, lw)
    return score_head(z[n:], final), kv
