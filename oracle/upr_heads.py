"""CPU oracle for the per-action ranking heads and utility top-K (UniPinRec).

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import, call or
link this module; only the tests, the smoke check and the benchmark's CPU
baseline leg use it.  It shares no code with the GPU library.

What is computed (paper, Sec. 3):

* Action prediction (ranking objective of Masked Action Modeling): for each
  action type c = 1..C a dedicated MLP head h_psi_c maps the transformer's
  hidden state z of a position to a scalar logit; the action probability is
  its sigmoid (the loss is a per-action binary cross-entropy on these logits,
  so sigmoid is the matching link).
* Serving (Sec. 3, deployment configurations): the unified L0 + L1 service
  ranks the overfetched candidates with the ranking heads and returns the top
  K by the heads' utility functions.

Readings where the paper is silent (each is listed in the design notes):
z is the final LayerNorm of the candidate's hidden state (the input the
single score head also uses); each head is one hidden layer of width Fh with
the same tanh-form GELU as the FFN, h_c(z) = w2_c . GELU(W1_c z + b1_c) + b2_c;
the utility of a candidate is a weighted sum of its action probabilities,
U = sum_c u_c p_c, with caller-given weights u_c (negative for actions such as
hide); the top K of a user are its candidates by utility, highest first, ties
broken by the lower candidate row, NaN utilities last, and a user with fewer
than K candidates returns all of them followed by padding (row -1).

Everything is plain numpy in float64.  Parity status: pinned in
tests/test_heads_pins.py (torch's Linear/GELU/Linear on CPU in float64 as the
textbook MLP, closed forms for zero weights, sigmoid symmetry, brute-force
ordering of small cases with explicit ties).
"""
from __future__ import annotations

import numpy as np

from .upr_oracle import gelu_tanh, layer_norm, linear


def heads_blob_size(d, C, Fh):
    """Values in the heads blob: per head W1[Fh, d] b1[Fh] w2[Fh] b2[1]."""
    return C * (Fh * d + 2 * Fh + 1)


def unpack_heads(blob, d, C, Fh):
    """Split the heads blob (per head, in order: W1 [Fh, d] row-major [out, in],
    b1 [Fh], w2 [Fh], b2 [1]) into a list of float64 dicts."""
    blob = np.asarray(blob, dtype=np.float64).reshape(-1)
    if blob.size != heads_blob_size(d, C, Fh):
        raise ValueError(f"heads blob has {blob.size} values, layout needs {heads_blob_size(d, C, Fh)}")
    heads, pos = [], 0
    for _ in range(C):
        W1 = blob[pos:pos + Fh * d].reshape(Fh, d); pos += Fh * d
        b1 = blob[pos:pos + Fh]; pos += Fh
        w2 = blob[pos:pos + Fh]; pos += Fh
        b2 = blob[pos]; pos += 1
        heads.append({"W1": W1, "b1": b1, "w2": w2, "b2": b2})
    return heads


def action_logits(hidden, final, heads_blob, d, C, Fh):
    """Logits [rows, C] of the C action heads on z = LN_f(hidden)."""
    z = layer_norm(np.asarray(hidden, dtype=np.float64), final["lnf_g"], final["lnf_b"])
    heads = unpack_heads(heads_blob, d, C, Fh)
    out = np.empty((z.shape[0], C))
    for c, hw in enumerate(heads):
        out[:, c] = gelu_tanh(linear(z, hw["W1"], hw["b1"])) @ hw["w2"] + hw["b2"]
    return out


def sigmoid(x):
    """1 / (1 + exp(-x)), computed without overflow for large |x|."""
    x = np.asarray(x, dtype=np.float64)
    e = np.exp(-np.abs(x))
    return np.where(x >= 0, 1.0 / (1.0 + e), e / (1.0 + e))


def utility(probs, weights):
    """U = sum_c u_c p_c per row."""
    return np.asarray(probs, dtype=np.float64) @ np.asarray(weights, dtype=np.float64)


def topk_by_utility(util, cand_offsets, K):
    """Per user, the K candidate rows of highest utility (ties: lower row
    first; NaN utilities after every number).  Returns (rows [U, K] int64,
    values [U, K] float64) with row -1 / NaN padding past a user's k_u."""
    util = np.asarray(util)
    coffs = np.asarray(cand_offsets, dtype=np.int64)
    U = len(coffs) - 1
    rows = np.full((U, K), -1, dtype=np.int64)
    vals = np.full((U, K), np.nan)
    for u in range(U):
        r = np.arange(coffs[u], coffs[u + 1])
        v = util[r]
        nan = np.isnan(v)
        # python's sort on (is NaN, -value, row) is the definition itself
        order = sorted(range(r.size), key=lambda i: (bool(nan[i]), 0.0 if nan[i] else -float(v[i]), int(r[i])))
        take = order[:K]
        rows[u, :len(take)] = r[take]
        vals[u, :len(take)] = v[take]
    return rows, vals
