"""Planted mistakes in a copy of the oracle must fail at least one pin.

Each case rewrites one expression in the oracle's source (a dropped term, a
wrong sign, scale or index, a transposed operand), loads the result as a
separate module and runs the pins of test_oracle_pins against it.  The real
oracle is untouched.
"""
import types

import pytest

import oracle.upr_oracle as real_oracle
import tests.test_oracle_pins as pins

SRC_PATH = real_oracle.__file__

MUTATIONS = {
    "self key dropped from value sum": ("+ p[:, -1:] * vs[j]", "+ 0.0 * vs[j]"),
    "self logit dropped": ("s = np.concatenate([s_hist, s_self[:, None]], axis=1)",
                           "s = np.concatenate([s_hist, s_self[:, None] - 1e9], axis=1)"),
    "attention scale 1/D": ("s = (q @ k.T) / math.sqrt(D)", "s = (q @ k.T) / D"),
    "rank scale missing": ("s_hist = (q[j] @ Kh.T) / math.sqrt(D)", "s_hist = (q[j] @ Kh.T)"),
    "causal mask without diagonal": ("causal = np.tril(np.ones((n, n), dtype=bool))",
                                     "causal = np.tril(np.ones((n, n), dtype=bool), -1) | (np.arange(n)[:, None] == 0)"),
    "mask lets candidates see each other": ("cand_row = (i >= n) & ((j < n) | (j == i))",
                                            "cand_row = (i >= n) & (j <= i)"),
    "Wo transposed in rank": ("g = g + lin(o.transpose(1, 0, 2).reshape(kc_rows, d), lw[\"Wo\"], lw[\"bo\"])",
                              "g = g + lin(o.transpose(1, 0, 2).reshape(kc_rows, d), lw[\"Wo\"].T, lw[\"bo\"])"),
    "value bias dropped in rank": ("vs = _split_heads(lin(a, lw[\"Wv\"], lw[\"bv\"]), H)",
                                   "vs = _split_heads(lin(a, lw[\"Wv\"], 0.0), H)"),
    "gelu constant": ("0.044715", "0.04715"),
    "unbiased variance": ("var = ((x - mu) ** 2).mean(axis=-1, keepdims=True)",
                          "var = ((x - mu) ** 2).sum(axis=-1, keepdims=True) / (x.shape[-1] - 1)"),
    "layernorm eps changed": ("def layer_norm(x, gain, shift, eps=1e-5)", "def layer_norm(x, gain, shift, eps=1e-3)"),
    "head split transposed": ("return x.reshape(rows, H, d // H).transpose(1, 0, 2)",
                              "return x.reshape(rows, d // H, H).transpose(2, 0, 1)"),
    "score bias dropped": ("@ final[\"w_score\"] + final[\"b_score\"]", "@ final[\"w_score\"]"),
    "ffn residual sign": ("g = g + ffn(g, lw, lin)", "g = g - ffn(g, lw, lin)"),
    "cache index kv/head swapped": ("return (((layer * 2 + kv) * H + head) * capacity_rows + row) * D + e",
                                    "return (((layer * H + head) * 2 + kv) * capacity_rows + row) * D + e"),
    "encode stores pre-projection keys": ("cache[l, 0, :, lo:hi, :] = k", "cache[l, 0, :, lo:hi, :] = q"),
    "softmax normalised over candidates": ("p = p / p.sum(axis=1, keepdims=True)",
                                           "p = p / p.sum(axis=0, keepdims=True)"),
    "ln2 uses ln1 params": ("a = layer_norm(x, lw[\"ln2_g\"], lw[\"ln2_b\"])",
                            "a = layer_norm(x, lw[\"ln1_g\"], lw[\"ln1_b\"])"),
}

PINS = [
    lambda: pins.test_cached_equals_full_sequence("perturbed"),
    lambda: pins.test_oracle_matches_torch_encoder_layer(False, "sharp"),
    pins.test_building_blocks_match_torch,
    pins.test_empty_history_is_a_per_token_mlp,
    pins.test_zero_query_weights_average_history_and_self,
    pins.test_cache_index_matches_row_major_shape,
    pins.test_mask_shape_counts,
    pins.test_single_key_attention_returns_value_exactly,
]


def _mutant(old, new):
    src = open(SRC_PATH).read()
    assert src.count(old) >= 1, f"mutation anchor not found: {old!r}"
    mod = types.ModuleType("oracle_mutant")
    mod.__file__ = SRC_PATH
    exec(compile(src.replace(old, new), SRC_PATH + "[mutant]", "exec"), mod.__dict__)
    return mod


def _failures(mod, monkeypatch):
    monkeypatch.setattr(pins, "oracle", mod)
    failed = 0
    for pin in PINS:
        try:
            with __import__("warnings").catch_warnings():
                __import__("warnings").simplefilter("ignore")
                pin()
        except (AssertionError, ValueError, FloatingPointError, IndexError):
            failed += 1
    return failed


def test_unmutated_oracle_passes_every_pin(monkeypatch):
    mod = _mutant("", "")
    assert _failures(mod, monkeypatch) == 0


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_planted_mistake_is_caught(name, monkeypatch):
    old, new = MUTATIONS[name]
    mod = _mutant(old, new)
    assert _failures(mod, monkeypatch) >= 1, f"no pin caught: {name}"
