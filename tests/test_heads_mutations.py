"""Planted mistakes in a copy of the heads oracle must fail at least one pin.

Each case rewrites one expression of oracle/upr_heads.py, loads the result as
a separate module inside the oracle package and runs the pins of
test_heads_pins against it.  The real oracle is untouched.
"""
import types
import warnings

import pytest

import oracle.upr_heads as real_heads
import tests.test_heads_pins as pins

SRC_PATH = real_heads.__file__

MUTATIONS = {
    "LN_f skipped": ('z = layer_norm(np.asarray(hidden, dtype=np.float64), final["lnf_g"], final["lnf_b"])',
                     'z = np.asarray(hidden, dtype=np.float64)'),
    "ReLU instead of GELU": ('gelu_tanh(linear(z, hw["W1"], hw["b1"]))', 'np.maximum(linear(z, hw["W1"], hw["b1"]), 0.0)'),
    "output bias dropped": ('@ hw["w2"] + hw["b2"]', '@ hw["w2"]'),
    "W1 transposed layout": ('W1 = blob[pos:pos + Fh * d].reshape(Fh, d)',
                             'W1 = blob[pos:pos + Fh * d].reshape(d, Fh).T'),
    "b1 and w2 swapped": ('b1 = blob[pos:pos + Fh]; pos += Fh\n        w2 = blob[pos:pos + Fh]; pos += Fh',
                          'w2 = blob[pos:pos + Fh]; pos += Fh\n        b1 = blob[pos:pos + Fh]; pos += Fh'),
    "sigmoid sign": ("return np.where(x >= 0, 1.0 / (1.0 + e), e / (1.0 + e))",
                     "return np.where(x >= 0, e / (1.0 + e), 1.0 / (1.0 + e))"),
    "utility ignores weights": ("@ np.asarray(weights, dtype=np.float64)", ".sum(axis=1)"),
    "ascending utility": ("0.0 if nan[i] else -float(v[i])", "0.0 if nan[i] else float(v[i])"),
    "ties to higher row": ("int(r[i])))", "-int(r[i])))"),
    "NaN first": ("key=lambda i: (bool(nan[i]),", "key=lambda i: (not bool(nan[i]),"),
    "K off by one": ("take = order[:K]", "take = order[:K - 1]"),
}

PINS = [
    lambda: pins.test_action_logits_match_torch_mlp("perturbed"),
    pins.test_zero_first_layer_gives_constant_logits,
    pins.test_sigmoid_identities,
    pins.test_utility_is_the_weighted_sum,
    pins.test_topk_hand_worked_with_ties_and_nan,
    pins.test_topk_matches_lexsort_on_random_cases,
    pins.test_heads_blob_size_and_layout,
]


def _mutant(old, new):
    src = open(SRC_PATH).read()
    assert src.count(old) >= 1, f"mutation anchor not found: {old!r}"
    mod = types.ModuleType("oracle.upr_heads_mutant")
    mod.__file__ = SRC_PATH
    mod.__package__ = "oracle"
    exec(compile(src.replace(old, new), SRC_PATH + "[mutant]", "exec"), mod.__dict__)
    return mod


def _failures(mod, monkeypatch):
    monkeypatch.setattr(pins, "heads_oracle", mod)
    failed = 0
    for pin in PINS:
        try:
            with warnings.catch_warnings():
                warnings.simplefilter("ignore")
                pin()
        except (AssertionError, ValueError, FloatingPointError, IndexError):
            failed += 1
    return failed


def test_real_heads_oracle_passes_every_pin(monkeypatch):
    assert _failures(real_heads, monkeypatch) == 0


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_planted_mistake_is_caught(name, monkeypatch):
    old, new = MUTATIONS[name]
    assert _failures(_mutant(old, new), monkeypatch) >= 1, f"mutation '{name}' passed every pin"
