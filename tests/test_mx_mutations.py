"""Planted mistakes in a copy of the MXFP8 oracle must fail at least one pin.

Each case rewrites one expression of oracle/upr_mx.py, loads the result as a
separate module and runs the pins of test_mx_pins against it (the ranking
pins use the real oracle's rank with the mutant's linear map).  A second set
rewrites the fp8 composition in oracle/upr_oracle.py (which projection inputs
are encoded) and runs the ranking pins against that copy.  The real oracle is
untouched.
"""
import types
import warnings

import pytest

import oracle.upr_mx as real_mx
import tests.test_mx_pins as pins

SRC_PATH = real_mx.__file__

MUTATIONS = {
    "emax 7": ("E4M3_EMAX = 8", "E4M3_EMAX = 7"),
    "ceil for the block exponent": ("e = np.floor(np.log2(", "e = np.ceil(np.log2("),
    "ties away from zero": ("((d_hi == d_lo) & (hi % 2 == 0))", "(d_hi == d_lo)"),
    "ties to odd": ("((d_hi == d_lo) & (hi % 2 == 0))", "((d_hi == d_lo) & (hi % 2 == 1))"),
    "blocks of 16": ("MX_BLOCK = 32", "MX_BLOCK = 16"),
    "subnormal step off by 2": ("m / 8.0 * 2.0 ** -6", "m / 8.0 * 2.0 ** -7"),
    "exponent bias 8": ("(1.0 + m / 8.0) * 2.0 ** (e - 7)", "(1.0 + m / 8.0) * 2.0 ** (e - 8)"),
    "scale multiplied": ("scaled = blocks / np.exp2(", "scaled = blocks * np.exp2("),
    "sign of zero dropped": ("sign = np.where(np.signbit(x), 0x80, 0)",
                             "sign = np.where(np.signbit(x) & (code != 0), 0x80, 0)"),
    "no saturation (NaN code)": ("    return (code | sign).astype(np.uint8)",
                                 "    code = np.where(np.abs(x) > 464.0, 0x7F, code)\n    return (code | sign).astype(np.uint8)"),
    "zero block exponent 0": ("e = np.where(amax > 0, e, -127.0)", "e = np.where(amax > 0, e, 0.0)"),
    "activation blocks across rows": ("return mx_round(x) @ mx_round(W).T", "return mx_round(x.T).T @ mx_round(W).T"),
    "weights not encoded": ("return mx_round(x) @ mx_round(W).T", "return mx_round(x) @ W.T"),
}

PINS = [
    pins.test_e4m3_values_of_all_codes,
    pins.test_e4m3_rounding_matches_torch_in_range,
    pins.test_e4m3_saturates_above_448,
    lambda: [pins.test_block_exponent_closed_forms(a, e) for a, e in
             [(1.0, -8), (448.0, 0), (256.0, 0), (511.99, 0), (512.0, 1), (0.75, -9),
              (2.0 ** -120, -127), (2.0 ** -140, -127), (0.0, -127), (2.0 ** 200, 127)]],
    pins.test_block_scale_puts_the_maximum_in_256_512,
    pins.test_representable_blocks_round_trip_exactly,
    pins.test_error_within_half_an_element_ulp,
    pins.test_all_zero_and_mixed_sign_blocks,
    pins.test_linear_mx_matches_torch_fp8_when_every_scale_is_one,
    pins.test_linear_mx_on_representable_operands_is_exact,
    pins.test_mxfp8_rank_is_per_candidate,
    pins.test_mxfp8_rank_stays_near_the_exact_model,
    pins.test_mxfp8_rank_matches_an_independent_composition,
]


def _mutant(old, new):
    src = open(SRC_PATH).read()
    assert src.count(old) >= 1, f"mutation anchor not found: {old!r}"
    mod = types.ModuleType("oracle.upr_mx_mutant")
    mod.__file__ = SRC_PATH
    mod.__package__ = "oracle"
    exec(compile(src.replace(old, new), SRC_PATH + "[mutant]", "exec"), mod.__dict__)
    return mod


def _failures(mod, monkeypatch):
    import oracle.upr_oracle as uo
    monkeypatch.setattr(pins, "mx_oracle", mod)
    real_rule = uo._projection_rule
    monkeypatch.setattr(uo, "_projection_rule",
                        lambda proj: mod.linear_mx if proj == "mxfp8" else real_rule(proj))
    failed = 0
    for pin in PINS:
        try:
            with warnings.catch_warnings():
                warnings.simplefilter("ignore")
                pin()
        except (AssertionError, ValueError, FloatingPointError, IndexError):
            failed += 1
    return failed


def test_real_mx_oracle_passes_every_pin(monkeypatch):
    assert _failures(real_mx, monkeypatch) == 0


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_planted_mistake_is_caught(name, monkeypatch):
    old, new = MUTATIONS[name]
    assert _failures(_mutant(old, new), monkeypatch) >= 1, f"mutation '{name}' passed every pin"


# Mistakes in how the ranking pass composes the fp8 projections
# (oracle/upr_oracle.py): a quantization point dropped or one added.
COMPOSITION_MUTATIONS = {
    "attention output not encoded": (
        'g = g + lin(o.transpose(1, 0, 2).reshape(kc_rows, d), lw["Wo"], lw["bo"])',
        'g = g + linear(o.transpose(1, 0, 2).reshape(kc_rows, d), lw["Wo"], lw["bo"])'),
    "GELU output not encoded": (
        'return lin(gelu_tanh(lin(a, lw["W1"], lw["b1"])), lw["W2"], lw["b2"])',
        'return linear(gelu_tanh(lin(a, lw["W1"], lw["b1"])), lw["W2"], lw["b2"])'),
    "attention output held in fp16 first": (
        'g = g + lin(o.transpose(1, 0, 2).reshape(kc_rows, d), lw["Wo"], lw["bo"])',
        'g = g + lin(o.transpose(1, 0, 2).reshape(kc_rows, d).astype(np.float16).astype(np.float64), '
        'lw["Wo"], lw["bo"])'),
}


@pytest.mark.parametrize("name", sorted(COMPOSITION_MUTATIONS))
def test_planted_composition_mistake_is_caught(name, monkeypatch):
    import oracle
    import oracle.upr_oracle as uo
    old, new = COMPOSITION_MUTATIONS[name]
    src = open(uo.__file__).read()
    assert src.count(old) == 1, f"mutation anchor not found: {old!r}"
    mod = types.ModuleType("oracle.upr_oracle_mutant")
    mod.__file__ = uo.__file__
    mod.__package__ = "oracle"
    exec(compile(src.replace(old, new), uo.__file__ + "[mutant]", "exec"), mod.__dict__)
    monkeypatch.setattr(oracle, "rank", mod.rank)
    with pytest.raises(AssertionError):
        pins.test_mxfp8_rank_matches_an_independent_composition()
