"""MXFP8 (OCP microscaling, E4M3 elements) for the fp8 projection variant.

TEST INFRASTRUCTURE ONLY: used by the tests and nothing in the product path.
It shares no code with the GPU library.

The paper runs its serving forward in FP8 with E4M3 in the forward pass
(Sec. 3, "FP8 quantization"), quantizing the inputs of the fused
LayerNorm/linear/activation modules.  It does not say at which granularity
the scales are taken.  The reading used here is the OCP Microscaling (MX)
format, which gfx950's matrix cores consume natively:

* elements are OCP FP8 E4M3 ("E4M3FN"): sign, 4 exponent bits with bias 7,
  3 mantissa bits; exponent field 0 encodes subnormals m/8 * 2^-6; the code
  S.1111.111 is NaN and there is no infinity, so the largest magnitude is
  1.75 * 2^8 = 448;
* every 32 consecutive values along the contraction axis share one scale
  X = 2^e stored as an E8M0 byte (e + 127), e in [-127, 127];
* e = floor(log2(max |v|)) - 8 (8 is the exponent of E4M3's largest normal),
  and each element is v / X rounded to the nearest E4M3 value, ties to the
  even code, with magnitudes above 448 saturated to 448 (the scaled block
  maximum lies in [256, 512), so the top of each block can exceed 448).
  An all-zero block takes e = -127.

Parity status: pinned against torch's float8_e4m3fn conversion (a library
rounding routine) for in-range values, against the format definition for all
256 codes, and by closed forms (block exponents, exactly representable
blocks, the half-ulp error bound).
"""
from __future__ import annotations

import numpy as np

E4M3_MAX = 448.0
E4M3_EMAX = 8          # exponent of the largest normal E4M3 value
MX_BLOCK = 32


def e4m3_value(codes):
    """Value of each E4M3 code (uint8) from the format definition; NaN for
    the two NaN codes."""
    c = np.asarray(codes, dtype=np.int64)
    sign = np.where(c & 0x80, -1.0, 1.0)
    e = (c >> 3) & 0xF
    m = (c & 0x7).astype(np.float64)
    mag = np.where(e == 0, m / 8.0 * 2.0 ** -6, (1.0 + m / 8.0) * 2.0 ** (e - 7))
    mag = np.where((c & 0x7F) == 0x7F, np.nan, mag)
    return sign * mag


_GRID = e4m3_value(np.arange(0x7F))          # codes 0..126: +0 .. 448, increasing


def e4m3_round_codes(x):
    """Codes of x rounded to the nearest E4M3 value (ties to the even code),
    magnitudes above 448 saturated to 448; negative values (also those that
    round to zero) carry the sign bit.  x must be finite."""
    x = np.asarray(x, dtype=np.float64)
    a = np.minimum(np.abs(x), E4M3_MAX)
    hi = np.searchsorted(_GRID, a, side="left")            # _GRID[hi-1] < a <= _GRID[hi]
    hi = np.minimum(hi, len(_GRID) - 1)
    lo = np.maximum(hi - 1, 0)
    d_lo = a - _GRID[lo]
    d_hi = _GRID[hi] - a
    pick_hi = (d_hi < d_lo) | ((d_hi == d_lo) & (hi % 2 == 0))
    code = np.where(pick_hi, hi, lo)
    code = np.where(a == _GRID[hi], hi, code)
    sign = np.where(np.signbit(x), 0x80, 0)           # a negative value keeps its sign at zero
    return (code | sign).astype(np.uint8)


def mx_block_exponent(amax):
    """Shared exponent of a block whose largest magnitude is amax."""
    amax = np.asarray(amax, dtype=np.float64)
    with np.errstate(divide="ignore"):
        e = np.floor(np.log2(np.where(amax > 0, amax, 1.0))) - E4M3_EMAX
    e = np.where(amax > 0, e, -127.0)
    return np.clip(e, -127, 127).astype(np.int64)


def mx_quantize(x):
    """MXFP8 encoding of x [..., K] (K a multiple of 32) along its last axis:
    (codes uint8 [..., K], scale bytes uint8 [..., K/32] = e + 127)."""
    x = np.asarray(x, dtype=np.float64)
    K = x.shape[-1]
    assert K % MX_BLOCK == 0, "the contraction length must be a multiple of 32"
    blocks = x.reshape(x.shape[:-1] + (K // MX_BLOCK, MX_BLOCK))
    e = mx_block_exponent(np.max(np.abs(blocks), axis=-1))
    scaled = blocks / np.exp2(e.astype(np.float64))[..., None]     # exact: power of two
    codes = e4m3_round_codes(scaled).reshape(x.shape)
    return codes, (e + 127).astype(np.uint8)


def mx_dequantize(codes, scales):
    """Values of an MXFP8 encoding."""
    codes = np.asarray(codes)
    K = codes.shape[-1]
    v = e4m3_value(codes).reshape(codes.shape[:-1] + (K // MX_BLOCK, MX_BLOCK))
    e = np.asarray(scales, dtype=np.int64) - 127
    return (v * np.exp2(e.astype(np.float64))[..., None]).reshape(codes.shape)


def mx_round(x):
    """x replaced by the values of its MXFP8 encoding along the last axis."""
    return mx_dequantize(*mx_quantize(x))


def linear_mx(x, W, b):
    """x W^T + b with x (rows) and W (rows of the [out, in] matrix) both
    MXFP8-encoded along the input axis; the products and sums are exact
    (float64)."""
    return mx_round(x) @ mx_round(W).T + np.asarray(b, dtype=np.float64)
