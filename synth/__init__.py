"""Seeded synthetic inputs for the candidate-ranking path.

This module only *draws* inputs: segment lengths, weights, history tokens and
candidate tokens, in the packed layouts the library's C interface documents.
It holds none of the ranking method's arithmetic (no normalisation, no
projection, no attention), so both the CPU oracle and the GPU path can be fed
from it without sharing any computation.

Value recipe (the paper's data and trained weights are private, so these
stand in for them):

* history and candidate tokens: i.i.d. N(0, 1)/sqrt(d), one row per token;
* every weight matrix: Xavier-uniform, a = sqrt(6 / (fan_in + fan_out)),
  drawn per matrix (Wq, Wk, Wv separately);
* biases 0, LayerNorm gain 1 and shift 0 (``variant="base"``), or small
  uniform perturbations of them (``"perturbed"``), optionally with the query
  projection scaled by 4 so attention logits are sharp (``"sharp"``);
* bf16 workloads round every drawn value to bf16 (round to nearest even) and
  hand it over as float32, so both sides start from identical inputs.

Draw order from ``numpy.random.default_rng(seed)``: ragged lengths (history
lengths, then candidate counts) if the workload is ragged; then the weight
blob entry by entry in blob order (matrices always, vectors only for the
perturbed variants); then the score weight; then history tokens; then
candidate tokens.
"""
from __future__ import annotations

import dataclasses
import math

import numpy as np

# Named workloads.  Shapes follow the paper's ranking setting: per-user action
# histories of up to a few thousand tokens, thousands of candidates per user
# (Sec. 3 serving design; Sec. 4.2 ranking-pass benchmark), with the model
# width and depth a ranking service of this kind uses.
WORKLOADS = {
    # 1 user, 64 history tokens, 128 candidates, d=64, 2 heads, 1 layer, fp32.
    "tiny_f32": dict(U=1, n=64, k=128, d=64, H=2, L=1, F=256, dtype="f32"),
    # 16 users x 256 history tokens, 1000 candidates each, d=256, 4 heads, 2 layers.
    "u16_n256_k1000": dict(U=16, n=256, k=1000, d=256, H=4, L=2, F=1024, dtype="bf16"),
    # 64 users x 1024 history tokens, 2000 candidates each, d=512, 8 heads, 4 layers.
    "u64_n1024_k2000": dict(U=64, n=1024, k=2000, d=512, H=8, L=4, F=2048, dtype="bf16"),
    # 64 users, history ~U[32,2048], candidates ~U[200,3000], d=512, 8 heads, 4 layers.
    "ragged_u64": dict(U=64, n=(32, 2048), k=(200, 3000), d=512, H=8, L=4, F=2048, dtype="bf16"),
    # 8 users x 8192 history tokens, 4096 candidates each, d=512, 8 heads, 4 layers.
    "u8_n8192_k4096": dict(U=8, n=8192, k=4096, d=512, H=8, L=4, F=2048, dtype="bf16"),
}

VARIANTS = ("base", "perturbed", "sharp")


@dataclasses.dataclass
class Inputs:
    """One seeded problem instance in the library's packed layouts."""

    d: int
    H: int
    L: int
    F: int
    dtype: str                      # "f32" or "bf16": the model's arithmetic type
    hist_offsets: np.ndarray        # int32 [U+1]
    cand_offsets: np.ndarray        # int32 [U+1]
    weights: np.ndarray             # float32 blob, blob order (see blob_layout)
    hist_emb: np.ndarray            # float32 [T, d]
    cand_emb: np.ndarray            # float32 [Kc, d]
    ln_eps: float = 1e-5

    @property
    def D(self) -> int:
        return self.d // self.H

    @property
    def U(self) -> int:
        return int(self.hist_offsets.shape[0] - 1)

    @property
    def hist_lens(self) -> np.ndarray:
        return np.diff(self.hist_offsets).astype(np.int64)

    @property
    def cand_lens(self) -> np.ndarray:
        return np.diff(self.cand_offsets).astype(np.int64)


def round_bf16(x: np.ndarray) -> np.ndarray:
    """Round float32 values to the nearest bf16 (ties to even), as float32."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) & 0xFFFF0000
    return u.astype(np.uint32).view(np.float32)


def blob_layout(d: int, L: int, F: int):
    """Entries of the weight blob in order: (name, shape, kind).

    kind is "mat" (Xavier-drawn), "gain" (LayerNorm gain), "vec" (bias or
    LayerNorm shift).  Linear weights use the [out, in] convention.
    """
    ent = []
    for l in range(L):
        p = f"l{l}."
        ent += [(p + "ln1_g", (d,), "gain"), (p + "ln1_b", (d,), "vec"),
                (p + "Wq", (d, d), "mat"), (p + "bq", (d,), "vec"),
                (p + "Wk", (d, d), "mat"), (p + "bk", (d,), "vec"),
                (p + "Wv", (d, d), "mat"), (p + "bv", (d,), "vec"),
                (p + "Wo", (d, d), "mat"), (p + "bo", (d,), "vec"),
                (p + "ln2_g", (d,), "gain"), (p + "ln2_b", (d,), "vec"),
                (p + "W1", (F, d), "mat"), (p + "b1", (F,), "vec"),
                (p + "W2", (d, F), "mat"), (p + "b2", (d,), "vec")]
    ent += [("lnf_g", (d,), "gain"), ("lnf_b", (d,), "vec"),
            ("w_score", (1, d), "mat"), ("b_score", (1,), "vec")]
    return ent


def blob_size(d: int, L: int, F: int) -> int:
    return sum(int(np.prod(s)) for _, s, _ in blob_layout(d, L, F))


def _draw_weights(rng, d, L, F, variant):
    parts = []
    for name, shape, kind in blob_layout(d, L, F):
        if kind == "mat":
            fan_out, fan_in = shape
            a = math.sqrt(6.0 / (fan_in + fan_out))
            w = rng.uniform(-a, a, size=shape)
            if variant == "sharp" and name.endswith("Wq"):
                w = w * 4.0
        elif variant == "base":
            w = np.ones(shape) if kind == "gain" else np.zeros(shape)
        else:
            w = rng.uniform(-0.1, 0.1, size=shape)
            if kind == "gain":
                w = 1.0 + w
        parts.append(np.asarray(w, dtype=np.float64).reshape(-1))
    return np.concatenate(parts).astype(np.float32)


def make_inputs(hist_lens, cand_lens, d, H, L, F, dtype="bf16", seed=0,
                variant="base", rng=None) -> Inputs:
    """Draw weights and tokens for explicit per-user lengths."""
    if variant not in VARIANTS:
        raise ValueError(f"unknown variant {variant!r}")
    if d % H:
        raise ValueError("d must be a multiple of H")
    rng = np.random.default_rng(seed) if rng is None else rng
    hist_lens = np.asarray(hist_lens, dtype=np.int64)
    cand_lens = np.asarray(cand_lens, dtype=np.int64)
    hoff = np.zeros(len(hist_lens) + 1, dtype=np.int64)
    coff = np.zeros(len(cand_lens) + 1, dtype=np.int64)
    hoff[1:] = np.cumsum(hist_lens)
    coff[1:] = np.cumsum(cand_lens)
    w = _draw_weights(rng, d, L, F, variant)
    T, Kc = int(hoff[-1]), int(coff[-1])
    X = (rng.standard_normal((T, d)) / math.sqrt(d)).astype(np.float32)
    C = (rng.standard_normal((Kc, d)) / math.sqrt(d)).astype(np.float32)
    if dtype == "bf16":
        w, X, C = round_bf16(w), round_bf16(X), round_bf16(C)
    elif dtype != "f32":
        raise ValueError(f"unknown dtype {dtype!r}")
    return Inputs(d=d, H=H, L=L, F=F, dtype=dtype,
                  hist_offsets=hoff.astype(np.int32), cand_offsets=coff.astype(np.int32),
                  weights=w, hist_emb=X, cand_emb=C)


def make_workload(name: str, seed: int = 0, variant: str = "base") -> Inputs:
    """Draw one of the named workloads."""
    spec = WORKLOADS[name]
    rng = np.random.default_rng(seed)
    U = spec["U"]
    if isinstance(spec["n"], tuple):
        lo, hi = spec["n"]
        n = rng.integers(lo, hi + 1, U)
        lo, hi = spec["k"]
        k = rng.integers(lo, hi + 1, U)
    else:
        n = np.full(U, spec["n"])
        k = np.full(U, spec["k"])
    return make_inputs(n, k, spec["d"], spec["H"], spec["L"], spec["F"],
                       dtype=spec["dtype"], variant=variant, rng=rng)


def workload_shape(name: str) -> dict:
    """The named workload's sizes, without drawing anything heavy."""
    spec = dict(WORKLOADS[name])
    if isinstance(spec["n"], tuple):
        rng = np.random.default_rng(0)
        U = spec["U"]
        spec["n_list"] = rng.integers(spec["n"][0], spec["n"][1] + 1, U)
        spec["k_list"] = rng.integers(spec["k"][0], spec["k"][1] + 1, U)
    else:
        spec["n_list"] = np.full(spec["U"], spec["n"])
        spec["k_list"] = np.full(spec["U"], spec["k"])
    return spec


# ----------------------------------------------------------------------------
# Per-action ranking heads (inputs only)
# ----------------------------------------------------------------------------

# Default action set of the heads workloads: C = 3 action types (for example
# save, click, hide) with utility weights that reward the first two and
# penalise the third; hidden width d/2.
DEFAULT_UTILITY = (1.0, 0.5, -2.0)


def heads_layout(d: int, C: int, Fh: int):
    """Entries of the heads blob in order: per head W1 [Fh, d], b1 [Fh],
    w2 [1, Fh] (stored flat), b2 [1]."""
    ent = []
    for c in range(C):
        p = f"h{c}."
        ent += [(p + "W1", (Fh, d), "mat"), (p + "b1", (Fh,), "vec"),
                (p + "w2", (1, Fh), "mat"), (p + "b2", (1,), "vec")]
    return ent


def make_heads(d: int, C: int = 3, Fh: int = None, dtype: str = "bf16", seed: int = 0,
               variant: str = "perturbed") -> np.ndarray:
    """Draw a heads blob (float32; bf16-rounded for bf16 models): Xavier-uniform
    matrices; biases 0 for ``base``, uniform +-0.1 otherwise."""
    Fh = d // 2 if Fh is None else Fh
    rng = np.random.default_rng(seed + 7919)
    parts = []
    for _, shape, kind in heads_layout(d, C, Fh):
        if kind == "mat":
            fan_out, fan_in = shape
            a = math.sqrt(6.0 / (fan_in + fan_out))
            w = rng.uniform(-a, a, size=shape)
        elif variant == "base":
            w = np.zeros(shape)
        else:
            w = rng.uniform(-0.1, 0.1, size=shape)
        parts.append(np.asarray(w, dtype=np.float64).reshape(-1))
    blob = np.concatenate(parts).astype(np.float32)
    return round_bf16(blob) if dtype == "bf16" else blob
