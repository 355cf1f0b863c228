"""MXFP8 projection variant (UPR_BF16_MXFP8) on the GPU vs the CPU oracle,
through the C ABI.

* Encoding is an integer decision: the device encoder and the oracle encode
  the same float32 / float16 / bfloat16 values, so codes and scale bytes are
  compared bit for bit.
* The scaled fp8 linear map runs on identical encoded operands and is
  compared with float64 products of the decoded values.  The matrix
  instruction sums the 64 products of one instruction in reduced precision
  (measured on gfx950: up to 1.4e-4 of the sum of |products|) and then
  accumulates in fp32, so |gpu - ref| <= 2.5e-4 (|A| |W|^T) + 1e-6.
* Scores of a UPR_BF16_MXFP8 model against oracle.rank(proj="mxfp8"): an
  envelope derived from the fp8 rule's own sensitivity (see MX_RMS below).
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2606_00422_amd import upr
from synth import make_inputs, make_workload
from tests.gpu_util import GpuRun, say

pytestmark = pytest.mark.gpu


def _encode_on_gpu(x_t):
    rows, k = x_t.shape
    codes = torch.full((rows, k), 0x55, dtype=torch.uint8, device="cuda")
    scales = torch.full((rows, k // 32), 0x55, dtype=torch.uint8, device="cuda")
    upr.upr_mx_quantize(x_t, codes, scales)
    torch.cuda.synchronize()
    return codes.cpu().numpy(), scales.cpu().numpy()


@pytest.mark.parametrize("dtype", ["float32", "float16", "bfloat16"])
@pytest.mark.parametrize("shape", [(1, 32), (7, 96), (33, 512), (5, 1056), (130, 2048)])
def test_device_encoding_matches_oracle_bit_for_bit(dtype, shape):
    rng = np.random.default_rng(1000 * ["float32", "float16", "bfloat16"].index(dtype) + shape[0] + shape[1])
    rows, k = shape
    x = rng.standard_normal((rows, k)) * np.exp2(rng.integers(-12, 12, (rows, 1)))
    if rows > 3:
        x[0, :32] = 0.0
        x[1, :32] = -0.0
        x[2, :32] *= 1e-3
        x[3, 3] = 460.0 * 2.0 ** 4                     # block top saturating after scaling
    xt = torch.from_numpy(x).to(getattr(torch, dtype))
    say(f"[gpu] mx encode {dtype} {shape}")
    codes, scales = _encode_on_gpu(xt.cuda())
    exact = xt.to(torch.float64).numpy()               # the values the GPU encodes
    oc, os_ = oracle.mx_quantize(exact)
    np.testing.assert_array_equal(scales, os_)
    np.testing.assert_array_equal(codes, oc)


@pytest.mark.parametrize("M,N,K", [(1, 8, 128), (257, 64, 256), (300, 512, 512), (513, 1536, 512),
                                   (260, 512, 2048)])
def test_scaled_fp8_linear_matches_decoded_products(M, N, K):
    rng = np.random.default_rng(M * 7 + N + K)
    a = rng.standard_normal((M, K)) * np.exp2(rng.integers(-4, 4, (M, 1)))
    w = rng.standard_normal((N, K)) * np.exp2(rng.integers(-4, 4, (N, 1))) / np.sqrt(K)
    ac, as_ = oracle.mx_quantize(a)
    wc, ws = oracle.mx_quantize(w)
    bias = rng.standard_normal(N).astype(np.float32)
    out0 = rng.standard_normal((M, N)).astype(np.float32)
    A = oracle.mx_dequantize(ac, as_)
    Wd = oracle.mx_dequantize(wc, ws)
    ref = out0.astype(np.float64) + A @ Wd.T + bias
    bound = 2.5e-4 * (np.abs(A) @ np.abs(Wd).T) + 1e-6 + 1e-6 * np.abs(out0)
    dev = lambda v: torch.from_numpy(np.ascontiguousarray(v)).cuda()
    out = dev(out0)
    say(f"[gpu] mx linear M={M} N={N} K={K}")
    upr.upr_mx_linear(dev(ac), dev(as_), dev(wc), dev(ws), dev(bias), out)
    torch.cuda.synchronize()
    err = np.abs(out.cpu().numpy().astype(np.float64) - ref)
    assert np.all(err <= bound), f"max err {err.max():.3e}, worst ratio {(err / bound).max():.2f}"


def _mx_scores(inp, users=None, cand_rows=None):
    cache = oracle.encode(inp.weights, inp.d, inp.H, inp.L, inp.F, inp.hist_emb, inp.hist_offsets,
                          users=users)
    return oracle.rank(inp.weights, inp.d, inp.H, inp.L, inp.F, cache, inp.hist_offsets,
                       inp.cand_emb, inp.cand_offsets, users=users, cand_rows=cand_rows, proj="mxfp8")


# (hist lens, cand lens, d, H, L, F)
CASES = [
    ([64, 200, 0], [100, 37, 5], 256, 4, 2, 512),
    ([300, 17], [129, 260], 256, 8, 1, 1024),            # head_dim 32: reference attention
    ([1000, 3], [513, 64], 512, 8, 2, 2048),
]

# Envelope for the MXFP8 scores.  The fp8 rounding is discontinuous: a value
# that moves by a relative 1e-3 (the order of the bf16 path's own rounding:
# bf16 queries, keys, values and probabilities, fp32 against float64) crosses
# an E4M3 rounding boundary for ~1-2% of the elements, each by a whole E4M3
# step (6-12% of the value), and later layers amplify the difference.  The
# oracle's own rule shows it (tests/test_mx_pins.py,
# test_mxfp8_rule_sensitivity): 1e-3 relative noise on its projection outputs
# moves the scores of these cases by rms 0.04-0.06 and at most 0.13-0.21.
# The GPU is held to that envelope with margin, and must follow the fp8 rule
# more closely than the rule follows the exact model (measured: 0.4-0.6 of
# the rule's own rms distance) while staying away from the exact scores.
MX_RMS, MX_MAX, MX_CORR = 0.1, 0.3, 0.98


def _check_mx_scores(g, rule, exact, label):
    rms = lambda v: float(np.sqrt(np.mean(v ** 2)))
    d_rule, d_exact, d_own = rms(g - rule), rms(g - exact), rms(rule - exact)
    err = np.abs(g - rule)
    corr = float(np.corrcoef(g, rule)[0, 1])
    say(f"[gpu]   {label}: rms(gpu-rule) {d_rule:.3e}, max {err.max():.3e}, rms(rule-exact) "
        f"{d_own:.3e}, rms(gpu-exact) {d_exact:.3e}, corr {corr:.5f}")
    assert np.all(np.isfinite(g))
    assert d_rule <= MX_RMS and err.max() <= MX_MAX and corr >= MX_CORR
    assert d_rule < 0.8 * d_own          # follows the fp8 rule ...
    assert d_exact > 0.5 * d_own         # ... and really quantizes


def test_mxfp8_rank_matches_oracle():
    for n, (hl, kl, d, H, L, F) in enumerate(CASES):
        inp = make_inputs(hl, kl, d, H, L, F, dtype="bf16", seed=400 + n, variant="perturbed")
        say(f"[gpu] mxfp8 rank case {n}: U={inp.U} Kc={inp.cand_offsets[-1]} d={d} H={H} L={L}")
        run = GpuRun(inp, model_dtype="bf16_mxfp8")
        run.encode()
        run.rank()
        g = run.scores_np()[: int(run.coff[-1])]
        rule = _mx_scores(inp)
        cache = oracle.encode(inp.weights, d, H, L, F, inp.hist_emb, inp.hist_offsets)
        exact = oracle.rank(inp.weights, d, H, L, F, cache, inp.hist_offsets, inp.cand_emb,
                            inp.cand_offsets)
        ok = ~np.isnan(rule)
        _check_mx_scores(g[ok], rule[ok], exact[ok], f"case {n}")


def test_mxfp8_headline_workload_sampled():
    inp = make_workload("u64_n1024_k2000", seed=0)
    say(f"[gpu] mxfp8 headline: U={inp.U} Kc={inp.cand_offsets[-1]}")
    run = GpuRun(inp, model_dtype="bf16_mxfp8")
    run.encode()
    run.rank()
    g = run.scores_np()
    rng = np.random.default_rng(78)
    users = sorted({0, inp.U - 1, int(rng.integers(inp.U))})
    rows = np.concatenate([rng.choice(np.arange(inp.cand_offsets[u], inp.cand_offsets[u + 1]), 16,
                                      replace=False) for u in users])
    o = _mx_scores(inp, users=users, cand_rows=rows)
    cache = oracle.encode(inp.weights, inp.d, inp.H, inp.L, inp.F, inp.hist_emb, inp.hist_offsets,
                          users=users)
    exact = oracle.rank(inp.weights, inp.d, inp.H, inp.L, inp.F, cache, inp.hist_offsets,
                        inp.cand_emb, inp.cand_offsets, users=users, cand_rows=rows)
    _check_mx_scores(g[rows], o[rows], exact[rows], "headline sample")
    assert np.all(np.isfinite(g[: int(run.coff[-1])]))


def test_mxfp8_action_heads_follow_the_rule():
    """Per-action heads on a UPR_BF16_MXFP8 model: the heads themselves keep
    the bf16 model's precision, so the probabilities move with the fp8
    hidden state only.  Held to the same relative envelope as the scores:
    closer to the oracle's fp8 rule than the rule is to the exact model,
    visibly away from the exact model, correlated; top-K is exact on the
    GPU's own utilities."""
    from synth import make_heads
    from tests.test_gpu_heads import _check_topk, _run_actions
    hl, kl, d, H, L, F = CASES[0]
    C, Fh = 3, 64
    inp = make_inputs(hl, kl, d, H, L, F, dtype="bf16", seed=410, variant="perturbed")
    hb = make_heads(d, C, Fh, dtype="bf16", seed=411, variant="perturbed")
    uw = np.array([1.0, 0.5, -2.0], dtype=np.float32)
    say(f"[gpu] mxfp8 heads: U={inp.U} Kc={inp.cand_offsets[-1]} d={d} C={C} Fh={Fh}")
    run = GpuRun(inp, model_dtype="bf16_mxfp8")
    run.encode()
    g_probs, g_util = _run_actions(run, hb, C, Fh, uw)
    _, final = oracle.unpack_weights(inp.weights, d, L, F)
    cache = oracle.encode(inp.weights, d, H, L, F, inp.hist_emb, inp.hist_offsets)

    def probs(proj):
        hid = oracle.rank_hidden(inp.weights, d, H, L, F, cache, inp.hist_offsets, inp.cand_emb,
                                 inp.cand_offsets, proj=proj)
        return oracle.sigmoid(oracle.action_logits(hid, final, hb, d, C, Fh))

    rule, exact = probs("mxfp8"), probs("exact")
    rows = int(inp.cand_offsets[-1])
    ok = ~np.isnan(rule[:rows]).any(axis=1)
    g, rule, exact = g_probs[:rows][ok].ravel(), rule[:rows][ok].ravel(), exact[:rows][ok].ravel()
    assert np.all(np.isfinite(g))
    rms = lambda v: float(np.sqrt(np.mean(v ** 2)))
    d_rule, d_exact, d_own = rms(g - rule), rms(g - exact), rms(rule - exact)
    corr = float(np.corrcoef(g, rule)[0, 1])
    say(f"[gpu]   rms(gpu-rule) {d_rule:.3e}, rms(rule-exact) {d_own:.3e}, rms(gpu-exact) {d_exact:.3e}, "
        f"corr {corr:.5f}, max {np.abs(g - rule).max():.3e}")
    assert d_rule < 0.8 * d_own and d_exact > 0.5 * d_own and corr >= MX_CORR
    assert np.abs(g - rule).max() <= 0.25 * MX_MAX      # sigmoid slope <= 1/4
    for K in (1, 5, 64):
        _check_topk(run, g_util[: max(rows, 1)], K)
