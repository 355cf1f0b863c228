"""Pins for the MXFP8 oracle (oracle/upr_mx.py) that do not reuse its code:
torch's float8_e4m3fn and bfloat16 conversions (library rounding routines),
the E4M3 format definition, and closed forms of the MX block scale."""
import numpy as np
import pytest
import torch

import oracle.upr_mx as mx_oracle

RNG = np.random.default_rng(2024)


def _f32(x):
    """Values exactly representable in float32: torch casts float64 to fp8
    through float32, which would round a second time."""
    return np.asarray(x, dtype=np.float32).astype(np.float64)


def _torch_codes(x):
    return torch.tensor(np.asarray(x, dtype=np.float64)).to(torch.float8_e4m3fn).view(torch.uint8).numpy()


def test_e4m3_values_of_all_codes():
    m = mx_oracle
    codes = np.arange(256, dtype=np.uint8)
    ours = m.e4m3_value(codes)
    ref = torch.from_numpy(codes).view(torch.float8_e4m3fn).to(torch.float64).numpy()
    np.testing.assert_array_equal(np.isnan(ours), np.isnan(ref))
    ok = ~np.isnan(ref)
    np.testing.assert_array_equal(ours[ok], ref[ok])
    # format landmarks: largest normal, smallest normal, smallest subnormal
    assert m.e4m3_value(0x7E) == 448.0 and m.e4m3_value(0x08) == 2.0 ** -6
    assert m.e4m3_value(0x01) == 2.0 ** -9 and np.isnan(m.e4m3_value(0x7F))


def test_e4m3_rounding_matches_torch_in_range():
    m = mx_oracle
    grid = m.e4m3_value(np.arange(0x7F))
    mids = (grid[1:] + grid[:-1]) / 2
    x = _f32(np.concatenate([RNG.uniform(-448, 448, 20000), RNG.uniform(-0.05, 0.05, 20000),
                             grid, -grid, mids, -mids, [0.0, -0.0, 464.0, -464.0]]))
    np.testing.assert_array_equal(m.e4m3_round_codes(x), _torch_codes(x))


def test_e4m3_saturates_above_448():
    m = mx_oracle
    x = np.array([448.0, 464.0, 464.5, 480.0, 511.9, 1e6, -470.0, -1e6])
    np.testing.assert_array_equal(m.e4m3_round_codes(x),
                                  [0x7E, 0x7E, 0x7E, 0x7E, 0x7E, 0x7E, 0xFE, 0xFE])


@pytest.mark.parametrize("amax,e", [(1.0, -8), (448.0, 0), (256.0, 0), (511.99, 0), (512.0, 1),
                                    (0.75, -9), (2.0 ** -120, -127), (2.0 ** -140, -127),
                                    (0.0, -127), (2.0 ** 200, 127), (3.0 * 2.0 ** 100, 93)])
def test_block_exponent_closed_forms(amax, e):
    assert int(mx_oracle.mx_block_exponent(amax)) == e


def test_block_scale_puts_the_maximum_in_256_512():
    m = mx_oracle
    x = RNG.standard_normal((64, 128)) * np.exp2(RNG.integers(-20, 20, (64, 1)))
    codes, scales = m.mx_quantize(x)
    assert codes.shape == x.shape and scales.shape == (64, 4)
    e = scales.astype(np.int64) - 127
    amax = np.abs(x).reshape(64, 4, 32).max(axis=-1)
    r = amax / np.exp2(e)
    assert np.all((r >= 256) & (r < 512))


def test_representable_blocks_round_trip_exactly():
    """A block built as E4M3 values times 2^e, whose largest value lies in
    [256, 448], is its own MXFP8 encoding."""
    m = mx_oracle
    grid = m.e4m3_value(np.arange(0x7F))
    top = grid[grid >= 256]
    rows = []
    for _ in range(50):
        e = int(RNG.integers(-30, 30))
        v = RNG.choice(grid, 32) * RNG.choice([-1.0, 1.0], 32)
        v[RNG.integers(32)] = RNG.choice(top)
        rows.append(v * 2.0 ** e)
    x = np.array(rows)
    np.testing.assert_array_equal(m.mx_round(x), x)


def test_error_within_half_an_element_ulp():
    m = mx_oracle
    x = RNG.standard_normal((200, 64)) * np.exp2(RNG.integers(-8, 8, (200, 1)))
    codes, scales = m.mx_quantize(x)
    X = np.repeat(np.exp2(scales.astype(np.float64) - 127), 32, axis=1)
    s = np.abs(x) / X
    ulp = np.where(s >= 2.0 ** -6, np.exp2(np.floor(np.log2(np.maximum(s, 2.0 ** -6))) - 3), 2.0 ** -9)
    sat = np.maximum(s - 448.0, 0.0)
    err = np.abs(m.mx_round(x) - x) / X
    assert np.all(err <= ulp / 2 + sat + 1e-12)
    assert np.any(sat > 0)            # the saturated top of some block is exercised


def test_all_zero_and_mixed_sign_blocks():
    m = mx_oracle
    z = np.zeros((2, 32))
    z[1, 5] = -0.0
    codes, scales = m.mx_quantize(z)
    assert np.all(scales == 0) and codes[1, 5] == 0x80 and np.all(np.delete(codes[1], 5) == 0)
    x = np.zeros(32)
    x[0], x[1] = 300.0, -2.0 ** -20          # far below the block's range: -0
    c, s = m.mx_quantize(x)
    assert s[0] == 127 and c[0] == m.e4m3_round_codes(300.0) and c[1] == 0x80


def test_linear_mx_matches_torch_fp8_when_every_scale_is_one():
    """Blocks whose largest magnitude is 300 take scale 2^0, so the MXFP8
    values are plain E4M3 roundings: torch's float8_e4m3fn cast gives the
    operands independently."""
    m = mx_oracle

    def scale_one(rows, k):
        v = RNG.uniform(-299.0, 299.0, (rows, k))
        for c in range(0, k, 32):
            v[np.arange(rows), c + RNG.integers(0, 32, rows)] = 300.0 * RNG.choice([-1.0, 1.0], rows)
        return _f32(v)

    def fp8(v):
        return torch.tensor(v).to(torch.float8_e4m3fn).to(torch.float64).numpy()

    x, W, b = scale_one(6, 64), scale_one(10, 64), RNG.standard_normal(10)
    np.testing.assert_allclose(m.linear_mx(x, W, b), fp8(x) @ fp8(W).T + b, rtol=1e-13, atol=1e-9)


def test_linear_mx_on_representable_operands_is_exact():
    m = mx_oracle
    xr = m.mx_round(RNG.standard_normal((8, 64)))
    Wr = m.mx_round(RNG.standard_normal((16, 64)))
    b = RNG.standard_normal(16)
    np.testing.assert_array_equal(m.linear_mx(xr, Wr, b), xr @ Wr.T + b)
    # and on general operands it is not the plain product
    x = RNG.standard_normal((8, 64))
    assert not np.allclose(m.linear_mx(x, Wr, b), x @ Wr.T + b, rtol=1e-4, atol=0)


# ---------------------------------------------------------------------------
# The MXFP8 projection rule inside the ranking pass
# ---------------------------------------------------------------------------

def _mx_scores(inp, cand_emb=None, cand_offsets=None, proj="mxfp8"):
    import oracle
    cache = oracle.encode(inp.weights, inp.d, inp.H, inp.L, inp.F, inp.hist_emb, inp.hist_offsets)
    return oracle.rank(inp.weights, inp.d, inp.H, inp.L, inp.F, cache, inp.hist_offsets,
                       inp.cand_emb if cand_emb is None else cand_emb,
                       inp.cand_offsets if cand_offsets is None else cand_offsets, proj=proj)


def test_mxfp8_rank_is_per_candidate():
    """Blocks run along each row's contraction axis, so a candidate's score
    does not depend on which other candidates share the call (a block taken
    across rows would break this)."""
    from synth import make_inputs
    inp = make_inputs([9, 4], [10, 6], d=64, H=2, L=2, F=128, dtype="bf16", seed=21)
    base = _mx_scores(inp)
    perm = np.concatenate([np.random.default_rng(0).permutation(10), 10 + np.arange(6)[::-1]])
    np.testing.assert_allclose(_mx_scores(inp, cand_emb=inp.cand_emb[perm]), base[perm],
                               rtol=1e-12, atol=1e-12)
    for c in [0, 7]:
        alone = _mx_scores(inp, cand_emb=inp.cand_emb[c:c + 1],
                           cand_offsets=np.array([0, 1, 1], np.int32))
        np.testing.assert_allclose(alone[0], base[c], rtol=1e-12, atol=1e-12)


def test_mxfp8_rank_stays_near_the_exact_model():
    """fp8 elements carry 3 mantissa bits (up to 2^-4 relative error per
    element, ~2.4% rms), compounded over 8 projections: the scores move by a
    few percent of their spread (measured 6-12%), keep their order almost
    everywhere (correlation >= 0.99 measured), and do move."""
    from synth import make_inputs
    inp = make_inputs([40, 17], [30, 25], d=64, H=2, L=2, F=128, dtype="bf16", seed=22)
    exact = _mx_scores(inp, proj="exact")
    mx = _mx_scores(inp)
    diff = mx - exact
    assert np.abs(diff).max() > 1e-4
    assert np.sqrt(np.mean(diff ** 2)) <= 0.25 * np.std(exact)
    assert np.corrcoef(exact, mx)[0, 1] >= 0.98


def test_mxfp8_rule_sensitivity():
    """The envelope the GPU's fp8 scores are held to (tests/test_gpu_mx.py):
    1e-3 relative noise on every projection output of the oracle's fp8 rule
    moves the scores by rms <= 0.07 and at most 0.25 on these workloads,
    because E4M3 rounding is discontinuous (a few percent of the values cross
    a rounding boundary by a whole step); the same noise moves the exact
    model's scores by an order of magnitude less (measured: 4%)."""
    import oracle
    import oracle.upr_oracle as uo
    from synth import make_inputs
    rms = lambda v: float(np.sqrt(np.mean(v ** 2)))
    m = mx_oracle
    for n, (hl, kl, d, H, L, F) in enumerate([([64, 200, 0], [100, 37, 5], 256, 4, 2, 512),
                                               ([300, 17], [129, 260], 256, 8, 1, 1024)]):
        inp = make_inputs(hl, kl, d, H, L, F, dtype="bf16", seed=400 + n, variant="perturbed")
        cache = oracle.encode(inp.weights, d, H, L, F, inp.hist_emb, inp.hist_offsets)
        args = (inp.weights, d, H, L, F, cache, inp.hist_offsets, inp.cand_emb, inp.cand_offsets)
        base = oracle.rank(*args, proj="mxfp8")
        exact = oracle.rank(*args)
        rng = np.random.default_rng(n)
        noisy = lambda x, W, b, f: f(x, W, b) * (1 + 1e-3 * rng.standard_normal((x.shape[0], W.shape[0])))
        real = uo._projection_rule
        try:
            uo._projection_rule = lambda proj: (lambda x, W, b: noisy(x, W, b, m.linear_mx))
            moved = oracle.rank(*args, proj="mxfp8")
            uo._projection_rule = lambda proj: (lambda x, W, b: noisy(x, W, b, uo.linear))
            moved_exact = oracle.rank(*args)
        finally:
            uo._projection_rule = real
        assert rms(moved - base) <= 0.07 and np.abs(moved - base).max() <= 0.25
        assert rms(moved - base) > 5e-3                       # it does move: the rounding is discontinuous
        assert rms(moved_exact - exact) < 0.1 * rms(moved - base)


# ---------------------------------------------------------------------------
# The composition, rebuilt from torch operations
# ---------------------------------------------------------------------------

def _torch_e4m3_round(s):
    """s rounded to E4M3 values, written independently of the oracle: three
    fraction bits by the add-and-subtract method in float64 (adding
    c = 1.5 * 2^(49 + e) puts the sum's last significand bit at 2^(e - 3),
    and float64 addition rounds to nearest, ties to even), exponents below
    -6 sharing the subnormal step 2^-9, magnitudes saturated at 448."""
    a = s.abs()
    _, ex = torch.frexp(a)                        # a = m 2^ex, m in [0.5, 1)
    e = torch.clamp(ex - 1, min=-6).to(torch.float64)
    c = 1.5 * torch.exp2(e + 49.0)
    r = torch.clamp((a + c) - c, max=448.0)
    return torch.copysign(r, s)


def _torch_mx_round(x):
    """x replaced by its MXFP8 values along the last axis: blocks of 32, scale
    2^(floor(log2 max|v|) - 8) (2^-127 for an all-zero block), from
    torch.frexp."""
    K = x.shape[-1]
    b = x.reshape(*x.shape[:-1], K // 32, 32)
    amax = b.abs().amax(dim=-1)
    _, ex = torch.frexp(amax)
    e = torch.where(amax > 0, ex - 9, torch.full_like(ex, -127)).clamp(-127, 127)
    sc = torch.exp2(e.to(torch.float64))[..., None]
    return (_torch_e4m3_round(b / sc) * sc).reshape(x.shape)


def _torch_mx_rank(inp, cache):
    """One candidate pass of the fp8 projection rule from torch.nn.functional
    pieces: LayerNorm, tanh GELU and softmax from torch, every projection
    input and weight through _torch_mx_round, attention over the cached
    history plus the candidate's own key; float64 elsewhere."""
    import torch.nn.functional as Fn
    from synth import blob_layout
    d, H, L, Fd = inp.d, inp.H, inp.L, inp.F
    D = d // H
    w, pos = {}, 0
    blob = torch.as_tensor(np.asarray(inp.weights, dtype=np.float64))
    for name, shape, _ in blob_layout(d, L, Fd):
        n = int(np.prod(shape))
        w[name] = blob[pos:pos + n].reshape(shape)
        pos += n
    lin = lambda x, W, b: _torch_mx_round(x) @ _torch_mx_round(W).T + b
    kv = torch.as_tensor(np.asarray(cache, dtype=np.float64))
    Cm = torch.as_tensor(np.asarray(inp.cand_emb, dtype=np.float64))
    ho, co = inp.hist_offsets, inp.cand_offsets
    out = torch.full((Cm.shape[0],), float("nan"), dtype=torch.float64)
    for u in range(inp.U):
        g = Cm[co[u]:co[u + 1]]
        if g.shape[0] == 0:
            continue
        lo, hi = int(ho[u]), int(ho[u + 1])
        for l in range(L):
            p = f"l{l}."
            a = Fn.layer_norm(g, (d,), w[p + "ln1_g"], w[p + "ln1_b"], eps=1e-5)
            q, k, v = (lin(a, w[p + "W" + t], w[p + "b" + t]) for t in "qkv")
            heads = []
            for j in range(H):
                sl = slice(j * D, (j + 1) * D)
                Kh, Vh = kv[l, 0, j, lo:hi], kv[l, 1, j, lo:hi]
                logits = torch.cat([q[:, sl] @ Kh.T, (q[:, sl] * k[:, sl]).sum(-1, keepdim=True)], 1)
                pr = torch.softmax(logits / np.sqrt(D), dim=-1)
                heads.append(pr[:, :-1] @ Vh + pr[:, -1:] * v[:, sl])
            g = g + lin(torch.cat(heads, 1), w[p + "Wo"], w[p + "bo"])
            a2 = Fn.layer_norm(g, (d,), w[p + "ln2_g"], w[p + "ln2_b"], eps=1e-5)
            g = g + lin(Fn.gelu(lin(a2, w[p + "W1"], w[p + "b1"]), approximate="tanh"),
                        w[p + "W2"], w[p + "b2"])
        z = Fn.layer_norm(g, (d,), w["lnf_g"], w["lnf_b"], eps=1e-5)
        out[co[u]:co[u + 1]] = z @ w["w_score"].reshape(-1) + w["b_score"].reshape(())
    return out.numpy()


def test_torch_e4m3_rounding_agrees_with_torch_cast():
    """The independent rounding above against torch's own float8_e4m3fn cast
    on float32-representable values (no double rounding there), saturation
    aside."""
    x = _f32(np.concatenate([RNG.uniform(-448, 448, 20000), RNG.uniform(-0.05, 0.05, 20000)]))
    ours = _torch_e4m3_round(torch.as_tensor(x)).numpy()
    ref = torch.tensor(x).to(torch.float8_e4m3fn).to(torch.float64).numpy()
    np.testing.assert_array_equal(ours, ref)


def test_mxfp8_rank_matches_an_independent_composition():
    """oracle.rank(proj="mxfp8") against the same forward pass assembled
    from torch operations with an independently written MX rounding: every
    quantization point (LN1 output, attention output, LN2 output, GELU
    output, each weight), its axis and block and nothing else rounded.  Both
    sides are float64 away from the E4M3 points, so they agree to rounding
    order."""
    import oracle
    from synth import make_inputs
    inp = make_inputs([37, 0, 70], [29, 6, 41], d=64, H=2, L=2, F=128, dtype="bf16", seed=23,
                      variant="perturbed")
    cache = oracle.encode(inp.weights, inp.d, inp.H, inp.L, inp.F, inp.hist_emb, inp.hist_offsets)
    ref = _torch_mx_rank(inp, cache)
    got = oracle.rank(inp.weights, inp.d, inp.H, inp.L, inp.F, cache, inp.hist_offsets,
                      inp.cand_emb, inp.cand_offsets, proj="mxfp8")
    np.testing.assert_allclose(got, ref, rtol=1e-9, atol=1e-9)
    exact = oracle.rank(inp.weights, inp.d, inp.H, inp.L, inp.F, cache, inp.hist_offsets,
                        inp.cand_emb, inp.cand_offsets)
    assert np.abs(got - exact).max() > 1e-3          # the quantization is really there
