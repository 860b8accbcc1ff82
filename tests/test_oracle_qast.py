"""Pins for the oracle's QAST low-rank scale step (CPU only).

Pinned against: exact integer products (no rounding anywhere, so the rank-r
sum must equal an integer matrix product, catching a dropped term or a
transposed factor), an error bound against exact rational arithmetic, the
Delta=0 control (a zero factor leaves every scale byte unchanged), the NVFP4
ceiling clamp and its gradient mask (stability recipe (ii)-(iii)), the
paper's merge check max|dW| = 0 (the QAST forward's weights equal the merged
model's), and central finite differences of the loss through the
straight-through estimator for dB and dA."""

from fractions import Fraction

import numpy as np
import pytest
import torch

from oracle import codec, linear, merge, qast
from paper_2609_04526_amd import inputs


def bf16(x):
    return torch.from_numpy(np.asarray(x, dtype=np.float32)).to(torch.bfloat16)


def test_delta_s_equals_integer_product_when_nothing_rounds():
    g = np.random.default_rng(7)
    B = g.integers(-8, 9, size=(40, 16))
    A = g.integers(-8, 9, size=(16, 24))
    for c in (1.0, 2.0 ** -5):
        d = qast.delta_s(bf16(B), bf16(A), c)
        assert d.dtype == np.float32
        assert np.array_equal(d.astype(np.float64), (B @ A).astype(np.float64) * c)


def test_delta_s_within_fp32_sum_bound_of_exact():
    g = np.random.default_rng(8)
    B = bf16(g.standard_normal((12, 32)) * 0.02)
    A = bf16(g.standard_normal((32, 10)) * 0.02)
    c = 2.0
    d = qast.delta_s(B, A, c)
    b = B.float().numpy().astype(np.float64)
    a = A.float().numpy().astype(np.float64)
    for o in range(12):
        for j in range(10):
            exact = sum(Fraction(float(b[o, k])) * Fraction(float(a[k, j])) for k in range(32)) * Fraction(c)
            mag = sum(abs(b[o, k] * a[k, j]) for k in range(32)) * c
            # r sequential fp32 additions and one multiply: |err| <= (r+1) u sum|terms|
            assert abs(float(d[o, j]) - float(exact)) <= 33 * 2.0 ** -24 * mag + 1e-45


@pytest.mark.parametrize("fmt", ["mx", "nv"])
def test_zero_factor_leaves_every_byte(fmt):
    O, G, r = 64, 16, 8
    base = (inputs.e8m0_uniform_exponents(11, O, G, -8, -3) if fmt == "mx"
            else inputs.e4m3_abs_normal(11, O, G))
    ws2 = 1.0 if fmt == "mx" else float(np.float32(1 / 448))
    A = bf16(np.random.default_rng(1).standard_normal((r, G)))
    out, m = qast.qast_scales(fmt, base, bf16(np.zeros((O, r))), A, 1.0, ws2)
    assert np.array_equal(out, base)
    assert np.all(m == 1)


def test_nv_ceiling_clamp_and_mask():
    ws2 = float(np.float32(1 / 448))
    base = np.array([[0x7E, 0x70, 0x40, 0x30]], dtype=np.uint8)
    eff = codec.E4M3_TABLE[base] * ws2
    cap = float(np.float32(448) * np.float32(ws2))
    # one rank: B = 1, A chosen so eff' = [2 cap, cap + tiny, exactly cap, below cap]
    target = np.array([[2 * cap, cap * 1.01, cap, eff[0, 3] * 1.5]])
    A = (target - eff).astype(np.float32)
    Ab = bf16(A)
    d = qast.delta_s(bf16([[1.0]]), Ab, 1.0)
    out, m = qast.qast_scales("nv", base, bf16([[1.0]]), Ab, 1.0, ws2)
    e2 = (codec.E4M3_TABLE[base].astype(np.float32) * np.float32(ws2)) + d
    over = e2 > np.float32(cap)
    assert np.all(out[over] == 0x7E) and np.all(m[over] == 0)
    assert np.all(m[~over] == 1)
    assert over[0, 0] and not over[0, 3]


@pytest.mark.parametrize("fmt", ["mx", "nv"])
def test_qast_forward_weights_equal_merged_weights(fmt):
    """The paper's merge check: max |W_trained - W_merged| = 0."""
    O, I, r = 32, 128, 4
    G = I // codec.BLOCK[fmt]
    codes = inputs.codes_uniform(21, O, I)
    base = (inputs.e8m0_uniform_exponents(22, O, G, -8, -3) if fmt == "mx"
            else inputs.e4m3_abs_normal(22, O, G))
    ws2 = 1.0 if fmt == "mx" else float(np.float32(1 / 448))
    eff = codec.effective_scales(fmt, base, ws2)
    g = np.random.default_rng(23)
    B = bf16(g.standard_normal((O, r)) * 0.3)
    A = bf16(g.standard_normal((r, G)) * float(np.median(np.abs(eff))))
    trained, _ = qast.qast_scales(fmt, base, B, A, 1.0, ws2)
    merged = merge.merge_delta(fmt, base, qast.delta_s(B, A, 1.0), ws2)
    assert np.array_equal(trained, merged)
    w_t = linear.dequant(fmt, codes, trained, ws2)
    w_m = linear.dequant(fmt, codes, merged, ws2)
    assert np.max(np.abs(w_t - w_m)) == 0.0
    assert np.any(trained != base)                       # the adapter did move scales


def test_factor_grads_match_finite_differences():
    """L(B, A) = sum (dS * m) * (c B A) is bilinear: central differences are exact."""
    g = np.random.default_rng(31)
    O, G, r, c = 6, 5, 3, 0.5
    dS = g.standard_normal((O, G))
    m = (g.random((O, G)) > 0.3).astype(np.uint8)
    B = bf16(g.standard_normal((O, r)))
    A = bf16(g.standard_normal((r, G)))
    dB, dA = qast.factor_grads(dS, m, B, A, c)
    b = B.float().numpy().astype(np.float64)
    a = A.float().numpy().astype(np.float64)

    def loss(bb, aa):
        return float(np.sum(dS * m * (c * (bb @ aa))))

    h = 0.25
    for o in range(O):
        for k in range(r):
            e = np.zeros_like(b); e[o, k] = h
            assert abs((loss(b + e, a) - loss(b - e, a)) / (2 * h) - dB[o, k]) < 1e-12
    for k in range(r):
        for j in range(G):
            e = np.zeros_like(a); e[k, j] = h
            assert abs((loss(b, a + e) - loss(b, a - e)) / (2 * h) - dA[k, j]) < 1e-12


def test_chain_rule_through_the_layer():
    """With the STE the forward's rounding is the identity for the gradient:
    d<dY, Y(eff + c B A)>/dB must equal factor_grads(backward_dscale(...))."""
    g = np.random.default_rng(41)
    fmt, T, O, I, r, c = "mx", 5, 8, 64, 2, 0.25
    G = I // 32
    codes = inputs.codes_uniform(42, O, I)
    base = inputs.e8m0_uniform_exponents(43, O, G, -4, -1)
    eff = codec.effective_scales(fmt, base, 1.0)
    X = g.standard_normal((T, I))
    dY = g.standard_normal((T, O))
    B = bf16(g.standard_normal((O, r)))
    A = bf16(g.standard_normal((r, G)) * 0.1)
    b = B.float().numpy().astype(np.float64)
    a = A.float().numpy().astype(np.float64)
    vals = codec.E2M1_TABLE[codec.unpack_nibbles(codes)]

    def loss(bb, aa):
        effp = eff + c * (bb @ aa)
        W = vals * np.repeat(effp, 32, axis=1)
        return float(np.sum(dY * (X @ W.T)))

    dS = linear.backward_dscale(fmt, X, dY, codes)
    dB, dA = qast.factor_grads(dS, np.ones((O, G), np.uint8), B, A, c)
    h = 0.5
    for o in range(O):
        for k in range(r):
            e = np.zeros_like(b); e[o, k] = h
            fd = (loss(b + e, a) - loss(b - e, a)) / (2 * h)
            assert abs(fd - dB[o, k]) <= 1e-9 * (1 + abs(fd))
    for k in range(r):
        for j in range(G):
            e = np.zeros_like(a); e[k, j] = h
            fd = (loss(b, a + e) - loss(b, a - e)) / (2 * h)
            assert abs(fd - dA[k, j]) <= 1e-9 * (1 + abs(fd))
