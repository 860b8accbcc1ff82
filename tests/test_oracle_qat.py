"""Pins for the QAT-LoRA weight-space STE oracle (CPU only).

Pinned against: a dyadic case where every step is exact, compared with the
fp64 product B @ A (orientation of B and A, the alpha/r factor, the base
weight); the fixed point B = 0 (re-quantisation returns the base codes and
scales); bf16 rounding against torch's own fp32 -> bf16 conversion; finite
differences of the bilinear loss sum(G * X W(B, A)^T), which fix dB and dA
without the oracle's formula; and the low-rank association
dB = c dY^T (X A^T), dA = c (dY B)^T X."""

import numpy as np
import pytest
import torch

from oracle import codec, linear, qat
from paper_2609_04526_amd import inputs


def test_bf16_round_matches_torch():
    g = np.random.default_rng(1)
    x = np.concatenate([g.standard_normal(100000).astype(np.float32) * np.float32(3.0),
                        np.array([np.inf, -np.inf, 3.3895314e38, -0.0, 1e-40, 3.4e38], np.float32)])
    want = torch.from_numpy(x).to(torch.bfloat16).float().numpy()
    assert np.array_equal(qat.bf16_round(x), want)
    assert np.isnan(qat.bf16_round(np.array([np.nan], np.float32)))[0]


def test_exact_dyadic_case():
    """Entries of B, A in {-1, 0, 1}/8, r = 4, alpha/r = 1/2: S, Delta and the
    sum with the base are exact in fp32 and bf16, so W_eff = base + c B @ A."""
    O, I, r = 16, 64, 4
    g = np.random.default_rng(2)
    B = g.integers(-1, 2, size=(O, r)).astype(np.float32) / 8
    A = g.integers(-1, 2, size=(r, I)).astype(np.float32) / 8
    codes = inputs.codes_uniform(3, O, I)
    sb = np.full((O, I // 32), 127 - 3, np.uint8)            # scale 2^-3
    W = qat.effective_weight("mx", codes, sb, 1.0, B, A, 0.5)
    want = linear.dequant("mx", codes, sb) + 0.5 * (B.astype(np.float64) @ A.astype(np.float64))
    assert np.count_nonzero(B @ A) > O * I // 4
    assert np.array_equal(W.astype(np.float64), want)


@pytest.mark.parametrize("fmt", ["mx", "nv"])
def test_zero_adapter_is_a_fixed_point(fmt):
    """B = 0: every block of the base holds a magnitude-6 code, so the nearest
    rule re-derives the same scale and the same codes, except that a -0 code
    comes back as +0 (the fp32 sum -0 + +0 is +0)."""
    O, I, r = 32, 256, 8
    codes = inputs.codes_uniform(10, O, I)
    nib = codec.unpack_nibbles(codes)
    block = codec.BLOCK[fmt]
    nib[:, ::block] = 7
    codes = codec.pack_nibbles(nib)
    if fmt == "mx":
        sb, ws2 = inputs.e8m0_uniform_exponents(11, O, I // block, -8, -3), 1.0
    else:
        sb, ws2 = inputs.e4m3_abs_normal(11, O, I // block), 2.0 ** -9      # ws2 a power of two: exact
        sb = np.where((sb & 0x7F) == 0, np.uint8(0x38), sb)    # a zero scale re-derives zero codes
    B = np.zeros((O, r), np.float32)
    A = inputs.rng(12).standard_normal((r, I)).astype(np.float32)
    c2, s2 = qat.requant(fmt, codes, sb, ws2, B, A, 2.0)
    want = codec.pack_nibbles(np.where(nib == 8, 0, nib).astype(np.uint8))
    assert np.any(nib == 8)
    assert np.array_equal(s2, sb) and np.array_equal(c2, want)


def test_finite_differences_fix_the_factor_gradients():
    """L(B, A) = sum(G * X W^T) with W = base + c B A is linear in B and in A
    separately, so a one-entry step gives the exact partial derivative."""
    T, O, I, r = 6, 8, 32, 3
    g = np.random.default_rng(4)
    X = g.standard_normal((T, I))
    G = g.standard_normal((T, O))
    B = g.standard_normal((O, r))
    A = g.standard_normal((r, I))
    base = g.standard_normal((O, I))
    c = 0.75

    def loss(B_, A_):
        return float(np.sum(G * (X @ (base + c * B_ @ A_).T)))

    dB, dA = qat.lora_grads(X.astype(np.float32), G.astype(np.float32), B.astype(np.float32),
                            A.astype(np.float32), c)
    Xf, Gf = X.astype(np.float32).astype(np.float64), G.astype(np.float32).astype(np.float64)
    Bf, Af = B.astype(np.float32).astype(np.float64), A.astype(np.float32).astype(np.float64)

    def loss_f(B_, A_):
        return float(np.sum(Gf * (Xf @ (base + c * B_ @ A_).T)))

    for (o, k) in [(0, 0), (7, 2), (3, 1)]:
        E = np.zeros_like(Bf)
        E[o, k] = 1.0
        assert abs((loss_f(Bf + E, Af) - loss_f(Bf, Af)) - dB[o, k]) < 1e-9 * max(1.0, abs(dB[o, k]))
    for (k, i) in [(0, 0), (2, 31), (1, 17)]:
        E = np.zeros_like(Af)
        E[k, i] = 1.0
        assert abs((loss_f(Bf, Af + E) - loss_f(Bf, Af)) - dA[k, i]) < 1e-9 * max(1.0, abs(dA[k, i]))


def test_low_rank_association():
    T, O, I, r = 40, 24, 64, 5
    g = np.random.default_rng(5)
    X, dY = g.standard_normal((T, I)).astype(np.float32), g.standard_normal((T, O)).astype(np.float32)
    B, A = g.standard_normal((O, r)).astype(np.float32), g.standard_normal((r, I)).astype(np.float32)
    dB, dA = qat.lora_grads(X, dY, B, A, 0.5)
    X64, dY64, B64, A64 = (v.astype(np.float64) for v in (X, dY, B, A))
    assert np.allclose(dB, 0.5 * dY64.T @ (X64 @ A64.T), rtol=1e-12, atol=1e-12)
    assert np.allclose(dA, 0.5 * (dY64 @ B64).T @ X64, rtol=1e-12, atol=1e-12)


def test_sampled_gradients_equal_the_full_ones():
    T, O, I, r = 30, 16, 48, 3
    g = np.random.default_rng(6)
    X, dY = g.standard_normal((T, I)).astype(np.float32), g.standard_normal((T, O)).astype(np.float32)
    B, A = g.standard_normal((O, r)).astype(np.float32), g.standard_normal((r, I)).astype(np.float32)
    dB, dA = qat.lora_grads(X, dY, B, A, 0.25)
    rows, cols = np.array([0, 5, 15]), np.array([1, 47, 20])
    sB, sA = qat.lora_grads_sampled(X, dY, B, A, 0.25, rows, cols)
    assert np.allclose(sB, dB[rows], rtol=1e-12, atol=1e-12)
    assert np.allclose(sA, dA[:, cols], rtol=1e-12, atol=1e-12)
