"""The per-element acceptance bound of the GEMM parity tests, checked on the
CPU: an fp32 evaluation of the products passes it, and a single corrupted
element (a neighbour's value, a dropped 64-deep K stage, a zero, a NaN)
fails it, where on an output of 8B size the normwise error would stay far
below 2e-3."""

import numpy as np

from oracle import linear
from paper_2609_04526_amd import inputs
from parity_check import check_elements

T, O, I = 64, 256, 512


def _layer():
    X = inputs.bf16_normal(1000, (T, I)).float().numpy()
    dY = inputs.bf16_normal(1001, (T, O)).float().numpy()
    codes = inputs.codes_uniform(1002, O, I)
    sb = inputs.e8m0_uniform_exponents(1003, O, I // 32, -8, -3)
    return X, dY, codes, sb


def _normwise(got, ref):
    return float(np.linalg.norm(got - ref) / np.linalg.norm(ref))


def test_fp32_products_pass_the_bound():
    X, dY, codes, sb = _layer()
    W = linear.dequant("mx", codes, sb)
    W32 = W.astype(np.float32)                       # exact: code * 2^e
    Y = X @ W32.T
    dX = dY @ W32
    dW32 = dY.T @ X
    c = linear.code_values(codes).astype(np.float32)
    dS = (c * dW32).reshape(O, I // 32, 32).sum(axis=2, dtype=np.float32)
    Xd, dYd = X.astype(np.float64), dY.astype(np.float64)
    aW, aX, adY = np.abs(W), np.abs(Xd), np.abs(dYd)
    assert check_elements(Y, linear.forward(Xd, W), aX @ aW.T, I).size == 0
    assert check_elements(dX, linear.backward_dx(dYd, W), adY @ aW, O).size == 0
    absdS = (np.abs(linear.code_values(codes)) * (adY.T @ aX)).reshape(O, I // 32, 32).sum(axis=2)
    assert check_elements(dS, linear.backward_dscale("mx", Xd, dYd, codes), absdS, T + 32 + 2).size == 0


def test_one_corrupted_element_fails_the_bound_but_not_the_norm():
    X, dY, codes, sb = _layer()
    W = linear.dequant("mx", codes, sb)
    Xd = X.astype(np.float64)
    ref = linear.forward(Xd, W)
    absref = np.abs(Xd) @ np.abs(W).T
    good = (X @ W.astype(np.float32).T).astype(np.float64)

    # a neighbour's value in one element
    d = np.abs(ref[:, :-1] - ref[:, 1:])
    t, o = np.unravel_index(np.argmax(d), d.shape)
    bad = good.copy()
    bad[t, o] = good[t, o + 1]
    assert [tuple(x) for x in check_elements(bad, ref, absref, I)] == [(t, o)]

    # one element missing one 64-deep K stage
    stage = Xd[:, 64:128] @ W[:, 64:128].T
    t, o = np.unravel_index(np.argmax(np.abs(stage)), stage.shape)
    bad = good.copy()
    bad[t, o] -= stage[t, o]
    # the same error in one element of a 4096-token 14336-wide output with
    # this RMS moves the normwise error by far less than 2e-3
    rms = float(np.sqrt(np.mean(ref ** 2)))
    assert abs(stage[t, o]) / (rms * np.sqrt(4096 * 14336)) < 2e-3 < _normwise(bad, ref)
    assert [tuple(x) for x in check_elements(bad, ref, absref, I)] == [(t, o)]

    # one element zeroed
    t, o = np.unravel_index(np.argmax(np.abs(ref)), ref.shape)
    bad = good.copy()
    bad[t, o] = 0.0
    assert [tuple(x) for x in check_elements(bad, ref, absref, I)] == [(t, o)]

    # NaN never passes
    bad = good.copy()
    bad[0, 0] = np.nan
    assert [tuple(x) for x in check_elements(bad, ref, absref, I)] == [(0, 0)]
