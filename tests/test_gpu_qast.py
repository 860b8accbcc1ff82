"""GPU parity of the QAST low-rank scale step against the oracle.

Scale bytes and clamp masks are integers decided by fp32 arithmetic that both
sides perform in the same order, so they must match bit for bit; the factor
gradients are fp32 sums compared with the fp64 oracle (normwise relative error
<= 1e-5, far inside the 2e-3 bar, since each is a short fp32 dot product)."""

import numpy as np
import pytest
import torch

from conftest import ensure_library, gpu_ready
from oracle import codec, linear, qast
from paper_2609_04526_amd import inputs

pytestmark = [pytest.mark.gpu, pytest.mark.skipif(not gpu_ready(), reason="needs a GPU")]

TOL = 1e-5


@pytest.fixture(scope="module")
def sq():
    ensure_library()
    from paper_2609_04526_amd import sq as _sq
    return _sq


def normwise(got, ref):
    ref = np.asarray(ref, np.float64)
    den = np.linalg.norm(ref)
    return float(np.linalg.norm(np.asarray(got, np.float64) - ref) / (den if den > 0 else 1.0))


def plane(fmt, O, G, seed):
    if fmt == "mx":
        return inputs.e8m0_normal_exponents(seed, O, G, -6.0, 1.5), 1.0
    return inputs.e4m3_abs_normal(seed, O, G), float(np.float32(1.0 / 448.0))


def factors(fmt, base, ws2, r, seed, push=1.0):
    """bf16 B [O, r], A [r, G] whose product moves scales by about `push` times their size."""
    O, G = base.shape
    g = inputs.rng(seed)
    eff = codec.effective_scales(fmt, base, ws2)
    scale = float(np.median(np.abs(eff[eff > 0]))) if np.any(eff > 0) else 1.0
    B = g.standard_normal((O, r)).astype(np.float32) / np.sqrt(r)
    A = (g.standard_normal((r, G)) * scale * push).astype(np.float32)
    return torch.from_numpy(B).to(torch.bfloat16), torch.from_numpy(A).to(torch.bfloat16)


CASES = [("mx", 64, 16, 8), ("nv", 64, 32, 16), ("mx", 136, 300, 32), ("nv", 200, 77, 5),
         ("mx", 8, 1, 1), ("nv", 520, 520, 64), ("mx", 1000, 129, 33)]


@pytest.mark.parametrize("fmt,O,G,r", CASES)
def test_qast_scales_bit_exact(sq, fmt, O, G, r):
    print(f"[qast scales] fmt={fmt} O={O} G={G} r={r}", flush=True)
    base, ws2 = plane(fmt, O, G, 7000 + O + G)
    B, A = factors(fmt, base, ws2, r, 7100 + r, push=2.0)
    c = 0.5
    want, want_m = qast.qast_scales(fmt, base, B, A, c, ws2)
    got, got_m = sq.sq_qast_scales(fmt, torch.from_numpy(base).cuda(), B.cuda(), A.cuda(), c, ws2)
    torch.cuda.synchronize()
    assert np.array_equal(got.cpu().numpy(), want)
    assert np.array_equal(got_m.cpu().numpy(), want_m)
    assert np.any(want != base)


def test_nv_ceiling_clamp_binds_and_masks(sq):
    """Blocks pushed past 448 ws2 saturate at 0x7E with mask 0 (stability recipe (ii)-(iii))."""
    O, G, r = 64, 40, 2
    base, ws2 = plane("nv", O, G, 7200)
    g = inputs.rng(7201)
    B = np.stack([np.ones(O), g.standard_normal(O) * 0.1], axis=1).astype(np.float32)
    A = np.zeros((r, G), np.float32)
    A[0, :10] = 600.0 * ws2                      # beyond the ceiling for every row
    A[0, 10:20] = -0.5 * ws2
    A[1, :] = g.standard_normal(G) * ws2
    Bb = torch.from_numpy(B).to(torch.bfloat16)
    Ab = torch.from_numpy(A).to(torch.bfloat16)
    want, want_m = qast.qast_scales("nv", base, Bb, Ab, 1.0, ws2)
    got, got_m = sq.sq_qast_scales("nv", torch.from_numpy(base).cuda(), Bb.cuda(), Ab.cuda(), 1.0, ws2)
    torch.cuda.synchronize()
    assert np.array_equal(got.cpu().numpy(), want) and np.array_equal(got_m.cpu().numpy(), want_m)
    assert np.all(want[:, :10] == 0x7E) and np.all(want_m[:, :10] == 0)
    assert np.all(want_m[:, 10:] == 1)


def test_qast_scales_in_place_and_without_mask(sq):
    fmt, O, G, r = "nv", 96, 64, 8
    base, ws2 = plane(fmt, O, G, 7300)
    B, A = factors(fmt, base, ws2, r, 7301)
    want, _ = qast.qast_scales(fmt, base, B, A, 1.0, ws2)
    s = torch.from_numpy(base).cuda()
    sq.sq_qast_scales(fmt, s, B.cuda(), A.cuda(), 1.0, ws2, scales_out=s, want_mask=False)
    torch.cuda.synchronize()
    assert np.array_equal(s.cpu().numpy(), want)


@pytest.mark.parametrize("fmt", ["mx", "nv"])
def test_zero_adapter_and_merge_share_the_grid_path(sq, fmt):
    """B = 0 leaves every byte; and the GPU merge of the oracle's Delta_S writes
    exactly the bytes the GPU QAST forward uses (stability recipe (iii))."""
    O, G, r = 128, 96, 16
    base, ws2 = plane(fmt, O, G, 7400)
    B, A = factors(fmt, base, ws2, r, 7401, push=3.0)
    zero, m = sq.sq_qast_scales(fmt, torch.from_numpy(base).cuda(), torch.zeros_like(B).cuda(), A.cuda(), 1.0, ws2)
    fwd, _ = sq.sq_qast_scales(fmt, torch.from_numpy(base).cuda(), B.cuda(), A.cuda(), 1.0, ws2)
    merged = torch.from_numpy(base.reshape(-1).copy()).cuda()
    d = torch.from_numpy(qast.delta_s(B, A, 1.0).reshape(-1)).cuda()
    sq.sq_merge_scales(fmt, merged, delta=d, ws2=ws2)
    torch.cuda.synchronize()
    assert np.array_equal(zero.cpu().numpy(), base) and bool(torch.all(m == 1))
    assert np.array_equal(merged.cpu().numpy().reshape(O, G), fwd.cpu().numpy())


GRAD_CASES = [(64, 16, 8), (130, 77, 16), (1000, 129, 32), (257, 448, 64), (33, 5, 3)]


@pytest.mark.parametrize("O,G,r", GRAD_CASES)
@pytest.mark.parametrize("masked", [False, True])
def test_factor_grads(sq, O, G, r, masked):
    print(f"[qast grads] O={O} G={G} r={r} masked={masked}", flush=True)
    g = inputs.rng(7500 + O + G + r)
    dS = (g.standard_normal((O, G)) * 1e-2).astype(np.float32)
    mask = (g.random((O, G)) > 0.2).astype(np.uint8) if masked else np.ones((O, G), np.uint8)
    B = torch.from_numpy(g.standard_normal((O, r)).astype(np.float32)).to(torch.bfloat16)
    A = torch.from_numpy(g.standard_normal((r, G)).astype(np.float32)).to(torch.bfloat16)
    c = 0.25
    wB, wA = qast.factor_grads(dS, mask, B, A, c)
    m_dev = torch.from_numpy(mask).cuda() if masked else None
    dB, dA = sq.sq_qast_factor_grads(torch.from_numpy(dS).cuda(), m_dev, B.cuda(), A.cuda(), c)
    dB2, dA2 = sq.sq_qast_factor_grads(torch.from_numpy(dS).cuda(), m_dev, B.cuda(), A.cuda(), c)
    torch.cuda.synchronize()
    assert normwise(dB.cpu().numpy(), wB) <= TOL
    assert normwise(dA.cpu().numpy(), wA) <= TOL
    assert torch.equal(dB, dB2) and torch.equal(dA, dA2)                 # fixed order


@pytest.mark.parametrize("fmt", ["mx", "nv"])
def test_qast_step_through_the_layer(sq, fmt):
    """QAST scales -> forward / dX on the on-grid bytes -> dS -> dB, dA, against the
    same chain in the oracle."""
    T, O, I, r = 96, 136, 256, 8
    G = I // codec.BLOCK[fmt]
    base, ws2 = plane(fmt, O, G, 7600)
    B, A = factors(fmt, base, ws2, r, 7601, push=1.5)
    X = inputs.bf16_normal(7602, (T, I))
    dY = inputs.bf16_normal(7603, (T, O))
    codes = inputs.codes_uniform(7604, O, I)
    c = 0.5
    sc, m = sq.sq_qast_scales(fmt, torch.from_numpy(base).cuda(), B.cuda(), A.cuda(), c, ws2)
    cd = torch.from_numpy(codes).cuda()
    Y = sq.sq_fwd(fmt, X.cuda(), cd, sc, ws2)
    dX = sq.sq_bwd_dx(fmt, dY.cuda(), cd, sc, ws2)
    dS = sq.sq_bwd_dscale(fmt, X.cuda(), dY.cuda(), cd)
    dB, dA = sq.sq_qast_factor_grads(dS, m, B.cuda(), A.cuda(), c)
    torch.cuda.synchronize()
    w_sc, w_m = qast.qast_scales(fmt, base, B, A, c, ws2)
    assert np.array_equal(sc.cpu().numpy(), w_sc) and np.array_equal(m.cpu().numpy(), w_m)
    W = linear.dequant(fmt, codes, w_sc, ws2)
    Xd, dYd = X.double().numpy(), dY.double().numpy()
    assert normwise(Y.cpu().numpy(), linear.forward(Xd, W)) <= 2e-3
    assert normwise(dX.cpu().numpy(), linear.backward_dx(dYd, W)) <= 2e-3
    w_dS = linear.backward_dscale(fmt, Xd, dYd, codes)
    wB, wA = qast.factor_grads(w_dS, w_m, B, A, c)
    assert normwise(dB.cpu().numpy(), wB) <= 2e-3
    assert normwise(dA.cpu().numpy(), wA) <= 2e-3


def test_qast_8b_gate_projection_nv(sq):
    """14336 x 4096 NVFP4 gate projection (G = 256), rank 32: every byte and mask."""
    O, G, r = 14336, 256, 32
    base, ws2 = plane("nv", O, G, 7700)
    B, A = factors("nv", base, ws2, r, 7701, push=1.0)
    want, want_m = qast.qast_scales("nv", base, B, A, 1.0, ws2)
    got, got_m = sq.sq_qast_scales("nv", torch.from_numpy(base).cuda(), B.cuda(), A.cuda(), 1.0, ws2)
    g = inputs.rng(7702)
    dS = (g.standard_normal((O, G)) * 1e-3).astype(np.float32)
    dB, dA = sq.sq_qast_factor_grads(torch.from_numpy(dS).cuda(), got_m, B.cuda(), A.cuda(), 1.0)
    torch.cuda.synchronize()
    assert np.array_equal(got.cpu().numpy(), want)
    assert np.array_equal(got_m.cpu().numpy(), want_m)
    wB, wA = qast.factor_grads(dS, want_m, B, A, 1.0)
    assert normwise(dB.cpu().numpy(), wB) <= TOL
    assert normwise(dA.cpu().numpy(), wA) <= TOL


@pytest.mark.parametrize("fmt,E,O,G,r", [("mx", 5, 64, 40, 8), ("nv", 3, 136, 77, 33), ("nv", 260, 8, 16, 4)])
def test_batched_experts_match_per_expert(sq, fmt, E, O, G, r):
    """E stacked experts in one launch sequence (260 experts: two tables of
    per-expert ws2): scale bytes and masks equal the oracle's per expert bit
    for bit, and the factor gradients equal the single-plane entry's bit for
    bit (the same order per expert)."""
    print(f"[qast batched] fmt={fmt} E={E} O={O} G={G} r={r}", flush=True)
    bases, ws2s, Bs, As = [], [], [], []
    for e in range(E):
        base, ws2 = plane(fmt, O, G, 7700 + e)
        if fmt == "nv":
            ws2 = float(np.float32(ws2 * (1 + e % 4)))
        B, A = factors(fmt, base, ws2, r, 7800 + e, push=2.0)
        bases.append(base), ws2s.append(ws2), Bs.append(B), As.append(A)
    base_d = torch.from_numpy(np.stack(bases)).cuda()
    B_d = torch.stack(Bs).cuda()
    A_d = torch.stack(As).cuda()
    got, got_m = sq.sq_qast_scales_batched(fmt, base_d, B_d, A_d, 0.5, ws2s if fmt == "nv" else None)
    g = inputs.rng(7900)
    dS = (g.standard_normal((E, O, G)) * 1e-2).astype(np.float32)
    dS_d = torch.from_numpy(dS).cuda()
    dB, dA = sq.sq_qast_factor_grads_batched(dS_d, got_m, B_d, A_d, 0.25)
    torch.cuda.synchronize()
    gs, gm = got.cpu().numpy(), got_m.cpu().numpy()
    for e in range(E) if E <= 8 else [0, 1, 255, 256, E - 1]:
        want, want_m = qast.qast_scales(fmt, bases[e], Bs[e], As[e], 0.5, ws2s[e])
        assert np.array_equal(gs[e], want) and np.array_equal(gm[e], want_m)
        dB1, dA1 = sq.sq_qast_factor_grads(dS_d[e], got_m[e], B_d[e], A_d[e], 0.25)
        torch.cuda.synchronize()
        assert torch.equal(dB1, dB[e]) and torch.equal(dA1, dA[e])
        wB, wA = qast.factor_grads(dS[e], gm[e], Bs[e], As[e], 0.25)
        assert normwise(dB[e].cpu().numpy(), wB) <= TOL and normwise(dA[e].cpu().numpy(), wA) <= TOL


def _rmax(r):
    return 8 if r <= 8 else 16 if r <= 16 else 32 if r <= 32 else 64


def wide_tiles_taken(E, O, G, r, cus=256):
    """Whether a batched call of this shape runs the wide tiles: the scale step's
    128-row x 32-block tiles and the dB pass's 4 rows per thread, each chosen
    when it still gives every CU two workgroups."""
    scales = E * -(-O // 128) * -(-G // 32) >= 2 * cus
    db_rows = 4 * (256 // (_rmax(r) // 4))
    return scales and E * -(-O // db_rows) >= 2 * cus


@pytest.mark.parametrize("fmt,E,O,G,r", [("mx", 130, 520, 40, 32), ("nv", 130, 520, 37, 33)])
def test_batched_wide_tiles(sq, fmt, E, O, G, r):
    """Stacked experts at MoE-like sizes, where the batched calls take the wide
    tiles (G % 4 == 0: word-wide byte planes and 16-byte dS loads; G = 37:
    byte-wide, ragged last block tile; rank 33: the 64-rank kernels).  Every
    expert's bytes, mask and gradients equal the single-plane calls' (narrow
    tiles) bit for bit, and sampled experts equal the oracle."""
    print(f"[qast wide] fmt={fmt} E={E} O={O} G={G} r={r}", flush=True)
    assert wide_tiles_taken(E, O, G, r) and not wide_tiles_taken(1, O, G, r)
    bases, ws2s, Bs, As = [], [], [], []
    for e in range(E):
        base, ws2 = plane(fmt, O, G, 8100 + e)
        if fmt == "nv":
            ws2 = float(np.float32(ws2 * (1 + e % 3)))
        B, A = factors(fmt, base, ws2, r, 8300 + e, push=2.0)
        if fmt == "nv":
            A[0, :4] = 6000.0 * ws2                # past the ceiling where B[o, 0] is large
        bases.append(base), ws2s.append(ws2), Bs.append(B), As.append(A)
    base_d = torch.from_numpy(np.stack(bases)).cuda()
    B_d, A_d = torch.stack(Bs).cuda(), torch.stack(As).cuda()
    got, got_m = sq.sq_qast_scales_batched(fmt, base_d, B_d, A_d, 0.5, ws2s if fmt == "nv" else None)
    dS = (inputs.rng(8500).standard_normal((E, O, G)) * 1e-2).astype(np.float32)
    dS_d = torch.from_numpy(dS).cuda()
    dB, dA = sq.sq_qast_factor_grads_batched(dS_d, got_m, B_d, A_d, 0.25)
    torch.cuda.synchronize()
    for e in range(E):
        one, one_m = sq.sq_qast_scales(fmt, base_d[e], B_d[e], A_d[e], 0.5, ws2s[e])
        dB1, dA1 = sq.sq_qast_factor_grads(dS_d[e], got_m[e], B_d[e], A_d[e], 0.25)
        torch.cuda.synchronize()
        assert torch.equal(one, got[e]) and torch.equal(one_m, got_m[e]), e
        assert torch.equal(dB1, dB[e]) and torch.equal(dA1, dA[e]), e
    gs, gm = got.cpu().numpy(), got_m.cpu().numpy()
    if fmt == "nv":
        assert 0 < int((gm == 0).sum()) < gm.size          # the ceiling binds somewhere
    for e in (0, 1, 64, E - 1):
        want, want_m = qast.qast_scales(fmt, bases[e], Bs[e], As[e], 0.5, ws2s[e])
        assert np.array_equal(gs[e], want) and np.array_equal(gm[e], want_m)
        wB, wA = qast.factor_grads(dS[e], gm[e], Bs[e], As[e], 0.25)
        assert normwise(dB[e].cpu().numpy(), wB) <= TOL and normwise(dA[e].cpu().numpy(), wA) <= TOL
