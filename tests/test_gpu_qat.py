"""GPU parity of the QAT-LoRA weight-space STE path against the oracle.

sq_qat_requant writes integers decided by fp32 arithmetic done in the same
order on both sides: codes and scales must match bit for bit.  sq_lora_grads
accumulates in fp32 and is compared with the fp64 oracle normwise (<= 1e-4,
inside the 2e-3 bar: fp32 sums over a few thousand tokens stay near 1e-6).
The forward on the re-quantised weight is the FP4 GEMM and is checked against
the oracle's forward on the oracle's fake-quantised weight (2e-3)."""

import numpy as np
import pytest
import torch

from conftest import ensure_library, gpu_ready
from oracle import codec, linear, qat
from paper_2609_04526_amd import inputs

pytestmark = [pytest.mark.gpu, pytest.mark.skipif(not gpu_ready(), reason="needs a GPU")]

GRAD_TOL = 1e-4
GEMM_TOL = 2e-3


@pytest.fixture(scope="module")
def sq():
    ensure_library()
    from paper_2609_04526_amd import sq as _sq
    return _sq


def normwise(got, ref):
    ref = np.asarray(ref, np.float64)
    den = np.linalg.norm(ref)
    return float(np.linalg.norm(np.asarray(got, np.float64) - ref) / (den if den > 0 else 1.0))


def layer(fmt, O, I, r, seed, std=0.02):
    """Base codes / scales, bf16 factors B [O, r], A [r, I]."""
    codes = inputs.codes_uniform(seed, O, I)
    if fmt == "mx":
        sb, ws2 = inputs.e8m0_normal_exponents(seed + 1, O, I // 32, -6, 1.5), 1.0
    else:
        sb, ws2 = inputs.e4m3_abs_normal(seed + 1, O, I // 16), float(np.float32(1 / 448))
    B, A = inputs.lora_factors(seed + 2, O, I, r, std)
    return codes, sb, ws2, torch.from_numpy(B).to(torch.bfloat16), torch.from_numpy(A).to(torch.bfloat16)


@pytest.mark.parametrize("fmt,O,I,r", [("mx", 264, 1056, 32), ("nv", 136, 784, 58), ("mx", 8, 32, 1),
                                       ("nv", 64, 4096, 64), ("mx", 1024, 4096, 16)])
def test_requant_matches_oracle(sq, fmt, O, I, r):
    """Ragged tiles in both directions (264 rows = 16 x 16 + 8; 1056 columns =
    2 x 512 + 32), ranks that are not multiples of 8, rank 1 and the maximum."""
    codes, sb, ws2, B, A = layer(fmt, O, I, r, seed=6000 + O + r)
    print(f"[qat requant] fmt={fmt} O={O} I={I} r={r}", flush=True)
    c, s = sq.sq_qat_requant(fmt, torch.from_numpy(codes).cuda(), torch.from_numpy(sb).cuda(), B.cuda(), A.cuda(),
                             2.0, ws2)
    torch.cuda.synchronize()
    rc, rs = qat.requant(fmt, codes, sb, ws2, B, A, 2.0)
    assert np.array_equal(s.cpu().numpy(), rs)
    assert np.array_equal(c.cpu().numpy(), rc)
    moved = np.mean(codec.unpack_nibbles(rc) != codec.unpack_nibbles(codes))
    print(f"  code nibbles moved by the adapter: {moved:.3f}")
    assert 0.0 < moved < 1.0


def test_requant_zero_adapter_and_specials(sq):
    """B = 0 returns the base (a -0 code returns as +0) when every block holds a
    magnitude-6 code; large factors push weights past the grid (saturation)."""
    O, I, r = 32, 512, 8
    codes = inputs.codes_uniform(6100, O, I)
    nib = codec.unpack_nibbles(codes)
    nib[:, ::32] = 7
    codes = codec.pack_nibbles(nib)
    sb = inputs.e8m0_uniform_exponents(6101, O, I // 32, -8, -3)
    A = torch.from_numpy(inputs.rng(6102).standard_normal((r, I)).astype(np.float32)).to(torch.bfloat16)
    B0 = torch.zeros((O, r), dtype=torch.bfloat16)
    c, s = sq.sq_qat_requant("mx", torch.from_numpy(codes).cuda(), torch.from_numpy(sb).cuda(), B0.cuda(),
                             A.cuda(), 2.0)
    torch.cuda.synchronize()
    want = codec.pack_nibbles(np.where(nib == 8, 0, nib).astype(np.uint8))
    assert np.array_equal(s.cpu().numpy(), sb) and np.array_equal(c.cpu().numpy(), want)
    Bbig = torch.from_numpy(inputs.rng(6103).standard_normal((O, r)).astype(np.float32) * 100).to(torch.bfloat16)
    c, s = sq.sq_qat_requant("mx", torch.from_numpy(codes).cuda(), torch.from_numpy(sb).cuda(), Bbig.cuda(),
                             A.cuda(), 2.0)
    torch.cuda.synchronize()
    rc, rs = qat.requant("mx", codes, sb, 1.0, Bbig, A, 2.0)
    assert np.array_equal(s.cpu().numpy(), rs) and np.array_equal(c.cpu().numpy(), rc)


@pytest.mark.parametrize("T,O,I,r", [(300, 264, 1056, 32), (1, 8, 16, 1), (129, 64, 512, 58),
                                     (256, 1024, 512, 64), (77, 520, 96, 7)])
def test_lora_grads_match_oracle(sq, T, O, I, r):
    """Token counts across the 128-token chunks (ragged, single token), row
    tiles of 32 with a ragged tail, both rank widths (<= 32 and <= 64)."""
    g = inputs.rng(6200 + T)
    X = inputs.bf16_normal(6201 + T, (T, I))
    dY = inputs.bf16_normal(6202 + T, (T, O))
    B = torch.from_numpy(g.standard_normal((O, r)).astype(np.float32) * 0.05).to(torch.bfloat16)
    A = torch.from_numpy(g.standard_normal((r, I)).astype(np.float32) * 0.05).to(torch.bfloat16)
    print(f"[lora grads] T={T} O={O} I={I} r={r}", flush=True)
    dB, dA = sq.sq_lora_grads(X.cuda(), dY.cuda(), B.cuda(), A.cuda(), 2.0)
    torch.cuda.synchronize()
    rB, rA = qat.lora_grads(X, dY, B, A, 2.0)
    eB, eA = normwise(dB.cpu().numpy(), rB), normwise(dA.cpu().numpy(), rA)
    print(f"  normwise dB {eB:.2e} dA {eA:.2e}")
    assert eB <= GRAD_TOL and eA <= GRAD_TOL
    dB2, dA2 = sq.sq_lora_grads(X.cuda(), dY.cuda(), B.cuda(), A.cuda(), 2.0)
    torch.cuda.synchronize()
    assert torch.equal(dB, dB2) and torch.equal(dA, dA2)         # deterministic


def test_lora_grads_no_tokens(sq):
    B = torch.ones((16, 4), dtype=torch.bfloat16, device="cuda")
    A = torch.ones((4, 32), dtype=torch.bfloat16, device="cuda")
    X = torch.empty((0, 32), dtype=torch.bfloat16, device="cuda")
    dY = torch.empty((0, 16), dtype=torch.bfloat16, device="cuda")
    dB = torch.full((16, 4), 7.0, device="cuda")
    dA = torch.full((4, 32), 7.0, device="cuda")
    sq.sq_lora_grads(X, dY, B, A, 1.0, dB=dB, dA=dA)
    torch.cuda.synchronize()
    assert torch.count_nonzero(dB).item() == 0 and torch.count_nonzero(dA).item() == 0


def test_lora_grads_attention_projection_sampled(sq):
    """The 4096 x 4096 projection at 4096 tokens, rank 32 (the comparator's
    shape): sampled rows of dB and columns of dA from the oracle."""
    T, O, I, r = 4096, 4096, 4096, 32
    X = inputs.bf16_normal(6300, (T, I))
    dY = inputs.bf16_normal(6301, (T, O))
    g = inputs.rng(6302)
    B = torch.from_numpy(g.standard_normal((O, r)).astype(np.float32) * 0.02).to(torch.bfloat16)
    A = torch.from_numpy(g.standard_normal((r, I)).astype(np.float32) * 0.02).to(torch.bfloat16)
    dB, dA = sq.sq_lora_grads(X.cuda(), dY.cuda(), B.cuda(), A.cuda(), 2.0)
    torch.cuda.synchronize()
    rows = np.sort(np.concatenate([g.choice(O, 15, replace=False), [O - 1]]))
    cols = np.sort(np.concatenate([g.choice(I, 15, replace=False), [I - 1]]))
    rB, rA = qat.lora_grads_sampled(X, dY, B, A, 2.0, rows, cols)
    eB = normwise(dB.cpu().numpy()[rows], rB)
    eA = normwise(dA.cpu().numpy()[:, cols], rA)
    print(f"  sampled normwise dB {eB:.2e} dA {eA:.2e}")
    assert eB <= GRAD_TOL and eA <= GRAD_TOL


@pytest.mark.parametrize("fmt", ["mx", "nv"])
def test_qat_step_forward_and_dx(sq, fmt):
    """One STE step's forward and dX on the re-quantised weight, against the
    oracle's forward / dX on its own fake-quantised weight."""
    T, O, I, r = 200, 264, 1024, 32
    codes, sb, ws2, B, A = layer(fmt, O, I, r, seed=6400)
    X = inputs.bf16_normal(6401, (T, I))
    dY = inputs.bf16_normal(6402, (T, O))
    c, s = sq.sq_qat_requant(fmt, torch.from_numpy(codes).cuda(), torch.from_numpy(sb).cuda(), B.cuda(), A.cuda(),
                             2.0, ws2)
    Y = sq.sq_fwd(fmt, X.cuda(), c, s, ws2)
    dX = sq.sq_bwd_dx(fmt, dY.cuda(), c, s, ws2)
    torch.cuda.synchronize()
    rc, rs = qat.requant(fmt, codes, sb, ws2, B, A, 2.0)
    Wq = linear.dequant(fmt, rc, rs, ws2)
    assert normwise(Y.float().cpu().numpy(), linear.forward(X.float().numpy(), Wq)) <= GEMM_TOL
    assert normwise(dX.float().cpu().numpy(), linear.backward_dx(dY.float().numpy(), Wq)) <= GEMM_TOL


# ---------------------------------------------------------------- MoE experts
@pytest.mark.parametrize("fmt,E,O,I,r", [("mx", 5, 264, 1056, 32), ("nv", 3, 136, 784, 58), ("nv", 300, 8, 32, 1)])
def test_requant_batched_equals_single_calls(sq, fmt, E, O, I, r):
    """Stacked experts (300: two launches of the 256-entry ws2 table), each
    with its own ws2 for NVFP4: every expert's codes and scales equal its own
    sq_qat_requant call bit for bit, and the first equals the oracle."""
    parts = [layer(fmt, O, I, r, seed=6600 + 7 * e) for e in range(E)]
    codes = torch.from_numpy(np.stack([p[0] for p in parts])).cuda()
    sb = torch.from_numpy(np.stack([p[1] for p in parts])).cuda()
    ws2 = [float(np.float32(p[2] * (1 + 0.25 * (e % 3)))) for e, p in enumerate(parts)]
    B = torch.stack([p[3] for p in parts]).cuda()
    A = torch.stack([p[4] for p in parts]).cuda()
    print(f"[qat requant batched] fmt={fmt} E={E} O={O} I={I} r={r}", flush=True)
    c, s = sq.sq_qat_requant_batched(fmt, codes, sb, B, A, 2.0, ws2 if fmt == "nv" else None)
    torch.cuda.synchronize()
    for e in range(E):
        ce, se = sq.sq_qat_requant(fmt, codes[e], sb[e], B[e], A[e], 2.0, ws2[e] if fmt == "nv" else 1.0)
        torch.cuda.synchronize()
        assert torch.equal(c[e], ce) and torch.equal(s[e], se), e
    rc, rs = qat.requant(fmt, parts[0][0], parts[0][1], ws2[0] if fmt == "nv" else 1.0, parts[0][3], parts[0][4], 2.0)
    assert np.array_equal(c[0].cpu().numpy(), rc) and np.array_equal(s[0].cpu().numpy(), rs)


@pytest.mark.parametrize("Ts,O,I,r", [([300, 0, 1, 129, 77], 264, 1056, 32),
                                      ([64] * 40 + [0, 513], 64, 512, 58),
                                      ([0, 0], 16, 32, 4)])
def test_lora_grads_batched_equals_single_calls(sq, Ts, O, I, r):
    """Experts with ragged, single, zero and repeated token counts (42 experts:
    two launch sets of 32): every expert's dB, dA equal its own sq_lora_grads
    call bit for bit, and match the oracle; experts without tokens get zeros."""
    E = len(Ts)
    g = inputs.rng(6700 + E)
    X = inputs.bf16_normal(6701 + E, (sum(Ts), I)).cuda()
    dY = inputs.bf16_normal(6702 + E, (sum(Ts), O)).cuda()
    B = torch.from_numpy(g.standard_normal((E, O, r)).astype(np.float32) * 0.05).to(torch.bfloat16).cuda()
    A = torch.from_numpy(g.standard_normal((E, r, I)).astype(np.float32) * 0.05).to(torch.bfloat16).cuda()
    print(f"[lora grads batched] E={E} T={Ts[:6]}... O={O} I={I} r={r}", flush=True)
    dB, dA = sq.sq_lora_grads_batched(Ts, X, dY, B, A, 2.0)
    torch.cuda.synchronize()
    t0 = 0
    for e, T in enumerate(Ts):
        Xe, dYe = X[t0:t0 + T], dY[t0:t0 + T]
        t0 += T
        sB, sA = sq.sq_lora_grads(Xe, dYe, B[e], A[e], 2.0)
        torch.cuda.synchronize()
        assert torch.equal(dB[e], sB) and torch.equal(dA[e], sA), e
        if T == 0:
            assert torch.count_nonzero(dB[e]).item() == 0 and torch.count_nonzero(dA[e]).item() == 0
        elif e < 4:
            rB, rA = qat.lora_grads(Xe.cpu(), dYe.cpu(), B[e].cpu(), A[e].cpu(), 2.0)
            assert normwise(dB[e].cpu().numpy(), rB) <= GRAD_TOL and normwise(dA[e].cpu().numpy(), rA) <= GRAD_TOL
