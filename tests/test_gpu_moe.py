"""GPU parity of the grouped MoE expert products (sq_fwd_grouped,
sq_bwd_dx_grouped, sq_bwd_dscale_grouped) against the oracle, per expert.

The grouped forward and dX accumulate every output element in the same order
as the single-product kernels, so they are also compared with sq_fwd /
sq_bwd_dx bit for bit; dS is compared with the oracle (normwise 2e-3, the
bar of the single products), and an expert with no tokens gets dS = 0."""

import numpy as np
import pytest
import torch

from conftest import ensure_library, gpu_ready
from oracle import linear
from paper_2609_04526_amd import inputs

pytestmark = [pytest.mark.gpu, pytest.mark.skipif(not gpu_ready(), reason="needs a GPU")]

TOL = 2e-3


@pytest.fixture(scope="module")
def sq():
    ensure_library()
    from paper_2609_04526_amd import sq as _sq
    return _sq


def normwise(got, ref):
    ref = np.asarray(ref, np.float64)
    den = np.linalg.norm(ref)
    return float(np.linalg.norm(np.asarray(got, np.float64) - ref) / (den if den > 0 else 1.0))


def experts(fmt, E, O, I, seed):
    codes, scales, ws2 = [], [], []
    for e in range(E):
        codes.append(inputs.codes_uniform(seed + 3 * e, O, I))
        if fmt == "mx":
            scales.append(inputs.e8m0_normal_exponents(seed + 3 * e + 1, O, I // 32, -6, 1.5))
            ws2.append(1.0)
        else:
            scales.append(inputs.e4m3_abs_normal(seed + 3 * e + 1, O, I // 16))
            ws2.append(float(np.float32(1.0 / (448 * (1 + e % 3)))))
    return codes, scales, ws2


def cuda(arrs):
    return [torch.from_numpy(a).cuda() for a in arrs]


@pytest.mark.parametrize("fmt", ["mx", "nv"])
def test_grouped_products_match_oracle_and_single(sq, fmt):
    """Eight experts with ragged token counts, including none and one."""
    O, I = 256, 512
    Ts = [0, 1, 37, 300, 64, 513, 128, 7]
    codes, scales, ws2 = experts(fmt, len(Ts), O, I, 7000)
    Xs = [inputs.bf16_normal(7100 + e, (T, I)) for e, T in enumerate(Ts)]
    dYs = [inputs.bf16_normal(7200 + e, (T, O)) for e, T in enumerate(Ts)]
    cd, sd = cuda(codes), cuda(scales)
    Xd, dYd = [x.cuda() for x in Xs], [d.cuda() for d in dYs]
    print(f"[moe grouped] fmt={fmt} T={Ts}", flush=True)
    Ys = sq.sq_fwd_grouped(fmt, Xd, cd, sd, ws2)
    dXs = sq.sq_bwd_dx_grouped(fmt, dYd, cd, sd, ws2)
    dSs = sq.sq_bwd_dscale_grouped(fmt, Xd, dYd, cd)
    torch.cuda.synchronize()
    for e, T in enumerate(Ts):
        W = linear.dequant(fmt, codes[e], scales[e], ws2[e])
        dS_ref = linear.backward_dscale(fmt, Xs[e].float().numpy(), dYs[e].float().numpy(), codes[e])
        if T == 0:
            assert Ys[e].numel() == 0 and dXs[e].numel() == 0
            assert torch.count_nonzero(dSs[e]).item() == 0
            continue
        assert normwise(Ys[e].cpu().numpy(), linear.forward(Xs[e].float().numpy(), W)) <= TOL
        assert normwise(dXs[e].cpu().numpy(), linear.backward_dx(dYs[e].float().numpy(), W)) <= TOL
        assert normwise(dSs[e].cpu().numpy(), dS_ref) <= TOL
        y1 = sq.sq_fwd(fmt, Xd[e], cd[e], sd[e], ws2[e])
        dx1 = sq.sq_bwd_dx(fmt, dYd[e], cd[e], sd[e], ws2[e])
        torch.cuda.synchronize()
        assert torch.equal(y1, Ys[e]) and torch.equal(dx1, dXs[e])


def test_more_experts_than_one_launch_holds(sq):
    """70 experts (two launches of at most 64), bf16 outputs."""
    O, I = 64, 128
    Ts = [(13 * e) % 97 for e in range(70)]
    codes, scales, ws2 = experts("mx", len(Ts), O, I, 7300)
    Xs = [inputs.bf16_normal(7400 + e, (T, I)) for e, T in enumerate(Ts)]
    dYs = [inputs.bf16_normal(7500 + e, (T, O)) for e, T in enumerate(Ts)]
    cd, sd = cuda(codes), cuda(scales)
    Xd, dYd = [x.cuda() for x in Xs], [d.cuda() for d in dYs]
    Ys = sq.sq_fwd_grouped("mx", Xd, cd, sd, out_dtype=torch.bfloat16)
    dSs = sq.sq_bwd_dscale_grouped("mx", Xd, dYd, cd)
    torch.cuda.synchronize()
    for e, T in enumerate(Ts):
        if T == 0:
            assert torch.count_nonzero(dSs[e]).item() == 0
            continue
        W = linear.dequant("mx", codes[e], scales[e])
        assert normwise(Ys[e].float().cpu().numpy(), linear.forward(Xs[e].float().numpy(), W)) <= TOL
        dS_ref = linear.backward_dscale("mx", Xs[e].float().numpy(), dYs[e].float().numpy(), codes[e])
        assert normwise(dSs[e].cpu().numpy(), dS_ref) <= TOL


def test_moe_layer_shapes_sampled(sq):
    """A 30B-A3B-style MoE layer: 128 experts of [768, 2048] (gate/up) and
    [2048, 768] (down), 4096 tokens routed top-8 (32768 expert tokens, ragged
    by a seeded multinomial); every expert runs, eight sampled experts are
    checked against the oracle."""
    E, tokens = 128, 4096 * 8
    g = inputs.rng(7600)
    Ts = g.multinomial(tokens, g.dirichlet(np.full(E, 2.0))).tolist()
    sample = sorted(set(g.choice(E, 8, replace=False).tolist()))
    for (O, I) in [(768, 2048), (2048, 768)]:
        codes, scales, ws2 = experts("mx", E, O, I, 7700 + O)
        cd, sd = cuda(codes), cuda(scales)
        Xd = [inputs.device_bf16_normal(7800 + e, (T, I)) for e, T in enumerate(Ts)]
        dYd = [inputs.device_bf16_normal(7900 + e, (T, O)) for e, T in enumerate(Ts)]
        print(f"[moe layer] O={O} I={I} experts={E} tokens={sum(Ts)}", flush=True)
        Ys = sq.sq_fwd_grouped("mx", Xd, cd, sd)
        dXs = sq.sq_bwd_dx_grouped("mx", dYd, cd, sd)
        dSs = sq.sq_bwd_dscale_grouped("mx", Xd, dYd, cd)
        torch.cuda.synchronize()
        for e in sample:
            X, dY = Xd[e].float().cpu().numpy(), dYd[e].float().cpu().numpy()
            W = linear.dequant("mx", codes[e], scales[e])
            assert normwise(Ys[e].cpu().numpy(), linear.forward(X, W)) <= TOL
            assert normwise(dXs[e].cpu().numpy(), linear.backward_dx(dY, W)) <= TOL
            assert normwise(dSs[e].cpu().numpy(), linear.backward_dscale("mx", X, dY, codes[e])) <= TOL
