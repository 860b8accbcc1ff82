"""GPU parity of the grouped MoE expert products (sq_fwd_grouped,
sq_bwd_dx_grouped, sq_bwd_dscale_grouped) against the oracle, per expert.

The grouped products accumulate every output element in the same order as
the single-product kernels, so they are also compared with sq_fwd /
sq_bwd_dx / sq_bwd_dscale bit for bit (dS where the single call does not
split its token sum, i.e. needs no workspace); against the oracle every
element is held to the summation bound of tests/parity_check.py besides the
normwise 2e-3 bar.  An expert with no tokens gets dS = 0."""

import numpy as np
import pytest
import torch

from conftest import ensure_library, gpu_ready
from oracle import codec, linear
from paper_2609_04526_amd import inputs
from parity_check import assert_elements

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


def check_elements(fmt, X, dY, codes, W, Y=None, dX=None, dS=None, what=""):
    """Every element of the given fp32 outputs within the summation bound of
    its K terms (Y: I terms, dX: O terms, dS: T terms, then the code
    multiply and the block sum)."""
    Xd, dYd = np.asarray(X, np.float64), np.asarray(dY, np.float64)
    T, I = Xd.shape
    O = W.shape[0]
    if Y is not None:
        assert_elements(Y, linear.forward(Xd, W), np.abs(Xd) @ np.abs(W).T, I + 2, what + " Y")
    if dX is not None:
        assert_elements(dX, linear.backward_dx(dYd, W), np.abs(dYd) @ np.abs(W), O + 2, what + " dX")
    if dS is not None:
        B = codec.BLOCK[fmt]
        aS = (np.abs(linear.code_values(codes)) * (np.abs(dYd).T @ np.abs(Xd))).reshape(O, I // B, B).sum(axis=2)
        assert_elements(dS, linear.backward_dscale(fmt, Xd, dYd, codes), aS, T + B + 2, what + " dS")


def single_dscale_equal(sq, fmt, X, dY, codes, dS):
    """dS of one expert equals the single call's bit for bit (when that call
    keeps the token sum whole); returns whether it was compared."""
    T, I = X.shape
    O = dY.shape[1]
    if sq.sq_bwd_dscale_workspace(fmt, T, O, I) != 0:
        return False
    one = sq.sq_bwd_dscale(fmt, X, dY, codes)
    torch.cuda.synchronize()
    assert torch.equal(one, dS)
    return True


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
        check_elements(fmt, Xs[e].float().numpy(), dYs[e].float().numpy(), codes[e], W,
                       Ys[e].cpu().numpy(), dXs[e].cpu().numpy(), dSs[e].cpu().numpy(), f"expert {e}")
        y1 = sq.sq_fwd(fmt, Xd[e], cd[e], sd[e], ws2[e])
        dx1 = sq.sq_bwd_dx(fmt, dYd[e], cd[e], sd[e], ws2[e])
        torch.cuda.synchronize()
        assert torch.equal(y1, Ys[e]) and torch.equal(dx1, dXs[e])
        single_dscale_equal(sq, fmt, Xd[e], dYd[e], cd[e], dSs[e])


def test_more_experts_than_one_launch_holds(sq):
    """150 experts (two launches of at most 128), bf16 outputs; under 96
    tokens per expert on average, so dX takes the 64-token tiles."""
    O, I = 64, 128
    Ts = [(13 * e) % 97 for e in range(150)]
    codes, scales, ws2 = experts("mx", len(Ts), O, I, 7300)
    Xs = [inputs.bf16_normal(7400 + e, (T, I)) for e, T in enumerate(Ts)]
    dYs = [inputs.bf16_normal(7500 + e, (T, O)) for e, T in enumerate(Ts)]
    cd, sd = cuda(codes), cuda(scales)
    Xd, dYd = [x.cuda() for x in Xs], [d.cuda() for d in dYs]
    Ys = sq.sq_fwd_grouped("mx", Xd, cd, sd, out_dtype=torch.bfloat16)
    dXs = sq.sq_bwd_dx_grouped("mx", dYd, cd, sd)
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
        check_elements("mx", Xs[e].float().numpy(), dYs[e].float().numpy(), codes[e], W,
                       dX=dXs[e].cpu().numpy(), what=f"expert {e}")
        dx1 = sq.sq_bwd_dx("mx", dYd[e], cd[e], sd[e])
        torch.cuda.synchronize()
        assert torch.equal(dx1, dXs[e])


@pytest.mark.parametrize("Ts", [[4096, 4096], [2048, 3000, 2500]])
def test_long_experts_grouped_forward(sq, Ts):
    """Experts of 2048 tokens and more whose 256 x 256 tiles would not fill
    the chip (the 8B step's k and v projections, 1024 x 4096, as one grouped
    forward; and a ragged set): the grouped forward takes 128 x 256 tiles and
    equals each single forward bit for bit; sampled rows against the oracle
    within the element bound."""
    O, I = 1024, 4096
    codes, scales, _ = experts("mx", len(Ts), O, I, 7800)
    cd, sd = cuda(codes), cuda(scales)
    Xs = [inputs.bf16_normal(7810 + e, (T, I)) for e, T in enumerate(Ts)]
    Xd = [x.cuda() for x in Xs]
    print(f"[moe long] Ts={Ts}", flush=True)
    Ys = sq.sq_fwd_grouped("mx", Xd, cd, sd)
    torch.cuda.synchronize()
    g = inputs.rng(7820)
    for e, T in enumerate(Ts):
        y1 = sq.sq_fwd("mx", Xd[e], cd[e], sd[e])
        torch.cuda.synchronize()
        assert torch.equal(y1, Ys[e])
        rows = np.sort(np.concatenate([g.choice(T, 7, replace=False), [T - 1]]))
        W = linear.dequant("mx", codes[e], scales[e])
        Xr = Xs[e].float().numpy()[rows]
        check_elements("mx", Xr, np.zeros((rows.size, O), np.float32), codes[e], W,
                       Y=Ys[e].float().cpu().numpy()[rows], what=f"expert {e}")


def test_experts_spread_over_more_than_4_gib(sq):
    """Expert activations and output gradients placed 4.5 GiB apart in one
    buffer: a launch's 32-bit offsets from one base cannot reach both, so the
    launch takes fewer experts.  Grouped products equal the single ones bit
    for bit and the oracle within the bar."""
    O, I, Ts = 64, 512, [40, 72, 16]
    codes, scales, _ = experts("mx", 3, O, I, 7700)
    cd, sd = cuda(codes), cuda(scales)
    far = 9 << 29                                            # 4.5 GiB in bytes
    places = [0, far, 1 << 25]                               # X_e at these byte offsets, dY_e 16 MiB after
    big = torch.empty((far + (1 << 26)) // 2, dtype=torch.bfloat16, device="cuda")
    Xs = [inputs.bf16_normal(7710 + e, (T, I)) for e, T in enumerate(Ts)]
    dYs = [inputs.bf16_normal(7720 + e, (T, O)) for e, T in enumerate(Ts)]
    Xd, dYd = [], []
    for e, T in enumerate(Ts):
        x0, d0 = places[e] // 2, (places[e] + (1 << 24)) // 2
        Xd.append(big[x0:x0 + T * I].view(T, I))
        dYd.append(big[d0:d0 + T * O].view(T, O))
        Xd[e].copy_(Xs[e].cuda())
        dYd[e].copy_(dYs[e].cuda())
    print("[moe spread] experts 4.5 GiB apart", flush=True)
    Ys = sq.sq_fwd_grouped("mx", Xd, cd, sd)
    dXs = sq.sq_bwd_dx_grouped("mx", dYd, cd, sd)
    dSs = sq.sq_bwd_dscale_grouped("mx", Xd, dYd, cd)
    torch.cuda.synchronize()
    for e in range(3):
        y1 = sq.sq_fwd("mx", Xd[e], cd[e], sd[e])
        dx1 = sq.sq_bwd_dx("mx", dYd[e], cd[e], sd[e])
        torch.cuda.synchronize()
        assert torch.equal(y1, Ys[e]) and torch.equal(dx1, dXs[e])
        assert single_dscale_equal(sq, "mx", Xd[e], dYd[e], cd[e], dSs[e])
        W = linear.dequant("mx", codes[e], scales[e])
        assert normwise(Ys[e].float().cpu().numpy(), linear.forward(Xs[e].float().numpy(), W)) <= TOL
        dS_ref = linear.backward_dscale("mx", Xs[e].float().numpy(), dYs[e].float().numpy(), codes[e])
        assert normwise(dSs[e].cpu().numpy(), dS_ref) <= TOL
    del big, Xd, dYd
    torch.cuda.empty_cache()


@pytest.mark.parametrize("fmt", ["mx", "nv"])
def test_thin_experts_64_token_tiles(sq, fmt):
    """Experts of 1 to 140 tokens (64-token tiles for the MXFP4 register
    forward and, at under 96 tokens per expert, for dX): every expert equals
    its single products bit for bit, sampled ones the oracle per element."""
    O, I = 768, 2048
    Ts = [1, 63, 64, 65, 0, 127, 128, 129, 140, 7, 33, 96]
    codes, scales, ws2 = experts(fmt, len(Ts), O, I, 7350)
    cd, sd = cuda(codes), cuda(scales)
    Xd = [inputs.device_bf16_normal(7360 + e, (T, I)) for e, T in enumerate(Ts)]
    dYd = [inputs.device_bf16_normal(7380 + e, (T, O)) for e, T in enumerate(Ts)]
    print(f"[moe thin] fmt={fmt} T={Ts}", flush=True)
    Ys = sq.sq_fwd_grouped(fmt, Xd, cd, sd, ws2)
    dXs = sq.sq_bwd_dx_grouped(fmt, dYd, cd, sd, ws2)
    torch.cuda.synchronize()
    for e, T in enumerate(Ts):
        if T == 0:
            continue
        y1 = sq.sq_fwd(fmt, Xd[e], cd[e], sd[e], ws2[e])
        dx1 = sq.sq_bwd_dx(fmt, dYd[e], cd[e], sd[e], ws2[e])
        torch.cuda.synchronize()
        assert torch.equal(y1, Ys[e]) and torch.equal(dx1, dXs[e]), e
    for e in (0, 3, 8):
        W = linear.dequant(fmt, codes[e], scales[e], ws2[e])
        check_elements(fmt, Xd[e].float().cpu().numpy(), dYd[e].float().cpu().numpy(), codes[e], W,
                       Ys[e].cpu().numpy(), dXs[e].cpu().numpy(), what=f"expert {e} T={Ts[e]}")


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
            check_elements("mx", X, dY, codes[e], W, Ys[e].cpu().numpy(), dXs[e].cpu().numpy(),
                           dSs[e].cpu().numpy(), f"O={O} I={I} expert {e} T={Ts[e]}")
        # every expert's dS equals its single product where that keeps the
        # token sum whole (here: fewer than 8 token stages, T <= 448)
        compared = sum(single_dscale_equal(sq, "mx", Xd[e], dYd[e], cd[e], dSs[e]) for e in range(E))
        assert compared >= sum(T <= 448 for T in Ts)
        # every expert's dX equals its single product bit for bit; for the
        # gate shape the experts whose last 128-token tile would hold 64 rows
        # or fewer run those rows in a second launch of 64 x 256 tiles
        if I == 2048:
            assert dx_tail_split_taken(Ts, I)
        for e in range(E):
            one = sq.sq_bwd_dx("mx", dYd[e], cd[e], sd[e])
            assert torch.equal(one, dXs[e]), (O, I, e, Ts[e])


def test_grouped_dx_tail_split_nvfp4_bf16(sq):
    """Grouped NVFP4 dX with bf16 outputs over the routed split of a MoE
    layer (gate shape), where the short last token tiles run in a second
    launch: every expert's dX equals its single product bit for bit."""
    E, O, I = 128, 768, 2048
    g = inputs.rng(7650)
    Ts = g.multinomial(4096 * 8, g.dirichlet(np.full(E, 2.0))).tolist()
    assert dx_tail_split_taken(Ts, I)
    codes, scales, ws2 = experts("nv", E, O, I, 7660)
    cd, sd = cuda(codes), cuda(scales)
    dYd = [inputs.device_bf16_normal(7670 + e, (T, O)) for e, T in enumerate(Ts)]
    print(f"[moe dx split] nv bf16 O={O} I={I} experts={E} tokens={sum(Ts)}", flush=True)
    dXs = sq.sq_bwd_dx_grouped("nv", dYd, cd, sd, ws2, out_dtype=torch.bfloat16)
    torch.cuda.synchronize()
    for e in range(E):
        one = sq.sq_bwd_dx("nv", dYd[e], cd[e], sd[e], ws2[e], out_dtype=torch.bfloat16)
        assert torch.equal(one, dXs[e]), (e, Ts[e])


def dx_tail_split_taken(Ts, I, cus=256):
    """Whether grouped dX (128 x 128 tiles) moves the short last token tiles
    of its experts to a 64 x 256 launch: when the moved tiles' rounds (two
    workgroups per CU, whole rounds, 1.15 times a 128 x 128 tile) and the
    kept tiles' take less than all tiles kept whole."""
    cols, cols_thin = (I + 127) // 128, (I + 255) // 256
    whole = sum((T + 127) // 128 for T in Ts) * cols
    kept = sum((T // 128 if 0 < T % 128 <= 64 else (T + 127) // 128) for T in Ts) * cols
    moved = sum(cols_thin for T in Ts if 0 < T % 128 <= 64)
    slots = 2 * cus
    return moved > 0 and kept / slots + 1.15 * ((moved + slots - 1) // slots) < whole / slots


# Grouped dS of short token sums runs each workgroup's share of the tiles as
# one pipeline (tiles of 1 to 5 token stages back to back, empty experts
# in between, fewer tiles than XCDs, workgroups with one tile and with many).
STREAM_CASES = [
    ("mx", 128, 128, [5, 0, 64, 65, 1, 0, 200]),          # 1 tile per expert, 7 tiles
    ("nv", 128, 144, [3, 130, 0, 66]),                   # 2 tiles per expert, ragged feature tile
    ("mx", 256, 384, [(37 * e) % 150 for e in range(64)]),
    ("nv", 768, 2048, [(97 * e + 13) % 300 for e in range(40)]),
]


@pytest.mark.parametrize("fmt,O,I,Ts", STREAM_CASES, ids=lambda x: str(x)[:40])
def test_streamed_dscale_tile_sequences(sq, fmt, O, I, Ts):
    codes, scales, ws2 = experts(fmt, len(Ts), O, I, 8100 + O + I)
    cd = cuda(codes)
    Xd = [inputs.device_bf16_normal(8200 + e, (T, I)) for e, T in enumerate(Ts)]
    dYd = [inputs.device_bf16_normal(8300 + e, (T, O)) for e, T in enumerate(Ts)]
    print(f"[moe stream ds] fmt={fmt} O={O} I={I} experts={len(Ts)} T={Ts[:8]}...", flush=True)
    dSs = sq.sq_bwd_dscale_grouped(fmt, Xd, dYd, cd)
    torch.cuda.synchronize()
    compared = 0
    for e, T in enumerate(Ts):
        if T == 0:
            assert torch.count_nonzero(dSs[e]).item() == 0
            continue
        compared += single_dscale_equal(sq, fmt, Xd[e], dYd[e], cd[e], dSs[e])
    assert compared >= len([T for T in Ts if T]) // 2
    g = inputs.rng(8400 + O)
    for e in sorted(set(g.choice(len(Ts), 4, replace=False).tolist())):
        if Ts[e] == 0:
            continue
        X, dY = Xd[e].float().cpu().numpy(), dYd[e].float().cpu().numpy()
        W = linear.dequant(fmt, codes[e], scales[e], ws2[e])
        check_elements(fmt, X, dY, codes[e], W, dS=dSs[e].cpu().numpy(), what=f"expert {e} T={Ts[e]}")
