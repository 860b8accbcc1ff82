"""GPU parity of sq_fwd / sq_bwd_dx / sq_bwd_dscale against the oracle.

Small and ragged shapes are compared on full outputs; full-size 8B shapes
(and the stacked q/k/v and gate/up projections) on 16 seeded rows and 16
seeded columns of every output, half of them drawn from the last 2048 rows or
columns, where a grid ending in a partial wave runs its second launch of half
tiles.  Two gates apply to every compared fp32 output: the normwise relative
error <= 2e-3 that the target sets for bf16 inputs with fp32 accumulation,
and a per-element bound of twice the fp32 summation bound gamma_K * sum|terms|
(tests/parity_check.py), which a single wrong element fails.  The full-size
checks add the exact identity sum(eff * dS) = <dY, Y> = <X, dX>."""

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
    got = np.asarray(got, np.float64)
    den = np.linalg.norm(ref)
    return float(np.linalg.norm(got - ref) / (den if den > 0 else 1.0))


def make_layer(fmt, T, O, I, seed, mx_exp=(-8, -3)):
    G = I // codec.BLOCK[fmt]
    X = inputs.bf16_normal(seed, (T, I))
    dY = inputs.bf16_normal(seed + 1, (T, O))
    codes = inputs.codes_uniform(seed + 2, O, I)
    if fmt == "mx":
        sb = inputs.e8m0_uniform_exponents(seed + 3, O, G, *mx_exp)
        ws2 = 1.0
    else:
        sb = inputs.e4m3_abs_normal(seed + 3, O, G)
        ws2 = float(np.float32(1.0 / 448.0))
    return X, dY, codes, sb, ws2


def to_dev(X, dY, codes, sb):
    return (X.cuda(), dY.cuda(), torch.from_numpy(codes).cuda(), torch.from_numpy(sb).cuda())


def run_all(sq, fmt, X, dY, codes, sb, ws2, out_dtype=torch.float32):
    print(f"[gemm] fmt={fmt} T={X.shape[0]} O={codes.shape[0]} I={X.shape[1]} out={out_dtype}", flush=True)
    dX_, dY_, c_, s_ = to_dev(X, dY, codes, sb)
    Y = sq.sq_fwd(fmt, dX_, c_, s_, ws2, out_dtype)
    dXo = sq.sq_bwd_dx(fmt, dY_, c_, s_, ws2, out_dtype)
    dS = sq.sq_bwd_dscale(fmt, dX_, dY_, c_)
    torch.cuda.synchronize()
    return Y.float().cpu().numpy(), dXo.float().cpu().numpy(), dS.cpu().numpy()


SHAPES = [
    ("mx", 64, 256, 512),       # the tiny MXFP4 workload
    ("nv", 64, 256, 512),
    ("mx", 300, 264, 416),      # several tiles and a ragged tail in every dimension
    ("nv", 300, 264, 208),
    ("mx", 1, 8, 32),           # smallest legal layer
    ("nv", 5, 8, 16),
    ("mx", 129, 136, 160),
    ("nv", 257, 520, 1040),
    # at least 256 workgroups of 256 x 256, so the large tile runs, with
    # ragged edges: forward, dX and dS in turn
    ("mx", 4100, 4104, 64),
    ("nv", 4100, 64, 4112),
    ("mx", 96, 4104, 4128),
    ("nv", 80, 4104, 4112),
    # few tiles and many token stages: dS splits the token sum (workspace)
    ("mx", 1000, 264, 512),
    ("nv", 700, 520, 256),
    # the MXFP4 forward's small tile with its four-stage pipeline over 16 and
    # 32 stages (its last stages wait for every load)
    ("mx", 256, 256, 1024),
    ("mx", 520, 264, 2048),
    # 256 x 256 grids ending in a short partial wave of whole tile-columns
    # (forward, dX) or tile-rows (dS), with ragged edges: those go to a second
    # launch of 256 x 128 or 128 x 256 tiles
    ("mx", 4096, 4360, 64),
    ("nv", 4096, 4360, 64),
    ("nv", 4096, 64, 4368),
    ("mx", 64, 4096, 4384),
    ("nv", 64, 4096, 4368),
    ("mx", 64, 4360, 4096),
    ("nv", 64, 4360, 4096),
    # the same dS half tiles over 4 token stages, so their three-stage
    # pipeline reaches its steady-state waits (128 x 256 half tiles for the
    # last input-feature rows, 256 x 128 for the last output columns)
    ("mx", 256, 4360, 4096),
    ("nv", 256, 4360, 4096),
    ("mx", 256, 4096, 4384),
    ("nv", 256, 4096, 4368),
]


def abs_sums(fmt, Xd, dYd, codes, W):
    """sum_k |terms| of every output element of Y, dX and dS."""
    aX, adY, aW = np.abs(Xd), np.abs(dYd), np.abs(W)
    B = codec.BLOCK[fmt]
    O, I = W.shape
    aS = (np.abs(linear.code_values(codes)) * (adY.T @ aX)).reshape(O, I // B, B).sum(axis=2)
    return aX @ aW.T, adY @ aW, aS


def depths(fmt, T, O, I):
    """Roundings per output element of Y, dX, dS (the K sums plus the NVFP4
    epilogue multiply; dS adds the code multiply and the block sum)."""
    return I + 2, O + 2, T + codec.BLOCK[fmt] + 2


@pytest.mark.parametrize("fmt,T,O,I", SHAPES)
def test_parity_full_outputs(sq, fmt, T, O, I):
    X, dY, codes, sb, ws2 = make_layer(fmt, T, O, I, seed=1000 + T + O + I)
    Y, dX, dS = run_all(sq, fmt, X, dY, codes, sb, ws2)
    Xd, dYd = X.double().numpy(), dY.double().numpy()
    W = linear.dequant(fmt, codes, sb, ws2)
    eY = normwise(Y, linear.forward(Xd, W))
    eX = normwise(dX, linear.backward_dx(dYd, W))
    rS = linear.backward_dscale(fmt, Xd, dYd, codes)
    eS = normwise(dS, rS)
    print(f"  normwise errors Y {eY:.2e} dX {eX:.2e} dS {eS:.2e}")
    assert eY <= TOL and eX <= TOL and eS <= TOL
    aY, aXo, aS = abs_sums(fmt, Xd, dYd, codes, W)
    kY, kX, kS = depths(fmt, T, O, I)
    assert_elements(Y, linear.forward(Xd, W), aY, kY, "Y")
    assert_elements(dX, linear.backward_dx(dYd, W), aXo, kX, "dX")
    assert_elements(dS, rS, aS, kS, "dS")


@pytest.mark.parametrize("fmt", ["mx", "nv"])
def test_bf16_outputs_within_one_ulp(sq, fmt):
    T, O, I = 192, 264, 416 if fmt == "mx" else 400
    X, dY, codes, sb, ws2 = make_layer(fmt, T, O, I, seed=2000)
    Y, dX, _ = run_all(sq, fmt, X, dY, codes, sb, ws2, torch.bfloat16)
    W = linear.dequant(fmt, codes, sb, ws2)
    for got, ref in ((Y, linear.forward(X.double().numpy(), W)), (dX, linear.backward_dx(dY.double().numpy(), W))):
        ref32 = ref.astype(np.float32)
        ref_bf = torch.from_numpy(ref32).to(torch.bfloat16).float().numpy()
        ulp = np.abs(np.spacing(ref_bf.astype(np.float32)) * 65536.0)       # bf16 ulp = 2^16 fp32 ulps
        assert np.all(np.abs(got - ref_bf) <= ulp + 1e-30)
        assert normwise(got, ref) <= 4e-3


@pytest.mark.parametrize("fmt,T,O,I", [("mx", 600, 520, 544), ("nv", 520, 776, 528), ("mx", 4096, 4096, 4096)])
def test_bf16_outputs_are_rounded_f32_outputs(sq, fmt, T, O, I):
    """Full 256 x 256 output tiles leave through the staged 16-byte store path,
    ragged ones through per-element stores; both must equal the fp32 result of
    the same contraction rounded to nearest even."""
    X, dY, codes, sb, ws2 = make_layer(fmt, T, O, I, seed=2100 + T)
    Y32, dX32, _ = run_all(sq, fmt, X, dY, codes, sb, ws2, torch.float32)
    Y16, dX16, _ = run_all(sq, fmt, X, dY, codes, sb, ws2, torch.bfloat16)
    for got, f32 in ((Y16, Y32), (dX16, dX32)):
        want = torch.from_numpy(f32).to(torch.bfloat16).float().numpy()
        assert np.array_equal(got, want)


@pytest.mark.parametrize("T,O,I", [(300, 264, 1024), (4100, 4104, 512), (64, 256, 512), (130, 72, 1536),
                                   (4096, 4360, 512)])
def test_mx_forward_both_dequant_paths(sq, T, O, I):
    """An MXFP4 forward with 16-byte aligned codes and scales and I a multiple
    of 512 dequantises each wave's operand in registers; codes that are only
    4-byte aligned take the path that dequantises W once into LDS.  Both
    match the oracle."""
    X, dY, codes, sb, ws2 = make_layer("mx", T, O, I, seed=2300 + T)
    Xc, sc = X.cuda(), torch.from_numpy(sb).cuda()
    c16 = torch.from_numpy(codes).cuda()
    buf = torch.empty(codes.size + 16, dtype=torch.uint8, device="cuda")
    c4 = buf[4:4 + codes.size].view(codes.shape)
    c4.copy_(c16)
    assert c16.data_ptr() % 16 == 0 and c4.data_ptr() % 16 == 4
    print(f"[gemm] mx forward, both dequant paths, T={T} O={O} I={I}", flush=True)
    ya = sq.sq_fwd("mx", Xc, c16, sc).cpu().numpy()
    yb = sq.sq_fwd("mx", Xc, c4, sc).cpu().numpy()
    ref = linear.forward(X.double().numpy(), linear.dequant("mx", codes, sb, ws2))
    ea, eb = normwise(ya, ref), normwise(yb, ref)
    print(f"  normwise errors: registers {ea:.2e}, LDS {eb:.2e}")
    assert ea <= TOL and eb <= TOL
    W = linear.dequant("mx", codes, sb, ws2)
    absY = np.abs(X.double().numpy()) @ np.abs(W).T
    assert_elements(ya, ref, absY, I + 2, "Y (registers)")
    assert_elements(yb, ref, absY, I + 2, "Y (LDS)")


def test_zero_tokens_gives_zero_dscale(sq):
    O, I = 64, 128
    codes = torch.from_numpy(inputs.codes_uniform(5, O, I)).cuda()
    X = torch.empty((0, I), dtype=torch.bfloat16, device="cuda")
    dY = torch.empty((0, O), dtype=torch.bfloat16, device="cuda")
    dS = torch.full((O, I // 32), 7.0, device="cuda")
    sq.sq_bwd_dscale("mx", X, dY, codes, dS=dS)
    torch.cuda.synchronize()
    assert torch.count_nonzero(dS).item() == 0


def test_dscale_deterministic_and_scale_independent(sq):
    fmt, T, O, I = "mx", 333, 136, 320
    X, dY, codes, _, _ = make_layer(fmt, T, O, I, seed=3000)
    Xc, dYc, cc = X.cuda(), dY.cuda(), torch.from_numpy(codes).cuda()
    a = sq.sq_bwd_dscale(fmt, Xc, dYc, cc)
    b = sq.sq_bwd_dscale(fmt, Xc, dYc, cc)
    torch.cuda.synchronize()
    assert torch.equal(a, b)


def test_split_dscale_deterministic(sq):
    """The split token sum adds its partial planes in a fixed order."""
    fmt, T, O, I = "mx", 1000, 264, 512
    assert sq.sq_bwd_dscale_workspace(fmt, T, O, I) > 0
    X, dY, codes, _, _ = make_layer(fmt, T, O, I, seed=3200)
    Xc, dYc, cc = X.cuda(), dY.cuda(), torch.from_numpy(codes).cuda()
    a = sq.sq_bwd_dscale(fmt, Xc, dYc, cc)
    b = sq.sq_bwd_dscale(fmt, Xc, dYc, cc)
    torch.cuda.synchronize()
    assert torch.equal(a, b)


def test_nan_scale_propagates(sq):
    fmt, T, O, I = "mx", 32, 64, 128
    X, dY, codes, sb, ws2 = make_layer(fmt, T, O, I, seed=3100)
    sb = sb.copy()
    sb[3, 1] = 0xFF                                          # NaN scale in row 3, block 1
    codes = codes.copy()
    codes[3, 16:32] = 0x11                                   # nonzero codes in that block
    Y, _, _ = run_all(sq, fmt, X, dY, codes, sb, ws2)
    assert np.all(np.isnan(Y[:, 3]))
    assert np.all(np.isfinite(np.delete(Y, 3, axis=1)))


def _pick(g, n, total, tail=2048):
    """n distinct indices below total: half from the last `tail`, half from the rest."""
    lo = max(total - tail, 0)
    a = g.choice(np.arange(lo, total), n // 2, replace=False)
    rest = np.setdiff1d(np.arange(total), a)
    b = g.choice(rest, n - n // 2, replace=False)
    return np.sort(np.concatenate([a, b]))


def _sampled_check(sq, fmt, T, O, I, seed, n=16):
    """16 rows and 16 columns of Y, dX and dS against the oracle computed for
    just those elements, each under both gates, plus the full-output identity."""
    X, dY, codes, sb, ws2 = make_layer(fmt, T, O, I, seed)
    if fmt == "mx":
        sb = inputs.e8m0_normal_exponents(seed + 3, O, I // 32, -6.0, 1.5)
    B = codec.BLOCK[fmt]
    G = I // B
    print(f"[gemm] sampled parity fmt={fmt} T={T} O={O} I={I}", flush=True)
    Xc, dYc, cc, sc = to_dev(X, dY, codes, sb)
    Yg = sq.sq_fwd(fmt, Xc, cc, sc, ws2, torch.float32)
    dXg = sq.sq_bwd_dx(fmt, dYc, cc, sc, ws2, torch.float32)
    dSg = sq.sq_bwd_dscale(fmt, Xc, dYc, cc)
    torch.cuda.synchronize()
    g = inputs.rng(seed + 99)
    t_rows, o_cols, i_cols = _pick(g, n, T), _pick(g, n, O), _pick(g, n, I)
    o_rows, b_cols = _pick(g, n, O), _pick(g, n, G, 2048 // B)

    def take_rows(t, idx):
        return t[torch.from_numpy(idx).cuda()].cpu().numpy()

    def take_cols(t, idx):
        return t[:, torch.from_numpy(idx).cuda()].cpu().numpy()

    W = linear.dequant(fmt, codes, sb, ws2)
    aW = np.abs(W)
    Xd, dYd = X.double().numpy(), dY.double().numpy()
    aX, adY = np.abs(Xd), np.abs(dYd)
    kY, kX, kS = depths(fmt, T, O, I)
    errs = []

    def gate(got, ref, absref, depth, what):
        errs.append(normwise(got, ref))
        assert errs[-1] <= TOL, (what, errs[-1])
        assert_elements(got, ref, absref, depth, what)

    # Y rows t and columns o
    gate(take_rows(Yg, t_rows), linear.forward(Xd[t_rows], W), aX[t_rows] @ aW.T, kY, "Y rows")
    gate(take_cols(Yg, o_cols), linear.forward(Xd, W[o_cols]), aX @ aW[o_cols].T, kY, "Y columns")
    # dX rows t and columns i
    gate(take_rows(dXg, t_rows), linear.backward_dx(dYd[t_rows], W), adY[t_rows] @ aW, kX, "dX rows")
    gate(take_cols(dXg, i_cols), linear.backward_dx(dYd, W[:, i_cols]), adY @ aW[:, i_cols], kX, "dX columns")
    # dS rows o (all blocks of those outputs) and block columns b (all outputs)
    cv = np.abs(linear.code_values(codes[o_rows]))
    aS = (cv * (adY[:, o_rows].T @ aX)).reshape(n, G, B).sum(axis=2)
    gate(take_rows(dSg, o_rows), linear.backward_dscale(fmt, Xd, dYd[:, o_rows], codes[o_rows]), aS, kS, "dS rows")
    ref_cols, abs_cols = [], []
    for b in b_cols:
        cb = codes[:, b * B // 2:(b + 1) * B // 2]
        ref_cols.append(linear.backward_dscale(fmt, Xd[:, b * B:(b + 1) * B], dYd, cb)[:, 0])
        abs_cols.append((np.abs(linear.code_values(cb)) * (adY.T @ aX[:, b * B:(b + 1) * B])).sum(axis=1))
    gate(take_cols(dSg, b_cols), np.stack(ref_cols, 1), np.stack(abs_cols, 1), kS, "dS block columns")

    # sum(eff * dS) = <dY, Y> = <X, dX> over the full outputs, in fp64 on the device
    eff = torch.from_numpy(codec.effective_scales(fmt, sb, ws2)).cuda()
    a = float((eff * dSg.double()).sum())
    b_ = float((dYc.double() * Yg.double()).sum())
    c = float((Xc.double() * dXg.double()).sum())
    scale = float(torch.sqrt((dYc.double() ** 2).sum() * (Yg.double() ** 2).sum()))
    print(f"  sampled normwise errors (Y r/c, dX r/c, dS r/c) {' '.join(f'{e:.1e}' for e in errs)}; "
          f"identity {a:.6e} {b_:.6e} {c:.6e}")
    assert abs(a - b_) <= TOL * scale and abs(c - b_) <= TOL * scale


def test_parity_8b_attention_projection_mx(sq):
    """4096 x 4096 MXFP4 projection, 4096 tokens, exponents rint(N(-6, 1.5))."""
    _sampled_check(sq, "mx", 4096, 4096, 4096, seed=2000)


def test_parity_8b_key_value_projection_mx(sq):
    """1024 x 4096 MXFP4 key/value projection, 4096 tokens: the forward and
    dS grids are too small for the large tile and take the small one."""
    _sampled_check(sq, "mx", 4096, 1024, 4096, seed=2500)


@pytest.mark.parametrize("O,I", [(14336, 4096), (4096, 14336), (6144, 4096), (28672, 4096)])
def test_parity_8b_mlp_and_stacked_mx(sq, O, I):
    """The MXFP4 shapes of the 8B model step at 4096 tokens: gate/up
    (14336 x 4096) and down (4096 x 14336), whose grids end in a half wave of
    whole tile-columns or tile-rows, and the stacked q/k/v (6144 x 4096) and
    gate/up (28672 x 4096) weights of the fused-projection layout."""
    _sampled_check(sq, "mx", 4096, O, I, seed=4000 + O + I)


@pytest.mark.parametrize("fmt,O,I", [("mx", 14336, 4096), ("mx", 4096, 14336), ("nv", 4096, 14336)])
def test_tail_split_equals_slices(sq, fmt, O, I):
    """8B MLP shapes at 4096 tokens (896 tiles of 256 x 256: three whole waves
    and a half wave, which runs as 256 x 128 tiles): the forward and dX equal,
    bit for bit, the same products over 2048-wide slices of W, which take the
    128 x 128 tile (each output element is summed in K order either way)."""
    T = 4096
    X, dY, codes, sb, ws2 = make_layer(fmt, T, O, I, seed=3500 + O)
    B = codec.BLOCK[fmt]
    Xd, dYd = X.cuda(), dY.cuda()
    cd, sd = torch.from_numpy(codes).cuda(), torch.from_numpy(sb).cuda()
    Y = sq.sq_fwd(fmt, Xd, cd, sd, ws2, out_dtype=torch.float32)
    dX = sq.sq_bwd_dx(fmt, dYd, cd, sd, ws2, out_dtype=torch.float32)
    torch.cuda.synchronize()
    for o0 in range(0, O, 2048):
        Ys = sq.sq_fwd(fmt, Xd, cd[o0:o0 + 2048].contiguous(), sd[o0:o0 + 2048].contiguous(), ws2,
                       out_dtype=torch.float32)
        torch.cuda.synchronize()
        assert torch.equal(Y[:, o0:o0 + 2048], Ys), o0
    for i0 in range(0, I, 2048):
        c = cd[:, i0 // 2:(i0 + 2048) // 2].contiguous()
        s_ = sd[:, i0 // B:(i0 + 2048) // B].contiguous()
        dXs = sq.sq_bwd_dx(fmt, dYd, c, s_, ws2, out_dtype=torch.float32)
        torch.cuda.synchronize()
        assert torch.equal(dX[:, i0:i0 + 2048], dXs), i0


@pytest.mark.parametrize("O,I", [(14336, 4096), (4096, 14336)])
def test_parity_8b_mlp_nv(sq, O, I):
    """NVFP4 gate/up (14336 x 4096) and down (4096 x 14336), 8192 tokens."""
    _sampled_check(sq, "nv", 8192, O, I, seed=3000 + O)
