"""GPU parity of sq_merge_scales(_grouped) and rtn_quantize against the oracle:
bit-exact bytes, with guard bytes around every written plane, and the code
plane untouched by merges."""

import numpy as np
import pytest
import torch

from conftest import ensure_library, gpu_ready
from oracle import codec, linear, merge, rtn
from paper_2609_04526_amd import inputs

pytestmark = [pytest.mark.gpu, pytest.mark.skipif(not gpu_ready(), reason="needs a GPU")]

GUARD = 256          # bytes of canary on each side (keeps 16-byte alignment)


@pytest.fixture(scope="module")
def sq():
    ensure_library()
    from paper_2609_04526_amd import sq as _sq
    return _sq


def guarded(host_bytes):
    """Device buffer = canary | plane | canary; returns (buffer, plane view)."""
    n = host_bytes.size
    buf = torch.full((n + 2 * GUARD,), 0xA5, dtype=torch.uint8, device="cuda")
    buf[GUARD:GUARD + n] = torch.from_numpy(np.ascontiguousarray(host_bytes).reshape(-1)).cuda()
    return buf, buf[GUARD:GUARD + n]


def guards_intact(buf):
    b = buf.cpu().numpy()
    return bool(np.all(b[:GUARD] == 0xA5) and np.all(b[-GUARD:] == 0xA5))


def test_merge_tiny_mx_perturbed_plane(sq):
    """The tiny MXFP4 workload: 256 x 16 scale plane, +-1 exponent step on 10% of blocks."""
    sb = inputs.e8m0_uniform_exponents(1003, 256, 16, -8, -3)
    d = inputs.e8m0_step_delta(1009, sb, 0.10)
    buf, plane = guarded(sb)
    sq.sq_merge_scales("mx", plane, delta=torch.from_numpy(d.reshape(-1)).cuda())
    torch.cuda.synchronize()
    ref = merge.merge_delta("mx", sb, d)
    assert np.array_equal(plane.cpu().numpy().reshape(sb.shape), ref)
    assert guards_intact(buf)
    assert (ref != sb).sum() == round(0.1 * sb.size)


@pytest.mark.parametrize("fmt,n", [("mx", 4096 * 3 + 20), ("nv", 4096 * 3 + 20), ("nv", 7), ("mx", 1000003)])
def test_merge_delta_random_matches_oracle(sq, fmt, n):
    g = inputs.rng(77 + n)
    if fmt == "mx":
        sb = g.integers(90, 150, size=n).astype(np.uint8)
        eff = np.ldexp(1.0, sb.astype(int) - 127)
        ws2 = 1.0
    else:
        sb = g.integers(0, 0x7F, size=n).astype(np.uint8)
        ws2 = float(np.float32(1 / 448))
        eff = codec.E4M3_TABLE[sb] * ws2
    d = (g.standard_normal(n) * 0.7 * eff).astype(np.float32)
    d[::97] = 0.0
    if fmt == "nv":
        d[5::101] = np.float32(1000 * ws2)        # past the ceiling: clamp, never NaN
    buf, plane = guarded(sb)
    sq.sq_merge_scales(fmt, plane, delta=torch.from_numpy(d).cuda(), ws2=ws2)
    torch.cuda.synchronize()
    got = plane.cpu().numpy()
    ref = merge.merge_delta(fmt, sb, d, ws2)
    assert np.array_equal(got, ref), np.flatnonzero(got != ref)[:10]
    assert guards_intact(buf)


LARGE = 1 << 24       # calls over this many scales in all take the multi-step spans


@pytest.mark.parametrize("fmt,n", [("mx", 8192 * 5 + 3), ("nv", 16384 * 2 + 4100), ("mx", 8192), ("nv", 16384),
                                   ("mx", 1024 * 7 + 1), ("nv", 1024),
                                   ("mx", LARGE + 8192 * 5 + 3), ("nv", LARGE + 16384 * 2 + 4100)])
def test_merge_delta_full_spans_and_tail(sq, fmt, n):
    """Planes of several whole workgroup spans plus a ragged tail: one-step
    spans of 1024 scales below LARGE scales, multi-step spans (8192 MXFP4 or
    16384 NVFP4 scales) above."""
    g = inputs.rng(91 + n)
    sb = g.integers(90, 150, size=n).astype(np.uint8) if fmt == "mx" else g.integers(0, 0x7E, size=n).astype(np.uint8)
    ws2 = 1.0 if fmt == "mx" else float(np.float32(1 / 448))
    eff = codec.effective_scales(fmt, sb, ws2)
    d = (g.standard_normal(n) * eff * 0.7).astype(np.float32)
    buf, plane = guarded(sb)
    sq.sq_merge_scales(fmt, plane, delta=torch.from_numpy(d).cuda(), ws2=ws2)
    torch.cuda.synchronize()
    assert np.array_equal(plane.cpu().numpy(), merge.merge_delta(fmt, sb, d, ws2))
    assert guards_intact(buf)


@pytest.mark.parametrize("n", [32768 * 3 + 100, 32768, 32768 * 2 + 16, 4096 * 5 + 7, LARGE + 32768 * 2 + 100])
def test_swap_full_spans_and_tail(sq, n):
    """Copies of several whole workgroup spans (4 KiB one-step spans below
    LARGE bytes, 32 KiB above) plus a ragged tail."""
    g = inputs.rng(93 + n)
    sb = g.integers(0, 256, size=n).astype(np.uint8)
    src = g.integers(0, 256, size=n).astype(np.uint8)
    buf, plane = guarded(sb)
    sq.sq_merge_scales("mx", plane, src=torch.from_numpy(src).cuda())
    torch.cuda.synchronize()
    assert np.array_equal(plane.cpu().numpy(), src)
    assert guards_intact(buf)


@pytest.mark.parametrize("fmt", ["mx", "nv"])
def test_merge_all_bytes_delta_zero_identity(sq, fmt):
    sb = np.arange(0, 255 if fmt == "mx" else 0x7F, dtype=np.uint8)
    sb = np.tile(sb, 33)
    buf, plane = guarded(sb)
    sq.sq_merge_scales(fmt, plane, delta=torch.zeros(sb.size, device="cuda"), ws2=float(np.float32(1 / 448)))
    torch.cuda.synchronize()
    assert np.array_equal(plane.cpu().numpy(), sb)
    assert guards_intact(buf)


def test_merge_special_values(sq):
    sb = np.array([0, 1, 127, 254, 255, 200, 50, 3] * 4, dtype=np.uint8)
    d = np.array([0.0, -1.0, np.inf, np.nan, 0.0, -np.inf, 1e-40, 3e38] * 4, dtype=np.float32)
    buf, plane = guarded(sb)
    sq.sq_merge_scales("mx", plane, delta=torch.from_numpy(d).cuda())
    torch.cuda.synchronize()
    assert np.array_equal(plane.cpu().numpy(), merge.merge_delta("mx", sb, d))


@pytest.mark.parametrize("ws2", [float(np.float32(1 / 448)), 0.37, 3.0e-3, 2.0 ** -70, 2.0 ** 70])
def test_merge_nv_special_values(sq, ws2):
    """NVFP4: NaN bytes (0x7F, 0xFF), negative bytes, signed zeros, NaN and
    infinite deltas, deltas far past the ceiling and far below zero; ws2 both
    inside and outside the range where the division runs through 1/ws2."""
    w = np.float32(ws2)
    sb = np.array([0x00, 0x80, 0x7F, 0xFF, 0x7E, 0xFE, 0x01, 0x81, 0x38, 0xB8, 0x40, 0x08], dtype=np.uint8)
    ds = np.array([0.0, -0.0, np.nan, -np.nan, np.inf, -np.inf, 3.0e38, -3.0e38, 1e-45, -1e-45,
                   float(w) * 1000, -float(w) * 1000, float(w) * 0.0009765625, -float(w) * 0.0009765625],
                  dtype=np.float32)
    b = np.repeat(sb, ds.size)
    d = np.tile(ds, sb.size)
    b = np.tile(b, 3)
    d = np.tile(d, 3)
    buf, plane = guarded(b)
    print(f"[merge nv special] ws2={ws2} n={b.size}", flush=True)
    sq.sq_merge_scales("nv", plane, delta=torch.from_numpy(d).cuda(), ws2=ws2)
    torch.cuda.synchronize()
    got = plane.cpu().numpy()
    ref = merge.merge_delta("nv", b, d, ws2)
    bad = np.flatnonzero(got != ref)
    assert bad.size == 0, [(int(b[i]), float(d[i]), int(got[i]), int(ref[i])) for i in bad[:8]]
    assert guards_intact(buf)


@pytest.mark.parametrize("ws2", [float(np.float32(1 / 448)), 0.0123, 2.0 ** -60, 5.5e17])
def test_merge_nv_quotients_at_e4m3_midpoints(sq, ws2):
    """NVFP4 deltas that put e2 / ws2 within a few fp32 ulps of every E4M3
    rounding midpoint (and of the values themselves), positive and negative:
    an ulp of error in the division would move bytes across a midpoint."""
    w = np.float32(ws2)
    vals = codec.E4M3_TABLE[:0x7F].astype(np.float64)
    pos = np.unique(vals[vals >= 0])
    mids = (pos[:-1] + pos[1:]) / 2
    targets = np.concatenate([mids, pos, -mids, -pos]).astype(np.float32)
    k = np.arange(-6, 7)
    t = targets[:, None]
    q = (t.astype(np.float64) * (1.0 + k[None, :] * 2.0 ** -23)).astype(np.float32).ravel()
    g = inputs.rng(4242)
    base = g.integers(0, 0x7F, size=q.size).astype(np.uint8)
    e = (codec.E4M3_TABLE[base].astype(np.float32) * w).astype(np.float32)
    e2_target = (q.astype(np.float64) * float(w)).astype(np.float32)
    d = (e2_target.astype(np.float64) - e.astype(np.float64)).astype(np.float32)
    buf, plane = guarded(base)
    print(f"[merge nv midpoints] ws2={ws2} n={base.size}", flush=True)
    sq.sq_merge_scales("nv", plane, delta=torch.from_numpy(d).cuda(), ws2=ws2)
    torch.cuda.synchronize()
    got = plane.cpu().numpy()
    ref = merge.merge_delta("nv", base, d, ws2)
    bad = np.flatnonzero(got != ref)
    assert bad.size == 0, [(int(base[i]), float(d[i]), int(got[i]), int(ref[i])) for i in bad[:8]]
    assert guards_intact(buf)


@pytest.mark.parametrize("rows", [1, 256])
def test_swap_and_grouped_merge_leave_codes_untouched(sq, rows):
    """A model-like set of planes: swap some, merge others, in one grouped call;
    the code planes (held next to them) keep their bytes.  rows = 256 puts the
    call above LARGE scales (multi-step spans)."""
    planes = []
    refs = []
    code_planes = []
    shapes = [("mx", 64, 4096), ("nv", 96, 4096), ("mx", 32, 14336), ("nv", 40, 14336), ("mx", 8, 1024)]
    assert (sum(O * I // codec.BLOCK[f] for f, O, I in shapes) * rows > LARGE) == (rows > 1)
    for k, (fmt, O, I) in enumerate(shapes):
        O *= rows
        B = codec.BLOCK[fmt]
        if fmt == "mx":
            sb = inputs.e8m0_normal_exponents(500 + k, O, I // B, -6, 1.5)
            eff = np.ldexp(1.0, sb.astype(int) - 127)
            ws2 = 1.0
        else:
            sb = inputs.e4m3_abs_normal(500 + k, O, I // B)
            ws2 = float(np.float32(1 / 448))
            eff = codec.E4M3_TABLE[sb] * ws2
        codes = inputs.codes_uniform(600 + k, O, I)
        cbuf, cplane = guarded(codes)
        code_planes.append((cbuf, cplane, codes))
        buf, plane = guarded(sb)
        if k % 2 == 0:
            d = inputs.relative_jitter(700 + k, eff, 0.3)
            planes.append(dict(fmt=fmt, scales=plane, delta=torch.from_numpy(d.reshape(-1)).cuda(), ws2=ws2))
            refs.append((buf, plane, merge.merge_delta(fmt, sb, d, ws2).reshape(-1)))
        else:
            src = inputs.e4m3_abs_normal(800 + k, O, I // B) if fmt == "nv" else \
                inputs.e8m0_normal_exponents(800 + k, O, I // B, -6, 1.5)
            planes.append(dict(fmt=fmt, scales=plane, src=torch.from_numpy(src.reshape(-1)).cuda()))
            refs.append((buf, plane, merge.merge_copy(sb, src).reshape(-1)))
    sq.sq_merge_scales_grouped(planes)
    torch.cuda.synchronize()
    for buf, plane, ref in refs:
        assert np.array_equal(plane.cpu().numpy(), ref)
        assert guards_intact(buf)
    for cbuf, cplane, codes in code_planes:
        assert np.array_equal(cplane.cpu().numpy().reshape(codes.shape), codes)
        assert guards_intact(cbuf)


def test_grouped_merge_many_planes(sq):
    """More planes than one launch takes, with sizes that leave ragged tails."""
    planes, refs = [], []
    for k in range(97):
        n = 16 * (1 + (k * 37) % 700)
        sb = inputs.rng(k).integers(100, 140, size=n).astype(np.uint8)
        d = inputs.relative_jitter(k + 1000, np.ldexp(1.0, sb.astype(int) - 127), 0.8)
        buf, plane = guarded(sb)
        planes.append(dict(fmt="mx", scales=plane, delta=torch.from_numpy(d).cuda()))
        refs.append((buf, plane, merge.merge_delta("mx", sb, d)))
    sq.sq_merge_scales_grouped(planes)
    torch.cuda.synchronize()
    for buf, plane, ref in refs:
        assert np.array_equal(plane.cpu().numpy(), ref)
        assert guards_intact(buf)


def _merged_weight(fmt, O, I, seed):
    """bf16(dequant(W) + B A) with a rank-16 update, the naive merge's input."""
    codes = inputs.codes_uniform(seed, O, I)
    if fmt == "mx":
        sb = inputs.e8m0_normal_exponents(seed + 1, O, I // 32, -6, 1.5)
        ws2 = 1.0
    else:
        sb = inputs.e4m3_abs_normal(seed + 1, O, I // 16)
        ws2 = float(np.float32(1 / 448))
    B, A = inputs.lora_factors(seed + 2, O, I, 16, 0.02)
    W = linear.dequant(fmt, codes, sb, ws2).astype(np.float32) + (B @ A).astype(np.float32)
    Wb = torch.from_numpy(W.astype(np.float32)).to(torch.bfloat16)
    return Wb, codes, sb, ws2


@pytest.mark.parametrize("fmt", ["mx", "nv"])
@pytest.mark.parametrize("tie", ["even", "away"])
@pytest.mark.parametrize("ws2_mode", ["fixed", "recompute"])
def test_rtn_matches_oracle(sq, fmt, tie, ws2_mode):
    if fmt == "mx" and ws2_mode == "recompute":
        pytest.skip("MXFP4 has no per-tensor scalar")
    O, I = 264, 1024
    Wb, codes, sb, ws2 = _merged_weight(fmt, O, I, seed=4000)
    Wf = Wb.float().numpy()
    tie_c = sq.TIE_EVEN if tie == "even" else sq.TIE_AWAY
    ws2_in = ws2 if ws2_mode == "fixed" else 0.0
    c, s, w2 = sq.rtn_quantize(fmt, Wb.cuda(), tie_c, ws2_in)
    torch.cuda.synchronize()
    rc, rs, rw = rtn.quantize(fmt, Wf, tie, ws2 if ws2_mode == "fixed" else None)
    assert np.array_equal(s.cpu().numpy(), rs)
    assert np.array_equal(c.cpu().numpy(), rc)
    if fmt == "nv":
        assert w2.cpu().numpy()[0] == rw
    # codes moved relative to the base plane (the naive merge rewrites codes)
    print(f"  {fmt} {tie} {ws2_mode}: code bytes changed vs base {np.mean(rc != codes):.3f}")


@pytest.mark.parametrize("fmt", ["mx", "nv"])
def test_rtn_8b_gate_projection_sampled_rows(sq, fmt):
    """14336 x 4096 merged weight (the gate projection): the whole plane is
    re-quantised on the GPU, and seeded rows are checked byte for byte against
    the oracle, for both tie rules (and, for NVFP4, the recomputed ws2, which the
    oracle takes from the whole tensor)."""
    O, I = 14336, 4096
    Wb, codes, sb, ws2 = _merged_weight(fmt, O, I, seed=4100)
    Wd = Wb.cuda()
    rows = np.sort(np.concatenate([inputs.rng(4101).choice(O, 47, replace=False), [O - 1]]))
    Wrows = Wb[torch.from_numpy(rows)].float().numpy()
    modes = [("even", sq.TIE_EVEN, ws2), ("away", sq.TIE_AWAY, ws2)]
    if fmt == "nv":
        modes.append(("even", sq.TIE_EVEN, 0.0))
    for tie, tie_c, w_in in modes:
        print(f"[rtn 8b] fmt={fmt} tie={tie} ws2_in={w_in}", flush=True)
        c, s, w2 = sq.rtn_quantize(fmt, Wd, tie_c, w_in)
        torch.cuda.synchronize()
        if fmt == "nv" and w_in == 0.0:
            w_ref = rtn.recompute_ws2(Wb.float().numpy())
            assert w2.cpu().numpy()[0] == w_ref
        else:
            w_ref = w_in if fmt == "nv" else None
        rc, rs, _ = rtn.quantize(fmt, Wrows, tie, w_ref)
        assert np.array_equal(c.cpu().numpy()[rows], rc)
        assert np.array_equal(s.cpu().numpy()[rows], rs)


def test_rtn_ties_and_specials(sq):
    """Exact midpoints of the E2M1 grid and zero / negative-zero weights."""
    O, I = 8, 64
    W = np.zeros((O, I), np.float32)
    mids = np.array([0.25, 0.75, 1.25, 1.75, 2.5, 3.5, 5.0, 6.0], np.float32)
    for o in range(O):
        W[o, :8] = mids
        W[o, 8:16] = -mids
        W[o, 32] = -0.0
        W[o, 33] = 1e-30
    Wb = torch.from_numpy(W).to(torch.bfloat16)
    for tie, tc in (("even", 0), ("away", 1)):
        c, s, _ = sq.rtn_quantize("mx", Wb.cuda(), tc)
        torch.cuda.synchronize()
        rc, rs, _ = rtn.quantize("mx", Wb.float().numpy(), tie)
        assert np.array_equal(s.cpu().numpy(), rs) and np.array_equal(c.cpu().numpy(), rc)


@pytest.mark.parametrize("ws2", [2.0 ** -70, 2.0 ** -64, 3e-3, float(np.float32(1 / 448)), 2.0 ** 64, 2.0 ** 70, 0.0])
def test_rtn_tiny_blocks_and_extreme_ws2(sq, ws2):
    """Block amax values on both sides of 2^-120 (where amax / 6 leaves the
    reciprocal path for a full division), bf16 subnormals, zeros, and a
    per-tensor ws2 inside and outside [2^-55, 2^55] (the range the NVFP4 kernels'
    shortened division assumes; 0: recomputed), in both
    formats against the oracle, for the two nearest rules and round toward
    zero."""
    O, I = 16, 512
    g = inputs.rng(4300)
    W = (g.standard_normal((O, I)) * 0.02).astype(np.float32)
    exps = [-125, -122, -121, -120, -119, -118, -100, -76, -60, -30, 0, 10, 60, 100, 110, 120]
    for o, e in enumerate(exps):
        W[o] *= np.float32(2.0 ** e) / np.float32(0.05)
        W[o, 32:64] = 0.0                                   # an all-zero block
    W[3, 64:96] = np.float32(2.0 ** -131)                   # bf16 subnormal blocks
    W[4, 96:128] = -np.float32(2.0 ** -133)
    Wb = torch.from_numpy(W).to(torch.bfloat16)
    Wf = Wb.float().numpy()
    for fmt in ("mx", "nv"):
        if fmt == "mx" and ws2 != 0.0:
            continue
        ws2_in = float(np.float32(ws2)) if fmt == "nv" else 0.0
        print(f"[rtn tiny] fmt={fmt} ws2={ws2_in}", flush=True)
        for tie, tc in (("even", sq.TIE_EVEN), ("away", sq.TIE_AWAY)):
            c, s, w2 = sq.rtn_quantize(fmt, Wb.cuda(), tc, ws2_in)
            torch.cuda.synchronize()
            rc, rs, rw = rtn.quantize(fmt, Wf, tie, ws2_in if (fmt == "nv" and ws2_in > 0) else None)
            assert np.array_equal(s.cpu().numpy(), rs), np.argwhere(s.cpu().numpy() != rs)[:5]
            assert np.array_equal(c.cpu().numpy(), rc)
            if fmt == "nv":
                got = w2.cpu().numpy()[0]
                assert got == rw or (np.isnan(got) and np.isnan(rw))
        # round toward zero takes the same block path for NVFP4
        ref_ws2 = ws2_in if (fmt == "nv" and ws2_in > 0) else None
        c, s, w2 = sq.rtn_quantize_rule(fmt, Wb.cuda(), "rtz", ws2_in, 0)
        torch.cuda.synchronize()
        rc, rs, rw = rtn.quantize_rule(fmt, Wf, "rtz", ref_ws2, 0)
        assert np.array_equal(s.cpu().numpy(), rs) and np.array_equal(c.cpu().numpy(), rc)
        if w2 is not None:
            got = w2.cpu().numpy()[0]
            assert got == rw or (np.isnan(got) and np.isnan(rw))


@pytest.mark.parametrize("ws2", [float(np.float32(1 / 448)), 2.0 ** -9, 0.0123])
def test_rtn_nv_quotients_on_change_points(sq, ws2):
    """NVFP4 blocks whose quotients w / eff fall on, or within a few fp32 steps
    of, the values where an E2M1 code changes (midpoints 0.25 .. 5, grid points
    0.5 .. 6), both signs: blocks whose scale is a power of two (scale bytes
    of mantissa 1.75 with ws2 = fp32(1/448), every byte of mantissa 1 with
    ws2 = 2^-9), where the product with the reciprocal is exact and lands on
    the midpoints themselves, and blocks of every other scale byte, where
    bf16 weights next to V eff give quotients a few steps from V.  Codes and
    scales under nearest even, nearest away and toward zero equal the
    oracle's byte for byte."""
    w2 = np.float32(ws2)
    change = np.array([0.25, 0.75, 1.25, 1.75, 2.5, 3.5, 5.0, 0.5, 1.0, 1.5, 2.0, 3.0, 4.0, 6.0])
    g = inputs.rng(4400)
    O, I = 96, 512
    G = I // 16
    W = np.zeros((O, G, 16), np.float32)
    pos = np.array([b for b in range(0x08, 0x7F) if 1e-30 < codec.E4M3_TABLE[b] * float(w2)])
    for o in range(O):
        for gb in range(G):
            s = codec.E4M3_TABLE[g.choice(pos)]
            eff = np.float32(s * float(w2))
            # the block amax, 6 eff rounded to bf16, picks back s (or a neighbour)
            blk = [bf16_round(6.0 * float(eff))]
            for k in range(15):
                v = change[g.integers(0, change.size)] * float(eff)
                v *= 1.0 + g.integers(-4, 5) * 2.0 ** -9 if g.integers(0, 3) == 0 else 1.0
                blk.append(bf16_round(v) * (1 if g.integers(0, 2) else -1))
            W[o, gb] = np.array(blk, np.float32)[g.permutation(16)]
    W = W.reshape(O, I)
    Wb = torch.from_numpy(W).to(torch.bfloat16)
    Wf = Wb.float().numpy()
    ws2_in = float(w2)
    print(f"[rtn change points] ws2={ws2_in}", flush=True)
    for tie, tc in (("even", sq.TIE_EVEN), ("away", sq.TIE_AWAY)):
        c, s_, _ = sq.rtn_quantize("nv", Wb.cuda(), tc, ws2_in)
        torch.cuda.synchronize()
        rc, rs, _ = rtn.quantize("nv", Wf, tie, ws2_in)
        assert np.array_equal(s_.cpu().numpy(), rs)
        bad = np.argwhere(c.cpu().numpy() != rc)
        assert bad.size == 0, (tie, bad[:5])
    c, s_, _ = sq.rtn_quantize_rule("nv", Wb.cuda(), "rtz", ws2_in, 0)
    torch.cuda.synchronize()
    rc, rs, _ = rtn.quantize_rule("nv", Wf, "rtz", ws2_in, 0)
    assert np.array_equal(s_.cpu().numpy(), rs) and np.array_equal(c.cpu().numpy(), rc)


def bf16_round(x):
    """x rounded to bf16 (nearest even), as a float."""
    return float(torch.tensor([x], dtype=torch.float32).to(torch.bfloat16).float()[0])


def test_rtn_delta_zero_fixed_point(sq):
    O, I = 64, 256
    codes = inputs.codes_uniform(4100, O, I)
    nib = codec.unpack_nibbles(codes)
    nib[:, ::32] = 7
    codes = codec.pack_nibbles(nib)
    sb = inputs.e8m0_uniform_exponents(4101, O, I // 32, -8, -3)
    W = torch.from_numpy(linear.dequant("mx", codes, sb).astype(np.float32)).to(torch.bfloat16)
    c, s, _ = sq.rtn_quantize("mx", W.cuda(), sq.TIE_EVEN)
    torch.cuda.synchronize()
    assert np.array_equal(s.cpu().numpy(), sb) and np.array_equal(c.cpu().numpy(), codes)
