"""GPU parity of rtn_quantize_rule (the deploy-side re-quantisers: round toward
zero, stochastic rounding from Philox4x64-10, one whole-tensor scale) against
the oracle: bit-exact code and scale bytes and the same ws2."""

import numpy as np
import pytest
import torch

from conftest import ensure_library, gpu_ready
from oracle import codec, linear, rtn
from paper_2609_04526_amd import inputs

pytestmark = [pytest.mark.gpu, pytest.mark.skipif(not gpu_ready(), reason="needs a GPU")]

RULES = ["rtz", "stochastic", "whole_tensor"]


@pytest.fixture(scope="module")
def sq():
    ensure_library()
    from paper_2609_04526_amd import sq as _sq
    return _sq


def _merged_weight(fmt, O, I, seed):
    """bf16(dequant(W) + B A) with a rank-16 update: the continuous merged tensor
    a deploy quantiser receives."""
    codes = inputs.codes_uniform(seed, O, I)
    if fmt == "mx":
        sb = inputs.e8m0_normal_exponents(seed + 1, O, I // 32, -6, 1.5)
        ws2 = 1.0
    else:
        sb = inputs.e4m3_abs_normal(seed + 1, O, I // 16)
        ws2 = float(np.float32(1 / 448))
    B, A = inputs.lora_factors(seed + 2, O, I, 16, 0.02)
    W = linear.dequant(fmt, codes, sb, ws2).astype(np.float32) + (B @ A).astype(np.float32)
    return torch.from_numpy(W).to(torch.bfloat16), ws2


def _check(sq, fmt, Wb, rule, ws2_in, seed, ref_ws2):
    c, s, w2 = sq.rtn_quantize_rule(fmt, Wb.cuda(), rule, ws2_in, seed)
    torch.cuda.synchronize()
    rc, rs, rw = rtn.quantize_rule(fmt, Wb.float().numpy(), rule, ref_ws2, seed)
    assert np.array_equal(s.cpu().numpy(), rs)
    assert np.array_equal(c.cpu().numpy(), rc)
    if w2 is not None:
        got = w2.cpu().numpy()[0]
        assert got == rw or (np.isnan(got) and np.isnan(rw))
    return c, s


@pytest.mark.parametrize("fmt", ["mx", "nv"])
@pytest.mark.parametrize("rule", RULES)
@pytest.mark.parametrize("ws2_mode", ["fixed", "recompute"])
def test_rule_matches_oracle(sq, fmt, rule, ws2_mode):
    """264 x 1056: 34848 chunks, a ragged last workgroup."""
    if fmt == "mx" and ws2_mode == "recompute":
        pytest.skip("MXFP4 has no per-tensor scalar")
    O, I = 264, 1056
    Wb, ws2 = _merged_weight(fmt, O, I, seed=5000)
    fixed = fmt == "nv" and ws2_mode == "fixed"
    print(f"[rule] fmt={fmt} rule={rule} ws2={ws2_mode}", flush=True)
    _check(sq, fmt, Wb, rule, ws2 if fixed else 0.0, 12345, ws2 if fixed else None)


@pytest.mark.parametrize("fmt", ["mx", "nv"])
@pytest.mark.parametrize("tie", ["even", "away"])
def test_nearest_rules_equal_rtn_quantize(sq, fmt, tie):
    Wb, ws2 = _merged_weight(fmt, 96, 512, seed=5100)
    Wd = Wb.cuda()
    c0, s0, _ = sq.rtn_quantize(fmt, Wd, sq.TIE_EVEN if tie == "even" else sq.TIE_AWAY, ws2)
    c1, s1, _ = sq.rtn_quantize_rule(fmt, Wd, tie, ws2)
    torch.cuda.synchronize()
    assert torch.equal(c0, c1) and torch.equal(s0, s1)


@pytest.mark.parametrize("seed", [0, 1, 0xFFFFFFFFFFFFFFFF])
def test_stochastic_seeds(sq, seed):
    """Each seed matches the oracle, and two seeds give different codes."""
    Wb, _ = _merged_weight("mx", 64, 512, seed=5200)
    c, _ = _check(sq, "mx", Wb, "stochastic", 0.0, seed, None)
    c2, _, _ = sq.rtn_quantize_rule("mx", Wb.cuda(), "stochastic", 0.0, seed ^ 0x5A5A)
    torch.cuda.synchronize()
    assert not torch.equal(c, c2)


@pytest.mark.parametrize("rule", ["rtz", "stochastic"])
def test_on_grid_weights_do_not_move(sq, rule):
    """Dequantised on-grid weights (every block holding a magnitude-6 code, so the
    scale rule returns the same byte) re-quantise to the same bytes."""
    O, I = 64, 512
    codes = inputs.codes_uniform(5300, O, I)
    nib = codec.unpack_nibbles(codes)
    nib[:, ::32] = 7
    codes = codec.pack_nibbles(nib)
    sb = inputs.e8m0_uniform_exponents(5301, O, I // 32, -8, -3)
    W = torch.from_numpy(linear.dequant("mx", codes, sb).astype(np.float32)).to(torch.bfloat16)
    c, s, _ = sq.rtn_quantize_rule("mx", W.cuda(), rule, 0.0, 77)
    torch.cuda.synchronize()
    assert np.array_equal(s.cpu().numpy(), sb) and np.array_equal(c.cpu().numpy(), codes)


def test_specials(sq):
    """Midpoints, zeros, signed zeros, tiny values and a NaN block; then a NaN
    anywhere makes the whole-tensor scale NaN for every block."""
    O, I = 8, 64
    W = np.zeros((O, I), np.float32)
    mids = np.array([0.25, 0.75, 1.25, 1.75, 2.5, 3.5, 5.0, 6.0], np.float32)
    for o in range(O):
        W[o, :8] = mids
        W[o, 8:16] = -mids * 0.999
        W[o, 32] = -0.0
        W[o, 33] = 1e-30
        W[o, 34] = -3e-3
    W[5, 40] = np.nan
    Wb = torch.from_numpy(W).to(torch.bfloat16)
    for fmt in ("mx", "nv"):
        for rule in RULES:
            fixed = fmt == "nv" and rule != "whole_tensor"
            _check(sq, fmt, Wb, rule, float(np.float32(1 / 448)) if fixed else 0.0, 3,
                   float(np.float32(1 / 448)) if fixed else None)


@pytest.mark.parametrize("fmt", ["mx", "nv"])
def test_8b_gate_projection_sampled_rows(sq, fmt):
    """14336 x 4096: the whole plane on the GPU, seeded rows checked byte for
    byte (the stochastic rule's element counter runs past 2^25; the
    whole-tensor rule needs the whole tensor's amax, taken by the oracle)."""
    O, I = 14336, 4096
    Wb, ws2 = _merged_weight(fmt, O, I, seed=5400)
    Wd = Wb.cuda()
    rows = np.sort(np.concatenate([inputs.rng(5401).choice(O, 31, replace=False), [O - 1]]))
    Wf = Wb.float().numpy()
    seed = 0x1234_5678_9ABC_DEF0
    for rule in ("rtz", "stochastic"):
        print(f"[rule 8b] fmt={fmt} rule={rule}", flush=True)
        c, s, _ = sq.rtn_quantize_rule(fmt, Wd, rule, ws2, seed)
        torch.cuda.synchronize()
        cc, sc = c.cpu().numpy(), s.cpu().numpy()
        for o in rows.tolist():
            rc, rs, _ = rtn.quantize_rule(fmt, Wf[o:o + 1], rule, ws2 if fmt == "nv" else None, seed, row0=o)
            assert np.array_equal(sc[o:o + 1], rs) and np.array_equal(cc[o:o + 1], rc)
    print(f"[rule 8b] fmt={fmt} rule=whole_tensor", flush=True)
    c, s, w2 = sq.rtn_quantize_rule(fmt, Wd, "whole_tensor", 0.0)
    torch.cuda.synchronize()
    amax = np.float32(np.max(np.abs(Wf)))
    sc = s.cpu().numpy()
    assert np.all(sc == sc[0, 0])
    # the oracle on the sampled rows with the tensor amax planted in an extra row
    probe = np.concatenate([Wf[rows], np.full((1, I), amax, np.float32)])
    ref_ws2 = rtn.recompute_ws2(Wf) if fmt == "nv" else None
    rc, rs, rw = rtn.quantize_rule(fmt, probe, "whole_tensor", ref_ws2)
    assert np.array_equal(c.cpu().numpy()[rows], rc[:-1]) and np.all(sc[0, 0] == rs)
    if fmt == "nv":
        assert w2.cpu().numpy()[0] == rw



ALL_RULES = ["even", "away", "rtz", "stochastic", "whole_tensor"]
GROUP_SHAPES = [(264, 1056), (8, 32), (96, 512), (1024, 4096), (8, 1024), (40, 3584)]


def _group_weights(sq, fmt, shapes, seed, ws2_in, unaligned=()):
    """Merged weights with output buffers for a grouped call and for single
    calls; planes listed in `unaligned` get scale planes at an odd address."""
    out = []
    for k, (O, I) in enumerate(shapes):
        Wb, _ = _merged_weight(fmt, O, I, seed=seed + 7 * k)
        G = I // codec.BLOCK[fmt]
        sbuf = torch.full((O * G + 1,), 0xA5, dtype=torch.uint8, device="cuda")
        sc = sbuf[1:].view(O, G) if k in unaligned else sbuf[:O * G].view(O, G)
        out.append(dict(W=Wb.cuda(), codes=torch.empty((O, I // 2), dtype=torch.uint8, device="cuda"),
                        scales=sc, ws2_out=torch.full((1,), -1.0, device="cuda"), ws2_in=ws2_in,
                        seed=0x9E37_79B9_7F4A_7C15 * (k + 1) & 0xFFFFFFFFFFFFFFFF, sbuf=sbuf))
    return out


@pytest.mark.parametrize("fmt", ["mx", "nv"])
@pytest.mark.parametrize("rule", ALL_RULES)
@pytest.mark.parametrize("ws2_mode", ["fixed", "recompute"])
def test_grouped_equals_single_calls(sq, fmt, rule, ws2_mode):
    """rtn_quantize_grouped over weights of several shapes (one with its scale
    plane at an odd address, so its scale bytes leave one by one) equals one
    rtn_quantize_rule call per weight, byte for byte, ws2_out included."""
    if fmt == "mx" and ws2_mode == "recompute":
        pytest.skip("MXFP4 has no per-tensor scalar")
    ws2_in = float(np.float32(1 / 448)) if (fmt == "nv" and ws2_mode == "fixed") else 0.0
    print(f"[grouped] fmt={fmt} rule={rule} ws2={ws2_mode}", flush=True)
    ws = _group_weights(sq, fmt, GROUP_SHAPES, 6000, ws2_in, unaligned=(2,))
    sq.rtn_quantize_grouped(fmt, rule, ws)
    torch.cuda.synchronize()
    for w in ws:
        c, s, w2 = sq.rtn_quantize_rule(fmt, w["W"], rule, ws2_in, w["seed"])
        torch.cuda.synchronize()
        assert torch.equal(w["codes"], c) and torch.equal(w["scales"], s)
        if w2 is not None:
            assert torch.equal(w["ws2_out"], w2)
        # the canary byte beside the plane is untouched
        canary = 0 if w["scales"].data_ptr() != w["sbuf"].data_ptr() else -1
        assert int(w["sbuf"][canary]) == 0xA5


def test_grouped_matches_oracle(sq):
    """One grouped NVFP4 call (recomputed ws2) against the oracle directly."""
    ws = _group_weights(sq, "nv", [(264, 1056), (96, 512)], 6100, 0.0)
    sq.rtn_quantize_grouped("nv", "even", ws)
    torch.cuda.synchronize()
    for w in ws:
        rc, rs, rw = rtn.quantize_rule("nv", w["W"].float().cpu().numpy(), "even", None, 0)
        assert np.array_equal(w["codes"].cpu().numpy(), rc) and np.array_equal(w["scales"].cpu().numpy(), rs)
        assert w["ws2_out"].cpu().numpy()[0] == rw


def test_grouped_more_weights_than_one_launch(sq):
    """61 weights (one launch takes 56), NVFP4 with every ws2 recomputed."""
    shapes = [(8 * (1 + k % 5), 16 * (2 + (k * 7) % 9)) for k in range(61)]
    ws = _group_weights(sq, "nv", shapes, 6200, 0.0, unaligned=(3, 60))
    sq.rtn_quantize_grouped("nv", "stochastic", ws)
    torch.cuda.synchronize()
    for w in ws:
        c, s, w2 = sq.rtn_quantize_rule("nv", w["W"], "stochastic", 0.0, w["seed"])
        torch.cuda.synchronize()
        assert torch.equal(w["codes"], c) and torch.equal(w["scales"], s) and torch.equal(w["ws2_out"], w2)


def test_grouped_rejects_a_shared_amax_slot(sq):
    ws = _group_weights(sq, "nv", [(8, 32), (8, 64)], 6300, 0.0)
    ws[1]["ws2_out"] = ws[0]["ws2_out"]
    with pytest.raises(sq.SqError):
        sq.rtn_quantize_grouped("nv", "even", ws)
    # with a fixed ws2 the slots only receive it, so sharing one is allowed
    for w in ws:
        w["ws2_in"] = float(np.float32(1 / 448))
    sq.rtn_quantize_grouped("nv", "even", ws)
    torch.cuda.synchronize()


@pytest.mark.parametrize("fmt", ["mx", "nv"])
def test_grouped_8b_layer_equals_single_calls(sq, fmt):
    """The seven linears of one 8B layer (q, k, v, o, gate, up, down), bf16
    weights drawn on the device, re-quantised in one grouped call and one call
    each: identical bytes."""
    B = codec.BLOCK[fmt]
    ws = []
    for k, (name, O, I) in enumerate(inputs.LLAMA8B_LAYER):
        W = (inputs.device_bf16_normal(7000 + k, (O, I)).float() * 0.02).to(torch.bfloat16)
        ws.append(dict(W=W, codes=torch.empty((O, I // 2), dtype=torch.uint8, device="cuda"),
                       scales=torch.empty((O, I // B), dtype=torch.uint8, device="cuda"),
                       ws2_out=torch.empty(1, device="cuda"), ws2_in=0.0))
    print(f"[grouped 8b] fmt={fmt}", flush=True)
    sq.rtn_quantize_grouped(fmt, "even", ws)
    torch.cuda.synchronize()
    for w in ws:
        c, s, w2 = sq.rtn_quantize(fmt, w["W"], sq.TIE_EVEN, 0.0)
        torch.cuda.synchronize()
        assert torch.equal(w["codes"], c) and torch.equal(w["scales"], s)
        if fmt == "nv":
            assert torch.equal(w["ws2_out"], w2)
