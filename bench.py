"""Benchmark of the Scale-QLoRA frozen-code FP4 layer on one MI355X.

    python bench.py [--gpus 1] [--steps 50] [--warmup 10] [--no-cpu-baseline]

One step is one pass of the whole hot path over one synthetic 8B-shaped
MXFP4 attention projection (O = I = 4096, 4096 tokens = batch 4 x seq 1024,
E8M0 exponents rint(N(-6, 1.5)), codes uniform, X and dY ~ N(0, 1) in bf16):

    sq_fwd (Y, bf16)  ->  sq_bwd_dx (dX, bf16)  ->  sq_bwd_dscale (dS, fp32)
    ->  sq_merge_scales copy (swap a base plane into the working plane)
    ->  sq_merge_scales delta (apply a task delta on the grid)
    ->  rtn_quantize (re-quantise the bf16 merged weight W + BA, the naive path)

`value` is the fused forward + backward throughput, 6*T*O*I flops over the
whole step's wall time (merge and re-quantisation time included), in TFLOP/s.
The timed steps carry no event records (on ROCm each record adds a
cache-flushing marker); per-kernel times come from a second pass that
launches each call back to back between two HIP events on the launch stream.
The line also carries those per-kernel times, the roofline of the dominant
kernel against MI355X's dense bf16 MFMA peak, the vendor bf16 GEMM at the same
shape, the whole-model scale-plane merge in GB/s against the 8 TB/s HBM peak,
the whole 8B-shaped model's scale-only step (32 layers x 7 linears) with the
weight-space STE comparator, and the CPU oracle timed on a bounded sample of
the same workload.
"""

import argparse
import json
import os
import sys
import time

import numpy as np
import torch

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

from paper_2609_04526_amd import inputs  # noqa: E402

PEAK_BF16_TFLOPS = 2500.0          # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0              # MI355X HBM3E

METRIC = "fused fwd+bwd scale-grad TFLOP/s and % bf16 MFMA peak at 8B shapes; merge GB/s"
T, O, I = 4096, 4096, 4096
FMT = "mx"
SEED = 2000


def kernel_source_digest():
    """sha256 of the GEMM kernel sources: counter readings are only reused
    while the kernels they were taken on are unchanged."""
    import hashlib
    h = hashlib.sha256()
    for f in ("sq_gemm.hip", "sq_device.h"):
        with open(os.path.join(ROOT, "paper_2609_04526_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def measured_traffic(kernel_name):
    """HBM bytes per launch of `kernel_name` from profiles/traffic.json (rocprofv3
    FETCH_SIZE / WRITE_SIZE, copy-calibrated), or None when absent or stale."""
    path = os.path.join(ROOT, "profiles", "traffic.json")
    try:
        with open(path) as f:
            rec = json.load(f)
    except (OSError, ValueError):
        return None
    if rec.get("source_sha256") != kernel_source_digest():
        return None
    k = rec.get("kernels", {}).get(kernel_name)
    return None if k is None else int(k["fetch_bytes"] + k["write_bytes"])


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=50)
    p.add_argument("--warmup", type=int, default=100,
                   help="untimed steps first; the clock settles after some tens of milliseconds of load")
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--no-model-merge", action="store_true")
    p.add_argument("--no-model-step", action="store_true")
    p.add_argument("--no-lifecycle", action="store_true")
    p.add_argument("--no-moe", action="store_true")
    p.add_argument("--no-mlp-nv", action="store_true")
    p.add_argument("--no-cpu-plan", action="store_true",
                   help="time only the main oracle sample, not the per-workload oracle plan")
    p.add_argument("--calib-copy-mib", type=int, default=0,
                   help="also run a plain device copy of this many MiB (the copy mode of "
                        "sq_merge_scales: reads N and writes N bytes) to calibrate HBM counters")
    return p.parse_args()


def layer_inputs():
    G = I // 32
    X = inputs.bf16_normal(SEED, (T, I))
    dY = inputs.bf16_normal(SEED + 1, (T, O))
    codes = inputs.codes_uniform(SEED + 2, O, I)
    sb = inputs.e8m0_normal_exponents(SEED + 3, O, G, -6.0, 1.5)
    # a task delta: +-1 exponent step on 5% of blocks plus 1% relative jitter
    eff = np.ldexp(1.0, sb.astype(np.int64) - 127)
    delta = inputs.e8m0_step_delta(SEED + 4, sb, 0.05) + inputs.relative_jitter(SEED + 5, eff, 0.01)
    src = inputs.e8m0_normal_exponents(SEED + 6, O, G, -6.0, 1.5)
    return X, dY, codes, sb, delta.astype(np.float32), src


def merged_weight_bf16(codes_d, sb_d, sq):
    """bf16(dequant(W) + B A), rank 16, built on the device outside the timed
    region: the layer's own forward on an identity batch gives dequant(W)^T."""
    eye = torch.eye(I, dtype=torch.bfloat16, device="cuda")
    Wt = sq.sq_fwd(FMT, eye, codes_d, sb_d, 1.0, torch.float32)       # [I, O] = W^T exactly
    B, A = inputs.lora_factors(SEED + 7, O, I, 16, 0.02)
    Wm = Wt.t() + torch.from_numpy(B).cuda() @ torch.from_numpy(A).cuda()
    return Wm.to(torch.bfloat16).contiguous()


def effective_scales_torch(fmt, scale_bytes, ws2):
    """fp32 effective scales of a scale plane with torch's decoders (input
    recipes and read-back only; the merge kernels decode on their own)."""
    if fmt == "mx":
        return torch.exp2(scale_bytes.float() - 127.0)
    return scale_bytes.view(torch.float8_e4m3fn).float() * ws2


def model_merge(sq, steps):
    """Grouped merges over every scale plane of the 8B model (32 layers x 7
    linears) with a task delta: MXFP4 (218,103,808 scales) and NVFP4
    (436,207,616 scales), 6 bytes moved per scale, and the MXFP4 hot swap
    (copy mode, 2 bytes per scale).  Base planes: MXFP4 exponents
    rint(N(-6, 1.5)), NVFP4 E4M3 of |N(0, 1)| with ws2 = 1/448.  Reports the
    fraction of scale bytes the merge changed."""
    out = {}
    ws2 = float(np.float32(1.0 / 448.0))
    # the model's code plane (224 linears, 0.5 B per weight), resident beside
    # the scale planes; after every merge it is compared byte for byte with a copy
    n_codes = sum(o * i // 2 for (_, o, i) in inputs.LLAMA8B_LAYER) * inputs.LLAMA8B_LAYERS
    code_plane = torch.randint(0, 256, (n_codes,), dtype=torch.uint8, device="cuda",
                               generator=inputs.device_generator(6900))
    code_copy = code_plane.clone()
    for name, fmt, block, mode in (("mx_delta", "mx", 32, "delta"), ("nv_delta", "nv", 16, "delta"),
                                   ("mx_swap", "mx", 32, "copy"), ("nv_swap", "nv", 16, "copy")):
        shapes = [(o, i // block) for _ in range(inputs.LLAMA8B_LAYERS) for (_, o, i) in inputs.LLAMA8B_LAYER]
        sizes = [o * g for (o, g) in shapes]
        total = sum(sizes)
        if fmt == "mx":
            base = torch.cat([inputs.device_e8m0_normal_exponents(7000 + k, o, g, -6.0, 1.5).reshape(-1)
                              for k, (o, g) in enumerate(shapes)])
        else:
            base = torch.cat([inputs.device_e4m3_abs_normal(7000 + k, o, g).reshape(-1)
                              for k, (o, g) in enumerate(shapes)])
        if mode == "delta":
            aux = inputs.device_task_delta(7500, effective_scales_torch(fmt, base, ws2), fmt).float()
        elif fmt == "mx":
            aux = torch.cat([inputs.device_e8m0_normal_exponents(7600 + k, o, g, -6.0, 1.5).reshape(-1)
                             for k, (o, g) in enumerate(shapes)])
        else:
            aux = torch.cat([inputs.device_e4m3_abs_normal(7600 + k, o, g).reshape(-1)
                             for k, (o, g) in enumerate(shapes)])
        scales = base.clone()
        descs, off = [], 0
        for n in sizes:
            d = dict(fmt=fmt, scales=scales[off:off + n], ws2=ws2)
            d["delta" if mode == "delta" else "src"] = aux[off:off + n]
            descs.append(d)
            off += n
        group = sq.MergeGroup(descs)
        sq.sq_merge_scales_grouped(group)              # the merge itself: base -> merged
        torch.cuda.synchronize()
        changed = float((scales != base).sum().item()) / total
        rb = None
        if mode == "delta":
            # rollback: the applied on-grid delta restores the base byte for byte
            applied = sq.sq_scale_applied_delta(fmt, base, scales)
            restored = scales.clone()
            sq.sq_scale_rollback(fmt, restored, applied)
            counts = sq.sq_byte_diff(restored, base)
            torch.cuda.synchronize()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            for _ in range(steps):
                sq.sq_scale_rollback(fmt, restored, applied)
            e1.record()
            torch.cuda.synchronize()
            rb_ms = e0.elapsed_time(e1) / steps
            e0.record()
            for _ in range(steps):
                sq.sq_byte_diff(restored, base, counts=torch.zeros(2, dtype=torch.int64, device="cuda"))
            e1.record()
            torch.cuda.synchronize()
            diff_ms = e0.elapsed_time(e1) / steps
            rb = {"restored_bytes_differing": int(counts[0].item()),
                  "rollback_ms": round(rb_ms, 4), "rollback_GB/s": round(6 * total / (rb_ms * 1e-3) / 1e9, 1),
                  "audit_ms": round(diff_ms, 4), "audit_GB/s": round(2 * total / (diff_ms * 1e-3) / 1e9, 1)}
            del applied, restored
        for _ in range(2):
            sq.sq_merge_scales_grouped(group)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(steps):
            sq.sq_merge_scales_grouped(group)
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / steps
        bps = 6 if mode == "delta" else 2
        gbs = bps * total / (ms * 1e-3) / 1e9
        code_diff = sq.sq_byte_diff(code_plane, code_copy)
        torch.cuda.synchronize()
        out[name] = {"scales": total, "planes": len(sizes), "bytes_per_scale": bps, "ms": round(ms, 4),
                     "code_bytes_checked": n_codes, "code_bytes_differing": int(code_diff[0].item()),
                     "GB/s": round(gbs, 1), "peak": PEAK_HBM_GBS, "frac": round(gbs / PEAK_HBM_GBS, 4),
                     "changed_byte_frac": round(changed, 5)}
        if rb is not None:
            out[name]["rollback"] = rb
        del scales, base, aux, descs, group
        torch.cuda.empty_cache()
    del code_plane, code_copy
    torch.cuda.empty_cache()
    out["note"] = ("delta merges are re-applied to the merged planes in the timed repetitions (same bytes "
                   "moved); the paper reports 4.7-7.7% of scale bytes changed by its task merges (context only)")
    return out


def model_lifecycle(sq, steps=3):
    """The naive merge's re-quantisation over the whole 8B model: for every
    linear, the bf16 merged weight W + B A (rank 16, A, B ~ N(0, 0.02), W the
    dequantised base) re-quantised with ties to even and ties away, and under
    the deploy-side rules (toward zero, stochastic, whole-tensor scale), each
    as one rtn_quantize_grouped call over all 224 linears (and nearest-even
    once more as one rtn_quantize call per linear).  Algorithmic
    bytes 2 + 0.5 + 1/B per weight.  The re-quantising swap of a task into the
    served model also runs as one fused pass per linear, base codes + scales +
    the task's rank-16 adapter -> new codes + scales (sq_qat_requant, nearest
    even), with no bf16 weight in between.  The diff census counts code nibbles that differ from the base
    plane (per tie rule) and between the tie rules, and changed scale bytes."""
    lut = torch.tensor([0.0, 0.5, 1.0, 1.5, 2.0, 3.0, 4.0, 6.0, -0.0, -0.5, -1.0, -1.5, -2.0, -3.0, -4.0, -6.0],
                       device="cuda")

    def nibbles(c):
        return torch.stack((c & 15, c >> 4), dim=-1).reshape(c.shape[0], -1)

    out = {}
    ws2 = float(np.float32(1.0 / 448.0))
    for fmt, block in (("mx", 32), ("nv", 16)):
        items = []
        for k, (name, o, i) in enumerate(inputs.LLAMA8B_LAYER * inputs.LLAMA8B_LAYERS):
            G = i // block
            codes = inputs.device_codes_uniform(8000 + k, o, i)
            sb = (inputs.device_e8m0_normal_exponents(8300 + k, o, G, -6.0, 1.5) if fmt == "mx"
                  else inputs.device_e4m3_abs_normal(8300 + k, o, G))
            g = inputs.device_generator(8600 + k)
            Bf = torch.randn((o, 16), generator=g, device="cuda") * 0.02
            Af = torch.randn((16, i), generator=g, device="cuda") * 0.02
            W = lut[nibbles(codes).long()] * effective_scales_torch(fmt, sb, ws2).repeat_interleave(block, dim=1)
            Wm = (W + Bf @ Af).to(torch.bfloat16)
            del W, Bf, Af
            items.append(dict(codes=codes, sb=sb, Wm=Wm,
                              ce=torch.empty_like(codes), se=torch.empty_like(sb),
                              ca=torch.empty_like(codes), sa=torch.empty_like(sb),
                              cr=torch.empty_like(codes), sr=torch.empty_like(sb),
                              w2=torch.empty(1, dtype=torch.float32, device="cuda")))
        weights = sum(it["Wm"].numel() for it in items)
        nbytes = weights * (2 + 0.5 + 1.0 / block)
        res = {"weights": weights, "linears": len(items), "bytes": int(nbytes)}
        runs = [("even", sq.TIE_EVEN, ws2, "ce", "se"), ("away", sq.TIE_AWAY, ws2, "ca", "sa")]
        if fmt == "nv":
            runs.append(("even_ws2_recomputed", sq.TIE_EVEN, 0.0, "ce", "se"))
        # deploy-side rules through rtn_quantize_rule (the whole-tensor rule
        # takes its amax in a pre-pass, so it reads W twice)
        runs += [("rtz", "rtz", ws2, "cr", "sr"), ("stochastic", "stochastic", ws2, "cr", "sr"),
                 ("whole_tensor", "whole_tensor", 0.0, "cr", "sr")]
        # the same nearest-even re-quantisation through one call per linear,
        # to show what sharing launches saves
        runs.append(("even_per_linear_calls", sq.TIE_EVEN, ws2, "ce", "se"))
        for label, tie, w_in, ck, sk in runs:
            rule = tie if isinstance(tie, str) else ("even" if tie == sq.TIE_EVEN else "away")
            group = sq.RtnGroup(fmt, rule, [dict(W=it["Wm"], codes=it[ck], scales=it[sk], ws2_out=it["w2"],
                                                 ws2_in=w_in if fmt == "nv" else 0.0, seed=1234) for it in items])

            def run():
                if label.endswith("per_linear_calls"):
                    for it in items:
                        sq.rtn_quantize(fmt, it["Wm"], tie, w_in, codes=it[ck], scales=it[sk],
                                        ws2_out=it["w2"] if fmt == "nv" else None)
                else:
                    sq.rtn_quantize_grouped(fmt, rule, group)
            run()
            torch.cuda.synchronize()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            for _ in range(steps):
                run()
            e1.record()
            torch.cuda.synchronize()
            ms = e0.elapsed_time(e1) / steps
            two_pass = (w_in == 0.0 and fmt == "nv") or tie == "whole_tensor"
            moved = nbytes + (weights * 2 if two_pass else 0)       # the amax pre-pass reads W once more
            res[label] = {"ms": round(ms, 3), "GB/s": round(moved / (ms * 1e-3) / 1e9, 1),
                          "frac": round(moved / (ms * 1e-3) / 1e9 / PEAK_HBM_GBS, 4)}
            if ck == "cr":
                nb_moved = sum(int((nibbles(it["cr"]) != nibbles(it["codes"])).sum().item()) for it in items)
                sb_moved = sum(int((it["sr"] != it["sb"]).sum().item()) for it in items)
                res[label]["code_nibbles_vs_base_frac"] = round(nb_moved / weights, 5)
                res[label]["scale_bytes_vs_base"] = sb_moved
        # the re-quantising swap from the base planes and the task adapter
        fused_items = []
        for k, it in enumerate(items):
            o, half = it["codes"].shape
            g = inputs.device_generator(8700 + k)
            fused_items.append((it, (torch.randn((o, 16), generator=g, device="cuda") * 0.02).to(torch.bfloat16),
                                (torch.randn((16, 2 * half), generator=g, device="cuda") * 0.02).to(torch.bfloat16)))

        def run_fused():
            for it, Bq, Aq in fused_items:
                sq.sq_qat_requant(fmt, it["codes"], it["sb"], Bq, Aq, 1.0, ws2 if fmt == "nv" else 1.0,
                                  codes_out=it["cr"], scales_out=it["sr"])
        run_fused()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(steps):
            run_fused()
        e1.record()
        torch.cuda.synchronize()
        fms = e0.elapsed_time(e1) / steps
        fbytes = weights * (0.5 + 1.0 / block) * 2            # codes + scales read, written
        res["requant_swap_fused"] = {"ms": round(fms, 3), "GB/s": round(fbytes / (fms * 1e-3) / 1e9, 1),
                                     "what": "sq_qat_requant over all 224 linears: base codes + scales + "
                                             "rank-16 task adapter -> re-quantised codes + scales"}
        del fused_items
        # census (ties to even and ties away, both with the fixed ws2 for NVFP4)
        sq.rtn_quantize_grouped(fmt, "even", [dict(W=it["Wm"], codes=it["ce"], scales=it["se"], ws2_out=it["w2"],
                                                   ws2_in=ws2 if fmt == "nv" else 0.0) for it in items])
        torch.cuda.synchronize()
        cen = {"code_nibbles_even_vs_base": 0, "code_nibbles_away_vs_base": 0, "code_nibbles_even_vs_away": 0,
               "scale_bytes_even_vs_base": 0, "scale_bytes_even_vs_away": 0}
        for it in items:
            nb, ne, na = nibbles(it["codes"]), nibbles(it["ce"]), nibbles(it["ca"])
            cen["code_nibbles_even_vs_base"] += int((ne != nb).sum().item())
            cen["code_nibbles_away_vs_base"] += int((na != nb).sum().item())
            cen["code_nibbles_even_vs_away"] += int((ne != na).sum().item())
            cen["scale_bytes_even_vs_base"] += int((it["se"] != it["sb"]).sum().item())
            cen["scale_bytes_even_vs_away"] += int((it["se"] != it["sa"]).sum().item())
        res["census"] = cen
        res["census_frac_even_vs_base"] = round(cen["code_nibbles_even_vs_base"] / weights, 5)
        out[fmt] = res
        del items
        torch.cuda.empty_cache()
    return out


def model_step_fused(sq, codes, scales, dys, xs, Tm, L, steps, warmup, flops):
    """The same step with the projections that share an input stored stacked,
    as fused-projection layouts keep them: q/k/v as one [6144, 4096] weight and
    gate/up as one [28672, 4096] weight (codes and scale rows concatenated;
    dY of the stacked product is the per-linear dY side by side).  Each
    stacked weight takes one forward, one dX (which is the sum of the
    projections' dX, what the shared input needs) and one dS, whose row
    ranges are the projections' dS.  The same flops in 4 + 4 + 4 products per
    layer instead of 7 + 7 + 7."""
    n_lin = len(inputs.LLAMA8B_LAYER)
    groups = (("qkv", (0, 1, 2)), ("o", (3,)), ("gate_up", (4, 5)), ("down", (6,)))
    layers = []
    for l in range(L):
        ent = []
        for name, ks in groups:
            ns = [l * n_lin + k for k in ks]
            c = torch.cat([codes[n] for n in ns]) if len(ns) > 1 else codes[ns[0]]
            sc = torch.cat([scales[n] for n in ns]) if len(ns) > 1 else scales[ns[0]]
            dy = torch.cat([dys[n] for n in ns], dim=1) if len(ns) > 1 else dys[ns[0]]
            x = xs[l][inputs.LLAMA8B_LAYER[ks[0]][0]]
            o, i = c.shape[0], x.shape[1]
            ent.append(dict(c=c, sc=sc, dy=dy, x=x, o=o, i=i,
                            ds=torch.empty((o, i // 32), dtype=torch.float32, device="cuda")))
        layers.append(ent)
    yb = {e["o"]: torch.empty((Tm, e["o"]), dtype=torch.bfloat16, device="cuda") for e in layers[0]}
    xb = {e["i"]: torch.empty((Tm, e["i"]), dtype=torch.bfloat16, device="cuda") for e in layers[0]}

    def run():
        for l in range(L):
            for e in layers[l]:
                sq.sq_fwd("mx", e["x"], e["c"], e["sc"], 1.0, Y=yb[e["o"]])
        for l in reversed(range(L)):
            for e in reversed(layers[l]):
                sq.sq_bwd_dx("mx", e["dy"], e["c"], e["sc"], 1.0, dX=xb[e["i"]])
                sq.sq_bwd_dscale("mx", e["x"], e["dy"], e["c"], dS=e["ds"])

    for _ in range(warmup):
        run()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(steps):
        run()
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / steps
    del layers, yb, xb
    torch.cuda.empty_cache()
    return {"what": "q/k/v and gate/up stacked into one weight each (fused projections), 171.5 TFLOP as above",
            "ms": round(ms, 3), "TFLOP/s": round(flops / (ms * 1e-3) / 1e12, 1),
            "frac_of_bf16_peak": round(flops / (ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 4)}


def model_step(sq, steps, warmup, comparator=True):
    """One scale-only training step of the whole 8B-shaped model in MXFP4: 32
    layers x {q, k, v, o, gate, up, down}, 4096 tokens, every linear's forward,
    dX and dS (171.5 TFLOP).  Inputs are drawn on the device (one X shared by
    q/k/v, one by gate/up, one each for o and down; one dY per linear); dS is
    kept per linear, Y and dX go to per-shape buffers.  The step runs every
    forward in layer order, then every backward in reverse order; k and v,
    which share their input and shape, run each product as one grouped launch
    of both (`per_linear_one_layer` times them apart too, as k_* and v_*).

    The QAST step reruns it with every linear's scales from a rank-32 adapter;
    the QAT-LoRA step runs the weight-space STE comparator on the native path
    (fused re-quantisation of W + B A, forward and dX on those codes, factor
    gradients through the rank).  A second, framework-style comparator repeats
    the paper's own construction on all 224 linears (rank 32, each with its own
    weight and factors): W' = deq(W) + B A, RTN fake-quantisation
    (rtn_quantize, then a torch dequant), the three dense bf16 GEMMs through
    torch (hipBLASLt) with dW materialised in fp32, then dB = dW A^T and
    dA = B^T dW."""
    Tm = 4096
    shapes = inputs.LLAMA8B_LAYER
    L = inputs.LLAMA8B_LAYERS
    seed = 4000
    codes, scales, dys, dss, xs = [], [], [], [], []
    for l in range(L):
        xa = inputs.device_bf16_normal(seed + 100 * l + 90, (Tm, 4096))
        xo = inputs.device_bf16_normal(seed + 100 * l + 91, (Tm, 4096))
        xm = inputs.device_bf16_normal(seed + 100 * l + 92, (Tm, 4096))
        xd = inputs.device_bf16_normal(seed + 100 * l + 93, (Tm, 14336))
        xs.append({"q": xa, "k": xa, "v": xa, "o": xo, "gate": xm, "up": xm, "down": xd})
        for k, (name, o, i) in enumerate(shapes):
            codes.append(inputs.device_codes_uniform(seed + 100 * l + 3 * k, o, i))
            scales.append(inputs.device_e8m0_normal_exponents(seed + 100 * l + 3 * k + 1, o, i // 32, -6.0, 1.5))
            dys.append(inputs.device_bf16_normal(seed + 100 * l + 3 * k + 2, (Tm, o)))
            dss.append(torch.empty((o, i // 32), dtype=torch.float32, device="cuda"))
    ybuf = {(o, i): torch.empty((Tm, o), dtype=torch.bfloat16, device="cuda") for (_, o, i) in shapes}
    dxbuf = {(o, i): torch.empty((Tm, i), dtype=torch.bfloat16, device="cuda") for (_, o, i) in shapes}
    # k and v share their input and shape: each of their products runs as one
    # grouped launch of both (512 tiles instead of two launches of 256 that
    # leave half of every CU's workgroup slots empty)
    KV = (1, 2)
    assert [shapes[k][0] for k in KV] == ["k", "v"]
    kv_y = [torch.empty((Tm, 1024), dtype=torch.bfloat16, device="cuda") for _ in KV]
    kv_dx = [torch.empty((Tm, 4096), dtype=torch.bfloat16, device="cuda") for _ in KV]

    def kv_tables(code_of, scale_of, with_ds=True):
        """Per layer, the grouped k+v tables over the given per-linear codes
        and scales (linear index n -> tensor)."""
        out = []
        for l in range(L):
            ns = [l * len(shapes) + k for k in KV]
            x = xs[l]["k"]
            c, sc = [code_of(n) for n in ns], [scale_of(n) for n in ns]
            t = dict(fwd=sq.ExpertTable("fwd", "mx", [x, x], c, sc, kv_y),
                     dx=sq.ExpertTable("dx", "mx", [dys[n] for n in ns], c, sc, kv_dx))
            if with_ds:
                t["ds"] = sq.ExpertTable("ds", "mx", [x, x], c, None, [dss[n] for n in ns],
                                         acts2=[dys[n] for n in ns])
            out.append(t)
        return out

    kv = kv_tables(lambda n: codes[n], lambda n: scales[n])

    def run(events=None):
        for l in range(L):
            for k, (name, o, i) in enumerate(shapes):
                n = l * len(shapes) + k
                if k == KV[0]:
                    kv[l]["fwd"].run()
                elif k not in KV:
                    sq.sq_fwd("mx", xs[l][name], codes[n], scales[n], 1.0, Y=ybuf[(o, i)])
        for l in reversed(range(L)):
            for k, (name, o, i) in reversed(list(enumerate(shapes))):
                n = l * len(shapes) + k
                if k == KV[1]:
                    kv[l]["dx"].run()
                    kv[l]["ds"].run()
                elif k not in KV:
                    sq.sq_bwd_dx("mx", dys[n], codes[n], scales[n], 1.0, dX=dxbuf[(o, i)])
                    sq.sq_bwd_dscale("mx", xs[l][name], dys[n], codes[n], dS=dss[n])

    for _ in range(warmup):
        run()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(steps):
        run()
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / steps
    flops = 6.0 * Tm * L * sum(o * i for (_, o, i) in shapes)

    # per-shape product times, one layer's worth repeated over all 32 layers
    per = {}
    for k, (name, o, i) in enumerate(shapes):
        for prod in ("fwd", "dx", "ds"):
            def one(l, prod=prod, k=k, name=name, o=o, i=i):
                n = l * len(shapes) + k
                if prod == "fwd":
                    sq.sq_fwd("mx", xs[l][name], codes[n], scales[n], 1.0, Y=ybuf[(o, i)])
                elif prod == "dx":
                    sq.sq_bwd_dx("mx", dys[n], codes[n], scales[n], 1.0, dX=dxbuf[(o, i)])
                else:
                    sq.sq_bwd_dscale("mx", xs[l][name], dys[n], codes[n], dS=dss[n])
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record()
            for l in range(L):
                one(l)
            b.record()
            torch.cuda.synchronize()
            t = a.elapsed_time(b) / L
            per[f"{name}_{prod}"] = {"ms": round(t, 4), "TFLOP/s": round(2.0 * Tm * o * i / (t * 1e-3) / 1e12, 1)}
    # k and v as the step runs them: one grouped launch of both per product
    for prod in ("fwd", "dx", "ds"):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for l in range(L):
            kv[l][prod].run()
        b.record()
        torch.cuda.synchronize()
        t = a.elapsed_time(b) / L
        per[f"kv_grouped_{prod}"] = {"ms": round(t, 4),
                                     "TFLOP/s": round(2 * 2.0 * Tm * 1024 * 4096 / (t * 1e-3) / 1e12, 1)}
    del kv
    fused = model_step_fused(sq, codes, scales, dys, xs, Tm, L, steps, warmup, flops)
    # The QAST step: every linear's scales come from its rank-32 adapter
    # (on-grid bytes + clamp mask), the products run on those bytes, and dS
    # turns into dB, dA.
    r = 32
    qa = []
    for n, (name, o, i) in enumerate(shapes * L):
        G = i // 32
        g = inputs.device_generator(6000 + n)
        qa.append(dict(B=(torch.randn((o, r), generator=g, device="cuda") * 0.02).to(torch.bfloat16),
                       A=(torch.randn((r, G), generator=g, device="cuda") * 1e-3).to(torch.bfloat16),
                       sc=torch.empty((o, G), dtype=torch.uint8, device="cuda"),
                       m=torch.empty((o, G), dtype=torch.uint8, device="cuda"),
                       dB=torch.empty((o, r), dtype=torch.float32, device="cuda"),
                       dA=torch.empty((r, G), dtype=torch.float32, device="cuda")))
    qws = torch.empty(max(sq.sq_qast_factor_grads_workspace(o, i // 32, r) for (_, o, i) in shapes),
                      dtype=torch.uint8, device="cuda")

    kv_qast = kv_tables(lambda n: codes[n], lambda n: qa[n]["sc"])

    def run_qast():
        for l in range(L):
            for k, (name, o, i) in enumerate(shapes):
                n = l * len(shapes) + k
                q = qa[n]
                sq.sq_qast_scales("mx", scales[n], q["B"], q["A"], 1.0, scales_out=q["sc"], mask_out=q["m"])
                if k == KV[1]:
                    kv_qast[l]["fwd"].run()
                elif k not in KV:
                    sq.sq_fwd("mx", xs[l][name], codes[n], q["sc"], 1.0, Y=ybuf[(o, i)])
        for l in reversed(range(L)):
            for k, (name, o, i) in reversed(list(enumerate(shapes))):
                n = l * len(shapes) + k
                q = qa[n]
                if k == KV[1]:
                    kv_qast[l]["dx"].run()
                    kv_qast[l]["ds"].run()
                elif k not in KV:
                    sq.sq_bwd_dx("mx", dys[n], codes[n], q["sc"], 1.0, dX=dxbuf[(o, i)])
                    sq.sq_bwd_dscale("mx", xs[l][name], dys[n], codes[n], dS=dss[n])
                sq.sq_qast_factor_grads(dss[n], q["m"], q["B"], q["A"], 1.0, dB=q["dB"], dA=q["dA"], workspace=qws)

    for _ in range(warmup):
        run_qast()
    torch.cuda.synchronize()
    e0.record()
    for _ in range(steps):
        run_qast()
    e1.record()
    torch.cuda.synchronize()
    qast_ms = e0.elapsed_time(e1) / steps
    del kv_qast

    # The QAT-LoRA comparator on the native path: every linear's weight
    # W = deq(W) + B A (rank 32) is re-quantised by the fused kernel before its
    # forward, the forward and dX run on those codes, and the STE gradients go
    # to B and A through the rank (dW is never formed).
    qt = []
    for n, (name, o, i) in enumerate(shapes * L):
        g = inputs.device_generator(7000 + n)
        qt.append(dict(B=(torch.randn((o, r), generator=g, device="cuda") * 0.02).to(torch.bfloat16),
                       A=(torch.randn((r, i), generator=g, device="cuda") * 0.02).to(torch.bfloat16),
                       c=torch.empty((o, i // 2), dtype=torch.uint8, device="cuda"),
                       s=torch.empty((o, i // 32), dtype=torch.uint8, device="cuda"),
                       dB=torch.empty((o, r), dtype=torch.float32, device="cuda"),
                       dA=torch.empty((r, i), dtype=torch.float32, device="cuda")))
    lws = torch.empty(max(sq.sq_lora_grads_workspace(Tm, o, i, r) for (_, o, i) in shapes),
                      dtype=torch.uint8, device="cuda")

    kv_qat = kv_tables(lambda n: qt[n]["c"], lambda n: qt[n]["s"], with_ds=False)

    def run_qat():
        for l in range(L):
            for k, (name, o, i) in enumerate(shapes):
                n = l * len(shapes) + k
                q = qt[n]
                sq.sq_qat_requant("mx", codes[n], scales[n], q["B"], q["A"], 1.0, codes_out=q["c"], scales_out=q["s"])
                if k == KV[1]:
                    kv_qat[l]["fwd"].run()
                elif k not in KV:
                    sq.sq_fwd("mx", xs[l][name], q["c"], q["s"], 1.0, Y=ybuf[(o, i)])
        for l in reversed(range(L)):
            for k, (name, o, i) in reversed(list(enumerate(shapes))):
                n = l * len(shapes) + k
                q = qt[n]
                if k == KV[1]:
                    kv_qat[l]["dx"].run()
                elif k not in KV:
                    sq.sq_bwd_dx("mx", dys[n], q["c"], q["s"], 1.0, dX=dxbuf[(o, i)])
                sq.sq_lora_grads(xs[l][name], dys[n], q["B"], q["A"], 1.0, dB=q["dB"], dA=q["dA"], workspace=lws)

    for _ in range(warmup):
        run_qat()
    torch.cuda.synchronize()
    e0.record()
    for _ in range(steps):
        run_qat()
    e1.record()
    torch.cuda.synchronize()
    qat_ms = e0.elapsed_time(e1) / steps
    del qt, lws, kv_qat

    out = {"workload": "MXFP4 8B-shaped model, 32 layers x 7 linears, 4096 tokens: fwd + dX + dS of every linear",
           "ms": round(ms, 3), "TFLOP": round(flops / 1e12, 2),
           "TFLOP/s": round(flops / (ms * 1e-3) / 1e12, 1),
           "frac_of_bf16_peak": round(flops / (ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 4),
           "per_linear_one_layer": per,
           "fused_projections": fused,
           "qast_step": {"what": "the same step with every linear's scales from a rank-32 adapter: "
                                 "sq_qast_scales before each forward, sq_qast_factor_grads after each dS",
                         "ms": round(qast_ms, 3), "overhead_ms": round(qast_ms - ms, 3),
                         "note": "the paper reports +49 ms per step for QAST on its own hardware and model "
                                 "(context only)"},
           "qat_lora_step": {"what": "QAT-LoRA weight-space STE on the native path, rank 32: sq_qat_requant "
                                     "(fused W + B A and nearest re-quantisation) before each forward, forward "
                                     "and dX on the re-quantised codes, sq_lora_grads (STE gradients of B, A "
                                     "through the rank) after each dX",
                             "ms": round(qat_ms, 3), "ratio_to_scale_step": round(qat_ms / ms, 3),
                             "ratio_to_qast_step": round(qat_ms / qast_ms, 3),
                             "note": "the paper reports QAT-LoRA at 3.9x its QAST step per step on its own "
                                     "hardware, through framework ops with dW materialised (context only)"}}
    del dys, xs, qa
    if comparator:
        out["weight_space_ste"] = weight_space_ste(sq, codes, scales, Tm, ms, L)
    return out


def model_moe(sq, steps=3, warmup=1):
    """One scale-only training step of a 30B-A3B-shaped MoE stack in MXFP4: 48
    layers, each with 128 experts of gate/up [768, 2048] and down [2048, 768];
    4096 tokens routed top-8 (32768 expert rows per layer, split over the
    experts by a seeded Dirichlet-multinomial, the same split for every
    layer).  Per layer and linear: one grouped forward, and in reverse order
    one grouped dX and one grouped dS, all 128 experts in each launch.  Every
    layer has its own expert weights; the routed activations and output
    buffers are shared across layers (values do not change the timing).  The
    fused variant stacks gate and up into one weight per expert (6 grouped
    products per layer, the pair's dX summed in one contraction).  The
    QAST variant adds the batched rank-32 scale step of all experts per linear
    (sq_qast_scales_batched before the forward, sq_qast_factor_grads_batched
    after dS).  The QAT-LoRA variant is the weight-space comparator on the
    same experts: sq_qat_requant_batched (all experts' W + B A re-quantised)
    before the grouped forward, then the grouped dX on those codes and
    sq_lora_grads_batched (rank 32) instead of dS."""
    L, E, topk, Tm, r = 48, 128, 8, 4096, 32
    g = inputs.rng(8800)
    Ts = g.multinomial(Tm * topk, g.dirichlet(np.full(E, 2.0))).tolist()
    shapes = (("gate", 768, 2048), ("up", 768, 2048), ("down", 2048, 768))
    acts = {}
    offs = np.concatenate([[0], np.cumsum(Ts)]).tolist()
    for k, (name, o, i) in enumerate(shapes):
        # the routed rows of all experts, expert after expert (the grouped layout)
        Xall = inputs.device_bf16_normal(8900 + k, (offs[-1], i))
        dYall = inputs.device_bf16_normal(9100 + k, (offs[-1], o))
        acts[name] = dict(Xall=Xall, dYall=dYall,
                          X=[Xall[offs[e]:offs[e + 1]] for e in range(E)],
                          dY=[dYall[offs[e]:offs[e + 1]] for e in range(E)],
                          Y=[torch.empty((T, o), dtype=torch.bfloat16, device="cuda") for T in Ts],
                          dX=[torch.empty((T, i), dtype=torch.bfloat16, device="cuda") for T in Ts],
                          dS=[torch.empty((o, i // 32), dtype=torch.float32, device="cuda") for _ in Ts])
    layers = []
    for l in range(L):
        lw = {}
        for k, (name, o, i) in enumerate(shapes):
            codes = inputs.device_codes_uniform(9300 + 10 * l + k, E * o, i).view(E, o, i // 2)
            sc = inputs.device_e8m0_normal_exponents(9600 + 10 * l + k, E * o, i // 32, -6.0, 1.5).view(E, o, i // 32)
            lw[name] = dict(codes=codes, scales=sc, cl=[codes[e] for e in range(E)], sl=[sc[e] for e in range(E)])
        layers.append(lw)

    # the expert descriptor tables are built once, as a training loop would
    tables = {}
    for l in range(L):
        for (name, _, _) in shapes:
            a, w = acts[name], layers[l][name]
            tables[(l, name)] = (sq.ExpertTable("fwd", "mx", a["X"], w["cl"], w["sl"], a["Y"]),
                                 sq.ExpertTable("dx", "mx", a["dY"], w["cl"], w["sl"], a["dX"]),
                                 sq.ExpertTable("ds", "mx", a["X"], w["cl"], None, a["dS"], acts2=a["dY"]))

    def run():
        for l in range(L):
            for (name, _, _) in shapes:
                tables[(l, name)][0].run()
        for l in reversed(range(L)):
            for (name, _, _) in reversed(shapes):
                tables[(l, name)][1].run()
                tables[(l, name)][2].run()

    def timed(fn):
        for _ in range(warmup):
            fn()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(steps):
            fn()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / steps

    ms = timed(run)
    rows = sum(Ts)
    flops = 6.0 * rows * L * sum(o * i for (_, o, i) in shapes)

    # the same stack with gate and up stacked into one [1536, 2048] weight per
    # expert (the fused-projection layout): one grouped forward, dX and dS for
    # the pair, the pair's dX summed inside one 1536-deep contraction
    gx = acts["gate"]
    dYgu_all = inputs.device_bf16_normal(9200, (offs[-1], 1536))
    dYgu = [dYgu_all[offs[e]:offs[e + 1]] for e in range(E)]
    Ygu = [torch.empty((T, 1536), dtype=torch.bfloat16, device="cuda") for T in Ts]
    dSgu = [torch.empty((1536, 2048 // 32), dtype=torch.float32, device="cuda") for _ in Ts]
    ftables = []
    for l in range(L):
        cg = torch.cat([layers[l]["gate"]["codes"], layers[l]["up"]["codes"]], dim=1)
        sg = torch.cat([layers[l]["gate"]["scales"], layers[l]["up"]["scales"]], dim=1)
        cl, sl = [cg[e] for e in range(E)], [sg[e] for e in range(E)]
        ftables.append((sq.ExpertTable("fwd", "mx", gx["X"], cl, sl, Ygu),
                        sq.ExpertTable("dx", "mx", dYgu, cl, sl, gx["dX"]),
                        sq.ExpertTable("ds", "mx", gx["X"], cl, None, dSgu, acts2=dYgu), cg, sg))

    def run_fused():
        for l in range(L):
            ftables[l][0].run()
            tables[(l, "down")][0].run()
        for l in reversed(range(L)):
            tables[(l, "down")][1].run()
            tables[(l, "down")][2].run()
            ftables[l][1].run()
            ftables[l][2].run()

    fused_ms = timed(run_fused)
    del ftables, dYgu, dYgu_all, Ygu, dSgu
    torch.cuda.empty_cache()
    # QAST: per layer and linear, stacked factors B [E, o, r], A [E, r, G]
    qa = {}
    for (name, o, i) in shapes:
        G = i // 32
        gg = inputs.device_generator(9900 + o)
        qa[name] = dict(B=(torch.randn((E, o, r), generator=gg, device="cuda") * 0.02).to(torch.bfloat16),
                        A=(torch.randn((E, r, G), generator=gg, device="cuda") * 1e-3).to(torch.bfloat16),
                        sc=torch.empty((E, o, G), dtype=torch.uint8, device="cuda"),
                        m=torch.empty((E, o, G), dtype=torch.uint8, device="cuda"),
                        dB=torch.empty((E, o, r), dtype=torch.float32, device="cuda"),
                        dA=torch.empty((E, r, G), dtype=torch.float32, device="cuda"))
        qa[name]["sl"] = [qa[name]["sc"][e] for e in range(E)]
        qa[name]["dSall"] = torch.empty((E, o, G), dtype=torch.float32, device="cuda")
        qa[name]["dSl"] = [qa[name]["dSall"][e] for e in range(E)]
        qa[name]["ws"] = torch.empty(max(1, int(sq.load().sq_qast_factor_grads_batched_workspace(E, o, G, r))),
                                     dtype=torch.uint8, device="cuda")

    qtables = {}
    for l in range(L):
        for (name, _, _) in shapes:
            a, w, q = acts[name], layers[l][name], qa[name]
            qtables[(l, name)] = (sq.ExpertTable("fwd", "mx", a["X"], w["cl"], q["sl"], a["Y"]),
                                  sq.ExpertTable("dx", "mx", a["dY"], w["cl"], q["sl"], a["dX"]),
                                  sq.ExpertTable("ds", "mx", a["X"], w["cl"], None, q["dSl"], acts2=a["dY"]))

    def run_qast():
        for l in range(L):
            for (name, _, _) in shapes:
                q = qa[name]
                sq.sq_qast_scales_batched("mx", layers[l][name]["scales"], q["B"], q["A"], 1.0,
                                          scales_out=q["sc"], mask_out=q["m"])
                qtables[(l, name)][0].run()
        for l in reversed(range(L)):
            for (name, _, _) in reversed(shapes):
                q = qa[name]
                qtables[(l, name)][1].run()
                qtables[(l, name)][2].run()
                sq.sq_qast_factor_grads_batched(q["dSall"], q["m"], q["B"], q["A"], 1.0, dB=q["dB"], dA=q["dA"],
                                                workspace=q["ws"])

    qast_ms = timed(run_qast)
    del qtables

    # QAT-LoRA on the same experts: per linear, stacked factors B [E, o, r],
    # A [E, r, i] and the re-quantised planes (shared across layers)
    qt = {}
    for (name, o, i) in shapes:
        gg = inputs.device_generator(9950 + o)
        qt[name] = dict(B=(torch.randn((E, o, r), generator=gg, device="cuda") * 0.02).to(torch.bfloat16),
                        A=(torch.randn((E, r, i), generator=gg, device="cuda") * 0.02).to(torch.bfloat16),
                        c=torch.empty((E, o, i // 2), dtype=torch.uint8, device="cuda"),
                        s=torch.empty((E, o, i // 32), dtype=torch.uint8, device="cuda"),
                        dB=torch.empty((E, o, r), dtype=torch.float32, device="cuda"),
                        dA=torch.empty((E, r, i), dtype=torch.float32, device="cuda"))
        qt[name]["ws"] = torch.empty(max(1, sq.sq_lora_grads_batched_workspace(Ts, o, i, r)), dtype=torch.uint8,
                                     device="cuda")
    ttables = {}
    for (name, _, _) in shapes:
        a, q = acts[name], qt[name]
        cl, sl = [q["c"][e] for e in range(E)], [q["s"][e] for e in range(E)]
        ttables[name] = (sq.ExpertTable("fwd", "mx", a["X"], cl, sl, a["Y"]),
                         sq.ExpertTable("dx", "mx", a["dY"], cl, sl, a["dX"]))

    def run_qat():
        for l in range(L):
            for (name, _, _) in shapes:
                q = qt[name]
                sq.sq_qat_requant_batched("mx", layers[l][name]["codes"], layers[l][name]["scales"], q["B"], q["A"],
                                          1.0, codes_out=q["c"], scales_out=q["s"])
                ttables[name][0].run()
        for l in reversed(range(L)):
            for (name, _, _) in reversed(shapes):
                q, a = qt[name], acts[name]
                ttables[name][1].run()
                sq.sq_lora_grads_batched(Ts, a["Xall"], a["dYall"], q["B"], q["A"], 1.0, dB=q["dB"], dA=q["dA"],
                                         workspace=q["ws"])

    qat_ms = timed(run_qat)
    out = {"workload": "MXFP4 30B-A3B-shaped MoE stack: 48 layers x 128 experts x {gate, up [768, 2048], "
                       "down [2048, 768]}, 4096 tokens top-8 (32768 routed rows per layer): grouped fwd + dX + dS",
           "expert_rows": {"min": int(min(Ts)), "max": int(max(Ts)), "mean": round(rows / E, 1)},
           "ms": round(ms, 3), "TFLOP": round(flops / 1e12, 2),
           "TFLOP/s": round(flops / (ms * 1e-3) / 1e12, 1),
           "frac_of_bf16_peak": round(flops / (ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 4),
           "fused_gate_up": {"what": "gate and up stacked into one [1536, 2048] weight per expert, as fused-"
                                     "projection MoE layouts store them: 6 grouped products per layer instead of 9, "
                                     "the pair's dX summed in one 1536-deep contraction (the same flops)",
                             "ms": round(fused_ms, 3), "TFLOP/s": round(flops / (fused_ms * 1e-3) / 1e12, 1),
                             "frac_of_bf16_peak": round(flops / (fused_ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 4)},
           "qast_step": {"ms": round(qast_ms, 3), "overhead_ms": round(qast_ms - ms, 3),
                         "note": "batched rank-32 QAST scale step of all experts per linear; the paper reports "
                                 "QAST within noise of its no-STE baseline on its MoE (context only)"},
           "qat_lora_step": {"what": "QAT-LoRA weight-space STE on the native path, rank 32: "
                                     "sq_qat_requant_batched before each grouped forward, grouped dX on the "
                                     "re-quantised codes, sq_lora_grads_batched instead of dS",
                             "ms": round(qat_ms, 3), "ratio_to_scale_step": round(qat_ms / ms, 3),
                             "ratio_to_qast_step": round(qat_ms / qast_ms, 3),
                             "note": "the paper reports 8882 vs 3958 ms per step (2.2x) for QAT-LoRA against "
                                     "Scale-QLoRA on its MoE, through framework ops (context only)"}}
    del layers, acts, qa, qt, tables, ttables
    torch.cuda.empty_cache()
    return out


def dequant_torch(codes, scales):
    """bf16 W from an MXFP4 code plane with torch ops (the comparator's fake-quant
    read-back; the scale-only path never forms W in HBM)."""
    lut = torch.tensor([0.0, 0.5, 1.0, 1.5, 2.0, 3.0, 4.0, 6.0, -0.0, -0.5, -1.0, -1.5, -2.0, -3.0, -4.0, -6.0],
                       device=codes.device)
    O, half = codes.shape
    nib = torch.stack((codes & 15, codes >> 4), dim=-1).reshape(O, 2 * half).long()
    eff = torch.exp2(scales.float() - 127.0).repeat_interleave(32, dim=1)
    return (lut[nib] * eff).to(torch.bfloat16)


def weight_space_ste(sq, codes, scales, Tm, scale_step_ms, L, r=32, steps=2):
    """The framework-style weight-space STE step over the whole model (every
    one of the L x 7 linears, each with its own weight and rank-r factors):
    W' = deq(W) + B A in fp32, RTN fake-quantisation (rtn_quantize, then a
    torch dequant), the three dense bf16 GEMMs through torch (hipBLASLt) with
    dW materialised in fp32, then dB = dW A^T and dA = B^T dW.  Activations
    are shared per shape."""
    shapes = inputs.LLAMA8B_LAYER
    acts = {}
    for k, (name, o, i) in enumerate(shapes):
        acts[name] = dict(X=inputs.device_bf16_normal(5100 + k, (Tm, i)), dY=inputs.device_bf16_normal(5200 + k, (Tm, o)),
                          qc=torch.empty((o, i // 2), dtype=torch.uint8, device="cuda"),
                          qs=torch.empty((o, i // 32), dtype=torch.uint8, device="cuda"))
    items = []
    for n, (name, o, i) in enumerate(shapes * L):
        g = inputs.device_generator(5300 + n)
        items.append(dict(name=name, Wd=dequant_torch(codes[n], scales[n]),
                          B=(torch.randn((o, r), generator=g, device="cuda") * 0.02).to(torch.bfloat16),
                          A=(torch.randn((r, i), generator=g, device="cuda") * 0.02).to(torch.bfloat16)))

    def run():
        for it in items:
            a = acts[it["name"]]
            Weff = (it["Wd"].float() + torch.mm(it["B"], it["A"], out_dtype=torch.float32)).to(torch.bfloat16)
            sq.rtn_quantize("mx", Weff, sq.TIE_EVEN, 0.0, codes=a["qc"], scales=a["qs"])
            Wfq = dequant_torch(a["qc"], a["qs"])
            torch.mm(a["X"], Wfq.t())                                              # Y
            torch.mm(a["dY"], Wfq)                                                 # dX
            dW = torch.mm(a["dY"].t(), a["X"], out_dtype=torch.float32)
            torch.mm(dW, it["A"].float().t())                                      # dB
            torch.mm(it["B"].float().t(), dW)                                      # dA

    run()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(steps):
        run()
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / steps
    del items, acts
    torch.cuda.empty_cache()
    return {"ms": round(ms, 2), "ratio_to_scale_step": round(ms / scale_step_ms, 2), "rank": r,
            "note": "all 224 linears measured; the paper reports 3.9x per step on its own hardware (context only)"}


def model_mlp_nv(sq, steps=10):
    """NVFP4 MLP projections at 8B shape, 8192 tokens: gate and up [14336, 4096],
    down [4096, 14336], block 16, E4M3 scales of |N(0, 1)| with ws2 = 1/448,
    codes uniform, X and dY ~ N(0, 1) bf16; forward, dX and dS of each, every
    product launched `steps` times back to back between two events."""
    Tm = 8192
    ws2 = float(np.float32(1.0 / 448.0))
    out, total_ms, total_flop = {}, 0.0, 0.0
    for k, (name, o, i) in enumerate((("gate", 14336, 4096), ("up", 14336, 4096), ("down", 4096, 14336))):
        codes = inputs.device_codes_uniform(9700 + k, o, i)
        sc = inputs.device_e4m3_abs_normal(9710 + k, o, i // 16)
        X = inputs.device_bf16_normal(9720 + k, (Tm, i))
        dY = inputs.device_bf16_normal(9730 + k, (Tm, o))
        Y = torch.empty((Tm, o), dtype=torch.bfloat16, device="cuda")
        dX = torch.empty((Tm, i), dtype=torch.bfloat16, device="cuda")
        dS = torch.empty((o, i // 16), dtype=torch.float32, device="cuda")
        calls = {"fwd": lambda: sq.sq_fwd("nv", X, codes, sc, ws2, Y=Y),
                 "dx": lambda: sq.sq_bwd_dx("nv", dY, codes, sc, ws2, dX=dX),
                 "ds": lambda: sq.sq_bwd_dscale("nv", X, dY, codes, dS=dS)}
        flop = 2.0 * Tm * o * i
        for prod, fn in calls.items():
            for _ in range(30):              # the first launches after the input generation run slower
                fn()
            torch.cuda.synchronize()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            for _ in range(steps):
                fn()
            e1.record()
            torch.cuda.synchronize()
            ms = e0.elapsed_time(e1) / steps
            out[f"{name}_{prod}"] = {"ms": round(ms, 4), "TFLOP/s": round(flop / (ms * 1e-3) / 1e12, 1)}
            total_ms += ms
            total_flop += flop
        del codes, sc, X, dY, Y, dX, dS
    out["all"] = {"ms": round(total_ms, 3), "TFLOP/s": round(total_flop / (total_ms * 1e-3) / 1e12, 1),
                  "frac_of_bf16_peak": round(total_flop / (total_ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 4)}
    out["workload"] = ("NVFP4 gate/up 14336x4096 and down 4096x14336, 8192 tokens: fwd + dX + dS of each "
                       "(the sum of the per-product times)")
    torch.cuda.empty_cache()
    return out


def cpu_baseline(X, dY, codes, sb, delta, src, Wm_host):
    """The oracle on the host cores over one whole step of the same layer:
    dequant + fwd + dX + dS (fp64 numpy matmuls over all 4096 tokens), scale
    swap + merge, and RTN re-quantisation of the merged weight.  Reported like
    `value`: 6*T*O*I flops over the step's time, in TFLOP/s."""
    from oracle import linear, merge, rtn
    try:
        from threadpoolctl import threadpool_info
        threads = max([d.get("num_threads", 1) for d in threadpool_info()] or [1])
    except Exception:
        threads = os.cpu_count()
    Xs = X.double().numpy()
    dYs = dY.double().numpy()
    reps, t_gemm, t_merge, t_rtn = 0, 0.0, 0.0, 0.0
    while reps < 1 or (t_gemm + t_merge + t_rtn < 10.0 and reps < 30):
        t0 = time.perf_counter()
        W = linear.dequant(FMT, codes, sb)
        linear.forward(Xs, W)
        linear.backward_dx(dYs, W)
        linear.backward_dscale(FMT, Xs, dYs, codes)
        t1 = time.perf_counter()
        plane = merge.merge_copy(sb, src)
        merge.merge_delta(FMT, plane, delta)
        t2 = time.perf_counter()
        rtn.quantize(FMT, Wm_host, rtn.TIE_EVEN)
        t3 = time.perf_counter()
        t_gemm += t1 - t0
        t_merge += t2 - t1
        t_rtn += t3 - t2
        reps += 1
    per_step = (t_gemm + t_merge + t_rtn) / reps
    flops = 6.0 * T * O * I
    return {"value": round(flops / per_step / 1e12, 5), "unit": "TFLOP/s", "cores": int(threads),
            "kind": "oracle",
            "sample": f"{reps} whole step(s) of the same 4096x4096 MXFP4 layer, 4096 tokens; per step "
                      f"dequant+fwd+dX+dS {t_gemm / reps:.2f} s (fp64 numpy matmuls), swap+merge "
                      f"{t_merge / reps:.3f} s, RTN {t_rtn / reps:.2f} s",
            "seconds": round(t_gemm + t_merge + t_rtn, 2),
            "host_cpus": os.cpu_count()}


def hbm_copy_ceiling(sq, mib=2048, reps=10):
    """Measured streaming ceilings beside the 8 TB/s spec: a 2 GiB
    device-to-device copy through torch (copy_) and through the copy mode of
    sq_merge_scales (one plane; 1:1 reads and writes), and a read-only pass
    over two 2 GiB buffers (the byte audit, sq_byte_diff), in bytes moved per
    second."""
    nb = mib << 20
    a = torch.empty(nb, dtype=torch.uint8, device="cuda").fill_(7)
    b = torch.empty_like(a)
    res = {"bytes_each_way": nb}
    counts = torch.zeros(2, dtype=torch.int64, device="cuda")
    for name, fn in (("torch_copy", lambda: b.copy_(a)), ("sq_merge_copy", lambda: sq.sq_merge_scales(FMT, b, src=a)),
                     ("read_only_sq_byte_diff", lambda: sq.sq_byte_diff(a, b, counts=counts))):
        for _ in range(2):
            fn()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            fn()
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / reps
        res[name] = {"ms": round(ms, 3), "GB/s": round(2 * nb / (ms * 1e-3) / 1e9, 1),
                     "frac_of_8TB/s": round(2 * nb / (ms * 1e-3) / 1e9 / PEAK_HBM_GBS, 4)}
    del counts
    del a, b
    torch.cuda.empty_cache()
    return res


def cpu_plan():
    """The oracle timed per workload on the host cores, with all BLAS threads
    and with one (threadpoolctl): the tiny MXFP4 layer in full (forward, dX,
    dS and the merge of its perturbed plane); the NVFP4 MLP projections at 8192
    tokens in full with all threads, and on 256 of the 8192 tokens with one
    (scaled by 32, labelled extrapolated); the 8B model step as layer 0's seven
    linears at 4096 tokens, reported x32 (extrapolated); the lifecycle over
    the model's first 8 linears (NVFP4 merge of their scale planes, MXFP4 RTN
    of the first 256 rows of their bf16 weights), scaled to all 224 by bytes
    (extrapolated)."""
    from oracle import linear, merge, rtn
    from threadpoolctl import threadpool_limits
    ws2 = float(np.float32(1.0 / 448.0))

    def gemms(fmt, X, dY, codes, sb, w2):
        W = linear.dequant(fmt, codes, sb, w2)
        linear.forward(X, W)
        linear.backward_dx(dY, W)
        linear.backward_dscale(fmt, X, dY, codes)

    def timed(fn):
        t0 = time.perf_counter()
        fn()
        return time.perf_counter() - t0

    def layer(fmt, Tn, o, i, seed):
        X = inputs.bf16_normal(seed, (Tn, i)).double().numpy()
        dY = inputs.bf16_normal(seed + 1, (Tn, o)).double().numpy()
        codes = inputs.codes_uniform(seed + 2, o, i)
        sb = (inputs.e8m0_uniform_exponents(seed + 3, o, i // 32, -8, -3) if fmt == "mx"
              else inputs.e4m3_abs_normal(seed + 3, o, i // 16))
        return X, dY, codes, sb

    out = {}
    # tiny MXFP4 layer, whole
    X, dY, codes, sb = layer("mx", 64, 256, 512, 1000)
    dlt = inputs.e8m0_step_delta(1009, sb, 0.10)
    fl = 6.0 * 64 * 256 * 512
    for label, nthreads in (("all_threads", None), ("one_thread", 1)):
        with threadpool_limits(limits=nthreads):
            tiny = lambda: (gemms("mx", X, dY, codes, sb, 1.0), merge.merge_delta("mx", sb, dlt))  # noqa: E731
            tiny()                                           # the thread pool starts up on the first call
            t = min(timed(tiny) for _ in range(3))
        out.setdefault("tiny_mxfp4_64x256x512", {})[label] = {"seconds": round(t, 4),
                                                             "GFLOP/s": round(fl / t / 1e9, 2)}
    # NVFP4 MLP at 8192 tokens
    mlp = (("gate", 14336, 4096), ("up", 14336, 4096), ("down", 4096, 14336))
    res = {}
    t_all = 0.0
    for k, (name, o, i) in enumerate(mlp):
        X, dY, codes, sb = layer("nv", 8192, o, i, 9000 + 10 * k)
        t_all += timed(lambda: gemms("nv", X, dY, codes, sb, ws2))
        del X, dY
    fl = 6.0 * 8192 * sum(o * i for (_, o, i) in mlp)
    res["all_threads"] = {"seconds": round(t_all, 2), "TFLOP/s": round(fl / t_all / 1e12, 4), "measured": "full"}
    t_one = 0.0
    with threadpool_limits(limits=1):
        for k, (name, o, i) in enumerate(mlp):
            X, dY, codes, sb = layer("nv", 256, o, i, 9100 + 10 * k)
            t_one += timed(lambda: gemms("nv", X, dY, codes, sb, ws2))
    res["one_thread"] = {"seconds_extrapolated": round(t_one * 32, 1), "TFLOP/s": round(fl / (t_one * 32) / 1e12, 5),
                         "measured": "256 of 8192 tokens, x32 (extrapolated)"}
    out["mlp_nvfp4_t8192"] = res
    # 8B step: layer 0 at 4096 tokens, x32
    t_l0 = 0.0
    for k, (name, o, i) in enumerate(inputs.LLAMA8B_LAYER):
        X, dY, codes, sb = layer("mx", 4096, o, i, 9200 + 10 * k)
        t_l0 += timed(lambda: gemms("mx", X, dY, codes, sb, 1.0))
        del X, dY
    fl = 6.0 * 4096 * sum(o * i for (_, o, i) in inputs.LLAMA8B_LAYER) * inputs.LLAMA8B_LAYERS
    out["step_8b"] = {"seconds_extrapolated": round(t_l0 * inputs.LLAMA8B_LAYERS, 1),
                      "TFLOP/s": round(fl / (t_l0 * inputs.LLAMA8B_LAYERS) / 1e12, 4),
                      "measured": f"layer 0 (7 linears) in {t_l0:.1f} s with all threads, x32 (extrapolated)"}
    # lifecycle: the first 8 linears' planes and weights, scaled by bytes to 224
    first = inputs.LLAMA8B_LAYER + inputs.LLAMA8B_LAYER[:1]
    t_merge = t_rtn = 0.0
    mbytes = rbytes = 0
    for k, (name, o, i) in enumerate(first):
        sbn = inputs.e4m3_abs_normal(9300 + k, o, i // 16)
        d = inputs.relative_jitter(9400 + k, sbn.astype(np.float64), 0.02)
        t_merge += timed(lambda: merge.merge_delta("nv", sbn, d, ws2))
        mbytes += 6 * sbn.size
        Wm = inputs.bf16_normal(9500 + k, (256, i)).float().numpy() * np.float32(0.01)
        t_rtn += timed(lambda: rtn.quantize("mx", Wm, rtn.TIE_EVEN))
        rbytes += 256 * i * 2 + 256 * i // 2 + 256 * i // 32
        del Wm
    tot_m = 6 * sum(o * i // 16 for (_, o, i) in inputs.LLAMA8B_LAYER) * inputs.LLAMA8B_LAYERS
    tot_r = sum(o * i * 2 + o * i // 2 + o * i // 32 for (_, o, i) in inputs.LLAMA8B_LAYER) * inputs.LLAMA8B_LAYERS
    out["lifecycle_8b"] = {"nv_merge": {"seconds_extrapolated": round(t_merge * tot_m / mbytes, 1),
                                        "GB/s": round(mbytes / t_merge / 1e9, 3)},
                           "mx_rtn": {"seconds_extrapolated": round(t_rtn * tot_r / rbytes, 1),
                                      "GB/s": round(rbytes / t_rtn / 1e9, 3)},
                           "measured": "merge: the first 8 linears' scale planes; RTN: the first 256 rows of "
                                       "each of the first 8 linears; both scaled to all 224 by bytes "
                                       "(extrapolated)"}
    out["cores"] = os.cpu_count()
    return out


def main():
    args = parse()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU: the library has no multi-GPU path (run with --gpus 1)", file=sys.stderr)
        sys.exit(2)
    from paper_2609_04526_amd import sq
    sq.load()
    torch.cuda.init()

    X, dY, codes, sb, delta, src = layer_inputs()
    Xd, dYd = X.cuda(), dY.cuda()
    codes_d = torch.from_numpy(codes).cuda()
    sb_d = torch.from_numpy(sb).cuda()
    base_plane = torch.from_numpy(src.reshape(-1)).cuda()
    work_plane = torch.empty_like(base_plane)
    delta_d = torch.from_numpy(delta.reshape(-1)).cuda()
    Wm = merged_weight_bf16(codes_d, sb_d, sq)
    Y = torch.empty((T, O), dtype=torch.bfloat16, device="cuda")
    dX = torch.empty((T, I), dtype=torch.bfloat16, device="cuda")
    dS = torch.empty((O, I // 32), dtype=torch.float32, device="cuda")
    rc = torch.empty((O, I // 2), dtype=torch.uint8, device="cuda")
    rs = torch.empty((O, I // 32), dtype=torch.uint8, device="cuda")

    calls = {
        "sq_fwd": lambda: sq.sq_fwd(FMT, Xd, codes_d, sb_d, 1.0, Y=Y),
        "sq_bwd_dx": lambda: sq.sq_bwd_dx(FMT, dYd, codes_d, sb_d, 1.0, dX=dX),
        "sq_bwd_dscale": lambda: sq.sq_bwd_dscale(FMT, Xd, dYd, codes_d, dS=dS),
        "merge_copy": lambda: sq.sq_merge_scales(FMT, work_plane, src=base_plane),
        "merge_delta": lambda: sq.sq_merge_scales(FMT, work_plane, delta=delta_d),
        "rtn_quantize": lambda: sq.rtn_quantize(FMT, Wm, sq.TIE_EVEN, 0.0, codes=rc, scales=rs),
    }
    names = list(calls)

    def step():
        for n in names:
            calls[n]()

    # The chip needs some tens of milliseconds of load before its clock
    # settles: a fixed 300 ms of untimed steps comes before the warmup steps,
    # whatever --warmup asks for.
    t_pre = time.perf_counter()
    while time.perf_counter() - t_pre < 0.3:
        step()
        torch.cuda.synchronize()
    preheat_ms = (time.perf_counter() - t_pre) * 1e3
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms_step = wall * 1e3 / args.steps

    # Per-kernel durations: each call launched `steps` times back to back on
    # the launch stream between two HIP events (an event record between every
    # launch would add a cache-flushing marker to each, so the timed step loop
    # above carries none).
    per = {}
    stream = torch.cuda.current_stream()
    for n in names:
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        calls[n]()
        e0.record(stream)
        for _ in range(args.steps):
            calls[n]()
        e1.record(stream)
        torch.cuda.synchronize()
        per[n] = e0.elapsed_time(e1) / args.steps
    # the vendor library's dense bf16 GEMM of the same shape (hipBLASLt through
    # torch), as a measured ceiling next to the spec peak
    Wd = Wm  # any bf16 [O, I] operand
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.mm(Xd, Wd.t())
    e0.record(stream)
    for _ in range(args.steps):
        torch.mm(Xd, Wd.t())
    e1.record(stream)
    torch.cuda.synchronize()
    vendor_ms = e0.elapsed_time(e1) / args.steps

    copy_ceiling = hbm_copy_ceiling(sq)

    gemm_flops = 2.0 * T * O * I
    tflops = 3 * gemm_flops / (ms_step * 1e-3) / 1e12
    kernels = {}
    for n in names[:3]:
        kernels[n] = {"ms": round(per[n], 4), "TFLOP/s": round(gemm_flops / (per[n] * 1e-3) / 1e12, 1)}
    for n in names[3:5]:
        nbytes = (2 if n == "merge_copy" else 6) * O * (I // 32)
        kernels[n] = {"ms": round(per[n], 4), "GB/s": round(nbytes / (per[n] * 1e-3) / 1e9, 1)}
    rtn_bytes = O * I * 2 + O * I // 2 + O * I // 32
    kernels["rtn_quantize"] = {"ms": round(per["rtn_quantize"], 4),
                               "GB/s": round(rtn_bytes / (per["rtn_quantize"] * 1e-3) / 1e9, 1)}
    dom = max(names[:3], key=lambda n: per[n])
    ach = gemm_flops / (per[dom] * 1e-3) / 1e12
    roofline = {"bound": "mfma", "kernel": dom, "achieved": round(ach, 1), "peak": PEAK_BF16_TFLOPS,
                "unit": "TFLOP/s", "frac": round(ach / PEAK_BF16_TFLOPS, 4),
                "traffic": measured_traffic(dom)}

    out = {
        "metric": METRIC,
        "value": round(tflops, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "preheat_ms": round(preheat_ms, 1),
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": "MXFP4 attention projection 4096x4096, 4096 tokens (4x1024): "
                               "fwd+dX+dS, scale swap+merge, RTN re-quantisation",
                   "T": T, "O": O, "I": I, "format": "mxfp4", "block": 32},
        "frac_of_bf16_peak": round(tflops / PEAK_BF16_TFLOPS, 4),
        "kernels": kernels,
        "roofline": roofline,
        "vendor_bf16_gemm": {"what": "torch.mm bf16 X W^T, same 4096^3 shape (hipBLASLt)",
                             "ms": round(vendor_ms, 4),
                             "TFLOP/s": round(gemm_flops / (vendor_ms * 1e-3) / 1e12, 1)},
        "hbm_copy_ceiling": copy_ceiling,
    }
    if args.calib_copy_mib:
        nb = args.calib_copy_mib << 20
        a = torch.randint(0, 255, (nb,), dtype=torch.uint8, device="cuda")
        b = torch.empty_like(a)
        for _ in range(3):
            sq.sq_merge_scales(FMT, b, src=a)
        torch.cuda.synchronize()
        out["calib_copy_bytes"] = nb
    if not args.no_model_merge:
        out["merge_8b"] = model_merge(sq, 20)
    if not args.no_model_step:
        out["step_8b"] = model_step(sq, 3, 1)
        torch.cuda.empty_cache()
    if not args.no_mlp_nv:
        out["mlp_nvfp4_t8192"] = model_mlp_nv(sq)
    if not args.no_moe:
        out["moe_30b_a3b"] = model_moe(sq)
        torch.cuda.empty_cache()
    if not args.no_lifecycle:
        out["lifecycle_8b"] = model_lifecycle(sq)
        torch.cuda.empty_cache()
    if "merge_8b" in out and "lifecycle_8b" in out:
        # a hot swap of the served task: the scale-only swap (NVFP4 planes
        # copied) against re-quantising every linear's weights
        sw = out["merge_8b"]["nv_swap"]["ms"]
        rq = out["lifecycle_8b"]["nv"]
        out["swap_nvfp4_8b"] = {
            "scale_swap_ms": sw,
            "requant_swap_rtn_ms": rq["even"]["ms"],
            "requant_swap_fused_ms": rq["requant_swap_fused"]["ms"],
            "ratio_rtn": round(rq["even"]["ms"] / sw, 1),
            "ratio_fused": round(rq["requant_swap_fused"]["ms"] / sw, 1),
            "what": "scale-only swap of all 224 NVFP4 scale planes (sq_merge_scales_grouped copy) against "
                    "re-quantising all 224 linears: rtn_quantize_grouped of the resident bf16 W + B A, and the "
                    "fused pass from base codes + scales + adapter (sq_qat_requant)",
            "note": "the paper reports 0.059 s against 7.45 s (~125x) for Llama-8B NVFP4 on one H200, "
                    "through its own loaders (context only)"}
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(X, dY, codes, sb, delta, src, Wm.float().cpu().numpy())
        if not args.no_cpu_plan:
            out["cpu_baseline"]["plan"] = cpu_plan()
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
