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
The line also carries per-kernel times from HIP events on the launch stream,
the roofline of the dominant kernel against MI355X's dense bf16 MFMA peak,
the whole-model scale-plane merge in GB/s against the 8 TB/s HBM peak, and
the CPU oracle timed on a bounded sample of the same workload.
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
    p.add_argument("--warmup", type=int, default=10)
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--no-model-merge", action="store_true")
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


def model_merge(sq, steps):
    """Grouped merges over every scale plane of the 8B model (32 layers x 7
    linears): MXFP4 delta merge (218,103,808 scales, 6 bytes per scale moved),
    NVFP4 delta merge (436,207,616 scales, 6 bytes) and the MXFP4 hot swap
    (copy mode, 2 bytes per scale)."""
    out = {}
    for name, fmt, block, mode in (("mx_delta", "mx", 32, "delta"), ("nv_delta", "nv", 16, "delta"),
                                   ("mx_swap", "mx", 32, "copy")):
        sizes = [o * (i // block) for _ in range(inputs.LLAMA8B_LAYERS) for (_, o, i) in inputs.LLAMA8B_LAYER]
        total = sum(sizes)
        if fmt == "mx":
            scales = torch.randint(100, 140, (total,), dtype=torch.uint8, device="cuda")
        else:
            scales = torch.randint(0x20, 0x70, (total,), dtype=torch.uint8, device="cuda")
        aux = (torch.randn(total, device="cuda") * 1e-3).float() if mode == "delta" else \
            torch.randint(100, 140, (total,), dtype=torch.uint8, device="cuda")
        descs, off = [], 0
        for n in sizes:
            d = dict(fmt=fmt, scales=scales[off:off + n], ws2=1.0 / 448.0)
            d["delta" if mode == "delta" else "src"] = aux[off:off + n]
            descs.append(d)
            off += n
        group = sq.MergeGroup(descs)
        for _ in range(3):
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
        out[name] = {"scales": total, "planes": len(sizes), "bytes_per_scale": bps, "ms": round(ms, 4),
                     "GB/s": round(gbs, 1), "peak": PEAK_HBM_GBS, "frac": round(gbs / PEAK_HBM_GBS, 4)}
        del scales, aux, descs, group
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


def main():
    args = parse()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU: this build has no multi-GPU path (run with --gpus 1)", file=sys.stderr)
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

    names = ["sq_fwd", "sq_bwd_dx", "sq_bwd_dscale", "merge_copy", "merge_delta", "rtn_quantize"]
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(len(names) + 1)] for _ in range(args.steps)]

    def step(e=None):
        if e: e[0].record()
        sq.sq_fwd(FMT, Xd, codes_d, sb_d, 1.0, Y=Y)
        if e: e[1].record()
        sq.sq_bwd_dx(FMT, dYd, codes_d, sb_d, 1.0, dX=dX)
        if e: e[2].record()
        sq.sq_bwd_dscale(FMT, Xd, dYd, codes_d, dS=dS)
        if e: e[3].record()
        sq.sq_merge_scales(FMT, work_plane, src=base_plane)
        if e: e[4].record()
        sq.sq_merge_scales(FMT, work_plane, delta=delta_d)
        if e: e[5].record()
        sq.rtn_quantize(FMT, Wm, sq.TIE_EVEN, 0.0, codes=rc, scales=rs)
        if e: e[6].record()

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for k in range(args.steps):
        step(ev[k])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms_step = wall * 1e3 / args.steps
    per = {n: sum(ev[k][i].elapsed_time(ev[k][i + 1]) for k in range(args.steps)) / args.steps
           for i, n in enumerate(names)}
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
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(X, dY, codes, sb, delta, src, Wm.float().cpu().numpy())
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
