"""Seeded synthetic inputs for the frozen-code linear layer.

Shared by the tests, the smoke entry and the benchmark so that the GPU path and
the oracle consume the same bytes.  This module draws random numbers and lays
them out in the storage formats' byte layouts; it performs none of the
method's arithmetic (no dequantisation, GEMM, merge or re-quantisation).  bf16
and E4M3 bytes are produced with torch's own dtype casts.

Every generator takes a seed; the workload recipes use numpy PCG64 seeded with
1000 * workload_id + tensor_id.
"""

import numpy as np
import torch


def rng(seed: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(seed))


def bf16_normal(seed: int, shape) -> torch.Tensor:
    """N(0, 1) samples rounded to bf16 (CPU tensor)."""
    x = rng(seed).standard_normal(size=shape, dtype=np.float32)
    return torch.from_numpy(x).to(torch.bfloat16)


def codes_uniform(seed: int, O: int, I: int) -> np.ndarray:
    """Packed E2M1 code plane [O, I/2]: every nibble uniform over all 16 codes."""
    return rng(seed).integers(0, 256, size=(O, I // 2), dtype=np.uint8)


def e8m0_uniform_exponents(seed: int, O: int, G: int, lo: int, hi: int) -> np.ndarray:
    """E8M0 bytes whose exponents are uniform integers in [lo, hi] (inclusive)."""
    e = rng(seed).integers(lo, hi + 1, size=(O, G))
    return (e + 127).astype(np.uint8)


def e8m0_normal_exponents(seed: int, O: int, G: int, mean: float, std: float) -> np.ndarray:
    """E8M0 bytes with exponents rint(N(mean, std)), kept inside [-127, 127]."""
    e = np.rint(rng(seed).normal(mean, std, size=(O, G)))
    return (np.clip(e, -127, 127) + 127).astype(np.uint8)


def e4m3_abs_normal(seed: int, O: int, G: int) -> np.ndarray:
    """E4M3 bytes of |N(0, 1)| samples (torch float8_e4m3fn cast, round to nearest even)."""
    x = np.abs(rng(seed).standard_normal(size=(O, G), dtype=np.float32))
    return torch.from_numpy(x).to(torch.float8_e4m3fn).view(torch.uint8).numpy()


def e8m0_step_delta(seed: int, scale_bytes: np.ndarray, frac: float) -> np.ndarray:
    """fp32 delta that moves round(frac * n) seeded blocks one exponent step up or
    down (fair coin) and leaves the others at zero: for a block at 2**e the delta
    is +2**e (up) or -2**(e-1) (down)."""
    b = np.asarray(scale_bytes, dtype=np.uint8)
    g = rng(seed)
    n = b.size
    pick = g.permutation(n)[: int(round(frac * n))]
    up = g.integers(0, 2, size=pick.size).astype(bool)
    e = b.reshape(-1)[pick].astype(np.int64) - 127
    d = np.zeros(n, dtype=np.float32)
    d[pick] = np.where(up, np.ldexp(1.0, e), -np.ldexp(1.0, e - 1)).astype(np.float32)
    return d.reshape(b.shape)


def relative_jitter(seed: int, magnitudes: np.ndarray, rel_std: float) -> np.ndarray:
    """fp32 N(0, rel_std * |m|) noise, elementwise."""
    m = np.asarray(magnitudes, dtype=np.float64)
    return (rng(seed).standard_normal(size=m.shape) * rel_std * np.abs(m)).astype(np.float32)


def lora_factors(seed: int, O: int, I: int, r: int, std: float):
    """B [O, r], A [r, I] ~ N(0, std) fp32 (the rank-r weight delta of the naive merge)."""
    g = rng(seed)
    B = (g.standard_normal(size=(O, r)) * std).astype(np.float32)
    A = (g.standard_normal(size=(r, I)) * std).astype(np.float32)
    return B, A


# Llama-3.1-8B dense linear shapes (out, in) per decoder layer; 32 layers.
LLAMA8B_LAYER = (
    ("q", 4096, 4096), ("k", 1024, 4096), ("v", 1024, 4096), ("o", 4096, 4096),
    ("gate", 14336, 4096), ("up", 14336, 4096), ("down", 4096, 14336),
)
LLAMA8B_LAYERS = 32


# ---------------------------------------------------------------- on device
# Whole-model workloads (tens of GB of activations) are drawn on the GPU with
# torch's seeded Philox generator instead of numpy; a test that checks such an
# output reads the same device bytes back.

def device_generator(seed: int) -> torch.Generator:
    g = torch.Generator(device="cuda")
    g.manual_seed(seed)
    return g


def device_bf16_normal(seed: int, shape) -> torch.Tensor:
    """N(0, 1) samples in bf16, drawn on the current GPU."""
    return torch.randn(shape, generator=device_generator(seed), device="cuda", dtype=torch.float32).to(torch.bfloat16)


def device_codes_uniform(seed: int, O: int, I: int) -> torch.Tensor:
    """Packed E2M1 code plane [O, I/2] on the GPU, every nibble uniform."""
    return torch.randint(0, 256, (O, I // 2), generator=device_generator(seed), device="cuda", dtype=torch.uint8)


def device_e8m0_normal_exponents(seed: int, O: int, G: int, mean: float, std: float) -> torch.Tensor:
    """E8M0 bytes with exponents rint(N(mean, std)) clipped to [-127, 127], on the GPU."""
    e = torch.randn((O, G), generator=device_generator(seed), device="cuda") * std + mean
    return (torch.round(e).clamp_(-127, 127) + 127).to(torch.uint8)


def device_task_delta(seed: int, eff: torch.Tensor, fmt: str) -> torch.Tensor:
    """A task's fp32 scale delta on the device, for effective scales `eff` (fp32):
    MXFP4: a one-exponent step (up: +eff, down: -eff/2, fair coin) on a seeded 5%
    of blocks plus N(0, 0.01 eff) jitter (which rounds away on the log grid);
    NVFP4: N(0, 0.02 eff)."""
    g = device_generator(seed)
    if fmt == "mx":
        pick = torch.rand(eff.shape, generator=g, device="cuda") < 0.05
        up = torch.rand(eff.shape, generator=g, device="cuda") < 0.5
        step = torch.where(up, eff, -0.5 * eff)
        jitter = torch.randn(eff.shape, generator=g, device="cuda") * (0.01 * eff)
        return torch.where(pick, step, torch.zeros_like(eff)) + jitter
    return torch.randn(eff.shape, generator=g, device="cuda") * (0.02 * eff)


def device_e4m3_abs_normal(seed: int, O: int, G: int) -> torch.Tensor:
    """E4M3 bytes of |N(0, 1)| samples on the GPU (torch's round-to-nearest-even cast)."""
    x = torch.randn((O, G), generator=device_generator(seed), device="cuda").abs()
    return x.to(torch.float8_e4m3fn).view(torch.uint8)
