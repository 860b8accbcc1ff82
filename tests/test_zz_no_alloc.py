"""sq_bwd_dscale_noalloc (static device scratch) against sq_bwd_dscale (caller
workspace): bitwise equal dS on consecutive calls, the second smaller than the
first, on shapes that split the token sum (partial planes in the scratch) and
on one that does not; and within the oracle's tolerance."""

import numpy as np
import pytest
import torch

from conftest import ensure_library, gpu_ready
from oracle import codec, linear
from paper_2609_04526_amd import inputs

pytestmark = [pytest.mark.gpu, pytest.mark.skipif(not gpu_ready(), reason="needs a GPU")]


@pytest.fixture(scope="module")
def sq():
    ensure_library()
    from paper_2609_04526_amd import sq as _sq
    return _sq


def _layer(fmt, T, O, I, seed):
    X = inputs.bf16_normal(seed, (T, I)).cuda()
    dY = inputs.bf16_normal(seed + 1, (T, O)).cuda()
    codes = torch.from_numpy(inputs.codes_uniform(seed + 2, O, I)).cuda()
    return X, dY, codes


# (fmt, T, O, I): the first two split the token sum; the third is the NVFP4
# key/value projection shape (64 tiles of 256 x 256, 4 token ranges: partial
# planes of exactly the scratch's 4 MiB); the last runs without a split
CALLS = [("nv", 1000, 520, 512), ("mx", 700, 264, 256), ("nv", 4096, 1024, 4096), ("mx", 64, 256, 512)]


def test_noalloc_equals_workspace_entry_point(sq):
    for k, (fmt, T, O, I) in enumerate(CALLS):
        ws = sq.sq_bwd_dscale_workspace(fmt, T, O, I)
        print(f"[no-alloc] call {k}: fmt={fmt} T={T} O={O} I={I} workspace={ws}", flush=True)
        assert ws <= 4 << 20
        X, dY, codes = _layer(fmt, T, O, I, seed=7000 + 10 * k)
        want = sq.sq_bwd_dscale(fmt, X, dY, codes)
        # the static scratch keeps the previous call's planes: poison the
        # output so a stale or missing write shows
        got = torch.full_like(want, float("nan"))
        sq.sq_bwd_dscale_noalloc(fmt, X, dY, codes, got)
        torch.cuda.synchronize()
        assert torch.equal(got, want), k
        if T * O * I <= 1000 * 520 * 512:
            Xd, dYd = X.double().cpu().numpy(), dY.double().cpu().numpy()
            ref = linear.backward_dscale(fmt, Xd, dYd, codes.cpu().numpy())
            err = np.linalg.norm(got.cpu().numpy() - ref) / np.linalg.norm(ref)
            assert err <= 2e-3, (k, err)
            assert codec.BLOCK[fmt] * got.shape[1] == I


def test_noalloc_zero_tokens_writes_zeros(sq):
    O, I = 64, 128
    codes = torch.from_numpy(inputs.codes_uniform(5, O, I)).cuda()
    X = torch.empty((0, I), dtype=torch.bfloat16, device="cuda")
    dY = torch.empty((0, O), dtype=torch.bfloat16, device="cuda")
    dS = torch.full((O, I // 32), 7.0, device="cuda")
    sq.sq_bwd_dscale_noalloc("mx", X, dY, codes, dS)
    torch.cuda.synchronize()
    assert torch.count_nonzero(dS).item() == 0
