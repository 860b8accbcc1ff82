"""C-ABI checks that need no GPU: the library loads, exports every entry point
the header declares, and rejects bad arguments on the host before any launch."""

import ctypes
import os
import re

import pytest

from conftest import ROOT, ensure_library

HEADER = os.path.join(ROOT, "include", "scaleqlora.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return re.findall(r"^(?:int|size_t|const char\s*\*)\s*(\w+)\s*\(", text, flags=re.M)


@pytest.fixture(scope="module")
def lib():
    return ensure_library()


def test_header_declares_the_boundary():
    names = set(declared_functions())
    assert {"sq_fwd", "sq_bwd_dx", "sq_bwd_dscale", "sq_merge_scales", "rtn_quantize"} <= names


def test_every_declared_symbol_is_exported(lib):
    for name in declared_functions():
        assert hasattr(lib, name), name


def test_status_strings_and_version(lib):
    from paper_2609_04526_amd import sq
    assert lib.sq_status_str(0) == b"SQ_OK"
    assert lib.sq_status_str(-2).startswith(b"SQ_ERR_SHAPE")
    assert sq.abi_version() == 1


def test_merge_desc_layout_matches_header():
    from paper_2609_04526_amd import sq
    assert ctypes.sizeof(sq.MergeDesc) == 48
    assert sq.MergeDesc.ws2.offset == 32 and sq.MergeDesc.reserved.offset == 44


def test_descriptor_layouts_match_the_c_compiler(tmp_path):
    """sizeof / offsetof of the header's descriptor structs, printed by a C
    program built with gcc, against the ctypes mirrors."""
    import subprocess
    from paper_2609_04526_amd import sq
    src = tmp_path / "layout.c"
    src.write_text(
        '#include <stddef.h>\n#include <stdio.h>\n#include "scaleqlora.h"\n'
        'int main(void) {\n'
        '  printf("%zu %zu %zu\\n", sizeof(sq_merge_desc), offsetof(sq_merge_desc, ws2),'
        ' offsetof(sq_merge_desc, reserved));\n'
        '  printf("%zu %zu %zu %zu\\n", sizeof(sq_expert_desc), offsetof(sq_expert_desc, T),'
        ' offsetof(sq_expert_desc, ws2), offsetof(sq_expert_desc, reserved));\n'
        '  printf("%zu %zu %zu %zu %zu\\n", sizeof(sq_rtn_desc), offsetof(sq_rtn_desc, ws2_out),'
        ' offsetof(sq_rtn_desc, ws2_in), offsetof(sq_rtn_desc, reserved), offsetof(sq_rtn_desc, seed));\n'
        '  return 0;\n}\n')
    exe = tmp_path / "layout"
    subprocess.run(["gcc", "-std=c99", "-I", os.path.join(ROOT, "include"), str(src), "-o", str(exe)], check=True)
    out = subprocess.run([str(exe)], check=True, capture_output=True, text=True).stdout.split("\n")
    m = [int(v) for v in out[0].split()]
    e = [int(v) for v in out[1].split()]
    assert m == [ctypes.sizeof(sq.MergeDesc), sq.MergeDesc.ws2.offset, sq.MergeDesc.reserved.offset]
    assert e == [ctypes.sizeof(sq.ExpertDesc), sq.ExpertDesc.T.offset, sq.ExpertDesc.ws2.offset,
                 sq.ExpertDesc.reserved.offset]
    r = [int(v) for v in out[2].split()]
    assert r == [ctypes.sizeof(sq.RtnDesc), sq.RtnDesc.ws2_out.offset, sq.RtnDesc.ws2_in.offset,
                 sq.RtnDesc.reserved.offset, sq.RtnDesc.seed.offset]


FAKE = 0x10000            # a 16-byte-aligned address that is never dereferenced
MISALIGNED = 0x10008


def _fwd(lib, fmt=0, T=64, O=256, I=512, X=FAKE, codes=FAKE, scales=FAKE, ws2=1.0, Y=FAKE, dt=0):
    return lib.sq_fwd(fmt, T, O, I, X, codes, scales, ws2, Y, dt, None)


@pytest.mark.parametrize("kw,status", [
    (dict(fmt=2), -4),
    (dict(O=0), -2),
    (dict(O=12), -2),                      # O % 8
    (dict(I=48), -2),                      # MX needs I % 32
    (dict(fmt=1, I=40), -2),               # NV needs I % 16
    (dict(T=-1), -2),
    (dict(I=1 << 31), -2),
    (dict(T=1 << 17, I=1 << 13), -2),      # X would reach 2 GiB
    (dict(dt=7), -1),
    (dict(codes=None), -1),
    (dict(X=None), -1),
    (dict(fmt=1, ws2=0.0), -1),
    (dict(fmt=1, ws2=float("nan")), -1),
    (dict(X=MISALIGNED), -3),
    (dict(Y=MISALIGNED), -3),
    (dict(codes=FAKE + 2), -3),
])
def test_fwd_validation(lib, kw, status):
    assert _fwd(lib, **kw) == status


def test_empty_token_batch_is_a_noop(lib):
    # T = 0: nothing to compute for Y / dX, and nothing is launched
    assert _fwd(lib, T=0, X=None, Y=None) == 0
    assert lib.sq_bwd_dx(0, 0, 256, 512, None, FAKE, FAKE, 1.0, None, 0, None) == 0


def test_dx_and_dscale_validation(lib):
    assert lib.sq_bwd_dx(0, 8, 250, 512, FAKE, FAKE, FAKE, 1.0, FAKE, 0, None) == -2
    assert lib.sq_bwd_dscale(0, 8, 256, 500, FAKE, FAKE, FAKE, FAKE, None, 0, None) == -2
    assert lib.sq_bwd_dscale(0, 8, 256, 512, FAKE, FAKE, FAKE, None, None, 0, None) == -1
    assert lib.sq_bwd_dscale(0, 8, 256, 512, MISALIGNED, FAKE, FAKE, FAKE, None, 0, None) == -3
    assert lib.sq_bwd_dscale(0, 8, 256, 512, FAKE, FAKE, FAKE, FAKE + 2, None, 0, None) == -3
    assert lib.sq_bwd_dscale_workspace(0, 4096, 4096, 4096) == 0


def test_dscale_workspace_for_split_token_sum(lib):
    # a 1024 x 4096 projection gives 64 tiles of 256 x 256: the token sum is
    # split four ways into partial [O, G] planes held in the workspace
    need = lib.sq_bwd_dscale_workspace(0, 4096, 1024, 4096)
    assert need == 4 * 1024 * 128 * 4
    assert lib.sq_bwd_dscale_workspace(1, 4096, 1024, 4096) == 4 * 1024 * 256 * 4
    assert lib.sq_bwd_dscale_workspace(0, 0, 1024, 4096) == 0            # nothing to split
    assert lib.sq_bwd_dscale_workspace(0, 64, 256, 512) == 0             # too few K stages
    assert lib.sq_bwd_dscale_workspace(0, 64, 250, 512) == 0             # invalid shape
    assert lib.sq_bwd_dscale(0, 4096, 1024, 4096, FAKE, FAKE, FAKE, FAKE, None, 0, None) == -5
    assert lib.sq_bwd_dscale(0, 4096, 1024, 4096, FAKE, FAKE, FAKE, FAKE, FAKE, need - 1, None) == -5
    assert lib.sq_bwd_dscale(0, 4096, 1024, 4096, FAKE, FAKE, FAKE, FAKE, FAKE + 4, need, None) == -3


def test_merge_validation(lib):
    from paper_2609_04526_amd import sq
    assert lib.sq_merge_scales(0, 0, None, None, None, 1.0, 0, None) == 0          # empty plane
    assert lib.sq_merge_scales(3, 16, FAKE, FAKE, None, 1.0, 0, None) == -4
    assert lib.sq_merge_scales(0, -1, FAKE, FAKE, None, 1.0, 0, None) == -2
    assert lib.sq_merge_scales(0, 16, FAKE, None, None, 1.0, 0, None) == -1         # delta missing
    assert lib.sq_merge_scales(0, 16, FAKE, None, None, 1.0, 1, None) == -1         # src missing
    assert lib.sq_merge_scales(0, 16, FAKE, FAKE, None, 1.0, 2, None) == -1         # bad mode
    assert lib.sq_merge_scales(1, 16, FAKE, FAKE, None, -1.0, 0, None) == -1        # NV ws2
    assert lib.sq_merge_scales(0, 16, FAKE + 1, FAKE, None, 1.0, 0, None) == -3
    assert lib.sq_merge_scales(0, 16, FAKE, MISALIGNED, None, 1.0, 0, None) == -3
    # grouped: one bad descriptor rejects the whole call before anything runs
    arr = (sq.MergeDesc * 2)()
    arr[0] = sq.MergeDesc(16, FAKE, FAKE, 0, 1.0, 0, 0, 0)
    arr[1] = sq.MergeDesc(16, FAKE, 0, 0, 1.0, 0, 0, 0)
    assert lib.sq_merge_scales_grouped(2, arr, None) == -1
    arr[1] = sq.MergeDesc(16, FAKE, FAKE, 0, 1.0, 0, 0, 5)
    assert lib.sq_merge_scales_grouped(2, arr, None) == -1                           # reserved != 0
    assert lib.sq_merge_scales_grouped(-1, arr, None) == -1
    assert lib.sq_merge_scales_grouped(0, None, None) == 0


def test_rtn_validation(lib):
    assert lib.rtn_quantize(0, 256, 500, FAKE, 0.0, 0, FAKE, FAKE, None, None) == -2
    assert lib.rtn_quantize(0, 256, 512, FAKE, 0.0, 3, FAKE, FAKE, None, None) == -1
    assert lib.rtn_quantize(1, 256, 512, FAKE, 0.0, 0, FAKE, FAKE, None, None) == -1   # NV recompute needs ws2_out
    assert lib.rtn_quantize(1, 256, 512, FAKE, float("inf"), 0, FAKE, FAKE, None, None) == -1
    assert lib.rtn_quantize(0, 256, 512, MISALIGNED, 0.0, 0, FAKE, FAKE, None, None) == -3
    assert lib.rtn_quantize(0, 256, 512, None, 0.0, 0, FAKE, FAKE, None, None) == -1


def test_qast_batched_validation(lib):
    ws2 = (ctypes.c_float * 3)(1.0, 0.5, 0.0)
    assert lib.sq_qast_scales_batched(0, 0, 64, 16, 8, FAKE, FAKE, FAKE, 1.0, None, FAKE, None, None) == -2
    assert lib.sq_qast_scales_batched(0, 65536, 8, 8, 8, FAKE, FAKE, FAKE, 1.0, None, FAKE, None, None) == -2
    assert lib.sq_qast_scales_batched(0, 4096, 4096, 256, 8, FAKE, FAKE, FAKE, 1.0, None, FAKE, None, None) == -2
    assert lib.sq_qast_scales_batched(1, 3, 64, 16, 8, FAKE, FAKE, FAKE, 1.0, None, FAKE, None, None) == -1
    assert lib.sq_qast_scales_batched(1, 3, 64, 16, 8, FAKE, FAKE, FAKE, 1.0, ctypes.cast(ws2, ctypes.c_void_p),
                                      FAKE, None, None) == -1              # expert 2's ws2 is 0
    assert lib.sq_qast_factor_grads_batched_workspace(3, 64, 16, 8) == 3 * 2 * 8 * 16 * 4
    assert lib.sq_qast_factor_grads_batched_workspace(0, 64, 16, 8) == 0
    assert lib.sq_qast_factor_grads_batched(3, 64, 16, 8, FAKE, None, FAKE, FAKE, 1.0, FAKE, FAKE, FAKE, 10,
                                            None) == -5


def test_grouped_validation(lib):
    from paper_2609_04526_amd import sq

    def table(*rows):
        arr = (sq.ExpertDesc * len(rows))()
        for d, (act, act2, codes, scales, out, T, ws2, res) in zip(arr, rows):
            d.act, d.act2, d.codes, d.scales, d.out = act, act2, codes, scales, out
            d.T, d.ws2, d.reserved = T, ws2, res
        return arr

    ok = (FAKE, FAKE, FAKE, FAKE, FAKE, 64, 1.0, 0)
    empty = (None, None, FAKE, FAKE, None, 0, 1.0, 0)
    assert lib.sq_fwd_grouped(0, 256, 512, 0, None, 0, None) == 0            # nothing to do
    assert lib.sq_fwd_grouped(0, 256, 512, 2, table(empty, empty), 0, None) == 0
    assert lib.sq_fwd_grouped(0, 256, 512, -1, None, 0, None) == -1
    assert lib.sq_fwd_grouped(0, 256, 512, 1, None, 0, None) == -1
    assert lib.sq_fwd_grouped(2, 256, 512, 1, table(ok), 0, None) == -4
    assert lib.sq_fwd_grouped(0, 256, 500, 1, table(ok), 0, None) == -2
    assert lib.sq_fwd_grouped(0, 256, 512, 1, table(ok), 5, None) == -1
    assert lib.sq_fwd_grouped(0, 256, 512, 2, table(ok, ok[:7] + (1,)), 0, None) == -1      # reserved
    assert lib.sq_fwd_grouped(0, 256, 512, 1, table(ok[:5] + (-1,) + ok[6:]), 0, None) == -2
    assert lib.sq_fwd_grouped(0, 256, 512, 1, table((None,) + ok[1:]), 0, None) == -1
    assert lib.sq_fwd_grouped(0, 256, 512, 1, table((MISALIGNED,) + ok[1:]), 0, None) == -3
    assert lib.sq_fwd_grouped(1, 256, 512, 1, table(ok[:6] + (0.0, 0)), 0, None) == -1     # NVFP4 ws2
    assert lib.sq_bwd_dx_grouped(0, 256, 512, 1, table(ok[:3] + (None,) + ok[4:]), 0, None) == -1
    # dS is written even for an expert without tokens, so its output is required
    assert lib.sq_bwd_dscale_grouped(0, 256, 512, 1, table(empty[:4] + (None,) + empty[5:]), None) == -1
    assert lib.sq_bwd_dscale_grouped(0, 256, 512, 1, table((FAKE, None) + ok[2:]), None) == -1
    assert lib.sq_bwd_dscale_grouped(0, 256, 512, 1, table(ok[:4] + (FAKE + 2,) + ok[5:]), None) == -3


def test_rtn_rule_validation(lib):
    assert lib.rtn_quantize_rule(0, 256, 500, FAKE, 0.0, 2, 0, FAKE, FAKE, None, None) == -2
    assert lib.rtn_quantize_rule(0, 256, 512, FAKE, 0.0, 5, 0, FAKE, FAKE, None, None) == -1
    assert lib.rtn_quantize_rule(0, 256, 512, FAKE, 0.0, -1, 0, FAKE, FAKE, None, None) == -1
    # the whole-tensor rule needs the amax slot in both formats
    assert lib.rtn_quantize_rule(0, 256, 512, FAKE, 0.0, 4, 0, FAKE, FAKE, None, None) == -1
    assert lib.rtn_quantize_rule(1, 256, 512, FAKE, 0.5, 4, 0, FAKE, FAKE, None, None) == -1
    assert lib.rtn_quantize_rule(1, 256, 512, FAKE, 0.0, 3, 7, FAKE, FAKE, None, None) == -1
    assert lib.rtn_quantize_rule(0, 256, 512, FAKE, 0.0, 4, 0, FAKE, FAKE, MISALIGNED + 2, None) == -3
    assert lib.rtn_quantize_rule(0, 256, 512, MISALIGNED, 0.0, 2, 0, FAKE, FAKE, None, None) == -3
    assert lib.rtn_quantize_rule(0, 256, 512, FAKE, 0.0, 2, 0, FAKE, None, None, None) == -1


def test_rtn_grouped_validation(lib):
    from paper_2609_04526_amd import sq

    def table(*rows):
        arr = (sq.RtnDesc * len(rows))()
        for k, r in enumerate(rows):
            arr[k] = sq.RtnDesc(*r)
        return arr

    ok = (256, 512, FAKE, FAKE, FAKE, FAKE + 256, 0.0, 0, 0)
    assert lib.rtn_quantize_grouped(0, 0, 0, None, None) == 0                    # nothing to do
    assert lib.rtn_quantize_grouped(2, 0, 1, table(ok), None) == -4
    assert lib.rtn_quantize_grouped(0, 5, 1, table(ok), None) == -1
    assert lib.rtn_quantize_grouped(0, 0, -1, table(ok), None) == -1
    assert lib.rtn_quantize_grouped(0, 0, 1, None, None) == -1
    assert lib.rtn_quantize_grouped(0, 0, 2, table(ok, (256, 500) + ok[2:]), None) == -2
    assert lib.rtn_quantize_grouped(0, 0, 1, table(ok[:7] + (1, 0)), None) == -1     # reserved
    assert lib.rtn_quantize_grouped(0, 0, 1, table(ok[:2] + (MISALIGNED,) + ok[3:]), None) == -3
    assert lib.rtn_quantize_grouped(0, 0, 1, table(ok[:3] + (FAKE + 2,) + ok[4:]), None) == -3
    assert lib.rtn_quantize_grouped(0, 0, 1, table(ok[:4] + (None,) + ok[5:]), None) == -1
    # an amax slot is required (whole tensor; NVFP4 recompute), aligned and not shared
    assert lib.rtn_quantize_grouped(0, 4, 1, table(ok[:5] + (None,) + ok[6:]), None) == -1
    assert lib.rtn_quantize_grouped(1, 0, 1, table(ok[:5] + (None,) + ok[6:]), None) == -1
    assert lib.rtn_quantize_grouped(1, 0, 1, table(ok[:5] + (FAKE + 2,) + ok[6:]), None) == -3
    assert lib.rtn_quantize_grouped(1, 0, 2, table(ok, ok), None) == -1
    assert lib.rtn_quantize_grouped(1, 0, 1, table(ok[:6] + (float("inf"),) + ok[7:]), None) == -1


def test_qat_validation(lib):
    assert lib.sq_qat_requant(2, 256, 512, 32, FAKE, FAKE, 1.0, FAKE, FAKE, 0.5, FAKE, FAKE, None) == -4
    assert lib.sq_qat_requant(0, 256, 500, 32, FAKE, FAKE, 1.0, FAKE, FAKE, 0.5, FAKE, FAKE, None) == -2
    assert lib.sq_qat_requant(0, 256, 512, 0, FAKE, FAKE, 1.0, FAKE, FAKE, 0.5, FAKE, FAKE, None) == -2
    assert lib.sq_qat_requant(0, 256, 512, 65, FAKE, FAKE, 1.0, FAKE, FAKE, 0.5, FAKE, FAKE, None) == -2
    assert lib.sq_qat_requant(0, 65535 * 16 + 8, 512, 8, FAKE, FAKE, 1.0, FAKE, FAKE, 0.5, FAKE, FAKE, None) == -2
    assert lib.sq_qat_requant(0, 256, 512, 32, None, FAKE, 1.0, FAKE, FAKE, 0.5, FAKE, FAKE, None) == -1
    assert lib.sq_qat_requant(0, 256, 512, 32, FAKE, FAKE, 1.0, FAKE, FAKE, float("nan"), FAKE, FAKE, None) == -1
    assert lib.sq_qat_requant(1, 256, 512, 32, FAKE, FAKE, 0.0, FAKE, FAKE, 0.5, FAKE, FAKE, None) == -1
    assert lib.sq_qat_requant(0, 256, 512, 32, FAKE, FAKE, 1.0, FAKE, MISALIGNED, 0.5, FAKE, FAKE, None) == -3
    assert lib.sq_qat_requant(0, 256, 512, 32, FAKE + 1, FAKE, 1.0, FAKE, FAKE, 0.5, FAKE, FAKE, None) == -3
    # workspace: P^T and Q^T as bf16 hi/lo [2, RW, Tp] (Tp = T rounded up to 64), B^T [RW, O] bf16,
    # partial sums [splits, N, RW] fp32 for each product (64-token stages, about 256 workgroups each),
    # then the projections' partial sums over 1024-wide K-chunks [chunks, Tp, RW] fp32
    assert lib.sq_lora_grads_workspace(256, 128, 512, 32) == \
        2 * (2 * 32 * 256 * 2) + 32 * 128 * 2 + 4 * 512 * 32 * 4 + 4 * 128 * 32 * 4 + 2 * 256 * 32 * 4
    assert lib.sq_lora_grads_workspace(0, 128, 512, 32) == 0
    assert lib.sq_lora_grads_workspace(256, 128, 512, 65) == 0
    assert lib.sq_lora_grads_workspace(256, 124, 512, 8) == 0
    need = lib.sq_lora_grads_workspace(256, 128, 512, 33)
    assert need == 2 * (2 * 64 * 256 * 2) + 64 * 128 * 2 + 4 * 512 * 64 * 4 + 4 * 128 * 64 * 4 + 2 * 256 * 64 * 4
    # 4096 tokens over a 4096-wide product: 16 column tiles -> 16 splits of 256 tokens
    assert lib.sq_lora_grads_workspace(4096, 4096, 4096, 32) == \
        2 * (2 * 32 * 4096 * 2) + 32 * 4096 * 2 + 2 * 16 * 4096 * 32 * 4 + 2 * 4 * 4096 * 32 * 4
    args = (256, 128, 512, 32, FAKE, FAKE, FAKE, FAKE, 0.5, FAKE, FAKE)
    assert lib.sq_lora_grads(*args, FAKE, 10, None) == -5
    assert lib.sq_lora_grads(*args, None, 1 << 30, None) == -5
    assert lib.sq_lora_grads(*args, MISALIGNED + 4, 1 << 30, None) == -3
    assert lib.sq_lora_grads(256, 128, 512, 32, MISALIGNED, FAKE, FAKE, FAKE, 0.5, FAKE, FAKE, FAKE, 1 << 30,
                             None) == -3
    assert lib.sq_lora_grads(256, 128, 512, 32, None, FAKE, FAKE, FAKE, 0.5, FAKE, FAKE, FAKE, 1 << 30, None) == -1
    assert lib.sq_lora_grads(256, 128, 512, 32, FAKE, FAKE, FAKE, FAKE, float("inf"), FAKE, FAKE, FAKE, 1 << 30,
                             None) == -1
    assert lib.sq_lora_grads(-1, 128, 512, 32, FAKE, FAKE, FAKE, FAKE, 0.5, FAKE, FAKE, FAKE, 1 << 30, None) == -2
    assert lib.sq_lora_grads(65535 * 128 + 1, 128, 512, 32, FAKE, FAKE, FAKE, FAKE, 0.5, FAKE, FAKE, FAKE,
                             1 << 30, None) == -2


def test_qast_validation(lib):
    nan = float("nan")
    q = lib.sq_qast_scales
    assert q(3, 8, 4, 2, FAKE, FAKE, FAKE, 1.0, 1.0, FAKE, None, None) == -4        # format
    assert q(0, 0, 4, 2, FAKE, FAKE, FAKE, 1.0, 1.0, FAKE, None, None) == -2        # O = 0
    assert q(0, 8, 4, 0, FAKE, FAKE, FAKE, 1.0, 1.0, FAKE, None, None) == -2        # rank 0
    assert q(0, 8, 4, 65, FAKE, FAKE, FAKE, 1.0, 1.0, FAKE, None, None) == -2       # rank above 64
    assert q(0, 1 << 20, 1 << 12, 2, FAKE, FAKE, FAKE, 1.0, 1.0, FAKE, None, None) == -2   # O*G >= 2^31
    assert q(0, 8, 4, 2, None, FAKE, FAKE, 1.0, 1.0, FAKE, None, None) == -1
    assert q(0, 8, 4, 2, FAKE, FAKE, FAKE, nan, 1.0, FAKE, None, None) == -1        # alpha/r
    assert q(1, 8, 4, 2, FAKE, FAKE, FAKE, 1.0, 0.0, FAKE, None, None) == -1        # NV ws2
    assert q(0, 8, 4, 2, FAKE, FAKE + 1, FAKE, 1.0, 1.0, FAKE, None, None) == -3    # bf16 B
    assert lib.sq_qast_factor_grads_workspace(32, 128, 32) == 1 * 32 * 128 * 4
    assert lib.sq_qast_factor_grads_workspace(33, 128, 32) == 2 * 32 * 128 * 4
    assert lib.sq_qast_factor_grads_workspace(64, 128, 0) == 0
    need = lib.sq_qast_factor_grads_workspace(8, 4, 2)
    g = lib.sq_qast_factor_grads
    assert g(8, 4, 2, FAKE, None, FAKE, FAKE, 1.0, FAKE, FAKE, None, 0, None) == -5            # no workspace
    assert g(8, 4, 2, FAKE, None, FAKE, FAKE, 1.0, FAKE, FAKE, FAKE, need - 1, None) == -5
    assert g(8, 4, 2, FAKE + 2, None, FAKE, FAKE, 1.0, FAKE, FAKE, FAKE, need, None) == -3     # dS
    assert g(8, 4, 2, FAKE, None, FAKE, FAKE, 1.0, None, FAKE, FAKE, need, None) == -1         # dB
    assert g(8, 4, 65, FAKE, None, FAKE, FAKE, 1.0, FAKE, FAKE, FAKE, need, None) == -2


def test_rollback_and_audit_validation(lib):
    assert lib.sq_scale_applied_delta(2, 16, FAKE, FAKE, FAKE, None) == -4
    assert lib.sq_scale_applied_delta(0, -1, FAKE, FAKE, FAKE, None) == -2
    assert lib.sq_scale_applied_delta(0, 0, None, None, None, None) == 0          # empty plane
    assert lib.sq_scale_applied_delta(0, 16, FAKE, None, FAKE, None) == -1
    assert lib.sq_scale_applied_delta(1, 16, FAKE, FAKE, FAKE + 4, None) == -3
    assert lib.sq_scale_rollback(0, 16, FAKE + 1, FAKE, None) == -3
    assert lib.sq_scale_rollback(0, 16, FAKE, None, None) == -1
    assert lib.sq_byte_diff(16, FAKE, FAKE, None, None) == -1
    assert lib.sq_byte_diff(16, FAKE, FAKE + 8, FAKE, None) == -3
    assert lib.sq_byte_diff(16, FAKE, FAKE, FAKE + 4, None) == -3
    assert lib.sq_byte_diff(0, None, None, FAKE, None) == 0


# ---------------------------------------------------------------- binding checks
# The C ABI sees bare pointers, so the Python binding checks dtype, contiguity
# and shape agreement before any call.  These run on CPU tensors: the checks
# come before the device check, and nothing reaches the library.
def _layer_cpu(T=8, O=16, I=64, fmt="mx"):
    import torch
    B = 32 if fmt == "mx" else 16
    X = torch.zeros((T, I), dtype=torch.bfloat16)
    dY = torch.zeros((T, O), dtype=torch.bfloat16)
    codes = torch.zeros((O, I // 2), dtype=torch.uint8)
    scales = torch.zeros((O, I // B), dtype=torch.uint8)
    return X, dY, codes, scales


def _cases():
    import torch
    from paper_2609_04526_amd import sq
    X, dY, codes, scales = _layer_cpu()
    return [
        ("fwd: X fp32", lambda: sq.sq_fwd("mx", X.float(), codes, scales)),
        ("fwd: X transposed view", lambda: sq.sq_fwd("mx", torch.zeros((64, 8), dtype=torch.bfloat16).t(),
                                                       codes, scales)),
        ("fwd: Y int32", lambda: sq.sq_fwd("mx", X, codes, scales, Y=torch.zeros((8, 16), dtype=torch.int32))),
        ("fwd: Y too small", lambda: sq.sq_fwd("mx", X, codes, scales, Y=torch.zeros((8, 8)))),
        ("fwd: scales too few blocks", lambda: sq.sq_fwd("mx", X, codes, scales[:, :1].contiguous())),
        ("fwd: codes for another I", lambda: sq.sq_fwd("mx", X, codes[:, :16].contiguous(), scales)),
        ("fwd: I not a multiple of the block", lambda: sq.sq_fwd("mx", X[:, :48].contiguous(),
                                                                   codes[:, :24].contiguous(), scales)),
        ("dx: dY fp16", lambda: sq.sq_bwd_dx("mx", dY.half(), codes, scales)),
        ("dx: dX wrong shape", lambda: sq.sq_bwd_dx("mx", dY, codes, scales, dX=torch.zeros((8, 32)))),
        ("dx: codes rows != dY columns", lambda: sq.sq_bwd_dx("mx", dY[:, :8].contiguous(), codes, scales)),
        ("ds: codes rows != dY columns", lambda: sq.sq_bwd_dscale("mx", X, dY[:, :8].contiguous(), codes)),
        ("ds: dY rows != X rows", lambda: sq.sq_bwd_dscale("mx", X, dY[:4].contiguous(), codes)),
        ("ds: dS bf16", lambda: sq.sq_bwd_dscale("mx", X, dY, codes,
                                                 dS=torch.zeros((16, 2), dtype=torch.bfloat16))),
        ("ds: dS too small", lambda: sq.sq_bwd_dscale("mx", X, dY, codes, dS=torch.zeros((16, 1)))),
        ("merge: delta shorter", lambda: sq.sq_merge_scales("mx", scales.reshape(-1),
                                                            delta=torch.zeros(scales.numel() - 1))),
        ("merge: delta fp64", lambda: sq.sq_merge_scales("mx", scales.reshape(-1),
                                                         delta=torch.zeros(scales.numel(), dtype=torch.float64))),
        ("swap: src shorter", lambda: sq.sq_merge_scales("mx", scales.reshape(-1),
                                                         src=torch.zeros(3, dtype=torch.uint8))),
        ("rtn: W fp32", lambda: sq.rtn_quantize("mx", torch.zeros((16, 64)))),
        ("rtn: codes_out too small", lambda: sq.rtn_quantize("mx", torch.zeros((16, 64), dtype=torch.bfloat16),
                                                             codes=torch.zeros((16, 16), dtype=torch.uint8))),
        ("grouped fwd: outputs per expert", lambda: sq.sq_fwd_grouped("mx", [X, X], [codes, codes],
                                                                      [scales, scales], Ys=[torch.zeros((8, 16))])),
        ("grouped ds: dS wrong shape", lambda: sq.sq_bwd_dscale_grouped("mx", [X], [dY], [codes],
                                                                        dSs=[torch.zeros((16, 4))])),
        ("qat: A wrong shape", lambda: sq.sq_qat_requant("mx", codes, scales,
                                                         torch.zeros((16, 4), dtype=torch.bfloat16),
                                                         torch.zeros((4, 32), dtype=torch.bfloat16), 1.0)),
        ("lora: dY rows != X rows", lambda: sq.sq_lora_grads(X, dY[:4].contiguous(),
                                                             torch.zeros((16, 4), dtype=torch.bfloat16),
                                                             torch.zeros((4, 64), dtype=torch.bfloat16), 1.0)),
        ("qast: A wrong shape", lambda: sq.sq_qast_scales("mx", scales, torch.zeros((16, 4), dtype=torch.bfloat16),
                                                          torch.zeros((4, 3), dtype=torch.bfloat16), 1.0)),
        ("qast grads: mask wrong shape", lambda: sq.sq_qast_factor_grads(
            torch.zeros((16, 2)), torch.zeros((16, 3), dtype=torch.uint8),
            torch.zeros((16, 4), dtype=torch.bfloat16), torch.zeros((4, 2), dtype=torch.bfloat16), 1.0)),
        ("rollback: applied shorter", lambda: sq.sq_scale_rollback("mx", scales.reshape(-1), torch.zeros(3))),
        ("byte diff: b shorter", lambda: sq.sq_byte_diff(scales.reshape(-1), torch.zeros(3, dtype=torch.uint8))),
    ]


@pytest.mark.parametrize("k", range(27))
def test_binding_rejects_bad_tensors(k):
    cases = _cases()
    assert len(cases) == 27
    name, call = cases[k]
    with pytest.raises(ValueError):
        call()


def test_binding_rejects_host_tensors_that_pass_the_checks():
    from paper_2609_04526_amd import sq
    X, dY, codes, scales = _layer_cpu()
    with pytest.raises(ValueError, match="device tensors"):
        sq.sq_fwd("mx", X, codes, scales)
