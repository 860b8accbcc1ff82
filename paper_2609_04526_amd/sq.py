"""ctypes binding of libscaleqlora (C ABI in include/scaleqlora.h).

Argument marshalling only: each function takes torch tensors that already live
on the current HIP device, passes their data pointers, sizes and the current
torch stream to the entry point of the same name, and raises on a non-zero
status.  All compute happens in the library's HIP kernels.  The library must
have been built (``python -m paper_2609_04526_amd.build``); there is no
fallback path.
"""

import ctypes
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libscaleqlora.so")

MXFP4, NVFP4 = 0, 1
OUT_F32, OUT_BF16 = 0, 1
TIE_EVEN, TIE_AWAY = 0, 1
MERGE_DELTA, MERGE_COPY = 0, 1
FORMATS = {"mx": MXFP4, "nv": NVFP4}
RULE_NEAREST_EVEN, RULE_NEAREST_AWAY, RULE_RTZ, RULE_STOCHASTIC, RULE_WHOLE_TENSOR = 0, 1, 2, 3, 4
RULES = {"even": RULE_NEAREST_EVEN, "away": RULE_NEAREST_AWAY, "rtz": RULE_RTZ,
         "stochastic": RULE_STOCHASTIC, "whole_tensor": RULE_WHOLE_TENSOR}
BLOCK = {MXFP4: 32, NVFP4: 16}

_c_i64 = ctypes.c_int64
_c_p = ctypes.c_void_p


class SqError(RuntimeError):
    def __init__(self, fn, status, msg):
        super().__init__(f"{fn} failed with status {status}: {msg}")
        self.status = status


class MergeDesc(ctypes.Structure):
    """Mirror of sq_merge_desc."""
    _fields_ = [
        ("n", ctypes.c_int64),
        ("scales", ctypes.c_void_p),
        ("delta", ctypes.c_void_p),
        ("src", ctypes.c_void_p),
        ("ws2", ctypes.c_float),
        ("fmt", ctypes.c_int32),
        ("mode", ctypes.c_int32),
        ("reserved", ctypes.c_int32),
    ]


class ExpertDesc(ctypes.Structure):
    """Mirror of sq_expert_desc."""
    _fields_ = [
        ("act", ctypes.c_void_p),
        ("act2", ctypes.c_void_p),
        ("codes", ctypes.c_void_p),
        ("scales", ctypes.c_void_p),
        ("out", ctypes.c_void_p),
        ("T", ctypes.c_int64),
        ("ws2", ctypes.c_float),
        ("reserved", ctypes.c_int32),
    ]


class RtnDesc(ctypes.Structure):
    """Mirror of sq_rtn_desc."""
    _fields_ = [
        ("O", ctypes.c_int64),
        ("I", ctypes.c_int64),
        ("W", ctypes.c_void_p),
        ("codes_out", ctypes.c_void_p),
        ("scales_out", ctypes.c_void_p),
        ("ws2_out", ctypes.c_void_p),
        ("ws2_in", ctypes.c_float),
        ("reserved", ctypes.c_int32),
        ("seed", ctypes.c_uint64),
    ]


_lib = None


def load():
    """Load the library (once).  Raises if it was not built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is missing: run `python -m paper_2609_04526_amd.build` first")
    lib = ctypes.CDLL(LIB_PATH)
    sigs = {
        "sq_fwd": (ctypes.c_int, [ctypes.c_int, _c_i64, _c_i64, _c_i64, _c_p, _c_p, _c_p, ctypes.c_float,
                                  _c_p, ctypes.c_int, _c_p]),
        "sq_bwd_dx": (ctypes.c_int, [ctypes.c_int, _c_i64, _c_i64, _c_i64, _c_p, _c_p, _c_p, ctypes.c_float,
                                     _c_p, ctypes.c_int, _c_p]),
        "sq_bwd_dscale": (ctypes.c_int, [ctypes.c_int, _c_i64, _c_i64, _c_i64, _c_p, _c_p, _c_p, _c_p,
                                         _c_p, ctypes.c_size_t, _c_p]),
        "sq_bwd_dscale_workspace": (ctypes.c_size_t, [ctypes.c_int, _c_i64, _c_i64, _c_i64]),
        "sq_merge_scales": (ctypes.c_int, [ctypes.c_int, _c_i64, _c_p, _c_p, _c_p, ctypes.c_float,
                                           ctypes.c_int, _c_p]),
        "sq_merge_scales_grouped": (ctypes.c_int, [ctypes.c_int, ctypes.POINTER(MergeDesc), _c_p]),
        "sq_fwd_grouped": (ctypes.c_int, [ctypes.c_int, _c_i64, _c_i64, ctypes.c_int, ctypes.POINTER(ExpertDesc),
                                          ctypes.c_int, _c_p]),
        "sq_bwd_dx_grouped": (ctypes.c_int, [ctypes.c_int, _c_i64, _c_i64, ctypes.c_int,
                                             ctypes.POINTER(ExpertDesc), ctypes.c_int, _c_p]),
        "sq_bwd_dscale_grouped": (ctypes.c_int, [ctypes.c_int, _c_i64, _c_i64, ctypes.c_int,
                                                 ctypes.POINTER(ExpertDesc), _c_p]),
        "rtn_quantize": (ctypes.c_int, [ctypes.c_int, _c_i64, _c_i64, _c_p, ctypes.c_float, ctypes.c_int,
                                        _c_p, _c_p, _c_p, _c_p]),
        "rtn_quantize_rule": (ctypes.c_int, [ctypes.c_int, _c_i64, _c_i64, _c_p, ctypes.c_float, ctypes.c_int,
                                             ctypes.c_uint64, _c_p, _c_p, _c_p, _c_p]),
        "rtn_quantize_grouped": (ctypes.c_int, [ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.POINTER(RtnDesc),
                                                _c_p]),
        "sq_qat_requant": (ctypes.c_int, [ctypes.c_int, _c_i64, _c_i64, ctypes.c_int, _c_p, _c_p, ctypes.c_float,
                                          _c_p, _c_p, ctypes.c_float, _c_p, _c_p, _c_p]),
        "sq_lora_grads_workspace": (ctypes.c_size_t, [_c_i64, _c_i64, _c_i64, ctypes.c_int]),
        "sq_lora_grads": (ctypes.c_int, [_c_i64, _c_i64, _c_i64, ctypes.c_int, _c_p, _c_p, _c_p, _c_p,
                                         ctypes.c_float, _c_p, _c_p, _c_p, ctypes.c_size_t, _c_p]),
        "sq_qast_scales": (ctypes.c_int, [ctypes.c_int, _c_i64, _c_i64, ctypes.c_int, _c_p, _c_p, _c_p,
                                          ctypes.c_float, ctypes.c_float, _c_p, _c_p, _c_p]),
        "sq_qast_factor_grads_workspace": (ctypes.c_size_t, [_c_i64, _c_i64, ctypes.c_int]),
        "sq_qast_scales_batched": (ctypes.c_int, [ctypes.c_int, _c_i64, _c_i64, _c_i64, ctypes.c_int, _c_p, _c_p,
                                                  _c_p, ctypes.c_float, _c_p, _c_p, _c_p, _c_p]),
        "sq_qast_factor_grads_batched_workspace": (ctypes.c_size_t, [_c_i64, _c_i64, _c_i64, ctypes.c_int]),
        "sq_qast_factor_grads_batched": (ctypes.c_int, [_c_i64, _c_i64, _c_i64, ctypes.c_int, _c_p, _c_p, _c_p,
                                                        _c_p, ctypes.c_float, _c_p, _c_p, _c_p, ctypes.c_size_t,
                                                        _c_p]),
        "sq_qast_factor_grads": (ctypes.c_int, [_c_i64, _c_i64, ctypes.c_int, _c_p, _c_p, _c_p, _c_p,
                                                ctypes.c_float, _c_p, _c_p, _c_p, ctypes.c_size_t, _c_p]),
        "sq_scale_applied_delta": (ctypes.c_int, [ctypes.c_int, _c_i64, _c_p, _c_p, _c_p, _c_p]),
        "sq_scale_rollback": (ctypes.c_int, [ctypes.c_int, _c_i64, _c_p, _c_p, _c_p]),
        "sq_byte_diff": (ctypes.c_int, [_c_i64, _c_p, _c_p, _c_p, _c_p]),
        "sq_status_str": (ctypes.c_char_p, [ctypes.c_int]),
        "sq_abi_version": (ctypes.c_int, []),
    }
    for name, (res, args) in sigs.items():
        f = getattr(lib, name)
        f.restype = res
        f.argtypes = args
    _lib = lib
    return lib


def _check(fn, status):
    if status != 0:
        raise SqError(fn, status, load().sq_status_str(status).decode())


def _stream():
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def _ptr(t):
    return ctypes.c_void_p(t.data_ptr()) if t is not None else ctypes.c_void_p(0)


def _fmt(fmt):
    return FORMATS.get(fmt, fmt)


def _dev(*ts):
    for t in ts:
        if t is not None and not t.is_cuda:
            raise ValueError("libscaleqlora takes device tensors")


# ---------------------------------------------------------------- entry points
def sq_fwd(fmt, X, codes, scales, ws2=1.0, out_dtype=torch.float32, Y=None):
    """Y = X W^T.  X bf16 [T, I], codes uint8 [O, I/2], scales uint8 [O, G]."""
    fmt = _fmt(fmt)
    T, I = X.shape
    O = codes.shape[0]
    if Y is None:
        Y = torch.empty((T, O), dtype=out_dtype, device=X.device)
    _dev(X, codes, scales, Y)
    _check("sq_fwd", load().sq_fwd(fmt, T, O, I, _ptr(X), _ptr(codes), _ptr(scales), float(ws2), _ptr(Y),
                                   OUT_BF16 if Y.dtype == torch.bfloat16 else OUT_F32, _stream()))
    return Y


def sq_bwd_dx(fmt, dY, codes, scales, ws2=1.0, out_dtype=torch.float32, dX=None):
    """dX = dY W.  dY bf16 [T, O] -> dX [T, I]."""
    fmt = _fmt(fmt)
    T, O = dY.shape
    I = codes.shape[1] * 2
    if dX is None:
        dX = torch.empty((T, I), dtype=out_dtype, device=dY.device)
    _dev(dY, codes, scales, dX)
    _check("sq_bwd_dx", load().sq_bwd_dx(fmt, T, O, I, _ptr(dY), _ptr(codes), _ptr(scales), float(ws2),
                                         _ptr(dX), OUT_BF16 if dX.dtype == torch.bfloat16 else OUT_F32,
                                         _stream()))
    return dX


def sq_bwd_dscale_workspace(fmt, T, O, I):
    return int(load().sq_bwd_dscale_workspace(_fmt(fmt), T, O, I))


def sq_bwd_dscale(fmt, X, dY, codes, dS=None, workspace=None):
    """dS[o,b] = sum_{j in b} code[o,j] (dY^T X)[o,j], fp32 [O, G]."""
    fmt = _fmt(fmt)
    T, I = X.shape
    O = dY.shape[1]
    if dS is None:
        dS = torch.empty((O, I // BLOCK[fmt]), dtype=torch.float32, device=X.device)
    _dev(X, dY, codes, dS)
    ws_bytes = sq_bwd_dscale_workspace(fmt, T, O, I)
    if ws_bytes and workspace is None:
        workspace = torch.empty(ws_bytes, dtype=torch.uint8, device=X.device)
    wsz = workspace.numel() * workspace.element_size() if workspace is not None else 0
    _check("sq_bwd_dscale", load().sq_bwd_dscale(fmt, T, O, I, _ptr(X), _ptr(dY), _ptr(codes), _ptr(dS),
                                                 _ptr(workspace), wsz, _stream()))
    return dS


def sq_merge_scales(fmt, scales, delta=None, src=None, ws2=1.0, mode=None):
    """In-place merge (delta given) or swap (src given) of one scale plane."""
    fmt = _fmt(fmt)
    if mode is None:
        mode = MERGE_COPY if src is not None else MERGE_DELTA
    _dev(scales, delta, src)
    _check("sq_merge_scales", load().sq_merge_scales(fmt, scales.numel(), _ptr(scales), _ptr(delta),
                                                     _ptr(src), float(ws2), mode, _stream()))
    return scales


class MergeGroup:
    """A prepared descriptor table for sq_merge_scales_grouped (built once,
    reused across calls; the tensors it names must stay alive)."""

    def __init__(self, planes):
        self.planes = planes
        self.arr = (MergeDesc * max(len(planes), 1))()
        for k, p in enumerate(planes):
            mode = p.get("mode", MERGE_COPY if p.get("src") is not None else MERGE_DELTA)
            _dev(p["scales"], p.get("delta"), p.get("src"))
            self.arr[k] = MergeDesc(p["scales"].numel(), p["scales"].data_ptr(),
                                    p["delta"].data_ptr() if p.get("delta") is not None else 0,
                                    p["src"].data_ptr() if p.get("src") is not None else 0,
                                    float(p.get("ws2", 1.0)), _fmt(p["fmt"]), mode, 0)


def sq_merge_scales_grouped(planes):
    """planes: a MergeGroup, or a list of dicts with keys fmt, scales,
    delta / src, ws2, mode."""
    group = planes if isinstance(planes, MergeGroup) else MergeGroup(planes)
    _check("sq_merge_scales_grouped",
           load().sq_merge_scales_grouped(len(group.planes), group.arr, _stream()))


def _expert_table(acts, acts2, codes, scales, outs, ws2):
    n = len(codes)
    arr = (ExpertDesc * max(n, 1))()
    for e in range(n):
        d = arr[e]
        d.act = acts[e].data_ptr() if acts[e] is not None and acts[e].numel() else None
        d.act2 = acts2[e].data_ptr() if acts2 is not None and acts2[e].numel() else None
        d.codes = codes[e].data_ptr()
        d.scales = scales[e].data_ptr() if scales is not None else None
        d.out = outs[e].data_ptr() if outs[e].numel() else None
        d.T = acts[e].shape[0]
        d.ws2 = float(ws2[e]) if ws2 is not None else 1.0
        d.reserved = 0
    return arr


_DTYPE_CODE = {torch.float32: OUT_F32, torch.bfloat16: OUT_BF16}


class ExpertTable:
    """A prebuilt sq_expert_desc table for repeated grouped calls on the same
    tensors (building the table is host work that a training loop need not
    repeat).  Holds references to every tensor it points at."""

    def __init__(self, kind, fmt, acts, codes, scales=None, outs=None, acts2=None, ws2=None,
                 out_dtype=torch.float32):
        self.kind, self.fmt = kind, _fmt(fmt)
        self.O, self.I = codes[0].shape[0], codes[0].shape[1] * 2
        dev = codes[0].device
        if outs is None:
            if kind == "fwd":
                outs = [torch.empty((x.shape[0], self.O), dtype=out_dtype, device=dev) for x in acts]
            elif kind == "dx":
                outs = [torch.empty((d.shape[0], self.I), dtype=out_dtype, device=dev) for d in acts]
            else:
                outs = [torch.empty((self.O, self.I // BLOCK[self.fmt]), dtype=torch.float32, device=dev)
                        for _ in codes]
        _dev(*acts, *codes, *(scales or []), *outs, *(acts2 or []))
        self.refs = (acts, codes, scales, outs, acts2)
        self.outs = outs
        self.n = len(codes)
        self.arr = _expert_table(acts, acts2, codes, scales, outs, ws2)
        self.dtype = _DTYPE_CODE[outs[0].dtype] if (outs and kind != "ds") else OUT_F32

    def run(self):
        lib = load()
        if self.kind == "fwd":
            st = lib.sq_fwd_grouped(self.fmt, self.O, self.I, self.n, self.arr, self.dtype, _stream())
        elif self.kind == "dx":
            st = lib.sq_bwd_dx_grouped(self.fmt, self.O, self.I, self.n, self.arr, self.dtype, _stream())
        else:
            st = lib.sq_bwd_dscale_grouped(self.fmt, self.O, self.I, self.n, self.arr, _stream())
        _check(f"sq_{self.kind}_grouped", st)
        return self.outs


def sq_fwd_grouped(fmt, Xs, codes, scales, ws2=None, out_dtype=torch.float32, Ys=None):
    """Per-expert Y_e = X_e W_e^T in one grouped launch; Xs[e] bf16 [T_e, I]."""
    return ExpertTable("fwd", fmt, Xs, codes, scales, Ys, None, ws2, out_dtype).run()


def sq_bwd_dx_grouped(fmt, dYs, codes, scales, ws2=None, out_dtype=torch.float32, dXs=None):
    """Per-expert dX_e = dY_e W_e in one grouped launch; dYs[e] bf16 [T_e, O]."""
    return ExpertTable("dx", fmt, dYs, codes, scales, dXs, None, ws2, out_dtype).run()


def sq_bwd_dscale_grouped(fmt, Xs, dYs, codes, dSs=None):
    """Per-expert dS_e (fp32 [O, G]) in one grouped launch."""
    return ExpertTable("ds", fmt, Xs, codes, None, dSs, dYs).run()


def rtn_quantize(fmt, W, tie=TIE_EVEN, ws2_in=0.0, codes=None, scales=None, ws2_out=None):
    """Round-to-nearest re-quantisation of bf16 W [O, I] -> (codes, scales, ws2_out)."""
    fmt = _fmt(fmt)
    O, I = W.shape
    dev = W.device
    if codes is None:
        codes = torch.empty((O, I // 2), dtype=torch.uint8, device=dev)
    if scales is None:
        scales = torch.empty((O, I // BLOCK[fmt]), dtype=torch.uint8, device=dev)
    if fmt == NVFP4 and ws2_out is None:
        ws2_out = torch.empty(1, dtype=torch.float32, device=dev)
    _dev(W, codes, scales, ws2_out)
    _check("rtn_quantize", load().rtn_quantize(fmt, O, I, _ptr(W), float(ws2_in), int(tie), _ptr(codes),
                                               _ptr(scales), _ptr(ws2_out), _stream()))
    return codes, scales, ws2_out


def rtn_quantize_rule(fmt, W, rule, ws2_in=0.0, seed=0, codes=None, scales=None, ws2_out=None):
    """Re-quantisation of bf16 W [O, I] under a deploy rule (RULE_*) -> (codes, scales, ws2_out).
    ws2_out is allocated where the call needs it (NVFP4, or the whole-tensor rule)."""
    fmt = _fmt(fmt)
    rule = RULES.get(rule, rule)
    O, I = W.shape
    dev = W.device
    if codes is None:
        codes = torch.empty((O, I // 2), dtype=torch.uint8, device=dev)
    if scales is None:
        scales = torch.empty((O, I // BLOCK[fmt]), dtype=torch.uint8, device=dev)
    if (fmt == NVFP4 or rule == RULE_WHOLE_TENSOR) and ws2_out is None:
        ws2_out = torch.empty(1, dtype=torch.float32, device=dev)
    _dev(W, codes, scales, ws2_out)
    _check("rtn_quantize_rule", load().rtn_quantize_rule(fmt, O, I, _ptr(W), float(ws2_in), int(rule),
                                                         int(seed) & 0xFFFFFFFFFFFFFFFF, _ptr(codes),
                                                         _ptr(scales), _ptr(ws2_out), _stream()))
    return codes, scales, ws2_out


class RtnGroup:
    """A prepared descriptor table for rtn_quantize_grouped (built once, reused
    across calls; the tensors it names must stay alive).  weights: dicts with
    keys W, codes, scales and optionally ws2_out, ws2_in, seed."""

    def __init__(self, fmt, rule, weights):
        self.fmt = _fmt(fmt)
        self.rule = RULES.get(rule, rule)
        self.weights = weights
        self.arr = (RtnDesc * max(len(weights), 1))()
        for k, w in enumerate(weights):
            O, I = w["W"].shape
            _dev(w["W"], w["codes"], w["scales"], w.get("ws2_out"))
            self.arr[k] = RtnDesc(O, I, w["W"].data_ptr(), w["codes"].data_ptr(), w["scales"].data_ptr(),
                                  w["ws2_out"].data_ptr() if w.get("ws2_out") is not None else 0,
                                  float(w.get("ws2_in", 0.0)), 0, int(w.get("seed", 0)) & 0xFFFFFFFFFFFFFFFF)


def rtn_quantize_grouped(fmt, rule, weights):
    """rtn_quantize_rule over many weights (an RtnGroup, or the list of dicts
    RtnGroup takes) in shared launches; outputs are written in place."""
    group = weights if isinstance(weights, RtnGroup) else RtnGroup(fmt, rule, weights)
    _check("rtn_quantize_grouped", load().rtn_quantize_grouped(group.fmt, group.rule, len(group.weights),
                                                               group.arr, _stream()))


def sq_qat_requant(fmt, codes, scales, B, A, alpha_over_r, ws2=1.0, codes_out=None, scales_out=None):
    """Fake-quantised QAT-LoRA weight quantize(base + alpha_over_r B A) as (codes_out, scales_out).
    codes uint8 [O, I/2], scales uint8 [O, G], B bf16 [O, r], A bf16 [r, I]."""
    fmt = _fmt(fmt)
    O, I = codes.shape[0], codes.shape[1] * 2
    r = B.shape[1]
    if codes_out is None:
        codes_out = torch.empty_like(codes)
    if scales_out is None:
        scales_out = torch.empty_like(scales)
    _dev(codes, scales, B, A, codes_out, scales_out)
    _check("sq_qat_requant", load().sq_qat_requant(fmt, O, I, r, _ptr(codes), _ptr(scales), float(ws2), _ptr(B),
                                                   _ptr(A), float(alpha_over_r), _ptr(codes_out),
                                                   _ptr(scales_out), _stream()))
    return codes_out, scales_out


def sq_lora_grads_workspace(T, O, I, r):
    return int(load().sq_lora_grads_workspace(T, O, I, r))


def sq_lora_grads(X, dY, B, A, alpha_over_r, dB=None, dA=None, workspace=None):
    """STE factor gradients dB [O, r], dA [r, I] (fp32) of W = base + alpha_over_r B A."""
    T, I = X.shape
    O, r = B.shape
    dev = B.device
    if dB is None:
        dB = torch.empty((O, r), dtype=torch.float32, device=dev)
    if dA is None:
        dA = torch.empty((r, I), dtype=torch.float32, device=dev)
    need = sq_lora_grads_workspace(T, O, I, r)
    if workspace is None and need > 0:
        workspace = torch.empty(need, dtype=torch.uint8, device=dev)
    _dev(X, dY, B, A, dB, dA, workspace)
    nbytes = workspace.numel() * workspace.element_size() if workspace is not None else 0
    _check("sq_lora_grads", load().sq_lora_grads(T, O, I, r, _ptr(X), _ptr(dY), _ptr(B), _ptr(A),
                                                 float(alpha_over_r), _ptr(dB), _ptr(dA), _ptr(workspace),
                                                 nbytes, _stream()))
    return dB, dA


def sq_qast_scales(fmt, base_scales, B, A, alpha_over_r, ws2=1.0, scales_out=None, mask_out=None,
                   want_mask=True):
    """On-grid scale bytes of the QAST forward for Delta_S = alpha_over_r * B A, and the
    clamp mask (1 where the gradient passes).  base_scales uint8 [O, G], B bf16 [O, r],
    A bf16 [r, G].  Returns (scales_out, mask_out or None)."""
    fmt = _fmt(fmt)
    O, G = base_scales.shape
    r = B.shape[1]
    if scales_out is None:
        scales_out = torch.empty_like(base_scales)
    if want_mask and mask_out is None:
        mask_out = torch.empty_like(base_scales)
    _dev(base_scales, B, A, scales_out, mask_out)
    _check("sq_qast_scales", load().sq_qast_scales(fmt, O, G, r, _ptr(base_scales), _ptr(B), _ptr(A),
                                                   float(alpha_over_r), float(ws2), _ptr(scales_out),
                                                   _ptr(mask_out), _stream()))
    return scales_out, mask_out


def sq_qast_scales_batched(fmt, base_scales, B, A, alpha_over_r, ws2=None, scales_out=None, mask_out=None,
                           want_mask=True):
    """QAST scale bytes for E stacked experts: base_scales [E, O, G], B [E, O, r],
    A [E, r, G] (bf16); ws2: E per-expert NVFP4 scalars.  Returns (scales_out, mask)."""
    fmt = _fmt(fmt)
    E, O, G = base_scales.shape
    r = B.shape[2]
    if scales_out is None:
        scales_out = torch.empty_like(base_scales)
    if want_mask and mask_out is None:
        mask_out = torch.empty_like(base_scales)
    w = None
    if fmt == NVFP4:
        w = (ctypes.c_float * E)(*[float(v) for v in ws2])
    _dev(base_scales, B, A, scales_out, mask_out)
    _check("sq_qast_scales_batched", load().sq_qast_scales_batched(
        fmt, E, O, G, r, _ptr(base_scales), _ptr(B), _ptr(A), float(alpha_over_r),
        ctypes.cast(w, ctypes.c_void_p) if w is not None else None, _ptr(scales_out), _ptr(mask_out), _stream()))
    return scales_out, mask_out


def sq_qast_factor_grads_batched(dS, mask, B, A, alpha_over_r, dB=None, dA=None, workspace=None):
    """dB [E, O, r], dA [E, r, G] (fp32) for E stacked experts."""
    E, O, G = dS.shape
    r = B.shape[2]
    if dB is None:
        dB = torch.empty((E, O, r), dtype=torch.float32, device=dS.device)
    if dA is None:
        dA = torch.empty((E, r, G), dtype=torch.float32, device=dS.device)
    need = int(load().sq_qast_factor_grads_batched_workspace(E, O, G, r))
    if workspace is None:
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=dS.device)
    _dev(dS, mask, B, A, dB, dA, workspace)
    _check("sq_qast_factor_grads_batched", load().sq_qast_factor_grads_batched(
        E, O, G, r, _ptr(dS), _ptr(mask), _ptr(B), _ptr(A), float(alpha_over_r), _ptr(dB), _ptr(dA),
        _ptr(workspace), workspace.numel(), _stream()))
    return dB, dA


def sq_qast_factor_grads_workspace(O, G, r):
    return int(load().sq_qast_factor_grads_workspace(O, G, r))


def sq_qast_factor_grads(dS, mask, B, A, alpha_over_r, dB=None, dA=None, workspace=None):
    """dB [O, r] and dA [r, G] (fp32) from dS [O, G] through the clamp mask (None: all pass)."""
    O, G = dS.shape
    r = B.shape[1]
    if dB is None:
        dB = torch.empty((O, r), dtype=torch.float32, device=dS.device)
    if dA is None:
        dA = torch.empty((r, G), dtype=torch.float32, device=dS.device)
    need = sq_qast_factor_grads_workspace(O, G, r)
    if workspace is None:
        workspace = torch.empty(max(need, 4), dtype=torch.uint8, device=dS.device)
    _dev(dS, mask, B, A, dB, dA, workspace)
    wsz = workspace.numel() * workspace.element_size()
    _check("sq_qast_factor_grads", load().sq_qast_factor_grads(O, G, r, _ptr(dS), _ptr(mask), _ptr(B), _ptr(A),
                                                               float(alpha_over_r), _ptr(dB), _ptr(dA),
                                                               _ptr(workspace), wsz, _stream()))
    return dB, dA


def sq_scale_applied_delta(fmt, before, after, applied=None):
    """fp32 on-grid delta value(after) - value(before) of two scale planes (same shape)."""
    fmt = _fmt(fmt)
    if applied is None:
        applied = torch.empty(before.shape, dtype=torch.float32, device=before.device)
    _dev(before, after, applied)
    _check("sq_scale_applied_delta", load().sq_scale_applied_delta(fmt, before.numel(), _ptr(before), _ptr(after),
                                                                   _ptr(applied), _stream()))
    return applied


def sq_scale_rollback(fmt, scales, applied):
    """In place: scales := encode(value(scales) - applied)."""
    fmt = _fmt(fmt)
    _dev(scales, applied)
    _check("sq_scale_rollback", load().sq_scale_rollback(fmt, scales.numel(), _ptr(scales), _ptr(applied), _stream()))
    return scales


def sq_byte_diff(a, b, counts=None):
    """Adds (differing bytes, differing nibbles) of two byte planes to a device int64 [2] tensor."""
    if counts is None:
        counts = torch.zeros(2, dtype=torch.int64, device=a.device)
    _dev(a, b, counts)
    _check("sq_byte_diff", load().sq_byte_diff(a.numel(), _ptr(a), _ptr(b), _ptr(counts), _stream()))
    return counts


def abi_version():
    return int(load().sq_abi_version())
