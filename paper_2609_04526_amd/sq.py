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
        "sq_bwd_dscale_noalloc": (ctypes.c_int, [ctypes.c_int, _c_i64, _c_i64, _c_i64, _c_p, _c_p, _c_p, _c_p,
                                                 _c_p]),
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
        "sq_qat_requant_batched": (ctypes.c_int, [ctypes.c_int, _c_i64, _c_i64, _c_i64, ctypes.c_int, _c_p, _c_p,
                                                  _c_p, _c_p, _c_p, ctypes.c_float, _c_p, _c_p, _c_p]),
        "sq_lora_grads_batched_workspace": (ctypes.c_size_t, [_c_i64, _c_p, _c_i64, _c_i64, ctypes.c_int]),
        "sq_lora_grads_batched": (ctypes.c_int, [_c_i64, _c_p, _c_i64, _c_i64, ctypes.c_int, _c_p, _c_p, _c_p, _c_p,
                                                 ctypes.c_float, _c_p, _c_p, _c_p, ctypes.c_size_t, _c_p]),
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
    """Every tensor lives on the current HIP device (the library launches there)."""
    dev = None
    for t in ts:
        if t is None:
            continue
        if not t.is_cuda:
            raise ValueError("libscaleqlora takes device tensors")
        if dev is None:
            dev = torch.cuda.current_device()
        if t.device.index != dev:
            raise ValueError(f"tensor on {t.device}, but the current device is cuda:{dev}")


# The C ABI receives bare pointers and cannot see a buffer's size, dtype or
# strides, so the binding checks them before every call: a wrong dtype, a
# non-contiguous view or a short buffer raises ValueError instead of reaching
# the kernels.
def _need(t, name, dtypes, shape=None, numel=None):
    if not isinstance(t, torch.Tensor):
        raise ValueError(f"{name} must be a torch.Tensor")
    if not isinstance(dtypes, tuple):
        dtypes = (dtypes,)
    if t.dtype not in dtypes:
        raise ValueError(f"{name} must be {' or '.join(str(d) for d in dtypes)}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} has shape {tuple(t.shape)}, expected {tuple(shape)}")
    if numel is not None and t.numel() != numel:
        raise ValueError(f"{name} has {t.numel()} elements, expected {numel}")
    return t


def _dims2(t, name):
    if not isinstance(t, torch.Tensor) or t.dim() != 2:
        raise ValueError(f"{name} must be a 2-D tensor")
    return t.shape


def _block(fmt, I):
    if fmt not in BLOCK:
        raise ValueError(f"unknown format {fmt}")
    B = BLOCK[fmt]
    if I % B:
        raise ValueError(f"the input dimension {I} is not a multiple of the block {B}")
    return I // B


def _layer(fmt, O, I, codes, scales=None):
    """codes uint8 [O, I/2] and scales uint8 [O, I/B] of one layer."""
    G = _block(fmt, I)
    _need(codes, "codes", torch.uint8, (O, I // 2))
    if scales is not None:
        _need(scales, "scales", torch.uint8, (O, G))
    return G


_BF16 = torch.bfloat16
_F32 = torch.float32
_OUT = (torch.float32, torch.bfloat16)


# ---------------------------------------------------------------- entry points
def sq_fwd(fmt, X, codes, scales, ws2=1.0, out_dtype=torch.float32, Y=None):
    """Y = X W^T.  X bf16 [T, I], codes uint8 [O, I/2], scales uint8 [O, G]."""
    fmt = _fmt(fmt)
    T, I = _dims2(X, "X")
    O = _dims2(codes, "codes")[0]
    _need(X, "X", _BF16)
    _layer(fmt, O, I, codes, scales)
    if Y is None:
        Y = torch.empty((T, O), dtype=out_dtype, device=X.device)
    _need(Y, "Y", _OUT, (T, O))
    _dev(X, codes, scales, Y)
    _check("sq_fwd", load().sq_fwd(fmt, T, O, I, _ptr(X), _ptr(codes), _ptr(scales), float(ws2), _ptr(Y),
                                   OUT_BF16 if Y.dtype == torch.bfloat16 else OUT_F32, _stream()))
    return Y


def sq_bwd_dx(fmt, dY, codes, scales, ws2=1.0, out_dtype=torch.float32, dX=None):
    """dX = dY W.  dY bf16 [T, O] -> dX [T, I]."""
    fmt = _fmt(fmt)
    T, O = _dims2(dY, "dY")
    I = _dims2(codes, "codes")[1] * 2
    _need(dY, "dY", _BF16)
    _layer(fmt, O, I, codes, scales)
    if dX is None:
        dX = torch.empty((T, I), dtype=out_dtype, device=dY.device)
    _need(dX, "dX", _OUT, (T, I))
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
    T, I = _dims2(X, "X")
    O = _dims2(dY, "dY")[1]
    _need(X, "X", _BF16)
    _need(dY, "dY", _BF16, (T, O))
    G = _layer(fmt, O, I, codes)
    if dS is None:
        dS = torch.empty((O, G), dtype=torch.float32, device=X.device)
    _need(dS, "dS", _F32, (O, G))
    ws_bytes = sq_bwd_dscale_workspace(fmt, T, O, I)
    if ws_bytes and workspace is None:
        workspace = torch.empty(ws_bytes, dtype=torch.uint8, device=X.device)
    if workspace is not None:
        _need(workspace, "workspace", torch.uint8)
    _dev(X, dY, codes, dS, workspace)
    wsz = workspace.numel() if workspace is not None else 0
    _check("sq_bwd_dscale", load().sq_bwd_dscale(fmt, T, O, I, _ptr(X), _ptr(dY), _ptr(codes), _ptr(dS),
                                                 _ptr(workspace), wsz, _stream()))
    return dS


def sq_bwd_dscale_noalloc(fmt, X, dY, codes, dS):
    """sq_bwd_dscale with the library's static device scratch instead of a
    workspace (the caller passes dS; nothing is allocated)."""
    fmt = _fmt(fmt)
    T, I = _dims2(X, "X")
    O = _dims2(dY, "dY")[1]
    _need(X, "X", _BF16)
    _need(dY, "dY", _BF16, (T, O))
    G = _layer(fmt, O, I, codes)
    _need(dS, "dS", _F32, (O, G))
    _dev(X, dY, codes, dS)
    _check("sq_bwd_dscale_noalloc", load().sq_bwd_dscale_noalloc(fmt, T, O, I, _ptr(X), _ptr(dY), _ptr(codes),
                                                                 _ptr(dS), _stream()))
    return dS


def sq_merge_scales(fmt, scales, delta=None, src=None, ws2=1.0, mode=None):
    """In-place merge (delta given) or swap (src given) of one scale plane."""
    fmt = _fmt(fmt)
    if mode is None:
        mode = MERGE_COPY if src is not None else MERGE_DELTA
    _check_plane(scales, delta, src, mode)
    _dev(scales, delta, src)
    _check("sq_merge_scales", load().sq_merge_scales(fmt, scales.numel(), _ptr(scales), _ptr(delta),
                                                     _ptr(src), float(ws2), mode, _stream()))
    return scales


def _check_plane(scales, delta, src, mode):
    _need(scales, "scales", torch.uint8)
    if mode == MERGE_DELTA:
        _need(delta, "delta", _F32, numel=scales.numel())
    elif mode == MERGE_COPY:
        _need(src, "src", torch.uint8, numel=scales.numel())


class MergeGroup:
    """A prepared descriptor table for sq_merge_scales_grouped (built once,
    reused across calls; the tensors it names must stay alive)."""

    def __init__(self, planes):
        self.planes = planes
        self.arr = (MergeDesc * max(len(planes), 1))()
        for k, p in enumerate(planes):
            mode = p.get("mode", MERGE_COPY if p.get("src") is not None else MERGE_DELTA)
            _check_plane(p["scales"], p.get("delta"), p.get("src"), mode)
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
        if kind not in ("fwd", "dx", "ds"):
            raise ValueError(f"unknown grouped product {kind}")
        if len(codes) == 0:
            raise ValueError("no experts")
        self.O, self.I = _dims2(codes[0], "codes[0]")[0], codes[0].shape[1] * 2
        dev = codes[0].device
        if outs is None:
            if kind == "fwd":
                outs = [torch.empty((x.shape[0], self.O), dtype=out_dtype, device=dev) for x in acts]
            elif kind == "dx":
                outs = [torch.empty((d.shape[0], self.I), dtype=out_dtype, device=dev) for d in acts]
            else:
                outs = [torch.empty((self.O, self.I // BLOCK[self.fmt]), dtype=torch.float32, device=dev)
                        for _ in codes]
        self._validate(acts, codes, scales, outs, acts2, ws2)
        _dev(*acts, *codes, *(scales or []), *outs, *(acts2 or []))
        self.refs = (acts, codes, scales, outs, acts2)
        self.outs = outs
        self.n = len(codes)
        self.arr = _expert_table(acts, acts2, codes, scales, outs, ws2)
        self.dtype = _DTYPE_CODE[outs[0].dtype] if (outs and kind != "ds") else OUT_F32

    def _validate(self, acts, codes, scales, outs, acts2, ws2):
        O, I, n = self.O, self.I, len(codes)
        G = _block(self.fmt, I)
        lists = [("acts", acts), ("outs", outs)] + ([("scales", scales)] if self.kind != "ds" else []) \
            + ([("acts2", acts2)] if self.kind == "ds" else [])
        for name, lst in lists:
            if lst is None or len(lst) != n:
                raise ValueError(f"{name} needs one tensor per expert ({n})")
        if self.fmt == NVFP4 and self.kind != "ds" and (ws2 is None or len(ws2) != n):
            raise ValueError("NVFP4 needs one ws2 per expert")
        out_dtypes = set()
        for e in range(n):
            _layer(self.fmt, O, I, codes[e], scales[e] if self.kind != "ds" else None)
            T = _dims2(acts[e], f"acts[{e}]")[0]
            if self.kind == "fwd":
                _need(acts[e], f"acts[{e}]", _BF16, (T, I))
                _need(outs[e], f"outs[{e}]", _OUT, (T, O))
                out_dtypes.add(outs[e].dtype)
            elif self.kind == "dx":
                _need(acts[e], f"acts[{e}]", _BF16, (T, O))
                _need(outs[e], f"outs[{e}]", _OUT, (T, I))
                out_dtypes.add(outs[e].dtype)
            else:
                _need(acts[e], f"acts[{e}]", _BF16, (T, I))
                _need(acts2[e], f"acts2[{e}]", _BF16, (T, O))
                _need(outs[e], f"outs[{e}]", _F32, (O, G))
        if len(out_dtypes) > 1:
            raise ValueError("every expert's output must have the same dtype")

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
    O, I = _dims2(W, "W")
    _need(W, "W", _BF16)
    G = _block(fmt, I)
    dev = W.device
    if codes is None:
        codes = torch.empty((O, I // 2), dtype=torch.uint8, device=dev)
    if scales is None:
        scales = torch.empty((O, G), dtype=torch.uint8, device=dev)
    if fmt == NVFP4 and ws2_out is None:
        ws2_out = torch.empty(1, dtype=torch.float32, device=dev)
    _layer(fmt, O, I, codes, scales)
    if ws2_out is not None:
        _need(ws2_out, "ws2_out", _F32, numel=1)
    _dev(W, codes, scales, ws2_out)
    _check("rtn_quantize", load().rtn_quantize(fmt, O, I, _ptr(W), float(ws2_in), int(tie), _ptr(codes),
                                               _ptr(scales), _ptr(ws2_out), _stream()))
    return codes, scales, ws2_out


def rtn_quantize_rule(fmt, W, rule, ws2_in=0.0, seed=0, codes=None, scales=None, ws2_out=None):
    """Re-quantisation of bf16 W [O, I] under a deploy rule (RULE_*) -> (codes, scales, ws2_out).
    ws2_out is allocated where the call needs it (NVFP4, or the whole-tensor rule)."""
    fmt = _fmt(fmt)
    rule = RULES.get(rule, rule)
    O, I = _dims2(W, "W")
    _need(W, "W", _BF16)
    G = _block(fmt, I)
    dev = W.device
    if codes is None:
        codes = torch.empty((O, I // 2), dtype=torch.uint8, device=dev)
    if scales is None:
        scales = torch.empty((O, G), dtype=torch.uint8, device=dev)
    if (fmt == NVFP4 or rule == RULE_WHOLE_TENSOR) and ws2_out is None:
        ws2_out = torch.empty(1, dtype=torch.float32, device=dev)
    _layer(fmt, O, I, codes, scales)
    if ws2_out is not None:
        _need(ws2_out, "ws2_out", _F32, numel=1)
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
            O, I = _dims2(w["W"], f"weights[{k}].W")
            _need(w["W"], f"weights[{k}].W", _BF16)
            _layer(self.fmt, O, I, w["codes"], w["scales"])
            if w.get("ws2_out") is not None:
                _need(w["ws2_out"], f"weights[{k}].ws2_out", _F32, numel=1)
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
    O, I = _dims2(codes, "codes")[0], codes.shape[1] * 2
    r = _dims2(B, "B")[1]
    _layer(fmt, O, I, codes, scales)
    _need(B, "B", _BF16, (O, r))
    _need(A, "A", _BF16, (r, I))
    if codes_out is None:
        codes_out = torch.empty_like(codes)
    if scales_out is None:
        scales_out = torch.empty_like(scales)
    _layer(fmt, O, I, codes_out, scales_out)
    _dev(codes, scales, B, A, codes_out, scales_out)
    _check("sq_qat_requant", load().sq_qat_requant(fmt, O, I, r, _ptr(codes), _ptr(scales), float(ws2), _ptr(B),
                                                   _ptr(A), float(alpha_over_r), _ptr(codes_out),
                                                   _ptr(scales_out), _stream()))
    return codes_out, scales_out


def sq_qat_requant_batched(fmt, codes, scales, B, A, alpha_over_r, ws2=None, codes_out=None, scales_out=None):
    """sq_qat_requant for E stacked experts: codes uint8 [E, O, I/2], scales uint8 [E, O, G],
    B bf16 [E, O, r], A bf16 [E, r, I]; ws2: E per-expert NVFP4 scalars."""
    fmt = _fmt(fmt)
    if not isinstance(codes, torch.Tensor) or codes.dim() != 3 or not isinstance(B, torch.Tensor) or B.dim() != 3:
        raise ValueError("codes and B must be 3-D (stacked experts)")
    E, O, I = codes.shape[0], codes.shape[1], codes.shape[2] * 2
    r = B.shape[2]
    G = _block(fmt, I)
    _need(codes, "codes", torch.uint8)
    _need(scales, "scales", torch.uint8, (E, O, G))
    _need(B, "B", _BF16, (E, O, r))
    _need(A, "A", _BF16, (E, r, I))
    if codes_out is None:
        codes_out = torch.empty_like(codes)
    if scales_out is None:
        scales_out = torch.empty_like(scales)
    _need(codes_out, "codes_out", torch.uint8, (E, O, I // 2))
    _need(scales_out, "scales_out", torch.uint8, (E, O, G))
    w = None
    if fmt == NVFP4:
        if ws2 is None or len(ws2) != E:
            raise ValueError("NVFP4 needs one ws2 per expert")
        w = (ctypes.c_float * E)(*[float(v) for v in ws2])
    _dev(codes, scales, B, A, codes_out, scales_out)
    _check("sq_qat_requant_batched", load().sq_qat_requant_batched(
        fmt, E, O, I, r, _ptr(codes), _ptr(scales), ctypes.cast(w, ctypes.c_void_p) if w is not None else None,
        _ptr(B), _ptr(A), float(alpha_over_r), _ptr(codes_out), _ptr(scales_out), _stream()))
    return codes_out, scales_out


def _tokens(T):
    arr = (ctypes.c_int64 * max(len(T), 1))(*[int(t) for t in T])
    return arr


def sq_lora_grads_batched_workspace(T, O, I, r):
    return int(load().sq_lora_grads_batched_workspace(len(T), ctypes.cast(_tokens(T), ctypes.c_void_p), O, I, r))


def sq_lora_grads_batched(T, X, dY, B, A, alpha_over_r, dB=None, dA=None, workspace=None):
    """STE factor gradients of E experts: T the E token counts; X bf16 [sum T, I] and
    dY bf16 [sum T, O] with the experts' token rows one after another; B bf16 [E, O, r],
    A bf16 [E, r, I] -> dB fp32 [E, O, r], dA fp32 [E, r, I]."""
    T = [int(t) for t in T]
    E = len(T)
    if not isinstance(B, torch.Tensor) or B.dim() != 3 or B.shape[0] != E:
        raise ValueError("B must be [E, O, r] with one expert per token count")
    _, O, r = B.shape
    Ttot, I = _dims2(X, "X")
    if Ttot != sum(T):
        raise ValueError(f"X has {Ttot} rows, the token counts add to {sum(T)}")
    _need(X, "X", _BF16)
    _need(dY, "dY", _BF16, (Ttot, O))
    _need(B, "B", _BF16)
    _need(A, "A", _BF16, (E, r, I))
    dev = B.device
    if dB is None:
        dB = torch.empty((E, O, r), dtype=torch.float32, device=dev)
    if dA is None:
        dA = torch.empty((E, r, I), dtype=torch.float32, device=dev)
    _need(dB, "dB", _F32, (E, O, r))
    _need(dA, "dA", _F32, (E, r, I))
    tarr = _tokens(T)
    need = int(load().sq_lora_grads_batched_workspace(E, ctypes.cast(tarr, ctypes.c_void_p), O, I, r))
    if workspace is None and need > 0:
        workspace = torch.empty(need, dtype=torch.uint8, device=dev)
    if workspace is not None:
        _need(workspace, "workspace", torch.uint8)
    _dev(X, dY, B, A, dB, dA, workspace)
    nbytes = workspace.numel() if workspace is not None else 0
    _check("sq_lora_grads_batched", load().sq_lora_grads_batched(
        E, ctypes.cast(tarr, ctypes.c_void_p), O, I, r, _ptr(X), _ptr(dY), _ptr(B), _ptr(A), float(alpha_over_r),
        _ptr(dB), _ptr(dA), _ptr(workspace), nbytes, _stream()))
    return dB, dA


def sq_lora_grads_workspace(T, O, I, r):
    return int(load().sq_lora_grads_workspace(T, O, I, r))


def sq_lora_grads(X, dY, B, A, alpha_over_r, dB=None, dA=None, workspace=None):
    """STE factor gradients dB [O, r], dA [r, I] (fp32) of W = base + alpha_over_r B A."""
    T, I = _dims2(X, "X")
    O, r = _dims2(B, "B")
    _need(X, "X", _BF16)
    _need(dY, "dY", _BF16, (T, O))
    _need(B, "B", _BF16)
    _need(A, "A", _BF16, (r, I))
    dev = B.device
    if dB is None:
        dB = torch.empty((O, r), dtype=torch.float32, device=dev)
    if dA is None:
        dA = torch.empty((r, I), dtype=torch.float32, device=dev)
    _need(dB, "dB", _F32, (O, r))
    _need(dA, "dA", _F32, (r, I))
    need = sq_lora_grads_workspace(T, O, I, r)
    if workspace is None and need > 0:
        workspace = torch.empty(need, dtype=torch.uint8, device=dev)
    if workspace is not None:
        _need(workspace, "workspace", torch.uint8)
    _dev(X, dY, B, A, dB, dA, workspace)
    nbytes = workspace.numel() if workspace is not None else 0
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
    O, G = _dims2(base_scales, "base_scales")
    r = _dims2(B, "B")[1]
    _need(base_scales, "base_scales", torch.uint8)
    _need(B, "B", _BF16, (O, r))
    _need(A, "A", _BF16, (r, G))
    if scales_out is None:
        scales_out = torch.empty_like(base_scales)
    if want_mask and mask_out is None:
        mask_out = torch.empty_like(base_scales)
    _need(scales_out, "scales_out", torch.uint8, (O, G))
    if mask_out is not None:
        _need(mask_out, "mask_out", torch.uint8, (O, G))
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
    if base_scales.dim() != 3 or B.dim() != 3:
        raise ValueError("base_scales and B must be 3-D (stacked experts)")
    E, O, G = base_scales.shape
    r = B.shape[2]
    _need(base_scales, "base_scales", torch.uint8)
    _need(B, "B", _BF16, (E, O, r))
    _need(A, "A", _BF16, (E, r, G))
    if scales_out is None:
        scales_out = torch.empty_like(base_scales)
    if want_mask and mask_out is None:
        mask_out = torch.empty_like(base_scales)
    _need(scales_out, "scales_out", torch.uint8, (E, O, G))
    if mask_out is not None:
        _need(mask_out, "mask_out", torch.uint8, (E, O, G))
    w = None
    if fmt == NVFP4:
        if ws2 is None or len(ws2) != E:
            raise ValueError("NVFP4 needs one ws2 per expert")
        w = (ctypes.c_float * E)(*[float(v) for v in ws2])
    _dev(base_scales, B, A, scales_out, mask_out)
    _check("sq_qast_scales_batched", load().sq_qast_scales_batched(
        fmt, E, O, G, r, _ptr(base_scales), _ptr(B), _ptr(A), float(alpha_over_r),
        ctypes.cast(w, ctypes.c_void_p) if w is not None else None, _ptr(scales_out), _ptr(mask_out), _stream()))
    return scales_out, mask_out


def sq_qast_factor_grads_batched(dS, mask, B, A, alpha_over_r, dB=None, dA=None, workspace=None):
    """dB [E, O, r], dA [E, r, G] (fp32) for E stacked experts."""
    if dS.dim() != 3 or B.dim() != 3:
        raise ValueError("dS and B must be 3-D (stacked experts)")
    E, O, G = dS.shape
    r = B.shape[2]
    _need(dS, "dS", _F32)
    if mask is not None:
        _need(mask, "mask", torch.uint8, (E, O, G))
    _need(B, "B", _BF16, (E, O, r))
    _need(A, "A", _BF16, (E, r, G))
    if dB is None:
        dB = torch.empty((E, O, r), dtype=torch.float32, device=dS.device)
    if dA is None:
        dA = torch.empty((E, r, G), dtype=torch.float32, device=dS.device)
    _need(dB, "dB", _F32, (E, O, r))
    _need(dA, "dA", _F32, (E, r, G))
    need = int(load().sq_qast_factor_grads_batched_workspace(E, O, G, r))
    if workspace is None:
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=dS.device)
    _need(workspace, "workspace", torch.uint8)
    _dev(dS, mask, B, A, dB, dA, workspace)
    _check("sq_qast_factor_grads_batched", load().sq_qast_factor_grads_batched(
        E, O, G, r, _ptr(dS), _ptr(mask), _ptr(B), _ptr(A), float(alpha_over_r), _ptr(dB), _ptr(dA),
        _ptr(workspace), workspace.numel(), _stream()))
    return dB, dA


def sq_qast_factor_grads_workspace(O, G, r):
    return int(load().sq_qast_factor_grads_workspace(O, G, r))


def sq_qast_factor_grads(dS, mask, B, A, alpha_over_r, dB=None, dA=None, workspace=None):
    """dB [O, r] and dA [r, G] (fp32) from dS [O, G] through the clamp mask (None: all pass)."""
    O, G = _dims2(dS, "dS")
    r = _dims2(B, "B")[1]
    _need(dS, "dS", _F32)
    if mask is not None:
        _need(mask, "mask", torch.uint8, (O, G))
    _need(B, "B", _BF16, (O, r))
    _need(A, "A", _BF16, (r, G))
    if dB is None:
        dB = torch.empty((O, r), dtype=torch.float32, device=dS.device)
    if dA is None:
        dA = torch.empty((r, G), dtype=torch.float32, device=dS.device)
    _need(dB, "dB", _F32, (O, r))
    _need(dA, "dA", _F32, (r, G))
    need = sq_qast_factor_grads_workspace(O, G, r)
    if workspace is None:
        workspace = torch.empty(max(need, 4), dtype=torch.uint8, device=dS.device)
    _need(workspace, "workspace", torch.uint8)
    _dev(dS, mask, B, A, dB, dA, workspace)
    wsz = workspace.numel()
    _check("sq_qast_factor_grads", load().sq_qast_factor_grads(O, G, r, _ptr(dS), _ptr(mask), _ptr(B), _ptr(A),
                                                               float(alpha_over_r), _ptr(dB), _ptr(dA),
                                                               _ptr(workspace), wsz, _stream()))
    return dB, dA


def sq_scale_applied_delta(fmt, before, after, applied=None):
    """fp32 on-grid delta value(after) - value(before) of two scale planes (same shape)."""
    fmt = _fmt(fmt)
    _need(before, "before", torch.uint8)
    _need(after, "after", torch.uint8, numel=before.numel())
    if applied is None:
        applied = torch.empty(before.shape, dtype=torch.float32, device=before.device)
    _need(applied, "applied", _F32, numel=before.numel())
    _dev(before, after, applied)
    _check("sq_scale_applied_delta", load().sq_scale_applied_delta(fmt, before.numel(), _ptr(before), _ptr(after),
                                                                   _ptr(applied), _stream()))
    return applied


def sq_scale_rollback(fmt, scales, applied):
    """In place: scales := encode(value(scales) - applied)."""
    fmt = _fmt(fmt)
    _need(scales, "scales", torch.uint8)
    _need(applied, "applied", _F32, numel=scales.numel())
    _dev(scales, applied)
    _check("sq_scale_rollback", load().sq_scale_rollback(fmt, scales.numel(), _ptr(scales), _ptr(applied), _stream()))
    return scales


def sq_byte_diff(a, b, counts=None):
    """Adds (differing bytes, differing nibbles) of two byte planes to a device int64 [2] tensor."""
    _need(a, "a", torch.uint8)
    _need(b, "b", torch.uint8, numel=a.numel())
    if counts is None:
        counts = torch.zeros(2, dtype=torch.int64, device=a.device)
    _need(counts, "counts", torch.int64, numel=2)
    _dev(a, b, counts)
    _check("sq_byte_diff", load().sq_byte_diff(a.numel(), _ptr(a), _ptr(b), _ptr(counts), _stream()))
    return counts


def abi_version():
    return int(load().sq_abi_version())
