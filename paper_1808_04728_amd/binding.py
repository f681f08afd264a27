"""ctypes binding of the C ABI in include/cosmoflow.h.

Argument marshalling only: every function here has the name of its C entry
point, turns torch tensors into device pointers and the current torch stream
into a hipStream_t, calls the library and raises ``CfError`` on a non-zero
status.  All computation happens in the HIP kernels of libcosmoflow_hip.so;
if the library is missing this module raises instead of computing anything
another way.
"""
from __future__ import annotations

import ctypes
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libcosmoflow_hip.so")

CF_OK, CF_ERR_INVALID_ARG, CF_ERR_UNSUPPORTED, CF_ERR_ALIGNMENT, CF_ERR_ALIAS, \
    CF_ERR_WORKSPACE, CF_ERR_LAUNCH = range(7)
CF_F32, CF_BF16 = 0, 1
CF_PAD_SAME_TF, CF_PAD_VALID = 0, 1
CF_FUSE_POOL2 = 1
CF_FUSE_MASK = 2
FUSED_FWD, FUSED_BWD_WEIGHT, FUSED_BWD_DATA, FUSED_BWD_WEIGHT_DZ = 1, 2, 4, 8

STATUS_NAMES = {0: "CF_OK", 1: "CF_ERR_INVALID_ARG", 2: "CF_ERR_UNSUPPORTED", 3: "CF_ERR_ALIGNMENT",
                4: "CF_ERR_ALIAS", 5: "CF_ERR_WORKSPACE", 6: "CF_ERR_LAUNCH"}

# every symbol the header declares
EXPORTS = [
    "cf_version", "cf_last_error", "cf_conv3d_out_shape", "cf_conv3d_fwd", "cf_conv3d_bwd_data",
    "cf_conv3d_bwd_weight_workspace_size", "cf_conv3d_bwd_weight", "cf_bias_lrelu_fwd",
    "cf_bias_lrelu_bwd_workspace_size", "cf_bias_lrelu_bwd", "cf_avgpool3d_fwd", "cf_avgpool3d_bwd",
    "cf_conv3d_fused_supported", "cf_conv3d_mask_bytes", "cf_conv3d_fwd_fused",
    "cf_conv3d_bwd_weight_fused_workspace_size", "cf_conv3d_bwd_weight_fused", "cf_conv3d_bwd_weight_fused_dz",
    "cf_conv3d_bwd_data_fused", "cf_reduce_partials", "cf_conv3d_bwd_weight_deferred", "cf_bias_lrelu_bwd_deferred",
    "cf_conv3d_bwd_weight_fused_deferred", "cf_adam_larc_workspace_size", "cf_adam_larc_step",
    "cf_fc_fwd_workspace_size", "cf_fc_fwd", "cf_fc_bwd_data", "cf_fc_bwd_weight", "cf_mse_loss",
    "cf_fc_head_workspace_size", "cf_fc_head",
    "cf_conv3d_bwd_weight_noalloc", "cf_avgpool3d_lrelu_bwd_workspace_size", "cf_avgpool3d_lrelu_bwd",
    "cf_avgpool3d_lrelu_bwd_deferred", "cf_conv3d_bwd_fused", "cf_conv3d_bwd_fused_deferred",
    "cf_conv3d_bwd", "cf_conv3d_bwd_deferred",
]


class CfError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{STATUS_NAMES.get(status, status)}: {msg}")
        self.status = status


class cf_conv3d_desc(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in
                ("n", "d", "h", "w", "c_in", "c_out", "kd", "kh", "kw", "sd", "sh", "sw", "pad", "dtype")]


class cf_reduction(ctypes.Structure):
    _fields_ = [("part", ctypes.c_void_p), ("out", ctypes.c_void_p), ("rows", ctypes.c_int32),
                ("cols", ctypes.c_int32)]


CF_MAX_PENDING = 4


class cf_adam_larc_hparams(ctypes.Structure):
    _fields_ = [("eta0", ctypes.c_double), ("eta_min", ctypes.c_double), ("t_decay", ctypes.c_int64),
                ("beta1", ctypes.c_double), ("beta2", ctypes.c_double), ("eps_hat", ctypes.c_double),
                ("larc_coef", ctypes.c_double), ("larc_fallback", ctypes.c_double), ("larc_clip", ctypes.c_double)]


CF_ADAM_MAX_GROUPS = 128
#: the paper's hyperparameters (Section III-B); t_decay is the caller's choice
PAPER_HPARAMS = dict(eta0=2e-3, eta_min=1e-4, beta1=0.9, beta2=0.999, eps_hat=1e-8,
                     larc_coef=0.002, larc_fallback=6.25e-5, larc_clip=1.0)


def make_hparams(t_decay, **kw) -> cf_adam_larc_hparams:
    h = dict(PAPER_HPARAMS)
    h.update(kw)
    return cf_adam_larc_hparams(h["eta0"], h["eta_min"], int(t_decay), h["beta1"], h["beta2"], h["eps_hat"],
                                h["larc_coef"], h["larc_fallback"], h["larc_clip"])


_lib = None


def lib():
    """Load libcosmoflow_hip.so (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is missing: build it with `python -m paper_1808_04728_amd.build` "
                          "(there is no fallback implementation)")
    L = ctypes.CDLL(LIB_PATH)
    vp, i32, i64, f32, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_float, ctypes.c_size_t
    D = ctypes.POINTER(cf_conv3d_desc)
    sig = {
        "cf_version": ([], ctypes.c_char_p),
        "cf_last_error": ([], ctypes.c_char_p),
        "cf_conv3d_out_shape": ([D, ctypes.POINTER(i32)], ctypes.c_int),
        "cf_conv3d_fwd": ([D, vp, vp, vp, vp], ctypes.c_int),
        "cf_conv3d_bwd_data": ([D, vp, vp, vp, vp], ctypes.c_int),
        "cf_conv3d_bwd_weight_workspace_size": ([D], sz),
        "cf_conv3d_bwd_weight": ([D, vp, vp, vp, vp, sz, vp], ctypes.c_int),
        "cf_conv3d_bwd_weight_noalloc": ([D, vp, vp, vp, vp], ctypes.c_int),
        "cf_bias_lrelu_fwd": ([i64, i32, i32, vp, vp, f32, vp, vp], ctypes.c_int),
        "cf_bias_lrelu_bwd_workspace_size": ([i64, i32], sz),
        "cf_bias_lrelu_bwd": ([i64, i32, i32, vp, vp, f32, vp, vp, vp, sz, vp], ctypes.c_int),
        "cf_avgpool3d_fwd": ([i32] * 8 + [vp, vp, vp], ctypes.c_int),
        "cf_avgpool3d_bwd": ([i32] * 8 + [vp, vp, vp], ctypes.c_int),
        "cf_avgpool3d_lrelu_bwd_workspace_size": ([i32] * 5, sz),
        "cf_avgpool3d_lrelu_bwd": ([i32] * 6 + [vp, vp, f32, vp, vp, vp, sz, vp], ctypes.c_int),
        "cf_avgpool3d_lrelu_bwd_deferred": ([i32] * 6 + [vp, vp, f32, vp, vp, vp, sz, ctypes.POINTER(cf_reduction),
                                                         ctypes.POINTER(i32), vp], ctypes.c_int),
        "cf_conv3d_fused_supported": ([D, ctypes.c_uint32], i32),
        "cf_conv3d_mask_bytes": ([D], sz),
        "cf_conv3d_fwd_fused": ([D, vp, vp, vp, f32, ctypes.c_uint32, vp, vp, vp], ctypes.c_int),
        "cf_conv3d_bwd_weight_fused_workspace_size": ([D, ctypes.c_uint32], sz),
        "cf_conv3d_bwd_weight_fused": ([D, vp, vp, vp, f32, ctypes.c_uint32, vp, vp, vp, sz, vp], ctypes.c_int),
        "cf_conv3d_bwd_weight_fused_dz": ([D, vp, vp, vp, f32, ctypes.c_uint32, vp, vp, vp, vp, sz, vp],
                                          ctypes.c_int),
        "cf_conv3d_bwd_data_fused": ([D, vp, vp, vp, f32, ctypes.c_uint32, vp, vp], ctypes.c_int),
        "cf_conv3d_bwd": ([D, vp, vp, vp, vp, vp, vp, sz, vp], ctypes.c_int),
        "cf_conv3d_bwd_deferred": ([D, vp, vp, vp, vp, vp, vp, sz, ctypes.POINTER(cf_reduction),
                                    ctypes.POINTER(i32), vp], ctypes.c_int),
        "cf_conv3d_bwd_fused": ([D, vp, vp, vp, vp, f32, ctypes.c_uint32, vp, vp, vp, vp, sz, vp], ctypes.c_int),
        "cf_conv3d_bwd_fused_deferred": ([D, vp, vp, vp, vp, f32, ctypes.c_uint32, vp, vp, vp, vp, sz,
                                          ctypes.POINTER(cf_reduction), ctypes.POINTER(i32), vp], ctypes.c_int),
        "cf_reduce_partials": ([i32, ctypes.POINTER(cf_reduction), vp], ctypes.c_int),
        "cf_conv3d_bwd_weight_deferred": ([D, vp, vp, vp, vp, sz, ctypes.POINTER(cf_reduction),
                                           ctypes.POINTER(i32), vp], ctypes.c_int),
        "cf_bias_lrelu_bwd_deferred": ([i64, i32, i32, vp, vp, f32, vp, vp, vp, sz, ctypes.POINTER(cf_reduction),
                                        ctypes.POINTER(i32), vp], ctypes.c_int),
        "cf_conv3d_bwd_weight_fused_deferred": ([D, vp, vp, vp, f32, ctypes.c_uint32, vp, vp, vp, vp, sz,
                                                 ctypes.POINTER(cf_reduction), ctypes.POINTER(i32), vp],
                                                ctypes.c_int),
        "cf_adam_larc_workspace_size": ([i32, ctypes.POINTER(i64)], sz),
        "cf_adam_larc_step": ([i32, ctypes.POINTER(i64), i64, ctypes.POINTER(cf_adam_larc_hparams), vp, vp, vp, vp,
                               vp, vp, sz, vp], ctypes.c_int),
        "cf_fc_fwd_workspace_size": ([i32, i32, i32], sz),
        "cf_fc_fwd": ([i32, i32, i32, i32, vp, vp, vp, vp, sz, vp], ctypes.c_int),
        "cf_fc_bwd_data": ([i32, i32, i32, i32, vp, vp, vp, vp], ctypes.c_int),
        "cf_fc_bwd_weight": ([i32, i32, i32, i32, vp, vp, vp, vp], ctypes.c_int),
        "cf_mse_loss": ([i32, i32, i32, vp, vp, vp, vp, vp], ctypes.c_int),
        "cf_fc_head_workspace_size": ([i32, i32, ctypes.POINTER(i32)], sz),
        "cf_fc_head": ([i32, i32, ctypes.POINTER(i32), i32, vp, ctypes.POINTER(vp), ctypes.POINTER(vp), f32, vp,
                        ctypes.POINTER(vp), ctypes.POINTER(vp), ctypes.POINTER(vp), ctypes.POINTER(vp),
                        ctypes.POINTER(vp), vp, vp, sz, vp], ctypes.c_int),
    }
    for name, (args, res) in sig.items():
        f = getattr(L, name)
        f.argtypes = args
        f.restype = res
    _lib = L
    return L


def _check(status: int):
    if status != CF_OK:
        raise CfError(status, lib().cf_last_error().decode())


def _ptr(t):
    """Device pointer of a tensor, or an int/None passed through."""
    if t is None:
        return None
    if isinstance(t, int):
        return t
    return t.data_ptr()


def _stream(stream):
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def dtype_code(dt) -> int:
    if dt in (torch.float32, "f32", CF_F32):
        return CF_F32
    if dt in (torch.bfloat16, "bf16", CF_BF16):
        return CF_BF16
    raise ValueError(f"unsupported dtype {dt}")


def make_desc(n, dhw, c_in, c_out, k, stride=1, pad="same", dtype=CF_F32) -> cf_conv3d_desc:
    k3 = tuple(k) if isinstance(k, (tuple, list)) else (k,) * 3
    s3 = tuple(stride) if isinstance(stride, (tuple, list)) else (stride,) * 3
    return cf_conv3d_desc(n, *dhw, c_in, c_out, *k3, *s3,
                          CF_PAD_SAME_TF if pad == "same" else CF_PAD_VALID, dtype_code(dtype))


# ---------------------------------------------------------------------------
# entry points (same names as the C ABI)
# ---------------------------------------------------------------------------

def cf_version() -> str:
    return lib().cf_version().decode()


def cf_last_error() -> str:
    return lib().cf_last_error().decode()


def cf_conv3d_out_shape(desc):
    out = (ctypes.c_int32 * 3)()
    _check(lib().cf_conv3d_out_shape(ctypes.byref(desc), out))
    return tuple(out)


def cf_conv3d_fwd(desc, x, w, z, stream=None):
    _check(lib().cf_conv3d_fwd(ctypes.byref(desc), _ptr(x), _ptr(w), _ptr(z), _stream(stream)))


def cf_conv3d_bwd_data(desc, dz, w, dx, stream=None):
    _check(lib().cf_conv3d_bwd_data(ctypes.byref(desc), _ptr(dz), _ptr(w), _ptr(dx), _stream(stream)))


def cf_conv3d_bwd_weight_workspace_size(desc) -> int:
    return int(lib().cf_conv3d_bwd_weight_workspace_size(ctypes.byref(desc)))


def cf_conv3d_bwd_weight(desc, x, dz, dw, ws, ws_bytes=None, stream=None):
    if ws_bytes is None:
        ws_bytes = 0 if ws is None or isinstance(ws, int) else ws.numel() * ws.element_size()
    _check(lib().cf_conv3d_bwd_weight(ctypes.byref(desc), _ptr(x), _ptr(dz), _ptr(dw), _ptr(ws),
                                      ws_bytes, _stream(stream)))


def cf_conv3d_bwd_weight_noalloc(desc, x, dz, dw, stream=None):
    _check(lib().cf_conv3d_bwd_weight_noalloc(ctypes.byref(desc), _ptr(x), _ptr(dz), _ptr(dw), _stream(stream)))


def cf_bias_lrelu_fwd(nvox, c, dtype, z, bias, alpha, y, stream=None):
    _check(lib().cf_bias_lrelu_fwd(nvox, c, dtype_code(dtype), _ptr(z), _ptr(bias), alpha, _ptr(y),
                                   _stream(stream)))


def cf_bias_lrelu_bwd_workspace_size(nvox, c) -> int:
    return int(lib().cf_bias_lrelu_bwd_workspace_size(nvox, c))


def cf_bias_lrelu_bwd(nvox, c, dtype, dy, y, alpha, dz, db, ws, ws_bytes=None, stream=None):
    if ws_bytes is None:
        ws_bytes = 0 if ws is None or isinstance(ws, int) else ws.numel() * ws.element_size()
    _check(lib().cf_bias_lrelu_bwd(nvox, c, dtype_code(dtype), _ptr(dy), _ptr(y), alpha, _ptr(dz), _ptr(db),
                                   _ptr(ws), ws_bytes, _stream(stream)))


def cf_avgpool3d_fwd(n, d, h, w, c, k, s, dtype, y, p, stream=None):
    _check(lib().cf_avgpool3d_fwd(n, d, h, w, c, k, s, dtype_code(dtype), _ptr(y), _ptr(p), _stream(stream)))


def cf_avgpool3d_bwd(n, d, h, w, c, k, s, dtype, dp, dy, stream=None):
    _check(lib().cf_avgpool3d_bwd(n, d, h, w, c, k, s, dtype_code(dtype), _ptr(dp), _ptr(dy), _stream(stream)))


def cf_avgpool3d_lrelu_bwd_workspace_size(n, d, h, w, c) -> int:
    return int(lib().cf_avgpool3d_lrelu_bwd_workspace_size(n, d, h, w, c))


def cf_avgpool3d_lrelu_bwd(n, d, h, w, c, dtype, dp, mask, alpha, dz, db, ws, ws_bytes=None, stream=None):
    if ws_bytes is None:
        ws_bytes = 0 if ws is None or isinstance(ws, int) else ws.numel() * ws.element_size()
    _check(lib().cf_avgpool3d_lrelu_bwd(n, d, h, w, c, dtype_code(dtype), _ptr(dp), _ptr(mask), alpha, _ptr(dz),
                                        _ptr(db), _ptr(ws), ws_bytes, _stream(stream)))


def cf_conv3d_fused_supported(desc, flags=CF_FUSE_POOL2) -> int:
    return int(lib().cf_conv3d_fused_supported(ctypes.byref(desc), flags))


def cf_conv3d_mask_bytes(desc) -> int:
    return int(lib().cf_conv3d_mask_bytes(ctypes.byref(desc)))


def cf_conv3d_fwd_fused(desc, x, w, bias, alpha, flags, out, mask, stream=None):
    _check(lib().cf_conv3d_fwd_fused(ctypes.byref(desc), _ptr(x), _ptr(w), _ptr(bias), alpha, flags, _ptr(out),
                                     _ptr(mask), _stream(stream)))


def cf_conv3d_bwd_weight_fused_workspace_size(desc, flags=CF_FUSE_POOL2) -> int:
    return int(lib().cf_conv3d_bwd_weight_fused_workspace_size(ctypes.byref(desc), flags))


def cf_conv3d_bwd_weight_fused(desc, x, g, mask, alpha, flags, dw, db, ws, ws_bytes=None, stream=None):
    if ws_bytes is None:
        ws_bytes = 0 if ws is None or isinstance(ws, int) else ws.numel() * ws.element_size()
    _check(lib().cf_conv3d_bwd_weight_fused(ctypes.byref(desc), _ptr(x), _ptr(g), _ptr(mask), alpha, flags,
                                            _ptr(dw), _ptr(db), _ptr(ws), ws_bytes, _stream(stream)))


def cf_conv3d_bwd_weight_fused_dz(desc, x, g, mask, alpha, flags, dw, db, dz, ws, ws_bytes=None, stream=None):
    if ws_bytes is None:
        ws_bytes = 0 if ws is None or isinstance(ws, int) else ws.numel() * ws.element_size()
    _check(lib().cf_conv3d_bwd_weight_fused_dz(ctypes.byref(desc), _ptr(x), _ptr(g), _ptr(mask), alpha, flags,
                                               _ptr(dw), _ptr(db), _ptr(dz), _ptr(ws), ws_bytes, _stream(stream)))


def cf_conv3d_bwd_data_fused(desc, g, mask, w, alpha, flags, dx, stream=None):
    _check(lib().cf_conv3d_bwd_data_fused(ctypes.byref(desc), _ptr(g), _ptr(mask), _ptr(w), alpha, flags, _ptr(dx),
                                          _stream(stream)))


def cf_conv3d_bwd(desc, x, dz, w, dw, dx, ws, ws_bytes=None, stream=None):
    if ws_bytes is None:
        ws_bytes = 0 if ws is None or isinstance(ws, int) else ws.numel() * ws.element_size()
    _check(lib().cf_conv3d_bwd(ctypes.byref(desc), _ptr(x), _ptr(dz), _ptr(w), _ptr(dw), _ptr(dx), _ptr(ws),
                               ws_bytes, _stream(stream)))


def cf_conv3d_bwd_fused(desc, x, g, mask, w, alpha, flags, dw, db, dx, ws, ws_bytes=None, stream=None):
    if ws_bytes is None:
        ws_bytes = 0 if ws is None or isinstance(ws, int) else ws.numel() * ws.element_size()
    _check(lib().cf_conv3d_bwd_fused(ctypes.byref(desc), _ptr(x), _ptr(g), _ptr(mask), _ptr(w), alpha, flags,
                                     _ptr(dw), _ptr(db), _ptr(dx), _ptr(ws), ws_bytes, _stream(stream)))


# ---- deferred gradient sums --------------------------------------------------
# The _deferred calls return a list of pending cf_reduction jobs (host
# structures holding device pointers); cf_reduce_partials runs any collection
# of them.

def _pending_list(arr, n):
    return [cf_reduction(arr[i].part, arr[i].out, arr[i].rows, arr[i].cols) for i in range(n.value)]


def cf_reduce_partials(jobs, stream=None):
    n = len(jobs)
    arr = (cf_reduction * max(n, 1))(*jobs)
    _check(lib().cf_reduce_partials(n, arr, _stream(stream)))


def cf_conv3d_bwd_weight_deferred(desc, x, dz, dw, ws, ws_bytes=None, stream=None):
    if ws_bytes is None:
        ws_bytes = 0 if ws is None or isinstance(ws, int) else ws.numel() * ws.element_size()
    arr, n = (cf_reduction * CF_MAX_PENDING)(), ctypes.c_int32(0)
    _check(lib().cf_conv3d_bwd_weight_deferred(ctypes.byref(desc), _ptr(x), _ptr(dz), _ptr(dw), _ptr(ws), ws_bytes,
                                               arr, ctypes.byref(n), _stream(stream)))
    return _pending_list(arr, n)


def cf_bias_lrelu_bwd_deferred(nvox, c, dtype, dy, y, alpha, dz, db, ws, ws_bytes=None, stream=None):
    if ws_bytes is None:
        ws_bytes = 0 if ws is None or isinstance(ws, int) else ws.numel() * ws.element_size()
    arr, n = (cf_reduction * CF_MAX_PENDING)(), ctypes.c_int32(0)
    _check(lib().cf_bias_lrelu_bwd_deferred(nvox, c, dtype_code(dtype), _ptr(dy), _ptr(y), alpha, _ptr(dz), _ptr(db),
                                            _ptr(ws), ws_bytes, arr, ctypes.byref(n), _stream(stream)))
    return _pending_list(arr, n)


def cf_avgpool3d_lrelu_bwd_deferred(n, d, h, w, c, dtype, dp, mask, alpha, dz, db, ws, ws_bytes=None,
                                    stream=None):
    if ws_bytes is None:
        ws_bytes = 0 if ws is None or isinstance(ws, int) else ws.numel() * ws.element_size()
    arr, n_ = (cf_reduction * CF_MAX_PENDING)(), ctypes.c_int32(0)
    _check(lib().cf_avgpool3d_lrelu_bwd_deferred(n, d, h, w, c, dtype_code(dtype), _ptr(dp), _ptr(mask), alpha,
                                                 _ptr(dz), _ptr(db), _ptr(ws), ws_bytes, arr, ctypes.byref(n_),
                                                 _stream(stream)))
    return _pending_list(arr, n_)


def cf_conv3d_bwd_weight_fused_deferred(desc, x, g, mask, alpha, flags, dw, db, dz, ws, ws_bytes=None,
                                        stream=None):
    if ws_bytes is None:
        ws_bytes = 0 if ws is None or isinstance(ws, int) else ws.numel() * ws.element_size()
    arr, n = (cf_reduction * CF_MAX_PENDING)(), ctypes.c_int32(0)
    _check(lib().cf_conv3d_bwd_weight_fused_deferred(ctypes.byref(desc), _ptr(x), _ptr(g), _ptr(mask), alpha, flags,
                                                     _ptr(dw), _ptr(db), _ptr(dz), _ptr(ws), ws_bytes, arr,
                                                     ctypes.byref(n), _stream(stream)))
    return _pending_list(arr, n)


def cf_conv3d_bwd_deferred(desc, x, dz, w, dw, dx, ws, ws_bytes=None, stream=None):
    if ws_bytes is None:
        ws_bytes = 0 if ws is None or isinstance(ws, int) else ws.numel() * ws.element_size()
    arr, n = (cf_reduction * CF_MAX_PENDING)(), ctypes.c_int32(0)
    _check(lib().cf_conv3d_bwd_deferred(ctypes.byref(desc), _ptr(x), _ptr(dz), _ptr(w), _ptr(dw), _ptr(dx), _ptr(ws),
                                        ws_bytes, arr, ctypes.byref(n), _stream(stream)))
    return _pending_list(arr, n)


def cf_conv3d_bwd_fused_deferred(desc, x, g, mask, w, alpha, flags, dw, db, dx, ws, ws_bytes=None, stream=None):
    if ws_bytes is None:
        ws_bytes = 0 if ws is None or isinstance(ws, int) else ws.numel() * ws.element_size()
    arr, n = (cf_reduction * CF_MAX_PENDING)(), ctypes.c_int32(0)
    _check(lib().cf_conv3d_bwd_fused_deferred(ctypes.byref(desc), _ptr(x), _ptr(g), _ptr(mask), _ptr(w), alpha,
                                              flags, _ptr(dw), _ptr(db), _ptr(dx), _ptr(ws), ws_bytes, arr,
                                              ctypes.byref(n), _stream(stream)))
    return _pending_list(arr, n)


def _offsets(offsets):
    """(ngroups, ctypes int64 array); an already built pair passes through."""
    if isinstance(offsets, tuple) and len(offsets) == 2 and isinstance(offsets[1], ctypes.Array):
        return offsets
    arr = (ctypes.c_int64 * max(len(offsets), 1))(*[int(o) for o in offsets])
    return len(offsets) - 1, arr


def adam_offsets(offsets):
    """Pre-marshalled offsets for repeated cf_adam_larc_step calls."""
    return _offsets(offsets)


def cf_adam_larc_workspace_size(offsets) -> int:
    n, arr = _offsets(offsets)
    return lib().cf_adam_larc_workspace_size(n, arr)


def cf_adam_larc_step(offsets, t, hp, v, g, m, s, v16, ws, ws_bytes=None, stream=None):
    """offsets: ngroups + 1 host integers; hp: a cf_adam_larc_hparams (see make_hparams)."""
    if ws_bytes is None:
        ws_bytes = 0 if ws is None or isinstance(ws, int) else ws.numel() * ws.element_size()
    n, arr = _offsets(offsets)
    _check(lib().cf_adam_larc_step(n, arr, int(t), ctypes.byref(hp), _ptr(v), _ptr(g), _ptr(m), _ptr(s), _ptr(v16),
                                   _ptr(ws), ws_bytes, _stream(stream)))


# ---- fully-connected head and loss ---------------------------------------------

def cf_fc_fwd_workspace_size(m, k, n) -> int:
    return int(lib().cf_fc_fwd_workspace_size(m, k, n))


def cf_fc_fwd(m, k, n, dtype, x, w, z, ws, ws_bytes=None, stream=None):
    if ws_bytes is None:
        ws_bytes = 0 if ws is None or isinstance(ws, int) else ws.numel() * ws.element_size()
    _check(lib().cf_fc_fwd(m, k, n, dtype_code(dtype), _ptr(x), _ptr(w), _ptr(z), _ptr(ws), ws_bytes,
                           _stream(stream)))


def cf_fc_bwd_data(m, k, n, dtype, dz, w, dx, stream=None):
    _check(lib().cf_fc_bwd_data(m, k, n, dtype_code(dtype), _ptr(dz), _ptr(w), _ptr(dx), _stream(stream)))


def cf_fc_bwd_weight(m, k, n, dtype, x, dz, dw, stream=None):
    _check(lib().cf_fc_bwd_weight(m, k, n, dtype_code(dtype), _ptr(x), _ptr(dz), _ptr(dw), _stream(stream)))


def _i32s(v):
    return (ctypes.c_int32 * len(v))(*[int(a) for a in v])


def _ptrs(ts):
    """Host array of the device pointers of a list of tensors."""
    return (ctypes.c_void_p * max(len(ts), 1))(*[_ptr(t) for t in ts])


def cf_fc_head_workspace_size(m, dims) -> int:
    return int(lib().cf_fc_head_workspace_size(m, len(dims) - 1, _i32s(dims)))


def cf_fc_head(m, dims, dtype, x, w, b, alpha, target, y, dz, dx, dw, db, loss, ws, ws_bytes=None, stream=None):
    """Forward, loss and backward of the whole head (lists of per-layer tensors)."""
    if ws_bytes is None:
        ws_bytes = 0 if ws is None or isinstance(ws, int) else ws.numel() * ws.element_size()
    _check(lib().cf_fc_head(m, len(dims) - 1, _i32s(dims), dtype_code(dtype), _ptr(x), _ptrs(w), _ptrs(b),
                            float(alpha), _ptr(target), _ptrs(y), _ptrs(dz), _ptrs(dx), _ptrs(dw), _ptrs(db),
                            _ptr(loss), _ptr(ws), ws_bytes, _stream(stream)))


def cf_mse_loss(m, n, dtype, p, t, loss, dp, stream=None):
    _check(lib().cf_mse_loss(m, n, dtype_code(dtype), _ptr(p), _ptr(t), _ptr(loss), _ptr(dp), _stream(stream)))
