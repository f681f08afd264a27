"""CPU oracle for the CosmoFlow 3D-convolution hot path (arXiv:1808.04728).

TEST INFRASTRUCTURE, NOT PRODUCT CODE.  Only the tests, the smoke check and
the CPU-baseline leg of the benchmark may import this package.  It shares no
code with the GPU library (``paper_1808_04728_amd``) and never imports it.

The arithmetic lives in ``cfref.c`` (plain C, IEEE double, loops in the order
of the definitions; see that file's header for the passages of the paper each
function follows).  This module only compiles it with gcc, marshals numpy
arrays, and composes the per-layer definitions into the layer stack.

Conventions: activations NDHWC, weights DHWIO ``[kd][kh][kw][ci][co]``,
every array is converted to contiguous float64 before the call.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
import threading

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "cfref.c")
_LIB_PATH = os.path.join(_HERE, "libcfref.so")
_lock = threading.Lock()
_lib = None


def build(force: bool = True) -> str:
    """Compile cfref.c into libcfref.so with gcc (no fast-math)."""
    if force or not os.path.exists(_LIB_PATH):
        tmp = _LIB_PATH + ".tmp%d" % os.getpid()
        cmd = ["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-fopenmp",
               "-fno-fast-math", "-ffp-contract=off", _SRC, "-o", tmp, "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def _load():
    global _lib
    with _lock:
        if _lib is not None:
            return _lib
        if not os.path.exists(_LIB_PATH):
            build(force=False)
        lib = ctypes.CDLL(_LIB_PATH)
        P = ctypes.POINTER(ctypes.c_double)
        I = ctypes.c_int
        conv_args = [P, P, P] + [I] * 18
        for name in ("ref_conv3d_fwd", "ref_conv3d_bwd_data", "ref_conv3d_bwd_weight"):
            f = getattr(lib, name)
            f.argtypes = conv_args
            f.restype = None
        lib.ref_conv_geometry.argtypes = [I, I, I, I, ctypes.POINTER(I), ctypes.POINTER(I)]
        lib.ref_conv_geometry.restype = I
        lib.ref_conv3d_fwd_point.argtypes = [P, P] + [I] * 14 + [I] * 5
        lib.ref_conv3d_fwd_point.restype = ctypes.c_double
        lib.ref_conv3d_bwd_data_point.argtypes = [P, P] + [I] * 17 + [I] * 5
        lib.ref_conv3d_bwd_data_point.restype = ctypes.c_double
        lib.ref_conv3d_bwd_weight_point.argtypes = [P, P] + [I] * 18 + [I] * 5
        lib.ref_conv3d_bwd_weight_point.restype = ctypes.c_double
        lib.ref_bias_lrelu_fwd.argtypes = [P, P, ctypes.c_double, P, ctypes.c_int64, I]
        lib.ref_bias_lrelu_fwd.restype = None
        lib.ref_bias_lrelu_bwd.argtypes = [P, P, ctypes.c_double, P, P, ctypes.c_int64, I]
        lib.ref_bias_lrelu_bwd.restype = None
        for name in ("ref_avgpool3d_fwd", "ref_avgpool3d_bwd"):
            f = getattr(lib, name)
            f.argtypes = [P, P] + [I] * 7
            f.restype = None
        I64 = ctypes.c_int64
        lib.ref_lr_schedule.argtypes = [I64, I64, ctypes.c_double, ctypes.c_double]
        lib.ref_lr_schedule.restype = ctypes.c_double
        lib.ref_adam_larc_step.argtypes = [I, ctypes.POINTER(I64), I64, I64, P, P, P, P, P, P]
        lib.ref_adam_larc_step.restype = None
        for name in ("ref_fc_fwd", "ref_fc_bwd_data", "ref_fc_bwd_weight"):
            f = getattr(lib, name)
            f.argtypes = [P, P, P, I, I, I]
            f.restype = None
        lib.ref_mse_loss.argtypes = [P, P, P, I, I]
        lib.ref_mse_loss.restype = ctypes.c_double
        _lib = lib
        return lib


def _f64(a) -> np.ndarray:
    if hasattr(a, "detach"):  # torch tensor on the CPU
        a = a.detach().to("cpu").double().numpy()
    return np.ascontiguousarray(a, dtype=np.float64)


def _ptr(a: np.ndarray):
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_double))


def geometry(size: int, k: int, s: int, pad: str):
    """(out, pad_before) for one spatial dimension; pad is 'same' or 'valid'."""
    lib = _load()
    out = ctypes.c_int()
    pb = ctypes.c_int()
    rc = lib.ref_conv_geometry(size, k, s, 1 if pad == "same" else 0,
                               ctypes.byref(out), ctypes.byref(pb))
    if rc != 0:
        raise ValueError(f"kernel {k} does not fit extent {size} ({pad})")
    return out.value, pb.value


def _geom3(dhw, ksz, stride, pad):
    res = [geometry(dhw[i], ksz[i], stride[i], pad) for i in range(3)]
    return [r[0] for r in res], [r[1] for r in res]


def _triple(v):
    return tuple(v) if isinstance(v, (tuple, list)) else (v, v, v)


def conv3d_fwd(x, w, stride=1, pad="same"):
    """z = conv(x, W): x [N,D,H,W,CI], w [KD,KH,KW,CI,CO] -> z [N,OD,OH,OW,CO]."""
    x = _f64(x)
    w = _f64(w)
    N, D, H, W, CI = x.shape
    KD, KH, KW, CI2, CO = w.shape
    assert CI2 == CI
    s = _triple(stride)
    (OD, OH, OW), (pd, ph, pw) = _geom3((D, H, W), (KD, KH, KW), s, pad)
    z = np.zeros((N, OD, OH, OW, CO), np.float64)
    _load().ref_conv3d_fwd(_ptr(x), _ptr(w), _ptr(z), N, D, H, W, CI, CO,
                           KD, KH, KW, *s, pd, ph, pw, OD, OH, OW)
    return z


def conv3d_bwd_data(dz, w, in_dhw, stride=1, pad="same"):
    """dx = adjoint of conv w.r.t. x; in_dhw is the forward input's (D,H,W)."""
    dz = _f64(dz)
    w = _f64(w)
    N, OD, OH, OW, CO = dz.shape
    KD, KH, KW, CI, CO2 = w.shape
    assert CO2 == CO
    D, H, W = in_dhw
    s = _triple(stride)
    (od, oh, ow), (pd, ph, pw) = _geom3((D, H, W), (KD, KH, KW), s, pad)
    assert (od, oh, ow) == (OD, OH, OW), "dz shape does not match the geometry"
    dx = np.zeros((N, D, H, W, CI), np.float64)
    _load().ref_conv3d_bwd_data(_ptr(dz), _ptr(w), _ptr(dx), N, D, H, W, CI, CO,
                                KD, KH, KW, *s, pd, ph, pw, OD, OH, OW)
    return dx


def conv3d_bwd_weight(x, dz, ksize, stride=1, pad="same"):
    """dW = adjoint of conv w.r.t. W: x [N,D,H,W,CI], dz [N,OD,OH,OW,CO]."""
    x = _f64(x)
    dz = _f64(dz)
    N, D, H, W, CI = x.shape
    CO = dz.shape[-1]
    KD, KH, KW = _triple(ksize)
    s = _triple(stride)
    (OD, OH, OW), (pd, ph, pw) = _geom3((D, H, W), (KD, KH, KW), s, pad)
    assert dz.shape == (N, OD, OH, OW, CO)
    dw = np.zeros((KD, KH, KW, CI, CO), np.float64)
    _load().ref_conv3d_bwd_weight(_ptr(x), _ptr(dz), _ptr(dw), N, D, H, W, CI, CO,
                                  KD, KH, KW, *s, pd, ph, pw, OD, OH, OW)
    return dw


def conv3d_fwd_points(x, w, idx, stride=1, pad="same"):
    """z at the listed output indices idx[:, (n, od, oh, ow, co)]."""
    x = _f64(x)
    w = _f64(w)
    N, D, H, W, CI = x.shape
    KD, KH, KW, _, CO = w.shape
    s = _triple(stride)
    _, (pd, ph, pw) = _geom3((D, H, W), (KD, KH, KW), s, pad)
    f = _load().ref_conv3d_fwd_point
    return np.array([f(_ptr(x), _ptr(w), D, H, W, CI, CO, KD, KH, KW, *s, pd, ph, pw,
                       *[int(t) for t in i]) for i in idx], np.float64)


def conv3d_bwd_data_points(dz, w, in_dhw, idx, stride=1, pad="same"):
    """dx at the listed input indices idx[:, (n, id, ih, iw, ci)]."""
    dz = _f64(dz)
    w = _f64(w)
    N, OD, OH, OW, CO = dz.shape
    KD, KH, KW, CI, _ = w.shape
    D, H, W = in_dhw
    s = _triple(stride)
    _, (pd, ph, pw) = _geom3((D, H, W), (KD, KH, KW), s, pad)
    f = _load().ref_conv3d_bwd_data_point
    return np.array([f(_ptr(dz), _ptr(w), D, H, W, CI, CO, KD, KH, KW, *s, pd, ph, pw,
                       OD, OH, OW, *[int(t) for t in i]) for i in idx], np.float64)


def conv3d_bwd_weight_points(x, dz, ksize, idx, stride=1, pad="same"):
    """dW at the listed indices idx[:, (kd, kh, kw, ci, co)]."""
    x = _f64(x)
    dz = _f64(dz)
    N, D, H, W, CI = x.shape
    OD, OH, OW, CO = dz.shape[1:]
    KD, KH, KW = _triple(ksize)
    s = _triple(stride)
    _, (pd, ph, pw) = _geom3((D, H, W), (KD, KH, KW), s, pad)
    f = _load().ref_conv3d_bwd_weight_point
    return np.array([f(_ptr(x), _ptr(dz), N, D, H, W, CI, CO, KD, KH, KW, *s, pd, ph, pw,
                       OD, OH, OW, *[int(t) for t in i]) for i in idx], np.float64)


def bias_lrelu_fwd(z, b, alpha):
    z = _f64(z)
    b = _f64(b)
    C = z.shape[-1]
    assert b.shape == (C,)
    y = np.empty_like(z)
    _load().ref_bias_lrelu_fwd(_ptr(z), _ptr(b), float(alpha), _ptr(y), z.size // C, C)
    return y


def bias_lrelu_bwd(dy, y, alpha):
    """Returns (dz, db)."""
    dy = _f64(dy)
    y = _f64(y)
    assert dy.shape == y.shape
    C = y.shape[-1]
    dz = np.empty_like(y)
    db = np.zeros(C, np.float64)
    _load().ref_bias_lrelu_bwd(_ptr(dy), _ptr(y), float(alpha), _ptr(dz), _ptr(db),
                               y.size // C, C)
    return dz, db


def avgpool3d_fwd(y, k=2, s=2):
    y = _f64(y)
    N, D, H, W, C = y.shape
    OD, OH, OW = [(t - k) // s + 1 for t in (D, H, W)]
    p = np.zeros((N, OD, OH, OW, C), np.float64)
    _load().ref_avgpool3d_fwd(_ptr(y), _ptr(p), N, D, H, W, C, k, s)
    return p


def avgpool3d_bwd(dp, in_dhw, k=2, s=2):
    dp = _f64(dp)
    N = dp.shape[0]
    C = dp.shape[-1]
    D, H, W = in_dhw
    dy = np.zeros((N, D, H, W, C), np.float64)
    _load().ref_avgpool3d_bwd(_ptr(dp), _ptr(dy), N, D, H, W, C, k, s)
    return dy


# --------------------------------------------------------------------------
# The layer stack: conv -> bias + leaky ReLU -> (optional) 2^3 stride-2 pool,
# composed from the per-layer definitions above in the network's order
# (Section III-A: every conv is followed by leaky ReLU; pooling with stride
# (2,2,2) follows the early convolutions).
# --------------------------------------------------------------------------

def stack_forward(x, layers, weights, biases, alpha):
    """Run the forward chain.  ``layers`` is a list of dicts with keys
    k, stride, pool (bool).  Returns per-layer dict of x, z, y, out."""
    acts = []
    h = _f64(x)
    for L, w, b in zip(layers, weights, biases):
        z = conv3d_fwd(h, w, stride=L["stride"], pad=L.get("pad", "same"))
        y = bias_lrelu_fwd(z, b, alpha)
        out = avgpool3d_fwd(y) if L["pool"] else y
        acts.append(dict(x=h, z=z, y=y, out=out))
        h = out
    return acts


def stack_backward(acts, layers, weights, dout, alpha, skip_first_dgrad=True):
    """Backward chain from the upstream gradient on the last layer's output.
    Returns per-layer dict of dy, dz, db, dw, dx (dx None when skipped)."""
    grads = [None] * len(layers)
    g = _f64(dout)
    for i in range(len(layers) - 1, -1, -1):
        L, w, a = layers[i], weights[i], acts[i]
        dy = avgpool3d_bwd(g, a["y"].shape[1:4]) if L["pool"] else g
        dz, db = bias_lrelu_bwd(dy, a["y"], alpha)
        k = np.asarray(w).shape[:3]
        dw = conv3d_bwd_weight(a["x"], dz, k, stride=L["stride"], pad=L.get("pad", "same"))
        dx = None
        if not (i == 0 and skip_first_dgrad):
            dx = conv3d_bwd_data(dz, w, a["x"].shape[1:4], stride=L["stride"],
                                 pad=L.get("pad", "same"))
        grads[i] = dict(dy=dy, dz=dz, db=db, dw=dw, dx=dx)
        g = dx
    return grads


# ----------------------------------------------------------------------
# Parameter update (Section III-B): Adam + LARC + linear learning-rate decay

#: the paper's hyperparameters (Section III-B); t_decay is not given there
PAPER_HPARAMS = dict(eta0=2e-3, eta_min=1e-4, beta1=0.9, beta2=0.999, eps_hat=1e-8,
                     larc_coef=0.002, larc_fallback=6.25e-5, larc_clip=1.0)


def lr_schedule(t, t_decay, eta0=2e-3, eta_min=1e-4):
    """Global learning rate of step t (linear decay, clamped after t_decay)."""
    return _load().ref_lr_schedule(int(t), int(t_decay), float(eta0), float(eta_min))


def adam_larc_step(offsets, t, t_decay, v, g, m, s, **hp):
    """One update of every group; returns (v, m, s, eta_dagger) as new float64
    arrays.  offsets has ngroups + 1 entries; group l is [offsets[l],
    offsets[l+1]).  hp overrides PAPER_HPARAMS."""
    h = dict(PAPER_HPARAMS)
    h.update(hp)
    off = np.ascontiguousarray(offsets, dtype=np.int64)
    ng = len(off) - 1
    v = _f64(v).copy()
    g = _f64(g)
    m = _f64(m).copy()
    s = _f64(s).copy()
    assert v.shape == g.shape == m.shape == s.shape and v.ndim == 1 and off[-1] <= v.size
    hpa = np.array([h["eta0"], h["eta_min"], h["beta1"], h["beta2"], h["eps_hat"],
                    h["larc_coef"], h["larc_fallback"], h["larc_clip"]], np.float64)
    dag = np.zeros(max(ng, 1), np.float64)
    _load().ref_adam_larc_step(ng, off.ctypes.data_as(ctypes.POINTER(ctypes.c_int64)), int(t), int(t_decay),
                               _ptr(hpa), _ptr(v), _ptr(g), _ptr(m), _ptr(s), _ptr(dag))
    return v, m, s, dag[:ng]


# ----------------------------------------------------------------------
# Fully-connected head and loss (Section III-A: three FC layers, leaky ReLU
# on every layer, three outputs).  x rows are [M][K], W is [K][N].

def fc_fwd(x, w):
    """z = x W for x [M][K] (a batch of flattened feature rows) and W [K][N]."""
    x = _f64(x)
    w = _f64(w)
    M = x.shape[0]
    x = x.reshape(M, -1)
    K, N = w.shape
    assert x.shape[1] == K
    z = np.empty((M, N), np.float64)
    _load().ref_fc_fwd(_ptr(x), _ptr(w), _ptr(z), M, K, N)
    return z


def fc_bwd_data(dz, w):
    """dx = dz W^T, shape [M][K]."""
    dz = _f64(dz)
    w = _f64(w)
    K, N = w.shape
    M = dz.shape[0]
    assert dz.shape == (M, N)
    dx = np.empty((M, K), np.float64)
    _load().ref_fc_bwd_data(_ptr(dz), _ptr(w), _ptr(dx), M, K, N)
    return dx


def fc_bwd_weight(x, dz):
    """dW = x^T dz, shape [K][N]."""
    x = _f64(x)
    dz = _f64(dz)
    M = x.shape[0]
    x = x.reshape(M, -1)
    K = x.shape[1]
    N = dz.shape[1]
    assert dz.shape == (M, N)
    dw = np.empty((K, N), np.float64)
    _load().ref_fc_bwd_weight(_ptr(x), _ptr(dz), _ptr(dw), M, K, N)
    return dw


def mse_loss(p, t):
    """(loss, dL/dp) of the mean squared error over all M x N outputs."""
    p = _f64(p)
    t = _f64(t)
    assert p.shape == t.shape and p.ndim == 2
    dp = np.empty_like(p)
    loss = _load().ref_mse_loss(_ptr(p), _ptr(t), _ptr(dp), p.shape[0], p.shape[1])
    return loss, dp


def head_forward(feat, weights, biases, alpha, target):
    """FC layers (each fc -> bias + leaky ReLU) on feature rows feat [M][K0],
    then the loss against target [M][N_last].  Returns (loss, dL/d(last
    output), acts) with acts a per-layer list of dicts x, z, y."""
    acts = []
    h = _f64(feat).reshape(np.asarray(feat).shape[0], -1)
    for w, b in zip(weights, biases):
        z = fc_fwd(h, w)
        y = bias_lrelu_fwd(z, b, alpha)
        acts.append(dict(x=h, z=z, y=y))
        h = y
    loss, dp = mse_loss(h, target)
    return loss, dp, acts


def head_backward(acts, weights, dp, alpha):
    """Backward through the FC layers from dL/d(last output).  Returns
    (per-layer dicts dz, db, dw, dx; gradient of the feature rows)."""
    grads = [None] * len(acts)
    g = _f64(dp)
    for i in range(len(acts) - 1, -1, -1):
        a = acts[i]
        dz, db = bias_lrelu_bwd(g, a["y"], alpha)
        dw = fc_bwd_weight(a["x"], dz)
        dx = fc_bwd_data(dz, weights[i])
        grads[i] = dict(dz=dz, db=db, dw=dw, dx=dx)
        g = dx
    return grads, g
