"""fp64 oracle primitives: numpy in, numpy out, computed by ``liboracle.so``.

Test infrastructure only (see the package docstring).  Shapes: activations are
NHWC ``[N, H, W, C]`` (or ``[m, C]`` for per-channel ops), conv weights
``[K, K, C_in, C_out]``.
"""
import ctypes
import os

import numpy as np

from . import build as _build

_lib = None
_D = ctypes.POINTER(ctypes.c_double)


def lib():
    global _lib
    if _lib is None:
        path = _build.LIB
        if not os.path.exists(path) or os.path.getmtime(path) < os.path.getmtime(_build.SRC):
            _build.build()
        _lib = ctypes.CDLL(path)
    return _lib


def _f64(a):
    return np.ascontiguousarray(a, dtype=np.float64)


def _p(a):
    return a.ctypes.data_as(_D)


def _out_dim(n, k, s, p):
    return (n + 2 * p - k) // s + 1


# ----------------------------------------------------------------- CONV ----
def conv_fwd(x, wt, stride=1, pad=None):
    x, wt = _f64(x), _f64(wt)
    N, H, W, Ci = x.shape
    K, K2, Ci2, Co = wt.shape
    assert K == K2 and Ci == Ci2
    pad = K // 2 if pad is None else pad
    out = np.empty((N, _out_dim(H, K, stride, pad), _out_dim(W, K, stride, pad), Co))
    lib().orc_conv_fwd(N, H, W, Ci, Co, K, stride, pad, _p(x), _p(wt), _p(out))
    return out


def conv_dgrad(g, wt, in_hw, stride=1, pad=None):
    g, wt = _f64(g), _f64(wt)
    N = g.shape[0]
    K, _, Ci, Co = wt.shape
    H, W = in_hw
    pad = K // 2 if pad is None else pad
    assert g.shape == (N, _out_dim(H, K, stride, pad), _out_dim(W, K, stride, pad), Co)
    din = np.empty((N, H, W, Ci))
    lib().orc_conv_dgrad(N, H, W, Ci, Co, K, stride, pad, _p(g), _p(wt), _p(din))
    return din


def conv_wgrad(x, g, K, stride=1, pad=None):
    x, g = _f64(x), _f64(g)
    N, H, W, Ci = x.shape
    Co = g.shape[3]
    pad = K // 2 if pad is None else pad
    assert g.shape[:3] == (N, _out_dim(H, K, stride, pad), _out_dim(W, K, stride, pad))
    dwt = np.empty((K, K, Ci, Co))
    lib().orc_conv_wgrad(N, H, W, Ci, Co, K, stride, pad, _p(x), _p(g), _p(dwt))
    return dwt


# ------------------------------------------------------------------- BN ----
def bn_fwd(x, gamma, beta, eps):
    """Returns (y, mean, var, rstd); x is [..., C], statistics over all but C."""
    shape = x.shape
    x2 = _f64(x).reshape(-1, shape[-1])
    m, C = x2.shape
    g, b = _f64(gamma), _f64(beta)
    mean, var, rstd, y = np.empty(C), np.empty(C), np.empty(C), np.empty((m, C))
    lib().orc_bn_fwd(ctypes.c_long(m), C, _p(x2), _p(g), _p(b), ctypes.c_double(eps),
                     _p(mean), _p(var), _p(rstd), _p(y))
    return y.reshape(shape), mean, var, rstd


def bn_stats(x, eps):
    _, mean, var, rstd = bn_fwd(x, np.ones(x.shape[-1]), np.zeros(x.shape[-1]), eps)
    return mean, var, rstd


def mvf_stats(x):
    x2 = _f64(x).reshape(-1, x.shape[-1])
    m, C = x2.shape
    mean, var = np.empty(C), np.empty(C)
    lib().orc_mvf_stats(ctypes.c_long(m), C, _p(x2), _p(mean), _p(var))
    return mean, var


def mvf_stats_shifted(x, K):
    """One-sweep statistics around a per-channel shift K: (mean, var)."""
    x2 = _f64(x).reshape(-1, x.shape[-1])
    m, C = x2.shape
    k = np.ascontiguousarray(np.broadcast_to(_f64(K), (C,)))
    mean, var = np.empty(C), np.empty(C)
    lib().orc_mvf_stats_shifted(ctypes.c_long(m), C, _p(x2), _p(k), _p(mean), _p(var))
    return mean, var


def running_update(rmean, rvar, mean, var, m, momentum):
    """Exponential moving average of the batch statistics (unbiased variance); returns new arrays."""
    C = len(mean)
    rm, rv = _f64(rmean).copy(), _f64(rvar).copy()
    lib().orc_running_update(C, ctypes.c_long(m), ctypes.c_double(momentum), _p(_f64(mean)), _p(_f64(var)),
                             _p(rm), _p(rv))
    return rm, rv


def bn_bwd(x, dy, gamma, mean, rstd, want_dx=True):
    """Returns (dx or None, dgamma, dbeta)."""
    shape = x.shape
    x2 = _f64(x).reshape(-1, shape[-1])
    dy2 = _f64(dy).reshape(-1, shape[-1])
    m, C = x2.shape
    dg, db = np.empty(C), np.empty(C)
    dx = np.empty((m, C)) if want_dx else None
    lib().orc_bn_bwd(ctypes.c_long(m), C, _p(x2), _p(dy2), _p(_f64(gamma)), _p(_f64(mean)),
                     _p(_f64(rstd)), _p(dg), _p(db), _p(dx) if want_dx else None)
    return (dx.reshape(shape) if want_dx else None), dg, db


# ----------------------------------------------------------------- ReLU ----
def relu_fwd(y):
    y = _f64(y)
    z = np.empty_like(y)
    lib().orc_relu_fwd(ctypes.c_long(y.size), _p(y), _p(z))
    return z


def relu_bwd(dz, y):
    dz, y = _f64(dz), _f64(y)
    dy = np.empty_like(dz)
    lib().orc_relu_bwd(ctypes.c_long(dz.size), _p(dz), _p(y), _p(dy))
    return dy


# -------------------------------------------------------------- pooling ----
def avgpool2_fwd(x):
    x = _f64(x)
    N, H, W, C = x.shape
    out = np.empty((N, H // 2, W // 2, C))
    lib().orc_avgpool2_fwd(N, H, W, C, _p(x), _p(out))
    return out


def avgpool2_bwd(gout, in_hw):
    gout = _f64(gout)
    N, _, _, C = gout.shape
    H, W = in_hw
    gin = np.empty((N, H, W, C))
    lib().orc_avgpool2_bwd(N, H, W, C, _p(gout), _p(gin))
    return gin


def maxpool_fwd(x, K=3, stride=2, pad=1):
    x = _f64(x)
    N, H, W, C = x.shape
    out = np.empty((N, _out_dim(H, K, stride, pad), _out_dim(W, K, stride, pad), C))
    lib().orc_maxpool_fwd(N, H, W, C, K, stride, pad, _p(x), _p(out))
    return out


def maxpool_bwd(x, gout, K=3, stride=2, pad=1):
    x, gout = _f64(x), _f64(gout)
    N, H, W, C = x.shape
    gin = np.empty_like(x)
    lib().orc_maxpool_bwd(N, H, W, C, K, stride, pad, _p(x), _p(gout), _p(gin))
    return gin


# ------------------------------------------------------------- storage ----
def round_bf16(a):
    """Nearest bf16 value of every element (ties to even), as fp64."""
    a = np.array(a, dtype=np.float64, copy=True)
    lib().orc_round_bf16(ctypes.c_long(a.size), _p(a))
    return a


# ------------------------------------------------------- network head ----
# The paper names the network's single fully connected layer (Sec. 2.2: 120
# CONV layers plus one FC layer) but gives no equations for the head; these
# are the standard classifier: global average pooling, an affine layer and
# the softmax cross-entropy averaged over the mini-batch.  numpy fp64.
def global_avgpool_fwd(x):
    """[N, H, W, C] -> [N, C]: mean over the H*W positions of each image."""
    x = _f64(x)
    return x.sum(axis=(1, 2)) / (x.shape[1] * x.shape[2])


def global_avgpool_bwd(gout, hw):
    """Every position of image n receives gout[n, c] / (H*W)."""
    gout = _f64(gout)
    H, W = hw
    return np.broadcast_to((gout / (H * W))[:, None, None, :], (gout.shape[0], H, W, gout.shape[1])).copy()


def fc_fwd(f, wt, bias):
    """logits[n, j] = sum_c f[n, c] * wt[c, j] + bias[j]."""
    return _f64(f) @ _f64(wt) + _f64(bias)[None, :]


def fc_bwd(f, wt, glogits):
    """(df, dwt, dbias) of L = sum(logits * glogits)."""
    f, wt, gl = _f64(f), _f64(wt), _f64(glogits)
    return gl @ wt.T, f.T @ gl, gl.sum(axis=0)


def softmax_ce(logits, labels):
    """Mean over the batch of -log softmax(logits)[n, label[n]], and its
    gradient with respect to the logits: (softmax - onehot) / N."""
    z = _f64(logits)
    N, K = z.shape
    lab = np.asarray(labels, dtype=np.int64)
    s = z - z.max(axis=1, keepdims=True)
    lse = np.log(np.exp(s).sum(axis=1))
    loss = float(np.mean(lse - s[np.arange(N), lab]))
    p = np.exp(s - lse[:, None])
    p[np.arange(N), lab] -= 1.0
    return loss, p / N
