"""Thin ctypes binding of ``libbnr.so`` (C ABI in ``include/bnr.h``).

Argument marshalling only: tensors are torch device tensors (PyTorch supplies
device memory and the current stream); every step of the computation runs in
the library's HIP kernels.  There is no fallback: if ``libbnr.so`` is missing
or fails to load, importing this module raises.

Tensor views.  A view argument is a torch tensor whose last dimension holds
the channels with unit stride and whose leading dimensions collapse to one
pixel stride (e.g. ``buf[..., c0:c0 + c]`` of a contiguous NHWC buffer): the
binding passes its data pointer and that pixel stride (``ldc``).
"""
import ctypes
import os

import torch

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libbnr.so")

if not os.path.exists(LIB_PATH):
    raise ImportError("libbnr.so is not built (run __graft_entry__.build())")
_lib = ctypes.CDLL(LIB_PATH)

BNR_F32, BNR_BF16 = 0, 1
GRAD_DENSE, GRAD_BN, GRAD_AVGPOOL2, GRAD_SPLIT = 0, 1, 2, 3
MODE_BASELINE, MODE_RCF, MODE_RCF_MVF = 0, 1, 2
STATUS = ["BNR_OK", "BNR_ERR_NULL", "BNR_ERR_SHAPE", "BNR_ERR_DTYPE", "BNR_ERR_ALIGN", "BNR_ERR_WORKSPACE",
          "BNR_ERR_UNSUPPORTED", "BNR_ERR_HIP", "BNR_ERR_ALIAS"]

c_i32, c_i64, c_vp, c_sz, c_f = ctypes.c_int32, ctypes.c_int64, ctypes.c_void_p, ctypes.c_size_t, ctypes.c_float


class ConvDesc(ctypes.Structure):
    _fields_ = [("n", c_i32), ("h", c_i32), ("w", c_i32), ("c_in", c_i32), ("c_out", c_i32), ("k", c_i32),
                ("in_ldc", c_i32), ("out_ldc", c_i32), ("dtype", ctypes.c_int)]


class BNStruct(ctypes.Structure):
    _fields_ = [("gamma", c_vp), ("beta", c_vp), ("mean", c_vp), ("var", c_vp), ("rstd", c_vp), ("eps", c_f),
                ("shift", c_vp), ("running_mean", c_vp), ("running_var", c_vp), ("momentum", c_f),
                ("mean_lo", c_vp)]


class GradSrc(ctypes.Structure):
    _fields_ = [("kind", ctypes.c_int), ("g", c_vp), ("g_ldc", c_i32), ("dy", c_vp), ("x", c_vp), ("x_ldc", c_i32),
                ("bn", ctypes.POINTER(BNStruct)), ("dgamma", c_vp), ("dbeta", c_vp), ("alpha", c_vp), ("betap", c_vp)]


class BnReluRefArgs(ctypes.Structure):
    _fields_ = [("x", c_vp), ("x_ldc", c_i32), ("bn", ctypes.POINTER(BNStruct)), ("y", c_vp), ("z", c_vp),
                ("gz", c_vp), ("gz_ldc", c_i32), ("dy", c_vp), ("dgamma", c_vp), ("dbeta", c_vp), ("dx", c_vp),
                ("dx_ldc", c_i32)]


class StemDesc(ctypes.Structure):
    _fields_ = [("n", c_i32), ("h", c_i32), ("w", c_i32), ("c_in", c_i32), ("dtype", ctypes.c_int)]


class RefArgs(ctypes.Structure):
    _fields_ = [("x", c_vp), ("bn", ctypes.POINTER(BNStruct)), ("w", c_vp), ("y", c_vp), ("z", c_vp), ("out", c_vp),
                ("g", c_vp), ("g_ldc", c_i32), ("dz", c_vp), ("dy", c_vp), ("dw", c_vp), ("dgamma", c_vp),
                ("dbeta", c_vp), ("dx", c_vp), ("dx_ldc", c_i32), ("dx_accumulate", c_i32)]


class AddReluRefArgs(ctypes.Structure):
    _fields_ = [("y", c_vp), ("y_ldc", c_i32), ("bn", ctypes.POINTER(BNStruct)), ("id", c_vp), ("id_ldc", c_i32),
                ("out", c_vp), ("out_ldc", c_i32), ("tmp", c_vp), ("g", c_vp), ("g_ldc", c_i32), ("gm", c_vp),
                ("dgamma", c_vp), ("dbeta", c_vp), ("dx", c_vp), ("dx_ldc", c_i32)]


def _sig(name, res, *args):
    f = getattr(_lib, name)
    f.restype = res
    f.argtypes = list(args)
    return f


_P = ctypes.POINTER
_lib_fns = dict(
    bnr_status_string=_sig("bnr_status_string", ctypes.c_char_p, ctypes.c_int),
    bnr_last_error=_sig("bnr_last_error", ctypes.c_char_p),
    bnr_stats_workspace_size=_sig("bnr_stats_workspace_size", c_sz, c_i64, c_i32),
    bnr_workspace_size=_sig("bnr_workspace_size", c_sz, _P(ConvDesc)),
    bnr_bn_stats=_sig("bnr_bn_stats", ctypes.c_int, c_i64, c_i32, c_i32, ctypes.c_int, c_vp, _P(BNStruct), c_vp, c_sz,
                      c_vp),
    bnr_conv_bn_stats_fwd=_sig("bnr_conv_bn_stats_fwd", ctypes.c_int, _P(ConvDesc), c_vp, c_vp, c_vp, _P(BNStruct),
                               c_vp, c_sz, c_vp),
    bnr_bn_relu_conv_fwd=_sig("bnr_bn_relu_conv_fwd", ctypes.c_int, _P(ConvDesc), c_vp, _P(BNStruct), c_vp, c_vp,
                              _P(BNStruct), c_vp, c_sz, c_vp),
    bnr_bn_add_relu_conv_fwd=_sig("bnr_bn_add_relu_conv_fwd", ctypes.c_int, _P(ConvDesc), c_vp, _P(BNStruct), c_vp,
                                  c_i32, c_vp, c_i32, c_vp, c_vp, _P(BNStruct), c_vp, c_sz, c_vp),
    bnr_bn_relu_conv_pool_fwd=_sig("bnr_bn_relu_conv_pool_fwd", ctypes.c_int, _P(ConvDesc), c_vp, _P(BNStruct), c_vp,
                                   c_vp, _P(BNStruct), c_vp, c_sz, c_vp),
    bnr_bn_relu_conv_fwd_o2=_sig("bnr_bn_relu_conv_fwd_o2", ctypes.c_int, _P(ConvDesc), c_vp, _P(BNStruct), c_vp,
                                 c_vp, _P(BNStruct), c_vp, c_i32, c_vp, c_sz, c_vp),
    bnr_bwd_fused_o2=_sig("bnr_bwd_fused_o2", ctypes.c_int, _P(ConvDesc), c_vp, _P(BNStruct), c_vp, c_i32, c_vp,
                          _P(GradSrc), c_vp, c_vp, c_vp, c_vp, c_vp, c_i32, c_i32, c_vp, c_sz, c_vp),
    bnr_bn_relu_conv_fwd_static=_sig("bnr_bn_relu_conv_fwd_static", ctypes.c_int, _P(ConvDesc), c_vp, _P(BNStruct),
                                     c_vp, c_vp, _P(BNStruct), c_vp),
    bnr_avgpool2_fwd=_sig("bnr_avgpool2_fwd", ctypes.c_int, c_i32, c_i32, c_i32, c_i32, ctypes.c_int, c_vp, c_i32,
                          c_vp, c_i32, c_vp),
    bnr_avgpool2_bwd=_sig("bnr_avgpool2_bwd", ctypes.c_int, c_i32, c_i32, c_i32, c_i32, ctypes.c_int, c_vp, c_i32,
                          c_vp, c_i32, c_vp),
    bnr_bwd_fused=_sig("bnr_bwd_fused", ctypes.c_int, _P(ConvDesc), c_vp, _P(BNStruct), c_vp, _P(GradSrc), c_vp,
                       c_vp, c_vp, c_vp, c_vp, c_i32, c_i32, c_vp, c_sz, c_vp),
    bnr_bwd_fused_split=_sig("bnr_bwd_fused_split", ctypes.c_int, _P(ConvDesc), c_vp, _P(BNStruct), c_vp,
                             _P(GradSrc), c_vp, c_vp, c_vp, c_vp, c_i32, c_i32, c_vp, c_vp, c_vp, c_sz, c_vp),
    bnr_bwd_data=_sig("bnr_bwd_data", ctypes.c_int, _P(ConvDesc), c_vp, _P(BNStruct), c_vp, _P(GradSrc), c_vp, c_vp,
                      c_vp, c_vp, c_i32, c_i32, c_vp, c_sz, c_vp),
    bnr_bwd_data_split=_sig("bnr_bwd_data_split", ctypes.c_int, _P(ConvDesc), c_vp, _P(BNStruct), c_vp, _P(GradSrc),
                            c_vp, c_vp, c_vp, c_i32, c_i32, c_vp, c_vp, c_vp, c_sz, c_vp),
    bnr_bwd_weights=_sig("bnr_bwd_weights", ctypes.c_int, _P(ConvDesc), c_vp, _P(BNStruct), _P(GradSrc), c_vp, c_vp,
                         c_sz, c_vp),
    bnr_split_dx=_sig("bnr_split_dx", ctypes.c_int, c_i64, c_i32, ctypes.c_int, c_vp, c_i32, c_vp, c_i32,
                      _P(BNStruct), c_vp, c_vp, c_vp, c_i32, c_i32, c_vp),
    bnr_bn_dx=_sig("bnr_bn_dx", ctypes.c_int, c_i64, c_i32, ctypes.c_int, c_vp, c_vp, c_i32, _P(BNStruct), c_vp, c_vp,
                   c_vp, c_i32, c_i32, c_vp),
    bnr_reference_path=_sig("bnr_reference_path", ctypes.c_int, ctypes.c_int, c_i32, _P(ConvDesc), _P(RefArgs), c_vp,
                            c_sz, c_vp),
    bnr_hbm_copy=_sig("bnr_hbm_copy", ctypes.c_int, c_vp, c_vp, c_sz, c_vp),
    bnr_conv_fwd=_sig("bnr_conv_fwd", ctypes.c_int, _P(ConvDesc), c_vp, c_vp, c_vp, c_vp, c_sz, c_vp),
    bnr_bn_add_relu_fwd=_sig("bnr_bn_add_relu_fwd", ctypes.c_int, c_i64, c_i32, ctypes.c_int, c_vp, c_i32,
                             _P(BNStruct), c_vp, c_i32, c_vp, c_i32, c_vp),
    bnr_bn_add_relu_bwd=_sig("bnr_bn_add_relu_bwd", ctypes.c_int, c_i64, c_i32, ctypes.c_int, c_vp, c_i32, c_vp, c_i32,
                             c_vp, c_i32, _P(BNStruct), c_vp, c_i32, c_vp, c_vp, c_vp, c_sz, c_vp),
    bnr_reference_bn_add_relu=_sig("bnr_reference_bn_add_relu", ctypes.c_int, c_i32, c_i64, c_i32, ctypes.c_int,
                                   _P(AddReluRefArgs), c_vp, c_sz, c_vp),
    bnr_reference_bn_relu=_sig("bnr_reference_bn_relu", ctypes.c_int, c_i32, c_i64, c_i32, ctypes.c_int,
                               _P(BnReluRefArgs), c_vp, c_sz, c_vp),
    bnr_stem_workspace_size=_sig("bnr_stem_workspace_size", c_sz, _P(StemDesc)),
    bnr_stem_conv_fwd=_sig("bnr_stem_conv_fwd", ctypes.c_int, _P(StemDesc), c_vp, c_vp, c_vp, _P(BNStruct), c_vp,
                           c_sz, c_vp),
    bnr_stem_wgrad=_sig("bnr_stem_wgrad", ctypes.c_int, _P(StemDesc), c_vp, _P(GradSrc), c_vp, c_vp, c_sz, c_vp),
    bnr_pool_workspace_size=_sig("bnr_pool_workspace_size", c_sz, c_i32, c_i32, c_i32, c_i32),
    bnr_bn_relu_maxpool_fwd=_sig("bnr_bn_relu_maxpool_fwd", ctypes.c_int, c_i32, c_i32, c_i32, c_i32, ctypes.c_int,
                                 c_vp, c_i32, _P(BNStruct), c_vp, c_i32, _P(BNStruct), c_vp, c_sz, c_vp),
    bnr_maxpool_bn_bwd=_sig("bnr_maxpool_bn_bwd", ctypes.c_int, c_i32, c_i32, c_i32, c_i32, ctypes.c_int, c_vp, c_i32,
                            _P(BNStruct), c_vp, c_i32, c_vp, c_vp, c_vp, c_vp, c_sz, c_vp),
    bnr_head_workspace_size=_sig("bnr_head_workspace_size", c_sz, c_i32, c_i32, c_i32, c_i32),
    bnr_head_fwd=_sig("bnr_head_fwd", ctypes.c_int, c_i32, c_i32, c_i32, c_i32, c_i32, ctypes.c_int, c_vp, c_i32,
                      _P(BNStruct), c_vp, c_vp, c_vp, c_vp, c_vp, c_vp, c_vp, c_vp),
    bnr_head_bwd=_sig("bnr_head_bwd", ctypes.c_int, c_i32, c_i32, c_i32, c_i32, c_i32, ctypes.c_int, c_vp, c_i32,
                      _P(BNStruct), c_vp, c_vp, c_vp, c_vp, c_vp, c_vp, c_vp, c_vp, c_vp, c_i32, c_vp, c_vp, c_vp,
                      c_sz, c_vp),
    bnr_trace_begin=_sig("bnr_trace_begin", ctypes.c_int, c_i32, c_i32),
    bnr_trace_end=_sig("bnr_trace_end", c_i32, ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_double),
                       ctypes.POINTER(ctypes.c_double), ctypes.POINTER(c_i32), c_i32),
)

KERNEL_IDS = {1: "conv1x1", 2: "conv3x3", 3: "wgrad1x1", 4: "wgrad3x3", 5: "stats_sweep", 6: "elementwise",
              7: "stats_combine", 8: "weight_pack", 9: "splitk_sum", 10: "pool", 11: "copy", 12: "stem_conv",
              13: "stem_wgrad", 14: "maxpool", 15: "head"}


class BnrError(RuntimeError):
    def __init__(self, status, msg):
        super().__init__("%s: %s" % (STATUS[status] if 0 <= status < len(STATUS) else status, msg))
        self.status = status


def _check(status):
    if status != 0:
        raise BnrError(status, _lib_fns["bnr_last_error"]().decode())


def status_string(s):
    return _lib_fns["bnr_status_string"](s).decode()


# --------------------------------------------------------------- helpers ----
def dtype_code(t):
    if t.dtype == torch.bfloat16:
        return BNR_BF16
    if t.dtype == torch.float32:
        return BNR_F32
    raise TypeError("unsupported dtype %s" % t.dtype)


def view(t):
    """(data pointer, pixels, channels, pixel stride) of a channel view."""
    if t.dim() < 2 or t.stride(-1) != 1:
        raise ValueError("view needs a unit-stride channel dimension")
    ldc = t.stride(-2)
    for i in range(t.dim() - 2):
        if t.shape[i] > 1 and t.stride(i) != t.stride(i + 1) * t.shape[i + 1]:
            raise ValueError("leading dimensions of a view must collapse to one pixel stride")
    m = 1
    for s in t.shape[:-1]:
        m *= s
    return t.data_ptr(), m, t.shape[-1], ldc


def _ptr(t):
    return None if t is None else t.data_ptr()


def _stream():
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


_ws_cache = {}


def workspace(nbytes, device=None, slot=0):
    """Grow-only per-device workspace (device memory from torch); calls that
    may be in flight at the same time (on different streams) use different
    slots."""
    dev = torch.device(device) if device is not None else torch.device("cuda", torch.cuda.current_device())
    cur = _ws_cache.get((dev, slot))
    if cur is None or cur.numel() < nbytes:
        cur = torch.empty(max(int(nbytes), 256) + 256, dtype=torch.uint8, device=dev)
        _ws_cache[(dev, slot)] = cur
    base = cur.data_ptr()
    aligned = (base + 255) // 256 * 256
    return aligned, cur.numel() - (aligned - base)


class BN:
    """Per-channel BN state: gamma, beta (inputs), mean, var, rstd (batch statistics), eps.

    Optional robust one-sweep statistics: ``shift`` (per-channel K: the
    one-sweep producers sum x - K and (x - K)^2) and running statistics
    (``running_mean``, ``running_var``, ``momentum``) updated by the producer;
    set them with :meth:`robust`, which also allocates ``mean_lo`` (the low
    part of the float64 mean, written by the producers; float32 consumers
    normalise (x - mean) - mean_lo with it)."""

    shift = running_mean = running_var = mean_lo = None
    momentum = 0.0

    def __init__(self, gamma, beta, eps=1e-5, mean=None, var=None, rstd=None):
        dev, c = gamma.device, gamma.shape[0]
        self.gamma, self.beta, self.eps = gamma, beta, float(eps)
        self.mean = mean if mean is not None else torch.empty(c, dtype=torch.float32, device=dev)
        self.var = var if var is not None else torch.empty(c, dtype=torch.float32, device=dev)
        self.rstd = rstd if rstd is not None else torch.empty(c, dtype=torch.float32, device=dev)

    def robust(self, shift=None, running_mean=None, running_var=None, momentum=0.1):
        """Sum around shift (may be running_mean itself) and/or update running statistics; returns self."""
        self.shift, self.running_mean, self.running_var = shift, running_mean, running_var
        self.momentum = float(momentum)
        self.mean_lo = torch.empty_like(self.mean)
        return self

    @classmethod
    def stats_only(cls, c, device, eps=1e-5):
        """Statistics holder for a BN whose gamma/beta are not needed (producer side)."""
        b = cls.__new__(cls)
        b.gamma = b.beta = None
        b.eps = float(eps)
        b.mean = torch.empty(c, dtype=torch.float32, device=device)
        b.var = torch.empty(c, dtype=torch.float32, device=device)
        b.rstd = torch.empty(c, dtype=torch.float32, device=device)
        return b

    @classmethod
    def stats_view(cls, eps, mean, var, rstd):
        """Statistics holder on caller-provided arrays (e.g. channel slices of
        per-channel arrays shared by several BN layers)."""
        b = cls.__new__(cls)
        b.gamma = b.beta = None
        b.eps = float(eps)
        b.mean, b.var, b.rstd = mean, var, rstd
        return b

    def struct(self):
        return BNStruct(_ptr(self.gamma), _ptr(self.beta), _ptr(self.mean), _ptr(self.var), _ptr(self.rstd),
                        self.eps, _ptr(self.shift), _ptr(self.running_mean), _ptr(self.running_var),
                        self.momentum, _ptr(self.mean_lo))


def conv_desc(n, h, w, c_in, c_out, k, in_ldc, out_ldc, dtype):
    return ConvDesc(n, h, w, c_in, c_out, k, in_ldc, out_ldc, dtype)


def desc_for(x, y, k, n, h, w):
    """Descriptor of a CONV from view x ([.., c_in]) to view y ([.., c_out])."""
    _, mx, ci, ldx = view(x)
    _, my, co, ldy = view(y)
    assert mx == my == n * h * w, (mx, my, n, h, w)
    return ConvDesc(n, h, w, ci, co, k, ldx, ldy, dtype_code(x))


# ----------------------------------------------------------- entry points --
def bnr_workspace_size(desc):
    return _lib_fns["bnr_workspace_size"](ctypes.byref(desc))


def bnr_stats_workspace_size(m, c):
    return _lib_fns["bnr_stats_workspace_size"](m, c)


def bnr_bn_stats(x, bn):
    """Standalone sub-BN1: batch statistics of the view x into bn."""
    p, m, c, ldc = view(x)
    ws, wsb = workspace(bnr_stats_workspace_size(m, c), x.device)
    s = bn.struct()
    _check(_lib_fns["bnr_bn_stats"](m, c, ldc, dtype_code(x), p, ctypes.byref(s), ws, wsb, _stream()))


def bnr_conv_bn_stats_fwd(desc, x, w, y, y_bn):
    ws, wsb = workspace(bnr_workspace_size(desc), x.device)
    ys = y_bn.struct()
    _check(_lib_fns["bnr_conv_bn_stats_fwd"](ctypes.byref(desc), _ptr(x), _ptr(w), _ptr(y), ctypes.byref(ys), ws, wsb,
                                             _stream()))


def bnr_bn_relu_conv_fwd(desc, x, x_bn, w, y, y_bn=None):
    ws, wsb = workspace(bnr_workspace_size(desc), x.device)
    xs = x_bn.struct()
    ys = y_bn.struct() if y_bn is not None else None
    _check(_lib_fns["bnr_bn_relu_conv_fwd"](ctypes.byref(desc), _ptr(x), ctypes.byref(xs), _ptr(w), _ptr(y),
                                            ctypes.byref(ys) if ys is not None else None, ws, wsb, _stream()))


def bnr_bn_add_relu_conv_fwd(desc, y, y_bn, ident, r, w, out, out_bn=None):
    """r = relu(bn(y) + ident) (written), out = conv1x1(r) [+ statistics of out]."""
    ws, wsb = workspace(bnr_workspace_size(desc), y.device)
    pi, _, _, ldi = view(ident)
    pr, _, _, ldr = view(r)
    ys = y_bn.struct()
    os_ = out_bn.struct() if out_bn is not None else None
    _check(_lib_fns["bnr_bn_add_relu_conv_fwd"](ctypes.byref(desc), _ptr(y), ctypes.byref(ys), pi, ldi, pr, ldr,
                                                _ptr(w), _ptr(out), ctypes.byref(os_) if os_ is not None else None,
                                                ws, wsb, _stream()))


def bnr_bn_relu_conv_pool_fwd(desc, x, x_bn, w, y, y_bn=None):
    """Transition layer: y (pooled view) = avgpool2x2(conv1x1(relu(bn(x)))), pooled before the CONV."""
    ws, wsb = workspace(bnr_workspace_size(desc), x.device)
    xs = x_bn.struct()
    ys = y_bn.struct() if y_bn is not None else None
    _check(_lib_fns["bnr_bn_relu_conv_pool_fwd"](ctypes.byref(desc), _ptr(x), ctypes.byref(xs), _ptr(w), _ptr(y),
                                                 ctypes.byref(ys) if ys is not None else None, ws, wsb, _stream()))


def bnr_bn_relu_conv_fwd_o2(desc, x, x_bn, w, y, z, y_bn=None):
    """bnr_bn_relu_conv_fwd that also writes z = relu(bn(x)) (the O2' sweep) to the view z."""
    ws, wsb = workspace(bnr_workspace_size(desc), x.device)
    xs = x_bn.struct()
    ys = y_bn.struct() if y_bn is not None else None
    pz, _, _, ldz = view(z)
    _check(_lib_fns["bnr_bn_relu_conv_fwd_o2"](ctypes.byref(desc), _ptr(x), ctypes.byref(xs), _ptr(w), _ptr(y),
                                               ctypes.byref(ys) if ys is not None else None, pz, ldz, ws, wsb,
                                               _stream()))


def bnr_bn_relu_conv_fwd_static(desc, x, x_bn, w, y, y_bn=None):
    """bnr_bn_relu_conv_fwd on the library's static per-GPU scratch (no workspace, no allocation)."""
    xs = x_bn.struct()
    ys = y_bn.struct() if y_bn is not None else None
    _check(_lib_fns["bnr_bn_relu_conv_fwd_static"](ctypes.byref(desc), _ptr(x), ctypes.byref(xs), _ptr(w), _ptr(y),
                                                   ctypes.byref(ys) if ys is not None else None, _stream()))


def bnr_avgpool2_fwd(x, y, n, h, w):
    p, m, c, ldc = view(x)
    py, _, _, ldy = view(y)
    _check(_lib_fns["bnr_avgpool2_fwd"](n, h, w, c, dtype_code(x), p, ldc, py, ldy, _stream()))


def bnr_avgpool2_bwd(g, gx, n, h, w):
    pd, _, c, ldc = view(gx)
    pg, _, _, ldg = view(g)
    _check(_lib_fns["bnr_avgpool2_bwd"](n, h, w, c, dtype_code(gx), pg, ldg, pd, ldc, _stream()))


def grad_dense(g):
    p, _, _, ldc = view(g)
    return dict(kind=GRAD_DENSE, g=p, g_ldc=ldc, keep=(g,))


def grad_avgpool2(gp):
    p, _, _, ldc = view(gp)
    return dict(kind=GRAD_AVGPOOL2, g=p, g_ldc=ldc, keep=(gp,))


def grad_bn(dy, x, bn, dgamma, dbeta):
    """Deferred gradient of a CONV output x that feeds BN `bn` (dy dense)."""
    px, _, _, ldx = view(x)
    return dict(kind=GRAD_BN, dy=_ptr(dy), x=px, x_ldc=ldx, bn=bn, dgamma=_ptr(dgamma), dbeta=_ptr(dbeta),
                keep=(dy, x, dgamma, dbeta))


def grad_split(gsum, x, bn, alpha, betap):
    """Summed gradient of a concatenation slice x read by several BNs with the
    statistics in bn: g = gsum + alpha + betap * (x - mean) * rstd."""
    pg, _, _, ldg = view(gsum)
    px, _, _, ldx = view(x)
    return dict(kind=GRAD_SPLIT, g=pg, g_ldc=ldg, x=px, x_ldc=ldx, bn=bn, alpha=_ptr(alpha), betap=_ptr(betap),
                keep=(gsum, x, alpha, betap))


def _grad_struct(g):
    bns = g["bn"].struct() if g.get("bn") is not None else None
    gs = GradSrc(g["kind"], g.get("g"), g.get("g_ldc", 0), g.get("dy"), g.get("x"), g.get("x_ldc", 0),
                 ctypes.pointer(bns) if bns is not None else None, g.get("dgamma"), g.get("dbeta"), g.get("alpha"),
                 g.get("betap"))
    return gs, bns


def bnr_bwd_fused(desc, x, x_bn, w, g_src, dw, dgamma=None, dbeta=None, dy=None, dx=None, dx_accumulate=False):
    ws, wsb = workspace(bnr_workspace_size(desc), x.device)
    gs, keep = _grad_struct(g_src)
    xs = x_bn.struct() if x_bn is not None else None
    dxp, dx_ldc = (None, 0)
    if dx is not None:
        dxp, _, _, dx_ldc = view(dx)
    _check(_lib_fns["bnr_bwd_fused"](ctypes.byref(desc), _ptr(x), ctypes.byref(xs) if xs is not None else None,
                                     _ptr(w), ctypes.byref(gs), _ptr(dw), _ptr(dgamma), _ptr(dbeta), _ptr(dy), dxp,
                                     dx_ldc, 1 if dx_accumulate else 0, ws, wsb, _stream()))
    del keep


def bnr_bwd_fused_o2(desc, x, x_bn, z, w, g_src, dw, dgamma, dbeta, dy, dx=None, dx_accumulate=False):
    """bnr_bwd_fused reading the forward's stored z (O2') instead of recomputing it from x."""
    ws, wsb = workspace(bnr_workspace_size(desc), x.device)
    gs, keep = _grad_struct(g_src)
    xs = x_bn.struct()
    pz, _, _, ldz = view(z)
    dxp, dx_ldc = (None, 0)
    if dx is not None:
        dxp, _, _, dx_ldc = view(dx)
    _check(_lib_fns["bnr_bwd_fused_o2"](ctypes.byref(desc), _ptr(x), ctypes.byref(xs), pz, ldz, _ptr(w),
                                        ctypes.byref(gs), _ptr(dw), _ptr(dgamma), _ptr(dbeta), _ptr(dy), dxp, dx_ldc,
                                        1 if dx_accumulate else 0, ws, wsb, _stream()))
    del keep


def bnr_bwd_fused_split(desc, x, x_bn, w, g_src, dw, dgamma, dbeta, gsum, alpha, betap, accumulate=False):
    """bnr_bwd_fused for a concatenation-slice BN input: gamma*rstd*dy goes to
    (or is added into) the view gsum and the combine writes (adds) alpha, betap."""
    ws, wsb = workspace(bnr_workspace_size(desc), x.device)
    gs, keep = _grad_struct(g_src)
    xs = x_bn.struct()
    pg, _, _, ldg = view(gsum)
    _check(_lib_fns["bnr_bwd_fused_split"](ctypes.byref(desc), _ptr(x), ctypes.byref(xs), _ptr(w), ctypes.byref(gs),
                                           _ptr(dw), _ptr(dgamma), _ptr(dbeta), pg, ldg, 1 if accumulate else 0,
                                           _ptr(alpha), _ptr(betap), ws, wsb, _stream()))
    del keep


def bnr_bwd_data(desc, x, x_bn, w, g_src, dgamma=None, dbeta=None, dy=None, dx=None, dx_accumulate=False, slot=0):
    """Steps 1-2 (and the optional dx) of bnr_bwd_fused."""
    ws, wsb = workspace(bnr_workspace_size(desc), x.device, slot)
    gs, keep = _grad_struct(g_src)
    xs = x_bn.struct() if x_bn is not None else None
    dxp, dx_ldc = (None, 0)
    if dx is not None:
        dxp, _, _, dx_ldc = view(dx)
    _check(_lib_fns["bnr_bwd_data"](ctypes.byref(desc), _ptr(x), ctypes.byref(xs) if xs is not None else None,
                                    _ptr(w), ctypes.byref(gs), _ptr(dgamma), _ptr(dbeta), _ptr(dy), dxp, dx_ldc,
                                    1 if dx_accumulate else 0, ws, wsb, _stream()))
    del keep


def bnr_bwd_data_split(desc, x, x_bn, w, g_src, dgamma, dbeta, gsum, alpha, betap, accumulate=False, slot=0):
    """Steps 1-2 of bnr_bwd_fused_split."""
    ws, wsb = workspace(bnr_workspace_size(desc), x.device, slot)
    gs, keep = _grad_struct(g_src)
    xs = x_bn.struct()
    pg, _, _, ldg = view(gsum)
    _check(_lib_fns["bnr_bwd_data_split"](ctypes.byref(desc), _ptr(x), ctypes.byref(xs), _ptr(w), ctypes.byref(gs),
                                          _ptr(dgamma), _ptr(dbeta), pg, ldg, 1 if accumulate else 0, _ptr(alpha),
                                          _ptr(betap), ws, wsb, _stream()))
    del keep


def bnr_bwd_weights(desc, x, x_bn, g_src, dw, slot=0):
    """Step 3 of the fused backward: the weight gradient alone."""
    ws, wsb = workspace(bnr_workspace_size(desc), x.device, slot)
    gs, keep = _grad_struct(g_src)
    xs = x_bn.struct() if x_bn is not None else None
    _check(_lib_fns["bnr_bwd_weights"](ctypes.byref(desc), _ptr(x), ctypes.byref(xs) if xs is not None else None,
                                       ctypes.byref(gs), _ptr(dw), ws, wsb, _stream()))
    del keep


def bnr_split_dx(gsum, x, bn, alpha, betap, dx, dx_accumulate=False):
    """dx = gsum + alpha + betap * (x - mean) * rstd (views [.., c])."""
    pg, m, c, ldg = view(gsum)
    px, _, _, ldx = view(x)
    pd, _, _, ldd = view(dx)
    bs = bn.struct()
    _check(_lib_fns["bnr_split_dx"](m, c, dtype_code(x), pg, ldg, px, ldx, ctypes.byref(bs), _ptr(alpha), _ptr(betap),
                                    pd, ldd, 1 if dx_accumulate else 0, _stream()))


def bnr_bn_dx(dy, x, bn, dgamma, dbeta, dx, dx_accumulate=False):
    px, m, c, ldx = view(x)
    pd, _, _, ldd = view(dx)
    bs = bn.struct()
    _check(_lib_fns["bnr_bn_dx"](m, c, dtype_code(x), _ptr(dy), px, ldx, ctypes.byref(bs), _ptr(dgamma), _ptr(dbeta),
                                 pd, ldd, 1 if dx_accumulate else 0, _stream()))


def bnr_reference_path(mode, backward, desc, x, bn, w, y, z=None, out=None, g=None, dz=None, dy=None, dw=None,
                       dgamma=None, dbeta=None, dx=None, dx_accumulate=False):
    ws, wsb = workspace(bnr_workspace_size(desc), x.device)
    bs = bn.struct()
    g_ldc = view(g)[3] if g is not None else 0
    dxp, dx_ldc = (None, 0)
    if dx is not None:
        dxp, _, _, dx_ldc = view(dx)
    a = RefArgs(_ptr(x), ctypes.pointer(bs), _ptr(w), _ptr(y), _ptr(z), _ptr(out), _ptr(g), g_ldc, _ptr(dz), _ptr(dy),
                _ptr(dw), _ptr(dgamma), _ptr(dbeta), dxp, dx_ldc, 1 if dx_accumulate else 0)
    _check(_lib_fns["bnr_reference_path"](mode, 1 if backward else 0, ctypes.byref(desc), ctypes.byref(a), ws, wsb,
                                          _stream()))


def bnr_conv_fwd(desc, x, w, y):
    ws, wsb = workspace(bnr_workspace_size(desc), x.device)
    _check(_lib_fns["bnr_conv_fwd"](ctypes.byref(desc), _ptr(x), _ptr(w), _ptr(y), ws, wsb, _stream()))


def bnr_bn_add_relu_fwd(y, bn, ident, out):
    py, m, c, ldy = view(y)
    pi, _, _, ldi = view(ident)
    po, _, _, ldo = view(out)
    bs = bn.struct()
    _check(_lib_fns["bnr_bn_add_relu_fwd"](m, c, dtype_code(y), py, ldy, ctypes.byref(bs), pi, ldi, po, ldo, _stream()))


def bnr_bn_add_relu_bwd(g, out, y, bn, gm, dgamma, dbeta):
    pg, m, c, ldg = view(g)
    po, _, _, ldo = view(out)
    py, _, _, ldy = view(y)
    pm, _, _, ldm = view(gm)
    ws, wsb = workspace(bnr_stats_workspace_size(m, c), y.device)
    bs = bn.struct()
    _check(_lib_fns["bnr_bn_add_relu_bwd"](m, c, dtype_code(y), pg, ldg, po, ldo, py, ldy, ctypes.byref(bs), pm, ldm,
                                           _ptr(dgamma), _ptr(dbeta), ws, wsb, _stream()))


def bnr_reference_bn_add_relu(backward, y, bn, out, ident=None, tmp=None, g=None, gm=None, dgamma=None, dbeta=None,
                              dx=None):
    py, m, c, ldy = view(y)
    po, _, _, ldo = view(out)
    pi, ldi = (view(ident)[0], view(ident)[3]) if ident is not None else (None, 0)
    pg, ldg = (view(g)[0], view(g)[3]) if g is not None else (None, 0)
    pdx, lddx = (view(dx)[0], view(dx)[3]) if dx is not None else (None, 0)
    bs = bn.struct()
    a = AddReluRefArgs(py, ldy, ctypes.pointer(bs), pi, ldi, po, ldo, _ptr(tmp), pg, ldg, _ptr(gm), _ptr(dgamma),
                       _ptr(dbeta), pdx, lddx)
    ws, wsb = workspace(bnr_stats_workspace_size(m, c), y.device)
    _check(_lib_fns["bnr_reference_bn_add_relu"](1 if backward else 0, m, c, dtype_code(y), ctypes.byref(a), ws, wsb,
                                                 _stream()))


def bnr_hbm_copy(src, dst):
    nbytes = src.numel() * src.element_size()
    _check(_lib_fns["bnr_hbm_copy"](_ptr(src), _ptr(dst), nbytes, _stream()))


def bnr_trace_begin(kernel_classes=0xF, capacity=100000):
    _check(_lib_fns["bnr_trace_begin"](kernel_classes, capacity))


def bnr_trace_end(capacity=100000):
    """[(kernel name, ms, algorithmic bytes, flops)] of the traced launches."""
    ms = (ctypes.c_double * capacity)()
    by = (ctypes.c_double * capacity)()
    fl = (ctypes.c_double * capacity)()
    kid = (c_i32 * capacity)()
    n = _lib_fns["bnr_trace_end"](ms, by, fl, kid, capacity)
    return [(KERNEL_IDS.get(kid[i], str(kid[i])), ms[i], by[i], fl[i]) for i in range(n)]


# ------------------------------------------------------ network ends ----
def stem_desc(img, c_in):
    """First-CONV descriptor of an image tensor [n, h, w, 4] with c_in channels used."""
    n, h, w, pix = img.shape
    assert pix == 4 and img.is_contiguous()
    return StemDesc(n, h, w, c_in, dtype_code(img))


def bnr_stem_conv_fwd(img, w, s, s_bn=None):
    d = stem_desc(img, w.shape[2])
    ws, wsb = workspace(_lib_fns["bnr_stem_workspace_size"](ctypes.byref(d)), img.device)
    bs = s_bn.struct() if s_bn is not None else None
    _check(_lib_fns["bnr_stem_conv_fwd"](ctypes.byref(d), _ptr(img), _ptr(w), _ptr(s),
                                         ctypes.byref(bs) if bs is not None else None, ws, wsb, _stream()))


def bnr_stem_wgrad(img, c_in, g_src, dw):
    d = stem_desc(img, c_in)
    ws, wsb = workspace(_lib_fns["bnr_stem_workspace_size"](ctypes.byref(d)), img.device)
    gs, keep = _grad_struct(g_src)
    _check(_lib_fns["bnr_stem_wgrad"](ctypes.byref(d), _ptr(img), ctypes.byref(gs), _ptr(dw), ws, wsb, _stream()))
    del keep


def bnr_bn_relu_maxpool_fwd(x, x_bn, y, n, h, w, y_bn=None):
    """y = maxpool3x3/2(relu(bn(x))) (x_bn None: of x) [+ statistics of y]."""
    px, _, c, ldx = view(x)
    py, _, _, ldy = view(y)
    ws, wsb = workspace(_lib_fns["bnr_pool_workspace_size"](n, h, w, c), x.device)
    xs = x_bn.struct() if x_bn is not None else None
    ys = y_bn.struct() if y_bn is not None else None
    _check(_lib_fns["bnr_bn_relu_maxpool_fwd"](n, h, w, c, dtype_code(x), px, ldx,
                                               ctypes.byref(xs) if xs is not None else None, py, ldy,
                                               ctypes.byref(ys) if ys is not None else None, ws, wsb, _stream()))


def bnr_maxpool_bn_bwd(x, x_bn, gy, dy, n, h, w, dgamma=None, dbeta=None):
    px, _, c, ldx = view(x)
    pg, _, _, ldg = view(gy)
    ws, wsb = workspace(_lib_fns["bnr_pool_workspace_size"](n, h, w, c), x.device)
    xs = x_bn.struct() if x_bn is not None else None
    _check(_lib_fns["bnr_maxpool_bn_bwd"](n, h, w, c, dtype_code(x), px, ldx, ctypes.byref(xs) if xs is not None else None,
                                          pg, ldg, _ptr(dy), _ptr(dgamma), _ptr(dbeta), ws, wsb, _stream()))


def bnr_head_fwd(x, x_bn, wfc, bfc, labels, f, logits, dlogits, loss, n, h, w):
    px, _, c, ldx = view(x)
    xs = x_bn.struct()
    _check(_lib_fns["bnr_head_fwd"](n, h, w, c, wfc.shape[1], dtype_code(x), px, ldx, ctypes.byref(xs), _ptr(wfc),
                                    _ptr(bfc), _ptr(labels), _ptr(f), _ptr(logits), _ptr(dlogits), _ptr(loss),
                                    _stream()))


def bnr_head_bwd(x, x_bn, wfc, f, dlogits, df, dwfc, dbfc, dgamma, dbeta, gx, n, h, w, alpha=None, betap=None):
    px, _, c, ldx = view(x)
    pg, _, _, ldg = view(gx)
    ws, wsb = workspace(_lib_fns["bnr_head_workspace_size"](n, h, w, c), x.device)
    xs = x_bn.struct()
    _check(_lib_fns["bnr_head_bwd"](n, h, w, c, wfc.shape[1], dtype_code(x), px, ldx, ctypes.byref(xs), _ptr(wfc),
                                    _ptr(f), _ptr(dlogits), _ptr(df), _ptr(dwfc), _ptr(dbfc), _ptr(dgamma),
                                    _ptr(dbeta), pg, ldg, _ptr(alpha), _ptr(betap), ws, wsb, _stream()))


def bnr_reference_bn_relu(backward, x, bn, y, z=None, gz=None, dy=None, dgamma=None, dbeta=None, dx=None):
    """Unfused BN -> ReLU (forward: stats, y, z; backward: dy, dgamma, dbeta, dx)."""
    px, m, c, ldx = view(x)
    pgz, ldgz = (view(gz)[0], view(gz)[3]) if gz is not None else (None, 0)
    pdx, lddx = (view(dx)[0], view(dx)[3]) if dx is not None else (None, 0)
    bs = bn.struct()
    a = BnReluRefArgs(px, ldx, ctypes.pointer(bs), _ptr(y), _ptr(z), pgz, ldgz, _ptr(dy), _ptr(dgamma), _ptr(dbeta),
                      pdx, lddx)
    ws, wsb = workspace(bnr_stats_workspace_size(m, c), x.device)
    _check(_lib_fns["bnr_reference_bn_relu"](1 if backward else 0, m, c, dtype_code(x), ctypes.byref(a), ws, wsb,
                                             _stream()))
