"""Host-side checks of the C ABI (CPU only, no kernel launches): the library
loads, exports every entry point that include/bnr.h declares, and rejects bad
arguments with the documented status before launching anything."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    src = open(os.path.join(ROOT, "include", "bnr.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(bnr_[a-z0-9_]+)\s*\(", src)))


@pytest.fixture(scope="module")
def B():
    from paper_1807_01702_amd import bnr
    return bnr


def test_exports_every_declared_symbol(B):
    names = _declared()
    assert len(names) >= 12, names
    lib = ctypes.CDLL(B.LIB_PATH)
    missing = [n for n in names if not hasattr(lib, n)]
    assert not missing, missing


def test_status_strings(B):
    for i, name in enumerate(B.STATUS):
        assert B.status_string(i) == name


def _desc(B, **kw):
    d = dict(n=2, h=4, w=4, c_in=16, c_out=8, k=1, in_ldc=16, out_ldc=8, dtype=B.BNR_BF16)
    d.update(kw)
    return B.ConvDesc(**d)


def test_workspace_sizes(B):
    assert B.bnr_workspace_size(_desc(B)) > 0
    assert B.bnr_workspace_size(_desc(B, k=5)) == 0
    assert B.bnr_stats_workspace_size(100, 64) > 0
    assert B.bnr_stats_workspace_size(0, 64) == 0


# fake, 16-byte aligned, never dereferenced addresses (validation fails first)
A = 0x10000
WS = 0x100000


@pytest.mark.parametrize("kw,status", [
    (dict(k=5), "BNR_ERR_UNSUPPORTED"),
    (dict(n=0), "BNR_ERR_SHAPE"),
    (dict(c_in=12), "BNR_ERR_ALIGN"),
    (dict(in_ldc=8), "BNR_ERR_SHAPE"),
    (dict(dtype=7), "BNR_ERR_DTYPE"),
    (dict(k=3, w=65), "BNR_ERR_UNSUPPORTED"),
])
def test_conv_fwd_rejects_bad_descriptor(B, kw, status):
    d = _desc(B, **kw)
    bn = B.BNStruct(None, None, A, A, A, 1e-5)
    r = B._lib_fns["bnr_conv_bn_stats_fwd"](ctypes.byref(d), A, A + 0x1000, A + 0x2000, ctypes.byref(bn), WS, 1 << 30, None)
    assert B.STATUS[r] == status, B._lib_fns["bnr_last_error"]()


def test_conv_fwd_rejects_pointers_workspace_alias(B):
    d = _desc(B)
    bn = B.BNStruct(None, None, A, A, A, 1e-5)
    f = B._lib_fns["bnr_conv_bn_stats_fwd"]
    assert B.STATUS[f(ctypes.byref(d), None, A, A + 0x2000, ctypes.byref(bn), WS, 1 << 30, None)] == "BNR_ERR_NULL"
    assert B.STATUS[f(ctypes.byref(d), A + 8, A, A + 0x2000, ctypes.byref(bn), WS, 1 << 30, None)] == "BNR_ERR_ALIGN"
    assert B.STATUS[f(ctypes.byref(d), A, A + 0x1000, A + 0x2000, ctypes.byref(bn), WS, 16, None)] == "BNR_ERR_WORKSPACE"
    assert B.STATUS[f(ctypes.byref(d), A, A + 0x1000, A + 0x2000, ctypes.byref(bn), None, 0, None)] == "BNR_ERR_WORKSPACE"
    assert B.STATUS[f(ctypes.byref(d), A, A + 0x1000, A + 0x40, ctypes.byref(bn), WS, 1 << 30, None)] == "BNR_ERR_ALIAS"
    bad = B.BNStruct(None, None, A, A, A, 0.0)
    assert B.STATUS[f(ctypes.byref(d), A, A + 0x1000, A + 0x2000, ctypes.byref(bad), WS, 1 << 30, None)] == "BNR_ERR_SHAPE"


def test_robust_statistics_fields_validate(B):
    """The shift / running-statistics fields of bnr_bn are checked before any launch."""
    st = B._lib_fns["bnr_bn_stats"]
    def status(**kw):
        f = dict(shift=None, running_mean=None, running_var=None, momentum=0.0)
        f.update(kw)
        bn = B.BNStruct(None, None, A, A, A, 1e-5, f["shift"], f["running_mean"], f["running_var"], f["momentum"])
        return B.STATUS[st(64, 8, 8, B.BNR_BF16, A, ctypes.byref(bn), WS, 1 << 20, None)]
    assert status(running_mean=A, momentum=1.5) == "BNR_ERR_SHAPE"
    assert status(running_mean=A, momentum=-0.1) == "BNR_ERR_SHAPE"
    assert status(running_var=A) == "BNR_ERR_NULL"
    assert status(shift=A + 2) == "BNR_ERR_ALIGN"
    assert status(running_mean=A + 1, momentum=0.1) == "BNR_ERR_ALIGN"


def test_other_entry_points_validate(B):
    bn = B.BNStruct(A, A, A, A, A, 1e-5)
    st = B._lib_fns["bnr_bn_stats"]
    assert B.STATUS[st(0, 8, 8, B.BNR_BF16, A, ctypes.byref(bn), WS, 1 << 20, None)] == "BNR_ERR_SHAPE"
    assert B.STATUS[st(10, 12, 16, B.BNR_BF16, A, ctypes.byref(bn), WS, 1 << 20, None)] == "BNR_ERR_ALIGN"
    assert B.STATUS[st(10, 8, 8, B.BNR_BF16, A, None, WS, 1 << 20, None)] == "BNR_ERR_NULL"
    d = _desc(B)
    g = B.GradSrc(9, A, 8, None, None, 0, None, None, None)
    r = B._lib_fns["bnr_bwd_fused"](ctypes.byref(d), A, ctypes.byref(bn), A, ctypes.byref(g), A, A, A, A, None, 0, 0,
                                     WS, 1 << 30, None)
    assert B.STATUS[r] == "BNR_ERR_UNSUPPORTED"
    g = B.GradSrc(B.GRAD_DENSE, A + 0x4000, 8, None, None, 0, None, None, None)
    r = B._lib_fns["bnr_bwd_fused"](ctypes.byref(d), A, None, A, ctypes.byref(g), A, None, None, None, None, 0, 0,
                                     WS, 1 << 30, None)
    assert B.STATUS[r] == "BNR_ERR_NULL"          # no BN and no dx
    pool = B._lib_fns["bnr_avgpool2_fwd"]
    assert B.STATUS[pool(1, 3, 4, 8, B.BNR_BF16, A, 8, A + 0x1000, 8, None)] == "BNR_ERR_SHAPE"
    assert B.STATUS[pool(1, 4, 4, 8, B.BNR_BF16, A, 8, A + 0x1000, 4, None)] == "BNR_ERR_SHAPE"
    assert B.STATUS[B._lib_fns["bnr_hbm_copy"](A, A + 0x1000, 24, None)] == "BNR_ERR_SHAPE"
    assert B.STATUS[B._lib_fns["bnr_hbm_copy"](A, A + 0x8, 64, None)] == "BNR_ERR_ALIGN"
    a = B.RefArgs()
    assert B.STATUS[B._lib_fns["bnr_reference_path"](5, 0, ctypes.byref(d), ctypes.byref(a), WS, 1 << 30, None)] \
        == "BNR_ERR_UNSUPPORTED"


def test_network_end_entry_points_validate(B):
    f = B._lib_fns
    sd = B.StemDesc(2, 30, 30, 3, B.BNR_BF16)
    assert f["bnr_stem_workspace_size"](ctypes.byref(sd)) > 0
    assert f["bnr_stem_workspace_size"](ctypes.byref(B.StemDesc(2, 30, 300, 3, B.BNR_BF16))) == 0
    bn = B.BNStruct(None, None, A, A, A, 1e-5)
    conv = f["bnr_stem_conv_fwd"]
    for desc, status in ((B.StemDesc(2, 30, 30, 5, B.BNR_BF16), "BNR_ERR_UNSUPPORTED"),
                         (B.StemDesc(2, 30, 257, 3, B.BNR_BF16), "BNR_ERR_UNSUPPORTED"),
                         (B.StemDesc(0, 30, 30, 3, B.BNR_BF16), "BNR_ERR_SHAPE"),
                         (B.StemDesc(2, 30, 30, 3, 9), "BNR_ERR_DTYPE")):
        assert B.STATUS[conv(ctypes.byref(desc), A, A + 0x100000, A + 0x200000, ctypes.byref(bn), WS, 1 << 30,
                             None)] == status
    assert B.STATUS[conv(ctypes.byref(sd), A, A + 0x100000, A + 0x200000, ctypes.byref(bn), WS, 64, None)] \
        == "BNR_ERR_WORKSPACE"
    assert B.STATUS[conv(ctypes.byref(sd), A, A + 0x100000, A + 0x10, None, WS, 1 << 30, None)] == "BNR_ERR_ALIAS"
    g = B.GradSrc(B.GRAD_AVGPOOL2, A, 64, None, None, 0, None, None, None)
    assert B.STATUS[f["bnr_stem_wgrad"](ctypes.byref(sd), A, ctypes.byref(g), A + 0x10000, WS, 1 << 30, None)] \
        == "BNR_ERR_UNSUPPORTED"
    g = B.GradSrc(B.GRAD_DENSE, A, 60, None, None, 0, None, None, None)
    assert B.STATUS[f["bnr_stem_wgrad"](ctypes.byref(sd), A, ctypes.byref(g), A + 0x10000, WS, 1 << 30, None)] \
        == "BNR_ERR_SHAPE"
    mp, mb = f["bnr_bn_relu_maxpool_fwd"], f["bnr_maxpool_bn_bwd"]
    assert f["bnr_pool_workspace_size"](2, 112, 112, 64) > 0
    assert B.STATUS[mp(2, 8, 8, 12, B.BNR_BF16, A, 16, None, A + 0x100000, 16, None, None, 0, None)] == "BNR_ERR_ALIGN"
    assert B.STATUS[mp(2, 8, 8, 16, B.BNR_BF16, A, 16, None, A + 0x10, 16, None, None, 0, None)] == "BNR_ERR_ALIAS"
    assert B.STATUS[mp(2, 8, 8, 16, B.BNR_BF16, A, 16, None, A + 0x100000, 16, ctypes.byref(bn), None, 0, None)] \
        == "BNR_ERR_WORKSPACE"
    assert B.STATUS[mb(2, 8, 8, 128, B.BNR_BF16, A, 128, None, A + 0x100000, 128, A + 0x200000, None, None, None, 0,
                       None)] == "BNR_ERR_UNSUPPORTED"
    assert B.STATUS[mb(2, 8, 8, 48, B.BNR_BF16, A, 48, None, A + 0x100000, 48, A + 0x200000, None, None, None, 0,
                       None)] == "BNR_ERR_UNSUPPORTED"
    assert B.STATUS[mb(2, 8, 300, 64, B.BNR_BF16, A, 64, None, A + 0x1000000, 64, A + 0x2000000, None, None, None, 0,
                       None)] == "BNR_ERR_UNSUPPORTED"
    full = B.BNStruct(A, A, A, A, A, 1e-5)
    assert B.STATUS[mb(2, 8, 8, 64, B.BNR_BF16, A, 64, ctypes.byref(full), A + 0x100000, 64, A + 0x200000, None, None,
                       WS, 1 << 30, None)] == "BNR_ERR_NULL"      # dgamma / dbeta required with a BN
    hf, hb = f["bnr_head_fwd"], f["bnr_head_bwd"]
    assert B.STATUS[hf(2, 7, 7, 64, 10, B.BNR_BF16, A, 64, ctypes.byref(full), A, A, None, A, A, A, A, None)] \
        == "BNR_ERR_NULL"                                          # labels
    assert B.STATUS[hf(2, 7, 7, 64, 0, B.BNR_BF16, A, 64, ctypes.byref(full), A, A, A, A, A, A, A, None)] \
        == "BNR_ERR_SHAPE"
    assert f["bnr_head_workspace_size"](2, 7, 7, 64) > 0
    assert B.STATUS[hb(2, 7, 7, 64, 10, B.BNR_BF16, A, 64, ctypes.byref(full), A, A, A, A, A, A, A, A, A + 0x40, 64,
                       None, None, WS, 1 << 30, None)] == "BNR_ERR_ALIAS"
    assert B.STATUS[hb(2, 7, 7, 64, 10, B.BNR_BF16, A, 64, ctypes.byref(full), A, A, A, A, A, A, A, A, A + 0x100000,
                       64, None, None, WS, 8, None)] == "BNR_ERR_WORKSPACE"
    a = B.BnReluRefArgs()
    assert B.STATUS[f["bnr_reference_bn_relu"](0, 100, 16, B.BNR_BF16, ctypes.byref(a), WS, 1 << 30, None)] \
        == "BNR_ERR_SHAPE"                                         # x_ldc 0


def test_bwd_fused_rejects_outputs_over_gradient_source(B):
    """dy / dx may not overlap any view the gradient source reads (the data
    gradient's workgroups read it while others already write the outputs)."""
    d = _desc(B)                                    # m = 32, c_in 16, c_out 8, bf16
    bn = B.BNStruct(A, A, A, A, A, 1e-5)
    f = B._lib_fns["bnr_bwd_fused"]
    x, w, g = A, A + 0x1000, A + 0x4000
    dense = B.GradSrc(B.GRAD_DENSE, g, 8, None, None, 0, None, None, None)
    def st(gs, dy, dx, xbn=True):
        return B.STATUS[f(ctypes.byref(d), x, ctypes.byref(bn) if xbn else None, w, ctypes.byref(gs), A + 0x8000,
                          A + 0x9000, A + 0x9100, dy, dx, 16 if dx else 0, 0, WS, 1 << 30, None)]
    assert st(dense, g + 0x10, None) == "BNR_ERR_ALIAS"          # dy over the dense gradient
    assert st(dense, A + 0x10000, g + 0x20) == "BNR_ERR_ALIAS"   # dx over the dense gradient
    assert st(dense, None, g, xbn=False) == "BNR_ERR_ALIAS"      # no BN: dx over the gradient
    assert st(dense, None, x + 0x10, xbn=False) == "BNR_ERR_ALIAS"   # no BN: dx over x
    gb = B.GradSrc(B.GRAD_BN, None, 0, A + 0x20000, A + 0x30000, 8, ctypes.pointer(bn), A, A, None, None)
    assert st(gb, A + 0x20000, None) == "BNR_ERR_ALIAS"          # dy over the deferred gradient's dy
    assert st(gb, A + 0x10000, A + 0x30010) == "BNR_ERR_ALIAS"   # dx over the deferred gradient's x


def test_static_scratch_entry_point_limit(B):
    """bnr_bn_relu_conv_fwd_static takes every forward CONV of the workloads
    (dense block and bottleneck, ResNet-50 conv2_x, DenseNet-121 at N = 128)
    and refuses one whose forward workspace exceeds its 16 MiB array, before
    any launch.  y is NULL, so no call here can launch: a shape that fits
    stops at the NULL check (or, without a GPU, at the device lookup)."""
    f = B._lib_fns["bnr_bn_relu_conv_fwd_static"]
    bn = B.BNStruct(A, A, A, A, A, 1e-5)
    ybn = B.BNStruct(None, None, A, A, A, 1e-5)

    def status(n, h, w, ci, co, k, dtype=B.BNR_BF16):
        d = B.ConvDesc(n, h, w, ci, co, k, ci, co, dtype)
        return B.STATUS[f(ctypes.byref(d), A, ctypes.byref(bn), A + 0x1000, None, ctypes.byref(ybn), None)]

    shapes = [(32, 56, 56, 256, 128, 1), (32, 56, 56, 128, 32, 3), (64, 56, 56, 256, 128, 1),
              (128, 56, 56, 256, 64, 1), (128, 56, 56, 64, 64, 3), (128, 56, 56, 64, 256, 1)]
    shapes += [(64, 56, 56, 64 + 32 * l, 128, 1) for l in range(6)]
    for hw, c0, layers in ((56, 64, 6), (28, 128, 12), (14, 256, 24), (7, 512, 16)):
        shapes += [(128, hw, hw, c0 + 32 * l, 128, 1) for l in range(layers)] + [(128, hw, hw, 128, 32, 3)]
        shapes.append((128, hw, hw, c0 + 32 * layers, (c0 + 32 * layers) // 2, 1))       # transition
    for s in shapes:
        assert status(*s) in ("BNR_ERR_NULL", "BNR_ERR_HIP"), s
    assert status(8, 8, 8, 64, 32, 1, B.BNR_F32) in ("BNR_ERR_NULL", "BNR_ERR_HIP")
    assert status(256, 64, 64, 256, 256, 1, B.BNR_F32) == "BNR_ERR_WORKSPACE"
    d = _desc(B)
    assert B.STATUS[f(ctypes.byref(d), A, None, A + 0x1000, A + 0x2000, None, None)] == "BNR_ERR_NULL"   # x_bn
