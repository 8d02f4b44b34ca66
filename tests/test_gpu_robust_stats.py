"""Robust one-sweep statistics and running statistics (GPU against the oracle).

The one-sweep producers (statistics sweep, CONV statistics epilogues, first
CONV, max pooling) sum x - K and (x - K)^2 around a per-channel shift K when a
BN carries one; the finalisation forms mean = K + S1/m and
var = S2/m - (S1/m)^2 and, when asked, updates the running statistics.  The
reference is the fp64 two-pass statistics of the values the GPU stored (and
the oracle's running-average update), on data whose |mean| / std makes the
unshifted E[x^2] - E[x]^2 lose the variance in float32.
"""
import numpy as np
import pytest
import torch

from helpers import dev, f32dev, host
from oracle import prims as P
from paper_1807_01702_amd import synth

pytestmark = pytest.mark.gpu

TOL = 1e-4          # statistics of stored values, float32 partial sums around a shift near the mean


def assert_stats(name, mean_g, var_g, mean_r, var_r, tol):
    """Mean within tol std plus the float32 resolution of the stored mean
    (|mean| 2^-22: the mean array itself is float32), variance within tol
    relative.  Returns the errors."""
    mean_g, var_g = np.asarray(mean_g, np.float64), np.asarray(var_g, np.float64)
    sig = np.sqrt(var_r)
    em = np.abs(mean_g - mean_r) - np.abs(mean_r) * 2.0 ** -22
    ev = np.abs(var_g - var_r) / np.maximum(var_r, 1e-30)
    assert np.all(em <= tol * sig), "%s mean: %.3e std" % (name, float(np.max(em / sig)))
    assert np.all(ev <= tol), "%s var: relative %.3e" % (name, float(np.max(ev)))
    return float(np.max(em / sig)), float(np.max(ev))


@pytest.fixture(scope="module")
def B():
    from paper_1807_01702_amd import bnr
    return bnr


def _robust(B, c, shift, rmean0, rvar0, momentum=0.1, alias=False):
    """Statistics holder with a shift and running statistics (alias: the shift is running_mean itself)."""
    bn = B.BN.stats_only(c, "cuda")
    rm, rv = f32dev(rmean0), f32dev(rvar0)
    sh = rm if alias else (f32dev(shift) if shift is not None else None)
    return bn.robust(shift=sh, running_mean=rm, running_var=rv, momentum=momentum)


def _check_running(bn, rmean0, rvar0, mean_r, var_r, m, momentum=0.1):
    rm_r, rv_r = P.running_update(rmean0, rvar0, mean_r, var_r, m, momentum)
    scale = np.maximum(np.abs(rm_r), 1.0)
    assert np.max(np.abs(host(bn.running_mean) - rm_r) / scale) < 1e-5, "running mean"
    np.testing.assert_allclose(host(bn.running_var), rv_r, rtol=1e-3, atol=1e-6 * momentum)


# --------------------------------------------------------- statistics sweep ----
@pytest.mark.parametrize("bf16,offset,m,c,ldc", [
    (False, 1.0e4, 65536, 16, 16),      # |mean| / std = 1e4, float32
    (False, 3.0e3, 20011, 40, 48),      # ragged rows, channel view
    (True, 1.0e2, 30000, 72, 72),       # bf16 storage (stats of the stored values)
])
def test_sweep_shift_and_running(B, bf16, offset, m, c, ldc):
    full = synth.normal(3, "robust", (m, ldc), bf16=False) + np.float32(offset)
    full = synth.round_to_bf16(full) if bf16 else full
    x = dev(full, bf16)
    mean_r, var_r, _ = P.bn_stats(full[:, :c].astype(np.float64), 0.0)
    shift = (mean_r + synth.normal(3, "shift", (c,))).astype(np.float32)      # a shift near the mean
    rmean0, rvar0 = shift, np.ones(c, np.float32)
    bn = _robust(B, c, None, rmean0, rvar0, alias=True)                       # K = running mean (read first)
    B.bnr_bn_stats(x[:, :c], bn)
    torch.cuda.synchronize()
    em, ev = assert_stats("shifted sweep", host(bn.mean), host(bn.var), mean_r, var_r, TOL)
    _check_running(bn, rmean0, rvar0, mean_r, var_r, m)
    if not bf16 and offset >= 1e4:
        plain = B.BN.stats_only(c, "cuda")
        B.bnr_bn_stats(x[:, :c], plain)
        torch.cuda.synchronize()
        ev_plain = np.max(np.abs(host(plain.var) - var_r) / var_r)
        print("variance error: unshifted %.2e, shifted %.2e" % (ev_plain, ev))
        assert ev_plain > 100 * max(ev, 1e-7), "the unshifted sums should lose the variance here"


def test_zero_shift_and_momentum_edges(B):
    """A zero shift gives the unshifted results bit for bit; momentum 0 keeps
    the running statistics, momentum 1 replaces them."""
    m, c = 4096, 32
    full = synth.normal(4, "edge", (m, c)) + np.float32(2.0)
    x = dev(full, False)
    plain = B.BN.stats_only(c, "cuda")
    B.bnr_bn_stats(x, plain)
    z = _robust(B, c, np.zeros(c, np.float32), np.full(c, 5.0, np.float32), np.full(c, 7.0, np.float32),
                momentum=0.0)
    B.bnr_bn_stats(x, z)
    one = _robust(B, c, None, np.zeros(c, np.float32), np.zeros(c, np.float32), momentum=1.0)
    B.bnr_bn_stats(x, one)
    torch.cuda.synchronize()
    assert np.array_equal(host(z.mean), host(plain.mean)) and np.array_equal(host(z.var), host(plain.var))
    assert np.all(host(z.running_mean) == 5.0) and np.all(host(z.running_var) == 7.0)
    np.testing.assert_allclose(host(one.running_mean), host(one.mean), rtol=1e-7)
    np.testing.assert_allclose(host(one.running_var), host(one.var).astype(np.float64) * m / (m - 1), rtol=1e-6)


# ----------------------------------------------- CONV statistics epilogues ----
CONV_CASES = [
    # bf16, k, n, h, w, c_in, c_out: the persistent 1x1 and 3x3 kernels, the row-tile kernel (fp32), a ragged view
    (True, 1, 4, 14, 14, 96, 128),
    (True, 3, 2, 14, 14, 128, 32),
    (False, 3, 2, 9, 11, 24, 40),
    (True, 1, 1, 9, 11, 40, 136),
]


@pytest.mark.parametrize("case", CONV_CASES)
def test_conv_stats_epilogue_shift(B, case):
    bf16, k, n, h, w, ci, co = case
    rnd = P.round_bf16 if bf16 else (lambda a: np.asarray(a, np.float64))
    xf = synth.normal(5, "x", (n, h, w, ci), bf16=False) + np.float32(4.0)
    xf = synth.round_to_bf16(xf) if bf16 else xf
    wt = synth.conv_weight(5, "w", k, ci, co, False) * np.float32(0.5) + np.float32(0.02)
    wt = synth.round_to_bf16(wt) if bf16 else wt
    out_r = rnd(P.conv_fwd(xf.astype(np.float64), wt.astype(np.float64)))
    mean_r, var_r, _ = P.bn_stats(out_r, 0.0)
    shift = (mean_r * (1 + 1e-3) + 0.1).astype(np.float32)
    rmean0, rvar0 = synth.normal(5, "rm", (co,)), np.full(co, 2.0, np.float32)
    x = dev(xf, bf16)
    y = torch.zeros((n, h, w, co), dtype=x.dtype, device=x.device)
    ybn = _robust(B, co, shift, rmean0, rvar0)
    B.bnr_conv_bn_stats_fwd(B.desc_for(x, y, k, n, h, w), x, dev(wt, bf16), y, ybn)
    torch.cuda.synchronize()
    got = host(y).astype(np.float64)
    mg, vg, _ = P.bn_stats(got, 0.0)                  # statistics of the stored outputs
    print("|mean|/std up to %.0f" % np.max(np.abs(mg) / np.sqrt(vg)))
    assert_stats("shifted epilogue stats", host(ybn.mean), host(ybn.var), mg, vg, TOL)
    _check_running(ybn, rmean0, rvar0, mg, vg, n * h * w)


# ------------------------------------------------- first CONV, max pooling ----
def test_stem_and_maxpool_shift(B):
    from test_gpu_densenet import _img4
    n, h, w = 2, 30, 30
    img = synth.round_to_bf16(synth.normal(6, "img", (n, h, w, 3)) + np.float32(8.0))
    wt = synth.round_to_bf16(synth.conv_weight(6, "w", 7, 3, 64, False) + np.float32(0.01))
    ho, wo = (h - 1) // 2 + 1, (w - 1) // 2 + 1
    s = torch.empty((n, ho, wo, 64), dtype=torch.bfloat16, device="cuda")
    ref = P.round_bf16(P.conv_fwd(img, wt, stride=2, pad=3))
    mr, _, _ = P.bn_stats(ref, 0.0)
    rmean0, rvar0 = np.zeros(64, np.float32), np.ones(64, np.float32)
    bn = _robust(B, 64, (mr + 0.3).astype(np.float32), rmean0, rvar0)
    B.bnr_stem_conv_fwd(_img4(img, True), dev(wt, True), s, bn)
    torch.cuda.synchronize()
    got = host(s).astype(np.float64)
    mg, vg, _ = P.bn_stats(got, 0.0)
    assert_stats("first CONV shifted stats", host(bn.mean), host(bn.var), mg, vg, TOL)
    _check_running(bn, rmean0, rvar0, mg, vg, n * ho * wo)
    # plain max pooling (float32) of data with |mean| / std ~ 1e3
    c = 32
    xp = synth.normal(6, "pool", (n, h, w, c)) + np.float32(1.0e3)
    po, qo = (h - 1) // 2 + 1, (w - 1) // 2 + 1
    out = torch.empty((n, po, qo, c), dtype=torch.float32, device="cuda")
    pr = P.maxpool_fwd(xp.astype(np.float64), 3, 2, 1)
    m2, v2, _ = P.bn_stats(pr, 0.0)
    pbn = _robust(B, c, (m2 - 0.2).astype(np.float32), np.zeros(c, np.float32), np.ones(c, np.float32))
    B.bnr_bn_relu_maxpool_fwd(dev(xp, False), None, out, n, h, w, y_bn=pbn)
    torch.cuda.synchronize()
    mg, vg, _ = P.bn_stats(host(out).astype(np.float64), 0.0)
    assert_stats("pooled shifted stats", host(pbn.mean), host(pbn.var), mg, vg, TOL)


# ----------------------------------------- unfused (two-pass) reference ----
def test_reference_two_pass_running(B):
    """The unfused BN layer (two-pass statistics) ignores the shift and updates
    the running statistics from its exact mean and variance."""
    m, c = 6000, 48
    full = synth.normal(7, "ref", (m, c)) + np.float32(50.0)
    x = dev(full, False)
    gamma, beta = np.ones(c, np.float32), np.zeros(c, np.float32)
    bn = B.BN(f32dev(gamma), f32dev(beta), 1e-5)
    rmean0, rvar0 = np.full(c, 1.0, np.float32), np.full(c, 3.0, np.float32)
    bn.robust(shift=f32dev(np.full(c, 1.0e6, np.float32)), running_mean=f32dev(rmean0),
              running_var=f32dev(rvar0), momentum=0.25)
    y = torch.empty_like(x)
    z = torch.empty_like(x)
    B.bnr_reference_bn_relu(False, x, bn, y, z)
    torch.cuda.synchronize()
    mean_r, var_r, _ = P.bn_stats(full.astype(np.float64), 0.0)
    assert_stats("two-pass stats", host(bn.mean), host(bn.var), mean_r, var_r, TOL)
    _check_running(bn, rmean0, rvar0, mean_r, var_r, m, momentum=0.25)


# ------------------------------------------------ consumers at large offsets ----
@pytest.mark.parametrize("offset", [1.0e3, 1.0e4])
@pytest.mark.parametrize("k", [1, 3])
def test_consumers_at_large_offset(B, offset, k):
    """fp32 data whose channels sit at |mean| / std = offset: the robust
    statistics of x (summed around a shift near the mean), the BN+ReLU
    prologue of the CONV that reads x, the BN-backward epilogue of its data
    gradient and the deferred input gradient of a BN on a large-offset CONV
    output, each against the oracle at the fp32 tolerance."""
    from helpers import assert_close, relu_ambiguous
    n, h, w, ci, co = 2, 6, 7, 16, 24
    xf = synth.normal(21, "x", (n, h, w, ci)) + np.float32(offset)
    wt = synth.conv_weight(21, "w", k, ci, co, False)
    bp = synth.bn_params(21, "bn", ci)
    x64 = xf.astype(np.float64)
    mean_r, var_r, _ = P.bn_stats(x64, 0.0)
    x = dev(xf, False)
    bn = B.BN(f32dev(bp["gamma"]), f32dev(bp["beta"]), 1e-5)
    bn.robust(shift=f32dev(mean_r + synth.normal(21, "shift", (ci,))))
    B.bnr_bn_stats(x, bn)
    y = torch.empty((n, h, w, co), dtype=torch.float32, device="cuda")
    desc = B.desc_for(x, y, k, n, h, w)
    B.bnr_bn_relu_conv_fwd(desc, x, bn, dev(wt, False), y)
    # backward: dense upstream gradient; BN-backward epilogue, dW with the recompute
    gf = synth.normal(21, "g", (n, h, w, co))
    dw = torch.empty(wt.shape, dtype=torch.float32, device="cuda")
    dg = torch.empty(ci, dtype=torch.float32, device="cuda")
    db = torch.empty_like(dg)
    dy = torch.empty_like(x)
    dx = torch.empty_like(x)
    B.bnr_bwd_fused(desc, x, bn, dev(wt, False), B.grad_dense(dev(gf, False)), dw, dg, db, dy, dx)
    torch.cuda.synchronize()
    yr, mu, var, rstd = P.bn_fwd(x64, bp["gamma"], bp["beta"], 1e-5)
    amb = relu_ambiguous(yr, False)
    z = P.relu_fwd(yr)
    assert_close("conv out", host(y), P.conv_fwd(z, wt.astype(np.float64)), 1e-4)
    dz = P.conv_dgrad(gf.astype(np.float64), wt.astype(np.float64), (h, w))
    dyr = P.relu_bwd(dz, yr)
    dxr, dgr, dbr = P.bn_bwd(x64, dyr, bp["gamma"], mu, rstd)
    assert_close("dy", host(dy), dyr, 1e-4, exclude=amb)
    assert_close("dx", host(dx), dxr, 1e-4, exclude=amb)
    assert_close("dW", host(dw), P.conv_wgrad(z, gf.astype(np.float64), k), 1e-4)
    assert_close("dgamma", host(dg), dgr, 1e-4)
    # the deferred input gradient of a BN whose input is this large-offset x,
    # formed on load by the backward of the CONV that produced x (input xin)
    xin_f = synth.normal(21, "xin", (n, h, w, co))
    wp = synth.conv_weight(21, "wp", k, co, ci, False)
    dwp = torch.empty(wp.shape, dtype=torch.float32, device="cuda")
    dxin = torch.empty((n, h, w, co), dtype=torch.float32, device="cuda")
    descp = B.desc_for(dev(xin_f, False), x, k, n, h, w)
    B.bnr_bwd_fused(descp, dev(xin_f, False), None, dev(wp, False), B.grad_bn(dy, x, bn, dg, db), dwp, dx=dxin)
    torch.cuda.synchronize()
    g_r = P.bn_bwd(x64, host(dy), bp["gamma"], mu, rstd)[0]
    assert_close("deferred dx -> producer dx", host(dxin), P.conv_dgrad(g_r, wp.astype(np.float64), (h, w)), 1e-4)
    assert_close("deferred dx -> producer dW", host(dwp), P.conv_wgrad(xin_f.astype(np.float64), g_r, k), 1e-4)


@pytest.mark.parametrize("offset", [1.0e4])
def test_sweeps_at_large_offset(B, offset):
    """The standalone float32 BN sweeps on data at |mean| / std = offset: BN
    input gradient, summed-gradient input gradient and the summed gradient
    formed in a CONV prologue, BN + add + ReLU forward and backward, and the
    unfused (two-pass) BN -> ReLU layer, each against the oracle."""
    from helpers import assert_close, relu_ambiguous
    n, h, w, c, co = 2, 5, 9, 32, 16
    m = n * h * w
    xf = synth.normal(22, "x", (n, h, w, c)) + np.float32(offset)
    x64 = xf.astype(np.float64)
    bp = synth.bn_params(22, "bn", c)
    x = dev(xf, False)

    def robust_bn():
        bn = B.BN(f32dev(bp["gamma"]), f32dev(bp["beta"]), 1e-5)
        return bn.robust(shift=f32dev(P.bn_stats(x64, 0.0)[0] + synth.normal(22, "shift", (c,))))

    yr, mu, var, rstd = P.bn_fwd(x64, bp["gamma"], bp["beta"], 1e-5)
    amb = relu_ambiguous(yr, False)
    bn = robust_bn()
    B.bnr_bn_stats(x, bn)
    # BN input gradient from dy and the sums
    dyf = synth.normal(22, "dy", (n, h, w, c))
    dxr, dgr, dbr = P.bn_bwd(x64, dyf.astype(np.float64), bp["gamma"], mu, rstd)
    dx = torch.empty_like(x)
    B.bnr_bn_dx(dev(dyf, False), x, bn, f32dev(dgr), f32dev(dbr), dx)
    torch.cuda.synchronize()
    assert_close("bn dx", host(dx), dxr, 1e-4)
    # summed gradient: dx = gsum + alpha + betap xhat, and the same term in a CONV prologue
    gs = synth.normal(22, "gsum", (n, h, w, c))
    al, bt = synth.normal(22, "alpha", (c,)), synth.normal(22, "betap", (c,))
    xh = (x64 - mu) * rstd
    dsr = gs + al + bt * xh
    B.bnr_split_dx(dev(gs, False), x, bn, f32dev(al), f32dev(bt), dx)
    xin = synth.normal(22, "xin", (n, h, w, co))
    wp = synth.conv_weight(22, "wp", 1, co, c, False)
    dxin = torch.empty((n, h, w, co), dtype=torch.float32, device="cuda")
    dwp = torch.empty(wp.shape, dtype=torch.float32, device="cuda")
    desc = B.desc_for(dev(xin, False), x, 1, n, h, w)
    B.bnr_bwd_fused(desc, dev(xin, False), None, dev(wp, False),
                    B.grad_split(dev(gs, False), x, bn, f32dev(al), f32dev(bt)), dwp, dx=dxin)
    torch.cuda.synchronize()
    assert_close("split dx", host(dx), dsr, 1e-4)
    assert_close("summed gradient prologue -> dx", host(dxin), P.conv_dgrad(dsr, wp.astype(np.float64), (h, w)), 1e-4)
    assert_close("summed gradient prologue -> dW", host(dwp), P.conv_wgrad(xin.astype(np.float64), dsr, 1), 1e-4)
    # BN + add + ReLU and its backward
    idf = synth.normal(22, "id", (n, h, w, c))
    t = yr + idf
    amb_t = relu_ambiguous(t, False)
    outr = P.relu_fwd(t)
    out = torch.empty_like(x)
    B.bnr_bn_add_relu_fwd(x, bn, dev(idf, False), out)
    g = synth.normal(22, "g", (n, h, w, c))
    gm = torch.empty_like(x)
    dg = torch.empty(c, dtype=torch.float32, device="cuda")
    db = torch.empty_like(dg)
    B.bnr_bn_add_relu_bwd(dev(g, False), out, x, bn, gm, dg, db)
    torch.cuda.synchronize()
    assert_close("bn+add+relu", host(out), outr, 1e-4, exclude=amb_t)
    gmr = P.relu_bwd(g.astype(np.float64), t)
    _, dg2, db2 = P.bn_bwd(x64, gmr, bp["gamma"], mu, rstd)
    assert_close("bn+add+relu bwd dgamma", host(dg), dg2, 1e-4)
    assert_close("bn+add+relu bwd dbeta", host(db), db2, 1e-4)
    # unfused BN -> ReLU (two-pass statistics) forward and backward.  Its mean
    # is a plain float32 sum of x (the two-pass layer takes no shift), good to
    # about 1e-3 std at this offset; the consumers are checked against the
    # oracle's formulas at the statistics the GPU produced (mean + mean_lo in
    # float64, rstd), which is what they can be held to.
    bn2 = robust_bn()
    y = torch.empty_like(x)
    z = torch.empty_like(x)
    B.bnr_reference_bn_relu(False, x, bn2, y, z)
    gz = synth.normal(22, "gz", (n, h, w, c))
    dy = torch.empty_like(x)
    dx2 = torch.empty_like(x)
    torch.cuda.synchronize()
    mu2 = host(bn2.mean).astype(np.float64) + host(bn2.mean_lo).astype(np.float64)
    rs2 = host(bn2.rstd).astype(np.float64)
    assert np.max(np.abs(mu2 - mu) * rstd) < 1e-2, "two-pass mean"
    y2r = bp["gamma"] * ((x64 - mu2) * rs2) + bp["beta"]
    amb2 = relu_ambiguous(y2r, False)
    B.bnr_reference_bn_relu(True, x, bn2, y, z, gz=dev(gz, False), dy=dy, dgamma=dg, dbeta=db, dx=dx2)
    torch.cuda.synchronize()
    assert_close("two-pass y", host(y), y2r, 1e-4)
    dyr = P.relu_bwd(gz.astype(np.float64), y2r)
    dxr2, dgr2, _ = P.bn_bwd(x64, dyr, bp["gamma"], mu2, rs2)
    assert_close("two-pass dx", host(dx2), dxr2, 1e-4, exclude=amb2)
    assert_close("two-pass dgamma", host(dg), dgr2, 1e-4)
    # one-sweep statistics around the shift: mean + mean_lo is the float64 mean
    full = host(bn.mean).astype(np.float64) + host(bn.mean_lo).astype(np.float64)
    assert np.max(np.abs(full - mu) * rstd) < 1e-6, "mean + mean_lo"


def test_net_ends_at_large_offset(B):
    """BN-ReLU-max-pooling forward and backward and the classifier head's
    pooled features on float32 data at |mean| / std = 1e4, with the mean
    given as its float32 value plus the low part, against the oracle."""
    from helpers import assert_close
    n, h, w, c = 2, 14, 14, 32
    xf = synth.normal(23, "x", (n, h, w, c)) + np.float32(1.0e4)
    x64 = xf.astype(np.float64)
    bp = synth.bn_params(23, "bn", c)
    yr, mu, var, rstd = P.bn_fwd(x64, bp["gamma"], bp["beta"], 1e-5)
    m32 = mu.astype(np.float32)
    lo32 = (mu - m32.astype(np.float64)).astype(np.float32)
    r32 = rstd.astype(np.float32)
    bn = B.BN(f32dev(bp["gamma"]), f32dev(bp["beta"]), 1e-5, mean=f32dev(m32), rstd=f32dev(r32))
    bn.mean_lo = f32dev(lo32)
    y = bp["gamma"] * ((x64 - mu) * r32.astype(np.float64)) + bp["beta"]
    z = P.relu_fwd(y)
    x = dev(xf, False)
    ho, wo = (h - 1) // 2 + 1, (w - 1) // 2 + 1
    out = torch.empty((n, ho, wo, c), dtype=torch.float32, device="cuda")
    B.bnr_bn_relu_maxpool_fwd(x, bn, out, n, h, w)
    gy = synth.normal(23, "gy", (n, ho, wo, c))
    dy = torch.empty_like(x)
    dg = torch.empty(c, dtype=torch.float32, device="cuda")
    db = torch.empty_like(dg)
    B.bnr_maxpool_bn_bwd(x, bn, dev(gy, False), dy, n, h, w, dg, db)
    # head: pooled features of relu(bn(x))
    K = 10
    wfc = synth.normal(23, "wfc", (c, K)) * np.float32(0.1)
    bfc = synth.normal(23, "bfc", (K,))
    labels = synth._gen(23, "labels").integers(0, K, size=n).astype(np.int32)
    f32 = dict(dtype=torch.float32, device="cuda")
    ft, lg, dl, ls = torch.empty((n, c), **f32), torch.empty((n, K), **f32), torch.empty((n, K), **f32), torch.empty(1 + n, **f32)
    B.bnr_head_fwd(x, bn, dev(wfc, False), f32dev(bfc), torch.from_numpy(labels).cuda(), ft, lg, dl, ls, n, h, w)
    torch.cuda.synchronize()
    assert_close("BN-ReLU-max-pool", host(out), P.maxpool_fwd(z, 3, 2, 1), 1e-5)
    dyr = P.relu_bwd(P.maxpool_bwd(z, gy.astype(np.float64), 3, 2, 1), y)
    _, dgr, dbr = P.bn_bwd(x64, dyr, bp["gamma"], mu, r32.astype(np.float64))
    assert_close("max-pool BN backward dy", host(dy), dyr, 1e-5)
    assert_close("max-pool BN backward dgamma", host(dg), dgr, 1e-5)
    assert_close("max-pool BN backward dbeta", host(db), dbr, 1e-5)
    assert_close("head features", host(ft), P.global_avgpool_fwd(z), 1e-5)
