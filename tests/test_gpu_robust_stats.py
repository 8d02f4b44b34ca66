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
