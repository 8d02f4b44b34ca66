"""Pins of the CPU oracle against what the paper and the mathematics fix.

None of these compare the oracle with itself: they use hand-worked examples
(tests/golden), invariants of BN training, adjoint identities, finite
differences, textbook special cases (1x1 CONV = matrix product, delta filters)
and independent library routines (numpy matmul, torch CPU fp64 conv2d /
batch_norm / autograd, torch's bf16 cast).  Runs on the CPU only.
"""
import os

import numpy as np
import pytest
import torch
import torch.nn.functional as F

from oracle import compose as OC
from oracle import prims as P

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
RNG = np.random.default_rng(1234)


def _golden(name):
    d = {}
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            if line.startswith("#") or not line.strip():
                continue
            k, *v = line.split()
            d[k] = np.array([float(t) for t in v])
    return d


def _nchw(a):
    return torch.from_numpy(np.ascontiguousarray(np.asarray(a, np.float64).transpose(0, 3, 1, 2)))


def _nhwc(t):
    return t.detach().numpy().transpose(0, 2, 3, 1)


def _oihw(w):
    return torch.from_numpy(np.ascontiguousarray(np.asarray(w, np.float64).transpose(3, 2, 0, 1)))


def _is_bf16(a):
    a = np.asarray(a, np.float64)
    return np.array_equal(P.round_bf16(a), a)


# ------------------------------------------------------------- golden ----
def test_bn_worked_example():
    g = _golden("bn_worked_example.txt")
    x = g["x"].reshape(4, 1)
    y, mean, var, rstd = P.bn_fwd(x, g["gamma"], g["beta"], float(g["eps"][0]))
    np.testing.assert_allclose(mean, g["mean"], rtol=0, atol=1e-15)
    np.testing.assert_allclose(var, g["var"], rtol=0, atol=1e-15)
    np.testing.assert_allclose(rstd, g["rstd"], rtol=1e-14)
    np.testing.assert_allclose(y[:, 0], g["y"], rtol=1e-14)
    m1, v1 = P.mvf_stats(x)
    np.testing.assert_allclose(v1, g["var"], rtol=0, atol=1e-15)
    dx, dgamma, dbeta = P.bn_bwd(x, g["dy"].reshape(4, 1), g["gamma"], mean, rstd)
    np.testing.assert_allclose(dbeta, g["dbeta"], rtol=1e-14)
    np.testing.assert_allclose(dgamma, g["dgamma"], rtol=1e-14)
    np.testing.assert_allclose(dx[:, 0], g["dx"], rtol=1e-13, atol=1e-15)


def test_conv_worked_example():
    g = _golden("conv_worked_example.txt")
    x = g["input"].reshape(1, 3, 3, 1)
    ones = np.ones((3, 3, 1, 1))
    np.testing.assert_array_equal(P.conv_fwd(x, ones).ravel(), g["ones"])
    w = np.zeros((3, 3, 1, 1)); w[0, 0] = 1
    np.testing.assert_array_equal(P.conv_fwd(x, w).ravel(), g["tap00"])
    w = np.zeros((3, 3, 1, 1)); w[2, 1] = 1
    np.testing.assert_array_equal(P.conv_fwd(x, w).ravel(), g["tap21"])


# ------------------------------------------------------------ BN forward ----
@pytest.mark.parametrize("m,C,shift", [(512, 7, 0.0), (3000, 5, 10.0), (2, 3, 0.0)])
def test_bn_fwd_normalised_moments(m, C, shift):
    x = RNG.standard_normal((m, C)) * RNG.uniform(0.1, 5, C) + shift
    y, mean, var, rstd = P.bn_fwd(x, np.ones(C), np.zeros(C), 0.0)
    assert np.max(np.abs(y.mean(0))) < 1e-12
    assert np.max(np.abs((y * y).mean(0) - 1)) < 1e-12
    eps = 1e-5
    y, mean, var, rstd = P.bn_fwd(x, np.ones(C), np.zeros(C), eps)
    assert np.max(np.abs(y.mean(0))) < 1e-12
    np.testing.assert_allclose((y * y).mean(0), var / (var + eps), rtol=0, atol=1e-12)


def test_bn_fwd_affine_and_special_cases():
    C = 4
    x = RNG.standard_normal((100, C))
    gamma, beta = RNG.uniform(0.5, 1.5, C), RNG.normal(0, 0.1, C)
    y0, *_ = P.bn_fwd(x, np.ones(C), np.zeros(C), 1e-5)
    y, *_ = P.bn_fwd(x, gamma, beta, 1e-5)
    np.testing.assert_allclose(y, gamma * y0 + beta, rtol=0, atol=1e-13)
    # one value per channel: xhat = 0, so y = beta
    y1, *_ = P.bn_fwd(x[:1], gamma, beta, 1e-5)
    np.testing.assert_array_equal(y1[0], beta)
    # a constant channel: y = beta
    yc, mean, var, _ = P.bn_fwd(np.full((50, C), 3.25), gamma, beta, 1e-5)
    np.testing.assert_array_equal(var, 0.0)
    np.testing.assert_array_equal(yc, np.broadcast_to(beta, (50, C)))


def test_bn_fwd_matches_torch_batch_norm():
    x = RNG.standard_normal((6, 5, 7, 9)) * 2 + 1
    gamma, beta = RNG.uniform(0.5, 1.5, 9), RNG.normal(0, 0.1, 9)
    y, mean, var, rstd = P.bn_fwd(x, gamma, beta, 1e-5)
    ref = F.batch_norm(_nchw(x), None, None, torch.from_numpy(gamma), torch.from_numpy(beta),
                       training=True, eps=1e-5)
    np.testing.assert_allclose(y, _nhwc(ref), rtol=0, atol=1e-12)
    np.testing.assert_allclose(var, x.reshape(-1, 9).var(0), rtol=1e-13)     # biased (ddof=0)


def test_mvf_stats_equal_two_pass():
    # small integers over m = 2^10 values: both forms are exact in fp64
    x = RNG.integers(-50, 50, (1024, 6)).astype(np.float64)   # m = 2^10: every step exact
    m1, v1 = P.mvf_stats(x)
    m2, v2, _ = P.bn_stats(x, 0.0)
    np.testing.assert_array_equal(m1, m2)
    np.testing.assert_array_equal(v1, v2)
    x = RNG.standard_normal((4096, 3)) + 3.0
    m1, v1 = P.mvf_stats(x)
    np.testing.assert_allclose(v1, x.var(0), rtol=1e-12)
    np.testing.assert_allclose(m1, x.mean(0), rtol=1e-14)


def test_mvf_shifted_statistics():
    """One-sweep statistics around a shift K (the robust MVF reading): exact
    small-integer data against the two-pass definition for several K; the
    closed form mean = mu, var = sigma^2 of a +-sigma pattern; the textbook
    two-pass mean/var of torch when K is the exact mean."""
    x = RNG.integers(-50, 50, (1024, 5)).astype(np.float64)
    m2, v2, _ = P.bn_stats(x, 0.0)
    for K in (np.zeros(5), np.array([3.0, -7.0, 11.0, 0.5, -64.0]), m2):
        m1, v1 = P.mvf_stats_shifted(x, K)
        np.testing.assert_allclose(m1, m2, rtol=0, atol=1e-12)
        np.testing.assert_allclose(v1, v2, rtol=1e-13, atol=1e-12)
    # K = 0 is the unshifted one-sweep identity
    np.testing.assert_array_equal(P.mvf_stats_shifted(x, np.zeros(5))[1], P.mvf_stats(x)[1])
    # x = mu + sigma * (+-1): mean mu, variance sigma^2, from a shift near mu
    mu, sg = np.array([1.0e4, -2.5e3]), np.array([1.0, 0.25])
    s = np.where(np.arange(2048) % 2 == 0, 1.0, -1.0)[:, None]
    x = mu[None, :] + sg[None, :] * s
    m1, v1 = P.mvf_stats_shifted(x, mu + np.array([0.5, -0.125]))
    np.testing.assert_allclose(m1, mu, rtol=0, atol=1e-12)
    np.testing.assert_allclose(v1, sg ** 2, rtol=1e-12)
    t = torch.from_numpy(RNG.standard_normal((3000, 4)) * 2 + 5)
    m1, v1 = P.mvf_stats_shifted(t.numpy(), t.mean(0).numpy())
    np.testing.assert_allclose(v1, t.var(0, unbiased=False).numpy(), rtol=1e-12)


def test_mvf_shift_removes_single_precision_cancellation():
    """The reason for the shift (a property of the method, not of the oracle):
    float32 one-sweep sums of data with |mean|/std = 1e4 lose the variance,
    the same sums around a shift near the mean keep it."""
    r = np.random.default_rng(7)
    x = (1.0e4 + r.standard_normal(65536)).astype(np.float32)
    ref = P.bn_stats(x[:, None], 0.0)[1][0]
    def one_sweep(d):
        s1, s2 = np.float32(0), np.float32(0)
        for blk in d.reshape(256, 256):                  # float32 partial sums per block, like the producers
            s1 += blk.sum(dtype=np.float32)
            s2 += (blk * blk).sum(dtype=np.float32)
        e1 = np.float64(s1) / d.size
        return np.float64(s2) / d.size - e1 * e1
    assert abs(one_sweep(x) - ref) / ref > 0.5
    assert abs(one_sweep(x - np.float32(1.0e4)) - ref) / ref < 1e-3


def test_running_update_closed_form():
    rm, rv = P.running_update([1.0, -2.0], [4.0, 0.5], [5.0, 2.0], [3.0, 6.0], 4, 0.1)
    np.testing.assert_allclose(rm, [0.9 * 1.0 + 0.1 * 5.0, 0.9 * -2.0 + 0.1 * 2.0], rtol=1e-15)
    np.testing.assert_allclose(rv, [0.9 * 4.0 + 0.1 * 3.0 * 4 / 3, 0.9 * 0.5 + 0.1 * 6.0 * 4 / 3], rtol=1e-15)
    # momentum 1 replaces, 0 keeps; the unbiased variance of torch's BN update
    rm, rv = P.running_update([7.0], [7.0], [1.0], [2.0], 9, 1.0)
    assert rm[0] == 1.0 and rv[0] == 2.0 * 9 / 8
    t = torch.randn(50, 3, 4, 4, dtype=torch.float64)
    run_m, run_v = torch.zeros(3, dtype=torch.float64), torch.ones(3, dtype=torch.float64)
    F.batch_norm(t, run_m, run_v, training=True, momentum=0.1)
    x = t.permute(0, 2, 3, 1).reshape(-1, 3).numpy()
    mean, var, _ = P.bn_stats(x, 0.0)
    rm, rv = P.running_update(np.zeros(3), np.ones(3), mean, var, x.shape[0], 0.1)
    np.testing.assert_allclose(rm, run_m.numpy(), rtol=1e-12)
    np.testing.assert_allclose(rv, run_v.numpy(), rtol=1e-12)


# ----------------------------------------------------------- BN backward ----
def test_bn_bwd_invariants():
    m, C = 777, 6
    x = RNG.standard_normal((m, C)) * 3 - 1
    dy = RNG.standard_normal((m, C))
    for gamma, beta in ((np.ones(C), np.zeros(C)), (RNG.uniform(0.5, 1.5, C), RNG.normal(0, 0.1, C))):
        for eps in (0.0, 1e-5):
            _, mean, var, rstd = P.bn_fwd(x, gamma, beta, eps)
            dx, dgamma, dbeta = P.bn_bwd(x, dy, gamma, mean, rstd)
            assert np.max(np.abs(dx.sum(0))) < 1e-10
            xhat = (x - mean) * rstd
            if eps == 0.0:
                assert np.max(np.abs((dx * xhat).sum(0))) < 1e-10
    # one value per channel, and gamma = 0: dx = 0
    _, mean, var, rstd = P.bn_fwd(x[:1], np.ones(C), np.zeros(C), 1e-5)
    dx, _, _ = P.bn_bwd(x[:1], dy[:1], np.ones(C), mean, rstd)
    np.testing.assert_array_equal(dx, 0.0)
    _, mean, var, rstd = P.bn_fwd(x, np.zeros(C), np.zeros(C), 1e-5)
    dx, _, _ = P.bn_bwd(x, dy, np.zeros(C), mean, rstd)
    np.testing.assert_array_equal(dx, 0.0)


def test_bn_bwd_matches_torch_autograd():
    x = RNG.standard_normal((4, 5, 6, 7))
    gamma, beta = RNG.uniform(0.5, 1.5, 7), RNG.normal(0, 0.1, 7)
    g = RNG.standard_normal(x.shape)
    xt = _nchw(x).requires_grad_()
    gt = torch.from_numpy(gamma).requires_grad_()
    bt = torch.from_numpy(beta).requires_grad_()
    yt = F.batch_norm(xt, None, None, gt, bt, training=True, eps=1e-5)
    (yt * _nchw(g)).sum().backward()
    _, mean, var, rstd = P.bn_fwd(x, gamma, beta, 1e-5)
    dx, dgamma, dbeta = P.bn_bwd(x, g, gamma, mean, rstd)
    np.testing.assert_allclose(dx, _nhwc(xt.grad), rtol=0, atol=1e-11)
    np.testing.assert_allclose(dgamma, gt.grad.numpy(), rtol=1e-11)
    np.testing.assert_allclose(dbeta, bt.grad.numpy(), rtol=1e-11)


# ------------------------------------------------------------------ ReLU ----
def test_relu():
    y = np.array([-2.0, -0.0, 0.0, 1e-300, 3.0])
    np.testing.assert_array_equal(P.relu_fwd(y), [0, 0, 0, 1e-300, 3.0])
    np.testing.assert_array_equal(P.relu_bwd(np.full(5, 7.0), y), [0, 0, 0, 7.0, 7.0])


# ------------------------------------------------------------------ CONV ----
def test_conv1x1_is_matrix_product():
    x = RNG.standard_normal((3, 5, 4, 11))
    w = RNG.standard_normal((1, 1, 11, 6))
    out = P.conv_fwd(x, w)
    np.testing.assert_allclose(out.reshape(-1, 6), x.reshape(-1, 11) @ w[0, 0], rtol=0, atol=1e-12)
    g = RNG.standard_normal(out.shape)
    np.testing.assert_allclose(P.conv_dgrad(g, w, (5, 4)).reshape(-1, 11), g.reshape(-1, 6) @ w[0, 0].T,
                               rtol=0, atol=1e-12)
    np.testing.assert_allclose(P.conv_wgrad(x, g, 1)[0, 0], x.reshape(-1, 11).T @ g.reshape(-1, 6),
                               rtol=0, atol=1e-11)


def test_conv3x3_centre_delta_is_identity():
    x = RNG.standard_normal((2, 4, 5, 3))
    w = np.zeros((3, 3, 3, 3))
    w[1, 1] = np.eye(3)
    np.testing.assert_array_equal(P.conv_fwd(x, w), x)


@pytest.mark.parametrize("K,stride,pad,H,W", [(1, 1, 0, 5, 6), (3, 1, 1, 5, 6), (3, 1, 1, 1, 1),
                                              (7, 2, 3, 11, 10), (3, 2, 1, 7, 7)])
def test_conv_matches_torch(K, stride, pad, H, W):
    x = RNG.standard_normal((2, H, W, 4))
    w = RNG.standard_normal((K, K, 4, 5))
    g = None
    xt = _nchw(x).requires_grad_()
    wt = _oihw(w).requires_grad_()
    out_t = F.conv2d(xt, wt, stride=stride, padding=pad)
    out = P.conv_fwd(x, w, stride, pad)
    np.testing.assert_allclose(out, _nhwc(out_t), rtol=0, atol=1e-12)
    g = RNG.standard_normal(out.shape)
    (out_t * _nchw(g)).sum().backward()
    np.testing.assert_allclose(P.conv_dgrad(g, w, (H, W), stride, pad), _nhwc(xt.grad), rtol=0, atol=1e-12)
    np.testing.assert_allclose(P.conv_wgrad(x, g, K, stride, pad), wt.grad.numpy().transpose(2, 3, 1, 0),
                               rtol=0, atol=1e-11)


def test_conv_adjoint_identities():
    x = RNG.standard_normal((2, 6, 7, 5))
    w = RNG.standard_normal((3, 3, 5, 4))
    out = P.conv_fwd(x, w)
    g = RNG.standard_normal(out.shape)
    lhs = np.sum(out * g)
    np.testing.assert_allclose(np.sum(x * P.conv_dgrad(g, w, (6, 7))), lhs, rtol=1e-12)
    np.testing.assert_allclose(np.sum(w * P.conv_wgrad(x, g, 3)), lhs, rtol=1e-12)


# --------------------------------------------------------------- pooling ----
def test_avgpool2():
    x = RNG.standard_normal((2, 6, 4, 3))
    out = P.avgpool2_fwd(x)
    np.testing.assert_allclose(_nchw(out).numpy(), F.avg_pool2d(_nchw(x), 2).numpy(), rtol=0, atol=1e-14)
    g = RNG.standard_normal(out.shape)
    np.testing.assert_allclose(np.sum(x * P.avgpool2_bwd(g, (6, 4))), np.sum(out * g), rtol=1e-13)


def test_maxpool():
    x = RNG.standard_normal((2, 9, 8, 3))
    out = P.maxpool_fwd(x)
    xt = _nchw(x).requires_grad_()
    ref = F.max_pool2d(xt, 3, 2, 1)
    np.testing.assert_array_equal(out, _nhwc(ref))
    g = RNG.standard_normal(out.shape)
    (ref * _nchw(g)).sum().backward()
    np.testing.assert_allclose(P.maxpool_bwd(x, g), _nhwc(xt.grad), rtol=0, atol=1e-14)
    # ties go to the first maximum in row-major window order
    t = np.zeros((1, 3, 3, 1))
    gi = P.maxpool_bwd(t, np.ones((1, 2, 2, 1)))
    # windows start at (-1,-1), (-1,1), (1,-1), (1,1): first in-image tap of each
    expect = np.zeros((1, 3, 3, 1))
    expect[0, 0, 0] = expect[0, 0, 1] = expect[0, 1, 0] = expect[0, 1, 1] = 1.0
    np.testing.assert_array_equal(gi, expect)


# ------------------------------------------------------------ bf16 cast ----
def test_round_bf16():
    a = np.array([1 + 2.0 ** -8, 1 + 3 * 2.0 ** -8, -(1 + 2.0 ** -8 + 2.0 ** -30), 0.0, 2.0 ** -140,
                  3.0e38, 3.4e38, 1e-40])
    r = P.round_bf16(a)
    assert r[0] == 1.0 and r[1] == 1 + 2.0 ** -6 and r[2] == -(1 + 2.0 ** -7)
    ref = torch.from_numpy(a.astype(np.float32)).to(torch.bfloat16).to(torch.float64).numpy()
    np.testing.assert_array_equal(r[3:], ref[3:])
    x = RNG.standard_normal(100000) * np.exp(RNG.uniform(-20, 20, 100000))
    x32 = x.astype(np.float32).astype(np.float64)          # fp32 inputs: no double rounding
    ref = torch.from_numpy(x32).to(torch.bfloat16).to(torch.float64).numpy()
    np.testing.assert_array_equal(P.round_bf16(x32), ref)


# ----------------------------------------------- finite-difference checks ----
def _fd(f, arr, idx, h=1e-6):
    old = arr[idx]
    arr[idx] = old + h
    lp = f()
    arr[idx] = old - h
    lm = f()
    arr[idx] = old
    return (lp - lm) / (2 * h)


def _check_fd(f, arr, grad, n=12, tol=1e-6):
    flat = arr.reshape(-1)
    gflat = np.asarray(grad).reshape(-1)
    picks = RNG.choice(flat.size, size=min(n, flat.size), replace=False)
    for i in picks:
        num = _fd(f, flat, i)
        assert abs(num - gflat[i]) <= tol * max(1.0, abs(num)), (i, num, gflat[i])


@pytest.mark.parametrize("K", [1, 3])
def test_unit_gradients_finite_difference(K):
    rnd = OC.storage(False)
    x = RNG.standard_normal((2, 3, 3, 3))
    gamma, beta = RNG.uniform(0.5, 1.5, 3), RNG.normal(0, 0.1, 3)
    w = RNG.standard_normal((K, K, 3, 2))
    g = RNG.standard_normal((2, 3, 3, 2))

    def loss():
        return np.sum(OC.unit_fwd(x, gamma, beta, w, 1e-5, rnd)["out"] * g)

    c = OC.unit_fwd(x, gamma, beta, w, 1e-5, rnd)
    b = OC.unit_bwd(c, g, rnd)
    _check_fd(loss, x, b["dx"], n=18)
    _check_fd(loss, gamma, b["dgamma"])
    _check_fd(loss, beta, b["dbeta"])
    _check_fd(loss, w, b["dw"])


def test_bottleneck_gradients_finite_difference():
    rnd = OC.storage(False)
    X = RNG.standard_normal((2, 3, 4, 4))
    p = dict(gamma1=RNG.uniform(0.5, 1.5, 4), beta1=RNG.normal(0, .1, 4), w1=RNG.standard_normal((1, 1, 4, 5)),
             gamma2=RNG.uniform(0.5, 1.5, 5), beta2=RNG.normal(0, .1, 5), w2=RNG.standard_normal((3, 3, 5, 2)))
    dY = RNG.standard_normal((2, 3, 4, 6))

    def loss():
        return np.sum(OC.bottleneck_fwd(X, 2, p, 1e-5, rnd)[0] * dY)

    _, c = OC.bottleneck_fwd(X, 2, p, 1e-5, rnd)
    dX, g = OC.bottleneck_bwd(c, dY, rnd)
    _check_fd(loss, X, dX, n=20)
    _check_fd(loss, p["w1"], g["b1"]["dw"])
    _check_fd(loss, p["w2"], g["b2"]["dw"])
    _check_fd(loss, p["gamma1"], g["b1"]["dgamma"])
    _check_fd(loss, p["beta2"], g["b2"]["dbeta"])


def _tiny_block():
    C0, width, growth, layers = 3, 4, 2, 2
    cpls, c = [], C0
    for _ in range(layers):
        cpls.append(dict(gamma1=RNG.uniform(0.5, 1.5, c), beta1=RNG.normal(0, .1, c),
                         w1=RNG.standard_normal((1, 1, c, width)), gamma2=RNG.uniform(0.5, 1.5, width),
                         beta2=RNG.normal(0, .1, width), w2=RNG.standard_normal((3, 3, width, growth))))
        c += growth
    trans = dict(gamma=RNG.uniform(0.5, 1.5, c), beta=RNG.normal(0, .1, c), w=RNG.standard_normal((1, 1, c, 3)))
    return RNG.standard_normal((2, 4, 4, C0)), cpls, trans, c


def test_block_gradients_finite_difference():
    rnd = OC.storage(False)
    X0, cpls, trans, ct = _tiny_block()
    dp = RNG.standard_normal((2, 2, 2, 3))

    def loss():
        return np.sum(OC.block_fwd(X0, cpls, trans, 1e-5, rnd, ct)[0] * dp)

    _, c = OC.block_fwd(X0, cpls, trans, 1e-5, rnd, ct)
    dX0, g = OC.block_bwd(c, dp, rnd)
    _check_fd(loss, X0, dX0, n=20)
    _check_fd(loss, cpls[0]["w1"], g["cpls"][0]["b1"]["dw"])
    _check_fd(loss, cpls[0]["gamma2"], g["cpls"][0]["b2"]["dgamma"])
    _check_fd(loss, cpls[1]["w2"], g["cpls"][1]["b2"]["dw"])
    _check_fd(loss, trans["w"], g["trans"]["dw"])
    _check_fd(loss, trans["beta"], g["trans"]["dbeta"])


def test_resnet_block_gradients_finite_difference():
    rnd = OC.storage(False)
    C, Wd = 4, 3
    p = dict(w1=RNG.standard_normal((1, 1, C, Wd)), w2=RNG.standard_normal((3, 3, Wd, Wd)),
             w3=RNG.standard_normal((1, 1, Wd, C)))
    for i, ch in ((1, Wd), (2, Wd), (3, C)):
        p["gamma%d" % i], p["beta%d" % i] = RNG.uniform(0.5, 1.5, ch), RNG.normal(0, .1, ch)
    X = RNG.standard_normal((2, 3, 3, C))
    dr = RNG.standard_normal((2, 3, 3, C))

    def loss():
        return np.sum(OC.resnet_block_fwd(X, p, 1e-5, rnd)[0] * dr)

    _, c = OC.resnet_block_fwd(X, p, 1e-5, rnd)
    dX, g = OC.resnet_block_bwd(c, dr, rnd)
    _check_fd(loss, X, dX, n=20)
    _check_fd(loss, p["w1"], g["dw1"])
    _check_fd(loss, p["w2"], g["b2"]["dw"])
    _check_fd(loss, p["gamma3"], g["dgamma3"])
    _check_fd(loss, p["beta1"], g["b2"]["dbeta"])


# ------------------------------------- compositions vs torch nn (forward) ----
def test_block_forward_matches_torch():
    rnd = OC.storage(False)
    X0, cpls, trans, ct = _tiny_block()
    pooled, _ = OC.block_fwd(X0, cpls, trans, 1e-5, rnd, ct)

    def bn_relu_conv(t, gamma, beta, w):
        t = F.batch_norm(t, None, None, torch.from_numpy(gamma), torch.from_numpy(beta), training=True, eps=1e-5)
        k = w.shape[0]
        return F.conv2d(F.relu(t), _oihw(w), padding=k // 2)

    feats = _nchw(X0)
    for p in cpls:
        h = bn_relu_conv(feats, p["gamma1"], p["beta1"], p["w1"])
        h = bn_relu_conv(h, p["gamma2"], p["beta2"], p["w2"])
        feats = torch.cat([feats, h], 1)
    ref = F.avg_pool2d(bn_relu_conv(feats, trans["gamma"], trans["beta"], trans["w"]), 2)
    np.testing.assert_allclose(pooled, _nhwc(ref), rtol=0, atol=1e-12)
    # the transition pooled before its (linear) CONV: the same result in exact arithmetic
    pooled_pf, _ = OC.block_fwd(X0, cpls, trans, 1e-5, rnd, ct, pool_first=True)
    np.testing.assert_allclose(pooled_pf, _nhwc(ref), rtol=0, atol=1e-12)


def test_bf16_pool_first_transition_storage():
    """Pooled before the CONV, the bf16 model stores the pooled CONV operand
    and the pooled output in bf16 and stays within bf16 rounding of the
    conv-then-pool order."""
    rnd = OC.storage(True)
    x = P.round_bf16(RNG.standard_normal((2, 6, 8, 16)))
    g, b = RNG.uniform(0.5, 1.5, 16), RNG.normal(0, 0.1, 16)
    w = P.round_bf16(RNG.standard_normal((1, 1, 16, 8)) * 0.3)
    c, pooled = OC.unit_pool_fwd(x, g, b, w, 1e-5, rnd)
    assert _is_bf16(c["zp"]) and _is_bf16(pooled) and _is_bf16(c["z"])
    ref = P.round_bf16(P.avgpool2_fwd(OC.unit_fwd(x, g, b, w, 1e-5, rnd)["out"]))
    e = np.max(np.abs(pooled - ref)) / np.max(np.abs(ref))
    assert 0 < e < 2e-2, e


def test_bf16_storage_model_rounds_stored_tensors():
    rnd = OC.storage(True)
    x = P.round_bf16(RNG.standard_normal((2, 4, 4, 3)))
    c = OC.unit_fwd(x, np.ones(3), np.zeros(3), P.round_bf16(RNG.standard_normal((3, 3, 3, 2))), 1e-5, rnd)
    for key in ("z", "out"):
        np.testing.assert_array_equal(P.round_bf16(c[key]), c[key])




def _bf16_backward_runs():
    """Every bf16 composition's backward, fed upstream gradients that are NOT
    bf16-representable (fp64 normal draws), so that every rounding site in the
    backward has something to round.  Returns [(name, stored, fp32_results)]:
    the tensors the storage model stores in bf16 and those it keeps in fp32."""
    rnd = OC.storage(True)
    r = lambda a: P.round_bf16(a)
    runs = []
    # bottleneck: dY -> G (initial value), the 3x3 unit's dy, the deferred
    # dx2 handed to the 1x1 unit, its dy, the Split accumulation into G
    X = r(RNG.standard_normal((2, 4, 4, 4)))
    pb = dict(gamma1=RNG.uniform(0.5, 1.5, 4), beta1=RNG.normal(0, .1, 4), w1=r(RNG.standard_normal((1, 1, 4, 5))),
              gamma2=RNG.uniform(0.5, 1.5, 5), beta2=RNG.normal(0, .1, 5), w2=r(RNG.standard_normal((3, 3, 5, 2))))
    _, c = OC.bottleneck_fwd(X, 2, pb, 1e-5, rnd)
    dX, g = OC.bottleneck_bwd(c, RNG.standard_normal((2, 4, 4, 6)), rnd)
    runs.append(("bottleneck", [dX, g["b2"]["g"], g["b2"]["dy"], g["b1"]["g"], g["b1"]["dy"]],
                 [g[b][k] for b in ("b1", "b2") for k in ("dw", "dgamma", "dbeta")]))
    # dense block + transition: the transition's unpooled gradient, G after the
    # transition's BN input gradient and after every reader's addition
    X0, cpls, trans, ct = _tiny_block()
    X0 = r(X0)
    for q in cpls:
        q["w1"], q["w2"] = r(q["w1"]), r(q["w2"])
    trans = dict(trans, w=r(trans["w"]))
    _, c = OC.block_fwd(X0, cpls, trans, 1e-5, rnd, ct)
    dX0, g = OC.block_bwd(c, RNG.standard_normal((2, 2, 2, 3)), rnd)
    stored = [dX0, g["G"], g["trans"]["g"], g["trans"]["dy"]]
    for q in g["cpls"]:
        stored += [q["b1"]["g"], q["b1"]["dy"], q["b2"]["g"], q["b2"]["dy"]]
    runs.append(("block", stored, [g["trans"]["dw"], g["trans"]["dgamma"], g["cpls"][0]["b1"]["dw"],
                                   g["cpls"][1]["b2"]["dbeta"]]))
    # ResNet block: ds, the deferred BN3 gradient, BN2's, BN1's, dX
    C, Wd = 4, 3
    pr = dict(w1=r(RNG.standard_normal((1, 1, C, Wd))), w2=r(RNG.standard_normal((3, 3, Wd, Wd))),
              w3=r(RNG.standard_normal((1, 1, Wd, C))))
    for i, ch in ((1, Wd), (2, Wd), (3, C)):
        pr["gamma%d" % i], pr["beta%d" % i] = RNG.uniform(0.5, 1.5, ch), RNG.normal(0, .1, ch)
    _, c = OC.resnet_block_fwd(r(RNG.standard_normal((2, 3, 3, C))), pr, 1e-5, rnd)
    dX, g = OC.resnet_block_bwd(c, RNG.standard_normal((2, 3, 3, C)), rnd)
    runs.append(("resnet", [dX, g["ds"], g["b3"]["g"], g["b3"]["dy"], g["b2"]["g"], g["b2"]["dy"], g["g1"]],
                 [g["dw1"], g["dgamma3"], g["dbeta3"], g["b2"]["dw"], g["b3"]["dgamma"]]))
    # whole DenseNet: the head BN's input gradient G, the stem BN's dy and input gradient
    from paper_1807_01702_amd import synth
    d = _f64_tree(synth.densenet(seed=5, n=2, hw=16, c_img=3, c_stem=4, growth=2, width=4, blocks=(2, 1),
                                 classes=5, bf16=True))
    _, c = OC.densenet_fwd(d, d["eps"], rnd)
    g = OC.densenet_bwd(c, rnd)
    runs.append(("densenet", [g["blocks"][-1]["G"], g["stem"]["dy"], g["stem"]["g"], g["stem"]["dX"]],
                 [g["stem"]["dw"], g["stem"]["dgamma"], g["head"]["dw"], g["head"]["dgamma"]]))
    return runs


def test_bf16_storage_model_backward_rounding_sites():
    """The bf16 compositions store every backward tensor that the GPU path
    stores (dy, the deferred BN input gradient a CONV's backward consumes,
    the concatenation gradient, dX) in bf16, and keep dW, dgamma, dbeta in
    fp32 (here fp64: not bf16-rounded)."""
    for name, stored, wide in _bf16_backward_runs():
        for i, t in enumerate(stored):
            assert np.any(t != 0), (name, i)
            assert _is_bf16(t), "%s: stored backward tensor %d is not bf16" % (name, i)
        for i, t in enumerate(wide):
            assert not _is_bf16(t), "%s: fp32 result %d was rounded to bf16" % (name, i)


def test_bf16_storage_model_backward_is_a_rounding_of_fp64():
    """With identical bf16 inputs and ReLU decisions that keep a margin, the
    bf16 model's backward differs from the exact composition only by the
    storage roundings: a few bf16 half-ulps (2^-9) per stored tensor, well
    under 2e-2 relative, and not zero (the roundings happen)."""
    r = lambda a: P.round_bf16(a)
    for seed in range(200):
        rng = np.random.default_rng(100 + seed)
        X = r(rng.standard_normal((2, 4, 4, 4)))
        p = dict(gamma1=rng.uniform(0.5, 1.5, 4), beta1=rng.normal(0, .1, 4), w1=r(rng.standard_normal((1, 1, 4, 5))),
                 gamma2=rng.uniform(0.5, 1.5, 5), beta2=rng.normal(0, .1, 5), w2=r(rng.standard_normal((3, 3, 5, 2))))
        dY = r(rng.standard_normal((2, 4, 4, 6)))
        _, ce = OC.bottleneck_fwd(X, 2, p, 1e-5, OC.storage(False))
        _, cb = OC.bottleneck_fwd(X, 2, p, 1e-5, OC.storage(True))
        # the first BN sees identical inputs and statistics on both sides; the
        # second one's input differs by the rounding of the first CONV's output
        if min(float(np.min(np.abs(y))) for y in (ce["u2"]["y"], cb["u2"]["y"])) < 0.01:
            continue                       # a ReLU decision near 0: the two need not agree
        dXe, ge = OC.bottleneck_bwd(ce, dY, OC.storage(False))
        dXb, gb = OC.bottleneck_bwd(cb, dY, OC.storage(True))
        for name, a, b in (("dX", dXb, dXe), ("dy2", gb["b2"]["dy"], ge["b2"]["dy"]),
                           ("dy1", gb["b1"]["dy"], ge["b1"]["dy"]), ("dW1", gb["b1"]["dw"], ge["b1"]["dw"])):
            e = np.max(np.abs(a - b)) / np.max(np.abs(b))
            assert 0 < e < 0.02, (seed, name, e)
        return
    pytest.fail("no seed with a ReLU margin")


# ------------------------------------------------- classifier head (C5) ----
def test_softmax_ce_uniform_logits_closed_form():
    # equal logits: every class has probability 1/K, the loss is ln K and the
    # gradient is (1/K - onehot) / N, whatever the common value
    N, K = 5, 1000
    labels = RNG.integers(0, K, N)
    loss, dl = P.softmax_ce(np.full((N, K), 3.25), labels)
    assert abs(loss - np.log(K)) <= 1e-12
    ref = np.full((N, K), 1.0 / K)
    ref[np.arange(N), labels] -= 1.0
    np.testing.assert_allclose(dl, ref / N, rtol=0, atol=1e-15)
    # a one-hot-dominant row: loss -> 0 and no gradient
    big = np.zeros((1, 4))
    big[0, 2] = 800.0
    l2, d2 = P.softmax_ce(big, [2])
    assert l2 == 0.0 and np.all(np.abs(d2) < 1e-300 + 1e-12)


def test_head_matches_torch():
    N, H, W, C, K = 3, 2, 3, 6, 7
    x = RNG.standard_normal((N, H, W, C))
    wt, b = RNG.standard_normal((C, K)), RNG.standard_normal(K)
    labels = RNG.integers(0, K, N)
    f = P.global_avgpool_fwd(x)
    logits = P.fc_fwd(f, wt, b)
    loss, dl = P.softmax_ce(logits, labels)
    df, dwt, db = P.fc_bwd(f, wt, dl)
    dx = P.global_avgpool_bwd(df, (H, W))
    xt = _nchw(x).requires_grad_(True)
    wtt = torch.from_numpy(wt).requires_grad_(True)
    bt = torch.from_numpy(b).requires_grad_(True)
    lt = F.cross_entropy(F.linear(F.adaptive_avg_pool2d(xt, 1).flatten(1), wtt.T, bt), torch.from_numpy(labels))
    lt.backward()
    assert abs(loss - lt.item()) <= 1e-12
    np.testing.assert_allclose(dwt, wtt.grad.numpy(), rtol=0, atol=1e-13)
    np.testing.assert_allclose(db, bt.grad.numpy(), rtol=0, atol=1e-13)
    np.testing.assert_allclose(dx, _nhwc(xt.grad), rtol=0, atol=1e-13)


def _f64_tree(o):
    """float64 copies of every float array (finite differences perturb them in place)."""
    if isinstance(o, dict):
        return {k: _f64_tree(v) for k, v in o.items()}
    if isinstance(o, list):
        return [_f64_tree(v) for v in o]
    if isinstance(o, np.ndarray) and o.dtype.kind == "f":
        return o.astype(np.float64)
    return o


def _tiny_densenet():
    from paper_1807_01702_amd import synth
    return _f64_tree(synth.densenet(seed=3, n=2, hw=16, c_img=3, c_stem=4, growth=2, width=4, blocks=(2, 1),
                                    classes=5, bf16=False))


def _torch_densenet(d):
    """The same network written with torch CPU fp64 modules (second opinion)."""
    t = lambda a: torch.from_numpy(np.ascontiguousarray(np.asarray(a, np.float64))).requires_grad_(True)
    params = []

    def P_(a):
        p = t(a)
        params.append(p)
        return p

    def bn_relu(h, gamma, beta):
        return F.relu(F.batch_norm(h, None, None, P_(gamma), P_(beta), training=True, eps=d["eps"]))

    def conv(h, w, stride=1, pad=None):
        wt = P_(w)
        k = w.shape[0]
        return F.conv2d(h, wt.permute(3, 2, 0, 1), stride=stride, padding=k // 2 if pad is None else pad)

    st = d["stem"]
    h = conv(_nchw(d["img"]), st["w"], 2, 3)
    h = F.max_pool2d(bn_relu(h, st["gamma"], st["beta"]), 3, 2, 1)
    for b in d["blocks"]:
        for p in b["cpls"]:
            y = conv(bn_relu(h, p["gamma1"], p["beta1"]), p["w1"])
            y = conv(bn_relu(y, p["gamma2"], p["beta2"]), p["w2"])
            h = torch.cat([h, y], 1)
        if b["trans"] is not None:
            tr = b["trans"]
            h = F.avg_pool2d(conv(bn_relu(h, tr["gamma"], tr["beta"]), tr["w"]), 2)
    hp = d["head"]
    f = bn_relu(h, hp["gamma"], hp["beta"]).mean(dim=(2, 3))
    wfc, bfc = P_(hp["w"]), P_(hp["b"])
    loss = F.cross_entropy(f @ wfc + bfc, torch.from_numpy(np.asarray(d["labels"], np.int64)))
    loss.backward()
    return loss.item(), [p.grad.numpy() for p in params]


def _oracle_densenet_grads(d, g):
    """Parameter gradients of the oracle in the order _torch_densenet creates them."""
    out = [g["stem"]["dw"], g["stem"]["dgamma"], g["stem"]["dbeta"]]
    for b, gb in zip(d["blocks"], g["blocks"]):
        for gc in gb["cpls"]:
            out += [gc["b1"]["dgamma"], gc["b1"]["dbeta"], gc["b1"]["dw"], gc["b2"]["dgamma"], gc["b2"]["dbeta"],
                    gc["b2"]["dw"]]
        if b["trans"] is not None:
            out += [gb["trans"]["dgamma"], gb["trans"]["dbeta"], gb["trans"]["dw"]]
    h = g["head"]
    return out + [h["dgamma"], h["dbeta"], h["dw"], h["db"]]


def test_densenet_matches_torch_autograd():
    d = _tiny_densenet()
    rnd = OC.storage(False)
    loss, c = OC.densenet_fwd(d, d["eps"], rnd)
    g = OC.densenet_bwd(c, rnd)
    lt, grads_t = _torch_densenet(d)
    assert abs(loss - lt) <= 1e-12
    ours = _oracle_densenet_grads(d, g)
    assert len(ours) == len(grads_t)
    for i, (a, b) in enumerate(zip(ours, grads_t)):
        b = b.transpose(2, 3, 1, 0) if b.ndim == 4 and np.asarray(a).ndim == 4 and b.shape != np.shape(a) else b
        np.testing.assert_allclose(a, b, rtol=0, atol=1e-11 * max(1.0, float(np.max(np.abs(b)))), err_msg=str(i))


def test_densenet_gradients_finite_difference():
    d = _tiny_densenet()
    rnd = OC.storage(False)

    def loss():
        return OC.densenet_fwd(d, d["eps"], rnd)[0]

    _, c = OC.densenet_fwd(d, d["eps"], rnd)
    g = OC.densenet_bwd(c, rnd)
    _check_fd(loss, d["stem"]["w"], g["stem"]["dw"], n=8)
    _check_fd(loss, d["stem"]["gamma"], g["stem"]["dgamma"], n=4)
    _check_fd(loss, d["blocks"][0]["cpls"][1]["w2"], g["blocks"][0]["cpls"][1]["b2"]["dw"], n=8)
    _check_fd(loss, d["blocks"][0]["trans"]["w"], g["blocks"][0]["trans"]["dw"], n=6)
    _check_fd(loss, d["blocks"][1]["cpls"][0]["beta1"], g["blocks"][1]["cpls"][0]["b1"]["dbeta"], n=4)
    _check_fd(loss, d["head"]["gamma"], g["head"]["dgamma"], n=4)
    _check_fd(loss, d["head"]["w"], g["head"]["dw"], n=8)
    _check_fd(loss, d["head"]["b"], g["head"]["db"], n=5)


def test_densenet121_loss_at_init_near_log_classes():
    # random init, N(0,1) images: the classifier is near uniform at step 0
    from paper_1807_01702_amd import synth
    d = synth.densenet(seed=0, n=1, hw=32, blocks=(1, 1, 1, 1), bf16=False)
    loss, _ = OC.densenet_fwd(d, d["eps"], OC.storage(False))
    assert abs(loss - np.log(1000)) < 1.0, loss
