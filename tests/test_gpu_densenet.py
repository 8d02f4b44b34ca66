"""Whole-DenseNet parity (GPU): the network's first CONV (7x7/2), the
BN-ReLU-max-pooling layer, the classifier head, and one whole training step,
against the CPU oracle on the same seeded inputs, through the C ABI.

Per-op tests feed both sides identical inputs (the BN statistics are the
oracle's, passed to the kernels in float32):

* first CONV forward with the statistics epilogue: odd output sizes (rows of
  an item and 16-pixel blocks straddle image rows), the full 224x224 image,
  bf16 (every element within one bf16 ulp of the rounded fp64 result) and
  fp32 (1e-5); statistics of the stored outputs at 1e-4;
* BN-ReLU-max pooling forward and backward with gamma of both signs and zero
  (the window's first maximum is taken of sign(gamma) * x) and inputs with
  many exact ties (first-maximum routing), plus plain max pooling;
* first-CONV weight gradient from a dense gradient and from the deferred BN
  input gradient;
* the head (loss, logits, dlogits, FC gradients, head BN gradients in the
  summed form and materialised).

Whole step: fp32 storage at 64x64 and 96x96 images (all four blocks, every
transition, two composite layers per block), every tensor against the pure
fp64 oracle at 1e-4, fused and unfused (ReLU margin precondition checked on
the oracle); bf16 DenseNet-121 at full
224x224 resolution (batch 2), at two composite layers per block and at
DenseNet-121's depth: loss, logits and dlogits, the first CONV, block 1 and
its BN statistics at 2e-2, and the deeper blocks and every parameter
gradient as accuracy equivalence of the fused path with the unfused path.
"""
import numpy as np
import pytest
import torch

from helpers import RTOL, assert_close, assert_close_pixels, assert_stats, bf16_round, dev, f32dev, host
from oracle import compose as OC
from oracle import prims as P
from paper_1807_01702_amd import synth

pytestmark = pytest.mark.gpu


def _B():
    from paper_1807_01702_amd import bnr as B
    return B


def _img4(img, bf16):
    n, h, w, c = img.shape
    a = np.zeros((n, h, w, 4), np.float32)
    a[..., :c] = img
    return dev(a, bf16)


def _bf16_ulp_close(name, gpu, ref):
    """Every element within one bf16 ulp of the rounded fp64 result (the two
    sides round the same exact value from different accumulation orders)."""
    gpu, ref = np.asarray(gpu, np.float64), np.asarray(ref, np.float64)
    ulp = np.exp2(np.floor(np.log2(np.maximum(np.abs(ref), 1e-30))) - 7)
    bad = np.abs(gpu - ref) > ulp + 1e-6 * np.max(np.abs(ref))
    assert not bad.any(), "%s: %d elements off by more than one bf16 ulp" % (name, int(bad.sum()))


def _stats_close(name, mean_g, var_g, mean_r, var_r, rtol):
    """Statistics comparison with the cancellation floor of one-sweep
    statistics: E[x^2] - E[x]^2 from float32 partial sums carries an absolute
    error of order 1e-7 mean^2 (a constant channel has variance 0)."""
    mean_g, var_g = np.asarray(mean_g, np.float64), np.asarray(var_g, np.float64)
    mean_r, var_r = np.asarray(mean_r, np.float64), np.maximum(np.asarray(var_r, np.float64), 0.0)
    em = np.abs(mean_g - mean_r) - (rtol * np.sqrt(var_r) + 1e-6 * np.abs(mean_r))
    ev = np.abs(var_g - var_r) - (rtol * var_r + 1e-6 * mean_r ** 2)
    assert np.all(em <= 0), "%s mean: channel %d" % (name, int(np.argmax(em)))
    assert np.all(ev <= 0), "%s var: channel %d" % (name, int(np.argmax(ev)))


# ------------------------------------------------------------ first CONV ----
@pytest.mark.parametrize("bf16", [True, False])
@pytest.mark.parametrize("n,h,w", [(2, 30, 30), (3, 17, 33), (1, 224, 224)])
def test_stem_conv_fwd_stats(bf16, n, h, w):
    B = _B()
    img = synth.normal(0, "img", (n, h, w, 3), bf16=bf16)
    wt = synth.conv_weight(0, "w", 7, 3, 64, bf16)
    ref = P.conv_fwd(img, wt, stride=2, pad=3)
    if bf16:
        ref = P.round_bf16(ref)
    ho, wo = (h - 1) // 2 + 1, (w - 1) // 2 + 1
    s = torch.empty((n, ho, wo, 64), dtype=torch.bfloat16 if bf16 else torch.float32, device="cuda")
    bn = B.BN.stats_only(64, "cuda")
    B.bnr_stem_conv_fwd(_img4(img, bf16), dev(wt, bf16), s, bn)
    torch.cuda.synchronize()
    got = host(s)
    if bf16:
        _bf16_ulp_close("first conv", got, ref)
    else:
        assert_close("first conv", got, ref, 1e-5)
    mean, var = P.mvf_stats(got)             # statistics of the values as stored
    _stats_close("first conv stats", host(bn.mean), host(bn.var), mean, var, 1e-4)


@pytest.mark.parametrize("bf16", [True, False])
@pytest.mark.parametrize("kind", ["bn", "dense"])
def test_stem_wgrad(bf16, kind):
    B = _B()
    n, h, w = 2, 30, 26
    ho, wo = (h - 1) // 2 + 1, (w - 1) // 2 + 1
    img = synth.normal(0, "img", (n, h, w, 3), bf16=bf16)
    s = synth.normal(0, "s", (n, ho, wo, 64), bf16=bf16) * 0.7 + 0.2
    s = bf16_round(s) if bf16 else s.astype(np.float64)
    gamma, beta = synth.uniform(0, "g", (64,), 0.5, 1.5), synth.normal(0, "b", (64,), 0.1)
    dy = synth.normal(0, "dy", (n, ho, wo, 64), bf16=bf16)
    dw = torch.empty((7, 7, 3, 64), dtype=torch.float32, device="cuda")
    if kind == "bn":
        _, mean, var, rstd = P.bn_fwd(s, gamma, beta, 1e-5)
        mean32, rstd32 = mean.astype(np.float32), rstd.astype(np.float32)
        dx, dg, db = P.bn_bwd(s, dy, gamma, mean32, rstd32)
        g = P.round_bf16(dx) if bf16 else dx
        bn = B.BN(f32dev(gamma), f32dev(beta), 1e-5, mean=f32dev(mean32), rstd=f32dev(rstd32))
        dyt, st = dev(dy, bf16), dev(s, bf16)
        dgt, dbt = f32dev(dg), f32dev(db)
        B.bnr_stem_wgrad(_img4(img, bf16), 3, B.grad_bn(dyt, st, bn, dgt, dbt), dw)
    else:
        g = np.asarray(dy, np.float64)
        B.bnr_stem_wgrad(_img4(img, bf16), 3, B.grad_dense(dev(dy, bf16)), dw)
    torch.cuda.synchronize()
    ref = P.conv_wgrad(img, g, 7, stride=2, pad=3)
    # bf16: the deferred gradient is rounded to bf16 on each side from float32
    # vs float64 coefficients: a few elements may round to neighbouring values
    assert_close("first conv dW", host(dw), ref, 2e-3 if (bf16 and kind == "bn") else (1e-5 if not bf16 else 1e-4))


# ------------------------------------------------------- max pooling ----
def _pool_inputs(n, h, w, c, bf16, seed=0):
    """Inputs with many exact ties; gamma of both signs and a zero."""
    s = np.round(synth.normal(seed, "s", (n, h, w, c)) * 3.0) / 4.0 + 0.25
    s = s.astype(np.float64)
    gamma = synth.uniform(seed, "g", (c,), 0.5, 1.5).astype(np.float64)
    gamma[1::5] *= -1.0
    gamma[3] = 0.0
    beta = synth.normal(seed, "b", (c,), 0.3).astype(np.float64)
    beta[3] = 0.7                                    # gamma = 0: constant positive output
    return s, gamma, beta


@pytest.mark.parametrize("bf16", [True, False])
@pytest.mark.parametrize("n,h,w", [(2, 112, 112), (2, 15, 15), (1, 13, 30)])
def test_bn_relu_maxpool_fwd(bf16, n, h, w):
    B = _B()
    c = 64
    s, gamma, beta = _pool_inputs(n, h, w, c, bf16)
    y, mean, var, rstd = P.bn_fwd(s, gamma, beta, 1e-5)
    mean32, rstd32 = mean.astype(np.float32), rstd.astype(np.float32)
    y = (s - mean32.astype(np.float64)) * rstd32.astype(np.float64) * gamma + beta    # BN with the float32 statistics
    ref = P.maxpool_fwd(P.relu_fwd(y), 3, 2, 1)
    if bf16:
        ref = P.round_bf16(ref)
    ho, wo = (h - 1) // 2 + 1, (w - 1) // 2 + 1
    buf = torch.zeros((n, ho, wo, c + 16), dtype=torch.bfloat16 if bf16 else torch.float32, device="cuda")
    bn = B.BN(f32dev(gamma), f32dev(beta), 1e-5, mean=f32dev(mean32), rstd=f32dev(rstd32))
    out_bn = B.BN.stats_only(c, "cuda")
    B.bnr_bn_relu_maxpool_fwd(dev(s, bf16), bn, buf[..., 8:8 + c], n, h, w, y_bn=out_bn)
    torch.cuda.synchronize()
    got = host(buf)
    if bf16:
        _bf16_ulp_close("bn-relu-maxpool", got[..., 8:8 + c], ref)
    else:
        assert_close("bn-relu-maxpool", got[..., 8:8 + c], ref, 1e-6)
    assert not np.any(got[..., :8]) and not np.any(got[..., 8 + c:]), "write outside the output view"
    m2, v2 = P.mvf_stats(got[..., 8:8 + c])
    _stats_close("pooled stats", host(out_bn.mean), host(out_bn.var), m2, v2, 1e-4)
    # plain max pooling of the stored ReLU output
    z = P.relu_fwd(s)
    zt = dev(z, bf16)
    out = torch.empty((n, ho, wo, c), dtype=zt.dtype, device="cuda")
    B.bnr_bn_relu_maxpool_fwd(zt, None, out, n, h, w)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(host(out), P.maxpool_fwd(host(zt), 3, 2, 1))


@pytest.mark.parametrize("bf16", [True, False])
@pytest.mark.parametrize("n,h,w", [(2, 112, 112), (2, 15, 15), (1, 13, 30)])
def test_maxpool_bn_bwd(bf16, n, h, w):
    B = _B()
    c = 64
    s, gamma, beta = _pool_inputs(n, h, w, c, bf16, seed=1)
    _, mean, var, rstd = P.bn_fwd(s, gamma, beta, 1e-5)
    mean32, rstd32 = mean.astype(np.float32), rstd.astype(np.float32)
    y = (s - mean32.astype(np.float64)) * rstd32.astype(np.float64) * gamma + beta
    z = P.relu_fwd(y)
    ho, wo = (h - 1) // 2 + 1, (w - 1) // 2 + 1
    gy = synth.normal(1, "gy", (n, ho, wo, c), bf16=bf16).astype(np.float64)
    dz = P.maxpool_bwd(z, gy, 3, 2, 1)
    dy_ref = P.relu_bwd(dz, y)
    if bf16:
        dy_ref = P.round_bf16(dy_ref)
    _, dg_ref, db_ref = P.bn_bwd(s, dy_ref, gamma, mean32, rstd32, want_dx=False)
    bn = B.BN(f32dev(gamma), f32dev(beta), 1e-5, mean=f32dev(mean32), rstd=f32dev(rstd32))
    gbuf = torch.zeros((n, ho, wo, c + 8), dtype=torch.bfloat16 if bf16 else torch.float32, device="cuda")
    gbuf[..., :c] = dev(gy, bf16)
    dyt = torch.empty((n, h, w, c), dtype=gbuf.dtype, device="cuda")
    dg, db = torch.empty(c, dtype=torch.float32, device="cuda"), torch.empty(c, dtype=torch.float32, device="cuda")
    B.bnr_maxpool_bn_bwd(dev(s, bf16), bn, gbuf[..., :c], dyt, n, h, w, dg, db)
    torch.cuda.synchronize()
    amb = (np.abs(y) <= 1e-6 * np.max(np.abs(y))).reshape(-1, c).any(axis=1)
    # bf16: the two sides may round a sum of window gradients to neighbouring values
    assert_close_pixels("pool bwd dy", host(dyt), dy_ref, 4e-3 if bf16 else 1e-6, amb)
    scale_b = np.abs(dy_ref).reshape(-1, c).sum(0).max()
    np.testing.assert_allclose(host(db), db_ref, rtol=0, atol=1e-5 * scale_b)
    np.testing.assert_allclose(host(dg), dg_ref, rtol=0, atol=1e-5 * scale_b * np.abs(y).max())
    # plain max-pooling backward on the stored ReLU output (exact ties included)
    zt = dev(P.relu_fwd(s), bf16)
    dzt = torch.empty_like(dyt)
    B.bnr_maxpool_bn_bwd(zt, None, gbuf[..., :c], dzt, n, h, w)
    torch.cuda.synchronize()
    assert_close("plain pool bwd", host(dzt), P.maxpool_bwd(host(zt), gy, 3, 2, 1), 1e-6 if not bf16 else 4e-3)


# -------------------------------------------------------------- head ----
@pytest.mark.parametrize("bf16", [True, False])
def test_head(bf16):
    B = _B()
    n, h, w, c, K = 6, 7, 7, 96, 130
    x = synth.normal(0, "x", (n, h, w, c)).astype(np.float64) * 0.8 + 0.1
    x = bf16_round(x) if bf16 else x.astype(np.float32).astype(np.float64)
    gamma, beta = synth.uniform(0, "g", (c,), 0.5, 1.5), synth.normal(0, "b", (c,), 0.1)
    wfc = synth.normal(0, "wfc", (c, K), std=float(1 / np.sqrt(c)), bf16=bf16).astype(np.float64)
    bfc = synth.normal(0, "bfc", (K,), 0.1)
    labels = synth._gen(0, "labels").integers(0, K, size=n).astype(np.int32)
    _, mean, var, rstd = P.bn_fwd(x, gamma, beta, 1e-5)
    mean32, rstd32 = mean.astype(np.float32), rstd.astype(np.float32)
    y = (x - mean32.astype(np.float64)) * rstd32.astype(np.float64) * gamma + beta
    f = P.global_avgpool_fwd(P.relu_fwd(y))
    logits = P.fc_fwd(f, wfc, bfc)
    loss, dlogits = P.softmax_ce(logits, labels)
    df, dwfc, dbfc = P.fc_bwd(f, wfc, dlogits)
    dy = P.relu_bwd(P.global_avgpool_bwd(df, (h, w)), y)
    dx, dgam, dbet = P.bn_bwd(x, dy, gamma, mean32, rstd32)
    bn = B.BN(f32dev(gamma), f32dev(beta), 1e-5, mean=f32dev(mean32), rstd=f32dev(rstd32))
    xt, wt = dev(x, bf16), dev(wfc, bf16)
    f32 = dict(dtype=torch.float32, device="cuda")
    ft, lg, dl, ls = torch.empty((n, c), **f32), torch.empty((n, K), **f32), torch.empty((n, K), **f32), torch.empty(1 + n, **f32)
    lab = torch.from_numpy(labels).cuda()
    B.bnr_head_fwd(xt, bn, wt, f32dev(bfc), lab, ft, lg, dl, ls, n, h, w)
    torch.cuda.synchronize()
    assert abs(float(host(ls)[0]) - loss) <= 1e-5 * abs(loss)
    rows = host(ls)[1:]
    assert np.all(np.isfinite(rows)) and abs(rows.mean() - loss) <= 1e-5 * abs(loss)
    assert_close("f", host(ft), f, 1e-5)
    assert_close("logits", host(lg), logits, 1e-5)
    assert_close("dlogits", host(dl), dlogits, 1e-5)
    dft, dwt, dbt = torch.empty((n, c), **f32), torch.empty((c, K), **f32), torch.empty(K, **f32)
    dg, db = torch.empty(c, **f32), torch.empty(c, **f32)
    al, bp = torch.empty(c, **f32), torch.empty(c, **f32)
    G = torch.empty_like(xt)
    B.bnr_head_bwd(xt, bn, wt, ft, dl, dft, dwt, dbt, dg, db, G, n, h, w, alpha=al, betap=bp)
    torch.cuda.synchronize()
    amb = (np.abs(y) <= 1e-6 * np.max(np.abs(y))).reshape(-1, c).any(axis=1)
    assert not amb.any()
    assert_close("df", host(dft), df, 1e-5)
    assert_close("dWfc", host(dwt), dwfc, 1e-5)
    assert_close("dbfc", host(dbt), dbfc, 1e-5)
    assert_close("head dgamma", host(dg), dgam, 1e-5)
    assert_close("head dbeta", host(db), dbet, 1e-5)
    k = gamma * rstd32
    assert_close("summed term D", host(G), k * dy, RTOL[bf16] if bf16 else 1e-5)
    m = n * h * w
    assert_close("alpha", host(al), -k * dbet / m, 1e-5)
    assert_close("betap", host(bp), -k * dgam / m, 1e-5)
    xh = (x - mean32) * rstd32
    assert_close("D + alpha + betap xhat", host(G) + host(al) + host(bp) * xh, dx, RTOL[bf16] if bf16 else 1e-5)
    # materialised input gradient
    B.bnr_head_bwd(xt, bn, wt, ft, dl, dft, dwt, dbt, dg, db, G, n, h, w)
    torch.cuda.synchronize()
    assert_close("head dx", host(G), dx, RTOL[bf16] if bf16 else 1e-5)


# ------------------------------------------------------- whole network ----
def _margin(c):
    """Smallest |y| / max|y| over every BN output whose ReLU decides a gradient."""
    ys = [c["stem"]["y"], c["head"]["y"]]
    for cb in c["blocks"]:
        for cc in cb["cpls"]:
            ys += [cc["u1"]["y"], cc["u2"]["y"]]
        if "ut" in cb:
            ys.append(cb["ut"]["y"])
    return min(float(np.min(np.abs(y)) / np.max(np.abs(y))) for y in ys)


def _sum_scales(dy, x, mean, rstd):
    """Scales of the BN-backward reductions dbeta = sum(dy), dgamma = sum(dy *
    xhat): the largest per-channel sum of |terms|.  A reduction's rounding
    error is bounded relative to that, not to the (possibly cancelling) sum."""
    dy = np.asarray(dy, np.float64)
    C = dy.shape[-1]
    dy = dy.reshape(-1, C)
    xh = (np.asarray(x, np.float64).reshape(-1, C) - mean) * rstd
    return float(np.abs(dy).sum(0).max()), float(np.abs(dy * xh).sum(0).max())


def _param_grads(wl, c, g):
    """(name, gpu tensor, oracle array, scale or None) of every parameter
    gradient; None: the max-norm of the oracle tensor."""
    st, gs = c["stem"], g["stem"]
    sb, sg = _sum_scales(gs["dy"], st["s"], st["mean"], st["rstd"])
    hd = c["head"]
    dy5 = P.relu_bwd(P.global_avgpool_bwd(g["head"]["df"], hd["x"].shape[1:3]), hd["y"])
    hb, hg = _sum_scales(dy5, hd["x"], hd["mean"], hd["rstd"])
    out = [("dW0", wl.dw0, gs["dw"], None), ("dgamma0", wl.g0.dgamma, gs["dgamma"], sg),
           ("dbeta0", wl.g0.dbeta, gs["dbeta"], sb), ("dWfc", wl.dwfc, g["head"]["dw"], None),
           ("dbfc", wl.dbfc, g["head"]["db"], None), ("dgamma5", wl.g5.dgamma, g["head"]["dgamma"], hg),
           ("dbeta5", wl.g5.dbeta, g["head"]["dbeta"], hb)]
    for i, (stg, cb, gb) in enumerate(zip(wl.stages, c["blocks"], g["blocks"])):
        if stg.ut is not None:
            bt, ut = gb["trans"], cb["ut"]
            tb, tg = _sum_scales(bt["dy"], ut["x"], ut["mean"], ut["rstd"])
            out += [("b%d trans dW" % i, stg.ut.dw, bt["dw"], None),
                    ("b%d trans dgamma" % i, stg.ut.g.dgamma, bt["dgamma"], tg),
                    ("b%d trans dbeta" % i, stg.ut.g.dbeta, bt["dbeta"], tb)]
        for l, ((c_l, k, u1, u2), cc, gg) in enumerate(zip(stg.cpl, cb["cpls"], gb["cpls"])):
            for nm, u, uc, bb in (("1", u1, cc["u1"], gg["b1"]), ("2", u2, cc["u2"], gg["b2"])):
                ub, ug = _sum_scales(bb["dy"], uc["x"], uc["mean"], uc["rstd"])
                out += [("b%d l%d dW%s" % (i, l, nm), u.dw, bb["dw"], None),
                        ("b%d l%d dgamma%s" % (i, l, nm), u.g.dgamma, bb["dgamma"], ug),
                        ("b%d l%d dbeta%s" % (i, l, nm), u.g.dbeta, bb["dbeta"], ub)]
    return out


def _check_grads(wl, c, g, rt):
    bad = []
    for name, t, ref, scale in _param_grads(wl, c, g):
        got = host(t)
        sc = scale if scale is not None else float(np.max(np.abs(ref)))
        e = float(np.max(np.abs(got - ref))) / max(sc, 1e-30)
        if e > rt:
            bad.append("%s %.2e" % (name, e))
    assert not bad, "relative errors over %.0e: %s" % (rt, ", ".join(bad))


def _check_forward(wl, loss, c, rt):
    assert abs(float(host(wl.loss)[0]) - loss) <= rt * abs(loss), (float(host(wl.loss)[0]), loss)
    assert_close("logits", host(wl.logits), c["head"]["logits"], rt)
    assert_close("first conv output", host(wl.s), c["stem"]["s"], rt)
    assert_stats("first bn", host(wl.stem_bn.mean), host(wl.stem_bn.var), c["stem"]["mean"], c["stem"]["var"], rt)
    for i, (st, cb) in enumerate(zip(wl.stages, c["blocks"])):
        assert_close("block %d buffer" % i, host(st.X), cb["buf"], rt)
        for l, ((c_l, k, u1, u2), cc) in enumerate(zip(st.cpl, cb["cpls"])):
            assert_stats("b%d l%d bn1" % (i, l), host(u1.bn.mean), host(u1.bn.var), cc["u1"]["mean"], cc["u1"]["var"], rt)
            assert_stats("b%d l%d bn2" % (i, l), host(u2.bn.mean), host(u2.bn.var), cc["u2"]["mean"], cc["u2"]["var"], rt)
        if st.ut is not None:
            assert_stats("b%d trans bn" % i, host(st.ut.bn.mean), host(st.ut.bn.var), cb["ut"]["mean"],
                         cb["ut"]["var"], rt)
    assert_stats("head bn", host(wl.head_bn.mean), host(wl.head_bn.var), c["head"]["mean"], c["head"]["var"], rt)


# (batch, image size, seed) at two composite layers per block: every BN
# normalises over at least 8 values per channel (smaller batches of pixels
# make the normalisation itself ill-conditioned at fp32) and every ReLU
# decision has margin >= 1e-6 (seeds chosen on the oracle).
@pytest.mark.parametrize("fused", [True, False])
@pytest.mark.parametrize("n,hw,seed", [(2, 64, 16), (1, 96, 17)])
def test_densenet_fp32_all_tensors(fused, n, hw, seed):
    from paper_1807_01702_amd import workloads as W
    d = synth.densenet(seed=seed, n=n, hw=hw, blocks=(2, 2, 2, 2), bf16=False)
    rnd = OC.storage(False)
    loss, c = OC.densenet_fwd(d, d["eps"], rnd, pool_first=fused)     # the fused transitions pool first
    assert _margin(c) >= 1e-6, "precondition: ReLU decisions must be unique at fp32 accuracy"
    g = OC.densenet_bwd(c, rnd)
    wl = W.DenseNet(d, fused=fused)
    wl.step()
    torch.cuda.synchronize()
    first = [host(t) for _, t, _, _ in _param_grads(wl, c, g)]
    wl.step()
    torch.cuda.synchronize()
    for a, (name, t, _, _) in zip(first, _param_grads(wl, c, g)):
        np.testing.assert_array_equal(a, host(t), err_msg=name)          # no state leaks between steps
    rt = RTOL[False]
    _check_forward(wl, loss, c, rt)
    assert_close("dX block 1", host(wl.stages[0].G[..., :wl.stages[0].c0]), g["stem"]["dX"], rt)
    _check_grads(wl, c, g, rt)


def _l2(a, b):
    a, b = np.asarray(a, np.float64), np.asarray(b, np.float64)
    return float(np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-30))


def _stats_rms(bn, mean_r, var_r):
    """RMS over channels of the mean error in units of sigma, and the relative
    L2 error of the variances."""
    mg, vg = host(bn.mean), host(bn.var)
    sig = np.sqrt(np.maximum(var_r, 1e-30))
    return float(np.sqrt(np.mean(((mg - mean_r) / sig) ** 2))), _l2(vg, var_r)


@pytest.mark.parametrize("blocks", [(2, 2, 2, 2), (6, 12, 24, 16)], ids=["depth2", "densenet121"])
def test_densenet_bf16_full_resolution(blocks):
    """bf16 DenseNet at 224x224 (batch 2).  Element-wise at 2e-2: the loss,
    the logits and their gradient, the first CONV, block 1 and the
    statistics of every BN up to block 1's transition.  The deeper blocks
    (buffers, BN statistics) and every parameter gradient (the classifier's
    included: it multiplies the last block's features) have no unique result
    at 2e-2 in bf16: each storage rounding of either side may land one ulp
    apart and the differences compound through the later layers (block 4's
    BNs normalise over 98 pixels; at DenseNet-121's depth both GPU paths'
    gradients sit at a median relative distance of about 0.07 from the
    oracle, 0.02 at two layers per block).  There the fused path must be as
    accurate as the unfused path in aggregate, since the two paths'
    per-tensor distances scatter independently once the forward passes have
    diverged (relative L2 / RMS distance to the oracle; BN reductions by their
    largest error over the sum of |terms|, since they cancel): median within
    15%, no tensor more than twice the unfused path's distance.  The exact
    checks of the same composition are the fp32 test above and the per-op
    tests."""
    from paper_1807_01702_amd import workloads as W
    d = synth.densenet(seed=0, n=2, blocks=blocks)
    rnd = OC.storage(True)
    rt = RTOL[True]
    errs, names = {}, []
    for fused in (True, False):
        # each path against the oracle with its own transition order (the
        # fused transitions pool before the CONV: rounding at other sites)
        loss, c = OC.densenet_fwd(d, d["eps"], rnd, pool_first=fused)
        g = OC.densenet_bwd(c, rnd)
        wl = W.DenseNet(d, fused=fused)
        wl.step()
        torch.cuda.synchronize()
        assert abs(float(host(wl.loss)[0]) - loss) <= rt * abs(loss), (float(host(wl.loss)[0]), loss)
        assert_close("logits", host(wl.logits), c["head"]["logits"], rt)
        assert_close("dlogits", host(wl.dlogits), c["head"]["dlogits"], rt)
        assert_close("first conv output", host(wl.s), c["stem"]["s"], rt)
        assert_close("block 1 buffer", host(wl.stages[0].X), c["blocks"][0]["buf"], rt)
        assert_stats("first bn", host(wl.stem_bn.mean), host(wl.stem_bn.var), c["stem"]["mean"], c["stem"]["var"], rt)
        st0, cb0 = wl.stages[0], c["blocks"][0]
        for l, ((c_l, k, u1, u2), cc) in enumerate(zip(st0.cpl, cb0["cpls"])):
            assert_stats("b0 l%d bn1" % l, host(u1.bn.mean), host(u1.bn.var), cc["u1"]["mean"], cc["u1"]["var"], rt)
            assert_stats("b0 l%d bn2" % l, host(u2.bn.mean), host(u2.bn.var), cc["u2"]["mean"], cc["u2"]["var"], rt)
        assert_stats("b0 trans bn", host(st0.ut.bn.mean), host(st0.ut.bn.var), cb0["ut"]["mean"], cb0["ut"]["var"],
                     rt)
        e, nm = [], []
        for i, (st, cb) in enumerate(zip(wl.stages[1:], c["blocks"][1:]), 1):
            e.append(_l2(host(st.X), cb["buf"]))
            nm.append("block %d buffer" % i)
            for l, ((c_l, k, u1, u2), cc) in enumerate(zip(st.cpl, cb["cpls"])):
                for which, u, uc in (("1", u1, cc["u1"]), ("2", u2, cc["u2"])):
                    e += list(_stats_rms(u.bn, uc["mean"], uc["var"]))
                    nm += ["b%d l%d bn%s mean" % (i, l, which), "b%d l%d bn%s var" % (i, l, which)]
            if st.ut is not None:
                e += list(_stats_rms(st.ut.bn, cb["ut"]["mean"], cb["ut"]["var"]))
                nm += ["b%d trans mean" % i, "b%d trans var" % i]
        e += list(_stats_rms(wl.head_bn, c["head"]["mean"], c["head"]["var"]))
        nm += ["head bn mean", "head bn var"]
        for name, t, ref, scale in _param_grads(wl, c, g):
            got = host(t)
            # BN reductions: error relative to the sum of |terms| (they cancel)
            e.append(_l2(got, ref) if scale is None else float(np.max(np.abs(got - ref))) / max(scale, 1e-30))
            nm.append(name)
        errs[fused] = np.array(e)
        names = nm
        del wl
    ef, eu = errs[True], errs[False]
    order = np.argsort(-(ef - 2.0 * eu))
    for j in order[:8]:
        print("%-24s fused %.3e unfused %.3e" % (names[j], ef[j], eu[j]))
    print("relative L2 / RMS to the oracle: fused max %.3e median %.3e; unfused max %.3e median %.3e" % (
        ef.max(), np.median(ef), eu.max(), np.median(eu)))
    assert np.median(ef) <= 1.15 * np.median(eu), (np.median(ef), np.median(eu))
    worse = [names[j] for j in range(len(ef)) if ef[j] > 2.0 * eu[j] + 2e-3]
    assert not worse, worse
