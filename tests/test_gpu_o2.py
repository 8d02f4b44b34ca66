"""The paper's O2' structure (Sec. 3.2): the fused BN+ReLU+CONV forward also
stores the BN+ReLU output z it feeds to the CONV, and the backward reads z
(ReLU mask, xhat for dgamma, the weight gradient's operand) instead of
recomputing it from x.  Checked against the oracle, and against the
recompute design where the two must agree bit for bit: the forward output and
its statistics, dy and dbeta (the same mask on the same dz), and dW (z holds
exactly the operand the recompute forms)."""
import numpy as np
import pytest
import torch

from helpers import RTOL, assert_close, dev, f32dev, host, relu_ambiguous
from oracle import prims as P
from paper_1807_01702_amd import synth

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def B():
    from paper_1807_01702_amd import bnr
    return bnr


CASES = [
    # bf16, k, n, h, w, c_in, c_out
    (False, 1, 8, 8, 8, 64, 32),          # float32: tiled kernel
    (False, 3, 2, 5, 6, 12, 20),          # float32 3x3, ragged
    (True, 1, 2, 14, 14, 256, 128),       # persistent 1x1
    (True, 1, 1, 9, 11, 40, 136),         # persistent 1x1, ragged channels and pixels
    (True, 3, 2, 14, 14, 128, 32),        # persistent 3x3
    (True, 3, 2, 7, 7, 64, 96),           # persistent 3x3, small images
    (True, 3, 1, 5, 62, 32, 8),           # 3x3 past the persistent kernel's width: tiled kernel
    (True, 1, 1, 9, 11, 288, 40),         # 1x1 with K > 256: tiled kernel
]


def _run(B, case, gamma_zero=False, seed=31):
    bf16, k, n, h, w, ci, co = case
    xf = synth.normal(seed, "x", (n, h, w, ci), bf16=bf16)
    wt = synth.conv_weight(seed, "w", k, ci, co, bf16)
    bp = synth.bn_params(seed, "bn", ci)
    gamma, beta = bp["gamma"].copy(), bp["beta"].copy()
    if gamma_zero:                        # a constant-output channel with a live ReLU and one with a dead ReLU
        gamma[3], beta[3] = 0.0, 0.5
        gamma[ci - 2], beta[ci - 2] = 0.0, -0.5
    gf = synth.normal(seed, "g", (n, h, w, co), bf16=bf16)
    x, wd, g = dev(xf, bf16), dev(wt, bf16), dev(gf, bf16)
    bn = B.BN(f32dev(gamma), f32dev(beta), 1e-5)
    B.bnr_bn_stats(x, bn)
    zl = ci + (8 if bf16 else 4)           # z as a view with a pixel stride past its channels
    zbuf = torch.full((n, h, w, zl), 7.0, dtype=x.dtype, device=x.device)
    z = zbuf[..., :ci]
    y1 = torch.empty((n, h, w, co), dtype=x.dtype, device=x.device)
    y2 = torch.empty_like(y1)
    s1, s2 = B.BN.stats_only(co, x.device), B.BN.stats_only(co, x.device)
    desc = B.desc_for(x, y1, k, n, h, w)
    B.bnr_bn_relu_conv_fwd(desc, x, bn, wd, y1, s1)
    B.bnr_bn_relu_conv_fwd_o2(desc, x, bn, wd, y2, z, s2)
    f32 = dict(dtype=torch.float32, device=x.device)
    out = {}
    for tag in ("re", "o2"):
        out[tag] = dict(dw=torch.empty(wt.shape, **f32), dg=torch.empty(ci, **f32), db=torch.empty(ci, **f32),
                        dy=torch.empty_like(x), dx=torch.empty_like(x))
    r, o = out["re"], out["o2"]
    B.bnr_bwd_fused(desc, x, bn, wd, B.grad_dense(g), r["dw"], r["dg"], r["db"], r["dy"], r["dx"])
    B.bnr_bwd_fused_o2(desc, x, bn, z, wd, B.grad_dense(g), o["dw"], o["dg"], o["db"], o["dy"], o["dx"])
    torch.cuda.synchronize()
    ref = dict(xf=xf, wt=wt, gamma=gamma, beta=beta, gf=gf)
    return (y1, y2, s1, s2, zbuf, z, out, ref)


def _bits(t):
    return t.view(torch.int16 if t.dtype == torch.bfloat16 else torch.int32)


def _eq(name, a, b):
    assert torch.equal(_bits(a), _bits(b)), name


@pytest.mark.parametrize("case", CASES)
def test_o2_against_recompute_and_oracle(B, case):
    bf16, k, n, h, w, ci, co = case
    rnd = P.round_bf16 if bf16 else (lambda a: np.asarray(a, np.float64))
    y1, y2, s1, s2, zbuf, z, out, ref = _run(B, case)
    r, o = out["re"], out["o2"]
    # forward: the same output and statistics; z is the CONV operand, written only inside its view
    _eq("forward output", y1, y2)
    _eq("forward mean", s1.mean, s2.mean)
    _eq("forward var", s1.var, s2.var)
    assert torch.all(zbuf[..., ci:] == 7.0), "z written outside its view"
    x64 = ref["xf"].astype(np.float64)
    yr, mu, var, rstd = P.bn_fwd(x64, ref["gamma"], ref["beta"], 1e-5)
    amb = relu_ambiguous(yr, bf16)
    rt = RTOL[bf16]
    assert_close("z", host(z), rnd(P.relu_fwd(yr)), rt, exclude=amb)
    # backward: dy, dbeta and dW bit for bit as in the recompute design
    _eq("dy", r["dy"], o["dy"])
    _eq("dbeta", r["db"], o["db"])
    _eq("dW", r["dw"], o["dw"])
    # dgamma (xhat from z) and the input gradient against the oracle
    dz = P.conv_dgrad(ref["gf"].astype(np.float64), ref["wt"].astype(np.float64), (h, w))
    dyr = rnd(P.relu_bwd(dz, yr))
    dxr, dgr, dbr = P.bn_bwd(x64, dyr, ref["gamma"], mu, rstd)
    assert_close("dgamma", host(o["dg"]), dgr, rt)
    assert_close("dbeta", host(o["db"]), dbr, rt)
    assert_close("dx", host(o["dx"]), rnd(dxr), rt, exclude=amb)
    # the two designs' dgamma differ only through xhat = (z - beta) / gamma
    # taken from the stored z: per element at most z's rounding over |gamma|
    # (half an ulp: 2^-9 |z| in bf16, 2^-24 |z| in float32) plus float32
    # noise, so per channel at most sum |dy| (2^-8 |z| + 2^-22 (|z| + |beta|)) / |gamma|
    u = 2.0 ** -8 if bf16 else 2.0 ** -23
    za, dya = np.abs(host(z)), np.abs(host(o["dy"]))
    g_abs = np.abs(ref["gamma"]).astype(np.float64)
    bound = (np.sum(dya * (u * za + 2.0 ** -22 * (za + np.abs(ref["beta"]))), axis=(0, 1, 2)) / g_abs +
             1e-6 * np.sum(np.abs(dyr * (x64 - mu) * rstd), axis=(0, 1, 2)))
    diff = np.abs(host(o["dg"]) - host(r["dg"]))
    assert np.all(diff <= bound), "dgamma vs recompute: worst %.3g of its bound" % np.max(diff / bound)


@pytest.mark.parametrize("case", [CASES[0], CASES[2], CASES[4], CASES[6]])
def test_o2_gamma_zero_channels(B, case):
    """A channel with gamma = 0 has the same output at every pixel, so z does
    not determine xhat: the threads whose channel vector holds it read x and
    give exactly the recompute design's dgamma for that vector."""
    bf16, k, n, h, w, ci, co = case
    vec = 8 if bf16 else 4
    _, _, _, _, _, _, out, ref = _run(B, case, gamma_zero=True)
    r, o = out["re"], out["o2"]
    dg_o = host(o["dg"])
    assert np.all(np.isfinite(dg_o))
    for c in (3, ci - 2):
        v = slice(c // vec * vec, c // vec * vec + vec)
        _eq("dgamma of the vector of channel %d" % c, o["dg"][v], r["dg"][v])
    _eq("dy", r["dy"], o["dy"])
    _eq("dW", r["dw"], o["dw"])
    rnd = P.round_bf16 if bf16 else (lambda a: np.asarray(a, np.float64))
    x64 = ref["xf"].astype(np.float64)
    yr, mu, var, rstd = P.bn_fwd(x64, ref["gamma"], ref["beta"], 1e-5)
    dz = P.conv_dgrad(ref["gf"].astype(np.float64), ref["wt"].astype(np.float64), (h, w))
    dyr = rnd(P.relu_bwd(dz, yr))
    _, dgr, _ = P.bn_bwd(x64, dyr, ref["gamma"], mu, rstd)
    assert_close("dgamma", dg_o, dgr, RTOL[bf16])
