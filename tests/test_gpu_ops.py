"""Per-entry-point parity of the HIP path against the CPU oracle (GPU).

Each test feeds identical seeded synthetic inputs to one C-ABI call and to
the fp64 oracle, at sizes the oracle finishes in seconds that still span
several tiles, a ragged pixel tail and channel counts that are not multiples
of the tile.
"""
import numpy as np
import pytest
import torch

from helpers import RTOL, assert_close, assert_stats, dev, f32dev, host, rel_err, relu_ambiguous
from oracle import prims as P
from paper_1807_01702_amd import synth

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def B():
    from paper_1807_01702_amd import bnr
    return bnr


def _bn_dev(gamma, beta, eps=1e-5):
    from paper_1807_01702_amd import bnr
    return bnr.BN(f32dev(gamma), f32dev(beta), eps)


# ------------------------------------------------------ standalone stats ----
@pytest.mark.parametrize("m,c,ldc,bf16,shift", [
    (512, 64, 64, False, 0.0),          # single-layer input, fp32
    (6272, 256, 288, True, 0.0),        # bottleneck input view of a 288-channel buffer
    (1, 8, 8, True, 0.0),               # one pixel: var = 0
    (7, 24, 40, False, 0.0),            # ragged
    (3001, 200, 256, True, 3.0),        # channel block tail, shifted mean
    (20000, 64, 64, False, 30.0),       # |mean| / sigma = 30 (one-pass statistics precision)
])
def test_bn_stats(B, m, c, ldc, bf16, shift):
    full = synth.normal(0, "stats", (m, ldc), bf16=bf16) + np.float32(shift)
    full = synth.round_to_bf16(full) if bf16 else full
    x = dev(full, bf16)
    bn = B.BN.stats_only(c, x.device)
    B.bnr_bn_stats(x[:, :c], bn)
    torch.cuda.synchronize()
    mean_r, var_r, rstd_r = P.bn_stats(full[:, :c].astype(np.float64), 1e-5)
    if m == 1:
        assert np.all(host(bn.var) == 0) and np.allclose(host(bn.mean), full[0, :c])
        return
    assert_stats("stats", host(bn.mean), host(bn.var), mean_r, var_r, RTOL[bf16])
    np.testing.assert_allclose(host(bn.rstd), rstd_r, rtol=RTOL[bf16])


def _poison_workspace(B, nbytes, device):
    """Grow the binding's workspace to nbytes and fill it with 0xFF bytes
    (NaN as float32): a combine that read a partial row its sweep did not
    write would return NaN."""
    B.workspace(nbytes, device)
    B._ws_cache[(torch.device(device), 0)].fill_(255)


@pytest.mark.parametrize("bf16", [False, True])
def test_stats_rows_launched_equal_rows_combined(B, bf16):
    """m = 20*56*56 = 62720 pixels of 64 channels: 123 rows per block give 510
    launched row blocks, fewer than the 512 the sizing rule aims at.  The
    standalone sweep and the unfused path's two-pass sweeps and backward sums
    must combine exactly the launched rows (workspace poisoned with NaN)."""
    n, h, w, c, co = 20, 56, 56, 64, 32
    m = n * h * w
    xf = synth.normal(7, "stats_rows", (n, h, w, c), bf16=bf16)
    x = dev(xf, bf16)
    bn = B.BN.stats_only(c, x.device)
    _poison_workspace(B, B.bnr_stats_workspace_size(m, c), x.device)
    B.bnr_bn_stats(x, bn)
    torch.cuda.synchronize()
    x64 = xf.reshape(m, c).astype(np.float64)
    mean_r, var_r, _ = P.bn_stats(x64, 1e-5)
    assert_stats("stats", host(bn.mean), host(bn.var), mean_r, var_r, RTOL[bf16])
    if bf16:
        return
    # unfused chain (fp32): two-pass statistics, then the backward reductions
    wt = synth.conv_weight(7, "w", 1, c, co, False)
    bp = synth.bn_params(7, "bn", c)
    gf = synth.normal(7, "g", (n, h, w, co), bf16=False)
    out = torch.empty((n, h, w, co), dtype=torch.float32, device=x.device)
    desc = B.desc_for(x, out, 1, n, h, w)
    rbn = _bn_dev(bp["gamma"], bp["beta"])
    y, z = torch.empty_like(x), torch.empty_like(x)
    wd = dev(wt, False)
    _poison_workspace(B, B.bnr_workspace_size(desc), x.device)
    B.bnr_reference_path(B.MODE_BASELINE, False, desc, x, rbn, wd, y, z=z, out=out)
    dz, dy, dx = torch.empty_like(x), torch.empty_like(x), torch.empty_like(x)
    dw = torch.empty(tuple(wt.shape), dtype=torch.float32, device=x.device)
    dg = torch.empty(c, dtype=torch.float32, device=x.device)
    db = torch.empty_like(dg)
    _poison_workspace(B, B.bnr_workspace_size(desc), x.device)
    B.bnr_reference_path(B.MODE_BASELINE, True, desc, x, rbn, wd, y, z=z, g=dev(gf, False), dz=dz, dy=dy, dw=dw,
                         dgamma=dg, dbeta=db, dx=dx)
    torch.cuda.synchronize()
    yr, mu, var, rstd = P.bn_fwd(x64, bp["gamma"], bp["beta"], 1e-5)
    assert_stats("two-pass stats", host(rbn.mean), host(rbn.var), mu, var, 1e-4)
    dzr = P.conv_dgrad(gf.astype(np.float64), wt.astype(np.float64), (h, w)).reshape(m, c)
    dyr = P.relu_bwd(dzr, yr)
    dxr, dgr, dbr = P.bn_bwd(x64, dyr, bp["gamma"], mu, rstd)
    xh = (x64 - mu) * rstd
    amb = relu_ambiguous(yr, False)
    scale_b = np.abs(dyr).sum(axis=0)
    scale_g = np.abs(dyr * xh).sum(axis=0)
    assert np.all(np.abs(host(db) - dbr) <= 1e-4 * scale_b), "dbeta"
    assert np.all(np.abs(host(dg) - dgr) <= 1e-4 * scale_g), "dgamma"
    assert_close("dx", host(dx).reshape(m, c), dxr, 1e-4, exclude=amb)


# --------------------------------------------------------- fused forward ----
FWD_CASES = [
    # dtype, k, n, h, w, c_in, c_out, in_ldc, out_ldc
    (False, 1, 8, 8, 8, 64, 32, 64, 32),         # single layer
    (False, 3, 2, 5, 7, 12, 20, 16, 24),         # fp32 3x3, ragged
    (True, 1, 2, 14, 14, 256, 128, 288, 128),    # bottleneck 1x1 on a concat view
    (True, 3, 2, 14, 14, 128, 32, 128, 288),     # growth 3x3 into a concat slice
    (True, 1, 1, 9, 11, 40, 136, 48, 136),       # ragged channels / pixels
    (True, 3, 3, 1, 1, 64, 64, 64, 64),          # H = W = 1: only the centre tap
    (True, 3, 1, 56, 56, 64, 64, 64, 64),        # full-width rows (W = 56)
    (True, 3, 2, 6, 61, 32, 8, 32, 8),           # widest rows of the persistent 3x3 kernel
    (True, 3, 1, 5, 62, 32, 8, 32, 8),           # one column past it (row-tile kernel)
    (True, 1, 2, 7, 7, 512, 128, 520, 128),      # 1x1 with K > 256: tiled kernel, caller's weights unpacked
    (True, 1, 1, 9, 11, 320, 96, 320, 104),      # same, partial output tile, output view
    (True, 1, 1, 5, 13, 296, 24, 304, 24),       # tiled 1x1: ragged last 64-channel chunk, 32-channel output tile
    (True, 1, 1, 3, 5, 1000, 64, 1000, 64),      # tiled 1x1: 16 chunks, 64-channel output tile
    (True, 1, 128, 7, 7, 992, 128, 992, 128),    # DenseNet-121 block 4 at batch 128: tiled 1x1 in 32-row tiles
    (True, 3, 128, 7, 7, 128, 32, 128, 32),      # its 3x3 at batch 128: one persistent workgroup per 32 pixels
    (True, 1, 5, 120, 110, 96, 128, 104, 128),   # persistent 1x1 forward over 66000 pixels: two whole rounds
                                                 # of 128-row tiles, then the 464 rows left split over the grid
]


@pytest.mark.parametrize("case", FWD_CASES)
@pytest.mark.parametrize("mode", ["bnrelu_stats", "bnrelu", "plain_stats"])
def test_conv_fwd(B, case, mode):
    bf16, k, n, h, w, ci, co, ildc, oldc = case
    rnd = P.round_bf16 if bf16 else (lambda a: np.asarray(a, np.float64))
    xf = synth.normal(1, "x", (n, h, w, ildc), bf16=bf16)
    wt = synth.conv_weight(1, "w", k, ci, co, bf16)
    bp = synth.bn_params(1, "bn", ci)
    beta = bp["beta"] + (np.float32(2.0) if k == 3 else np.float32(0))   # large beta: padding semantics
    x = dev(xf, bf16)
    y = torch.zeros((n, h, w, oldc), dtype=x.dtype, device=x.device)
    desc = B.desc_for(x[..., :ci], y[..., :co], k, n, h, w)
    wd = dev(wt, bf16)
    x64 = xf[..., :ci].astype(np.float64)
    ybn = B.BN.stats_only(co, x.device)
    if mode.startswith("bnrelu"):
        xbn = _bn_dev(bp["gamma"], beta)
        B.bnr_bn_stats(x[..., :ci], xbn)
        B.bnr_bn_relu_conv_fwd(desc, x[..., :ci], xbn, wd, y[..., :co], ybn if mode.endswith("stats") else None)
        yr, mu, var, rstd = P.bn_fwd(x64, bp["gamma"], beta, 1e-5)
        z = rnd(P.relu_fwd(yr))
    else:
        B.bnr_conv_bn_stats_fwd(desc, x[..., :ci], wd, y[..., :co], ybn)
        z = x64
    torch.cuda.synchronize()
    out_r = rnd(P.conv_fwd(z, wt.astype(np.float64)))
    assert_close("conv out", host(y[..., :co]), out_r, RTOL[bf16])
    assert np.all(host(y[..., co:]) == 0), "wrote outside the output view"
    if mode.endswith("stats"):
        mr, vr, _ = P.bn_stats(out_r, 1e-5)
        assert_stats("output stats", host(ybn.mean), host(ybn.var), mr, vr, RTOL[bf16])


# --------------------------------------- transition: BN-ReLU-pool-CONV ----
@pytest.mark.parametrize("case", [
    # dtype, n, h, w, c_in, c_out, in_ldc, out_ldc
    (True, 4, 56, 56, 256, 128, 256, 128),      # dense block 1's transition (persistent 1x1 kernel)
    (True, 2, 6, 10, 200, 64, 208, 96),         # ragged channels, output view of a wider buffer
    (True, 2, 14, 14, 512, 256, 512, 512),      # K > 256: tiled kernel (DenseNet-121 transition 2 shape)
    (False, 2, 4, 6, 40, 24, 48, 32),           # fp32 (tiled kernel)
])
@pytest.mark.parametrize("stats", [False, True])
def test_bn_relu_conv_pool_fwd(B, case, stats):
    """y = avgpool2x2(conv1x1(relu(bn(x)))): the fused path averages the
    normalised, rectified input over each window and runs the CONV on the
    pooled pixels; the oracle convolves at full resolution, then pools (equal
    in exact arithmetic; the bf16 path rounds the pooled operand)."""
    bf16, n, h, w, ci, co, ildc, oldc = case
    rnd = P.round_bf16 if bf16 else (lambda a: np.asarray(a, np.float64))
    xf = synth.normal(11, "x", (n, h, w, ildc), bf16=bf16)
    wt = synth.conv_weight(11, "w", 1, ci, co, bf16)
    bp = synth.bn_params(11, "bn", ci)
    x = dev(xf, bf16)
    y = torch.zeros((n, h // 2, w // 2, oldc), dtype=x.dtype, device=x.device)
    xbn = _bn_dev(bp["gamma"], bp["beta"])
    B.bnr_bn_stats(x[..., :ci], xbn)
    desc = B.conv_desc(n, h, w, ci, co, 1, ildc, oldc, B.dtype_code(x))
    ybn = B.BN.stats_only(co, x.device) if stats else None
    B.bnr_bn_relu_conv_pool_fwd(desc, x[..., :ci], xbn, dev(wt, bf16), y[..., :co], ybn)
    torch.cuda.synchronize()
    yr, _, _, _ = P.bn_fwd(xf[..., :ci].astype(np.float64), bp["gamma"], bp["beta"], 1e-5)
    out_r = P.avgpool2_fwd(P.conv_fwd(P.relu_fwd(yr), wt.astype(np.float64)))
    assert_close("pooled out", host(y[..., :co]), rnd(out_r), RTOL[bf16])
    assert np.all(host(y[..., co:]) == 0), "wrote outside the output view"
    if stats:
        mr, vr, _ = P.bn_stats(rnd(out_r), 1e-5)
        assert_stats("pooled output stats", host(ybn.mean), host(ybn.var), mr, vr, RTOL[bf16])


# ----------------------------- residual boundary: BN-add-ReLU-CONV ----
@pytest.mark.parametrize("case", [
    # dtype, n, h, w, c (y, identity, r), c_out, r_ldc
    (True, 2, 14, 14, 256, 64, 256),        # ResNet-50 conv2_x block boundary (persistent 1x1 kernel)
    (True, 1, 9, 11, 136, 40, 144),         # ragged pixels and channels, r into a wider view
    (False, 2, 5, 6, 24, 16, 24),           # fp32 (tiled kernel)
])
def test_bn_add_relu_conv_fwd(B, case):
    """r = relu(bn(y) + identity) formed while the next block's first CONV
    reads y and the identity, written as a side output, and out = conv(r)
    with statistics: r equals the standalone element-wise pass bit for bit,
    out and its statistics match the oracle."""
    bf16, n, h, w, c, co, rldc = case
    rnd = P.round_bf16 if bf16 else (lambda a: np.asarray(a, np.float64))
    yf = synth.normal(12, "y", (n, h, w, c), bf16=bf16) * np.float32(1.3)
    yf = synth.round_to_bf16(yf) if bf16 else yf
    idf = synth.normal(12, "id", (n, h, w, c), bf16=bf16)
    wt = synth.conv_weight(12, "w", 1, c, co, bf16)
    bp = synth.bn_params(12, "bn", c)
    y, ident = dev(yf, bf16), dev(idf, bf16)
    ybn = _bn_dev(bp["gamma"], bp["beta"])
    B.bnr_bn_stats(y, ybn)
    rbuf = torch.zeros((n, h, w, rldc), dtype=y.dtype, device=y.device)
    out = torch.empty((n, h, w, co), dtype=y.dtype, device=y.device)
    obn = B.BN.stats_only(co, y.device)
    desc = B.desc_for(y, out, 1, n, h, w)
    B.bnr_bn_add_relu_conv_fwd(desc, y, ybn, ident, rbuf[..., :c], dev(wt, bf16), out, obn)
    r_ew = torch.empty_like(y)
    B.bnr_bn_add_relu_fwd(y, ybn, ident, r_ew)
    torch.cuda.synchronize()
    assert torch.equal(rbuf[..., :c], r_ew), "side output differs from the element-wise pass"
    assert np.all(host(rbuf[..., c:]) == 0), "wrote outside the side view"
    yr, _, _, _ = P.bn_fwd(yf.astype(np.float64), bp["gamma"], bp["beta"], 1e-5)
    r_r = rnd(P.relu_fwd(yr + idf.astype(np.float64)))
    amb = relu_ambiguous(yr + idf.astype(np.float64), bf16)
    assert_close("r", host(rbuf[..., :c]), r_r, RTOL[bf16], exclude=amb)
    out_r = rnd(P.conv_fwd(host(r_ew), wt.astype(np.float64)))
    assert_close("out", host(out), out_r, RTOL[bf16])
    mr, vr, _ = P.bn_stats(out_r, 1e-5)
    assert_stats("out stats", host(obn.mean), host(obn.var), mr, vr, RTOL[bf16])


# -------------------------------------------------------- fused backward ----
BWD_CASES = [
    (False, 1, 8, 8, 8, 64, 32),
    (False, 3, 2, 5, 6, 12, 20),
    (True, 1, 2, 14, 14, 256, 128),
    (True, 3, 2, 14, 14, 128, 32),
    (True, 1, 1, 9, 11, 40, 136),
    (True, 3, 3, 1, 1, 16, 24),
    (True, 3, 1, 12, 56, 64, 64),
    (True, 3, 2, 7, 7, 128, 32),                # 7x7 rows: four image rows per K chunk
    (True, 3, 1, 5, 30, 64, 96),                # two rows per chunk, two output-channel tiles
    (False, 3, 2, 3, 62, 8, 12),                # widest rows, fp32
    (True, 1, 2, 7, 7, 512, 128),               # tiled 1x1 forward weights [k][n] and data gradient [n][k] unpacked
    (True, 1, 1, 9, 11, 288, 40),               # ragged: K and N past the 256-channel persistent kernel
    (True, 1, 1, 6, 7, 264, 24),                # tiled 1x1: one 8-channel tail chunk, 32-channel output tile
    (True, 1, 1, 5, 7, 1000, 128),              # persistent 1x1 data gradient in four column groups (256 x 3 + 232)
    (True, 1, 1, 6, 10, 512, 256),              # K = 256: four 128-column groups (256-column groups exceed the LDS)
    (True, 3, 4, 56, 56, 128, 32),              # 3x3 weight gradient: 5 chunks per split, Z rows carried between
                                                # chunks, splits crossing image boundaries
    (True, 3, 8, 30, 7, 64, 32),                # same with 14-row chunks of 7-pixel rows
    (True, 3, 128, 7, 7, 128, 32),              # DenseNet-121 block 4 at batch 128: 196 persistent 3x3
                                                # workgroups, 64-way split-K weight gradient (small-operand budget)
    (True, 1, 128, 7, 7, 992, 128),             # its 1x1: data gradient in four column groups, wide split-K dW
]


def _bwd_inputs(bf16, k, n, h, w, ci, co, seed=2):
    xf = synth.normal(seed, "x", (n, h, w, ci), bf16=bf16)
    wt = synth.conv_weight(seed, "w", k, ci, co, bf16)
    bp = synth.bn_params(seed, "bn", ci)
    g = synth.normal(seed, "g", (n, h, w, co), bf16=bf16)
    return xf, wt, bp, g


@pytest.mark.parametrize("case", BWD_CASES)
@pytest.mark.parametrize("dxmode", ["none", "write", "accumulate"])
def test_bwd_fused_dense(B, case, dxmode):
    bf16, k, n, h, w, ci, co = case
    rnd = P.round_bf16 if bf16 else (lambda a: np.asarray(a, np.float64))
    xf, wt, bp, gf = _bwd_inputs(bf16, k, n, h, w, ci, co)
    x, wd, g = dev(xf, bf16), dev(wt, bf16), dev(gf, bf16)
    xbn = _bn_dev(bp["gamma"], bp["beta"])
    B.bnr_bn_stats(x, xbn)
    dw = torch.empty(wt.shape, dtype=torch.float32, device=x.device)
    dgamma = torch.empty(ci, dtype=torch.float32, device=x.device)
    dbeta = torch.empty_like(dgamma)
    dy = torch.empty_like(x)
    old = synth.normal(3, "old", (n, h, w, ci), bf16=bf16)
    dx = dev(old, bf16) if dxmode != "none" else None
    desc = B.desc_for(x, g, k, n, h, w)
    B.bnr_bwd_fused(desc, x, xbn, wd, B.grad_dense(g), dw, dgamma, dbeta, dy, dx, dxmode == "accumulate")
    torch.cuda.synchronize()
    # oracle
    x64 = xf.astype(np.float64)
    yr, mu, var, rstd = P.bn_fwd(x64, bp["gamma"], bp["beta"], 1e-5)
    z = rnd(P.relu_fwd(yr))
    dz = P.conv_dgrad(gf.astype(np.float64), wt.astype(np.float64), (h, w))
    dyr = rnd(P.relu_bwd(dz, yr))
    dwr = P.conv_wgrad(z, gf.astype(np.float64), k)
    dxr, dgr, dbr = P.bn_bwd(x64, dyr, bp["gamma"], mu, rstd)
    amb = relu_ambiguous(yr, bf16)
    rt = RTOL[bf16]
    assert_close("dy", host(dy), dyr, rt, exclude=amb)
    assert_close("dW", host(dw), dwr, rt)
    assert_close("dgamma", host(dgamma), dgr, rt)
    assert_close("dbeta", host(dbeta), dbr, rt)
    if dxmode == "write":
        assert_close("dx", host(dx), rnd(dxr), rt, exclude=amb)
    elif dxmode == "accumulate":
        assert_close("dx (accumulated)", host(dx), rnd(old.astype(np.float64) + dxr), rt, exclude=amb)


@pytest.mark.parametrize("case", [(False, 1, 8, 8, 8, 32, 64), (True, 1, 2, 14, 14, 128, 256),
                                  (True, 3, 2, 10, 12, 64, 32), (True, 1, 1, 9, 11, 136, 40)])
def test_bwd_fused_deferred_bn_gradient(B, case):
    """Gradient source = the deferred input gradient of the next BN (the
    next-prologue backward fusion)."""
    bf16, k, n, h, w, ci, co = case
    rnd = P.round_bf16 if bf16 else (lambda a: np.asarray(a, np.float64))
    xf, wt, bp, _ = _bwd_inputs(bf16, k, n, h, w, ci, co, seed=4)
    # the CONV output x2 feeds BN2, whose masked output gradient dy2 is known
    x2f = synth.normal(4, "x2", (n, h, w, co), bf16=bf16) * np.float32(1.5) + np.float32(0.25)
    x2f = synth.round_to_bf16(x2f) if bf16 else x2f
    dy2f = synth.normal(4, "dy2", (n, h, w, co), bf16=bf16)
    bp2 = synth.bn_params(4, "bn2", co)
    x, wd, x2, dy2 = dev(xf, bf16), dev(wt, bf16), dev(x2f, bf16), dev(dy2f, bf16)
    xbn, bn2 = _bn_dev(bp["gamma"], bp["beta"]), _bn_dev(bp2["gamma"], bp2["beta"])
    B.bnr_bn_stats(x, xbn)
    B.bnr_bn_stats(x2, bn2)
    # dgamma2 / dbeta2 of BN2 from the oracle's own definition, uploaded as inputs
    x2_64, dy2_64 = x2f.astype(np.float64), dy2f.astype(np.float64)
    _, mu2, var2, rstd2 = P.bn_fwd(x2_64, bp2["gamma"], bp2["beta"], 1e-5)
    _, dg2, db2 = P.bn_bwd(x2_64, dy2_64, bp2["gamma"], mu2, rstd2, want_dx=False)
    dg2d, db2d = f32dev(dg2), f32dev(db2)
    dw = torch.empty(wt.shape, dtype=torch.float32, device=x.device)
    dgamma = torch.empty(ci, dtype=torch.float32, device=x.device)
    dbeta = torch.empty_like(dgamma)
    dy = torch.empty_like(x)
    desc = B.desc_for(x, x2, k, n, h, w)
    B.bnr_bwd_fused(desc, x, xbn, wd, B.grad_bn(dy2, x2, bn2, dg2d, db2d), dw, dgamma, dbeta, dy)
    torch.cuda.synchronize()
    g_r = rnd(P.bn_bwd(x2_64, dy2_64, bp2["gamma"], mu2, rstd2)[0])
    x64 = xf.astype(np.float64)
    yr, mu, var, rstd = P.bn_fwd(x64, bp["gamma"], bp["beta"], 1e-5)
    z = rnd(P.relu_fwd(yr))
    dz = P.conv_dgrad(g_r, wt.astype(np.float64), (h, w))
    dyr = rnd(P.relu_bwd(dz, yr))
    dwr = P.conv_wgrad(z, g_r, k)
    _, dgr, dbr = P.bn_bwd(x64, dyr, bp["gamma"], mu, rstd, want_dx=False)
    rt = RTOL[bf16]
    amb = relu_ambiguous(yr, bf16)
    assert_close("dy", host(dy), dyr, rt, exclude=amb)
    assert_close("dW", host(dw), dwr, rt)
    assert_close("dgamma", host(dgamma), dgr, rt)
    assert_close("dbeta", host(dbeta), dbr, rt)


@pytest.mark.parametrize("case", [
    # bf16, k, n, h, w, c_in (BN input), c_out (= the slice), ldc of the concatenation buffer, slice offset
    (True, 3, 2, 10, 12, 128, 32, 64, 32),     # the dense block's 3x3 CONV backward (persistent kernels)
    (True, 3, 1, 6, 56, 128, 32, 256, 224),    # full-width rows, last slice of a 256-channel buffer
    (True, 1, 2, 7, 9, 64, 128, 160, 32),      # 1x1
    (False, 3, 2, 5, 6, 16, 24, 40, 8),        # fp32 (tiled kernels)
])
def test_bwd_fused_summed_gradient_with_bn(B, case):
    """Gradient source = the summed input gradient of a concatenation slice
    (D + alpha + betap * xhat, formed on load) together with the BN-backward
    epilogue of the CONV's own input BN: the combination the dense block's
    3x3 CONVs run with inter-composite-layer fusion."""
    bf16, k, n, h, w, ci, co, ldc, off = case
    rnd = P.round_bf16 if bf16 else (lambda a: np.asarray(a, np.float64))
    xf, wt, bp, _ = _bwd_inputs(bf16, k, n, h, w, ci, co, seed=9)
    bufx = synth.normal(9, "slice_x", (n, h, w, ldc), bf16=bf16) * np.float32(1.4) + np.float32(0.3)
    bufx = synth.round_to_bf16(bufx) if bf16 else bufx
    bufd = synth.normal(9, "slice_d", (n, h, w, ldc), bf16=bf16) * np.float32(0.5)
    bufd = synth.round_to_bf16(bufd) if bf16 else bufd
    alpha_f = synth.normal(9, "alpha", (co,), std=0.05)
    betap_f = synth.normal(9, "betap", (co,), std=0.05)
    x, wd = dev(xf, bf16), dev(wt, bf16)
    X, D = dev(bufx, bf16), dev(bufd, bf16)
    xs, ds = X[..., off:off + co], D[..., off:off + co]
    xbn = _bn_dev(bp["gamma"], bp["beta"])
    B.bnr_bn_stats(x, xbn)
    st = B.BN.stats_only(co, x.device)
    B.bnr_bn_stats(xs, st)
    dw = torch.empty(wt.shape, dtype=torch.float32, device=x.device)
    dgamma = torch.empty(ci, dtype=torch.float32, device=x.device)
    dbeta = torch.empty_like(dgamma)
    dy = torch.empty_like(x)
    desc = B.desc_for(x, xs, k, n, h, w)
    B.bnr_bwd_fused(desc, x, xbn, wd, B.grad_split(ds, xs, st, f32dev(alpha_f), f32dev(betap_f)), dw, dgamma,
                    dbeta, dy)
    torch.cuda.synchronize()
    xs64 = bufx[..., off:off + co].astype(np.float64)
    mu_s, _, rstd_s = P.bn_stats(xs64, 1e-5)
    g_r = rnd(bufd[..., off:off + co].astype(np.float64) + alpha_f.astype(np.float64) +
              betap_f.astype(np.float64) * (xs64 - mu_s) * rstd_s)
    x64 = xf.astype(np.float64)
    yr, mu, var, rstd = P.bn_fwd(x64, bp["gamma"], bp["beta"], 1e-5)
    z = rnd(P.relu_fwd(yr))
    dz = P.conv_dgrad(g_r, wt.astype(np.float64), (h, w))
    dyr = rnd(P.relu_bwd(dz, yr))
    dwr = P.conv_wgrad(z, g_r, k)
    _, dgr, dbr = P.bn_bwd(x64, dyr, bp["gamma"], mu, rstd, want_dx=False)
    rt = RTOL[bf16]
    amb = relu_ambiguous(yr, bf16)
    assert_close("dy", host(dy), dyr, rt, exclude=amb)
    assert_close("dW", host(dw), dwr, rt)
    assert_close("dgamma", host(dgamma), dgr, rt)
    assert_close("dbeta", host(dbeta), dbr, rt)


@pytest.mark.parametrize("bf16", [False, True])
def test_bwd_fused_pooled_gradient_plain_input(B, bf16):
    """Transition-style backward: gradient from a 2x2 average pooling, and a
    CONV without a BN in front (x_bn = NULL: dx = dz written and accumulated)."""
    rnd = P.round_bf16 if bf16 else (lambda a: np.asarray(a, np.float64))
    n, h, w, ci, co = 2, 8, 12, 64, 32
    xf = synth.normal(5, "x", (n, h, w, ci), bf16=bf16)
    wt = synth.conv_weight(5, "w", 1, ci, co, bf16)
    gpf = synth.normal(5, "gp", (n, h // 2, w // 2, co), bf16=bf16)
    old = synth.normal(5, "old", (n, h, w, ci), bf16=bf16)
    x, wd, gp, dx = dev(xf, bf16), dev(wt, bf16), dev(gpf, bf16), dev(old, bf16)
    dw = torch.empty(wt.shape, dtype=torch.float32, device=x.device)
    desc = B.conv_desc(n, h, w, ci, co, 1, ci, co, B.dtype_code(x))
    B.bnr_bwd_fused(desc, x, None, wd, B.grad_avgpool2(gp), dw, dx=dx, dx_accumulate=True)
    torch.cuda.synchronize()
    g_r = P.avgpool2_bwd(gpf.astype(np.float64), (h, w))
    dz = P.conv_dgrad(g_r, wt.astype(np.float64), (h, w))
    rt = RTOL[bf16]
    assert_close("dx", host(dx), rnd(old.astype(np.float64) + dz), rt)
    assert_close("dW", host(dw), P.conv_wgrad(xf.astype(np.float64), g_r, 1), rt)


@pytest.mark.parametrize("bf16", [False, True])
def test_bn_dx_and_avgpool(B, bf16):
    rnd = P.round_bf16 if bf16 else (lambda a: np.asarray(a, np.float64))
    n, h, w, c, ldc = 3, 6, 10, 48, 64
    xf = synth.normal(6, "x", (n, h, w, ldc), bf16=bf16)
    dyf = synth.normal(6, "dy", (n, h, w, c), bf16=bf16)
    bp = synth.bn_params(6, "bn", c)
    x, dy = dev(xf, bf16), dev(dyf, bf16)
    bn = _bn_dev(bp["gamma"], bp["beta"])
    B.bnr_bn_stats(x[..., :c], bn)
    x64 = xf[..., :c].astype(np.float64)
    _, mu, var, rstd = P.bn_fwd(x64, bp["gamma"], bp["beta"], 1e-5)
    dxr, dg, db = P.bn_bwd(x64, dyf.astype(np.float64), bp["gamma"], mu, rstd)
    G = torch.zeros((n, h, w, ldc), dtype=x.dtype, device=x.device)
    B.bnr_bn_dx(dy, x[..., :c], bn, f32dev(dg), f32dev(db), G[..., :c])
    B.bnr_bn_dx(dy, x[..., :c], bn, f32dev(dg), f32dev(db), G[..., :c], dx_accumulate=True)
    pooled = torch.empty((n, h // 2, w // 2, c), dtype=x.dtype, device=x.device)
    B.bnr_avgpool2_fwd(x[..., :c], pooled, n, h, w)
    torch.cuda.synchronize()
    rt = RTOL[bf16]
    assert_close("dx twice", host(G[..., :c]), rnd(rnd(dxr) + dxr), rt)
    assert np.all(host(G[..., c:]) == 0)
    assert_close("avgpool", host(pooled), rnd(P.avgpool2_fwd(x64)), rt)


# ------------------------------------- concatenation BNs: summed gradient ----
@pytest.mark.parametrize("case", [
    # bf16, k of the producer, n, h, w, c (slice), ldc of the buffer, c_out of the two readers, producer c_in
    (False, 3, 2, 6, 7, 24, 40, (16, 40), 12),     # fp32: tiled kernels, ragged
    (True, 3, 2, 10, 12, 32, 96, (128, 64), 128),  # bf16: persistent 1x1 readers, 3x3 producer
    (True, 1, 1, 9, 11, 136, 160, (128, 256), 64),  # bf16: wide slice, 1x1 producer
    (True, 1, 1, 9, 11, 288, 320, (128, 64), 64),  # slice past 256 channels: readers' data gradients in two column groups
])
def test_split_fusion_two_readers(B, case):
    """A concatenation slice x read by two BN-ReLU-CONV1x1 layers that share
    its statistics (inter-composite-layer fusion, Sec. 3.2): each reader's
    backward leaves its BN input gradient in summed form (gsum, alpha, betap);
    the CONV that produced x consumes the sum on load (BNR_GRAD_SPLIT), and
    bnr_split_dx materialises it.  Oracle: the plain sum of the two readers'
    BN input gradients."""
    bf16, kp, n, h, w, c, ldc, cos, cp = case
    rnd = P.round_bf16 if bf16 else (lambda a: np.asarray(a, np.float64))
    buf_f = synth.normal(7, "buf", (n, h, w, ldc), bf16=bf16) * np.float32(1.3) + np.float32(0.2)
    buf_f = synth.round_to_bf16(buf_f) if bf16 else buf_f
    buf = dev(buf_f, bf16)
    x = buf[..., :c]
    shared = B.BN.stats_only(c, buf.device)
    B.bnr_bn_stats(x, shared)                       # the channels' one statistics sweep
    x64 = buf_f[..., :c].astype(np.float64)
    G = dev(synth.normal(7, "garbage", (n, h, w, ldc), bf16=bf16), bf16)     # overwritten by the first reader
    alpha = f32dev(synth.normal(7, "ga", (c,)))
    betap = f32dev(synth.normal(7, "gb", (c,)))
    readers = []
    for i, co in enumerate(cos):
        wt = synth.conv_weight(7, "w%d" % i, 1, c, co, bf16)
        bp = synth.bn_params(7, "bn%d" % i, c)
        gf = synth.normal(7, "g%d" % i, (n, h, w, co), bf16=bf16)
        bn = B.BN(f32dev(bp["gamma"]), f32dev(bp["beta"]), 1e-5, mean=shared.mean, var=shared.var, rstd=shared.rstd)
        dw = torch.empty(wt.shape, dtype=torch.float32, device=buf.device)
        dgamma = torch.empty(c, dtype=torch.float32, device=buf.device)
        dbeta = torch.empty_like(dgamma)
        g = dev(gf, bf16)
        desc = B.desc_for(x, g, 1, n, h, w)
        B.bnr_bwd_fused_split(desc, x, bn, dev(wt, bf16), B.grad_dense(g), dw, dgamma, dbeta, G[..., :c], alpha,
                              betap, accumulate=i > 0)
        readers.append((dw, dgamma, dbeta, wt, bp, gf))
    # the producer CONV of x (plain input): its backward takes the summed gradient on load
    xin_f = synth.normal(7, "xin", (n, h, w, cp), bf16=bf16)
    wp = synth.conv_weight(7, "wp", kp, cp, c, bf16)
    xin = dev(xin_f, bf16)
    dwp = torch.empty(wp.shape, dtype=torch.float32, device=buf.device)
    dxin = torch.empty_like(xin)
    descp = B.desc_for(xin, x, kp, n, h, w)
    B.bnr_bwd_fused(descp, xin, None, dev(wp, bf16), B.grad_split(G[..., :c], x, shared, alpha, betap), dwp,
                    dx=dxin)
    torch.cuda.synchronize()
    rest = host(G[..., c:])
    B.bnr_split_dx(G[..., :c], x, shared, alpha, betap, G[..., :c])
    torch.cuda.synchronize()
    rt = RTOL[bf16]
    np.testing.assert_array_equal(host(G[..., c:]), rest)          # channels beyond the slice untouched

    # Oracle.  A reader's ReLU decision within rounding of 0 has two correct
    # outcomes; with k such decisions there are 2^k correct results.  Every
    # tensor must match one and the same of them (no element excluded).
    x_flat = x64.reshape(-1, c)
    per_reader = []
    for dw, dgamma, dbeta, wt, bp, gf in readers:
        yr, mu, var, rstd = P.bn_fwd(x64, bp["gamma"], bp["beta"], 1e-5)
        dz = P.conv_dgrad(gf.astype(np.float64), wt.astype(np.float64), (h, w))
        amb = np.flatnonzero(relu_ambiguous(yr, bf16).reshape(-1))
        per_reader.append((yr, mu, rstd, dz, amb))
    k = sum(len(a) for *_, a in per_reader)
    assert k <= 6, "%d ambiguous reader decisions" % k

    def variant(bits):
        out, dx_true, j = [], np.zeros_like(x64), 0
        for (dw, dgamma, dbeta, wt, bp, gf), (yr, mu, rstd, dz, amb) in zip(readers, per_reader):
            dy = P.relu_bwd(dz, yr).reshape(-1)
            for e in amb:                                   # flip this decision if its bit is set
                if bits >> j & 1:
                    dy[e] = 0.0 if dy[e] != 0 or yr.reshape(-1)[e] > 0 else dz.reshape(-1)[e]
                j += 1
            dyr = rnd(dy.reshape(x64.shape))
            dxr, dgr, dbr = P.bn_bwd(x64, dyr, bp["gamma"], mu, rstd)
            dx_true += dxr
            out.append((P.conv_wgrad(rnd(P.relu_fwd(yr)), gf.astype(np.float64), 1), dgr, dbr))
        g_true = rnd(dx_true)
        return out, dx_true, P.conv_dgrad(g_true, wp.astype(np.float64), (h, w)), \
            P.conv_wgrad(xin_f.astype(np.float64), g_true, kp)

    got_dx, got_dxin, got_dwp = host(G[..., :c]), host(dxin), host(dwp)
    best = None
    for bits in range(1 << k):
        out, dx_true, dz_p, dwp_r = variant(bits)
        errs = [rel_err(got_dx, dx_true), rel_err(got_dxin, dz_p), rel_err(got_dwp, dwp_r)]
        for (dw, dgamma, dbeta, *_), (dwr, dgr, dbr) in zip(readers, out):
            errs += [rel_err(host(dw), dwr), rel_err(host(dgamma), dgr), rel_err(host(dbeta), dbr)]
        if best is None or max(errs) < max(best):
            best = errs
    names = ["summed dx", "producer dx", "producer dW (summed gradient on load)"] + \
        ["reader%d %s" % (i, t) for i in range(len(readers)) for t in ("dW", "dgamma", "dbeta")]
    bad = [(nm, e) for nm, e in zip(names, best) if e > rt]
    assert not bad, "no correct outcome of the %d ambiguous decisions matches: %s" % (k, bad)
