"""Training compositions built from the fp64 oracle primitives.

Test infrastructure only.  Each function follows the layer order the paper
describes and nothing else:

* ``unit_*``  -- one BN -> ReLU -> CONV chain (the BN whose sub-layers the
  paper's fission splits between the CONV before it and the CONV after it,
  Sec. 3.2, Fig. 5).
* ``cpl_*``   -- a DenseNet composite layer, BN-ReLU-CONV1x1-BN-ReLU-CONV3x3,
  whose k new channels are concatenated to its input (Sec. 2.3, Fig. 2).
  The backward of the concat is a channel split and the backward of the split
  (one tensor read by several later layers) is a sum over its readers.
* ``block_*`` -- dense block 1 of DenseNet-121 followed by its transition
  layer BN-ReLU-CONV1x1 + 2x2 average pooling (Sec. 2.3).
* ``densenet_*`` -- a whole DenseNet: 7x7 stem, dense blocks joined by
  transitions, and the classifier head (Sec. 2.2, Sec. 2.3, Sec. 3.1).
* ``resnet_*`` -- a ResNet bottleneck block CONV1x1-BN-ReLU-CONV3x3-BN-ReLU-
  CONV1x1-BN, element-wise sum with its input, ReLU (Sec. 2.2).

Storage model.  ``rnd`` is applied exactly where the configuration stores a
tensor (or hands it to a matrix unit) in its operand precision: identity for
the fp32 configuration (the oracle then runs fully in fp64), bf16
round-to-nearest-even for the bf16-operand configurations.  Everything between
those points, including all statistics and reductions, stays fp64.
The paper runs in fp32 only, so the rounding sites are a reading:
  forward   z = relu(bn(x)) and every CONV output (the MFMA operand and the
            stored activation), the pooled outputs, the residual block output;
  backward  the masked BN output gradient dy of every unit; the gradient
            operand a CONV's backward receives when it is a BN input gradient
            (the deferred dx formed on load); the concatenation gradient G
            after each reader's addition (Split backward) and its initial
            value; the transition's unpooled gradient; the residual block's
            masked gradient ds and its input gradient dX; the stem's BN input
            gradient.
  never     batch statistics, dgamma, dbeta and dW (fp32 results on the GPU,
            fp64 here).
"""
import numpy as np

from . import prims as P


def storage(bf16: bool):
    if bf16:
        return P.round_bf16
    return lambda a: np.asarray(a, dtype=np.float64)


# ------------------------------------------------------------ one unit ----
def unit_fwd(x, gamma, beta, wt, eps, rnd):
    """BN (training statistics) -> ReLU -> CONV (stride 1, pad K//2)."""
    y, mean, var, rstd = P.bn_fwd(x, gamma, beta, eps)
    z = rnd(P.relu_fwd(y))
    out = rnd(P.conv_fwd(z, wt))
    return dict(x=np.asarray(x, np.float64), y=y, z=z, out=out, mean=mean, var=var, rstd=rstd,
                gamma=np.asarray(gamma, np.float64), wt=np.asarray(wt, np.float64))


def unit_pool_fwd(x, gamma, beta, wt, eps, rnd):
    """The transition layer BN -> ReLU -> CONV1x1 -> 2x2 average pooling with
    the pooling applied to the CONV's input instead of its output (Sec. 2.3
    transition; both operations are linear, so the result is the same in
    exact arithmetic).  Storage: the pooled CONV operand and the pooled output
    are rounded; z, the full-resolution CONV input, is kept as the backward
    uses it.  Returns (cache as unit_fwd's without "out", pooled)."""
    y, mean, var, rstd = P.bn_fwd(x, gamma, beta, eps)
    z = rnd(P.relu_fwd(y))
    zp = rnd(P.avgpool2_fwd(P.relu_fwd(y)))
    pooled = rnd(P.conv_fwd(zp, wt))
    return dict(x=np.asarray(x, np.float64), y=y, z=z, zp=zp, mean=mean, var=var, rstd=rstd,
                gamma=np.asarray(gamma, np.float64), wt=np.asarray(wt, np.float64)), pooled


def unit_bwd(c, g, rnd):
    """Backward of ``unit_fwd`` for L = sum(out * g); g in operand precision.

    Returns g (the gradient operand as received), dz (CONV input gradient),
    dy (BN output gradient after the ReLU mask, stored), dW, dgamma, dbeta and
    dx (fp64, not rounded)."""
    K = c["wt"].shape[0]
    dz = P.conv_dgrad(g, c["wt"], c["x"].shape[1:3])
    dy = rnd(P.relu_bwd(dz, c["y"]))
    dw = P.conv_wgrad(c["z"], g, K)
    dx, dgamma, dbeta = P.bn_bwd(c["x"], dy, c["gamma"], c["mean"], c["rstd"])
    return dict(g=np.asarray(g, np.float64), dz=dz, dy=dy, dw=dw, dgamma=dgamma, dbeta=dbeta, dx=dx)


# ------------------------------------------------- DenseNet composite layer ----
def cpl_fwd(buf, c_l, p, eps, rnd):
    """Runs composite layer on buf[..., :c_l] and writes its k new channels
    into buf[..., c_l:c_l+k] (in place).  p: gamma1, beta1, w1, gamma2, beta2, w2."""
    u1 = unit_fwd(buf[..., :c_l], p["gamma1"], p["beta1"], p["w1"], eps, rnd)
    u2 = unit_fwd(u1["out"], p["gamma2"], p["beta2"], p["w2"], eps, rnd)
    k = p["w2"].shape[3]
    buf[..., c_l:c_l + k] = u2["out"]
    return dict(u1=u1, u2=u2, c_l=c_l, k=k)


def cpl_bwd(c, G, rnd):
    """G: gradient buffer of the concatenated tensor; its slice of this layer's
    new channels is complete when this is called.  Adds this layer's input
    gradient into G[..., :c_l] (in place) and returns the parameter gradients."""
    c_l, k = c["c_l"], c["k"]
    b2 = unit_bwd(c["u2"], G[..., c_l:c_l + k], rnd)
    b1 = unit_bwd(c["u1"], rnd(b2["dx"]), rnd)
    G[..., :c_l] = rnd(G[..., :c_l] + b1["dx"])
    return dict(b1=b1, b2=b2)


def bottleneck_fwd(X, k, p, eps, rnd):
    """One DenseNet bottleneck layer with its concatenated output:
    returns Y = concat(X, CPL(X)) and the cache."""
    N, H, W, C = X.shape
    buf = np.zeros((N, H, W, C + k))
    buf[..., :C] = X
    c = cpl_fwd(buf, C, p, eps, rnd)
    return buf, c


def bottleneck_bwd(c, dY, rnd):
    G = rnd(np.array(dY, dtype=np.float64, copy=True))
    g = cpl_bwd(c, G, rnd)
    return G[..., :c["c_l"]], g


# ------------------------------------------- dense block (+ transition) ----
def dense_layers_fwd(X0, cpls, eps, rnd, c_total):
    """The composite layers of one dense block on a buffer holding the block
    input X0 in channels [0, C0); returns (buffer, per-layer caches)."""
    N, H, W, C0 = X0.shape
    buf = np.zeros((N, H, W, c_total))
    buf[..., :C0] = X0
    caches, c_l = [], C0
    for p in cpls:
        caches.append(cpl_fwd(buf, c_l, p, eps, rnd))
        c_l += p["w2"].shape[3]
    assert c_l == c_total
    return buf, caches


def dense_layers_bwd(caches, G, rnd):
    """Backward of ``dense_layers_fwd`` on the complete gradient G of the
    block buffer (in place); returns the per-layer parameter gradients."""
    grads = [cpl_bwd(cc, G, rnd) for cc in reversed(caches)]
    grads.reverse()
    return grads


def block_fwd(X0, cpls, trans, eps, rnd, c_total, pool_first=False):
    """X0: block input [N,H,W,C0]; cpls: list of composite-layer params;
    trans: gamma, beta, w (1x1) of the transition.  Returns pooled output.
    pool_first: the transition pools before its CONV (unit_pool_fwd)."""
    buf, caches = dense_layers_fwd(X0, cpls, eps, rnd, c_total)
    if pool_first:
        ut, pooled = unit_pool_fwd(buf, trans["gamma"], trans["beta"], trans["w"], eps, rnd)
    else:
        ut = unit_fwd(buf, trans["gamma"], trans["beta"], trans["w"], eps, rnd)
        pooled = rnd(P.avgpool2_fwd(ut["out"]))
    return pooled, dict(buf=buf, cpls=caches, ut=ut, C0=X0.shape[3])


def block_bwd(c, dpool, rnd):
    ut = c["ut"]
    gt = rnd(P.avgpool2_bwd(dpool, ut["x"].shape[1:3]))
    bt = unit_bwd(ut, gt, rnd)
    G = rnd(bt["dx"])
    grads = dense_layers_bwd(c["cpls"], G, rnd)
    return G[..., :c["C0"]], dict(trans=bt, cpls=grads, G=G)


# ------------------------------------------------ ResNet bottleneck block ----
def resnet_block_fwd(X, p, eps, rnd):
    """CONV1x1 -> BN -> ReLU -> CONV3x3 -> BN -> ReLU -> CONV1x1 -> BN, + X, ReLU.
    p: w1, gamma1, beta1, w2, gamma2, beta2, w3, gamma3, beta3."""
    a1 = rnd(P.conv_fwd(X, p["w1"]))
    u2 = unit_fwd(a1, p["gamma1"], p["beta1"], p["w2"], eps, rnd)
    u3 = unit_fwd(u2["out"], p["gamma2"], p["beta2"], p["w3"], eps, rnd)
    y3, m3, v3, r3 = P.bn_fwd(u3["out"], p["gamma3"], p["beta3"], eps)
    s = y3 + np.asarray(X, np.float64)
    r = rnd(P.relu_fwd(s))
    return r, dict(X=np.asarray(X, np.float64), a1=a1, u2=u2, u3=u3, s=s, mean3=m3, var3=v3,
                   rstd3=r3, p=p)


def resnet_block_bwd(c, dr, rnd):
    p = c["p"]
    ds = rnd(P.relu_bwd(dr, c["s"]))
    dx3, dgamma3, dbeta3 = P.bn_bwd(c["u3"]["out"], ds, p["gamma3"], c["mean3"], c["rstd3"])
    b3 = unit_bwd(c["u3"], rnd(dx3), rnd)
    b2 = unit_bwd(c["u2"], rnd(b3["dx"]), rnd)
    g1 = rnd(b2["dx"])
    dX = rnd(ds + P.conv_dgrad(g1, p["w1"], c["X"].shape[1:3]))
    dw1 = P.conv_wgrad(c["X"], g1, p["w1"].shape[0])
    return dX, dict(ds=ds, g1=g1, dw1=dw1, b2=b2, b3=b3, dgamma3=dgamma3, dbeta3=dbeta3)


# ------------------------------------------------ full DenseNet(-121) ----
def densenet_fwd(d, eps, rnd, pool_first=False):
    """One training forward pass of a DenseNet (Sec. 2.3: dense blocks joined
    by transition layers; Sec. 3.1: a first 7x7 CONV):
      stem   CONV7x7/2 pad 3 -> BN -> ReLU -> max pooling 3x3/2 pad 1,
      blocks dense layers, then (all but the last) transition BN-ReLU-CONV1x1
             + 2x2 average pooling whose output is the next block's input,
      head   BN -> ReLU -> global average pooling -> FC -> softmax
             cross-entropy (mean over the batch).
    d: img [N,H,W,Ci], stem {w, gamma, beta}, blocks [{cpls, trans or None,
    c_total}], head {gamma, beta, w [C,K], b [K]}, labels [N].
    pool_first: every transition pools before its CONV (block_fwd).
    Returns (loss, cache)."""
    st = d["stem"]
    img = np.asarray(d["img"], np.float64)
    s = rnd(P.conv_fwd(img, st["w"], stride=2, pad=3))
    y0, m0, v0, r0 = P.bn_fwd(s, st["gamma"], st["beta"], eps)
    z0 = P.relu_fwd(y0)
    X = rnd(P.maxpool_fwd(z0, 3, 2, 1))
    stem = dict(img=img, s=s, y=y0, z=z0, mean=m0, var=v0, rstd=r0, out=X)
    blocks = []
    for b in d["blocks"]:
        if b["trans"] is not None:
            X, cb = block_fwd(X, b["cpls"], b["trans"], eps, rnd, b["c_total"], pool_first)
        else:
            buf, caches = dense_layers_fwd(X, b["cpls"], eps, rnd, b["c_total"])
            cb = dict(buf=buf, cpls=caches, C0=X.shape[3])
            X = buf
        blocks.append(cb)
    hp = d["head"]
    y5, m5, v5, r5 = P.bn_fwd(X, hp["gamma"], hp["beta"], eps)
    z5 = P.relu_fwd(y5)
    f = P.global_avgpool_fwd(z5)
    logits = P.fc_fwd(f, hp["w"], hp["b"])
    loss, dlogits = P.softmax_ce(logits, d["labels"])
    head = dict(x=X, y=y5, z=z5, mean=m5, var=v5, rstd=r5, f=f, logits=logits, dlogits=dlogits)
    return loss, dict(stem=stem, blocks=blocks, head=head, d=d)


def densenet_bwd(c, rnd):
    """Backward of ``densenet_fwd`` for the loss itself.  Returns the
    parameter gradients and the intermediate gradients the fused path
    materialises (stored ones rounded by ``rnd``)."""
    d, hd, st = c["d"], c["head"], c["stem"]
    hp = d["head"]
    df, dwfc, dbfc = P.fc_bwd(hd["f"], hp["w"], hd["dlogits"])
    dz5 = P.global_avgpool_bwd(df, hd["x"].shape[1:3])
    dy5 = P.relu_bwd(dz5, hd["y"])
    dx5, dg5, db5 = P.bn_bwd(hd["x"], dy5, hp["gamma"], hd["mean"], hd["rstd"])
    head = dict(df=df, dw=dwfc, db=dbfc, dgamma=dg5, dbeta=db5)
    blocks = [None] * len(c["blocks"])
    cb = c["blocks"][-1]
    G = rnd(dx5)
    blocks[-1] = dict(cpls=dense_layers_bwd(cb["cpls"], G, rnd), G=G)
    dX = G[..., :cb["C0"]]
    for i in range(len(c["blocks"]) - 2, -1, -1):
        dX, blocks[i] = block_bwd(c["blocks"][i], dX, rnd)
    dz0 = P.maxpool_bwd(st["z"], dX, 3, 2, 1)
    dy0 = rnd(P.relu_bwd(dz0, st["y"]))
    dx0, dg0, db0 = P.bn_bwd(st["s"], dy0, d["stem"]["gamma"], st["mean"], st["rstd"])
    g0 = rnd(dx0)
    dw0 = P.conv_wgrad(st["img"], g0, d["stem"]["w"].shape[0], stride=2, pad=3)
    stem = dict(dX=dX, dy=dy0, g=g0, dw=dw0, dgamma=dg0, dbeta=db0)
    return dict(head=head, blocks=blocks, stem=stem)
