"""Algorithmic HBM bytes of one training step, fused vs unfused.

"Algorithmic" = every kernel reads each of its input tensors once and writes
each output once (halo re-reads, weight re-reads from cache and the tiny
per-tile partial sums are not counted).  The unit of the model is the paper's
"memory sweep": reading or writing one feature-map tensor over the whole
mini-batch (Sec. 3.2, Fig. 5).  Per BN of C channels with S = m*C*bytes:

  forward   unfused: CONV1 writes x, mean and variance sweeps read x, the
                     normalisation reads x and writes y, ReLU reads y and writes
                     z, CONV2 reads z                           -> 8 S
            fused:   CONV1 writes x (statistics in its epilogue), CONV2 reads x
                     (normalise + ReLU in its prologue)         -> 2 S
  backward  unfused: CONV2 dgrad writes dz, wgrad reads z, ReLU backward reads
                     dz, y and writes dy, the reductions read dy and x, the
                     input gradient reads dy and x and writes dx, CONV1 dgrad and
                     wgrad read dx                              -> 12 S
            fused:   CONV2 dgrad reads x and writes dy (mask + sums in its
                     epilogue), wgrad reads x, CONV1 dgrad and wgrad each read
                     dy and x (deferred input gradient in their prologues)
                                                                -> 7 S
i.e. the backward restructuring removes 5 sweeps per BN, as the paper states.

Inter-composite-layer fusion (dense block, Sec. 3.2 last paragraph): the BN1
statistics come from the producers' epilogues (no sweep per layer, one sweep
of the block input), and each BN1's input gradient is added in summed form
into the concatenation gradient inside its data-gradient epilogue (read x, read
and write the sum: 3 S instead of writing dy and a separate read dy, x, G /
write G pass: 5 S); a slice's producer reads the sum and x (2 S of k channels
instead of 1).
``sweeps_per_bn()`` returns these counts; ``for_workload()`` sums the exact
byte traffic of each driver's kernel sequence.
"""


def sweeps_per_bn():
    # fwd_fused_o2: the paper's fused layer also writes the BN+ReLU output (O2')
    return {"fwd_unfused": 8, "fwd_fused": 2, "fwd_fused_o2": 3, "bwd_unfused": 12, "bwd_fused": 7}


class _Acc:
    def __init__(self):
        self.total = 0

    def __iadd__(self, v):
        self.total += int(v)
        return self


def _unit_fused_fwd(a, m, ci, co, k, e, stats_sweep, out_stats=True, save_z=False):
    if stats_sweep:
        a += m * ci * e                       # standalone sub-BN1: one read sweep
    a += m * ci * e + k * k * ci * co * e     # CONV reads x (normalise + ReLU on load) and weights
    a += m * co * e                           # writes its output (statistics of it in the epilogue)
    if save_z:
        a += m * ci * e                       # O2': also writes relu(bn(x)) (the backward reads it in place of x)


def _unit_fused_bwd(a, m, ci, co, k, e, g_bytes, dx_mode):
    """g_bytes: bytes of one read of the gradient source.  dx_mode: None
    (deferred), 'write' or 'accumulate'."""
    a += g_bytes + k * k * ci * co * e        # dgrad: gradient source, weights
    a += m * ci * e + m * ci * e              # epilogue: read x, write dy
    a += m * ci * e + g_bytes                 # wgrad: x (recomputed relu(bn(x))) and the gradient source
    a += k * k * ci * co * 4                  # dW (fp32)
    if dx_mode is not None:
        a += 2 * m * ci * e + m * ci * e      # read dy, x; write dx
        if dx_mode == "accumulate":
            a += m * ci * e


def _unit_split_bwd(a, m, ci, co, k, e, g_bytes, accumulate):
    """Backward of a concatenation-slice BN reader leaving its input gradient in
    summed form: the epilogue reads x and writes (or reads and writes) the sum."""
    a += g_bytes + k * k * ci * co * e        # dgrad: gradient source, weights
    a += m * ci * e + m * ci * e              # epilogue: read x, write the sum
    if accumulate:
        a += m * ci * e                       # ... and read its old contents
    a += m * ci * e + g_bytes                 # wgrad: x and the gradient source
    a += k * k * ci * co * 4                  # dW (fp32)


def _unit_ref_fwd(a, m, ci, co, k, e, ref="baseline"):
    """Unfused chain; ref 'rcf': the ReLU applied while the CONV reads y (no
    z), 'rcf_mvf': that with one statistics sweep (mean/variance fusion)."""
    a += (1 if ref == "rcf_mvf" else 2) * m * ci * e     # statistics: mean and variance sweeps (MVF: one)
    a += 2 * m * ci * e                       # normalise: read x, write y
    if ref == "baseline":
        a += 2 * m * ci * e                   # ReLU: read y, write z
    a += m * ci * e + k * k * ci * co * e + m * co * e   # CONV: read z (RCF: y), weights, write out


def _unit_ref_bwd(a, m, ci, co, k, e, g_bytes, accumulate, ref="baseline"):
    if ref == "baseline":
        a += g_bytes + k * k * ci * co * e + m * ci * e  # dgrad: read g, weights, write dz
        a += m * ci * e + g_bytes + k * k * ci * co * 4  # wgrad: read z, g, write dW
        a += 3 * m * ci * e                              # ReLU backward: read dz, y, write dy
    else:
        a += g_bytes + k * k * ci * co * e + 2 * m * ci * e   # dgrad with the ReLU mask: read g, weights, y; write dy
        a += m * ci * e + g_bytes + k * k * ci * co * 4  # wgrad: read y (ReLU on load), g, write dW
    a += 2 * m * ci * e                                  # reductions: read dy, x
    a += 3 * m * ci * e + (m * ci * e if accumulate else 0)   # dx: read dy, x (+dx), write dx


def single_layer(m, ci, co, e):
    f, u = _Acc(), _Acc()
    _unit_fused_fwd(f, m, ci, co, 1, e, True)
    _unit_fused_bwd(f, m, ci, co, 1, e, m * co * e, "write")
    _unit_ref_fwd(u, m, ci, co, 1, e)
    _unit_ref_bwd(u, m, ci, co, 1, e, m * co * e, False)
    return {"fused": f.total, "unfused": u.total}


def bottleneck(m, ci, width, k, e):
    f, u = _Acc(), _Acc()
    ct = ci + k
    for a in (f, u):
        a += 2 * m * ct * e                   # G = dY (split backward starts from the upstream gradient)
    _unit_fused_fwd(f, m, ci, width, 1, e, True)
    _unit_fused_fwd(f, m, width, k, 3, e, False)
    _unit_fused_bwd(f, m, width, k, 3, e, m * k * e, None)
    _unit_fused_bwd(f, m, ci, width, 1, e, 2 * m * width * e, "accumulate")
    _unit_ref_fwd(u, m, ci, width, 1, e)
    _unit_ref_fwd(u, m, width, k, 3, e)
    _unit_ref_bwd(u, m, width, k, 3, e, m * k * e, False)
    _unit_ref_bwd(u, m, ci, width, 1, e, m * width * e, True)
    return {"fused": f.total, "unfused": u.total}


def _block_fwd(a, m, c0, layers, width, k, trans_out, e, mode, in_sweep=True):
    """Forward of a dense block (+ transition) in mode 'icf' (fused with
    inter-composite-layer fusion), 'fused', 'o2' (fused, the composite layers'
    BN+ReLU outputs stored: the paper's O2' sweep), 'unfused', 'rcf' or
    'rcf_mvf' (the unfused chain with ReLU-CONV fusion, and with mean/variance
    fusion too); in_sweep (icf): the block input's statistics need their own
    sweep."""
    ref = {"unfused": "baseline", "rcf": "rcf", "rcf_mvf": "rcf_mvf"}.get(mode)
    c = c0
    if mode == "icf" and in_sweep:
        a += m * c0 * e                                          # the one statistics sweep (block input)
    for _ in range(layers):
        if ref:
            _unit_ref_fwd(a, m, c, width, 1, e, ref)
            _unit_ref_fwd(a, m, width, k, 3, e, ref)
        else:
            _unit_fused_fwd(a, m, c, width, 1, e, mode in ("fused", "o2"), save_z=mode == "o2")
            _unit_fused_fwd(a, m, width, k, 3, e, False, save_z=mode == "o2")
        c += k
    if trans_out:
        if ref:
            _unit_ref_fwd(a, m, c, trans_out, 1, e, ref)
            a += m * trans_out * e + m // 4 * trans_out * e      # avgpool forward
        else:
            # BN, ReLU and the 2x2 average in the CONV's prologue: read x,
            # write only the pooled output
            if mode in ("fused", "o2"):
                a += m * c * e                                   # the transition BN's statistics sweep
            a += m * c * e + c * trans_out * e + m // 4 * trans_out * e
    return c


def _block_bwd(a, m, c0, layers, width, k, trans_out, e, mode):
    """Backward of _block_fwd; without a transition the block's gradient
    buffer was written by the BN that reads the whole block (the head)."""
    ct = c0 + layers * k
    ref = {"unfused": "baseline", "rcf": "rcf", "rcf_mvf": "rcf_mvf"}.get(mode)
    if trans_out:
        if mode == "icf":
            _unit_split_bwd(a, m, ct, trans_out, 1, e, m // 4 * trans_out * e, False)
        elif mode in ("fused", "o2"):
            _unit_fused_bwd(a, m, ct, trans_out, 1, e, m // 4 * trans_out * e, "write")
        else:
            a += m // 4 * trans_out * e + m * trans_out * e      # unfused: materialised pooling gradient
            _unit_ref_bwd(a, m, ct, trans_out, 1, e, m * trans_out * e, False, ref)
    for layer in reversed(range(layers)):
        c = c0 + layer * k
        if mode == "icf":
            _unit_fused_bwd(a, m, width, k, 3, e, 2 * m * k * e, None)     # summed gradient + slice on load
            _unit_split_bwd(a, m, c, width, 1, e, 2 * m * width * e, True)
        elif mode in ("fused", "o2"):             # (o2: the epilogue and wgrad read z in place of x)
            _unit_fused_bwd(a, m, width, k, 3, e, m * k * e, None)
            _unit_fused_bwd(a, m, c, width, 1, e, 2 * m * width * e, "accumulate")
        else:
            _unit_ref_bwd(a, m, width, k, 3, e, m * k * e, False, ref)
            _unit_ref_bwd(a, m, c, width, 1, e, m * width * e, True, ref)
    if mode == "icf":
        a += 3 * m * c0 * e                                      # block-input gradient: read sum, x; write


def dense_block(m, c0, layers, width, k, trans_out, e):
    out = {}
    for mode in ("icf", "fused", "o2", "unfused", "rcf", "rcf_mvf"):
        a = _Acc()
        _block_fwd(a, m, c0, layers, width, k, trans_out, e, mode)
        _block_bwd(a, m, c0, layers, width, k, trans_out, e, mode)
        out[mode] = a.total
    return {"fused": out["icf"], "fused_no_icf": out["fused"], "fused_o2": out["o2"], "unfused": out["unfused"],
            "unfused_rcf": out["rcf"], "unfused_rcf_mvf": out["rcf_mvf"]}


def densenet(n, hw, c_in, c_stem, blocks, classes, e):
    """Whole DenseNet step.  blocks: [(c0, layers, width, k, trans_out or 0)].
    Fused: first CONV with statistics epilogue; BN-ReLU-max pooling reading s
    and writing block 1's input with its statistics; blocks with ICF (a
    transition writes the next block's input with its statistics); the head
    reads the last block (BN + ReLU + pooling) and its backward writes the
    summed gradient; max-pooling backward reads s and the block-1 input
    gradient and writes dy; the first CONV's weight gradient reads the image,
    dy and s.  Unfused: two-pass statistics, normalise and ReLU sweeps around
    a plain max pooling, materialised pooling / ReLU / BN input gradients."""
    ho = (hw - 1) // 2 + 1
    hp = (ho - 1) // 2 + 1
    S0 = n * ho * ho * c_stem * e
    Sp = n * hp * hp * c_stem * e
    img = n * hw * hw * 4 * e
    w0 = 49 * c_in * c_stem
    out = {}
    for mode in ("icf", "unfused"):
        a = _Acc()
        a += img + w0 * e + S0                                   # first CONV (statistics in its epilogue if fused)
        if mode == "icf":
            a += S0 + Sp                                         # BN-ReLU-max pooling (+ block-input statistics)
        else:
            a += 6 * S0 + S0 + Sp                                # stats (2), normalise (2), ReLU (2), pooling
        h, dims = hp, []
        for i, (c0, layers, width, k, to) in enumerate(blocks):
            m = n * h * h
            ct = _block_fwd(a, m, c0, layers, width, k, to, e, mode, in_sweep=False)
            dims.append(m)
            if to:
                h //= 2
        S4 = dims[-1] * ct * e
        if mode == "unfused":
            a += S4                                              # head BN statistics sweep
        a += S4 + ct * classes * e                               # head forward: x (BN + ReLU + pooling), FC weights
        a += ct * classes * (e + 4)                              # FC backward: weights, dW
        a += (2 if mode == "icf" else 3) * S4                    # head BN backward (summed form / sums + dx)
        for (c0, layers, width, k, to), m in reversed(list(zip(blocks, dims))):
            _block_bwd(a, m, c0, layers, width, k, to, e, mode)
        if mode == "icf":
            a += 2 * S0 + Sp                                     # pooling backward: s, block-input gradient; dy
            a += img + 2 * S0 + w0 * 4                           # first-CONV wgrad: image, dy, s; dW
        else:
            a += 2 * S0 + Sp                                     # plain pooling backward: z, gradient; dz
            a += 8 * S0                                          # ReLU backward (3), BN sums (2), BN dx (3)
            a += img + S0 + w0 * 4                               # first-CONV wgrad: image, dx; dW
        out[mode] = a.total
    return {"fused": out["icf"], "unfused": out["unfused"]}


def resnet_stack(m, c, width, blocks, e):
    """Bottleneck blocks CONV1x1(c->width)-BN-ReLU-CONV3x3-BN-ReLU-CONV1x1(width->c)-BN, + id, ReLU."""
    f, u = _Acc(), _Acc()
    S, Sw = m * c * e, m * width * e
    w1, w2, w3 = c * width * e, 9 * width * width * e, width * c * e
    for i in range(blocks):
        # forward: first CONV reads X and writes y1 with BN1's statistics (fused) / without (unfused);
        # fused, from the second block on it reads the previous y3 and identity and writes X itself
        # (the previous block's BN3 + add + ReLU in its prologue)
        f += (S if i == 0 else 3 * S) + w1 + Sw
        u += S + w1 + Sw
        _unit_fused_fwd(f, m, width, width, 3, e, False)
        _unit_fused_fwd(f, m, width, c, 1, e, False)
        if i == blocks - 1:
            f += 3 * S                        # the last block: BN3 + add + ReLU as one sweep
        _unit_ref_fwd(u, m, width, width, 3, e)
        _unit_ref_fwd(u, m, width, c, 1, e)
        u += 2 * S + 2 * S + 3 * S            # two-pass statistics, normalise (r, w), add + ReLU (r, r, w)
    for _ in range(blocks):
        f += 4 * S                            # mask + BN3 sums: read g, out, y3; write gm
        _unit_fused_bwd(f, m, width, c, 1, e, 2 * S, None)
        _unit_fused_bwd(f, m, width, width, 3, e, 2 * Sw, None)
        f += 2 * Sw + w1 + 2 * S              # first CONV dgrad: (dy1, y1) in, accumulate into gm
        f += S + 2 * Sw + 4 * c * width       # its wgrad: X and (dy1, y1)
        u += 3 * S + 2 * S + 3 * S            # ReLU backward (r, r, w), BN3 sums (r, r), BN3 dx (r, r, w)
        _unit_ref_bwd(u, m, width, c, 1, e, S, False)
        _unit_ref_bwd(u, m, width, width, 3, e, Sw, False)
        u += Sw + w1 + 2 * S + S + Sw + 4 * c * width
    return {"fused": f.total, "unfused": u.total}


def for_workload(name, data):
    e = 2 if data.get("bf16") else 4
    if name == "single_layer":
        n, h, w, ci = data["x"].shape
        return single_layer(n * h * w, ci, data["w"].shape[3], e)
    if name == "bottleneck":
        n, h, w, ci = data["x"].shape
        p = data["p"]
        return bottleneck(n * h * w, ci, p["w1"].shape[3], p["w2"].shape[3], e)
    if name == "resnet_stack":
        n, h, w, c = data["x"].shape
        return resnet_stack(n * h * w, c, data["blocks"][0]["w1"].shape[3], len(data["blocks"]), e)
    if name == "densenet121":
        n, hw, _, c_in = data["img"].shape
        blocks = [(b["c0"], len(b["cpls"]), b["cpls"][0]["w1"].shape[3], b["cpls"][0]["w2"].shape[3],
                   b["trans"]["w"].shape[3] if b["trans"] is not None else 0) for b in data["blocks"]]
        return densenet(n, hw, c_in, data["stem"]["w"].shape[3], blocks, data["head"]["w"].shape[1], e)
    n, h, w, c0 = data["x"].shape
    cp = data["cpls"]
    return dense_block(n * h * w, c0, len(cp), cp[0]["w1"].shape[3], cp[0]["w2"].shape[3],
                       data["trans"]["w"].shape[3], e)
