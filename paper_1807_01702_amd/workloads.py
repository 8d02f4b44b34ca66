"""Training-step drivers for the synthetic workloads, fused and unfused.

Each driver owns its device buffers (allocated once), sequences C-ABI calls of
``libbnr`` for one training step (forward + backward, no optimizer update) and
exposes the results for parity checks.  ``fused=True`` runs the BN
fission/fusion path (Sec. 3.2 of the paper); ``fused=False`` runs the same math
through ``bnr_reference_path`` (the unfused BN -> ReLU -> CONV chain with
materialised intermediates, Sec. 3.2 "before" picture).

Workloads (shapes of the paper's DenseNet-121 / ResNet-50 training):
* ``SingleLayer``  -- one BN-ReLU-CONV1x1 layer.
* ``Bottleneck``   -- one DenseNet composite layer BN-ReLU-CONV1x1(4k)-BN-ReLU-
                      CONV3x3(k) whose k new channels are concatenated (Sec. 2.3).
* ``DenseBlock``   -- dense block 1 (6 composite layers, growth 32, width 128,
                      64 -> 256 channels) + transition BN-ReLU-CONV1x1 + 2x2
                      average pooling.
* ``DenseNet``     -- the whole network: first CONV, max pooling, dense blocks
                      and transitions, classifier head with its loss.
* ``ResNetStack``  -- ResNet-50 conv2_x bottleneck blocks with identity
                      shortcuts.  Concat is a channel-offset buffer
                      (pointer passing, as the paper's reference does for
                      Split); Split's backward is the accumulation of every
                      reader's input gradient into that buffer's gradient.
"""
import numpy as np
import torch

from . import bnr as B

MODE = B.MODE_BASELINE


def _t(a, dev, bf16):
    t = torch.from_numpy(np.ascontiguousarray(np.asarray(a, dtype=np.float32))).to(dev)
    return t.to(torch.bfloat16) if bf16 else t


def _dense(flat, n, h, w, c):
    """Dense [n, h, w, c] tensor on the front of a flat scratch buffer."""
    return flat[:n * h * w * c].view(n, h, w, c)


def _f32(a, dev):
    return torch.from_numpy(np.ascontiguousarray(np.asarray(a, dtype=np.float32))).to(dev)


class _Grads:
    def __init__(self, c, dev):
        self.dgamma = torch.empty(c, dtype=torch.float32, device=dev)
        self.dbeta = torch.empty(c, dtype=torch.float32, device=dev)


class _Unit:
    """One BN -> ReLU -> CONV chain on views x (BN input) -> out (CONV output)."""

    def __init__(self, n, h, w, x, out, k, gamma, beta, wt, eps, dev, bf16, fused, ref_mode=MODE):
        self.n, self.h, self.w, self.k = n, h, w, k
        self.x, self.out = x, out
        self.desc = B.desc_for(x, out, k, n, h, w)
        self.bn = B.BN(_f32(gamma, dev), _f32(beta, dev), eps)
        self.wt = _t(wt, dev, bf16)
        ci, co = x.shape[-1], out.shape[-1]
        self.dw = torch.empty(tuple(wt.shape), dtype=torch.float32, device=dev)
        self.g = _Grads(ci, dev)
        self.fused, self.ref_mode = fused, ref_mode
        dt = torch.bfloat16 if bf16 else torch.float32
        if not fused:   # materialised intermediates of the unfused chain, kept from forward to backward
            self.y = torch.empty(x.shape[:-1] + (ci,), dtype=dt, device=dev)
            self.z = torch.empty_like(self.y) if ref_mode == B.MODE_BASELINE else None

    # unfused forward / backward through the reference path
    def ref_fwd(self):
        B.bnr_reference_path(self.ref_mode, False, self.desc, self.x, self.bn, self.wt, self.y, z=self.z,
                             out=self.out)

    def ref_bwd(self, g, dz, dy, dx, accumulate):
        B.bnr_reference_path(self.ref_mode, True, self.desc, self.x, self.bn, self.wt, self.y, z=self.z, g=g,
                             dz=dz if self.ref_mode == B.MODE_BASELINE else None, dy=dy, dw=self.dw,
                             dgamma=self.g.dgamma, dbeta=self.g.dbeta, dx=dx, dx_accumulate=accumulate)


class SingleLayer:
    """BN-ReLU-CONV1x1 (fp32 by default): x [n,h,w,c_in] -> out [n,h,w,c_out],
    upstream gradient dy of out given."""

    def __init__(self, data, device="cuda", fused=True, ref_mode=MODE):
        bf16 = data["bf16"]
        dev = torch.device(device)
        n, h, w, ci = data["x"].shape
        co = data["w"].shape[3]
        self.x = _t(data["x"], dev, bf16)
        self.out = torch.empty((n, h, w, co), dtype=self.x.dtype, device=dev)
        self.gout = _t(data["dy"], dev, bf16)
        self.u = _Unit(n, h, w, self.x, self.out, 1, data["gamma"], data["beta"], data["w"], data["eps"], dev, bf16,
                       fused, ref_mode)
        self.out_bn = B.BN.stats_only(co, dev, data["eps"])     # statistics of the CONV output (CONV-sub-BN1)
        self.dy = torch.empty_like(self.x)
        self.dx = torch.empty_like(self.x)
        self.dz = torch.empty_like(self.x) if not fused else None
        self.fused = fused
        self.images = n

    def forward(self):
        u = self.u
        if self.fused:
            B.bnr_bn_stats(u.x, u.bn)
            B.bnr_bn_relu_conv_fwd(u.desc, u.x, u.bn, u.wt, u.out, self.out_bn)
        else:
            u.ref_fwd()

    def backward(self):
        u = self.u
        if self.fused:
            B.bnr_bwd_fused(u.desc, u.x, u.bn, u.wt, B.grad_dense(self.gout), u.dw, u.g.dgamma, u.g.dbeta, self.dy,
                            self.dx)
        else:
            u.ref_bwd(self.gout, self.dz, self.dy, self.dx, False)

    def step(self):
        self.forward()
        self.backward()


class Bottleneck:
    """One DenseNet composite layer with concatenated output Y = [X, CPL(X)].
    The upstream gradient dY covers all of Y; dX = dY[..., :c_in] + dx."""

    def __init__(self, data, device="cuda", fused=True, ref_mode=MODE):
        bf16 = data["bf16"]
        dev = torch.device(device)
        p = data["p"]
        n, h, w, ci = data["x"].shape
        width, k = p["w1"].shape[3], p["w2"].shape[3]
        dt = torch.bfloat16 if bf16 else torch.float32
        self.n, self.h, self.w, self.ci, self.k = n, h, w, ci, k
        self.buf = torch.empty((n, h, w, ci + k), dtype=dt, device=dev)
        self.buf[..., :ci] = _t(data["x"], dev, bf16)
        self.x1 = torch.empty((n, h, w, width), dtype=dt, device=dev)
        eps = data["eps"]
        self.u1 = _Unit(n, h, w, self.buf[..., :ci], self.x1, 1, p["gamma1"], p["beta1"], p["w1"], eps, dev, bf16,
                        fused, ref_mode)
        self.u2 = _Unit(n, h, w, self.x1, self.buf[..., ci:], 3, p["gamma2"], p["beta2"], p["w2"], eps, dev, bf16,
                        fused, ref_mode)
        self.dY = _t(data["dy"], dev, bf16)
        self.G = torch.empty_like(self.dY)          # gradient of the concatenated buffer
        self.dy1 = torch.empty((n, h, w, ci), dtype=dt, device=dev)
        self.dy2 = torch.empty((n, h, w, width), dtype=dt, device=dev)
        if not fused:
            self.dz1 = torch.empty_like(self.dy1)
            self.dz2 = torch.empty_like(self.dy2) if ref_mode == B.MODE_BASELINE else None
            self.dx2 = torch.empty_like(self.dy2)
        self.fused = fused
        self.images = n

    def forward(self):
        if self.fused:
            u1, u2 = self.u1, self.u2
            B.bnr_bn_stats(u1.x, u1.bn)
            B.bnr_bn_relu_conv_fwd(u1.desc, u1.x, u1.bn, u1.wt, u1.out, u2.bn)     # BN2 statistics in the epilogue
            B.bnr_bn_relu_conv_fwd(u2.desc, u2.x, u2.bn, u2.wt, u2.out)
        else:
            self.u1.ref_fwd()
            self.u2.ref_fwd()

    def backward(self):
        B.bnr_hbm_copy(self.dY, self.G)             # Split backward starts from the upstream gradient
        ci = self.ci
        u1, u2 = self.u1, self.u2
        if self.fused:
            B.bnr_bwd_fused(u2.desc, u2.x, u2.bn, u2.wt, B.grad_dense(self.G[..., ci:]), u2.dw, u2.g.dgamma,
                            u2.g.dbeta, self.dy2)
            B.bnr_bwd_fused(u1.desc, u1.x, u1.bn, u1.wt,
                            B.grad_bn(self.dy2, u2.x, u2.bn, u2.g.dgamma, u2.g.dbeta),
                            u1.dw, u1.g.dgamma, u1.g.dbeta, self.dy1, self.G[..., :ci], dx_accumulate=True)
        else:
            u2.ref_bwd(self.G[..., ci:], self.dz2, self.dy2, self.dx2, False)
            u1.ref_bwd(self.dx2, self.dz1, self.dy1, self.G[..., :ci], True)

    def step(self):
        self.forward()
        self.backward()


class _DenseStage:
    """One dense block of composite layers over a concatenation buffer X
    [n, h, w, ct] whose channels [0, c0) hold the block input (layer l writes
    channels [c0 + l*k, c0 + (l+1)*k)), optionally followed by its transition
    BN-ReLU-CONV1x1 + 2x2 average pooling into a caller-provided view.

    ``icf`` (fused only): inter-composite-layer fusion (Sec. 3.2, last
    paragraph).  Every BN reading a channel of X sees the same values, so the
    statistics live once per channel in shared arrays: one sweep (or the
    producer's epilogue) for the block input, the 3x3 CONV epilogues for every
    new slice; no BN1 sweeps its input.  Backward: the concatenation gradient
    G holds the summed form D = sum_l gamma_l rstd dy_l (written by the BN
    that reads the whole block -- the transition's or the classifier head's --
    and added by each BN1's data-gradient epilogue) plus per-channel
    alpha/betap; each 3x3 CONV's backward forms its slice's gradient on load,
    and one pass materialises the block input's gradient at the end.  Without
    ICF each BN1 sweeps its input for statistics and its input gradient is
    formed by a separate pass accumulating into G.

    ``o2`` (fused without ICF only): the paper's own sweep structure -- each
    composite layer's fused forwards also store the BN+ReLU output they feed
    to their CONV (O2'), and the backwards read it in place of recomputing it
    from the BN input (bnr_bn_relu_conv_fwd_o2 / bnr_bwd_fused_o2); every
    layer keeps its two stored tensors from forward to backward."""

    def __init__(self, n, h, w, c0, ct, cpls, trans, eps, dev, bf16, fused, icf, ref_mode=MODE, overlap=False,
                 robust=False, o2=False):
        dt = torch.bfloat16 if bf16 else torch.float32
        self.n, self.h, self.w, self.c0, self.ct = n, h, w, c0, ct
        self.X = torch.zeros((n, h, w, ct), dtype=dt, device=dev)
        self.cpl = []
        c_l = c0
        width = cpls[0]["w1"].shape[3]
        for p in cpls:
            k = p["w2"].shape[3]
            x1 = torch.empty((n, h, w, width), dtype=dt, device=dev)
            u1 = _Unit(n, h, w, self.X[..., :c_l], x1, 1, p["gamma1"], p["beta1"], p["w1"], eps, dev, bf16, fused,
                       ref_mode)
            u2 = _Unit(n, h, w, x1, self.X[..., c_l:c_l + k], 3, p["gamma2"], p["beta2"], p["w2"], eps, dev, bf16,
                       fused, ref_mode)
            self.cpl.append((c_l, k, u1, u2))
            c_l += k
        assert c_l == ct
        self.ut = None
        if trans is not None:
            to = trans["w"].shape[3]
            # the fused transition writes only its pooled output (BN, ReLU and
            # the 2x2 average in the CONV's prologue): t is then a shape
            # placeholder that no kernel touches
            self.t = (torch.empty((n, h, w, to), dtype=dt, device=dev) if not fused else
                      torch.empty((1, 1, 1, to), dtype=dt, device=dev).expand(n, h, w, to))
            self.ut = _Unit(n, h, w, self.X, self.t, 1, trans["gamma"], trans["beta"], trans["w"], eps, dev, bf16,
                            fused, ref_mode)
            if fused:
                self.ut.desc.out_ldc = to     # the backward's descriptor: a dense full-resolution output
            self.dy_t = torch.empty((n, h, w, ct), dtype=dt, device=dev)
            if not fused:
                self.dt = torch.empty_like(self.t)
        self.G = torch.empty((n, h, w, ct), dtype=dt, device=dev)
        self.dy1_flat = torch.empty(n * h * w * ct, dtype=dt, device=dev)    # dense [m][c_l] scratch, c_l < ct
        self.dy2 = torch.empty((n, h, w, width), dtype=dt, device=dev)
        # overlap (off by default: measured no faster, the persistent CONV kernels hold every CU): every
        # layer's weight gradients run on a side stream while the data gradients of the layers before
        # it proceed; a layer's BN2 gradient dy2 is then read after the next layer's data gradient has
        # started, so each layer keeps its own dy2
        self.overlap = bool(overlap) and fused
        self.dy2s = ([torch.empty((n, h, w, width), dtype=dt, device=dev) for _ in cpls] if self.overlap
                     else [self.dy2] * len(cpls))
        self._side = torch.cuda.Stream(device=dev) if self.overlap else None
        if not fused:
            self.dz_flat = torch.empty(n * h * w * max(ct, width), dtype=dt, device=dev)
            self.dx2 = torch.empty_like(self.dy2)
        self.fused = fused
        # called as layer_hook(i) after composite layer i's backward calls have
        # been issued (i = 0 .. len(cpls)-1, in backward order), e.g. to take
        # that layer's dy2 before the next layer reuses the buffer
        self.layer_hook = None
        self.icf = bool(icf)
        if self.icf and not fused:
            raise ValueError("inter-composite-layer fusion needs the fused path")
        self.o2 = bool(o2)
        if self.o2 and (not fused or self.icf or self.overlap):
            raise ValueError("the stored-O2' variant is wired for the fused path without inter-composite-layer "
                             "fusion or overlap")
        # per layer: relu(bn1(X[..., :c_l])) and relu(bn2(x1)), written by the forward, read by the backward
        self.z = ([(torch.empty((n, h, w, c_l), dtype=dt, device=dev),
                    torch.empty((n, h, w, u2.x.shape[-1]), dtype=dt, device=dev)) for c_l, k, u1, u2 in self.cpl]
                  if self.o2 else None)
        if self.icf:
            f32 = dict(dtype=torch.float32, device=dev)
            self.mu, self.var, self.rstd = (torch.empty(ct, **f32) for _ in range(3))
            self.alpha, self.betap = torch.empty(ct, **f32), torch.empty(ct, **f32)
            self.in_stats = B.BN.stats_view(eps, **self.shared(0, c0))         # block input channels
            self.slice_stats = []
            for c_l, k, u1, u2 in self.cpl:
                u1.bn = B.BN(u1.bn.gamma, u1.bn.beta, eps, **self.shared(0, c_l))
                self.slice_stats.append(B.BN.stats_view(eps, **self.shared(c_l, c_l + k)))
            if self.ut is not None:
                self.ut.bn = B.BN(self.ut.bn.gamma, self.ut.bn.beta, eps, **self.shared(0, ct))
        # robust one-sweep statistics: every statistics producer of the block sums
        # around its channels' running mean (the shift, updated in place by the
        # producer's finalisation together with the running variance)
        self.robust = bool(robust)
        if self.robust:
            if not self.icf:
                raise ValueError("robust statistics are wired for the fused path with inter-composite-layer fusion")
            f32 = dict(dtype=torch.float32, device=dev)
            self.run_mean, self.run_var = torch.zeros(ct, **f32), torch.ones(ct, **f32)

            def rob(bn, rm, rv):
                bn.robust(shift=rm, running_mean=rm, running_var=rv, momentum=0.1)

            rob(self.in_stats, self.run_mean[:c0], self.run_var[:c0])
            for (c_l, k, u1, u2), st in zip(self.cpl, self.slice_stats):
                rob(st, self.run_mean[c_l:c_l + k], self.run_var[c_l:c_l + k])
                wd = u2.bn.gamma.shape[0]
                rob(u2.bn, torch.zeros(wd, **f32), torch.ones(wd, **f32))

    def shared(self, lo, hi):
        """Views of the shared per-channel statistics of channels [lo, hi)."""
        return dict(mean=self.mu[lo:hi], var=self.var[lo:hi], rstd=self.rstd[lo:hi])

    def _pool_desc(self, pooled):
        """Descriptor of the fused transition writing the pooled view."""
        ut = self.ut
        return B.conv_desc(self.n, self.h, self.w, ut.desc.c_in, ut.desc.c_out, 1, ut.desc.in_ldc, B.view(pooled)[3],
                           ut.desc.dtype)

    def forward(self, pooled=None, in_stats_done=False, pooled_bn=None):
        """Composite layers, then (with a transition) its CONV and the 2x2
        pooling into the view `pooled` (fused: pooled before the CONV, in its
        prologue; pooled_bn: statistics of the pooled output from the CONV's
        epilogue).  in_stats_done (ICF): the block input's statistics are
        already in the shared arrays."""
        if self.icf:
            if not in_stats_done:
                B.bnr_bn_stats(self.X[..., :self.c0], self.in_stats)           # the one statistics sweep
            for (c_l, k, u1, u2), st in zip(self.cpl, self.slice_stats):
                B.bnr_bn_relu_conv_fwd(u1.desc, u1.x, u1.bn, u1.wt, u1.out, u2.bn)
                B.bnr_bn_relu_conv_fwd(u2.desc, u2.x, u2.bn, u2.wt, u2.out, st)   # the new slice's statistics
            ut = self.ut
            if ut is not None:
                B.bnr_bn_relu_conv_pool_fwd(self._pool_desc(pooled), ut.x, ut.bn, ut.wt, pooled, pooled_bn)
        elif self.fused:
            for i, (c_l, k, u1, u2) in enumerate(self.cpl):
                B.bnr_bn_stats(u1.x, u1.bn)                                    # sub-BN1 of a concat: own sweep
                if self.o2:
                    z1, z2 = self.z[i]
                    B.bnr_bn_relu_conv_fwd_o2(u1.desc, u1.x, u1.bn, u1.wt, u1.out, z1, u2.bn)
                    B.bnr_bn_relu_conv_fwd_o2(u2.desc, u2.x, u2.bn, u2.wt, u2.out, z2)
                    continue
                B.bnr_bn_relu_conv_fwd(u1.desc, u1.x, u1.bn, u1.wt, u1.out, u2.bn)
                B.bnr_bn_relu_conv_fwd(u2.desc, u2.x, u2.bn, u2.wt, u2.out)
            ut = self.ut
            if ut is not None:
                B.bnr_bn_stats(ut.x, ut.bn)
                B.bnr_bn_relu_conv_pool_fwd(self._pool_desc(pooled), ut.x, ut.bn, ut.wt, pooled, pooled_bn)
        else:
            for c_l, k, u1, u2 in self.cpl:
                u1.ref_fwd()
                u2.ref_fwd()
            if self.ut is not None:
                self.ut.ref_fwd()
                B.bnr_avgpool2_fwd(self.t, pooled, self.n, self.h, self.w)

    def backward(self, dpool=None):
        """With a transition: dpool is the gradient view of the pooled output,
        and the transition's backward starts G.  Without one the BN that
        reads the whole block (the classifier head) has already written G
        (and, with ICF, alpha/betap).  On return G[..., :c0] holds the
        gradient of the block input (and, with overlap, the side stream's
        weight gradients are joined into the current stream)."""
        if self.overlap:
            self._backward_overlapped(dpool)
            return
        ut = self.ut
        n, h, w = self.n, self.h, self.w
        if self.icf:
            c0 = self.c0
            if ut is not None:
                B.bnr_bwd_fused_split(ut.desc, ut.x, ut.bn, ut.wt, B.grad_avgpool2(dpool), ut.dw, ut.g.dgamma,
                                      ut.g.dbeta, self.G, self.alpha, self.betap)
            for i, ((c_l, k, u1, u2), st) in reversed(list(enumerate(zip(self.cpl, self.slice_stats)))):
                sl = slice(c_l, c_l + k)
                B.bnr_bwd_fused(u2.desc, u2.x, u2.bn, u2.wt,
                                B.grad_split(self.G[..., sl], self.X[..., sl], st, self.alpha[sl], self.betap[sl]),
                                u2.dw, u2.g.dgamma, u2.g.dbeta, self.dy2)
                B.bnr_bwd_fused_split(u1.desc, u1.x, u1.bn, u1.wt,
                                      B.grad_bn(self.dy2, u2.x, u2.bn, u2.g.dgamma, u2.g.dbeta),
                                      u1.dw, u1.g.dgamma, u1.g.dbeta, self.G[..., :c_l], self.alpha[:c_l],
                                      self.betap[:c_l], accumulate=True)
                if self.layer_hook is not None:
                    self.layer_hook(i)
            B.bnr_split_dx(self.G[..., :c0], self.X[..., :c0], self.in_stats, self.alpha[:c0], self.betap[:c0],
                           self.G[..., :c0])
        elif self.fused:
            if ut is not None:
                B.bnr_bwd_fused(ut.desc, ut.x, ut.bn, ut.wt, B.grad_avgpool2(dpool), ut.dw, ut.g.dgamma,
                                ut.g.dbeta, self.dy_t, self.G)
            for i, (c_l, k, u1, u2) in reversed(list(enumerate(self.cpl))):
                if self.o2:
                    z1, z2 = self.z[i]
                    B.bnr_bwd_fused_o2(u2.desc, u2.x, u2.bn, z2, u2.wt, B.grad_dense(self.G[..., c_l:c_l + k]),
                                       u2.dw, u2.g.dgamma, u2.g.dbeta, self.dy2)
                    B.bnr_bwd_fused_o2(u1.desc, u1.x, u1.bn, z1, u1.wt,
                                       B.grad_bn(self.dy2, u2.x, u2.bn, u2.g.dgamma, u2.g.dbeta),
                                       u1.dw, u1.g.dgamma, u1.g.dbeta, _dense(self.dy1_flat, n, h, w, c_l),
                                       self.G[..., :c_l], dx_accumulate=True)
                    continue
                B.bnr_bwd_fused(u2.desc, u2.x, u2.bn, u2.wt, B.grad_dense(self.G[..., c_l:c_l + k]), u2.dw,
                                u2.g.dgamma, u2.g.dbeta, self.dy2)
                B.bnr_bwd_fused(u1.desc, u1.x, u1.bn, u1.wt,
                                B.grad_bn(self.dy2, u2.x, u2.bn, u2.g.dgamma, u2.g.dbeta),
                                u1.dw, u1.g.dgamma, u1.g.dbeta, _dense(self.dy1_flat, n, h, w, c_l),
                                self.G[..., :c_l], dx_accumulate=True)
        else:
            if ut is not None:
                B.bnr_avgpool2_bwd(dpool, self.dt, n, h, w)
                ut.ref_bwd(self.dt, _dense(self.dz_flat, n, h, w, self.ct), self.dy_t, self.G, False)
            for c_l, k, u1, u2 in reversed(self.cpl):
                width = u2.x.shape[-1]
                u2.ref_bwd(self.G[..., c_l:c_l + k], _dense(self.dz_flat, n, h, w, width), self.dy2, self.dx2, False)
                u1.ref_bwd(self.dx2, _dense(self.dz_flat, n, h, w, c_l), _dense(self.dy1_flat, n, h, w, c_l),
                           self.G[..., :c_l], True)

    def _weights(self, u, g_src):
        """u's weight gradient on the side stream, after everything issued so
        far on the current stream (which completes g_src)."""
        main = torch.cuda.current_stream()
        self._side.wait_stream(main)
        with torch.cuda.stream(self._side):
            B.bnr_bwd_weights(u.desc, u.x, u.bn, g_src, u.dw, slot=1)

    def _backward_overlapped(self, dpool):
        """The fused backward with every weight gradient on the side stream.
        A weight gradient reads its layer's input and gradient source only:
        the later data gradients on the current stream write other channels
        of G, alpha, betap (and their own dy2), never what it reads."""
        ut = self.ut
        n, h, w = self.n, self.h, self.w
        main = torch.cuda.current_stream()
        if self.icf:
            c0 = self.c0
            if ut is not None:
                g = B.grad_avgpool2(dpool)
                self._weights(ut, g)
                B.bnr_bwd_data_split(ut.desc, ut.x, ut.bn, ut.wt, g, ut.g.dgamma, ut.g.dbeta, self.G, self.alpha,
                                     self.betap)
            for (c_l, k, u1, u2), st, dy2 in zip(reversed(self.cpl), reversed(self.slice_stats), reversed(self.dy2s)):
                sl = slice(c_l, c_l + k)
                g2 = B.grad_split(self.G[..., sl], self.X[..., sl], st, self.alpha[sl], self.betap[sl])
                self._weights(u2, g2)
                B.bnr_bwd_data(u2.desc, u2.x, u2.bn, u2.wt, g2, u2.g.dgamma, u2.g.dbeta, dy2)
                g1 = B.grad_bn(dy2, u2.x, u2.bn, u2.g.dgamma, u2.g.dbeta)
                self._weights(u1, g1)
                B.bnr_bwd_data_split(u1.desc, u1.x, u1.bn, u1.wt, g1, u1.g.dgamma, u1.g.dbeta, self.G[..., :c_l],
                                     self.alpha[:c_l], self.betap[:c_l], accumulate=True)
            B.bnr_split_dx(self.G[..., :c0], self.X[..., :c0], self.in_stats, self.alpha[:c0], self.betap[:c0],
                           self.G[..., :c0])
        else:
            if ut is not None:
                g = B.grad_avgpool2(dpool)
                self._weights(ut, g)
                B.bnr_bwd_data(ut.desc, ut.x, ut.bn, ut.wt, g, ut.g.dgamma, ut.g.dbeta, self.dy_t, self.G)
            for (c_l, k, u1, u2), dy2 in zip(reversed(self.cpl), reversed(self.dy2s)):
                g2 = B.grad_dense(self.G[..., c_l:c_l + k])
                self._weights(u2, g2)
                B.bnr_bwd_data(u2.desc, u2.x, u2.bn, u2.wt, g2, u2.g.dgamma, u2.g.dbeta, dy2)
                g1 = B.grad_bn(dy2, u2.x, u2.bn, u2.g.dgamma, u2.g.dbeta)
                self._weights(u1, g1)
                B.bnr_bwd_data(u1.desc, u1.x, u1.bn, u1.wt, g1, u1.g.dgamma, u1.g.dbeta,
                               _dense(self.dy1_flat, n, h, w, c_l), self.G[..., :c_l], dx_accumulate=True)
        main.wait_stream(self._side)


class DenseBlock(_DenseStage):
    """Dense block 1 of DenseNet-121 + transition layer on a given block
    input; upstream gradient: dpool of the pooled output.  ``icf`` defaults
    to on for the fused path (see _DenseStage)."""

    def __init__(self, data, device="cuda", fused=True, ref_mode=MODE, icf=None, overlap=False, robust=False,
                 o2=False):
        bf16 = data["bf16"]
        dev = torch.device(device)
        dt = torch.bfloat16 if bf16 else torch.float32
        n, h, w, c0 = data["x"].shape
        super().__init__(n, h, w, c0, data["c_total"], data["cpls"], data["trans"], data["eps"], dev, bf16, fused,
                         fused if icf is None else icf, ref_mode, overlap, robust, o2)
        self.X[..., :c0] = _t(data["x"], dev, bf16)
        to = data["trans"]["w"].shape[3]
        self.pooled = torch.empty((n, h // 2, w // 2, to), dtype=dt, device=dev)
        self.dpool = _t(data["dpool"], dev, bf16)
        self.images = n

    def forward(self):
        super().forward(self.pooled)

    def backward(self):
        super().backward(self.dpool)

    def step(self):
        self.forward()
        self.backward()


class DenseNet:
    """A whole DenseNet training step (forward and backward of the mean
    softmax cross-entropy; no optimizer update): first CONV 7x7/2 -> BN ->
    ReLU -> 3x3/2 max pooling, dense blocks joined by transitions
    (_DenseStage), and the head BN -> ReLU -> global average pooling -> FC.

    fused=True: BN fission/fusion with inter-composite-layer fusion in every
    block.  The first CONV's epilogue produces its BN's statistics; the max
    pooling applies that BN and the ReLU while reading and produces the
    statistics of block 1's input; a transition's pooled output is written
    into the next block's buffer and swept once for statistics; the head's BN
    reads the shared statistics of the last block.  Backward: the head's BN
    backward writes the last block's summed gradient (D, alpha, betap); each
    block materialises the gradient of its input, which is the next-lower
    transition's pooled-output gradient (formed on load by its CONV) or, for
    block 1, the max pooling's output gradient; the pooling backward applies
    the ReLU mask and the first BN's reductions, and the first CONV's weight
    gradient forms that BN's input gradient on load.

    fused=False: the unfused chain: first CONV, two-pass BN statistics,
    normalise and ReLU sweeps, plain max pooling; blocks through
    bnr_reference_path; backward with materialised pooling, ReLU and BN input
    gradients.  (The head BN's statistics come from one sweep and its ReLU is
    applied while the head pools in both paths: its tensors are three orders
    of magnitude smaller than the first BN's.)"""

    def __init__(self, data, device="cuda", fused=True, ref_mode=MODE):
        bf16 = data["bf16"]
        dev = torch.device(device)
        dt = torch.bfloat16 if bf16 else torch.float32
        eps = data["eps"]
        img = np.asarray(data["img"], np.float32)
        n, H, W, ci = img.shape
        self.n, self.H, self.W, self.ci = n, H, W, ci
        img4 = np.zeros((n, H, W, 4), np.float32)
        img4[..., :ci] = img
        self.img = _t(img4, dev, bf16)
        st = data["stem"]
        self.w0 = _t(st["w"], dev, bf16)
        c_stem = st["w"].shape[3]
        self.hs, self.ws_ = (H - 1) // 2 + 1, (W - 1) // 2 + 1
        self.s = torch.empty((n, self.hs, self.ws_, c_stem), dtype=dt, device=dev)
        self.stem_bn = B.BN(_f32(st["gamma"], dev), _f32(st["beta"], dev), eps)
        self.dw0 = torch.empty(tuple(st["w"].shape), dtype=torch.float32, device=dev)
        self.g0 = _Grads(c_stem, dev)
        self.dy0 = torch.empty_like(self.s)
        h, w = (self.hs - 1) // 2 + 1, (self.ws_ - 1) // 2 + 1
        self.stages, self.hw = [], []
        for bd in data["blocks"]:
            self.stages.append(_DenseStage(n, h, w, bd["c0"], bd["c_total"], bd["cpls"], bd["trans"], eps, dev, bf16,
                                           fused, fused, ref_mode))
            self.hw.append((h, w))
            if bd["trans"] is not None:
                h, w = h // 2, w // 2
        last = self.stages[-1]
        hp = data["head"]
        C, K = hp["w"].shape
        self.C, self.K = C, K
        self.head_bn = B.BN(_f32(hp["gamma"], dev), _f32(hp["beta"], dev), eps,
                            **(last.shared(0, C) if fused else {}))
        self.wfc = _t(hp["w"], dev, bf16)
        self.bfc = _f32(hp["b"], dev)
        self.labels = torch.from_numpy(np.asarray(data["labels"], np.int32)).to(dev)
        f32 = dict(dtype=torch.float32, device=dev)
        self.f = torch.empty((n, C), **f32)
        self.logits, self.dlogits = torch.empty((n, K), **f32), torch.empty((n, K), **f32)
        self.loss = torch.empty(1 + n, **f32)
        self.df = torch.empty((n, C), **f32)
        self.dwfc, self.dbfc = torch.empty((C, K), **f32), torch.empty(K, **f32)
        self.g5 = _Grads(C, dev)
        if not fused:
            self.y0, self.z0 = torch.empty_like(self.s), torch.empty_like(self.s)
            self.dz0, self.dx0 = torch.empty_like(self.s), torch.empty_like(self.s)
        self.fused = fused
        self.images = n

    def forward(self):
        s0 = self.stages[0]
        n = self.n
        if self.fused:
            B.bnr_stem_conv_fwd(self.img, self.w0, self.s, self.stem_bn)
            B.bnr_bn_relu_maxpool_fwd(self.s, self.stem_bn, s0.X[..., :s0.c0], n, self.hs, self.ws_,
                                      y_bn=s0.in_stats)
        else:
            B.bnr_stem_conv_fwd(self.img, self.w0, self.s)
            B.bnr_reference_bn_relu(False, self.s, self.stem_bn, self.y0, z=self.z0)
            B.bnr_bn_relu_maxpool_fwd(self.z0, None, s0.X[..., :s0.c0], n, self.hs, self.ws_)
        for i, st in enumerate(self.stages):
            nxt = self.stages[i + 1] if i + 1 < len(self.stages) else None
            # fused: the transition's epilogue produces the next block's input statistics
            st.forward(nxt.X[..., :nxt.c0] if nxt is not None else None, in_stats_done=(i == 0 or self.fused),
                       pooled_bn=nxt.in_stats if nxt is not None and self.fused else None)
        last = self.stages[-1]
        h, w = self.hw[-1]
        if not self.fused:
            B.bnr_bn_stats(last.X, self.head_bn)
        B.bnr_head_fwd(last.X, self.head_bn, self.wfc, self.bfc, self.labels, self.f, self.logits, self.dlogits,
                       self.loss, n, h, w)

    def backward(self):
        n = self.n
        last = self.stages[-1]
        h, w = self.hw[-1]
        if self.fused:
            B.bnr_head_bwd(last.X, self.head_bn, self.wfc, self.f, self.dlogits, self.df, self.dwfc, self.dbfc,
                           self.g5.dgamma, self.g5.dbeta, last.G, n, h, w, alpha=last.alpha, betap=last.betap)
        else:
            B.bnr_head_bwd(last.X, self.head_bn, self.wfc, self.f, self.dlogits, self.df, self.dwfc, self.dbfc,
                           self.g5.dgamma, self.g5.dbeta, last.G, n, h, w)
        for i in range(len(self.stages) - 1, -1, -1):
            st = self.stages[i]
            nxt = self.stages[i + 1] if i + 1 < len(self.stages) else None
            st.backward(nxt.G[..., :nxt.c0] if nxt is not None else None)
        s0 = self.stages[0]
        dX = s0.G[..., :s0.c0]
        c_in = self.ci
        if self.fused:
            B.bnr_maxpool_bn_bwd(self.s, self.stem_bn, dX, self.dy0, n, self.hs, self.ws_, self.g0.dgamma,
                                 self.g0.dbeta)
            B.bnr_stem_wgrad(self.img, c_in, B.grad_bn(self.dy0, self.s, self.stem_bn, self.g0.dgamma, self.g0.dbeta),
                             self.dw0)
        else:
            B.bnr_maxpool_bn_bwd(self.z0, None, dX, self.dz0, n, self.hs, self.ws_)
            B.bnr_reference_bn_relu(True, self.s, self.stem_bn, self.y0, gz=self.dz0, dy=self.dy0,
                                    dgamma=self.g0.dgamma, dbeta=self.g0.dbeta, dx=self.dx0)
            B.bnr_stem_wgrad(self.img, c_in, B.grad_dense(self.dx0), self.dw0)

    def step(self):
        self.forward()
        self.backward()


class ResNetStack:
    """ResNet-50 conv2_x: bottleneck blocks CONV1x1(c -> width) - BN - ReLU -
    CONV3x3(width -> width) - BN - ReLU - CONV1x1(width -> c) - BN, + identity,
    ReLU (He et al., as used in the paper's ResNet-50 evaluation).

    Fused: every BN's statistics come from the epilogue of the CONV that
    produces its input; BN1/BN2 + ReLU run in the next CONV's prologue; the
    last BN of a block, the residual addition and the ReLU run in the
    prologue of the next block's first CONV, which also writes their result
    (the next block's identity); only the last block of the stack runs them
    as one element-wise sweep.  BN3's input gradient is consumed deferred by
    the third CONV's backward.  Unfused: the
    reference chain (two-pass statistics, materialised normalised / ReLU
    tensors and gradients)."""

    def __init__(self, data, device="cuda", fused=True, ref_mode=MODE):
        bf16 = data["bf16"]
        dev = torch.device(device)
        dt = torch.bfloat16 if bf16 else torch.float32
        n, h, w, c = data["x"].shape
        width = data["blocks"][0]["w1"].shape[3]
        self.n, self.h, self.w, self.c, self.width = n, h, w, c, width
        self.fused, self.images = fused, n
        eps = data["eps"]
        self.x0 = _t(data["x"], dev, bf16)
        self.gout = _t(data["dy"], dev, bf16)
        self.blocks = []
        xin = self.x0
        for p in data["blocks"]:
            b = dict(xin=xin)
            b["y1"] = torch.empty((n, h, w, width), dtype=dt, device=dev)
            b["y2"] = torch.empty_like(b["y1"])
            b["y3"] = torch.empty((n, h, w, c), dtype=dt, device=dev)
            b["out"] = torch.empty_like(b["y3"])
            b["w1"] = _t(p["w1"], dev, bf16)
            b["dw1"] = torch.empty(tuple(p["w1"].shape), dtype=torch.float32, device=dev)
            b["desc1"] = B.desc_for(xin, b["y1"], 1, n, h, w)
            # BN1 -> ReLU -> CONV3x3 and BN2 -> ReLU -> CONV1x1 as units
            b["u2"] = _Unit(n, h, w, b["y1"], b["y2"], 3, p["gamma1"], p["beta1"], p["w2"], eps, dev, bf16, fused,
                            ref_mode)
            b["u3"] = _Unit(n, h, w, b["y2"], b["y3"], 1, p["gamma2"], p["beta2"], p["w3"], eps, dev, bf16, fused,
                            ref_mode)
            b["bn3"] = B.BN(_f32(p["gamma3"], dev), _f32(p["beta3"], dev), eps)
            b["g3"] = _Grads(c, dev)
            self.blocks.append(b)
            xin = b["out"]
        self.out = xin
        self.gbuf = torch.empty_like(self.x0)                      # gradient of the current block input
        self.dyw = torch.empty((n, h, w, width), dtype=dt, device=dev)
        self.dyw2 = torch.empty_like(self.dyw)
        if not fused:
            self.tmp = torch.empty_like(self.x0)
            self.dx3 = torch.empty_like(self.x0)
            self.dyw3 = torch.empty_like(self.dyw)
            self.dzw = torch.empty_like(self.dyw)

    def forward(self):
        for i, b in enumerate(self.blocks):
            u2, u3 = b["u2"], b["u3"]
            if self.fused:
                if i == 0:
                    B.bnr_conv_bn_stats_fwd(b["desc1"], b["xin"], b["w1"], b["y1"], u2.bn)
                else:                          # the previous block's BN3 + identity + ReLU on load
                    pb = self.blocks[i - 1]
                    B.bnr_bn_add_relu_conv_fwd(b["desc1"], pb["y3"], pb["bn3"], pb["xin"], pb["out"], b["w1"],
                                               b["y1"], u2.bn)
                B.bnr_bn_relu_conv_fwd(u2.desc, u2.x, u2.bn, u2.wt, u2.out, u3.bn)
                B.bnr_bn_relu_conv_fwd(u3.desc, u3.x, u3.bn, u3.wt, u3.out, b["bn3"])
                if i == len(self.blocks) - 1:
                    B.bnr_bn_add_relu_fwd(b["y3"], b["bn3"], b["xin"], b["out"])
            else:
                B.bnr_conv_fwd(b["desc1"], b["xin"], b["w1"], b["y1"])
                u2.ref_fwd()
                u3.ref_fwd()
                B.bnr_reference_bn_add_relu(False, b["y3"], b["bn3"], b["out"], ident=b["xin"], tmp=self.tmp)

    def backward(self):
        g = self.gout
        for b in reversed(self.blocks):
            u2, u3, g3 = b["u2"], b["u3"], b["g3"]
            if self.fused:
                # gm = g * [out > 0] into gbuf (in place from the second block on), BN3 sums
                B.bnr_bn_add_relu_bwd(g, b["out"], b["y3"], b["bn3"], self.gbuf, g3.dgamma, g3.dbeta)
                B.bnr_bwd_fused(u3.desc, u3.x, u3.bn, u3.wt, B.grad_bn(self.gbuf, b["y3"], b["bn3"], g3.dgamma,
                                                                       g3.dbeta),
                                u3.dw, u3.g.dgamma, u3.g.dbeta, self.dyw)
                B.bnr_bwd_fused(u2.desc, u2.x, u2.bn, u2.wt, B.grad_bn(self.dyw, u3.x, u3.bn, u3.g.dgamma,
                                                                       u3.g.dbeta),
                                u2.dw, u2.g.dgamma, u2.g.dbeta, self.dyw2)
                # first CONV: its input has no BN in front; identity gradient + data gradient
                B.bnr_bwd_fused(b["desc1"], b["xin"], None, b["w1"], B.grad_bn(self.dyw2, u2.x, u2.bn,
                                                                               u2.g.dgamma, u2.g.dbeta),
                                b["dw1"], dx=self.gbuf, dx_accumulate=True)
            else:
                B.bnr_reference_bn_add_relu(True, b["y3"], b["bn3"], b["out"], g=g, gm=self.gbuf,
                                            dgamma=g3.dgamma, dbeta=g3.dbeta, dx=self.dx3)
                u3.ref_bwd(self.dx3, self.dzw, self.dyw, self.dyw2, False)
                u2.ref_bwd(self.dyw2, self.dzw, self.dyw, self.dyw3, False)
                B.bnr_bwd_fused(b["desc1"], b["xin"], None, b["w1"], B.grad_dense(self.dyw3), b["dw1"],
                                dx=self.gbuf, dx_accumulate=True)
            g = self.gbuf

    def step(self):
        self.forward()
        self.backward()
