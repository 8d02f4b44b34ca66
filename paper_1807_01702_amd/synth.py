"""Seeded synthetic inputs for the training workloads (host side, numpy).

This module only draws random numbers and rounds them to the storage format;
it holds none of the method's arithmetic.  Both the GPU path's callers and
the CPU oracle's callers take their inputs from here, so the two sides see
identical values.

Every tensor has its own stream: ``numpy.random.Generator(PCG64(SeedSequence
([seed, crc32(name)])))``, drawn in float64, cast to float32 and, for bf16
operands, rounded to the nearest bf16 value (ties to even).  Arrays are float32
(bf16 tensors hold bf16-representable values); ``bf16_bits`` gives the raw
16-bit words for upload.

Distributions (the configurations' own recipe): activations and upstream
gradients N(0, 1); BN scale gamma ~ U(0.5, 1.5); BN shift beta ~ N(0, 0.1)
(standard deviation 0.1); conv weights He-normal, std = sqrt(2 / (K*K*C_in)).
"""
import zlib

import numpy as np

EPS = 1e-5


def round_to_bf16(a):
    """float32 -> nearest bf16-representable float32 (ties to even)."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    u = a.view(np.uint32).astype(np.uint64)
    u = ((u + 0x7FFF + ((u >> 16) & 1)) >> 16) << 16
    return u.astype(np.uint32).view(np.float32).reshape(a.shape)


def bf16_bits(a):
    """bf16-representable float32 array -> uint16 words."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    return (a.view(np.uint32) >> 16).astype(np.uint16)


def from_bf16_bits(u16):
    u = np.ascontiguousarray(u16, dtype=np.uint16)
    return (u.astype(np.uint32) << 16).view(np.float32)


def _gen(seed, name):
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, zlib.crc32(name.encode())])))


def normal(seed, name, shape, std=1.0, bf16=False):
    a = (_gen(seed, name).standard_normal(size=shape) * std).astype(np.float32)
    return round_to_bf16(a) if bf16 else a


def uniform(seed, name, shape, lo, hi):
    return _gen(seed, name).uniform(lo, hi, size=shape).astype(np.float32)


def bn_params(seed, prefix, c):
    return dict(gamma=uniform(seed, prefix + ".gamma", (c,), 0.5, 1.5),
                beta=normal(seed, prefix + ".beta", (c,), 0.1))


def conv_weight(seed, name, k, c_in, c_out, bf16):
    return normal(seed, name, (k, k, c_in, c_out), std=float(np.sqrt(2.0 / (k * k * c_in))), bf16=bf16)


# ------------------------------------------------------ workload recipes ----
def single_layer(seed=0, n=8, h=8, w=8, c_in=64, c_out=32, bf16=False):
    """One BN-ReLU-CONV1x1 layer (fp32 NHWC, 8x8x8x64 -> 32 by default)."""
    p = bn_params(seed, "bn", c_in)
    return dict(x=normal(seed, "x", (n, h, w, c_in), bf16=bf16), gamma=p["gamma"], beta=p["beta"],
                w=conv_weight(seed, "w", 1, c_in, c_out, bf16), dy=normal(seed, "dy", (n, h, w, c_out), bf16=bf16),
                eps=EPS, bf16=bf16)


def cpl_params(seed, prefix, c_l, width, growth, bf16):
    p1, p2 = bn_params(seed, prefix + ".bn1", c_l), bn_params(seed, prefix + ".bn2", width)
    return dict(gamma1=p1["gamma"], beta1=p1["beta"], w1=conv_weight(seed, prefix + ".w1", 1, c_l, width, bf16),
                gamma2=p2["gamma"], beta2=p2["beta"], w2=conv_weight(seed, prefix + ".w2", 3, width, growth, bf16))


def bottleneck(seed=0, n=32, h=56, w=56, c_in=256, width=128, growth=32, bf16=True):
    """One DenseNet-121 bottleneck layer with concatenated output."""
    return dict(x=normal(seed, "x", (n, h, w, c_in), bf16=bf16),
                p=cpl_params(seed, "cpl", c_in, width, growth, bf16),
                dy=normal(seed, "dy", (n, h, w, c_in + growth), bf16=bf16), eps=EPS, bf16=bf16)


def dense_block(seed=0, n=64, h=56, w=56, c0=64, layers=6, width=128, growth=32, trans_out=128, bf16=True):
    """Dense block 1 of DenseNet-121 (6 composite layers) + transition layer."""
    cpls, c_l = [], c0
    for l in range(layers):
        cpls.append(cpl_params(seed, "cpl%d" % l, c_l, width, growth, bf16))
        c_l += growth
    tb = bn_params(seed, "trans.bn", c_l)
    trans = dict(gamma=tb["gamma"], beta=tb["beta"], w=conv_weight(seed, "trans.w", 1, c_l, trans_out, bf16))
    return dict(x=normal(seed, "x", (n, h, w, c0), bf16=bf16), cpls=cpls, trans=trans, c_total=c_l,
                dpool=normal(seed, "dpool", (n, h // 2, w // 2, trans_out), bf16=bf16), eps=EPS, bf16=bf16)


def resnet_stack(seed=0, n=128, h=56, w=56, c=256, width=64, blocks=3, bf16=True):
    """ResNet-50 conv2_x: `blocks` bottleneck blocks 256 -> 64 -> 64 -> 256."""
    ps = []
    for b in range(blocks):
        pre = "block%d" % b
        d = dict(w1=conv_weight(seed, pre + ".w1", 1, c, width, bf16),
                 w2=conv_weight(seed, pre + ".w2", 3, width, width, bf16),
                 w3=conv_weight(seed, pre + ".w3", 1, width, c, bf16))
        for i, ch in ((1, width), (2, width), (3, c)):
            bp = bn_params(seed, pre + ".bn%d" % i, ch)
            d["gamma%d" % i], d["beta%d" % i] = bp["gamma"], bp["beta"]
        ps.append(d)
    return dict(x=normal(seed, "x", (n, h, w, c), bf16=bf16), blocks=ps,
                dy=normal(seed, "dy", (n, h, w, c), bf16=bf16), eps=EPS, bf16=bf16)


def densenet(seed=0, n=128, hw=224, c_img=3, c_stem=64, growth=32, width=128, blocks=(6, 12, 24, 16),
             classes=1000, bf16=True):
    """A whole DenseNet training step: image [n, hw, hw, c_img] ~ N(0, 1),
    uniform random labels in [0, classes), 7x7 stem CONV (He-normal), BN
    parameters as everywhere, dense blocks of `blocks` composite layers with
    compression-1/2 transitions between them, and the classifier FC
    (weight N(0, 1/C), bias N(0, 0.1)).  Defaults: DenseNet-121 at 224x224."""
    stem_bn = bn_params(seed, "stem.bn", c_stem)
    d = dict(img=normal(seed, "img", (n, hw, hw, c_img), bf16=bf16),
             labels=_gen(seed, "labels").integers(0, classes, size=n).astype(np.int32),
             stem=dict(w=conv_weight(seed, "stem.w", 7, c_img, c_stem, bf16), gamma=stem_bn["gamma"],
                       beta=stem_bn["beta"]),
             blocks=[], eps=EPS, bf16=bf16)
    c0 = c_stem
    for b, layers in enumerate(blocks):
        cpls, c_l = [], c0
        for l in range(layers):
            cpls.append(cpl_params(seed, "b%d.cpl%d" % (b, l), c_l, width, growth, bf16))
            c_l += growth
        trans = None
        if b + 1 < len(blocks):
            tb = bn_params(seed, "b%d.trans.bn" % b, c_l)
            trans = dict(gamma=tb["gamma"], beta=tb["beta"],
                         w=conv_weight(seed, "b%d.trans.w" % b, 1, c_l, c_l // 2, bf16))
        d["blocks"].append(dict(cpls=cpls, trans=trans, c_total=c_l, c0=c0))
        c0 = c_l // 2
    hb = bn_params(seed, "head.bn", c_l)
    d["head"] = dict(gamma=hb["gamma"], beta=hb["beta"],
                     w=normal(seed, "head.w", (c_l, classes), std=float(1.0 / np.sqrt(c_l)), bf16=bf16),
                     b=normal(seed, "head.b", (classes,), 0.1))
    return d
