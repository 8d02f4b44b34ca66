"""Shared helpers of the GPU parity tests: upload/download, the tolerance
metric and the ReLU-decision ambiguity band.

Tolerance metric (per tensor): max |gpu - ref| / max |ref|, with rtol 1e-4 for
fp32 storage and 2e-2 for bf16 storage.  Batch statistics are compared per
channel: |mean_gpu - mean_ref| <= rtol * sigma_ref and
|var_gpu - var_ref| <= rtol * var_ref.

ReLU decisions.  dy = dz * [y > 0] is a discontinuous function of y: where the
oracle's fp64 y lies within the kernel's rounding of 0, both decisions are
correct.  Element-wise comparisons of tensors downstream of such a decision
exclude exactly those elements (their number is reported and bounded); all
reductions are compared without exclusions.
"""
import numpy as np
import torch

from paper_1807_01702_amd import synth

RTOL = {False: 1e-4, True: 2e-2}


def dev(a, bf16, device="cuda"):
    t = torch.from_numpy(np.ascontiguousarray(np.asarray(a, dtype=np.float32)))
    t = t.to(device)
    return t.to(torch.bfloat16) if bf16 else t


def f32dev(a, device="cuda"):
    return torch.from_numpy(np.ascontiguousarray(np.asarray(a, dtype=np.float32))).to(device)


def host(t):
    return t.detach().float().cpu().numpy().astype(np.float64)


def rel_err(gpu, ref, exclude=None):
    gpu = np.asarray(gpu, np.float64)
    ref = np.asarray(ref, np.float64)
    d = np.abs(gpu - ref)
    if exclude is not None:
        d = np.where(exclude, 0.0, d)
    scale = np.max(np.abs(ref))
    return float(np.max(d) / scale) if scale > 0 else float(np.max(d))


def assert_close(name, gpu, ref, rtol, exclude=None, max_excluded_frac=1e-3):
    if exclude is not None:
        frac = float(np.mean(exclude))
        assert frac <= max_excluded_frac, "%s: %.2e of elements in the ReLU ambiguity band" % (name, frac)
    e = rel_err(gpu, ref, exclude)
    assert e <= rtol, "%s: relative error %.3e > %.1e" % (name, e, rtol)
    return e


def assert_stats(name, mean_g, var_g, mean_r, var_r, rtol):
    mean_g, var_g = np.asarray(mean_g, np.float64), np.asarray(var_g, np.float64)
    sig = np.sqrt(var_r)
    em = np.max(np.abs(mean_g - mean_r) / np.maximum(sig, 1e-30))
    ev = np.max(np.abs(var_g - var_r) / np.maximum(var_r, 1e-30))
    assert em <= rtol, "%s mean: %.3e > %.1e (in units of sigma)" % (name, em, rtol)
    assert ev <= rtol, "%s var: relative %.3e > %.1e" % (name, ev, rtol)
    return em, ev


def relu_ambiguous(y, bf16):
    """Elements whose ReLU decision is within rounding of 0 at the kernel's
    precision (fp32 arithmetic on values the two sides hold identically)."""
    y = np.asarray(y, np.float64)
    band = (1e-5 if bf16 else 1e-6) * max(1.0, float(np.max(np.abs(y))))
    return np.abs(y) <= band


def relu_ambiguous_pixels(y, x_stored, gamma, rstd, bf16):
    """Pixels (rows of y [.., C]) holding a ReLU decision that the kernel's
    rounding can flip.  For a BN input that both sides hold exactly (an
    input tensor) the band is the fp32 arithmetic noise; for a BN input that
    each side rounds to bf16 itself (a CONV output) it is one bf16 ulp of that
    input, mapped through gamma * rstd."""
    y = np.asarray(y, np.float64)
    C = y.shape[-1]
    y2 = y.reshape(-1, C)
    band = relu_ambiguous(y2, bf16).astype(bool)
    if x_stored is not None and bf16:
        x = np.abs(np.asarray(x_stored, np.float64).reshape(-1, C))
        ulp = np.exp2(np.floor(np.log2(np.maximum(x, 1e-30))) - 7)
        band |= np.abs(y2) <= 2.0 * ulp * np.abs(np.asarray(gamma) * np.asarray(rstd))
    return band.any(axis=1)


def assert_close_pixels(name, gpu, ref, rtol, ambiguous_px, max_frac=1e-3):
    """Element-wise max-norm check in which a pixel may exceed the tolerance
    only if it holds an ambiguous ReLU decision (several results are correct
    there); such pixels must stay rare."""
    gpu = np.asarray(gpu, np.float64)
    ref = np.asarray(ref, np.float64)
    C = ref.shape[-1]
    err = np.abs(gpu - ref).reshape(-1, C)
    scale = np.max(np.abs(ref))
    bad_px = (err > rtol * scale).any(axis=1)
    unexplained = bad_px & ~ambiguous_px
    assert not unexplained.any(), "%s: %d pixels over %.1e not explained by an ambiguous ReLU decision" % (
        name, int(unexplained.sum()), rtol)
    assert bad_px.mean() <= max_frac, "%s: %.2e of pixels over tolerance" % (name, bad_px.mean())
    return int(bad_px.sum())


def bf16_round(a):
    return synth.round_to_bf16(np.asarray(a, np.float32)).astype(np.float64)
