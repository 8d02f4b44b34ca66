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


def bf16_round(a):
    return synth.round_to_bf16(np.asarray(a, np.float32)).astype(np.float64)
