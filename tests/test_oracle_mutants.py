"""Plants plausible mistakes in a copy of the CPU oracle and checks that the
pins in test_oracle_pins.py catch every one of them (CPU only).

Each mutant is a one-spot text edit of oracle/oracle.c, oracle/compose.py or
oracle/prims.py:
a flipped filter tap, a transposed weight index, an unbiased variance, a
dropped or sign-flipped term of the BN gradient, a wrong ReLU tie rule, a lost
concat-gradient accumulation, ...  The mutated copy (with the pins and the
golden fixtures) lives in a temporary directory; the real oracle is untouched.
"""
import os
import shutil
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

MUTANTS = [
    ("conv taps flipped (convolution, not correlation)", "oracle.c",
     "int iy = oy * stride + kh - pad, ix = ox * stride + kw - pad;\n                            if (iy < 0 || iy >= H || ix < 0 || ix >= W) continue;\n                            for (int ci",
     "int iy = oy * stride - kh + pad, ix = ox * stride - kw + pad;\n                            if (iy < 0 || iy >= H || ix < 0 || ix >= W) continue;\n                            for (int ci"),
    ("conv weight kh/kw transposed", "oracle.c",
     "acc += in[IDX4(n, iy, ix, ci, H, W, Ci)] *\n                                       wt[((long)(kh * K + kw)",
     "acc += in[IDX4(n, iy, ix, ci, H, W, Ci)] *\n                                       wt[((long)(kw * K + kh)"),
    ("dgrad tap offset sign", "oracle.c", "int ty = iy + pad - kh, tx = ix + pad - kw;",
     "int ty = iy - pad + kh, tx = ix - pad + kw;"),
    ("wgrad uses the wrong tap for the row", "oracle.c",
     "int iy = oy * stride + kh - pad, ix = ox * stride + kw - pad;\n                            if (iy < 0 || iy >= H || ix < 0 || ix >= W) continue;\n                            double a",
     "int iy = oy * stride + kw - pad, ix = ox * stride + kh - pad;\n                            if (iy < 0 || iy >= H || ix < 0 || ix >= W) continue;\n                            double a"),
    ("unbiased variance", "oracle.c", "double v = q / (double)m;", "double v = q / (double)(m > 1 ? m - 1 : 1);"),
    ("eps outside the square root", "oracle.c", "double r = 1.0 / sqrt(v + eps);", "double r = 1.0 / (sqrt(v) + eps);"),
    ("gamma and beta swapped", "oracle.c", "gamma[c] * ((x[i * C + c] - mu) * r) + beta[c]",
     "beta[c] * ((x[i * C + c] - mu) * r) + gamma[c]"),
    ("BN backward: xhat term sign", "oracle.c", "- xh * sg / (double)m);", "+ xh * sg / (double)m);"),
    ("BN backward: mean-gradient term dropped", "oracle.c", "(dy[i * C + c] - sb / (double)m - xh",
     "(dy[i * C + c] - xh"),
    ("BN backward: rstd factor dropped", "oracle.c", "dx[i * C + c] = gamma[c] * rstd[c] *", "dx[i * C + c] = gamma[c] *"),
    ("ReLU gradient passes at y == 0", "oracle.c", "dy[i] = y[i] > 0.0 ? dz[i] : 0.0;", "dy[i] = y[i] >= 0.0 ? dz[i] : 0.0;"),
    ("MVF drops the square of the mean", "oracle.c", "var[c] = e2 - e1 * e1;", "var[c] = e2 - e1;"),
    ("shifted MVF forgets to add the shift back", "oracle.c", "mean[c] = K[c] + d1;", "mean[c] = d1;"),
    ("shifted MVF squares the unshifted value", "oracle.c", "s += d; s2 += d * d; }",
     "s += d; s2 += x[i * C + c] * x[i * C + c]; }"),
    ("running variance kept biased", "oracle.c", "mo * var[c] * ((double)m / (double)(m - 1));", "mo * var[c];"),
    ("running mean momentum reversed", "oracle.c", "rmean[c] = (1.0 - mo) * rmean[c] + mo * mean[c];",
     "rmean[c] = mo * rmean[c] + (1.0 - mo) * mean[c];"),
    ("avgpool backward scale", "oracle.c", "gin[IDX4(n, iy, ix, c, H, W, C)] = 0.25 *", "gin[IDX4(n, iy, ix, c, H, W, C)] = 0.5 *"),
    ("maxpool backward picks the last maximum", "oracle.c", "if (in[j] > best) { best = in[j]; arg = j; }",
     "if (in[j] >= best) { best = in[j]; arg = j; }"),
    ("bf16 keeps 9 significant bits", "oracle.c", "r = ldexp(nearbyint(ldexp(f, 8)), e - 8);",
     "r = ldexp(nearbyint(ldexp(f, 9)), e - 9);"),
    ("split backward overwrites instead of accumulating", "compose.py",
     'G[..., :c_l] = rnd(G[..., :c_l] + b1["dx"])', 'G[..., :c_l] = rnd(b1["dx"])'),
    ("ReLU mask taken on the CONV input gradient", "compose.py",
     'dy = rnd(P.relu_bwd(dz, c["y"]))', 'dy = rnd(P.relu_bwd(dz, dz))'),
    ("wgrad on the un-normalised input", "compose.py", 'dw = P.conv_wgrad(c["z"], g, K)', 'dw = P.conv_wgrad(c["x"], g, K)'),
    ("transition backward skips the pooling gradient", "compose.py",
     'gt = rnd(P.avgpool2_bwd(dpool, ut["x"].shape[1:3]))', 'gt = rnd(np.repeat(np.repeat(dpool, 2, 1), 2, 2))'),
    ("residual gradient not added", "compose.py", 'dX = rnd(ds + P.conv_dgrad(', 'dX = rnd(0 * ds + P.conv_dgrad('),
    ("cross-entropy gradient not averaged over the batch", "prims.py", "return loss, p / N", "return loss, p"),
    ("FC bias dropped", "prims.py", "return _f64(f) @ _f64(wt) + _f64(bias)[None, :]", "return _f64(f) @ _f64(wt)"),
    ("global pooling gradient scaled by 1/H only", "prims.py", "(gout / (H * W))", "(gout / H)"),
    ("head ReLU mask taken on the BN input", "compose.py", 'dy5 = P.relu_bwd(dz5, hd["y"])',
     'dy5 = P.relu_bwd(dz5, hd["x"])'),
    ("stem weight gradient with the wrong padding", "compose.py",
     'd["stem"]["w"].shape[0], stride=2, pad=3)', 'd["stem"]["w"].shape[0], stride=2, pad=2)'),
    # the bf16 storage model's backward rounding sites (each dropped) and its
    # fp32 results (one rounded)
    ("bf16: masked BN output gradient dy not stored in bf16", "compose.py",
     'dy = rnd(P.relu_bwd(dz, c["y"]))', 'dy = P.relu_bwd(dz, c["y"])'),
    ("bf16: deferred dx of the 3x3 CONV's BN not rounded for the 1x1 backward", "compose.py",
     'b1 = unit_bwd(c["u1"], rnd(b2["dx"]), rnd)', 'b1 = unit_bwd(c["u1"], b2["dx"], rnd)'),
    ("bf16: Split accumulation into G not rounded", "compose.py",
     'G[..., :c_l] = rnd(G[..., :c_l] + b1["dx"])', 'G[..., :c_l] = G[..., :c_l] + b1["dx"]'),
    ("bf16: bottleneck upstream gradient not rounded", "compose.py",
     'G = rnd(np.array(dY, dtype=np.float64, copy=True))', 'G = np.array(dY, dtype=np.float64, copy=True)'),
    ("bf16: transition unpooled gradient not rounded", "compose.py",
     'gt = rnd(P.avgpool2_bwd(dpool, ut["x"].shape[1:3]))', 'gt = P.avgpool2_bwd(dpool, ut["x"].shape[1:3])'),
    ("bf16: block gradient G from the transition not rounded", "compose.py",
     'G = rnd(bt["dx"])', 'G = np.array(bt["dx"])'),
    ("bf16: residual masked gradient ds not rounded", "compose.py",
     'ds = rnd(P.relu_bwd(dr, c["s"]))', 'ds = P.relu_bwd(dr, c["s"])'),
    ("bf16: BN3 input gradient not rounded for the third CONV's backward", "compose.py",
     'b3 = unit_bwd(c["u3"], rnd(dx3), rnd)', 'b3 = unit_bwd(c["u3"], dx3, rnd)'),
    ("bf16: BN2 input gradient not rounded for the second CONV's backward", "compose.py",
     'b2 = unit_bwd(c["u2"], rnd(b3["dx"]), rnd)', 'b2 = unit_bwd(c["u2"], b3["dx"], rnd)'),
    ("bf16: BN1 input gradient not rounded for the first CONV's backward", "compose.py",
     'g1 = rnd(b2["dx"])', 'g1 = b2["dx"]'),
    ("bf16: residual block input gradient not rounded", "compose.py",
     'dX = rnd(ds + P.conv_dgrad(g1', 'dX = (ds + P.conv_dgrad(g1'),
    ("bf16: head BN input gradient not rounded", "compose.py", 'G = rnd(dx5)', 'G = np.array(dx5)'),
    ("bf16: stem masked gradient not rounded", "compose.py",
     'dy0 = rnd(P.relu_bwd(dz0, st["y"]))', 'dy0 = P.relu_bwd(dz0, st["y"])'),
    ("bf16: stem BN input gradient not rounded for the stem weight gradient", "compose.py",
     'g0 = rnd(dx0)', 'g0 = np.array(dx0)'),
    ("bf16: weight gradient rounded to bf16", "compose.py",
     'dw = P.conv_wgrad(c["z"], g, K)', 'dw = rnd(P.conv_wgrad(c["z"], g, K))'),
    ("pool-first transition: ReLU after the pooling", "compose.py",
     'zp = rnd(P.avgpool2_fwd(P.relu_fwd(y)))', 'zp = rnd(P.relu_fwd(P.avgpool2_fwd(y)))'),
    ("pool-first transition: pooled CONV operand not rounded", "compose.py",
     'zp = rnd(P.avgpool2_fwd(P.relu_fwd(y)))', 'zp = P.avgpool2_fwd(P.relu_fwd(y))'),
    ("bf16: BN reductions rounded to bf16", "compose.py",
     'dx, dgamma, dbeta = P.bn_bwd(c["x"], dy, c["gamma"], c["mean"], c["rstd"])',
     'dx, dgamma, dbeta = P.bn_bwd(c["x"], dy, c["gamma"], c["mean"], c["rstd"]); dgamma = rnd(dgamma)'),
]


def _run_mutant(tmp_root, idx, fname, old, new):
    d = os.path.join(tmp_root, "m%02d" % idx)
    shutil.copytree(os.path.join(ROOT, "oracle"), os.path.join(d, "oracle"),
                    ignore=shutil.ignore_patterns("*.so", "__pycache__"))
    os.makedirs(os.path.join(d, "tests"))
    shutil.copy(os.path.join(ROOT, "tests", "test_oracle_pins.py"), os.path.join(d, "tests"))
    shutil.copytree(os.path.join(ROOT, "tests", "golden"), os.path.join(d, "tests", "golden"))
    pkg = os.path.join(d, "paper_1807_01702_amd")        # the seeded input generator the pins draw from
    os.makedirs(pkg)
    for f in ("__init__.py", "synth.py"):
        shutil.copy(os.path.join(ROOT, "paper_1807_01702_amd", f), pkg)
    path = os.path.join(d, "oracle", fname)
    src = open(path).read()
    assert src.count(old) == 1, "mutation site not unique/found: %r" % old
    open(path, "w").write(src.replace(old, new))
    env = dict(os.environ, PYTHONPATH=d, OMP_NUM_THREADS="2")
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-p", "no:cacheprovider",
                        os.path.join(d, "tests", "test_oracle_pins.py")],
                       cwd=d, env=env, capture_output=True, text=True, timeout=600)
    return r.returncode, r.stdout[-400:]


def test_every_planted_mistake_is_caught(tmp_path):
    with ThreadPoolExecutor(max_workers=4) as ex:
        futs = [ex.submit(_run_mutant, str(tmp_path), i, f, o, n) for i, (_, f, o, n) in enumerate(MUTANTS)]
        results = [f.result() for f in futs]
    survivors = [MUTANTS[i][0] for i, (rc, _) in enumerate(results) if rc == 0]
    assert not survivors, "mutants not caught by any pin: %s" % survivors
    # a failure must be a test failure (exit 1), not a crash of the harness
    assert all(rc == 1 for rc, _ in results), [(MUTANTS[i][0], out) for i, (rc, out) in enumerate(results) if rc != 1]
