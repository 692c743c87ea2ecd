"""Shared helpers of the GPU parity tests: tolerances, comparisons, inputs."""
import math

import numpy as np
import torch

import synth

# Tolerances: bf16 inputs with fp32 accumulation -> max-abs <= 2e-2 and
# relative L2 <= 5e-3; the fp32 path -> 1e-5 for both.
TOL = {torch.bfloat16: (2e-2, 5e-3), torch.float32: (1e-5, 1e-5)}


def metrics(got, ref):
    g = got.detach().double().cpu().numpy() if hasattr(got, "detach") else np.asarray(got, np.float64)
    r = np.asarray(ref, np.float64)
    assert g.shape == r.shape, (g.shape, r.shape)
    gi, ri = np.isneginf(g), np.isneginf(r)
    assert np.array_equal(gi, ri), f"-inf pattern differs at {np.argwhere(gi != ri)[:5].tolist()}"
    g = np.where(gi, 0.0, g)
    r = np.where(ri, 0.0, r)
    assert np.all(np.isfinite(g)), "non-finite values"
    d = g - r
    max_abs = float(np.max(np.abs(d))) if d.size else 0.0
    nr = float(np.linalg.norm(r))
    rel = float(np.linalg.norm(d)) / nr if nr > 0 else float(np.linalg.norm(d))
    return max_abs, rel


def assert_close(name, got, ref, dtype, log=None):
    ma, rl = metrics(got, ref)
    tol_abs, tol_rel = TOL[dtype]
    line = f"{name}: max_abs={ma:.3e} rel_l2={rl:.3e} (tol {tol_abs:g}/{tol_rel:g})"
    print(line, flush=True)
    if log is not None:
        log.append(line)
    assert ma <= tol_abs and rl <= tol_rel, line


def assert_close_bf16_out(name, got, ref, log=None):
    """bf16-rounded outputs: the tolerance plus the output rounding (half a bf16 ulp <= 2^-8 |x|).

    Rounding a correct fp32 result to bf16 moves it by up to 2^-8 of its
    magnitude, which for |x| >= 8 alone exceeds 2e-2; the fp32-output tests
    carry the strict bar, this one bounds error = accumulation + output rounding.
    """
    g = got.detach().double().cpu().numpy()
    r = np.asarray(ref, np.float64)
    gi, ri = np.isneginf(g), np.isneginf(r)
    assert np.array_equal(gi, ri)
    g = np.where(gi, 0.0, g)
    r = np.where(ri, 0.0, r)
    d = np.abs(g - r)
    excess = float(np.max(d - 2.0 ** -8 * np.abs(r))) if d.size else 0.0
    rel = float(np.linalg.norm(g - r) / max(np.linalg.norm(r), 1e-300))
    line = f"{name} (bf16 out): max(|err| - 2^-8|ref|)={excess:.3e} rel_l2={rel:.3e} (tol 2e-2/5e-3)"
    print(line, flush=True)
    if log is not None:
        log.append(line)
    assert excess <= 2e-2 and rel <= 5e-3, line


def joint_inputs(L, Hq, Hkv, D, dtype, batch=1, seed=0):
    n = 2 * L
    q = synth.normal((batch, n, Hq, D), seed, dtype)
    k = synth.normal((batch, n, Hkv, D), seed + 1, dtype)
    v = synth.normal((batch, n, Hkv, D), seed + 2, dtype)
    do = synth.normal((batch, n, Hq, D), seed + 3, dtype)
    return q, k, v, do


def kv_group_heads(Hq, Hkv, groups):
    g = Hq // Hkv
    return [kv * g + i for kv in groups for i in range(g)]


def default_scale(D):
    return 1.0 / math.sqrt(D)
