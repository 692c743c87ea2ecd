"""Pins of the oracle's two mask generalisations: the sliding window and the
per-block clean context of DFlash2 draft blocks.

Independent sources, as for the base mask: a loop brute force written from
the prose rules with math.fsum sums, the per-block formula of
eq. ``eq:dflash2-block-attention`` evaluated directly on stacked K/V, closed
forms (a one-position window, pair counts), finite differences of the
backward, and reductions to the base mask (no window, the table M * b).
"""
import math

import numpy as np
import pytest

import oracle
from oracle import CLEAN, CORRUPTED, CLEAN_INTRA_BLOCK, CLEAN_INTRA_CAUSAL

READINGS = [CLEAN_INTRA_CAUSAL, CLEAN_INTRA_BLOCK]


def rand(shape, seed):
    return np.random.default_rng(seed).standard_normal(shape)


def joint_inputs(L, Hq, Hkv, d, seed):
    return (rand((1, 2 * L, Hq, d), seed), rand((1, 2 * L, Hkv, d), seed + 1),
            rand((1, 2 * L, Hkv, d), seed + 2), rand((1, 2 * L, Hq, d), seed + 3))


def anchors(L, M, seed):
    """A non-decreasing table of draft-block anchors in [0, L] (one per block)."""
    a = np.sort(np.random.default_rng(seed).integers(0, L + 1, size=L // M))
    return [int(x) for x in a]


def brute_force(q, k, v, L, M, reading, scale, window, prefix):
    """Loops over the allowed key positions, written from the prose rules."""
    _, n, Hq, d = q.shape
    g = Hq // k.shape[2]
    rows = [(CORRUPTED, p) for p in range(L)] + [(CLEAN, p) for p in range(L)]
    index = {r: i for i, r in enumerate(rows)}
    O = np.zeros_like(q)
    LSE = np.full((1, Hq, n), -np.inf)
    for i, (s, p) in enumerate(rows):
        blk = p // M
        if s == CLEAN:
            end = p + 1 if reading == CLEAN_INTRA_CAUSAL else (blk + 1) * M
            allowed = []
        else:
            end = blk * M if prefix is None else prefix[blk]
            allowed = [(CORRUPTED, x) for x in range(blk * M, (blk + 1) * M)]
        start = max(0, end - window) if window else 0
        allowed += [(CLEAN, x) for x in range(start, end)]
        keys = [index[r] for r in allowed]
        if not keys:
            continue
        for h in range(Hq):
            kv = h // g
            a = [scale * math.fsum(q[0, i, h, t] * k[0, j, kv, t] for t in range(d)) for j in keys]
            mx = max(a)
            w = [math.exp(x - mx) for x in a]
            den = math.fsum(w)
            for t in range(d):
                O[0, i, h, t] = math.fsum(wj * v[0, j, kv, t] for wj, j in zip(w, keys)) / den
            LSE[0, h, i] = mx + math.log(den)
    return O, LSE


@pytest.mark.parametrize("L,M", [(8, 2), (12, 4), (12, 3)])
@pytest.mark.parametrize("window", [1, 3, 5])
@pytest.mark.parametrize("reading", READINGS)
@pytest.mark.parametrize("with_prefix", [False, True], ids=["blocks", "anchors"])
def test_forward_matches_brute_force(L, M, window, reading, with_prefix):
    d = 3
    q, k, v, _ = joint_inputs(L, 2, 1, d, seed=L * 7 + M + window)
    prefix = anchors(L, M, seed=L + M) if with_prefix else None
    O, LSE = oracle.joint_fwd(q, k, v, L, M, clean_intra=reading, window=window, clean_prefix=prefix)
    Ob, LSEb = brute_force(q, k, v, L, M, reading, 1 / math.sqrt(d), window, prefix)
    np.testing.assert_allclose(O, Ob, rtol=0, atol=1e-12)
    np.testing.assert_array_equal(np.isneginf(LSE), np.isneginf(LSEb))
    fin = np.isfinite(LSEb)
    np.testing.assert_allclose(LSE[fin], LSEb[fin], rtol=0, atol=1e-12)


@pytest.mark.parametrize("reading", READINGS)
def test_anchor_prefix_without_window_matches_brute_force(reading):
    L, M, d = 12, 3, 3
    q, k, v, _ = joint_inputs(L, 2, 2, d, seed=41)
    prefix = anchors(L, M, seed=9)
    O, LSE = oracle.joint_fwd(q, k, v, L, M, clean_intra=reading, clean_prefix=prefix)
    Ob, _ = brute_force(q, k, v, L, M, reading, 1 / math.sqrt(d), 0, prefix)
    np.testing.assert_allclose(O, Ob, rtol=0, atol=1e-12)


def test_wide_window_and_block_table_reduce_to_the_base_mask():
    L, M, d = 16, 4, 4
    q, k, v, do = joint_inputs(L, 4, 2, d, seed=5)
    base = oracle.joint_fwd(q, k, v, L, M)
    for kw in ({"window": 2 * L}, {"clean_prefix": [b * M for b in range(L // M)]}):
        got = oracle.joint_fwd(q, k, v, L, M, **kw)
        np.testing.assert_array_equal(got[0], base[0])
        np.testing.assert_array_equal(got[1], base[1])


def test_one_position_window_closed_form():
    """W = 1: a clean query sees only itself (O = V_q); a corrupted query of
    block b > 0 sees its own block and the single clean key M b - 1."""
    L, M, d = 12, 4, 5
    q, k, v, _ = joint_inputs(L, 1, 1, d, seed=6)
    O, LSE = oracle.joint_fwd(q, k, v, L, M, window=1)
    scale = 1 / math.sqrt(d)
    for p in range(L):
        i = L + p
        np.testing.assert_allclose(O[0, i, 0], v[0, i, 0], rtol=0, atol=1e-14)
        np.testing.assert_allclose(LSE[0, 0, i], scale * q[0, i, 0] @ k[0, i, 0], rtol=0, atol=1e-14)
    for p in range(M, L):
        b = p // M
        keys = list(range(b * M, (b + 1) * M)) + [L + b * M - 1]
        s = scale * k[0, keys, 0] @ q[0, p, 0]
        w = np.exp(s - s.max())
        np.testing.assert_allclose(O[0, p, 0], w @ v[0, keys, 0] / w.sum(), rtol=0, atol=1e-13)


def test_draft_blocks_match_the_per_block_formula():
    """eq:dflash2-block-attention: O_b = Attn(Q_b, [K_b; K^tar_{<a_b}], [V_b; V^tar_{<a_b}])
    for every draft block, with draft blocks as the corrupted stream and the
    target features as the clean stream; the target rows themselves have no
    query role here, only the draft rows are checked."""
    L, M, Hq, Hkv, d = 24, 4, 4, 2, 6
    q, k, v, do = joint_inputs(L, Hq, Hkv, d, seed=8)
    prefix = anchors(L, M, seed=3)
    O, LSE = oracle.joint_fwd(q, k, v, L, M, clean_prefix=prefix)
    scale = 1 / math.sqrt(d)
    g = Hq // Hkv
    for b in range(L // M):
        rows = slice(b * M, (b + 1) * M)
        Kb = np.concatenate([k[0, rows], k[0, L:L + prefix[b]]], axis=0)
        Vb = np.concatenate([v[0, rows], v[0, L:L + prefix[b]]], axis=0)
        for h in range(Hq):
            S = scale * q[0, rows, h] @ Kb[:, h // g].T
            P = np.exp(S - S.max(axis=1, keepdims=True))
            ref = (P @ Vb[:, h // g]) / P.sum(axis=1, keepdims=True)
            np.testing.assert_allclose(O[0, rows, h], ref, rtol=0, atol=1e-12)
    # Blocks are independent: dO of one draft block moves no other block's dQ
    # or own-block dK/dV.
    dQ, dK, dV = oracle.joint_bwd(q, k, v, O, LSE, do, L, M, clean_prefix=prefix)
    do2 = do.copy()
    do2[0, 2 * M:3 * M] += 1.0
    dQ2, dK2, dV2 = oracle.joint_bwd(q, k, v, O, LSE, do2, L, M, clean_prefix=prefix)
    other = np.r_[0:2 * M, 3 * M:L]
    np.testing.assert_array_equal(dQ2[0, other], dQ[0, other])
    np.testing.assert_array_equal(dK2[0, other], dK[0, other])
    np.testing.assert_array_equal(dV2[0, other], dV[0, other])


@pytest.mark.parametrize("reading", READINGS)
@pytest.mark.parametrize("with_prefix", [False, True], ids=["blocks", "anchors"])
def test_backward_matches_finite_differences(reading, with_prefix):
    L, M, d, window = 8, 2, 3, 3
    q, k, v, do = joint_inputs(L, 2, 1, d, seed=21)
    prefix = anchors(L, M, seed=2) if with_prefix else None
    kw = dict(clean_intra=reading, window=window, clean_prefix=prefix)

    def f(q_, k_, v_):
        O, _ = oracle.joint_fwd(q_, k_, v_, L, M, **kw)
        return float(np.sum(do * O))

    O, LSE = oracle.joint_fwd(q, k, v, L, M, **kw)
    dQ, dK, dV = oracle.joint_bwd(q, k, v, O, LSE, do, L, M, **kw)
    h = 1e-6
    for name, x, gr in (("q", q, dQ), ("k", k, dK), ("v", v, dV)):
        fd = np.zeros_like(x)
        for idx in np.ndindex(x.shape):
            xp = x.copy(); xp[idx] += h
            xm = x.copy(); xm[idx] -= h
            args_p = {"q": (xp, k, v), "k": (q, xp, v), "v": (q, k, xp)}[name]
            args_m = {"q": (xm, k, v), "k": (q, xm, v), "v": (q, k, xm)}[name]
            fd[idx] = (f(*args_p) - f(*args_m)) / (2 * h)
        err = np.max(np.abs(fd - gr)) / max(1.0, np.max(np.abs(gr)))
        assert err < 1e-7, (name, err)


def windowed_pairs_closed_form(L, M, W, reading):
    """Valid pairs per head of the joint layout with a window of W clean positions."""
    nb = L // M
    if reading == CLEAN_INTRA_CAUSAL:
        clean = sum(min(p + 1, W) for p in range(L))
    else:
        clean = sum(M * min((b + 1) * M, W) for b in range(nb))
    corrupted = L * M + sum(M * min(b * M, W) for b in range(nb))
    return clean + corrupted


@pytest.mark.parametrize("L,M,W", [(64, 8, 1), (64, 8, 20), (96, 16, 64), (40, 4, 1000)])
@pytest.mark.parametrize("reading", READINGS)
def test_windowed_pair_count_closed_form(L, M, W, reading):
    r = oracle.joint_ranges(L)
    assert oracle.count_visible_pairs(r, r, M, reading, window=W) == windowed_pairs_closed_form(L, M, W, reading)


def test_anchor_pair_count_closed_form():
    L, M = 64, 8
    prefix = anchors(L, M, seed=17)
    r = oracle.joint_ranges(L)
    want = L * (L + 1) // 2 + L * M + sum(M * a for a in prefix)
    assert oracle.count_visible_pairs(r, r, M, clean_prefix=prefix) == want
