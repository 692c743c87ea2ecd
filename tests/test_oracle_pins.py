"""Pins of the fp64 oracle to facts fixed by the paper and by mathematics.

None of these re-types the oracle's own formula: each check comes from an
independent source -- a hand-written mask fixture, a loop-based brute force
written from the prose rules, finite differences, PyTorch's SDPA in float64
on special cases, closed-form pair counts (App. B), or an invariant the paper
proves (per-block separability, exact LSE merge of partials, the clean-gradient
sum of eq. ``eq:correctness-clean-gradient``).
"""
import math
import os

import numpy as np
import pytest
import torch

import oracle
from oracle import CLEAN, CORRUPTED, CLEAN_INTRA_BLOCK, CLEAN_INTRA_CAUSAL

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
READINGS = [CLEAN_INTRA_CAUSAL, CLEAN_INTRA_BLOCK]


def rand(shape, seed):
    return np.random.default_rng(seed).standard_normal(shape)


def joint_inputs(L, Hq, Hkv, d, seed, batch=1):
    q = rand((batch, 2 * L, Hq, d), seed)
    k = rand((batch, 2 * L, Hkv, d), seed + 1)
    v = rand((batch, 2 * L, Hkv, d), seed + 2)
    do = rand((batch, 2 * L, Hq, d), seed + 3)
    return q, k, v, do


# ---------------------------------------------------------------- mask fixture
def read_mask_fixture():
    grids, cur = {}, None
    with open(os.path.join(GOLDEN, "mask_L4_M2.txt")) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            if line in ("causal", "block"):
                cur = line
                grids[cur] = []
            else:
                grids[cur].append([int(c) for c in line])
    return {k: np.array(v, dtype=bool) for k, v in grids.items()}


def test_mask_matches_hand_written_fixture():
    grids = read_mask_fixture()
    s, p = oracle.rows_of(oracle.joint_ranges(4))
    for name, reading in (("causal", CLEAN_INTRA_CAUSAL), ("block", CLEAN_INTRA_BLOCK)):
        got = oracle.visible(s, p, s, p, 2, reading)
        np.testing.assert_array_equal(got, grids[name])


# ------------------------------------------------------ closed-form pair counts
def read_pair_counts():
    rows = []
    with open(os.path.join(GOLDEN, "pair_counts.txt")) as f:
        for line in f:
            if line.startswith("#") or not line.strip():
                continue
            rows.append(line.split())
    return rows


@pytest.mark.parametrize("row", [r for r in read_pair_counts() if r[0] in ("joint", "tiny", "4k")],
                         ids=lambda r: "-".join(r[:4]))
def test_pair_count_closed_form(row):
    name, Lf, Mf, reading, pairs = row
    L = int(Lf.split("=")[1])
    M = int(Mf.split("=")[1])
    rd = CLEAN_INTRA_CAUSAL if reading == "causal" else CLEAN_INTRA_BLOCK
    r = oracle.joint_ranges(L)
    assert oracle.count_visible_pairs(r, r, M, rd) == int(pairs)


def test_pair_count_csbp_rank_scaled():
    # Same structure as the 256K CSBP rank's share, scaled down by 64x in length:
    # target blocks b0..b1 over a full clean prefix; sum_b (b+1) M^2.
    M, n_local, pos0, clean = 4, 64, 512, 1024
    qr = [(CORRUPTED, pos0, n_local)]
    kr = [(CORRUPTED, pos0, n_local)] + [(CLEAN, s * 64, 64) for s in range(clean // 64)]
    want = sum((b + 1) * M * M for b in range(pos0 // M, (pos0 + n_local) // M))
    assert oracle.count_visible_pairs(qr, kr, M) == want


# ---------------------------------------------------------------- brute force
def brute_force(q, k, v, L, M, reading, scale):
    """Loop implementation from the prose rules, with math.fsum sums."""
    Bn, n, Hq, d = q.shape
    Hkv = k.shape[2]
    g = Hq // Hkv
    rows = [(CORRUPTED, p) for p in range(L)] + [(CLEAN, p) for p in range(L)]
    O = np.zeros_like(q)
    LSE = np.zeros((Bn, Hq, n))
    for i, (s, p) in enumerate(rows):
        blk = p // M
        if s == CLEAN:
            hi = p + 1 if reading == CLEAN_INTRA_CAUSAL else (blk + 1) * M
            allowed = {(CLEAN, x) for x in range(0, hi)}
        else:
            allowed = {(CORRUPTED, x) for x in range(blk * M, (blk + 1) * M)}
            allowed |= {(CLEAN, x) for x in range(0, blk * M)}
        keys = [j for j, r in enumerate(rows) if r in allowed]
        for b in range(Bn):
            for h in range(Hq):
                kv = h // g
                a = [scale * math.fsum(q[b, i, h, t] * k[b, j, kv, t] for t in range(d)) for j in keys]
                mx = max(a)
                w = [math.exp(x - mx) for x in a]
                den = math.fsum(w)
                for t in range(d):
                    O[b, i, h, t] = math.fsum(wj * v[b, j, kv, t] for wj, j in zip(w, keys)) / den
                LSE[b, h, i] = mx + math.log(den)
    return O, LSE


@pytest.mark.parametrize("L,M", [(4, 1), (4, 2), (4, 4), (8, 2), (8, 8), (12, 4)])
@pytest.mark.parametrize("heads", [(1, 1), (2, 1), (4, 2)])
@pytest.mark.parametrize("reading", READINGS)
def test_forward_matches_brute_force(L, M, heads, reading):
    Hq, Hkv = heads
    d = 4 if L == 8 else 2
    q, k, v, _ = joint_inputs(L, Hq, Hkv, d, seed=L * 100 + M * 10 + Hq)
    scale = 1.0 / math.sqrt(d)
    O, LSE = oracle.joint_fwd(q, k, v, L, M, clean_intra=reading)
    Ob, LSEb = brute_force(q, k, v, L, M, reading, scale)
    np.testing.assert_allclose(O, Ob, rtol=0, atol=1e-12)
    np.testing.assert_allclose(LSE, LSEb, rtol=0, atol=1e-12)


# ---------------------------------------------------------- finite differences
@pytest.mark.parametrize("reading", READINGS)
@pytest.mark.parametrize("L,M,heads", [(4, 2, (2, 1)), (6, 3, (2, 2)), (8, 2, (4, 2))])
def test_backward_matches_finite_differences(reading, L, M, heads):
    Hq, Hkv = heads
    d = 3
    q, k, v, do = joint_inputs(L, Hq, Hkv, d, seed=7 + L)

    def f(q_, k_, v_):
        O, _ = oracle.joint_fwd(q_, k_, v_, L, M, clean_intra=reading)
        return float(np.sum(do * O))

    O, LSE = oracle.joint_fwd(q, k, v, L, M, clean_intra=reading)
    dQ, dK, dV = oracle.joint_bwd(q, k, v, O, LSE, do, L, M, clean_intra=reading)
    h = 1e-6
    for name, x, g in (("q", q, dQ), ("k", k, dK), ("v", v, dV)):
        fd = np.zeros_like(x)
        for idx in np.ndindex(x.shape):
            xp = x.copy(); xp[idx] += h
            xm = x.copy(); xm[idx] -= h
            args_p = {"q": (xp, k, v), "k": (q, xp, v), "v": (q, k, xp)}[name]
            args_m = {"q": (xm, k, v), "k": (q, xm, v), "v": (q, k, xm)}[name]
            fd[idx] = (f(*args_p) - f(*args_m)) / (2 * h)
        err = np.max(np.abs(fd - g)) / max(1.0, np.max(np.abs(g)))
        assert err < 1e-7, (name, err)


# ------------------------------------------------- special cases against SDPA
def sdpa64(q, k, v, causal):
    """torch SDPA in float64 on the CPU, one sequence, GQA expanded by repeat."""
    Hq, Hkv = q.shape[1], k.shape[1]
    g = Hq // Hkv
    qt = torch.from_numpy(q).permute(1, 0, 2)[None]
    kt = torch.from_numpy(np.repeat(k, g, axis=1)).permute(1, 0, 2)[None]
    vt = torch.from_numpy(np.repeat(v, g, axis=1)).permute(1, 0, 2)[None]
    o = torch.nn.functional.scaled_dot_product_attention(qt, kt, vt, is_causal=causal)
    return o[0].permute(1, 0, 2).numpy()


@pytest.mark.parametrize("reading", READINGS)
def test_block_equals_length_is_bidirectional_over_corrupted(reading):
    # M = L: one block, no clean prefix for the corrupted copy (the b = 1 case of App. A).
    L, Hq, Hkv, d = 16, 4, 2, 8
    q, k, v, do = joint_inputs(L, Hq, Hkv, d, seed=3)
    O, LSE = oracle.joint_fwd(q, k, v, L, L, clean_intra=reading)
    ref = sdpa64(q[0, :L], k[0, :L], v[0, :L], causal=False)
    np.testing.assert_allclose(O[0, :L], ref, rtol=0, atol=1e-12)
    # gradients from the corrupted rows never reach the clean keys
    do_c = do.copy()
    do_c[:, L:] = 0.0
    _, dK, dV = oracle.joint_bwd(q, k, v, O, LSE, do_c, L, L, clean_intra=reading)
    assert np.all(dK[:, L:] == 0.0) and np.all(dV[:, L:] == 0.0)


@pytest.mark.parametrize("reading", READINGS)
def test_block_size_one_clean_rows_are_causal(reading):
    L, Hq, Hkv, d = 16, 4, 2, 8
    q, k, v, _ = joint_inputs(L, Hq, Hkv, d, seed=4)
    O, _ = oracle.joint_fwd(q, k, v, L, 1, clean_intra=reading)
    ref = sdpa64(q[0, L:], k[0, L:], v[0, L:], causal=True)
    np.testing.assert_allclose(O[0, L:], ref, rtol=0, atol=1e-12)


def test_clean_rows_under_block_reading_match_explicit_block_causal_sdpa():
    # block reading: clean query sees clean keys of blocks <= its own.  Checked
    # against SDPA with a block-lower-triangular boolean mask built by kron.
    L, M, Hq, d = 16, 4, 2, 8
    q, k, v, _ = joint_inputs(L, Hq, Hq, d, seed=5)
    O, _ = oracle.joint_fwd(q, k, v, L, M, clean_intra=CLEAN_INTRA_BLOCK)
    blockmask = torch.from_numpy(np.kron(np.tril(np.ones((L // M, L // M))), np.ones((M, M))).astype(bool))
    qt = torch.from_numpy(q[0, L:]).permute(1, 0, 2)[None]
    kt = torch.from_numpy(k[0, L:]).permute(1, 0, 2)[None]
    vt = torch.from_numpy(v[0, L:]).permute(1, 0, 2)[None]
    ref = torch.nn.functional.scaled_dot_product_attention(qt, kt, vt, attn_mask=blockmask)[0].permute(1, 0, 2).numpy()
    np.testing.assert_allclose(O[0, L:], ref, rtol=0, atol=1e-12)


# ---------------------------------------------------- per-block separability
@pytest.mark.parametrize("reading", READINGS)
def test_per_block_attention_equals_joint(reading):
    """eq. eq:csbp-block-attention: each target block alone = the joint corrupted rows."""
    L, M, Hq, Hkv, d = 24, 4, 4, 2, 6
    q, k, v, _ = joint_inputs(L, Hq, Hkv, d, seed=11)
    O, LSE = oracle.joint_fwd(q, k, v, L, M, clean_intra=reading)
    for b in range(L // M):
        rows = slice(b * M, (b + 1) * M)
        kk = np.concatenate([k[:, rows], k[:, L:L + b * M]], axis=1)
        vv = np.concatenate([v[:, rows], v[:, L:L + b * M]], axis=1)
        ob, lb = oracle.fwd(q[:, rows], kk, vv, [(CORRUPTED, b * M, M)],
                            [(CORRUPTED, b * M, M), (CLEAN, 0, b * M)], M, clean_intra=reading)
        np.testing.assert_allclose(ob, O[:, rows], rtol=0, atol=1e-13)
        np.testing.assert_allclose(lb, LSE[:, :, rows], rtol=0, atol=1e-13)


def test_block_gradients_do_not_depend_on_other_blocks():
    """eq. eq:correctness-block-dependency: dO of block b' != b leaves block b's corrupted grads unchanged."""
    L, M, Hq, Hkv, d = 16, 4, 2, 1, 4
    q, k, v, do = joint_inputs(L, Hq, Hkv, d, seed=12)
    O, LSE = oracle.joint_fwd(q, k, v, L, M)
    dQ, dK, dV = oracle.joint_bwd(q, k, v, O, LSE, do, L, M)
    do2 = do.copy()
    do2[:, 2 * M:3 * M] += rand(do2[:, 2 * M:3 * M].shape, 99)  # perturb corrupted block 2 only
    dQ2, dK2, dV2 = oracle.joint_bwd(q, k, v, O, LSE, do2, L, M)
    for b in (0, 1, 3):
        r = slice(b * M, (b + 1) * M)
        assert np.array_equal(dQ[:, r], dQ2[:, r])
        assert np.array_equal(dK[:, r], dK2[:, r])
        assert np.array_equal(dV[:, r], dV2[:, r])
    assert not np.allclose(dK[:, 2 * M:3 * M], dK2[:, 2 * M:3 * M])


@pytest.mark.parametrize("reading", READINGS)
def test_clean_gradient_is_sum_over_blocks_and_clean_queries(reading):
    """eq. eq:correctness-clean-gradient: clean dK/dV = sum over every query row's contribution."""
    L, M, Hq, Hkv, d = 16, 4, 4, 2, 5
    q, k, v, do = joint_inputs(L, Hq, Hkv, d, seed=13)
    O, LSE = oracle.joint_fwd(q, k, v, L, M, clean_intra=reading)
    _, dK, dV = oracle.joint_bwd(q, k, v, O, LSE, do, L, M, clean_intra=reading)
    acc_k = np.zeros_like(k[:, L:])
    acc_v = np.zeros_like(v[:, L:])
    # the clean queries over the clean keys
    _, ck, cv = oracle.bwd(q[:, L:], k[:, L:], v[:, L:], O[:, L:], LSE[:, :, L:], do[:, L:],
                           [(CLEAN, 0, L)], [(CLEAN, 0, L)], M, clean_intra=reading)
    acc_k += ck
    acc_v += cv
    # each target block separately over [own block ; full clean sequence]
    for b in range(L // M):
        r = slice(b * M, (b + 1) * M)
        kk = np.concatenate([k[:, r], k[:, L:]], axis=1)
        vv = np.concatenate([v[:, r], v[:, L:]], axis=1)
        _, bk, bv = oracle.bwd(q[:, r], kk, vv, O[:, r], LSE[:, :, r], do[:, r], [(CORRUPTED, b * M, M)],
                               [(CORRUPTED, b * M, M), (CLEAN, 0, L)], M, clean_intra=reading)
        np.testing.assert_allclose(bk[:, :M], dK[:, r], rtol=0, atol=1e-13)
        acc_k += bk[:, M:]
        acc_v += bv[:, M:]
    np.testing.assert_allclose(acc_k, dK[:, L:], rtol=0, atol=1e-12)
    np.testing.assert_allclose(acc_v, dV[:, L:], rtol=0, atol=1e-12)


# ------------------------------------------------------------------ LSE merge
def random_split(ranges, n_parts, rng):
    """Cut each range at random points and deal the pieces to n_parts parts (some parts may be empty)."""
    parts = [[] for _ in range(n_parts)]
    offset = 0
    for stream, pos0, n in ranges:
        cuts = sorted(rng.choice(np.arange(1, n), size=min(n - 1, 3), replace=False).tolist())
        bounds = [0] + cuts + [n]
        for a, b in zip(bounds[:-1], bounds[1:]):
            parts[int(rng.integers(n_parts - 1))].append((stream, pos0 + a, b - a, offset + a))
        offset += n
    return parts  # the last part is always empty


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_merge_of_partials_equals_unsplit(seed):
    """eq. eq:correctness-online-softmax-merge and eq. eq:csbp-lse-merge."""
    L, M, Hq, Hkv, d = 16, 4, 4, 2, 6
    rng = np.random.default_rng(seed)
    q, k, v, _ = joint_inputs(L, Hq, Hkv, d, seed=20 + seed, batch=2)
    r = oracle.joint_ranges(L)
    O, LSE = oracle.joint_fwd(q, k, v, L, M)
    o_parts, l_parts = [], []
    for part in random_split(r, 4, rng):
        rows = [x[3] + i for x in part for i in range(x[2])]
        o, l = oracle.fwd(q, k[:, rows], v[:, rows], r, [(s, p, n) for s, p, n, _ in part], M)
        o_parts.append(o)
        l_parts.append(l)
    assert np.all(np.isneginf(l_parts[-1])) and np.all(o_parts[-1] == 0.0)
    Om, Lm = oracle.lse_merge(o_parts, l_parts)
    np.testing.assert_allclose(Om, O, rtol=0, atol=1e-13)
    np.testing.assert_allclose(Lm, LSE, rtol=0, atol=1e-13)


def test_merge_of_all_empty_rows():
    o = [np.zeros((1, 3, 2, 4)), np.zeros((1, 3, 2, 4))]
    l = [np.full((1, 2, 3), -np.inf), np.full((1, 2, 3), -np.inf)]
    Om, Lm = oracle.lse_merge(o, l)
    assert np.all(Om == 0.0) and np.all(np.isneginf(Lm))


def test_merge_pairwise_formula_two_parts():
    """Two parts, written as the paper's pairwise rule on scalars."""
    z1, z2 = 1.5, -0.25
    o1, o2 = np.array([[[[1.0, 2.0]]]]), np.array([[[[-3.0, 0.5]]]])
    Om, Lm = oracle.lse_merge([o1, o2], [np.array([[[z1]]]), np.array([[[z2]]])])
    m = max(z1, z2)
    w1, w2 = math.exp(z1 - m), math.exp(z2 - m)
    np.testing.assert_allclose(Om[0, 0, 0], (w1 * o1[0, 0, 0] + w2 * o2[0, 0, 0]) / (w1 + w2), rtol=1e-15)
    assert abs(Lm[0, 0, 0] - (m + math.log(w1 + w2))) < 1e-15


# ------------------------------------------------------------------------ GQA
def test_gqa_reduces_to_mha():
    L, M, Hq, Hkv, d = 8, 2, 4, 2, 4
    q, k, v, do = joint_inputs(L, Hq, Hkv, d, seed=30)
    g = Hq // Hkv
    O, LSE = oracle.joint_fwd(q, k, v, L, M)
    kr, vr = np.repeat(k, g, axis=2), np.repeat(v, g, axis=2)
    O2, LSE2 = oracle.joint_fwd(q, kr, vr, L, M)
    np.testing.assert_allclose(O, O2, rtol=0, atol=1e-14)
    _, dK, dV = oracle.joint_bwd(q, k, v, O, LSE, do, L, M)
    _, dK2, dV2 = oracle.joint_bwd(q, kr, vr, O2, LSE2, do, L, M)
    np.testing.assert_allclose(dK, dK2.reshape(1, 2 * L, Hkv, g, d).sum(3), rtol=0, atol=1e-13)
    np.testing.assert_allclose(dV, dV2.reshape(1, 2 * L, Hkv, g, d).sum(3), rtol=0, atol=1e-13)


# ------------------------------------------------------------ row-level sanity
def test_row_bounds_and_convex_hull():
    L, M, Hq, Hkv, d = 16, 4, 2, 2, 4
    q, k, v, _ = joint_inputs(L, Hq, Hkv, d, seed=40)
    O, LSE = oracle.joint_fwd(q, k, v, L, M)
    s, p = oracle.rows_of(oracle.joint_ranges(L))
    mask = oracle.visible(s, p, s, p, M)
    for h in range(Hq):
        S = (q[0, :, h] @ k[0, :, h].T) / math.sqrt(d)
        for i in range(2 * L):
            vis = np.nonzero(mask[i])[0]
            mx = S[i, vis].max()
            assert mx - 1e-12 <= LSE[0, h, i] <= mx + math.log(len(vis)) + 1e-12
            vv = v[0, vis, h]
            assert np.all(O[0, i, h] >= vv.min(0) - 1e-12) and np.all(O[0, i, h] <= vv.max(0) + 1e-12)


def test_permuting_keys_inside_a_corrupted_block():
    L, M, Hq, Hkv, d = 16, 4, 2, 1, 4
    q, k, v, do = joint_inputs(L, Hq, Hkv, d, seed=41)
    O, LSE = oracle.joint_fwd(q, k, v, L, M)
    perm = np.arange(2 * L)
    perm[4:8] = [6, 4, 7, 5]  # corrupted block 1
    k2, v2 = k[:, perm], v[:, perm]
    O2, LSE2 = oracle.joint_fwd(q, k2, v2, L, M)
    np.testing.assert_allclose(O2, O, rtol=0, atol=1e-13)
    _, dK, dV = oracle.joint_bwd(q, k, v, O, LSE, do, L, M)
    _, dK2, dV2 = oracle.joint_bwd(q, k2, v2, O2, LSE2, do, L, M)
    np.testing.assert_allclose(dK2, dK[:, perm], rtol=0, atol=1e-13)
    np.testing.assert_allclose(dV2, dV[:, perm], rtol=0, atol=1e-13)


def test_empty_partial_rows():
    """A corrupted query of block 0 sees no clean key: its clean partial is O = 0, LSE = -inf."""
    L, M, Hq, d = 8, 4, 2, 4
    q, k, v, _ = joint_inputs(L, Hq, Hq, d, seed=42)
    o, l = oracle.fwd(q[:, :L], k[:, L:], v[:, L:], [(CORRUPTED, 0, L)], [(CLEAN, 0, L)], M)
    assert np.all(o[:, :M] == 0.0) and np.all(np.isneginf(l[:, :, :M]))
    assert np.all(np.isfinite(l[:, :, M:]))


# ----------------------------------------------------------- CSBP backward
def test_per_range_backward_with_merged_stats_equals_unsplit():
    """App. C fused backward: bwd over [local block ; clean shards] with the merged (O, LSE)."""
    M, n_local, pos0, shard, n_shards, Hq, Hkv, d = 4, 16, 32, 16, 4, 4, 2, 5
    q = rand((1, n_local, Hq, d), 50)
    kl, vl = rand((1, n_local, Hkv, d), 51), rand((1, n_local, Hkv, d), 52)
    kc, vc = rand((1, shard * n_shards, Hkv, d), 53), rand((1, shard * n_shards, Hkv, d), 54)
    do = rand((1, n_local, Hq, d), 55)
    qr = [(CORRUPTED, pos0, n_local)]
    kranges = [(CORRUPTED, pos0, n_local)] + [(CLEAN, s * shard, shard) for s in range(n_shards)]
    kall = np.concatenate([kl, kc], axis=1)
    vall = np.concatenate([vl, vc], axis=1)
    O, LSE = oracle.fwd(q, kall, vall, qr, kranges, M)
    # per-range partials then merge
    o_parts, l_parts = [], []
    for j, (s, p, n) in enumerate(kranges):
        off = 0 if j == 0 else n_local + (j - 1) * shard
        o, l = oracle.fwd(q, kall[:, off:off + n], vall[:, off:off + n], qr, [(s, p, n)], M)
        o_parts.append(o)
        l_parts.append(l)
    Om, Lm = oracle.lse_merge(o_parts, l_parts)
    np.testing.assert_allclose(Om, O, rtol=0, atol=1e-13)
    dQ, dK, dV = oracle.bwd(q, kall, vall, Om, Lm, do, qr, kranges, M)
    dQs = np.zeros_like(dQ)
    for j, (s, p, n) in enumerate(kranges):
        off = 0 if j == 0 else n_local + (j - 1) * shard
        dq, dk, dv = oracle.bwd(q, kall[:, off:off + n], vall[:, off:off + n], Om, Lm, do, qr, [(s, p, n)], M)
        dQs += dq
        np.testing.assert_allclose(dk, dK[:, off:off + n], rtol=0, atol=1e-13)
        np.testing.assert_allclose(dv, dV[:, off:off + n], rtol=0, atol=1e-13)
    np.testing.assert_allclose(dQs, dQ, rtol=0, atol=1e-13)


# ------------------------------------------------ head and row subsets of the oracle
# The full-size GPU tests call the oracle on a subset of query heads and rows.
# Pinned here against the full call by two facts that do not re-type the
# oracle: heads and query rows are independent in the forward, and in the
# backward a query row whose upstream gradient dO is zero contributes nothing
# to dK or dV (its dP and D vanish, so dS = 0 and P^T dO = 0).
@pytest.mark.parametrize("reading", READINGS)
def test_subset_heads_and_rows_equal_slices_of_the_full_call(reading):
    L, M, Hq, Hkv, d = 24, 4, 4, 2, 8
    q, k, v, do = joint_inputs(L, Hq, Hkv, d, seed=71, batch=2)
    r = oracle.joint_ranges(L)
    s_all, p_all = oracle.rows_of(r)
    O, LSE = oracle.fwd(q, k, v, r, r, M, clean_intra=reading)
    dQ, dK, dV = oracle.bwd(q, k, v, O, LSE, do, r, r, M, clean_intra=reading)

    # forward: q_rows and heads select rows and heads of the full result
    rows = np.array([0, 3, 5, L - 1, L, L + 7, 2 * L - 1])
    hs = [1, 2]
    Os, Ls = oracle.fwd(q, k, v, r, r, M, clean_intra=reading, heads=hs, q_rows=rows)
    np.testing.assert_allclose(Os, O[:, rows][:, :, hs], rtol=0, atol=1e-13)
    np.testing.assert_allclose(Ls, LSE[:, hs][:, :, rows], rtol=0, atol=1e-13)
    # the same rows passed as single-row ranges (the form the full-size GPU tests use)
    single = [(int(s_all[i]), int(p_all[i]), 1) for i in rows]
    Os2, Ls2 = oracle.fwd(q[:, rows], k, v, single, r, M, clean_intra=reading, heads=hs)
    np.testing.assert_allclose(Os2, Os, rtol=0, atol=1e-13)
    np.testing.assert_allclose(Ls2, Ls, rtol=0, atol=1e-13)

    # backward over one complete GQA group (KV head 1 = query heads 2, 3): its dQ
    # rows and the group's whole dK/dV
    grp = [2, 3]
    dQg, dKg, dVg = oracle.bwd(q, k, v, O[:, :, grp], LSE[:, grp], do[:, :, grp], r, r, M, clean_intra=reading,
                               heads=grp)
    np.testing.assert_allclose(dQg, dQ[:, :, grp], rtol=0, atol=1e-12)
    np.testing.assert_allclose(dKg[:, :, 1], dK[:, :, 1], rtol=0, atol=1e-12)
    np.testing.assert_allclose(dVg[:, :, 1], dV[:, :, 1], rtol=0, atol=1e-12)
    assert not dKg[:, :, 0].any() and not dVg[:, :, 0].any()

    # one head of a group: dK/dV equal the full call with dO zero on every other head
    do1 = np.zeros_like(do)
    do1[:, :, 2] = do[:, :, 2]
    _, dK1, dV1 = oracle.bwd(q, k, v, O, LSE, do1, r, r, M, clean_intra=reading)
    _, dKh, dVh = oracle.bwd(q, k, v, O[:, :, [2]], LSE[:, [2]], do[:, :, [2]], r, r, M, clean_intra=reading,
                             heads=[2])
    np.testing.assert_allclose(dKh, dK1, rtol=0, atol=1e-12)
    np.testing.assert_allclose(dVh, dV1, rtol=0, atol=1e-12)

    # a subset of query rows as single-row ranges: their dQ rows, and dK/dV equal
    # the full call with dO zero on every other row
    dQs, dKs, dVs = oracle.bwd(q[:, rows], k, v, O[:, rows], LSE[:, :, rows], do[:, rows], single, r, M,
                               clean_intra=reading)
    np.testing.assert_allclose(dQs, dQ[:, rows], rtol=0, atol=1e-12)
    dor = np.zeros_like(do)
    dor[:, rows] = do[:, rows]
    _, dKr, dVr = oracle.bwd(q, k, v, O, LSE, dor, r, r, M, clean_intra=reading)
    np.testing.assert_allclose(dKs, dKr, rtol=0, atol=1e-12)
    np.testing.assert_allclose(dVs, dVr, rtol=0, atol=1e-12)
