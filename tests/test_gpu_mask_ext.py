"""GPU parity of the mask generalisations against the fp64 oracle: the sliding
window and the per-block clean context of DFlash2 draft blocks.

Cases: windows from one position to more than a tile (and wider than the
sequence), both clean-to-clean readings, GQA, head_dim 64 and 128, batch 2,
fp32 and bf16; anchor tables with repeated entries, zeros and L; the drafter
layout (draft queries only, over draft and target-feature keys); the two
complementary views of the AR-to-BDLM objective as batch elements; and
workload-sized cases (a 1,024-position window at 4K, a drafter with 256
draft blocks over 8,192 target features) on a subset of heads.
"""
import pytest
import torch

import oracle
import paper_2609_19242_amd as bd
import synth
from paper_2609_19242_amd import CLEAN, CORRUPTED, Range
from tests.gpu_util import assert_close, joint_inputs, kv_group_heads

pytestmark = pytest.mark.gpu
DEV = "cuda"


def sorted_anchors(nblk, L, seed, n_used=None):
    """Non-decreasing anchors in [0, L]; blocks past n_used (no draft rows) get L."""
    n_used = nblk if n_used is None else n_used
    g = torch.Generator().manual_seed(seed)
    a = torch.sort(torch.randint(0, L + 1, (n_used,), generator=g)).values
    a[0] = 0  # a block with no clean context at all
    if n_used > 3:
        a[2] = a[3]  # repeated anchors
    return torch.cat([a, torch.full((nblk - n_used,), L)]).to(torch.int32)


def check_joint_ext(q, k, v, do, M, reading, dtype, window=0, prefix=None, heads=None, tag="", hilo=0):
    L = q.shape[1] // 2
    qd, kd, vd, dod = (t.to(DEV) for t in (q, k, v, do))
    pref_d = prefix.to(DEV) if prefix is not None else None
    o, lse = bd.joint_fwd(qd, kd, vd, M, clean_intra=reading, out_f32=True, window=window, clean_prefix=pref_d,
                          hilo=hilo)
    dq, dk, dv = bd.joint_bwd(qd, kd, vd, o, lse, dod, M, clean_intra=reading, out_f32=True, window=window,
                              clean_prefix=pref_d, hilo=hilo)
    torch.cuda.synchronize()
    hs = list(range(q.shape[2])) if heads is None else heads
    pl = None if prefix is None else prefix.tolist()
    O, LSE = oracle.joint_fwd(q, k, v, L, M, clean_intra=reading, heads=hs, window=window, clean_prefix=pl)
    dQ, dK, dV = oracle.joint_bwd(q, k, v, O, LSE, do[:, :, hs], L, M, clean_intra=reading, heads=hs,
                                  window=window, clean_prefix=pl)
    kvs = sorted(set(h // (q.shape[2] // k.shape[2]) for h in hs))
    assert_close(f"{tag} LSE", lse[:, hs], LSE, dtype)
    for name, got, ref in (("O", o[:, :, hs], O), ("dQ", dq[:, :, hs], dQ), ("dK", dk[:, :, kvs], dK[:, :, kvs]),
                           ("dV", dv[:, :, kvs], dV[:, :, kvs])):
        assert_close(f"{tag} {name}", got, ref, dtype)
    # the library's pair counter agrees with the oracle's explicit mask
    p = bd.make_problem(q.shape[0], L, M, q.shape[2], k.shape[2], q.shape[3], dtype, clean_intra=reading,
                        window=window, clean_prefix=pref_d)
    r = bd.joint_ranges(L)
    assert bd.visible_pairs(p, r, r) == oracle.count_visible_pairs(oracle.joint_ranges(L), oracle.joint_ranges(L), M,
                                                                   reading, window=window, clean_prefix=pl)


WINDOW_CASES = [
    # L, M, Hq, Hkv, D, batch, window
    (300, 12, 4, 2, 128, 1, 1),
    (300, 12, 4, 2, 128, 1, 37),
    (320, 16, 2, 1, 64, 2, 100),
    (520, 40, 2, 1, 128, 1, 130),
    (256, 8, 4, 1, 128, 1, 600),
]


# bf16 with adaptive two-term P and dS products: the wave-level tile skip and
# the adaptive selection on the same partly visible window tiles
HILO_OF_DT = {"bf16-adaptive": bd.HILO_ALL | bd.HILO_ADAPTIVE}


@pytest.mark.parametrize("dt", ["bf16", "bf16-adaptive", "fp32"])
@pytest.mark.parametrize("reading", [0, 1], ids=["causal", "block"])
@pytest.mark.parametrize("case", WINDOW_CASES, ids=lambda c: "L{}-M{}-H{}x{}-d{}-b{}-W{}".format(*c))
def test_window_small(case, reading, dt):
    L, M, Hq, Hkv, D, B, W = case
    dtype = torch.float32 if dt == "fp32" else torch.bfloat16
    q, k, v, do = joint_inputs(L, Hq, Hkv, D, dtype, batch=B, seed=L + W)
    check_joint_ext(q, k, v, do, M, reading, dtype, window=W, tag=f"L{L} M{M} W{W} r{reading} {dt}",
                    hilo=HILO_OF_DT.get(dt, 0))


@pytest.mark.parametrize("dt", ["bf16", "fp32"])
@pytest.mark.parametrize("window", [0, 45])
def test_anchor_table_joint(window, dt):
    L, M, Hq, Hkv, D = 320, 16, 4, 2, 128
    dtype = torch.float32 if dt == "fp32" else torch.bfloat16
    q, k, v, do = joint_inputs(L, Hq, Hkv, D, dtype, seed=77 + window)
    prefix = sorted_anchors(L // M, L, seed=4)
    check_joint_ext(q, k, v, do, M, 0, dtype, window=window, prefix=prefix, tag=f"anchors W{window}")


def drafter_case(T, M, n_blocks, Hq, Hkv, D, dtype, seed, window=0):
    """Draft queries only: draft blocks (corrupted rows [0, n_blocks M)) over
    themselves and the target features (clean rows [0, T))."""
    nd = n_blocks * M
    q = synth.normal((1, nd, Hq, D), seed, dtype)
    kd_ = synth.normal((1, nd, Hkv, D), seed + 1, dtype)
    vd_ = synth.normal((1, nd, Hkv, D), seed + 2, dtype)
    kt = synth.normal((1, T, Hkv, D), seed + 3, dtype)
    vt = synth.normal((1, T, Hkv, D), seed + 4, dtype)
    do = synth.normal((1, nd, Hq, D), seed + 5, dtype)
    prefix = sorted_anchors(T // M, T, seed=seed, n_used=n_blocks)
    return q, kd_, vd_, kt, vt, do, prefix


def check_drafter(T, M, n_blocks, Hq, Hkv, D, dtype, seed, heads=None, window=0, hilo=0):
    q, kd_, vd_, kt, vt, do, prefix = drafter_case(T, M, n_blocks, Hq, Hkv, D, dtype, seed, window)
    nd = n_blocks * M
    pref_d = prefix.to(DEV)
    p = bd.make_problem(1, T, M, Hq, Hkv, D, dtype, out_f32=True, window=window, clean_prefix=pref_d, hilo=hilo)
    qr = [Range(CORRUPTED, 0, nd)]
    kr = [Range(CORRUPTED, 0, nd), Range(CLEAN, 0, T)]
    qg, dog = q.to(DEV), do.to(DEV)
    ks = [kd_.to(DEV), kt.to(DEV)]
    vs = [vd_.to(DEV), vt.to(DEV)]
    o = torch.empty(q.shape, dtype=torch.float32, device=DEV)
    lse = torch.empty((1, Hq, nd), dtype=torch.float32, device=DEV)
    bd.attn_fwd(p, qr, [qg], [o], [lse], kr, ks, vs)
    dq = torch.empty(q.shape, dtype=torch.float32, device=DEV)
    dks = [torch.empty(t.shape, dtype=torch.float32, device=DEV) for t in ks]
    dvs = [torch.empty(t.shape, dtype=torch.float32, device=DEV) for t in vs]
    ws = torch.empty(bd.attn_bwd_workspace_bytes(p, qr), dtype=torch.uint8, device=DEV)
    bd.attn_bwd(p, qr, [qg], [o], [lse], [dog], [dq], kr, ks, vs, dks, dvs, ws)
    torch.cuda.synchronize()
    hs = list(range(Hq)) if heads is None else heads
    kk = torch.cat([kd_, kt], dim=1)
    vv = torch.cat([vd_, vt], dim=1)
    oq = [(CORRUPTED, 0, nd)]
    ok = [(CORRUPTED, 0, nd), (CLEAN, 0, T)]
    pl = prefix.tolist()
    O, LSE = oracle.fwd(q, kk, vv, oq, ok, M, heads=hs, window=window, clean_prefix=pl)
    dQ, dK, dV = oracle.bwd(q, kk, vv, O, LSE, do[:, :, hs], oq, ok, M, heads=hs, window=window, clean_prefix=pl)
    kvs = sorted(set(h // (Hq // Hkv) for h in hs))
    tag = f"drafter T{T} M{M} nb{n_blocks} W{window}"
    assert_close(f"{tag} LSE", lse[:, hs], LSE, dtype)
    assert_close(f"{tag} O", o[:, :, hs], O, dtype)
    assert_close(f"{tag} dQ", dq[:, :, hs], dQ, dtype)
    for name, got, ref in (("dK draft", dks[0], dK[:, :nd]), ("dK target", dks[1], dK[:, nd:]),
                           ("dV draft", dvs[0], dV[:, :nd]), ("dV target", dvs[1], dV[:, nd:])):
        assert_close(f"{tag} {name}", got[:, :, kvs], ref[:, :, kvs], dtype)
    assert bd.visible_pairs(p, qr, kr) == oracle.count_visible_pairs(oq, ok, M, window=window, clean_prefix=pl)


@pytest.mark.parametrize("dt", ["bf16", "bf16-adaptive", "fp32"])
@pytest.mark.parametrize("window", [0, 70])
def test_drafter_small(window, dt):
    dtype = torch.float32 if dt == "fp32" else torch.bfloat16
    check_drafter(608, 16, 24, 4, 2, 128, dtype, seed=13, window=window, hilo=HILO_OF_DT.get(dt, 0))


def test_two_complementary_views_are_batch_elements():
    """AR-to-BDLM conversion (eq:fast-dllm-v2-attention): the two noisy views
    share the clean sequence and are separate batch elements; each view's
    result equals the single-view computation."""
    L, M, Hq, Hkv, D = 256, 16, 4, 2, 128
    q, k, v, do = joint_inputs(L, Hq, Hkv, D, torch.bfloat16, batch=2, seed=90)
    for t in (q, k, v):
        t[1, L:] = t[0, L:]  # identical clean halves, different corrupted halves
    qd, kd, vd, dod = (t.to(DEV) for t in (q, k, v, do))
    o2, lse2 = bd.joint_fwd(qd, kd, vd, M, out_f32=True)
    dq2, dk2, dv2 = bd.joint_bwd(qd, kd, vd, o2, lse2, dod, M, out_f32=True)
    for b in range(2):
        sl = slice(b, b + 1)
        o1, lse1 = bd.joint_fwd(qd[sl].contiguous(), kd[sl].contiguous(), vd[sl].contiguous(), M, out_f32=True)
        dq1, dk1, dv1 = bd.joint_bwd(qd[sl].contiguous(), kd[sl].contiguous(), vd[sl].contiguous(), o1, lse1,
                                     dod[sl].contiguous(), M, out_f32=True)
        torch.cuda.synchronize()
        for a, r in ((o2[sl], o1), (lse2[sl], lse1), (dq2[sl], dq1), (dk2[sl], dk1), (dv2[sl], dv1)):
            assert torch.equal(a, r)
    O, LSE = oracle.joint_fwd(q, k, v, L, M)
    assert_close("two views O", o2, O, torch.bfloat16)


def test_workload_4k_window_1024():
    """The 4K workload (batch 2, block 32, 32/8 heads, d 128) with the paper's
    1,024-position sliding window, query heads of KV groups {0, 7}."""
    w = synth.WORKLOADS["4k"]
    q, k, v, do = synth.make_joint(w)
    hs = kv_group_heads(w.heads, w.kv_heads, [0, w.kv_heads - 1])
    check_joint_ext(q, k, v, do, w.block_size, 0, torch.bfloat16, window=1024, heads=hs, tag="4k W1024")


def test_workload_drafter_8k():
    """A drafter layout: 256 draft blocks of 16 over 8,192 target features,
    32/8 heads, d 128, bf16; query heads of KV group 0."""
    check_drafter(8192, 16, 256, 32, 8, 128, torch.bfloat16, seed=31, heads=kv_group_heads(32, 8, [0]))
