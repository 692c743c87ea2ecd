"""GPU parity at the full workload sizes (32K joint, one 256K CSBP rank, 128K joint, and the
32K sliding-window and drafter legs of the mask generalisations).

The GPU computes every head and row in the launch configuration bench.py
times.  The fp64 oracle checks, on the query heads of KV groups {0, last}:

* sampled query rows (block edges of both streams and seeded random rows):
  O, LSE and dQ -- each needs only its own row's keys;
* every key row whose visible queries are few enough to enumerate: the
  corrupted keys of sampled blocks (seen only by their own block's queries,
  eq:correctness-block-dependency) and the clean keys of the last two blocks:
  dK and dV complete;
* for all keys of every KV head, the identity sum_j dV_j = sum_i dO_i over the
  group's heads (softmax rows sum to one), which catches any lost or doubled
  key tile at any size.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2609_19242_amd as bd
import synth
from paper_2609_19242_amd import CLEAN, CORRUPTED, Range
from synth import WORKLOADS
from tests.gpu_util import assert_close, assert_close_bf16_out, kv_group_heads

pytestmark = pytest.mark.gpu
DEV = "cuda"
F32 = torch.float32
BF16 = torch.bfloat16  # tolerance class of these runs: bf16 inputs, fp32 accumulation, fp32 outputs


def sample_rows(L, M, n_random, seed):
    corr = [0, M - 1, M, L // 2, L - M, L - 1]
    clean = [L + x for x in (0, 1, M - 1, M, L // 2, L - 1)]
    rng = np.random.default_rng(seed)
    rnd = rng.choice(2 * L, size=n_random, replace=False).tolist()
    return sorted(set(corr + clean + rnd))


def to_cpu_heads(t, heads):
    return t[:, :, heads].cpu()


def dv_identity(dv, do, group, tag):
    """sum over all key rows of dV equals sum over all query rows of dO (per batch, KV head)."""
    B, _, Hkv, D = dv.shape
    lhs = dv.double().sum(dim=1)  # [B][Hkv][D]
    rhs = do.double().sum(dim=1).reshape(B, Hkv, group, D).sum(dim=2)
    err = float((lhs - rhs).norm() / rhs.norm())
    print(f"{tag} sum dV identity rel_l2={err:.3e}", flush=True)
    assert err < 5e-3, err


def joint_check(w, reading=0, n_random=24, hilo=False, window=0, outs=("f32",), hilos=None):
    """The workload's fused fwd+bwd against the oracle on sampled rows and enumerable key sets.

    ``outs``: output modes to run, each against the same oracle values: "f32"
    (the fp32 accumulators, strict tolerance) and "bf16" (outputs rounded to
    bf16 as bench.py times them: the backward then reads the rounded O, and the
    bound adds the output rounding).  ``hilos``: the two-term settings to run in
    each output mode (default: ``hilo`` alone).
    """
    L, M = w.L, w.block_size
    torch.cuda.empty_cache()
    q, k, v, do = synth.make_joint(w, device=DEV)
    tag = w.name
    kvs = [0, w.kv_heads - 1]
    hs = kv_group_heads(w.heads, w.kv_heads, kvs)
    qc, doc = to_cpu_heads(q, hs), to_cpu_heads(do, hs)  # bf16 on the host; rows are picked before upcasting
    kc, vc = k[:, :, kvs].cpu(), v[:, :, kvs].cpu()
    # the oracle sees the sampled heads renumbered 0..len(hs)-1 over KV heads 0..len(kvs)-1
    r = oracle.joint_ranges(L)
    s_all, p_all = oracle.rows_of(r)

    # ---- oracle: sampled query rows (O, LSE, dQ)
    rows = sample_rows(L, M, n_random, seed=w.index)
    single = [(int(s_all[i]), int(p_all[i]), 1) for i in rows]
    O, LSE = oracle.fwd(qc[:, rows], kc, vc, single, r, M, clean_intra=reading, chunk=128, window=window)
    dQ, _, _ = oracle.bwd(qc[:, rows], kc, vc, O, LSE, doc[:, rows], single, r, M, clean_intra=reading, chunk=128,
                          window=window)
    # ---- oracle: key rows with few visible queries: corrupted blocks and the last two clean blocks
    # (with a window of at least 2M positions the same query rows are all that see them)
    nb = L // M
    key_sets = []
    for blk in (0, 1, nb // 2, nb - 1):
        qrows = list(range(blk * M, (blk + 1) * M))
        key_sets.append((f"corrupted block {blk}", qrows, list(range(blk * M, (blk + 1) * M))))
    qrows = list(range(2 * L - 2 * M, 2 * L)) + list(range(L - M, L))
    key_sets.append(("last clean blocks", qrows, list(range(2 * L - 2 * M, 2 * L))))
    key_refs = []
    for name, qrows, krows in key_sets:
        single_k = [(int(s_all[i]), int(p_all[i]), 1) for i in qrows]
        Oq, Lq = oracle.fwd(qc[:, qrows], kc, vc, single_k, r, M, clean_intra=reading, chunk=128, window=window)
        _, dK, dV = oracle.bwd(qc[:, qrows], kc, vc, Oq, Lq, doc[:, qrows], single_k, r, M, clean_intra=reading,
                               chunk=128, window=window)
        key_refs.append((name, krows, dK[:, krows], dV[:, krows]))

    for mode, hl in [(m, h) for m in outs for h in (hilos or (hilo,))]:
        f32 = mode == "f32"
        o, lse = bd.joint_fwd(q, k, v, M, clean_intra=reading, out_f32=f32, hilo=hl, window=window)
        dq, dk, dv = bd.joint_bwd(q, k, v, o, lse, do, M, clean_intra=reading, out_f32=f32, hilo=hl,
                                  window=window)
        torch.cuda.synchronize()
        t = f"{tag} [{mode} out{'' if not hilos else f', hilo {int(hl)}'}]"
        assert torch.isfinite(o).all() and torch.isfinite(lse).all()
        assert torch.isfinite(dq).all() and torch.isfinite(dk).all() and torch.isfinite(dv).all()
        dv_identity(dv, do, w.heads // w.kv_heads, t)

        def close(name, got, ref):
            if f32:
                assert_close(f"{t} {name}", got, ref, BF16)
            else:
                assert_close_bf16_out(f"{t} {name}", got, ref)

        close("O rows", o[:, rows][:, :, hs], O)
        assert_close(f"{t} LSE rows", lse[:, hs][:, :, rows], LSE, BF16)
        close("dQ rows", dq[:, rows][:, :, hs], dQ)
        for name, krows, dK, dV in key_refs:
            close(f"dK {name}", dk[:, krows][:, :, kvs], dK)
            close(f"dV {name}", dv[:, krows][:, :, kvs], dV)
        del o, lse, dq, dk, dv
        torch.cuda.empty_cache()
    del q, k, v, do
    torch.cuda.empty_cache()


def test_workload_32k_causal():
    """The headline step in both output modes: fp32 outputs (strict bar) and bf16
    outputs, the arithmetic bench.py times."""
    joint_check(WORKLOADS["32k"], 0, outs=("f32", "bf16"))


def test_workload_32k_block_reading():
    joint_check(WORKLOADS["32k"], 1, n_random=12, outs=("f32", "bf16"))


def test_workload_32k_window_1024():
    """The 32K shape in a sliding-window layer (1,024 positions), as bench.py times it (bf16
    outputs), and with fp32 outputs."""
    w = WORKLOADS["32k-w1024"]
    assert w.window >= 2 * w.block_size
    joint_check(w, 0, n_random=16, window=w.window, outs=("f32", "bf16"))


def test_workload_drafter32k():
    """The drafter share as bench.py times it: 2,048 draft blocks of 16 over 32,768
    target-feature rows.  Sampled draft rows (O, LSE, dQ); the draft keys of
    sampled blocks (seen by their own block only) and the last 64 target rows
    (seen only by the blocks whose anchors pass them): dK, dV complete; the
    sum-dV identity over both key ranges."""
    w = WORKLOADS["drafter32k"]
    torch.cuda.empty_cache()
    q, kd, vd, kt, vt, do, anchors = synth.make_drafter(w, device=DEV)
    M, T = w.block_size, w.L
    nd = w.draft_blocks * M
    p = bd.make_problem(1, T, M, w.heads, w.kv_heads, w.head_dim, torch.bfloat16, out_f32=True, clean_prefix=anchors)
    qr = [Range(CORRUPTED, 0, nd)]
    kr = [Range(CORRUPTED, 0, nd), Range(CLEAN, 0, T)]
    o = torch.empty(q.shape, dtype=F32, device=DEV)
    lse = torch.empty((1, w.heads, nd), dtype=F32, device=DEV)
    bd.attn_fwd(p, qr, [q], [o], [lse], kr, [kd, kt], [vd, vt])
    dq = torch.empty(q.shape, dtype=F32, device=DEV)
    dks = [torch.empty(t.shape, dtype=F32, device=DEV) for t in (kd, kt)]
    dvs = [torch.empty(t.shape, dtype=F32, device=DEV) for t in (vd, vt)]
    ws = torch.empty(bd.attn_bwd_workspace_bytes(p, qr), dtype=torch.uint8, device=DEV)
    bd.attn_bwd(p, qr, [q], [o], [lse], [do], [dq], kr, [kd, kt], [vd, vt], dks, dvs, ws)
    torch.cuda.synchronize()
    tag = w.name
    assert torch.isfinite(o).all() and torch.isfinite(dq).all()
    dv_identity(torch.cat(dvs, dim=1), do, w.heads // w.kv_heads, tag)

    kvs = [0, w.kv_heads - 1]
    hs = kv_group_heads(w.heads, w.kv_heads, kvs)
    qc, doc = to_cpu_heads(q, hs), to_cpu_heads(do, hs)
    kc = torch.cat([kd[:, :, kvs], kt[:, :, kvs]], dim=1).cpu()
    vc = torch.cat([vd[:, :, kvs], vt[:, :, kvs]], dim=1).cpu()
    pl = anchors.cpu().tolist()
    okr = [(CORRUPTED, 0, nd), (CLEAN, 0, T)]

    rows = sorted(set([0, M - 1, M, nd // 2, nd - M, nd - 1] +
                      np.random.default_rng(w.index).choice(nd, size=16, replace=False).tolist()))
    single = [(CORRUPTED, int(i), 1) for i in rows]
    O, LSE = oracle.fwd(qc[:, rows], kc, vc, single, okr, M, chunk=128, clean_prefix=pl)
    assert_close(f"{tag} O rows", o[:, rows][:, :, hs], O, BF16)
    assert_close(f"{tag} LSE rows", lse[:, hs][:, :, rows], LSE, BF16)
    dQ, _, _ = oracle.bwd(qc[:, rows], kc, vc, O, LSE, doc[:, rows], single, okr, M, chunk=128, clean_prefix=pl)
    assert_close(f"{tag} dQ rows", dq[:, rows][:, :, hs], dQ, BF16)

    nb = w.draft_blocks
    last = list(range(T - 64, T))
    seers = [b for b in range(nb) if pl[b] > T - 64]  # blocks whose target context reaches the last 64 rows
    key_sets = [(f"draft block {b}", list(range(b * M, (b + 1) * M)), 0, list(range(b * M, (b + 1) * M)))
                for b in (0, 1, nb // 2, nb - 1)]
    key_sets.append(("last target rows", [i for b in seers for i in range(b * M, (b + 1) * M)], 1, last))
    for name, qrows, kidx, krows in key_sets:
        assert qrows, name
        single = [(CORRUPTED, int(i), 1) for i in qrows]
        Oq, Lq = oracle.fwd(qc[:, qrows], kc, vc, single, okr, M, chunk=128, clean_prefix=pl)
        _, dK, dV = oracle.bwd(qc[:, qrows], kc, vc, Oq, Lq, doc[:, qrows], single, okr, M, chunk=128,
                               clean_prefix=pl)
        off = 0 if kidx == 0 else nd
        kk = [off + x for x in krows]
        assert_close(f"{tag} dK {name}", dks[kidx][:, krows][:, :, kvs], dK[:, kk], BF16)
        assert_close(f"{tag} dV {name}", dvs[kidx][:, krows][:, :, kvs], dV[:, kk], BF16)
    del q, kd, vd, kt, vt, do, o, lse, dq, dks, dvs, ws
    torch.cuda.empty_cache()


HILO_128K = bd.HILO_ALL | bd.HILO_ADAPTIVE


def test_workload_128k():
    """128K with 1% of the keys scaled x8 (logits up to about +-40), in the arithmetic
    that meets the bar there and that bench.py times: fp32 outputs and every P and dS
    product in two bf16 terms on the tiles that hold a probability of 1/64 or more
    (and, for comparison, on every tile).  Single terms fail in each kernel: P V and
    dS K leave about 7e-2 in dQ (|dS| up to about 30, and D = rowsum(dO O) inherits
    O's P rounding), P^T dO leaves 5.4e-2 in dV of a corrupted block whose queries
    put P near 1 on one amplified key, and bf16 outputs add O's output rounding to D
    (about 0.1 in dQ)."""
    joint_check(WORKLOADS["128k"], 0, n_random=8, hilos=(HILO_128K, bd.HILO_ALL))


def test_workload_128k_block_reading():
    joint_check(WORKLOADS["128k"], 1, n_random=4, hilo=HILO_128K)


def csbp_ranges(w):
    qr = Range(CORRUPTED, w.local_pos0, w.local_tokens)
    krs = [Range(CORRUPTED, w.local_pos0, w.local_tokens)] + \
          [Range(CLEAN, s * w.shard_tokens, w.shard_tokens) for s in range(w.n_shards)]
    return qr, krs


def shard_views(t, w):
    """Pointers of the shards of a contiguous clean-prefix buffer [1][clean][Hkv][D]."""
    step = w.shard_tokens * t.shape[2] * t.shape[3] * t.element_size()
    return [t.data_ptr() + s * step for s in range(w.n_shards)]


def closer(f32, tag):
    """Comparison of one output mode: strict on fp32 outputs, rounding-aware on bf16 outputs."""
    def close(name, got, ref):
        if f32:
            assert_close(f"{tag} {name}", got, ref, BF16)
        else:
            assert_close_bf16_out(f"{tag} {name}", got, ref)
    return close


@pytest.mark.parametrize("mode", ["f32", "bf16"])
def test_workload_csbp256k(mode):
    """One CSBP rank's share as bench.py runs it (17 partials, the merge, the
    17-range backward); "bf16" is bench.py's arithmetic (bf16 partials, merged
    O and gradients), "f32" returns the fp32 accumulators."""
    w = WORKLOADS["csbp256k"]
    torch.cuda.empty_cache()
    q, kl, vl, kc, vc, do = synth.make_csbp_rank(w, device=DEV)
    qr, krs = csbp_ranges(w)
    f32 = mode == "f32"
    ODT = F32 if f32 else torch.bfloat16
    close = closer(f32, f"csbp256k [{mode} out]")
    p = bd.make_problem(1, w.L, w.block_size, w.heads, w.kv_heads, w.head_dim, torch.bfloat16, out_f32=f32)
    n = w.local_tokens
    ks = [kl.data_ptr()] + shard_views(kc, w)
    vs = [vl.data_ptr()] + shard_views(vc, w)
    o_parts, l_parts = [], []
    for j, kr in enumerate(krs):
        o = torch.empty(q.shape, dtype=ODT, device=DEV)
        lse = torch.empty((1, w.heads, n), dtype=F32, device=DEV)
        bd.attn_partial_fwd(p, qr, q, o, lse, kr, ks[j], vs[j])
        o_parts.append(o)
        l_parts.append(lse)
    om = torch.empty(q.shape, dtype=ODT, device=DEV)
    lm = torch.empty((1, w.heads, n), dtype=F32, device=DEV)
    bd.lse_merge(o_parts, l_parts, om, lm)
    of = torch.empty(q.shape, dtype=ODT, device=DEV)
    lf = torch.empty((1, w.heads, n), dtype=F32, device=DEV)
    bd.attn_fwd(p, [qr], [q], [of], [lf], krs, ks, vs)
    torch.cuda.synchronize()
    for j in range(9, 17):  # shards 8..15 start at or after the first local block's position
        if krs[j].pos0 >= w.local_pos0 + w.local_tokens - w.block_size:
            assert torch.isneginf(l_parts[j]).all() and (o_parts[j] == 0).all()
    # fused multi-range launch = merge of per-range partials (eq:correctness-online-softmax-merge)
    close("fused vs merged O", of, om.cpu().double().numpy())
    assert_close(f"csbp256k [{mode} out] fused vs merged LSE", lf, lm.cpu().double().numpy(), BF16)

    dq = torch.empty(q.shape, dtype=ODT, device=DEV)
    dkl, dvl = (torch.empty(t.shape, dtype=ODT, device=DEV) for t in (kl, vl))
    dkc, dvc = (torch.empty(t.shape, dtype=ODT, device=DEV) for t in (kc, vc))
    ws = torch.empty(bd.attn_bwd_workspace_bytes(p, [qr]), dtype=torch.uint8, device=DEV)
    bd.attn_bwd(p, [qr], [q], [om], [lm], [do], [dq], krs, ks, vs,
                [dkl.data_ptr()] + shard_views(dkc, w), [dvl.data_ptr()] + shard_views(dvc, w), ws)
    torch.cuda.synchronize()
    dv_all = torch.cat([dvl, dvc], dim=1)
    dv_identity(dv_all, do, w.heads // w.kv_heads, "csbp256k")
    # shards whose positions no local block reaches get exact zeros
    visible_end = w.local_pos0 + w.local_tokens - w.block_size
    first_dead = -(-visible_end // w.shard_tokens)
    assert (dkc[:, first_dead * w.shard_tokens:] == 0).all() and (dvc[:, first_dead * w.shard_tokens:] == 0).all()

    kvs = [0, w.kv_heads - 1]
    hs = kv_group_heads(w.heads, w.kv_heads, kvs)
    qcpu, docpu = q[:, :, hs].cpu(), do[:, :, hs].cpu()
    kall = torch.cat([kl, kc], dim=1)[:, :, kvs].cpu()
    vall = torch.cat([vl, vc], dim=1)[:, :, kvs].cpu()
    qranges = [(CORRUPTED, w.local_pos0, n)]
    kranges = [(r.stream, r.pos0, r.len) for r in krs]
    rng = np.random.default_rng(4)
    rows = sorted(set([0, 31, 32, n // 2, n - 32, n - 1] + rng.choice(n, 16, replace=False).tolist()))
    O, LSE = oracle.fwd(qcpu, kall, vall, qranges, kranges, w.block_size, q_rows=rows)
    close("merged O rows", om[:, rows][:, :, hs], O)
    assert_close(f"csbp256k [{mode} out] merged LSE rows", lm[:, hs][:, :, rows], LSE, BF16)
    single = [(CORRUPTED, w.local_pos0 + i, 1) for i in rows]
    dQ, _, _ = oracle.bwd(qcpu[:, rows], kall, vall, O, LSE, docpu[:, rows], single, kranges, w.block_size)
    close("dQ rows", dq[:, rows][:, :, hs], dQ)
    # local corrupted blocks (block-local keys) and the tail of the partly visible shard
    M = w.block_size
    for blk in (0, n // M // 2, n // M - 1):
        qrows = list(range(blk * M, (blk + 1) * M))
        Oq, Lq = oracle.fwd(qcpu, kall, vall, qranges, kranges, M, q_rows=qrows)
        single = [(CORRUPTED, w.local_pos0 + i, 1) for i in qrows]
        _, dK, dV = oracle.bwd(qcpu[:, qrows], kall, vall, Oq, Lq, docpu[:, qrows], single, kranges, M)
        kr = list(range(blk * M, (blk + 1) * M))
        close(f"dK local block {blk}", dkl[:, kr][:, :, kvs], dK[:, kr])
        close(f"dV local block {blk}", dvl[:, kr][:, :, kvs], dV[:, kr])
    # clean keys of the last visible clean block: seen only by the last local block's queries
    qrows = list(range(n - M, n))
    Oq, Lq = oracle.fwd(qcpu, kall, vall, qranges, kranges, M, q_rows=qrows)
    single = [(CORRUPTED, w.local_pos0 + i, 1) for i in qrows]
    _, dK, dV = oracle.bwd(qcpu[:, qrows], kall, vall, Oq, Lq, docpu[:, qrows], single, kranges, M)
    kpos = list(range(visible_end - M, visible_end))  # clean positions
    krow = [n + x for x in kpos]  # rows in the concatenated [local ; clean] key tensor
    close("dK last visible clean block", dkc[:, kpos][:, :, kvs], dK[:, krow])
    close("dV last visible clean block", dvc[:, kpos][:, :, kvs], dV[:, krow])


@pytest.mark.parametrize("mode", ["f32", "bf16"])
@pytest.mark.parametrize("reading", [0, 1], ids=["causal", "block"])
def test_workload_csbp256k_rank_operator(reading, mode):
    """One CSBP rank with its clean-shard queries too (Alg. 1/2 for one rank), in
    both readings of the clean-to-clean rule and both output modes.

    The rank owns clean shard 8 (the positions of its corrupted blocks); its
    clean queries attend causally to all gathered clean keys, i.e. shards 0..8.
    Forward: corrupted queries by per-range partials + merge, clean queries by
    one multi-range launch (checked against their own partials + merge);
    backward: one call over both query ranges and all 17 key ranges.
    """
    w = WORKLOADS["csbp256k"]
    torch.cuda.empty_cache()
    q, kl, vl, kc, vc, do = synth.make_csbp_rank(w, device=DEV)
    qc, doc = synth.make_csbp_clean_queries(w, device=DEV)
    own, S, n, M = synth.csbp_own_shard(w), w.shard_tokens, w.local_tokens, w.block_size
    qr, krs = csbp_ranges(w)
    qrc = Range(CLEAN, own * S, S)
    f32 = mode == "f32"
    ODT = F32 if f32 else torch.bfloat16
    close = closer(f32, f"csbp256k rank r{reading} [{mode} out]")
    p = bd.make_problem(1, w.L, w.block_size, w.heads, w.kv_heads, w.head_dim, torch.bfloat16, out_f32=f32,
                        clean_intra=reading)
    ks = [kl.data_ptr()] + shard_views(kc, w)
    vs = [vl.data_ptr()] + shard_views(vc, w)

    def partials_merged(qrange, qt, rows):
        o_parts, l_parts = [], []
        for j, kr in enumerate(krs):
            o = torch.empty(qt.shape, dtype=ODT, device=DEV)
            lse = torch.empty((1, w.heads, rows), dtype=F32, device=DEV)
            bd.attn_partial_fwd(p, qrange, qt, o, lse, kr, ks[j], vs[j])
            o_parts.append(o)
            l_parts.append(lse)
        om = torch.empty(qt.shape, dtype=ODT, device=DEV)
        lm = torch.empty((1, w.heads, rows), dtype=F32, device=DEV)
        bd.lse_merge(o_parts, l_parts, om, lm)
        return om, lm, l_parts

    om, lm, _ = partials_merged(qr, q, n)
    oc = torch.empty(qc.shape, dtype=ODT, device=DEV)
    lc = torch.empty((1, w.heads, S), dtype=F32, device=DEV)
    bd.attn_fwd(p, [qrc], [qc], [oc], [lc], krs, ks, vs)
    omc, lmc, lpc = partials_merged(qrc, qc, S)
    torch.cuda.synchronize()
    # clean queries never see corrupted keys nor shards past their own
    assert torch.isneginf(lpc[0]).all()
    for s in range(own + 1, w.n_shards):
        assert torch.isneginf(lpc[1 + s]).all()
    close("clean fused vs merged O", oc, omc.cpu().double().numpy())
    assert_close(f"rank r{reading} [{mode} out] clean fused vs merged LSE", lc, lmc.cpu().double().numpy(), BF16)

    dq = torch.empty(q.shape, dtype=ODT, device=DEV)
    dqc = torch.empty(qc.shape, dtype=ODT, device=DEV)
    dkl, dvl = (torch.empty(t.shape, dtype=ODT, device=DEV) for t in (kl, vl))
    dkc, dvc = (torch.empty(t.shape, dtype=ODT, device=DEV) for t in (kc, vc))
    ws = torch.empty(bd.attn_bwd_workspace_bytes(p, [qr, qrc]), dtype=torch.uint8, device=DEV)
    bd.attn_bwd(p, [qr, qrc], [q, qc], [om, oc], [lm, lc], [do, doc], [dq, dqc], krs, ks, vs,
                [dkl.data_ptr()] + shard_views(dkc, w), [dvl.data_ptr()] + shard_views(dvc, w), ws)
    torch.cuda.synchronize()
    dv_identity(torch.cat([dvl, dvc], dim=1), torch.cat([do, doc], dim=1), w.heads // w.kv_heads, "csbp256k rank")
    # clean keys past the rank's own shard are seen by nobody on this rank
    assert (dkc[:, (own + 1) * S:] == 0).all() and (dvc[:, (own + 1) * S:] == 0).all()

    kvs = [0, w.kv_heads - 1]
    hs = kv_group_heads(w.heads, w.kv_heads, kvs)
    qcat = torch.cat([q, qc], dim=1)[:, :, hs].cpu()
    docat = torch.cat([do, doc], dim=1)[:, :, hs].cpu()
    kall = torch.cat([kl, kc], dim=1)[:, :, kvs].cpu()
    vall = torch.cat([vl, vc], dim=1)[:, :, kvs].cpu()
    qranges = [(CORRUPTED, w.local_pos0, n), (CLEAN, own * S, S)]
    kranges = [(r.stream, r.pos0, r.len) for r in krs]

    def single(rows):
        return [(CORRUPTED, w.local_pos0 + i, 1) if i < n else (CLEAN, own * S + i - n, 1) for i in rows]

    rng = np.random.default_rng(5)
    crow = sorted(set([0, 1, M - 1, M, S // 2, S - M, S - 1] + rng.choice(S, 12, replace=False).tolist()))
    rows = [n + i for i in crow]
    O, LSE = oracle.fwd(qcat, kall, vall, qranges, kranges, M, q_rows=rows, clean_intra=reading)
    close("clean O rows", oc[:, crow][:, :, hs], O)
    assert_close(f"rank r{reading} [{mode} out] clean LSE rows", lc[:, hs][:, :, crow], LSE, BF16)
    dQ, _, _ = oracle.bwd(qcat[:, rows], kall, vall, O, LSE, docat[:, rows], single(rows), kranges, M,
                          clean_intra=reading)
    close("clean dQ rows", dqc[:, crow][:, :, hs], dQ)
    # the last two clean key blocks of the own shard: seen by the last two blocks of
    # clean queries and (for the earlier block) the last corrupted block
    qrows = list(range(n - M, n)) + [n + i for i in range(S - 2 * M, S)]
    Oq, Lq = oracle.fwd(qcat, kall, vall, qranges, kranges, M, q_rows=qrows, clean_intra=reading)
    _, dK, dV = oracle.bwd(qcat[:, qrows], kall, vall, Oq, Lq, docat[:, qrows], single(qrows), kranges, M,
                           clean_intra=reading)
    kpos = list(range((own + 1) * S - 2 * M, (own + 1) * S))
    krow = [n + x for x in kpos]
    close("own-shard tail dK", dkc[:, kpos][:, :, kvs], dK[:, krow])
    close("own-shard tail dV", dvc[:, kpos][:, :, kvs], dV[:, krow])
