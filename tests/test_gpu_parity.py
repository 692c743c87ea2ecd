"""GPU parity: the HIP library (through its C ABI) against the fp64 oracle.

Small shapes span several tiles and ragged tails in every dimension the
kernels tile (128- and 256-row forward and dQ query tiles, 64-key forward key tiles, 128-key
backward key tiles, 32-row backward query steps); they cover both readings of
the clean-to-clean rule, GQA groups, head_dim 64 and 128, batch > 1, the
degenerate block sizes (1 and L) and rows that see no key.
"""
import math

import numpy as np
import pytest
import torch

import oracle
import paper_2609_19242_amd as bd
from paper_2609_19242_amd import CLEAN, CORRUPTED, Range
from synth import WORKLOADS, make_joint
from tests.gpu_util import assert_close, assert_close_bf16_out, joint_inputs, kv_group_heads

pytestmark = pytest.mark.gpu
DEV = "cuda"


def run_joint(q, k, v, do, M, reading, out_f32, hilo=False):
    qd, kd, vd, dod = (t.to(DEV) for t in (q, k, v, do))
    o, lse = bd.joint_fwd(qd, kd, vd, M, clean_intra=reading, out_f32=out_f32, hilo=hilo)
    dq, dk, dv = bd.joint_bwd(qd, kd, vd, o, lse, dod, M, clean_intra=reading, out_f32=out_f32, hilo=hilo)
    torch.cuda.synchronize()
    return o, lse, dq, dk, dv


def check_joint(q, k, v, do, M, reading, dtype, heads=None, tag="", out_f32=True, hilo=False, outs=None):
    """GPU joint fwd+bwd against the oracle on the query heads ``heads`` (all by default).

    ``outs`` lists the output modes to run against one oracle result ("f32":
    the fp32 accumulators, strict tolerance; "bf16": outputs rounded to bf16,
    whose bound adds the output rounding, and whose backward reads the rounded
    O); by default the single mode ``out_f32`` selects.  Returns the GPU
    results of the last mode.
    """
    L = q.shape[1] // 2
    outs = outs or (("f32",) if out_f32 else ("bf16",))
    hs = list(range(q.shape[2])) if heads is None else heads
    O, LSE = oracle.joint_fwd(q, k, v, L, M, clean_intra=reading, heads=hs)
    dQ, dK, dV = oracle.joint_bwd(q, k, v, O, LSE, do[:, :, hs], L, M, clean_intra=reading, heads=hs)
    kvs = sorted(set(h // (q.shape[2] // k.shape[2]) for h in hs))
    for mode in outs:
        f32 = mode == "f32" or dtype == torch.float32
        o, lse, dq, dk, dv = run_joint(q, k, v, do, M, reading, f32, hilo)
        assert_close(f"{tag} [{mode} out] LSE", lse[:, hs], LSE, dtype)
        pairs = (("O", o[:, :, hs], O), ("dQ", dq[:, :, hs], dQ), ("dK", dk[:, :, kvs], dK[:, :, kvs]),
                 ("dV", dv[:, :, kvs], dV[:, :, kvs]))
        for name, got, ref in pairs:
            if f32:
                assert_close(f"{tag} [{mode} out] {name}", got, ref, dtype)
            else:
                assert_close_bf16_out(f"{tag} [{mode} out] {name}", got, ref)
    return o, lse, dq, dk, dv


SMALL = [
    # L, M, Hq, Hkv, D, batch
    (300, 12, 4, 2, 128, 1),
    (300, 20, 2, 2, 64, 2),
    (320, 1, 4, 1, 128, 1),
    (256, 256, 2, 1, 128, 1),
    (200, 8, 8, 2, 128, 1),
    (520, 40, 2, 1, 128, 1),
    # batch x KV heads a multiple of 8 above 8: the dK/dV kernels interleave the
    # (batch, KV head) pairs that share an XCD (2 per XCD here, 3 below)
    (200, 8, 16, 8, 128, 2),
    (150, 10, 8, 8, 64, 3),
]


HILO_OF_MODE = {"bf16-hilo": bd.HILO_ALL, "bf16-hilo-adaptive": bd.HILO_ALL | bd.HILO_ADAPTIVE}


@pytest.mark.parametrize("mode", ["bf16", "bf16-out-bf16", "bf16-hilo", "bf16-hilo-adaptive", "fp32"])
@pytest.mark.parametrize("reading", [0, 1], ids=["causal", "block"])
@pytest.mark.parametrize("shape", SMALL, ids=lambda s: "L{}-M{}-H{}x{}-d{}-b{}".format(*s))
def test_joint_small(shape, reading, mode):
    L, M, Hq, Hkv, D, B = shape
    dtype = torch.float32 if mode == "fp32" else torch.bfloat16
    q, k, v, do = joint_inputs(L, Hq, Hkv, D, dtype, batch=B, seed=L + M + D)
    check_joint(q, k, v, do, M, reading, dtype, tag=f"L{L} M{M} r{reading}", out_f32=(mode != "bf16-out-bf16"),
                hilo=HILO_OF_MODE.get(mode, 0))


@pytest.mark.parametrize("hilo", ["all", "adaptive"])
@pytest.mark.parametrize("shape", [SMALL[0], SMALL[4], SMALL[6]], ids=lambda s: "L{}-M{}-H{}x{}-d{}-b{}".format(*s))
def test_joint_small_two_terms_bf16_outputs(shape, hilo):
    """Two-term products with bf16 outputs, both output modes against one oracle result: the forward's
    bf16 O goes through its LDS-staged epilogue, the adaptive dQ kernel stores bf16 dQ directly."""
    L, M, Hq, Hkv, D, B = shape
    q, k, v, do = joint_inputs(L, Hq, Hkv, D, torch.bfloat16, batch=B, seed=L + M + D + 7)
    check_joint(q, k, v, do, M, 0, torch.bfloat16, tag=f"L{L} M{M} two-term {hilo}", outs=("f32", "bf16"),
                hilo=HILO_OF_MODE["bf16-hilo" if hilo == "all" else "bf16-hilo-adaptive"])


@pytest.mark.parametrize("reading", [0, 1], ids=["causal", "block"])
@pytest.mark.parametrize("hilo", ["all", "adaptive"])
@pytest.mark.parametrize("Hq", [8, 6], ids=["group4", "group3"])
def test_two_terms_amplified_keys(reading, hilo, Hq):
    """Keys of large norm (3% of the key rows x8, so many rows put nearly all of their
    probability on one key) with two-term products on every tile and on the adaptive
    selection: batch 1, L = 2048 + 2048, block 128, Hq/2 heads, d 128, every row and
    key against the oracle with fp32 outputs.  Both branches of the adaptive test run:
    tiles with a large probability and tiles without one; an even GQA group takes the
    scheduled dK/dV kernel, an odd one the general kernel."""
    import synth
    L, M, Hkv, D = 2048, 128, 2, 128
    q = synth.normal((1, 2 * L, Hq, D), 9100, torch.bfloat16)
    k32 = synth.normal((1, 2 * L, Hkv, D), 9101, torch.float32)
    k32[:, synth.amplified_rows(2 * L, 0.03, 9104)] *= 8.0
    k = k32.to(torch.bfloat16)
    v = synth.normal((1, 2 * L, Hkv, D), 9102, torch.bfloat16)
    do = synth.normal((1, 2 * L, Hq, D), 9103, torch.bfloat16)
    h = bd.HILO_ALL | (bd.HILO_ADAPTIVE if hilo == "adaptive" else 0)
    check_joint(q, k, v, do, M, reading, torch.bfloat16, tag=f"amplified {hilo} H{Hq} r{reading}", hilo=h)


@pytest.mark.parametrize("hilo", ["single", "adaptive"])
def test_forward_running_max_moves_mid_walk(hilo):
    """Scores that grow along the key positions (about 12 log2 units per 64-key tile,
    over 190 across the sequence), so the forward's running max moves several times
    inside a row's walk (the lazy rescale of O and of the row sum), not only on the
    row's first tile: O and LSE of every row against the oracle, batch 1,
    L = 1024 + 1024, block 32, 2/1 heads, d 128, fp32 outputs."""
    import synth
    L, M, Hq, Hkv, D = 1024, 32, 2, 1, 128
    q = synth.normal((1, 2 * L, Hq, D), 9200, torch.float32)
    q[..., 0] = 20.0
    k = synth.normal((1, 2 * L, Hkv, D), 9201, torch.float32) * 0.1
    ramp = 0.075 * torch.arange(L, dtype=torch.float32)
    k[0, :L, 0, 0] = ramp  # corrupted stream
    k[0, L:, 0, 0] = ramp  # clean stream
    q, k = q.to(torch.bfloat16), k.to(torch.bfloat16)
    v = synth.normal((1, 2 * L, Hkv, D), 9202, torch.bfloat16)
    s2 = (k[0, L:, 0].double() @ q[0, -1, 0].double()) / math.sqrt(D) * math.log2(math.e)
    assert float(s2.max() - s2.min()) > 3 * 64, "the test needs several moves of the running max"
    h = 0 if hilo == "single" else bd.HILO_ALL | bd.HILO_ADAPTIVE
    o, lse = bd.joint_fwd(q.to(DEV), k.to(DEV), v.to(DEV), M, out_f32=True, hilo=h)
    torch.cuda.synchronize()
    O, LSE = oracle.joint_fwd(q, k, v, L, M)
    assert_close(f"rising scores {hilo} O", o, O, torch.bfloat16)
    assert_close(f"rising scores {hilo} LSE", lse, LSE, torch.bfloat16)


@pytest.mark.parametrize("reading", [0, 1], ids=["causal", "block"])
def test_workload_tiny_fp32(reading):
    w = WORKLOADS["tiny"]
    q, k, v, do = make_joint(w)
    check_joint(q, k, v, do, w.block_size, reading, torch.float32, tag=f"tiny r{reading}")


@pytest.mark.parametrize("reading", [0, 1], ids=["causal", "block"])
def test_workload_4k_bf16_head_subset(reading):
    """The 4k workload (batch 2, L = 4096 + 4096, block 32, 32/8 heads): every row and
    every key of KV groups {0, 7}, with fp32 and with bf16 outputs (bench.py's arithmetic)."""
    w = WORKLOADS["4k"]
    q, k, v, do = make_joint(w)
    hs = kv_group_heads(w.heads, w.kv_heads, [0, w.kv_heads - 1])
    o, lse, *_ = check_joint(q, k, v, do, w.block_size, reading, torch.bfloat16, heads=hs, tag=f"4k r{reading}",
                             outs=("f32", "bf16"))
    assert torch.isfinite(o).all() and torch.isfinite(lse).all()


@pytest.mark.parametrize("reading", [0, 1], ids=["causal", "block"])
def test_complete_kv_group_8k_block64(reading):
    """Element by element over one whole KV group at a size where clean keys are
    seen by thousands of query rows: batch 1, L = 8192 + 8192, block 64, 32/8
    heads, d 128; every row of query heads 0-3 (O, LSE, dQ) and every key of KV
    head 0 (dK, dV summed over the group), with fp32 and with bf16 outputs."""
    import synth
    L, M, Hq, Hkv, D = 8192, 64, 32, 8, 128
    q = synth.normal((1, 2 * L, Hq, D), 9000, torch.bfloat16)
    k = synth.normal((1, 2 * L, Hkv, D), 9001, torch.bfloat16)
    v = synth.normal((1, 2 * L, Hkv, D), 9002, torch.bfloat16)
    do = synth.normal((1, 2 * L, Hq, D), 9003, torch.bfloat16)
    check_joint(q, k, v, do, M, reading, torch.bfloat16, heads=[0, 1, 2, 3], tag=f"8k group0 r{reading}",
                outs=("f32", "bf16"))


# ------------------------------------------------------ partial + merge, CSBP
def csbp_case(dtype, M=8, n_local=96, pos0=512, shard=256, n_shards=4, Hq=4, Hkv=2, D=128, seed=5):
    import synth
    q = synth.normal((1, n_local, Hq, D), seed, dtype)
    kl = synth.normal((1, n_local, Hkv, D), seed + 1, dtype)
    vl = synth.normal((1, n_local, Hkv, D), seed + 2, dtype)
    kc = synth.normal((1, shard * n_shards, Hkv, D), seed + 3, dtype)
    vc = synth.normal((1, shard * n_shards, Hkv, D), seed + 4, dtype)
    do = synth.normal((1, n_local, Hq, D), seed + 5, dtype)
    qr = Range(CORRUPTED, pos0, n_local)
    krs = [Range(CORRUPTED, pos0, n_local)] + [Range(CLEAN, s * shard, shard) for s in range(n_shards)]
    ks = [kl] + [kc[:, s * shard:(s + 1) * shard].contiguous() for s in range(n_shards)]
    vs = [vl] + [vc[:, s * shard:(s + 1) * shard].contiguous() for s in range(n_shards)]
    return q, ks, vs, do, qr, krs


@pytest.mark.parametrize("mode", ["bf16", "bf16-out-bf16", "fp32"])
def test_csbp_partials_merge_and_backward(mode):
    M = 8
    dtype = torch.float32 if mode == "fp32" else torch.bfloat16
    out_f32 = mode != "bf16-out-bf16"
    odt = torch.float32 if out_f32 else dtype
    q, ks, vs, do, qr, krs = csbp_case(dtype, M=M)
    B, n, Hq, D = q.shape
    Hkv = ks[0].shape[2]
    L = 2048
    p = bd.make_problem(1, L, M, Hq, Hkv, D, dtype, out_f32=out_f32)
    qd, dod = q.to(DEV), do.to(DEV)
    kd = [t.to(DEV) for t in ks]
    vd = [t.to(DEV) for t in vs]
    o_parts, l_parts = [], []
    for kr, kk, vv in zip(krs, kd, vd):
        o = torch.empty(qd.shape, dtype=odt, device=DEV)
        lse = torch.empty((1, Hq, n), dtype=torch.float32, device=DEV)
        bd.attn_partial_fwd(p, qr, qd, o, lse, kr, kk, vv)
        o_parts.append(o)
        l_parts.append(lse)
    om = torch.empty(qd.shape, dtype=odt, device=DEV)
    lm = torch.empty((1, Hq, n), dtype=torch.float32, device=DEV)
    bd.lse_merge(o_parts, l_parts, om, lm)
    # fused multi-range forward in one launch
    of = torch.empty(qd.shape, dtype=odt, device=DEV)
    lf = torch.empty((1, Hq, n), dtype=torch.float32, device=DEV)
    bd.attn_fwd(p, [qr], [qd], [of], [lf], krs, kd, vd)
    torch.cuda.synchronize()

    qranges = [(CORRUPTED, qr.pos0, qr.len)]
    kranges = [(r.stream, r.pos0, r.len) for r in krs]
    kall = torch.cat(ks, dim=1)
    vall = torch.cat(vs, dim=1)
    O, LSE = oracle.fwd(q, kall, vall, qranges, kranges, M)
    def close(name, got, ref):
        if out_f32:
            assert_close(name, got, ref, dtype)
        else:
            assert_close_bf16_out(name, got, ref)

    for j, (kr, kk, vv) in enumerate(zip(krs, ks, vs)):
        Oj, Lj = oracle.fwd(q, kk, vv, qranges, [kranges[j]], M)
        close(f"partial{j} O", o_parts[j], Oj)
        assert_close(f"partial{j} LSE", l_parts[j], Lj, dtype)
    # shard 3 covers clean positions 768..1023, beyond every local block's prefix
    assert torch.isneginf(l_parts[4]).all() and (o_parts[4] == 0).all()
    close("merged O", om, O)
    assert_close("merged LSE", lm, LSE, dtype)
    close("fused O", of, O)
    assert_close("fused LSE", lf, LSE, dtype)

    # backward over the key-range list with the merged (O, LSE)
    dq = torch.empty(qd.shape, dtype=odt, device=DEV)
    dks = [torch.empty(t.shape, dtype=odt, device=DEV) for t in kd]
    dvs = [torch.empty(t.shape, dtype=odt, device=DEV) for t in vd]
    ws = torch.empty(bd.attn_bwd_workspace_bytes(p, [qr]), dtype=torch.uint8, device=DEV)
    bd.attn_bwd(p, [qr], [qd], [om], [lm], [dod], [dq], krs, kd, vd, dks, dvs, ws)
    torch.cuda.synchronize()
    dQ, dK, dV = oracle.bwd(q, kall, vall, O, LSE, do, qranges, kranges, M)
    close("csbp dQ", dq, dQ)
    off = 0
    for j, kk in enumerate(ks):
        nrows = kk.shape[1]
        close(f"csbp dK{j}", dks[j], dK[:, off:off + nrows])
        close(f"csbp dV{j}", dvs[j], dV[:, off:off + nrows])
        off += nrows
    assert (dks[4] == 0).all() and (dvs[4] == 0).all()


def test_merge_kernel_random_partials():
    """Merge of arbitrary partials (including all-empty rows) against the oracle's merge."""
    g = torch.Generator().manual_seed(3)
    B, R, H, D, J = 2, 77, 3, 128, 5
    os_ = [torch.randn(B, R, H, D, generator=g) for _ in range(J)]
    ls = [torch.randn(B, H, R, generator=g) * 4 for _ in range(J)]
    for j in range(J):  # some parts empty for some rows
        mask = torch.rand(B, H, R, generator=g) < 0.3
        ls[j][mask] = -float("inf")
    ls[0][:, :, :5] = -float("inf")
    for j in range(1, J):
        ls[j][:, :, :5] = -float("inf")
    for j in range(J):
        os_[j] = torch.where(torch.isneginf(ls[j]).transpose(1, 2)[..., None], torch.zeros(()), os_[j]).contiguous()
    O, LSE = oracle.lse_merge(os_, ls)
    for pdt, odt in ((torch.float32, torch.float32), (torch.bfloat16, torch.bfloat16), (torch.bfloat16, torch.float32)):
        od = [t.to(pdt).to(DEV) for t in os_]
        ld = [t.to(DEV) for t in ls]
        o = torch.empty(B, R, H, D, dtype=odt, device=DEV)
        lse = torch.empty(B, H, R, dtype=torch.float32, device=DEV)
        bd.lse_merge(od, ld, o, lse)
        torch.cuda.synchronize()
        Or, Lr = oracle.lse_merge([t.to(pdt) for t in os_], ls)
        tol = torch.float32 if (pdt, odt) == (torch.float32, torch.float32) else torch.bfloat16
        assert_close(f"merge {pdt}->{odt} O", o, Or, tol)
        assert_close(f"merge {pdt}->{odt} LSE", lse, Lr, tol)
        assert (o[:, :5] == 0).all() and torch.isneginf(lse[:, :, :5]).all()


@pytest.mark.parametrize("pdt,odt", [(torch.bfloat16, torch.bfloat16), (torch.float32, torch.float32)],
                         ids=["bf16", "fp32"])
def test_merge_of_strided_views(pdt, odt):
    """bdlm_lse_merge_strided through lse_merge: partials that are row windows of larger tensors
    (batch stride 700, rows 100..399) merged into a window of another (batch stride 500, rows
    50..349), every padding row NaN.  The merged rows equal the dense merge of contiguous copies
    bit for bit and the oracle's merge; no padding row is read into or written."""
    g = torch.Generator().manual_seed(11)
    B, R, H, D, J, SP, SO, P0, Q0 = 2, 300, 4, 128, 4, 700, 500, 100, 50
    os_ = [torch.randn(B, R, H, D, generator=g) for _ in range(J)]
    ls = [torch.randn(B, H, R, generator=g) * 4 for _ in range(J)]
    ls[1][:, :, 7:40] = -float("inf")
    os_[1][:, 7:40] = 0.0
    big_o = [torch.full((B, SP, H, D), float("nan"), dtype=pdt, device=DEV) for _ in range(J)]
    big_l = [torch.full((B, H, SP), float("nan"), device=DEV) for _ in range(J)]
    for j in range(J):
        big_o[j][:, P0:P0 + R] = os_[j].to(pdt).to(DEV)
        big_l[j][:, :, P0:P0 + R] = ls[j].to(DEV)
    out_o = torch.full((B, SO, H, D), float("nan"), dtype=odt, device=DEV)
    out_l = torch.full((B, H, SO), float("nan"), device=DEV)
    bd.lse_merge([t[:, P0:P0 + R] for t in big_o], [t[:, :, P0:P0 + R] for t in big_l],
                 out_o[:, Q0:Q0 + R], out_l[:, :, Q0:Q0 + R])
    dense_o = torch.empty(B, R, H, D, dtype=odt, device=DEV)
    dense_l = torch.empty(B, H, R, device=DEV)
    bd.lse_merge([t[:, P0:P0 + R].contiguous() for t in big_o], [t[:, :, P0:P0 + R].contiguous() for t in big_l],
                 dense_o, dense_l)
    torch.cuda.synchronize()
    assert torch.equal(out_o[:, Q0:Q0 + R], dense_o) and torch.equal(out_l[:, :, Q0:Q0 + R], dense_l)
    assert torch.isnan(out_o[:, :Q0]).all() and torch.isnan(out_o[:, Q0 + R:]).all()
    assert torch.isnan(out_l[:, :, :Q0]).all() and torch.isnan(out_l[:, :, Q0 + R:]).all()
    Or, Lr = oracle.lse_merge([t.to(pdt) for t in os_], ls)
    tol = torch.float32 if pdt == torch.float32 else torch.bfloat16
    assert_close(f"strided merge {pdt} O", dense_o, Or, tol)
    assert_close(f"strided merge {pdt} LSE", dense_l, Lr, tol)


def test_backward_split_over_key_ranges():
    """A backward over key ranges A and B equals one call over A and one over B: each range's
    dK/dV bit for bit, and dQ as the sum of the two calls' dQ (fp32, summation order aside).
    This is how a caller with more key ranges than one call takes splits its backward."""
    L, M, Hq, Hkv, D = 384, 16, 4, 2, 128
    q, k, v, do = (t.to(DEV) for t in joint_inputs(L, Hq, Hkv, D, torch.bfloat16, seed=123))
    o, lse = bd.joint_fwd(q, k, v, M, out_f32=True)
    p = bd.make_problem(1, L, M, Hq, Hkv, D, torch.bfloat16, out_f32=True)
    r = bd.joint_ranges(L)
    halves = lambda t: bd._joint_ptrs(t, L)  # noqa: E731
    lp = [lse.data_ptr(), lse.data_ptr() + L * 4]
    ws = torch.empty(bd.attn_bwd_workspace_bytes(p, r), dtype=torch.uint8, device=DEV)

    def run(key_sel):
        dq = torch.zeros(q.shape, dtype=torch.float32, device=DEV)
        dk = torch.full(k.shape, float("nan"), dtype=torch.float32, device=DEV)
        dv = torch.full(v.shape, float("nan"), dtype=torch.float32, device=DEV)
        kr = [r[i] for i in key_sel]
        pick = lambda ptrs: [ptrs[i] for i in key_sel]  # noqa: E731
        bd.attn_bwd(p, r, halves(q), halves(o), lp, halves(do), halves(dq), kr, pick(halves(k)), pick(halves(v)),
                    pick(halves(dk)), pick(halves(dv)), ws)
        torch.cuda.synchronize()
        return dq, dk, dv

    dq, dk, dv = run([0, 1])
    dq0, dk0, dv0 = run([0])
    dq1, dk1, dv1 = run([1])
    rows0 = slice(0, L) if r[0].stream == CORRUPTED else slice(L, 2 * L)
    rows1 = slice(L, 2 * L) if rows0.start == 0 else slice(0, L)
    assert torch.equal(dk0[:, rows0], dk[:, rows0]) and torch.equal(dv0[:, rows0], dv[:, rows0])
    assert torch.equal(dk1[:, rows1], dk[:, rows1]) and torch.equal(dv1[:, rows1], dv[:, rows1])
    assert_close("split dQ", dq0 + dq1, dq.double().cpu().numpy(), torch.float32)


def test_empty_rows_partial():
    """Corrupted queries of block 0 over the clean stream: O = 0 exactly, LSE = -inf."""
    L, M, H, D = 256, 32, 2, 128
    q, k, v, _ = joint_inputs(L, H, H, D, torch.bfloat16, seed=9)
    p = bd.make_problem(1, L, M, H, H, D, torch.bfloat16)
    qd = q[:, :L].contiguous().to(DEV)
    kd, vd = k[:, L:].contiguous().to(DEV), v[:, L:].contiguous().to(DEV)
    o = torch.full(qd.shape, 7.0, dtype=torch.bfloat16, device=DEV)
    lse = torch.zeros((1, H, L), dtype=torch.float32, device=DEV)
    bd.attn_partial_fwd(p, Range(CORRUPTED, 0, L), qd, o, lse, Range(CLEAN, 0, L), kd, vd)
    torch.cuda.synchronize()
    assert (o[:, :M] == 0).all() and torch.isneginf(lse[:, :, :M]).all()
    O, LSE = oracle.fwd(q[:, :L], k[:, L:], v[:, L:], [(CORRUPTED, 0, L)], [(CLEAN, 0, L)], M)
    assert_close("empty-rows O", o, O, torch.bfloat16)
    assert_close("empty-rows LSE", lse, LSE, torch.bfloat16)


# ------------------------------------------- more than two query ranges
@pytest.mark.parametrize("split", ["q3-k3", "q4-k4"])
@pytest.mark.parametrize("heads", [(4, 2, 128), (3, 1, 64)], ids=["H4x2-d128", "H3x1-d64"])
def test_multi_range_fwd_bwd(split, heads):
    """The joint problem cut into three or four query ranges and as many key
    ranges (uneven cuts, each range its own tensor), forward and backward in one
    call each, against the oracle over the same ranges."""
    Hq, Hkv, D = heads
    L, M = 300, 12
    q, k, v, do = joint_inputs(L, Hq, Hkv, D, torch.bfloat16, seed=41 + D)
    cuts = {"q3-k3": ([(CORRUPTED, 0, 140), (CORRUPTED, 140, 160), (CLEAN, 0, 300)],
                      [(CLEAN, 0, 90), (CLEAN, 90, 210), (CORRUPTED, 0, 300)]),
            "q4-k4": ([(CLEAN, 170, 130), (CORRUPTED, 0, 97), (CLEAN, 0, 170), (CORRUPTED, 97, 203)],
                      [(CORRUPTED, 150, 150), (CLEAN, 0, 300), (CORRUPTED, 0, 33), (CORRUPTED, 33, 117)])}[split]
    qrs, krs = cuts

    def rows(t, rs):  # joint tensors hold corrupted rows [0, L) then clean rows [L, 2L)
        return [t[:, (L if s == CLEAN else 0) + p0:(L if s == CLEAN else 0) + p0 + n].contiguous() for s, p0, n in rs]

    qs, dos = rows(q, qrs), rows(do, qrs)
    ks, vs = rows(k, krs), rows(v, krs)
    p = bd.make_problem(1, L, M, Hq, Hkv, D, torch.bfloat16, out_f32=True)
    QR = [Range(*r) for r in qrs]
    KR = [Range(*r) for r in krs]
    qd, dod = [t.to(DEV) for t in qs], [t.to(DEV) for t in dos]
    kd, vd = [t.to(DEV) for t in ks], [t.to(DEV) for t in vs]
    od = [torch.empty(t.shape, dtype=torch.float32, device=DEV) for t in qd]
    ld = [torch.empty((1, Hq, t.shape[1]), dtype=torch.float32, device=DEV) for t in qd]
    bd.attn_fwd(p, QR, qd, od, ld, KR, kd, vd)
    dqd = [torch.empty(t.shape, dtype=torch.float32, device=DEV) for t in qd]
    dkd = [torch.empty(t.shape, dtype=torch.float32, device=DEV) for t in kd]
    dvd = [torch.empty(t.shape, dtype=torch.float32, device=DEV) for t in vd]
    ws = torch.empty(bd.attn_bwd_workspace_bytes(p, QR), dtype=torch.uint8, device=DEV)
    bd.attn_bwd(p, QR, qd, od, ld, dod, dqd, KR, kd, vd, dkd, dvd, ws)
    torch.cuda.synchronize()

    qall, doall = torch.cat(qs, dim=1), torch.cat(dos, dim=1)
    kall, vall = torch.cat(ks, dim=1), torch.cat(vs, dim=1)
    O, LSE = oracle.fwd(qall, kall, vall, qrs, krs, M)
    dQ, dK, dV = oracle.bwd(qall, kall, vall, O, LSE, doall, qrs, krs, M)
    assert_close(f"{split} O", torch.cat([t.cpu() for t in od], dim=1), O, torch.bfloat16)
    assert_close(f"{split} LSE", torch.cat([t.cpu() for t in ld], dim=2), LSE, torch.bfloat16)
    assert_close(f"{split} dQ", torch.cat([t.cpu() for t in dqd], dim=1), dQ, torch.bfloat16)
    assert_close(f"{split} dK", torch.cat([t.cpu() for t in dkd], dim=1), dK, torch.bfloat16)
    assert_close(f"{split} dV", torch.cat([t.cpu() for t in dvd], dim=1), dV, torch.bfloat16)


@pytest.mark.parametrize("layout", ["gap", "gap-reversed", "offset"])
def test_two_query_ranges_with_apart_spans(layout):
    """Two query ranges whose visible 32-row blocks for a key tile do not nest:
    for the clean key tile at 128 the spans are blocks [0, 2) and [4, 10) with a
    gap between them, in either range order, and in "offset" [2, 4) and [5, 7).
    Head_dim 128, bf16, an even GQA group and two query ranges: the backward runs
    the scheduled dK/dV kernel, whose walk over such spans has its own segments
    (walk_plan); checked against the oracle over the same ranges."""
    Hq, Hkv, D = 8, 2, 128
    L, M = 300, 12
    q, k, v, do = joint_inputs(L, Hq, Hkv, D, torch.bfloat16, seed=77)
    qrs = {"gap": [(CLEAN, 120, 60), (CORRUPTED, 0, 300)],
           "gap-reversed": [(CORRUPTED, 0, 300), (CLEAN, 120, 60)],
           "offset": [(CLEAN, 180, 120), (CORRUPTED, 100, 200)]}[layout]
    krs = [(CLEAN, 0, 300), (CORRUPTED, 0, 300)]

    def rows(t, rs):  # joint tensors hold corrupted rows [0, L) then clean rows [L, 2L)
        return [t[:, (L if s == CLEAN else 0) + p0:(L if s == CLEAN else 0) + p0 + n].contiguous() for s, p0, n in rs]

    qs, dos = rows(q, qrs), rows(do, qrs)
    ks, vs = rows(k, krs), rows(v, krs)
    p = bd.make_problem(1, L, M, Hq, Hkv, D, torch.bfloat16, out_f32=True)
    QR = [Range(*r) for r in qrs]
    KR = [Range(*r) for r in krs]
    qd, dod = [t.to(DEV) for t in qs], [t.to(DEV) for t in dos]
    kd, vd = [t.to(DEV) for t in ks], [t.to(DEV) for t in vs]
    od = [torch.empty(t.shape, dtype=torch.float32, device=DEV) for t in qd]
    ld = [torch.empty((1, Hq, t.shape[1]), dtype=torch.float32, device=DEV) for t in qd]
    bd.attn_fwd(p, QR, qd, od, ld, KR, kd, vd)
    dqd = [torch.empty(t.shape, dtype=torch.float32, device=DEV) for t in qd]
    dkd = [torch.empty(t.shape, dtype=torch.float32, device=DEV) for t in kd]
    dvd = [torch.empty(t.shape, dtype=torch.float32, device=DEV) for t in vd]
    ws = torch.empty(bd.attn_bwd_workspace_bytes(p, QR), dtype=torch.uint8, device=DEV)
    bd.attn_bwd(p, QR, qd, od, ld, dod, dqd, KR, kd, vd, dkd, dvd, ws)
    torch.cuda.synchronize()

    qall, doall = torch.cat(qs, dim=1), torch.cat(dos, dim=1)
    kall, vall = torch.cat(ks, dim=1), torch.cat(vs, dim=1)
    O, LSE = oracle.fwd(qall, kall, vall, qrs, krs, M)
    dQ, dK, dV = oracle.bwd(qall, kall, vall, O, LSE, doall, qrs, krs, M)
    assert_close(f"{layout} O", torch.cat([t.cpu() for t in od], dim=1), O, torch.bfloat16)
    assert_close(f"{layout} dQ", torch.cat([t.cpu() for t in dqd], dim=1), dQ, torch.bfloat16)
    assert_close(f"{layout} dK", torch.cat([t.cpu() for t in dkd], dim=1), dK, torch.bfloat16)
    assert_close(f"{layout} dV", torch.cat([t.cpu() for t in dvd], dim=1), dV, torch.bfloat16)


# ---------------------------------------------------------- degenerate calls
def test_degenerate_ranges():
    """Zero-length query and key ranges next to ordinary ones change nothing
    (bit for bit); a key range no query sees gets dK = dV = 0 exactly; a call
    whose only query range is empty writes nothing."""
    L, M, Hq, Hkv, D = 256, 16, 4, 2, 128
    q, k, v, do = joint_inputs(L, Hq, Hkv, D, torch.bfloat16, seed=61)
    qd, kd, vd, dod = (t.to(DEV) for t in (q, k, v, do))
    o_ref, lse_ref = bd.joint_fwd(qd, kd, vd, M, out_f32=True)
    dq_ref, dk_ref, dv_ref = bd.joint_bwd(qd, kd, vd, o_ref, lse_ref, dod, M, out_f32=True)

    p = bd.make_problem(1, L, M, Hq, Hkv, D, torch.bfloat16, out_f32=True)
    half = lambda t, s: t[:, (L if s == CLEAN else 0):(L if s == CLEAN else 0) + L].contiguous()
    dummy_q = torch.zeros((1, 1, Hq, D), dtype=torch.bfloat16, device=DEV)
    dummy_kv = torch.zeros((1, 1, Hkv, D), dtype=torch.bfloat16, device=DEV)
    # Same range order as the joint call (the order of ranges is the order of
    # accumulation), with an empty range between the two.
    QR = [Range(CORRUPTED, 0, L), Range(CLEAN, 100, 0), Range(CLEAN, 0, L)]
    KR = [Range(CORRUPTED, 0, L), Range(CORRUPTED, 50, 0), Range(CLEAN, 0, L)]
    qs = [half(qd, CORRUPTED), dummy_q, half(qd, CLEAN)]
    dos = [half(dod, CORRUPTED), dummy_q, half(dod, CLEAN)]
    ks = [half(kd, CORRUPTED), dummy_kv, half(kd, CLEAN)]
    vs = [half(vd, CORRUPTED), dummy_kv, half(vd, CLEAN)]
    os_ = [torch.empty(t.shape, dtype=torch.float32, device=DEV) for t in qs]
    ls = [torch.empty((1, Hq, t.shape[1]), dtype=torch.float32, device=DEV) for t in qs]
    bd.attn_fwd(p, QR, qs, os_, ls, KR, ks, vs)
    dqs = [torch.empty(t.shape, dtype=torch.float32, device=DEV) for t in qs]
    dks = [torch.empty(t.shape, dtype=torch.float32, device=DEV) for t in ks]
    dvs = [torch.empty(t.shape, dtype=torch.float32, device=DEV) for t in vs]
    ws = torch.empty(bd.attn_bwd_workspace_bytes(p, QR), dtype=torch.uint8, device=DEV)
    bd.attn_bwd(p, QR, qs, os_, ls, dos, dqs, KR, ks, vs, dks, dvs, ws)
    torch.cuda.synchronize()
    assert torch.equal(os_[0], o_ref[:, :L]) and torch.equal(os_[2], o_ref[:, L:])
    assert torch.equal(ls[0], lse_ref[:, :, :L]) and torch.equal(ls[2], lse_ref[:, :, L:])
    assert torch.equal(dqs[0], dq_ref[:, :L]) and torch.equal(dqs[2], dq_ref[:, L:])
    assert torch.equal(dks[0], dk_ref[:, :L]) and torch.equal(dks[2], dk_ref[:, L:])
    assert torch.equal(dvs[0], dv_ref[:, :L]) and torch.equal(dvs[2], dv_ref[:, L:])

    # clean queries only: the corrupted key range is seen by no query
    QR2 = [Range(CLEAN, 0, L)]
    KR2 = [Range(CLEAN, 0, L), Range(CORRUPTED, 0, L)]  # ks[2], ks[0] below
    o2 = torch.empty(qs[2].shape, dtype=torch.float32, device=DEV)
    l2 = torch.empty((1, Hq, L), dtype=torch.float32, device=DEV)
    bd.attn_fwd(p, QR2, [qs[2]], [o2], [l2], KR2, [ks[2], ks[0]], [vs[2], vs[0]])
    dq2 = torch.empty(qs[2].shape, dtype=torch.float32, device=DEV)
    dk2 = [torch.full(t.shape, 5.0, dtype=torch.float32, device=DEV) for t in (ks[2], ks[0])]
    dv2 = [torch.full(t.shape, 5.0, dtype=torch.float32, device=DEV) for t in (vs[2], vs[0])]
    ws2 = torch.empty(bd.attn_bwd_workspace_bytes(p, QR2), dtype=torch.uint8, device=DEV)
    bd.attn_bwd(p, QR2, [qs[2]], [o2], [l2], [dos[2]], [dq2], KR2, [ks[2], ks[0]], [vs[2], vs[0]], dk2, dv2, ws2)
    torch.cuda.synchronize()
    assert (dk2[1] == 0).all() and (dv2[1] == 0).all()
    O, LSE = oracle.fwd(q[:, L:], k[:, L:], v[:, L:], [(CLEAN, 0, L)], [(CLEAN, 0, L)], M)
    assert_close("clean-only O", o2, O, torch.bfloat16)

    # a call whose only query range is empty writes nothing
    sentinel = torch.full((1, 1, Hq, D), 3.0, dtype=torch.float32, device=DEV)
    lsent = torch.full((1, Hq, 1), 3.0, dtype=torch.float32, device=DEV)
    bd.attn_fwd(p, [Range(CLEAN, 0, 0)], [dummy_q], [sentinel], [lsent], KR2, [ks[2], ks[0]], [vs[2], vs[0]])
    torch.cuda.synchronize()
    assert (sentinel == 3.0).all() and (lsent == 3.0).all()


# ------------------------------------------ strided ranges, poisoned padding
@pytest.mark.parametrize("dt", ["bf16", "fp32"])
def test_strided_ranges_poisoned_padding(dt):
    """Ranges stored with batch_stride > len (batch 2) whose padding rows hold
    NaN in every input: results match the oracle on the dense data (no padding
    row is ever used), and the padding rows of every output (O, LSE, dQ, dK,
    dV) keep their sentinel (nothing is written outside a range)."""
    L, M, Hq, Hkv, D, B = 300, 12, 4, 2, 128, 2
    SQ, SK = L + 37, L + 21  # row strides of the query-side and key-side tensors
    dtype = torch.float32 if dt == "fp32" else torch.bfloat16
    q, k, v, do = joint_inputs(L, Hq, Hkv, D, dtype, batch=B, seed=71)
    streams = (CORRUPTED, CLEAN)

    def strided(t, s, stride, fill):  # one stream's rows of a joint tensor, padded to `stride` rows
        out = torch.full((B, stride) + tuple(t.shape[2:]), fill, dtype=t.dtype)
        out[:, :L] = t[:, (L if s == CLEAN else 0):(L if s == CLEAN else 0) + L]
        return out.to(DEV)

    nan = float("nan")
    QR = [Range(s, 0, L, SQ) for s in streams]
    KR = [Range(s, 0, L, SK) for s in streams]
    qs = [strided(q, s, SQ, nan) for s in streams]
    dos = [strided(do, s, SQ, nan) for s in streams]
    ks = [strided(k, s, SK, nan) for s in streams]
    vs = [strided(v, s, SK, nan) for s in streams]
    SENT = 7.0
    os_ = [torch.full((B, SQ, Hq, D), SENT, dtype=torch.float32, device=DEV) for _ in streams]
    ls = [torch.full((B, Hq, SQ), SENT, dtype=torch.float32, device=DEV) for _ in streams]
    p = bd.make_problem(B, L, M, Hq, Hkv, D, dtype, out_f32=True)
    bd.attn_fwd(p, QR, qs, os_, ls, KR, ks, vs)
    dqs = [torch.full((B, SQ, Hq, D), SENT, dtype=torch.float32, device=DEV) for _ in streams]
    dks = [torch.full((B, SK, Hkv, D), SENT, dtype=torch.float32, device=DEV) for _ in streams]
    dvs = [torch.full((B, SK, Hkv, D), SENT, dtype=torch.float32, device=DEV) for _ in streams]
    ws = torch.empty(bd.attn_bwd_workspace_bytes(p, QR), dtype=torch.uint8, device=DEV)
    bd.attn_bwd(p, QR, qs, os_, ls, dos, dqs, KR, ks, vs, dks, dvs, ws)
    torch.cuda.synchronize()

    for t in os_ + dqs + dks + dvs:
        assert (t[:, L:] == SENT).all(), "a padding row was written"
    for t in ls:
        assert (t[:, :, L:] == SENT).all(), "a padding LSE entry was written"
    joint = lambda ts: torch.cat([t[:, :L].cpu() for t in ts], dim=1)
    O, LSE = oracle.joint_fwd(q, k, v, L, M)
    dQ, dK, dV = oracle.joint_bwd(q, k, v, O, LSE, do, L, M)
    assert_close(f"{dt} strided O", joint(os_), O, dtype)
    assert_close(f"{dt} strided LSE", torch.cat([t[:, :, :L].cpu() for t in ls], dim=2), LSE, dtype)
    assert_close(f"{dt} strided dQ", joint(dqs), dQ, dtype)
    assert_close(f"{dt} strided dK", joint(dks), dK, dtype)
    assert_close(f"{dt} strided dV", joint(dvs), dV, dtype)


# ------------------------------------------------------------- side stream
def test_calls_run_on_the_given_stream():
    """Every entry point enqueues on the stream it is given: a forward and
    backward on a side stream (default priority), synchronised through that
    stream alone, equal the same calls on the current stream bit for bit, and
    the timing hooks record their kernels."""
    L, M, Hq, Hkv, D = 320, 16, 4, 2, 128
    q, k, v, do = joint_inputs(L, Hq, Hkv, D, torch.bfloat16, seed=83)
    qd, kd, vd, dod = (t.to(DEV) for t in (q, k, v, do))
    o_ref, lse_ref = bd.joint_fwd(qd, kd, vd, M, out_f32=True)
    dq_ref, dk_ref, dv_ref = bd.joint_bwd(qd, kd, vd, o_ref, lse_ref, dod, M, out_f32=True)
    torch.cuda.synchronize()

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        o = torch.empty(qd.shape, dtype=torch.float32, device=DEV)
        lse = torch.empty(lse_ref.shape, dtype=torch.float32, device=DEV)
        grads = tuple(torch.empty(t.shape, dtype=torch.float32, device=DEV) for t in (qd, kd, vd))
        p = bd.make_problem(1, L, M, Hq, Hkv, D, torch.bfloat16)
        ws = torch.empty(bd.attn_bwd_workspace_bytes(p, bd.joint_ranges(L)), dtype=torch.uint8, device=DEV)
    bd.timing_enable(True)
    bd.joint_fwd(qd, kd, vd, M, out_f32=True, out=(o, lse), stream=side)
    bd.joint_bwd(qd, kd, vd, o, lse, dod, M, out_f32=True, out=grads, workspace=ws, stream=side)
    side.synchronize()
    recs = bd.timing_collect()
    bd.timing_enable(False)
    assert [n for n, _ in recs] == ["fwd_bf16", "bwd_dq_bf16", "bwd_dkdv_bf16"], recs
    assert all(ms > 0 for _, ms in recs)
    assert torch.equal(o, o_ref) and torch.equal(lse, lse_ref)
    for a, b in zip(grads, (dq_ref, dk_ref, dv_ref)):
        assert torch.equal(a, b)


# ------------------------------------------------------- head_dim 64, more tiles
@pytest.mark.parametrize("reading", [0, 1], ids=["causal", "block"])
def test_medium_head_dim_64(reading):
    """head_dim 64 over many tiles: batch 2, L = 2,048 + 2,048, block 32, 16/4
    heads (the d = 64 kernels otherwise meet only the small shapes); query
    heads of KV groups {0, 3} against the oracle."""
    L, M, Hq, Hkv, D, B = 2048, 32, 16, 4, 64, 2
    q, k, v, do = joint_inputs(L, Hq, Hkv, D, torch.bfloat16, batch=B, seed=97 + reading)
    check_joint(q, k, v, do, M, reading, torch.bfloat16, heads=kv_group_heads(Hq, Hkv, [0, Hkv - 1]),
                tag=f"d64 L{L} r{reading}")


# ------------------------------------------------------- the call-size limits
@pytest.mark.parametrize("D", [64, 128])
def test_merge_max_parts(D):
    """A merge of the maximum 32 partials (head_dim 64: per-lane LSE loads;
    128: the two-register lane broadcast of parts 0-15 and 16-31), with empty
    parts per row, bf16 and fp32 partials, against the oracle's merge."""
    g = torch.Generator().manual_seed(5 + D)
    B, R, H, J = 1, 45, 2, bd.MAX_MERGE_PARTS
    os_ = [torch.randn(B, R, H, D, generator=g) for _ in range(J)]
    ls = [torch.randn(B, H, R, generator=g) * 3 for _ in range(J)]
    for j in range(J):
        ls[j][torch.rand(B, H, R, generator=g) < 0.4] = -float("inf")
    ls[J - 1][:, :, 7] = 9.0  # a row dominated by the last part
    for j in range(J):
        os_[j] = torch.where(torch.isneginf(ls[j]).transpose(1, 2)[..., None], torch.zeros(()), os_[j]).contiguous()
    for pdt in (torch.float32, torch.bfloat16):
        od = [t.to(pdt).to(DEV) for t in os_]
        ld = [t.to(DEV) for t in ls]
        o = torch.empty(B, R, H, D, dtype=torch.float32, device=DEV)
        lse = torch.empty(B, H, R, dtype=torch.float32, device=DEV)
        bd.lse_merge(od, ld, o, lse)
        torch.cuda.synchronize()
        Or, Lr = oracle.lse_merge([t.to(pdt) for t in os_], ls)
        tol = torch.float32 if pdt == torch.float32 else torch.bfloat16
        assert_close(f"merge J{J} d{D} {pdt} O", o, Or, tol)
        assert_close(f"merge J{J} d{D} {pdt} LSE", lse, Lr, tol)


def test_max_query_and_key_ranges():
    """The largest call: 4 query ranges and 32 key ranges (the clean stream cut
    into 31 uneven pieces, each its own tensor), forward and backward in one
    call each, against the oracle over the same ranges."""
    L, M, Hq, Hkv, D = 640, 16, 4, 2, 128
    q, k, v, do = joint_inputs(L, Hq, Hkv, D, torch.bfloat16, seed=101)
    cuts = sorted(set([0, L] + np.random.default_rng(7).choice(np.arange(1, L), size=30, replace=False).tolist()))
    assert len(cuts) == 32
    krs = [(CORRUPTED, 0, L)] + [(CLEAN, a, b - a) for a, b in zip(cuts[:-1], cuts[1:])]
    qrs = [(CLEAN, 300, 340), (CORRUPTED, 0, 333), (CLEAN, 0, 300), (CORRUPTED, 333, 307)]
    assert len(krs) == bd.MAX_K_RANGES and len(qrs) == bd.MAX_Q_RANGES

    def rows(t, rs):
        return [t[:, (L if s == CLEAN else 0) + p0:(L if s == CLEAN else 0) + p0 + n].contiguous() for s, p0, n in rs]

    qs, dos, ks, vs = rows(q, qrs), rows(do, qrs), rows(k, krs), rows(v, krs)
    p = bd.make_problem(1, L, M, Hq, Hkv, D, torch.bfloat16, out_f32=True)
    QR, KR = [Range(*r) for r in qrs], [Range(*r) for r in krs]
    qd, dod = [t.to(DEV) for t in qs], [t.to(DEV) for t in dos]
    kd, vd = [t.to(DEV) for t in ks], [t.to(DEV) for t in vs]
    od = [torch.empty(t.shape, dtype=torch.float32, device=DEV) for t in qd]
    ld = [torch.empty((1, Hq, t.shape[1]), dtype=torch.float32, device=DEV) for t in qd]
    bd.attn_fwd(p, QR, qd, od, ld, KR, kd, vd)
    dqd = [torch.empty(t.shape, dtype=torch.float32, device=DEV) for t in qd]
    dkd = [torch.empty(t.shape, dtype=torch.float32, device=DEV) for t in kd]
    dvd = [torch.empty(t.shape, dtype=torch.float32, device=DEV) for t in vd]
    ws = torch.empty(bd.attn_bwd_workspace_bytes(p, QR), dtype=torch.uint8, device=DEV)
    bd.attn_bwd(p, QR, qd, od, ld, dod, dqd, KR, kd, vd, dkd, dvd, ws)
    torch.cuda.synchronize()
    qall, doall = torch.cat(qs, dim=1), torch.cat(dos, dim=1)
    kall, vall = torch.cat(ks, dim=1), torch.cat(vs, dim=1)
    O, LSE = oracle.fwd(qall, kall, vall, qrs, krs, M)
    dQ, dK, dV = oracle.bwd(qall, kall, vall, O, LSE, doall, qrs, krs, M)
    cat1 = lambda ts: torch.cat([t.cpu() for t in ts], dim=1)
    assert_close("max ranges O", cat1(od), O, torch.bfloat16)
    assert_close("max ranges LSE", torch.cat([t.cpu() for t in ld], dim=2), LSE, torch.bfloat16)
    assert_close("max ranges dQ", cat1(dqd), dQ, torch.bfloat16)
    assert_close("max ranges dK", cat1(dkd), dK, torch.bfloat16)
    assert_close("max ranges dV", cat1(dvd), dV, torch.bfloat16)
