"""The bf16 forward and dQ kernels take 128-row query tiles (4 waves, two
workgroups per CU) when no row of a call can see many keys and 256-row tiles
(8 waves) otherwise, chosen from the longest key range of the call.  A row's
arithmetic does not depend on the tile height, so the same rows give the same
bits under either: here a long clean key range that no query can see (it lies
past every query's clean context) is added to a call, which moves the forward,
the dQ kernel or both to 256-row tiles; O, LSE, dQ, dK and dV of the other
ranges must not change in any bit, and the unseen keys get dK = dV = 0.  The
call without the extra range is checked against the oracle.
"""
import pytest
import torch

import oracle
import paper_2609_19242_amd as bd
import synth
from paper_2609_19242_amd import CLEAN, CORRUPTED, Range
from tests.gpu_util import assert_close, joint_inputs

pytestmark = pytest.mark.gpu
DEV = "cuda"
L, M, HQ, HKV, D, N = 40000, 16, 8, 2, 128, 600
FAR = 20000  # first clean position of the unseen key range (every query sits below position N)


def call(qs, dos, ks, vs, qrs, krs):
    p = bd.make_problem(1, L, M, HQ, HKV, D, torch.bfloat16, out_f32=True)
    QR, KR = [Range(*r) for r in qrs], [Range(*r) for r in krs]
    od = [torch.full(t.shape, float("nan"), dtype=torch.float32, device=DEV) for t in qs]
    ld = [torch.full((1, HQ, t.shape[1]), float("nan"), dtype=torch.float32, device=DEV) for t in qs]
    bd.attn_fwd(p, QR, qs, od, ld, KR, ks, vs)
    dqd = [torch.full(t.shape, float("nan"), dtype=torch.float32, device=DEV) for t in qs]
    dkd = [torch.full(t.shape, float("nan"), dtype=torch.float32, device=DEV) for t in ks]
    dvd = [torch.full(t.shape, float("nan"), dtype=torch.float32, device=DEV) for t in vs]
    ws = torch.empty(bd.attn_bwd_workspace_bytes(p, QR), dtype=torch.uint8, device=DEV)
    bd.attn_bwd(p, QR, qs, od, ld, dos, dqd, KR, ks, vs, dkd, dvd, ws)
    torch.cuda.synchronize()
    return od, ld, dqd, dkd, dvd


@pytest.fixture(scope="module")
def base():
    q, k, v, do = joint_inputs(N, HQ, HKV, D, torch.bfloat16, seed=91)
    qrs = [(CLEAN, 0, N), (CORRUPTED, 0, N)]
    krs = [(CLEAN, 0, N), (CORRUPTED, 0, N)]

    def rows(t, rs):  # joint tensors of length N hold corrupted rows [0, N) then clean rows [N, 2N)
        return [t[:, (N if s == CLEAN else 0) + p0:(N if s == CLEAN else 0) + p0 + n].contiguous() for s, p0, n in rs]

    qs, dos, ks, vs = rows(q, qrs), rows(do, qrs), rows(k, krs), rows(v, krs)
    dev = lambda ts: [t.to(DEV) for t in ts]  # noqa: E731
    inp = dict(qs=dev(qs), dos=dev(dos), ks=dev(ks), vs=dev(vs), qrs=qrs, krs=krs)
    out = call(**inp)
    return inp, out, (qs, dos, ks, vs)


def test_short_tiles_against_the_oracle(base):
    inp, (od, ld, dqd, dkd, dvd), (qs, dos, ks, vs) = base
    qall, doall = torch.cat(qs, dim=1), torch.cat(dos, dim=1)
    kall, vall = torch.cat(ks, dim=1), torch.cat(vs, dim=1)
    O, LSE = oracle.fwd(qall, kall, vall, inp["qrs"], inp["krs"], M)
    dQ, dK, dV = oracle.bwd(qall, kall, vall, O, LSE, doall, inp["qrs"], inp["krs"], M)
    assert_close("O", torch.cat([t.cpu() for t in od], dim=1), O, torch.bfloat16)
    assert_close("dQ", torch.cat([t.cpu() for t in dqd], dim=1), dQ, torch.bfloat16)
    assert_close("dK", torch.cat([t.cpu() for t in dkd], dim=1), dK, torch.bfloat16)
    assert_close("dV", torch.cat([t.cpu() for t in dvd], dim=1), dV, torch.bfloat16)


# 10,000 unseen keys: 128-row forward, 256-row dQ; 16,500: 256 rows for both.
@pytest.mark.parametrize("extra", [10000, 16500])
def test_tile_height_changes_no_bit(base, extra):
    inp, ref, _ = base
    k_far = synth.normal((1, extra, HKV, D), 93, torch.bfloat16).to(DEV)
    v_far = synth.normal((1, extra, HKV, D), 94, torch.bfloat16).to(DEV)
    od, ld, dqd, dkd, dvd = call(inp["qs"], inp["dos"], inp["ks"] + [k_far], inp["vs"] + [v_far], inp["qrs"],
                                 inp["krs"] + [(CLEAN, FAR, extra)])
    for name, got, want in (("O", od, ref[0]), ("LSE", ld, ref[1]), ("dQ", dqd, ref[2]),
                            ("dK", dkd[:2], ref[3]), ("dV", dvd[:2], ref[4])):
        for i, (g, w) in enumerate(zip(got, want)):
            assert torch.equal(g, w), f"{name}[{i}] with {extra} unseen keys: " \
                f"max diff {(g - w).abs().max().item()}"
    assert torch.count_nonzero(dkd[2]).item() == 0 and torch.count_nonzero(dvd[2]).item() == 0
    print(f"{extra} unseen keys: O, LSE, dQ, dK, dV bit-identical; unseen dK = dV = 0", flush=True)
