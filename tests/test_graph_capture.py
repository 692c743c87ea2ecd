"""The forward and both backward entry points under HIP graph capture.

The launch paths issue kernels only (no allocation, memset, copy or host
synchronisation), so a caller may record them into a graph.  Each graph here is
replayed several times, on new inputs copied into its static buffers, with
eager work and synchronisations between the replays and the outputs poisoned
with NaN before each replay; every replay must equal the eager call on the same
inputs bit for bit (the kernels are deterministic: no atomics in any result).
"""
import pytest
import torch

import paper_2609_19242_amd as bd
from tests.gpu_util import joint_inputs

pytestmark = pytest.mark.gpu
DEV = "cuda"
L, M, HQ, HKV, D, BATCH = 1536, 32, 8, 2, 128, 2


def eager(q, k, v, do):
    o, lse = bd.joint_fwd(q, k, v, M)
    dq, dk, dv = bd.joint_bwd(q, k, v, o, lse, do, M)
    torch.cuda.synchronize()
    return o, lse, dq, dk, dv


def noalloc_bwd(p, r, q, o, lse, do, k, v, dq, dk, dv):
    halves = lambda t: bd._joint_ptrs(t, L)  # noqa: E731
    lp = [lse.data_ptr(), lse.data_ptr() + L * 4]
    bd.attn_bwd_noalloc(p, r, halves(q), halves(o), lp, halves(do), halves(dq), r, halves(k), halves(v),
                        halves(dk), halves(dv))


def other_work():
    a = torch.randn(1024, 1024, device=DEV)
    return (a @ a).sum().item()


@pytest.mark.parametrize("bwd", ["workspace", "noalloc"])
def test_graph_replays_equal_eager_calls(bwd):
    seeds = (41, 43, 47, 53)
    inputs = [tuple(t.to(DEV) for t in joint_inputs(L, HQ, HKV, D, torch.bfloat16, batch=BATCH, seed=s))
              for s in seeds]
    expect = [eager(*x) for x in inputs]

    q, k, v, do = (t.clone() for t in inputs[0])
    o = torch.empty_like(q)
    lse = torch.empty((BATCH, HQ, 2 * L), dtype=torch.float32, device=DEV)
    grads = tuple(torch.empty_like(t) for t in (q, k, v))
    p = bd.make_problem(BATCH, L, M, HQ, HKV, D, torch.bfloat16)
    r = bd.joint_ranges(L)
    ws = torch.empty(bd.attn_bwd_workspace_bytes(p, r), dtype=torch.uint8, device=DEV)

    def step():
        bd.joint_fwd(q, k, v, M, out=(o, lse))
        if bwd == "workspace":
            bd.joint_bwd(q, k, v, o, lse, do, M, out=grads, workspace=ws)
        else:
            noalloc_bwd(p, r, q, o, lse, do, k, v, *grads)

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step()  # warm-up off the capture (the no-allocation call looks up its scratch address here)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()

    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step()
    torch.cuda.synchronize()

    for rep, idx in enumerate((1, 0, 3, 2, 1)):
        for dst, src in zip((q, k, v, do), inputs[idx]):
            dst.copy_(src)
        for t in (o, lse) + grads:
            t.fill_(float("nan"))
        other_work()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for name, got, want in zip(("o", "lse", "dq", "dk", "dv"), (o, lse) + grads, expect[idx]):
            assert torch.equal(got, want), f"replay {rep} (inputs {idx}) {name}: " \
                f"max diff {(got.float() - want.float()).abs().max().item()}"
        print(f"{bwd}: replay {rep} on inputs {idx} equals the eager call", flush=True)
