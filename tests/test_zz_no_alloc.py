"""bdlm_attn_bwd_noalloc (the backward without a workspace argument) against
bdlm_attn_bwd, through the C ABI: identical results on two calls in a row, the
second smaller than the first (the scratch array keeps the first call's
contents).  The rejection of calls beyond the array's size is a host test
(tests/test_abi_host.py)."""
import pytest
import torch

import paper_2609_19242_amd as bd
from tests.gpu_util import joint_inputs

pytestmark = pytest.mark.gpu
DEV = "cuda"


def run_both(L, M, Hq, Hkv, D, batch, seed, out_f32):
    q, k, v, do = (t.to(DEV) for t in joint_inputs(L, Hq, Hkv, D, torch.bfloat16, batch=batch, seed=seed))
    o, lse = bd.joint_fwd(q, k, v, M, out_f32=out_f32)
    p = bd.make_problem(batch, L, M, Hq, Hkv, D, torch.bfloat16, out_f32=out_f32)
    r = bd.joint_ranges(L)
    odt = torch.float32 if out_f32 else torch.bfloat16
    grads = [tuple(torch.full(t.shape, float("nan"), dtype=odt, device=DEV) for t in (q, k, v)) for _ in range(2)]
    ws = torch.empty(bd.attn_bwd_workspace_bytes(p, r), dtype=torch.uint8, device=DEV)
    halves = lambda t: bd._joint_ptrs(t, L)  # noqa: E731
    lp = [lse.data_ptr(), lse.data_ptr() + L * 4]
    args = [halves(q), halves(o), lp, halves(do)]
    (dq0, dk0, dv0), (dq1, dk1, dv1) = grads
    bd.attn_bwd(p, r, *args, halves(dq0), r, halves(k), halves(v), halves(dk0), halves(dv0), ws)
    bd.attn_bwd_noalloc(p, r, *args, halves(dq1), r, halves(k), halves(v), halves(dk1), halves(dv1))
    torch.cuda.synchronize()
    for name, a, b in (("dq", dq0, dq1), ("dk", dk0, dk1), ("dv", dv0, dv1)):
        assert torch.isfinite(a).all(), name
        assert torch.equal(a, b), f"{name}: max diff {(a.float() - b.float()).abs().max().item()}"
    print(f"L={L} batch={batch} {Hq}/{Hkv} heads: noalloc == workspace call (scratch bytes used "
          f"{bd.attn_bwd_workspace_bytes(p, r)})", flush=True)


def test_noalloc_matches_workspace_call_twice_smaller_second():
    run_both(1536, 32, 8, 2, 128, batch=2, seed=31, out_f32=False)
    run_both(320, 16, 4, 2, 64, batch=1, seed=37, out_f32=True)
