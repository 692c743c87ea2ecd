"""The Python binding rejects tensors of the wrong dtype, shape, layout or device
before any pointer reaches the C ABI (a bf16 buffer given where the kernels
write fp32, or a non-contiguous gradient, would otherwise be written past its
end or read wrong).  Host only: every call here fails validation first."""
import pytest
import torch

import paper_2609_19242_amd as bd

B, L, HQ, HKV, D = 1, 32, 4, 2, 64
N = 2 * L


def joint(dtype=torch.bfloat16):
    q = torch.zeros(B, N, HQ, D, dtype=dtype)
    k = torch.zeros(B, N, HKV, D, dtype=dtype)
    v = torch.zeros(B, N, HKV, D, dtype=dtype)
    return q, k, v


def lse_ok():
    return torch.zeros(B, HQ, N, dtype=torch.float32)


def test_fwd_rejects_out_of_wrong_dtype():
    q, k, v = joint()
    with pytest.raises(TypeError, match="o must be torch.float32"):
        bd.joint_fwd(q, k, v, 16, out_f32=True, out=(torch.zeros_like(q), lse_ok()))
    with pytest.raises(TypeError, match="o must be torch.bfloat16"):
        bd.joint_fwd(q, k, v, 16, out=(torch.zeros(q.shape), lse_ok()))


def test_fwd_rejects_lse_of_wrong_layout_or_dtype():
    q, k, v = joint()
    with pytest.raises(ValueError, match="lse must have shape"):
        bd.joint_fwd(q, k, v, 16, out=(torch.zeros_like(q), torch.zeros(B, N, HQ)))
    with pytest.raises(TypeError, match="lse must be torch.float32"):
        bd.joint_fwd(q, k, v, 16, out=(torch.zeros_like(q), lse_ok().double()))


def test_fwd_rejects_bad_inputs():
    q, k, v = joint()
    with pytest.raises(ValueError, match="q must be"):
        bd.joint_fwd(q[:, :N - 1], k, v, 16)
    with pytest.raises(TypeError, match="k must be torch.bfloat16"):
        bd.joint_fwd(q, k.float(), v, 16)
    with pytest.raises(ValueError, match="v must have shape"):
        bd.joint_fwd(q, k, v[:, :, :1], 16)
    with pytest.raises(ValueError, match="k must be contiguous"):
        bd.joint_fwd(q, k.transpose(2, 3).contiguous().transpose(2, 3), v, 16)
    with pytest.raises(TypeError, match="unsupported dtype"):
        bd.joint_fwd(q.half(), k.half(), v.half(), 16)


def test_fwd_rejects_host_tensors():
    q, k, v = joint()
    with pytest.raises(ValueError, match="must be on"):
        bd.joint_fwd(q, k, v, 16)


def test_bwd_rejects_o_lse_do_of_wrong_kind():
    q, k, v = joint()
    o, do = torch.zeros_like(q), torch.zeros_like(q)
    with pytest.raises(TypeError, match="o must be torch.float32"):
        bd.joint_bwd(q, k, v, o, lse_ok(), do, 16, out_f32=True)
    with pytest.raises(ValueError, match="lse must have shape"):
        bd.joint_bwd(q, k, v, o, torch.zeros(B, N, HQ), do, 16)
    with pytest.raises(TypeError, match="do must be torch.bfloat16"):
        bd.joint_bwd(q, k, v, o, lse_ok(), do.float(), 16)
    qf, kf, vf = joint(torch.float32)
    with pytest.raises(TypeError, match="do must be torch.float32"):
        bd.joint_bwd(qf, kf, vf, torch.zeros_like(qf), lse_ok(), do, 16)
    strided = torch.zeros(B, N, HQ, 2 * D, dtype=torch.bfloat16)[..., :D]
    with pytest.raises(ValueError, match="do must be contiguous"):
        bd.joint_bwd(q, k, v, o, lse_ok(), strided, 16)


def test_bwd_rejects_gradient_outputs_of_wrong_kind():
    q, k, v = joint()
    o, do = torch.zeros_like(q), torch.zeros_like(q)
    good = (torch.zeros_like(q), torch.zeros_like(k), torch.zeros_like(v))
    with pytest.raises(TypeError, match="dk must be torch.float32"):
        bd.joint_bwd(q, k, v, o.float(), lse_ok(), do, 16, out_f32=True,
                     out=(good[0].float(), good[1], good[2].float()))
    with pytest.raises(ValueError, match="dv must have shape"):
        bd.joint_bwd(q, k, v, o, lse_ok(), do, 16, out=(good[0], good[1], torch.zeros_like(q)))
    with pytest.raises(ValueError, match="out must be"):
        bd.joint_bwd(q, k, v, o, lse_ok(), do, 16, out=good[:2])
    with pytest.raises(ValueError, match="must be on"):
        bd.joint_bwd(q, k, v, o, lse_ok(), do, 16, out=good)


def test_merge_rejects_mismatched_parts():
    o = torch.zeros(B, 8, HQ, D, dtype=torch.bfloat16)
    lse = torch.zeros(B, HQ, 8)
    parts = [torch.zeros_like(o), torch.zeros_like(o)]
    with pytest.raises(ValueError, match="one LSE per partial"):
        bd.lse_merge(parts, [lse], o, lse.clone())
    with pytest.raises(ValueError, match=r"o_parts\[1\] must have shape"):
        bd.lse_merge([parts[0], torch.zeros(B, 9, HQ, D, dtype=torch.bfloat16)], [lse, lse], o, lse.clone())
    with pytest.raises(TypeError, match=r"o_parts\[1\] must be torch.bfloat16"):
        bd.lse_merge([parts[0], parts[1].float()], [lse, lse], o, lse.clone())
    with pytest.raises(ValueError, match=r"lse_parts\[0\] must have shape"):
        bd.lse_merge(parts, [torch.zeros(B, 8, HQ), lse], o, lse.clone())
    with pytest.raises(ValueError, match="must be on"):
        bd.lse_merge(parts, [lse, lse.clone()], o, lse.clone())


def test_merge_takes_row_packed_views_with_a_batch_stride():
    # one range's half of joint outputs [2][2R][H][D] / [2][H][2R]: accepted up to the device check
    R = 8
    jo = torch.zeros(2, 2 * R, HQ, D, dtype=torch.bfloat16)
    jl = torch.zeros(2, HQ, 2 * R)
    o, lse = torch.zeros(2, R, HQ, D, dtype=torch.bfloat16), torch.zeros(2, HQ, R)
    with pytest.raises(ValueError, match="must be on"):
        bd.lse_merge([jo[:, R:], jo[:, :R]], [jl[:, :, R:], jl[:, :, :R]], o, lse)
    with pytest.raises(ValueError, match="must be on"):
        bd.lse_merge([torch.zeros_like(o)], [torch.zeros_like(lse)], jo[:, :R], jl[:, :, :R])
    # not row-packed: heads and rows swapped, every other row
    with pytest.raises(ValueError, match="rows packed"):
        bd.lse_merge([torch.zeros(2, HQ, R, D, dtype=torch.bfloat16).transpose(1, 2)], [jl[:, :, R:]], o, lse)
    with pytest.raises(ValueError, match="rows packed"):
        bd.lse_merge([jo[:, ::2]], [jl[:, :, ::2]], o, lse)
    # parts with different batch strides, o and lse with different ones
    with pytest.raises(ValueError, match="share one batch stride"):
        bd.lse_merge([jo[:, R:], torch.zeros_like(o)], [jl[:, :, R:], torch.zeros_like(lse)], o, lse)
    with pytest.raises(ValueError, match="o and lse must share"):
        bd.lse_merge([torch.zeros_like(o)], [torch.zeros_like(lse)], jo[:, :R], lse)
