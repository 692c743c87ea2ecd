"""MI355X (gfx950) BDLM attention: Python binding of ``libbdlm_attn.so``.

The C ABI (``include/bdlm_attn.h``) does all the work in HIP kernels; this
module only marshals arguments: it builds the ``bdlm_problem`` / ``bdlm_range``
records, passes tensor data pointers and torch's current HIP stream, turns
status codes into exceptions, and allocates outputs with torch.

``torch`` is imported before the library is loaded so that the library binds
to the HIP runtime torch already holds (both carry the soname
``libamdhip64.so.7``).  If the library has not been built, every call raises:
there is no fallback path.
"""
from __future__ import annotations

import ctypes
import math
import os
from typing import List, Optional, Sequence

import torch  # noqa: F401  (load torch's HIP runtime first)

__all__ = [
    "Problem", "Range", "BdlmError", "lib", "library_path",
    "BF16", "F32", "CLEAN", "CORRUPTED", "CLEAN_INTRA_CAUSAL", "CLEAN_INTRA_BLOCK",
    "HILO_PV", "HILO_DKDV", "HILO_DQ", "HILO_ALL", "HILO_ADAPTIVE",
    "make_problem", "joint_ranges", "attn_fwd", "attn_partial_fwd", "lse_merge",
    "attn_bwd_workspace_bytes", "attn_bwd", "attn_bwd_noalloc", "visible_pairs",
    "joint_fwd", "joint_bwd", "timing_enable", "timing_collect", "useful_flops",
]

BF16, F32 = 0, 1
CLEAN, CORRUPTED = 0, 1
CLEAN_INTRA_CAUSAL, CLEAN_INTRA_BLOCK = 0, 1
# bdlm_problem.hilo bits: products that take P or dS as two bf16 terms
HILO_PV, HILO_DKDV, HILO_DQ = 1, 2, 4
HILO_ALL = HILO_PV | HILO_DKDV | HILO_DQ
HILO_ADAPTIVE = 8  # with the bits above: the second term only on tiles holding a probability >= 1/64
MAX_Q_RANGES, MAX_K_RANGES, MAX_MERGE_PARTS = 4, 32, 32
NOALLOC_SCRATCH_BYTES = 64 << 20  # BDLM_NOALLOC_SCRATCH_BYTES

_HERE = os.path.dirname(os.path.abspath(__file__))
# BDLM_LIBRARY points the binding at another build of the same C ABI (e.g. a
# differently tuned one); the default is the in-tree library.
library_path = os.environ.get("BDLM_LIBRARY") or os.path.join(_HERE, "libbdlm_attn.so")


class Problem(ctypes.Structure):
    _fields_ = [
        ("batch", ctypes.c_int64), ("L", ctypes.c_int64), ("block_size", ctypes.c_int64),
        ("heads", ctypes.c_int32), ("kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32),
        ("dtype", ctypes.c_int32), ("scale", ctypes.c_float), ("clean_intra", ctypes.c_int32),
        ("out_f32", ctypes.c_int32), ("hilo", ctypes.c_int32),
        ("window", ctypes.c_int64), ("clean_prefix", ctypes.c_void_p),
    ]


class Range(ctypes.Structure):
    _fields_ = [
        ("stream", ctypes.c_int32), ("reserved", ctypes.c_int32),
        ("pos0", ctypes.c_int64), ("len", ctypes.c_int64), ("batch_stride", ctypes.c_int64),
    ]

    def __init__(self, stream: int, pos0: int, length: int, batch_stride: int = 0):
        super().__init__(stream, 0, pos0, length, batch_stride)

    def __repr__(self):
        s = "CLEAN" if self.stream == CLEAN else "CORRUPTED"
        return f"Range({s}, pos0={self.pos0}, len={self.len}, batch_stride={self.batch_stride})"


class BdlmError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"bdlm status {status}: {msg}")
        self.status = status


_LIB = None
_VP = ctypes.c_void_p
_PP = ctypes.POINTER(ctypes.c_void_p)


def lib() -> ctypes.CDLL:
    """The loaded HIP library; raises if it has not been built."""
    global _LIB
    if _LIB is None:
        if not os.path.exists(library_path):
            raise RuntimeError(f"{library_path} is missing: build it first "
                               "(python -c 'import __graft_entry__ as g; g.build()')")
        L = ctypes.CDLL(library_path)
        L.bdlm_last_error.restype = ctypes.c_char_p
        L.bdlm_attn_fwd.argtypes = [ctypes.POINTER(Problem), ctypes.c_int32, ctypes.POINTER(Range), _PP, _PP, _PP,
                                    ctypes.c_int32, ctypes.POINTER(Range), _PP, _PP, _VP]
        L.bdlm_attn_partial_fwd.argtypes = [ctypes.POINTER(Problem), Range, _VP, _VP, _VP, Range, _VP, _VP, _VP]
        L.bdlm_lse_merge.argtypes = [ctypes.c_int64, ctypes.c_int64, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,
                                     _PP, _PP, ctypes.c_int32, _VP, _VP, ctypes.c_int32, _VP]
        L.bdlm_lse_merge_strided.argtypes = [ctypes.c_int64, ctypes.c_int64, ctypes.c_int32, ctypes.c_int32,
                                             ctypes.c_int32, _PP, _PP, ctypes.c_int32, ctypes.c_int64, _VP, _VP,
                                             ctypes.c_int32, ctypes.c_int64, _VP]
        L.bdlm_attn_bwd_workspace_bytes.argtypes = [ctypes.POINTER(Problem), ctypes.c_int32, ctypes.POINTER(Range)]
        L.bdlm_attn_bwd_workspace_bytes.restype = ctypes.c_size_t
        L.bdlm_attn_bwd.argtypes = [ctypes.POINTER(Problem), ctypes.c_int32, ctypes.POINTER(Range), _PP, _PP, _PP,
                                    _PP, _PP, ctypes.c_int32, ctypes.POINTER(Range), _PP, _PP, _PP, _PP,
                                    _VP, ctypes.c_size_t, _VP]
        L.bdlm_attn_bwd_noalloc.argtypes = [ctypes.POINTER(Problem), ctypes.c_int32, ctypes.POINTER(Range), _PP, _PP,
                                             _PP, _PP, _PP, ctypes.c_int32, ctypes.POINTER(Range), _PP, _PP, _PP, _PP,
                                             _VP]
        L.bdlm_visible_pairs.argtypes = [ctypes.POINTER(Problem), ctypes.c_int32, ctypes.POINTER(Range),
                                         ctypes.c_int32, ctypes.POINTER(Range)]
        L.bdlm_visible_pairs.restype = ctypes.c_int64
        L.bdlm_timing_enable.argtypes = [ctypes.c_int32]
        L.bdlm_timing_enable.restype = ctypes.c_int
        L.bdlm_timing_collect.argtypes = [ctypes.c_int32, ctypes.POINTER(ctypes.c_int32), ctypes.POINTER(ctypes.c_float)]
        L.bdlm_timing_collect.restype = ctypes.c_int32
        L.bdlm_kernel_name.argtypes = [ctypes.c_int32]
        L.bdlm_kernel_name.restype = ctypes.c_char_p
        for name in ("bdlm_attn_fwd", "bdlm_attn_partial_fwd", "bdlm_lse_merge", "bdlm_lse_merge_strided",
                     "bdlm_attn_bwd", "bdlm_attn_bwd_noalloc"):
            getattr(L, name).restype = ctypes.c_int
        _LIB = L
    return _LIB


def _check(status: int):
    if status != 0:
        raise BdlmError(status, lib().bdlm_last_error().decode())


def _ptr(x) -> int:
    """Device address of a tensor (which must be contiguous and on the GPU) or a raw pointer int."""
    if x is None:
        return 0
    if isinstance(x, int):
        return x
    if not x.is_contiguous():
        raise ValueError(f"tensor of shape {tuple(x.shape)} is not contiguous")
    if not x.is_cuda:
        raise ValueError("tensor is not on the GPU")
    return x.data_ptr()


def _parr(xs) -> ctypes.Array:
    return (ctypes.c_void_p * max(1, len(xs)))(*[_ptr(x) for x in xs])


def _rarr(rs: Sequence[Range]) -> ctypes.Array:
    return (Range * max(1, len(rs)))(*rs)


def _stream(stream) -> int:
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def _dtype_code(dt: torch.dtype) -> int:
    if dt == torch.bfloat16:
        return BF16
    if dt == torch.float32:
        return F32
    raise TypeError(f"unsupported dtype {dt}")


def make_problem(batch: int, L: int, block_size: int, heads: int, kv_heads: int, head_dim: int,
                 dtype, scale: float = 0.0, clean_intra: int = CLEAN_INTRA_CAUSAL, out_f32: bool = False,
                 hilo=False, window: int = 0, clean_prefix: Optional[torch.Tensor] = None) -> Problem:
    """Problem record.  ``hilo`` is a mask of ``HILO_*`` bits (``True`` means the three product bits): the
    products that take P or dS as two bf16 terms, on every tile or, with ``HILO_ADAPTIVE``, only on
    tiles holding a large probability.  ``window`` limits every query to the last ``window`` positions of its clean
    context (0: no limit); ``clean_prefix`` is an int32 device tensor of ``L // block_size`` entries,
    the end of corrupted block b's clean context (DFlash2 anchors), kept alive by the caller until the
    kernels that use it have run."""
    code = dtype if isinstance(dtype, int) else _dtype_code(dtype)
    pref = None
    if clean_prefix is not None:
        if clean_prefix.dtype != torch.int32 or not clean_prefix.is_cuda or not clean_prefix.is_contiguous() \
                or clean_prefix.numel() != L // block_size:
            raise ValueError("clean_prefix must be a contiguous int32 device tensor of L // block_size entries")
        pref = clean_prefix.data_ptr()
    hmask = HILO_ALL if hilo is True else int(hilo)
    return Problem(batch, L, block_size, heads, kv_heads, head_dim, code, scale, clean_intra, int(bool(out_f32)),
                   hmask, int(window), pref)


def joint_ranges(L: int) -> List[Range]:
    """The packed ``[x_t ; x]`` layout: corrupted rows [0, L), clean rows [L, 2L) per batch element."""
    return [Range(CORRUPTED, 0, L, 2 * L), Range(CLEAN, 0, L, 2 * L)]


def attn_fwd(p: Problem, q_ranges: Sequence[Range], q, o, lse, k_ranges: Sequence[Range], k, v, stream=None):
    """``bdlm_attn_fwd``: q/o/lse are lists (one per query range), k/v lists (one per key range)."""
    _check(lib().bdlm_attn_fwd(ctypes.byref(p), len(q_ranges), _rarr(q_ranges), _parr(q), _parr(o), _parr(lse),
                               len(k_ranges), _rarr(k_ranges), _parr(k), _parr(v), _stream(stream)))


def attn_partial_fwd(p: Problem, qr: Range, q, o, lse, kr: Range, k, v, stream=None):
    """``bdlm_attn_partial_fwd``: one query range over one key range."""
    _check(lib().bdlm_attn_partial_fwd(ctypes.byref(p), qr, _ptr(q), _ptr(o), _ptr(lse), kr, _ptr(k), _ptr(v),
                                       _stream(stream)))


def _batch_stride(name, t, dtype, shape, lse_layout):
    """Rows between batch elements of ``t``: a ``[batch][rows][heads][d]`` (or, with ``lse_layout``,
    ``[batch][heads][rows]``) tensor or view whose rows are packed as in a tensor of ``stride`` rows
    per batch element, e.g. one range's half of a joint output."""
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor, got {type(t).__name__}")
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} must have shape {tuple(shape)}, got {tuple(t.shape)}")
    st = t.stride()
    if lse_layout:
        B, H, R = shape
        S = st[1] if H > 1 else (st[0] if B > 1 else R)
        ok = (R <= 1 or st[2] == 1) and (B <= 1 or st[0] == H * S)
    else:
        B, R, H, D = shape
        S = st[0] // (H * D) if B > 1 else R
        ok = st[3] == 1 and (H <= 1 or st[2] == D) and (R <= 1 or st[1] == H * D) and (B <= 1 or st[0] == S * H * D)
    if not ok or S < R:
        raise ValueError(f"{name} must hold its rows packed (only the batch stride may exceed the row count)")
    return S


def lse_merge(o_parts, lse_parts, o, lse, stream=None):
    """``bdlm_lse_merge_strided`` of partials shaped ``[batch][rows][heads][d]`` / ``[batch][heads][rows]``.

    Each tensor may be a view whose batch elements lie further apart than ``rows`` (one range of a
    joint output, say); the parts share one batch stride, ``o`` and ``lse`` another."""
    if not isinstance(o, torch.Tensor) or o.dim() != 4:
        raise ValueError("o must be a [batch][rows][heads][head_dim] tensor")
    B, R, H, D = o.shape
    if len(o_parts) != len(lse_parts) or not o_parts:
        raise ValueError("need one LSE per partial output and at least one part")
    _dtype_code(o.dtype)
    pdt = o_parts[0].dtype
    _dtype_code(pdt)
    strides = set()
    for j, (op, lp) in enumerate(zip(o_parts, lse_parts)):
        strides.add(_batch_stride(f"o_parts[{j}]", op, pdt, o.shape, False))
        strides.add(_batch_stride(f"lse_parts[{j}]", lp, torch.float32, (B, H, R), True))
    if len(strides) != 1:
        raise ValueError("the partials and their LSEs must share one batch stride")
    so = _batch_stride("o", o, o.dtype, o.shape, False)
    if _batch_stride("lse", lse, torch.float32, (B, H, R), True) != so:
        raise ValueError("o and lse must share one batch stride")
    _on_device(o.device, o=o, lse=lse, **{f"o_parts[{j}]": t for j, t in enumerate(o_parts)},
               **{f"lse_parts[{j}]": t for j, t in enumerate(lse_parts)})
    # views: their addresses are taken as they are (the layout was checked above)
    _check(lib().bdlm_lse_merge_strided(B, R, H, D, len(o_parts), _parr([t.data_ptr() for t in o_parts]),
                                        _parr([t.data_ptr() for t in lse_parts]), _dtype_code(pdt), strides.pop(),
                                        o.data_ptr(), lse.data_ptr(), _dtype_code(o.dtype), so, _stream(stream)))


def attn_bwd_workspace_bytes(p: Problem, q_ranges: Sequence[Range]) -> int:
    return int(lib().bdlm_attn_bwd_workspace_bytes(ctypes.byref(p), len(q_ranges), _rarr(q_ranges)))


def attn_bwd(p: Problem, q_ranges, q, o, lse, dO, dq, k_ranges, k, v, dk, dv, workspace, stream=None):
    """``bdlm_attn_bwd``; ``workspace`` is a device tensor of at least ``attn_bwd_workspace_bytes`` bytes."""
    nbytes = workspace.numel() * workspace.element_size() if workspace is not None else 0
    _check(lib().bdlm_attn_bwd(ctypes.byref(p), len(q_ranges), _rarr(q_ranges), _parr(q), _parr(o), _parr(lse),
                               _parr(dO), _parr(dq), len(k_ranges), _rarr(k_ranges), _parr(k), _parr(v),
                               _parr(dk), _parr(dv), _ptr(workspace), nbytes, _stream(stream)))


def attn_bwd_noalloc(p: Problem, q_ranges, q, o, lse, dO, dq, k_ranges, k, v, dk, dv, stream=None):
    """``bdlm_attn_bwd_noalloc``: :func:`attn_bwd` without a workspace (the library's per-GPU scratch
    array of ``NOALLOC_SCRATCH_BYTES`` holds D); calls that overlap on one GPU race."""
    _check(lib().bdlm_attn_bwd_noalloc(ctypes.byref(p), len(q_ranges), _rarr(q_ranges), _parr(q), _parr(o),
                                       _parr(lse), _parr(dO), _parr(dq), len(k_ranges), _rarr(k_ranges), _parr(k),
                                       _parr(v), _parr(dk), _parr(dv), _stream(stream)))


def visible_pairs(p: Problem, q_ranges: Sequence[Range], k_ranges: Sequence[Range]) -> int:
    """Valid query-key pairs of the mask per (batch element, query head) (host computation)."""
    n = lib().bdlm_visible_pairs(ctypes.byref(p), len(q_ranges), _rarr(q_ranges), len(k_ranges), _rarr(k_ranges))
    if n < 0:
        raise BdlmError(-1, lib().bdlm_last_error().decode())
    return int(n)


def timing_enable(on: bool = True):
    """Bracket every kernel this thread enqueues with HIP events (see bdlm_timing_enable)."""
    _check(lib().bdlm_timing_enable(int(bool(on))))


def timing_collect(max_records: int = 1 << 16):
    """Wait for recorded kernels and return [(kernel_name, ms), ...] in launch order."""
    ids = (ctypes.c_int32 * max_records)()
    ms = (ctypes.c_float * max_records)()
    n = lib().bdlm_timing_collect(max_records, ids, ms)
    if n < 0:
        raise BdlmError(n, lib().bdlm_last_error().decode())
    return [(lib().bdlm_kernel_name(ids[i]).decode(), float(ms[i])) for i in range(n)]


# ----------------------------------------------------------- joint helpers
def _joint_ptrs(t: torch.Tensor, L: int):
    """Pointers of the corrupted and clean halves of a packed [B][2L][H][D] tensor."""
    step = L * t.shape[2] * t.shape[3] * t.element_size()
    return [t.data_ptr(), t.data_ptr() + step]


def _expect(name, t, dtype, shape):
    """Reject a tensor of the wrong type, dtype, shape or layout before any pointer reaches the library."""
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor, got {type(t).__name__}")
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} must have shape {tuple(shape)}, got {tuple(t.shape)}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")


def _on_device(device, **tensors):
    for name, t in tensors.items():
        if not t.is_cuda or t.device != device:
            raise ValueError(f"{name} must be on {device}, got {t.device}")


def _check_joint(q, k, v):
    """Packed ``[x_t ; x]`` inputs: q ``[B][2L][Hq][D]``, k and v ``[B][2L][Hkv][D]``, one dtype."""
    if not isinstance(q, torch.Tensor) or q.dim() != 4 or q.shape[1] % 2:
        raise ValueError(f"q must be a [batch][2L][heads][head_dim] tensor, got "
                         f"{tuple(q.shape) if isinstance(q, torch.Tensor) else type(q).__name__}")
    _dtype_code(q.dtype)
    B, n, _, D = q.shape
    if not isinstance(k, torch.Tensor) or k.dim() != 4:
        raise ValueError("k must be a [batch][2L][kv_heads][head_dim] tensor")
    _expect("q", q, q.dtype, q.shape)
    _expect("k", k, q.dtype, (B, n, k.shape[2], D))
    _expect("v", v, q.dtype, k.shape)


def _check_ws(workspace, device):
    if workspace is None:
        return
    if not isinstance(workspace, torch.Tensor) or not workspace.is_contiguous():
        raise ValueError("workspace must be a contiguous tensor")
    _on_device(device, workspace=workspace)


def joint_fwd(q, k, v, block_size: int, clean_intra: int = CLEAN_INTRA_CAUSAL, scale: float = 0.0,
              out_f32: bool = False, out: Optional[tuple] = None, stream=None, hilo=False,
              window: int = 0, clean_prefix: Optional[torch.Tensor] = None):
    """Fused forward over packed ``[x_t ; x]`` tensors ``q [B][2L][Hq][D]``, ``k, v [B][2L][Hkv][D]``.

    Returns ``(o, lse)`` with ``lse [B][Hq][2L]`` fp32; ``o`` is fp32 when ``out_f32``.
    """
    _check_joint(q, k, v)
    B, n, Hq, D = q.shape
    L = n // 2
    p = make_problem(B, L, block_size, Hq, k.shape[2], D, q.dtype, scale, clean_intra, out_f32, hilo,
                     window, clean_prefix)
    odt = torch.float32 if out_f32 else q.dtype
    if out is not None:
        if len(out) != 2:
            raise ValueError("out must be (o, lse)")
        o, lse = out
        _expect("o", o, odt, q.shape)
        _expect("lse", lse, torch.float32, (B, Hq, n))
    _on_device(q.device, q=q, k=k, v=v)
    if out is None:
        o = torch.empty(q.shape, dtype=odt, device=q.device)
        lse = torch.empty((B, Hq, n), dtype=torch.float32, device=q.device)
    else:
        _on_device(q.device, o=o, lse=lse)
    r = joint_ranges(L)
    lp = [lse.data_ptr(), lse.data_ptr() + L * 4]
    attn_fwd(p, r, _joint_ptrs(q, L), _joint_ptrs(o, L), lp, r, _joint_ptrs(k, L), _joint_ptrs(v, L), stream)
    return o, lse


def joint_bwd(q, k, v, o, lse, do, block_size: int, clean_intra: int = CLEAN_INTRA_CAUSAL, scale: float = 0.0,
              out_f32: bool = False, out: Optional[tuple] = None, workspace: Optional[torch.Tensor] = None,
              stream=None, hilo=False, window: int = 0, clean_prefix: Optional[torch.Tensor] = None):
    """Backward of :func:`joint_fwd`; returns ``(dq, dk, dv)`` (fp32 when ``out_f32``; ``o`` must match)."""
    _check_joint(q, k, v)
    B, n, Hq, D = q.shape
    L = n // 2
    p = make_problem(B, L, block_size, Hq, k.shape[2], D, q.dtype, scale, clean_intra, out_f32, hilo,
                     window, clean_prefix)
    r = joint_ranges(L)
    odt = torch.float32 if out_f32 else q.dtype
    _expect("o", o, odt, q.shape)
    _expect("lse", lse, torch.float32, (B, Hq, n))
    _expect("do", do, q.dtype, q.shape)
    if out is not None:
        if len(out) != 3:
            raise ValueError("out must be (dq, dk, dv)")
        for name, t, like in zip(("dq", "dk", "dv"), out, (q, k, v)):
            _expect(name, t, odt, like.shape)
    _on_device(q.device, q=q, k=k, v=v, o=o, lse=lse, do=do)
    _check_ws(workspace, q.device)
    if out is None:
        out = tuple(torch.empty(t.shape, dtype=odt, device=q.device) for t in (q, k, v))
    else:
        _on_device(q.device, dq=out[0], dk=out[1], dv=out[2])
    dq, dk, dv = out
    if workspace is None:
        workspace = torch.empty(attn_bwd_workspace_bytes(p, r), dtype=torch.uint8, device=q.device)
    lp = [lse.data_ptr(), lse.data_ptr() + L * 4]
    attn_bwd(p, r, _joint_ptrs(q, L), _joint_ptrs(o, L), lp, _joint_ptrs(do, L), _joint_ptrs(dq, L),
             r, _joint_ptrs(k, L), _joint_ptrs(v, L), _joint_ptrs(dk, L), _joint_ptrs(dv, L), workspace, stream)
    return dq, dk, dv


def useful_flops(pairs_per_head: int, heads: int, batch: int, head_dim: int) -> dict:
    """Useful FLOPs of the valid pairs: 4 d per pair forward (Q K^T, P V), 10 d backward (five products)."""
    n = pairs_per_head * heads * batch
    return {"fwd": 4 * head_dim * n, "bwd": 10 * head_dim * n, "total": 14 * head_dim * n}


def default_scale(head_dim: int) -> float:
    return 1.0 / math.sqrt(head_dim)
