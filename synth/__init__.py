"""Seeded synthetic workloads for BDLM attention.

This module only draws random numbers and describes shapes.  It holds none of
the attention arithmetic: both the fp64 oracle and the HIP path receive the
tensors made here, so neither depends on the other.

Layout conventions (shared vocabulary, not arithmetic):

* the joint problem packs, per batch element, the corrupted copy x_t first and
  the clean copy x second: rows ``[0, L)`` are x_t, rows ``[L, 2L)`` are x
  (the length-2L representation of Sec. 3.2 of the paper);
* Q/O/dO/dQ are ``[batch][rows][Hq][d]``, K/V/dK/dV are
  ``[batch][rows][Hkv][d]``, LSE is ``[batch][Hq][rows]`` (fp32, natural log);
* ``block_size`` is the number of tokens per block (the paper's M = L/B).

Seeds: tensor ``t`` of workload ``c`` is drawn from a generator seeded with
``1000 * c + t`` (Q=0, K=1, V=2, dO=3, the pick of amplified key rows=4).
Values are drawn in fp32 and then cast to the run dtype; the oracle receives
the cast values upcast to fp64.
"""
from __future__ import annotations

import dataclasses
from typing import Dict, Optional

import torch

CORRUPTED = 1
CLEAN = 0


@dataclasses.dataclass(frozen=True)
class Workload:
    """One synthetic BDLM attention workload.

    ``kind == "joint"``: the fused length-2L problem, queries and keys are the
    packed ``[x_t ; x]`` rows of ``batch`` independent sequences of length L.

    ``kind == "csbp_rank"``: one context-sharded block-parallel rank's share.
    Its queries are ``local_tokens`` corrupted rows whose first row sits at
    global position ``local_pos0``; its keys are the same rows' corrupted K/V
    plus a clean prefix of ``clean_tokens`` rows held as ``n_shards`` equal
    shards (Sec. 4.3 and Alg. 1 of the paper).

    ``kind == "drafter"``: DFlash2 drafter attention (App. "DFlash2 Drafter
    Training Methodology"): ``draft_blocks`` draft blocks of ``block_size``
    rows (the corrupted stream) attend to themselves and to the target
    features (the clean stream, ``L`` rows) before their anchors.
    """

    index: int
    name: str
    kind: str
    batch: int
    L: int
    block_size: int
    heads: int
    kv_heads: int
    head_dim: int
    dtype: str  # "fp32" or "bf16"
    amplified_key_fraction: float = 0.0
    amplified_key_factor: float = 1.0
    local_tokens: int = 0
    local_pos0: int = 0
    clean_tokens: int = 0
    n_shards: int = 0
    window: int = 0        # sliding window over the clean context (0: none)
    draft_blocks: int = 0  # kind "drafter": draft blocks of block_size rows over L target-feature rows

    @property
    def torch_dtype(self) -> torch.dtype:
        return torch.float32 if self.dtype == "fp32" else torch.bfloat16

    @property
    def q_rows(self) -> int:
        if self.kind == "joint":
            return 2 * self.L
        return self.draft_blocks * self.block_size if self.kind == "drafter" else self.local_tokens

    @property
    def shard_tokens(self) -> int:
        return self.clean_tokens // self.n_shards if self.n_shards else 0

    def describe(self) -> str:
        win = f", window {self.window}" if self.window else ""
        if self.kind == "joint":
            return (f"batch {self.batch}, L={self.L} clean + {self.L} corrupted, block {self.block_size}, "
                    f"{self.heads}/{self.kv_heads} heads, d={self.head_dim}, {self.dtype}{win}")
        if self.kind == "drafter":
            return (f"drafter: {self.draft_blocks} draft blocks of {self.block_size} over {self.L} target-feature "
                    f"rows, sorted uniform anchors, {self.heads}/{self.kv_heads} heads, d={self.head_dim}, "
                    f"{self.dtype}{win}")
        return (f"CSBP rank: {self.local_tokens} corrupted rows at {self.local_pos0}, block {self.block_size}, "
                f"clean prefix {self.clean_tokens} as {self.n_shards} shards, "
                f"{self.heads}/{self.kv_heads} heads, d={self.head_dim}, {self.dtype}")


WORKLOADS: Dict[str, Workload] = {
    "tiny": Workload(1, "tiny", "joint", 1, 256, 16, 2, 2, 64, "fp32"),
    "4k": Workload(2, "4k", "joint", 2, 4096, 32, 32, 8, 128, "bf16"),
    "32k": Workload(3, "32k", "joint", 1, 32768, 64, 32, 8, 128, "bf16"),
    "csbp256k": Workload(4, "csbp256k", "csbp_rank", 1, 262144, 32, 32, 8, 128, "bf16",
                         local_tokens=16384, local_pos0=131072, clean_tokens=262144, n_shards=16),
    "128k": Workload(5, "128k", "joint", 1, 131072, 128, 64, 8, 128, "bf16",
                     amplified_key_fraction=0.01, amplified_key_factor=8.0),
    # The 32K shape in a sliding-window layer (the paper's 1,024-position window).
    "32k-w1024": Workload(6, "32k-w1024", "joint", 1, 32768, 64, 32, 8, 128, "bf16", window=1024),
    # A drafter share: 2,048 draft blocks of 16 over 32K target features.
    "drafter32k": Workload(7, "drafter32k", "drafter", 1, 32768, 16, 32, 8, 128, "bf16", draft_blocks=2048),
}
BY_INDEX = {w.index: w for w in WORKLOADS.values()}


def generator(seed: int, device: str = "cpu") -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    return g


def normal(shape, seed: int, dtype: torch.dtype, device: str = "cpu") -> torch.Tensor:
    """N(0,1) draws in fp32 from ``seed``, cast to ``dtype``."""
    x = torch.randn(*shape, generator=generator(seed, device), dtype=torch.float32, device=device)
    return x.to(dtype)


def amplified_rows(n_rows: int, fraction: float, seed: int) -> torch.Tensor:
    """Indices of floor(fraction * n_rows) distinct rows, drawn without replacement."""
    n = int(fraction * n_rows)
    g = generator(seed, "cpu")
    return torch.randperm(n_rows, generator=g)[:n].sort().values


def make_joint(w: Workload, device: str = "cpu", dtype: Optional[torch.dtype] = None,
               seed_base: Optional[int] = None, need_do: bool = True):
    """Packed joint tensors ``q, k, v, do`` for a ``kind == 'joint'`` workload."""
    assert w.kind == "joint"
    dt = dtype or w.torch_dtype
    base = 1000 * w.index if seed_base is None else seed_base
    rows = 2 * w.L
    q = normal((w.batch, rows, w.heads, w.head_dim), base + 0, dt, device)
    if w.amplified_key_fraction > 0:
        k32 = normal((w.batch, rows, w.kv_heads, w.head_dim), base + 1, torch.float32, device)
        idx = amplified_rows(rows, w.amplified_key_fraction, base + 4).to(device)
        k32[:, idx] *= w.amplified_key_factor
        k = k32.to(dt)
        del k32
    else:
        k = normal((w.batch, rows, w.kv_heads, w.head_dim), base + 1, dt, device)
    v = normal((w.batch, rows, w.kv_heads, w.head_dim), base + 2, dt, device)
    do = normal((w.batch, rows, w.heads, w.head_dim), base + 3, dt, device) if need_do else None
    return q, k, v, do


def make_csbp_rank(w: Workload, device: str = "cpu", dtype: Optional[torch.dtype] = None,
                   seed_base: Optional[int] = None, need_do: bool = True):
    """One CSBP rank's tensors: ``q, k_local, v_local, k_clean, v_clean, do``.

    ``k_clean``/``v_clean`` hold the whole clean prefix contiguously; shard s is
    rows ``[s * shard_tokens, (s + 1) * shard_tokens)``.
    """
    assert w.kind == "csbp_rank"
    dt = dtype or w.torch_dtype
    base = 1000 * w.index if seed_base is None else seed_base
    n = w.local_tokens
    q = normal((1, n, w.heads, w.head_dim), base + 0, dt, device)
    kall = normal((1, n + w.clean_tokens, w.kv_heads, w.head_dim), base + 1, dt, device)
    vall = normal((1, n + w.clean_tokens, w.kv_heads, w.head_dim), base + 2, dt, device)
    k_local, k_clean = kall[:, :n].contiguous(), kall[:, n:].contiguous()
    v_local, v_clean = vall[:, :n].contiguous(), vall[:, n:].contiguous()
    del kall, vall
    do = normal((1, n, w.heads, w.head_dim), base + 3, dt, device) if need_do else None
    return q, k_local, v_local, k_clean, v_clean, do


def csbp_own_shard(w: Workload) -> int:
    """Index of the clean shard a CSBP rank owns: the one at its corrupted blocks' positions."""
    assert w.kind == "csbp_rank" and w.local_pos0 % w.shard_tokens == 0
    return w.local_pos0 // w.shard_tokens


def make_csbp_clean_queries(w: Workload, device: str = "cpu", dtype: Optional[torch.dtype] = None,
                            seed_base: Optional[int] = None):
    """The rank's clean-shard queries and their upstream gradient: ``q_clean, do_clean``.

    These are the ``shard_tokens`` clean rows the rank owns (positions
    ``[own * shard_tokens, (own + 1) * shard_tokens)``); seeds are tensors 5 and 6
    of the workload.
    """
    assert w.kind == "csbp_rank"
    dt = dtype or w.torch_dtype
    base = 1000 * w.index if seed_base is None else seed_base
    shape = (1, w.shard_tokens, w.heads, w.head_dim)
    return normal(shape, base + 5, dt, device), normal(shape, base + 6, dt, device)


def draft_anchors(w: Workload, device: str = "cpu") -> torch.Tensor:
    """Anchors of the draft blocks: ``draft_blocks`` positions drawn uniformly
    from [1, L] (seed tensor 4), sorted; one int32 entry per block of the
    L-row stream, the entries past the draft blocks set to L."""
    assert w.kind == "drafter"
    nblk = w.L // w.block_size
    g = generator(1000 * w.index + 4, "cpu")
    a = torch.sort(torch.randint(1, w.L + 1, (w.draft_blocks,), generator=g)).values
    a = torch.cat([a, torch.full((nblk - w.draft_blocks,), w.L)]).to(torch.int32)
    return a.to(device)


def make_drafter(w: Workload, device: str = "cpu", dtype: Optional[torch.dtype] = None, need_do: bool = True):
    """Drafter tensors: ``q, k_draft, v_draft, k_target, v_target, do`` and the anchor table."""
    assert w.kind == "drafter"
    dt = dtype or w.torch_dtype
    base = 1000 * w.index
    nd = w.draft_blocks * w.block_size
    q = normal((1, nd, w.heads, w.head_dim), base + 0, dt, device)
    kall = normal((1, nd + w.L, w.kv_heads, w.head_dim), base + 1, dt, device)
    vall = normal((1, nd + w.L, w.kv_heads, w.head_dim), base + 2, dt, device)
    kd, kt = kall[:, :nd].contiguous(), kall[:, nd:].contiguous()
    vd, vt = vall[:, :nd].contiguous(), vall[:, nd:].contiguous()
    del kall, vall
    do = normal((1, nd, w.heads, w.head_dim), base + 3, dt, device) if need_do else None
    return q, kd, vd, kt, vt, do, draft_anchors(w, device)
