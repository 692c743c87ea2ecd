"""Host-side checks of the C ABI: the library loads, exports every declared
symbol, rejects invalid arguments before any launch, and its pair counter
matches the paper's closed form and the oracle's explicit mask.

No GPU is touched: every call here fails validation (returns before any HIP
call) or is host-only (bdlm_visible_pairs, bdlm_attn_bwd_workspace_bytes).
"""
import ctypes
import os
import re

import pytest
import torch

import oracle
import paper_2609_19242_amd as bd
from paper_2609_19242_amd import CLEAN, CORRUPTED, Range
from synth import WORKLOADS

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "bdlm_attn.h")

pytestmark = pytest.mark.skipif(not os.path.exists(bd.library_path), reason="library not built")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(bdlm_[a-z_]+)\s*\(", text)))


def test_every_declared_symbol_is_exported():
    names = declared_functions()
    assert {"bdlm_attn_fwd", "bdlm_attn_bwd", "bdlm_attn_partial_fwd", "bdlm_lse_merge"} <= set(names)
    L = bd.lib()
    for n in names:
        assert hasattr(L, n), n


def _prob(**kw):
    base = dict(batch=1, L=64, block_size=16, heads=4, kv_heads=2, head_dim=128, dtype=bd.BF16)
    base.update(kw)
    return bd.make_problem(**base)


FAKE = 0x10000  # never dereferenced: these calls fail validation first
# Tests that pass unmapped pointers run only where no GPU is visible: should a
# validation bug let such a call through, nothing is launched on a device.
# (Counting devices does not initialise the HIP runtime.)
host_only = pytest.mark.skipif(torch.cuda.device_count() > 0,
                               reason="passes unmapped pointers that validation must reject; host-only test")


def _fwd(p, qr=None, kr=None, ptr=FAKE):
    qr = qr or [Range(CORRUPTED, 0, p.L)]
    kr = kr or [Range(CLEAN, 0, p.L)]
    return bd.lib().bdlm_attn_fwd(ctypes.byref(p), len(qr), bd._rarr(qr), bd._parr([ptr] * len(qr)),
                                  bd._parr([ptr] * len(qr)), bd._parr([ptr] * len(qr)), len(kr), bd._rarr(kr),
                                  bd._parr([ptr] * len(kr)), bd._parr([ptr] * len(kr)), None)


@pytest.mark.parametrize("kw,status,needle", [
    (dict(L=60, block_size=16), -1, "block_size"),
    (dict(heads=3, kv_heads=2), -1, "kv_heads"),
    (dict(head_dim=96), -2, "head_dim"),
    (dict(dtype=7), -2, "dtype"),
    (dict(batch=0), -1, "batch"),
    (dict(clean_intra=5), -1, "clean_intra"),
    (dict(hilo=16), -1, "hilo"),
    (dict(hilo=-1), -1, "hilo"),
])
@host_only
def test_invalid_problem_rejected(kw, status, needle):
    assert _fwd(_prob(**kw)) == status
    assert needle in bd.lib().bdlm_last_error().decode()


@host_only
def test_invalid_ranges_rejected():
    p = _prob()
    assert _fwd(p, qr=[Range(CORRUPTED, 60, 8)]) == -1  # past L
    assert "outside" in bd.lib().bdlm_last_error().decode()
    assert _fwd(p, qr=[Range(2, 0, 8)]) == -1  # bad stream
    assert _fwd(p, qr=[Range(CLEAN, 0, 8, 4)]) == -1  # batch_stride < len
    assert _fwd(p, kr=[Range(CLEAN, 0, 8)] * 33) == -2  # too many key ranges
    assert _fwd(p, ptr=FAKE + 8) == -1  # misaligned
    assert "aligned" in bd.lib().bdlm_last_error().decode()
    assert _fwd(p, ptr=0) == -1  # null
    L = bd.lib()
    assert L.bdlm_attn_fwd(ctypes.byref(p), 0, None, None, None, None, 1, bd._rarr([Range(CLEAN, 0, 8)]),
                           None, None, None) == -1


@host_only
def test_merge_and_bwd_validation():
    L = bd.lib()
    parts = bd._parr([FAKE])
    assert L.bdlm_lse_merge(1, 8, 2, 128, 0, parts, parts, 0, FAKE, FAKE, 0, None) == -1
    assert L.bdlm_lse_merge(1, 8, 2, 128, 33, parts, parts, 0, FAKE, FAKE, 0, None) == -2
    assert L.bdlm_lse_merge(1, 8, 2, 80, 1, parts, parts, 0, FAKE, FAKE, 0, None) == -2
    assert L.bdlm_lse_merge(1, 8, 2, 128, 1, parts, parts, 0, FAKE, FAKE + 64, 0, None) == -1  # o aliases a part
    # strided form: batch strides below the row count are invalid, above 2^30 unsupported
    assert L.bdlm_lse_merge_strided(2, 8, 2, 128, 1, parts, parts, 0, 7, FAKE + 4096, FAKE + 8192, 0, 0, None) == -1
    assert L.bdlm_lse_merge_strided(2, 8, 2, 128, 1, parts, parts, 0, 0, FAKE + 4096, FAKE + 8192, 0, 5, None) == -1
    assert L.bdlm_lse_merge_strided(2, 8, 2, 128, 1, parts, parts, 0, 1 << 31, FAKE + 4096, FAKE + 8192, 0, 0,
                                    None) == -2
    p = _prob()
    qr = [Range(CORRUPTED, 0, 64)]
    need = bd.attn_bwd_workspace_bytes(p, qr)
    assert need == 2 * 256 * (-(-64 * 4 * 4 // 256))  # fp32 LSE*log2(e) and D per (row, head), 256-byte aligned
    f = bd._parr([FAKE])
    rc = L.bdlm_attn_bwd(ctypes.byref(p), 1, bd._rarr(qr), f, f, f, f, f, 1, bd._rarr([Range(CLEAN, 0, 64)]),
                         f, f, f, f, FAKE, need - 1, None)
    assert rc == -4 and "workspace" in L.bdlm_last_error().decode()


# ------------------------------------------------------------ pair counter
def golden_pairs():
    out = {}
    with open(os.path.join(ROOT, "tests", "golden", "pair_counts.txt")) as f:
        for line in f:
            if line.startswith("#") or not line.strip():
                continue
            name, Lf, Mf, reading, pairs = line.split()
            out[(name, Lf, Mf, reading)] = int(pairs)
    return out


@pytest.mark.parametrize("name", ["tiny", "4k", "32k", "128k"])
@pytest.mark.parametrize("reading", ["causal", "block"])
def test_visible_pairs_match_closed_form(name, reading):
    w = WORKLOADS[name]
    rd = bd.CLEAN_INTRA_CAUSAL if reading == "causal" else bd.CLEAN_INTRA_BLOCK
    p = bd.make_problem(w.batch, w.L, w.block_size, w.heads, w.kv_heads, w.head_dim, bd.BF16, 0.0, rd)
    r = bd.joint_ranges(w.L)
    want = golden_pairs()[(name, f"L={w.L}", f"M={w.block_size}", reading)]
    assert bd.visible_pairs(p, r, r) == want


def test_visible_pairs_csbp_rank():
    w = WORKLOADS["csbp256k"]
    p = bd.make_problem(1, w.L, w.block_size, w.heads, w.kv_heads, w.head_dim, bd.BF16)
    qr = [Range(CORRUPTED, w.local_pos0, w.local_tokens)]
    kr = [Range(CORRUPTED, w.local_pos0, w.local_tokens)] + \
         [Range(CLEAN, s * w.shard_tokens, w.shard_tokens) for s in range(w.n_shards)]
    assert bd.visible_pairs(p, qr, kr) == 2281963520


@pytest.mark.parametrize("L,M", [(24, 4), (40, 8), (17, 17), (12, 1)])
@pytest.mark.parametrize("reading", [0, 1])
def test_visible_pairs_match_oracle_popcount(L, M, reading):
    p = bd.make_problem(1, L, M, 1, 1, 64, bd.BF16, 0.0, reading)
    qr = [Range(CORRUPTED, 0, L), Range(CLEAN, 0, L)]
    kr = [Range(CORRUPTED, 0, L), Range(CLEAN, 3, L - 5), Range(CLEAN, 0, 3)]
    got = bd.visible_pairs(p, qr, kr)
    want = oracle.count_visible_pairs([(CORRUPTED, 0, L), (CLEAN, 0, L)],
                                      [(CORRUPTED, 0, L), (CLEAN, 3, L - 5), (CLEAN, 0, 3)], M, reading)
    assert got == want


def test_visible_pairs_csbp_rank_with_clean_queries():
    """The rank's clean-shard queries (positions 131072..147455) see clean keys 0..p
    (clean->clean causal, Sec. 3.2): sum_p (p + 1) on top of the corrupted share."""
    w = WORKLOADS["csbp256k"]
    p = bd.make_problem(1, w.L, w.block_size, w.heads, w.kv_heads, w.head_dim, bd.BF16)
    S = w.shard_tokens
    own = w.local_pos0 // S
    qr = [Range(CORRUPTED, w.local_pos0, w.local_tokens), Range(CLEAN, own * S, S)]
    kr = [Range(CORRUPTED, w.local_pos0, w.local_tokens)] + \
         [Range(CLEAN, s * S, S) for s in range(w.n_shards)]
    first, last = own * S, own * S + S - 1
    clean = (last - first + 1) * (first + 1 + last + 1) // 2
    assert clean == 2281709568
    assert bd.visible_pairs(p, qr, kr) == 2281963520 + clean


# ------------------------------------------------------ mask generalisations
@host_only
def test_invalid_window_and_prefix_rejected():
    assert _fwd(_prob(window=-1)) == -1
    assert "window" in bd.lib().bdlm_last_error().decode()
    p = _prob()
    p.clean_prefix = FAKE + 2  # misaligned table pointer; never dereferenced
    assert _fwd(p) == -1
    assert "clean_prefix" in bd.lib().bdlm_last_error().decode()


@pytest.mark.parametrize("L,M,W", [(256, 16, 1), (256, 16, 40), (512, 32, 100), (128, 8, 10000)])
@pytest.mark.parametrize("reading", [bd.CLEAN_INTRA_CAUSAL, bd.CLEAN_INTRA_BLOCK])
def test_windowed_visible_pairs_match_oracle_popcount(L, M, W, reading):
    p = bd.make_problem(1, L, M, 2, 1, 128, bd.BF16, clean_intra=reading, window=W)
    qr = [Range(CORRUPTED, 0, L), Range(CLEAN, 0, L)]
    kr = [Range(CLEAN, 0, L // 2), Range(CORRUPTED, 0, L), Range(CLEAN, L // 2, L - L // 2)]
    want = oracle.count_visible_pairs([(CORRUPTED, 0, L), (CLEAN, 0, L)],
                                      [(CLEAN, 0, L // 2), (CORRUPTED, 0, L), (CLEAN, L // 2, L - L // 2)],
                                      M, reading, window=W)
    assert bd.visible_pairs(p, qr, kr) == want


# ---------------------------------------------------------------- size limits
@host_only
def test_size_limits_rejected_before_launch():
    L = bd.lib()
    # positions must stay below 2^30
    assert _fwd(_prob(L=1 << 30, block_size=1 << 20)) == -1
    assert "2^30" in L.bdlm_last_error().decode()
    # a query range whose batch * len * heads exceeds 2^28 is rejected by the backward
    n = 1 << 24  # 2^24 rows x 32 heads = 2^29
    p = bd.make_problem(1, n, 64, 32, 8, 128, bd.BF16)
    qr = [Range(CORRUPTED, 0, n)]
    need = bd.attn_bwd_workspace_bytes(p, qr)
    f = bd._parr([FAKE])
    rc = L.bdlm_attn_bwd(ctypes.byref(p), 1, bd._rarr(qr), f, f, f, f, f, 1, bd._rarr([Range(CLEAN, 0, 64)]),
                         f, f, f, f, FAKE, need, None)
    assert rc == -2 and "2^28" in L.bdlm_last_error().decode()
    # more query ranges than the kernel arguments hold
    assert _fwd(_prob(), qr=[Range(CORRUPTED, 0, 8)] * 5) == -2
    # a merge over 2^31 (row, head) pairs or more (the product is checked without overflowing)
    parts = bd._parr([FAKE])
    assert L.bdlm_lse_merge(1, 1 << 26, 32, 128, 1, parts, parts, 0, FAKE + 4096, FAKE + 8192, 0, None) == -2
    assert "2^31" in L.bdlm_last_error().decode()
    assert L.bdlm_lse_merge(1 << 40, 1 << 40, 1 << 30, 128, 1, parts, parts, 0, FAKE + 4096, FAKE + 8192, 0, None) == -2


@host_only
def test_noalloc_backward_rejects_scratch_overflow_before_launch():
    """bdlm_attn_bwd_noalloc: query ranges whose D arrays exceed the library's scratch array
    are rejected with BDLM_ERR_UNSUPPORTED before anything is enqueued."""
    L = 1 << 20  # 2 ranges x 2 arrays x 2^20 rows x 16 heads x 4 bytes = 256 MiB > 64 MiB
    p = _prob(L=L, block_size=64, heads=16, kv_heads=2)
    r = bd.joint_ranges(L)
    assert bd.attn_bwd_workspace_bytes(p, r) > bd.NOALLOC_SCRATCH_BYTES
    fake = [FAKE, FAKE]
    st = bd.lib().bdlm_attn_bwd_noalloc(ctypes.byref(p), 2, bd._rarr(r), bd._parr(fake), bd._parr(fake),
                                        bd._parr(fake), bd._parr(fake), bd._parr(fake), 2, bd._rarr(r),
                                        bd._parr(fake), bd._parr(fake), bd._parr(fake), bd._parr(fake), None)
    assert st == -2
    assert "scratch" in bd.lib().bdlm_last_error().decode()
    # the same call on a problem that fits passes the size check and stops at the next validation step
    p2 = _prob(L=64, block_size=16)
    r2 = bd.joint_ranges(64)
    st = bd.lib().bdlm_attn_bwd_noalloc(ctypes.byref(p2), 2, bd._rarr(r2), bd._parr(fake), bd._parr(fake),
                                        bd._parr(fake), bd._parr(fake), bd._parr([FAKE + 8, FAKE]), 2, bd._rarr(r2),
                                        bd._parr(fake), bd._parr(fake), bd._parr(fake), bd._parr(fake), None)
    assert st == -1 and "aligned" in bd.lib().bdlm_last_error().decode()
