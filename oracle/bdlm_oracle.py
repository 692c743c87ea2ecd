"""fp64 CPU oracle for BDLM attention -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this module.  The HIP library never calls it, and it
shares no code, tables or helpers with the HIP library.

What it computes is the plain definition of the method's result: masked
softmax attention over the length-2L clean-plus-corrupted representation and
its exact gradient.  The paper shows (Prop. ``prop:csbp-exactness``, App. A)
that block-parallel and context-sharded execution reach exactly this result up
to floating-point reduction order, so the oracle is that definition written
out in fp64 with the explicit boolean mask materialised.

Paper references (arXiv 2609.19242):

* mask: Sec. 3.2 (Block diffusion language models, last two paragraphs) and
  App. A step 1, eqs. ``eq:correctness-clean-attention`` and
  ``eq:correctness-corrupted-attention``;
* attention: eq. ``eq:context-parallel-attention`` (softmax(QK^T/sqrt(d_h) + M) V);
* partial attention over a key subset and its merge:
  eq. ``eq:correctness-online-softmax-merge`` and eq. ``eq:csbp-lse-merge``;
* backward: eqs. ``eq:correctness-corrupted-gradient`` to
  ``eq:correctness-query-gradient`` (clean dK/dV summed over every query row).

Conventions (0-based positions; the paper is 1-based):

* a row is ``(stream, pos)`` with stream ``CLEAN = 0`` or ``CORRUPTED = 1``;
  block of a position ``p`` is ``p // M`` with ``M`` the block size;
* arrays are ``[batch][rows][heads][d]``; LSE is ``[batch][heads][rows]``,
  natural log; query head ``h`` reads KV head ``h // (Hq // Hkv)``;
* a query row that sees no key gets ``O = 0`` and ``LSE = -inf``.
"""
from __future__ import annotations

import math
from typing import Iterable, List, Optional, Sequence, Tuple

import numpy as np

CLEAN = 0
CORRUPTED = 1

# Reading of the clean-to-clean rule inside a block (see the module docstring of
# ``visible``): the paper's token-causal rule is the default.
CLEAN_INTRA_CAUSAL = 0
CLEAN_INTRA_BLOCK = 1


def rows_of(ranges: Sequence[Tuple[int, int, int]]) -> Tuple[np.ndarray, np.ndarray]:
    """Row metadata for a tensor holding the given ``(stream, pos0, length)`` ranges in order."""
    streams, pos = [], []
    for stream, pos0, n in ranges:
        streams.append(np.full(n, stream, dtype=np.int64))
        pos.append(np.arange(pos0, pos0 + n, dtype=np.int64))
    if not streams:
        return np.zeros(0, np.int64), np.zeros(0, np.int64)
    return np.concatenate(streams), np.concatenate(pos)


def joint_ranges(L: int) -> List[Tuple[int, int, int]]:
    """The packed length-2L layout: corrupted copy x_t first, clean copy x second."""
    return [(CORRUPTED, 0, L), (CLEAN, 0, L)]


def visible(q_stream, q_pos, k_stream, k_pos, M: int, clean_intra: int = CLEAN_INTRA_CAUSAL,
            window: int = 0, clean_prefix: Optional[Sequence[int]] = None) -> np.ndarray:
    """Explicit BDLM mask ``mask[i, j]``: may query row i attend to key row j?

    Rules (Sec. 3.2; App. A step 1):

    * clean query, clean key: the clean prefix of earlier blocks plus causal
      access inside the own block, i.e. key position <= query position.  Under
      the alternative reading ``CLEAN_INTRA_BLOCK`` the whole own clean block
      is visible: block(key) <= block(query);
    * corrupted query, corrupted key: only the own corrupted block,
      bidirectionally: block(key) == block(query);
    * corrupted query, clean key: the clean prefix of earlier blocks,
      block(key) < block(query);
    * clean query, corrupted key: never.

    Two generalisations (the library's ``window`` and ``clean_prefix``):

    * ``clean_prefix[b]`` (DFlash2 drafter attention, App. "DFlash2 Drafter
      Training Methodology", eq. ``eq:dflash2-block-attention``): corrupted
      block b is a draft block that sees the clean rows (target features)
      before its anchor ``a_b = clean_prefix[b]`` instead of before ``M * b``;
    * ``window > 0`` (the sliding-window layers of App. "Savings Breakdowns";
      the paper gives only the width, this is the reading): with ``e`` the end
      of the clean context a query sees under the rules above (``q + 1``, the
      end of its block under the block reading, ``M * b`` or ``a_b`` for a
      corrupted query), only clean keys ``e - window <= k < e`` stay visible.
    """
    qs = np.asarray(q_stream)[:, None]
    qp = np.asarray(q_pos)[:, None]
    ks = np.asarray(k_stream)[None, :]
    kp = np.asarray(k_pos)[None, :]
    qb = qp // M
    kb = kp // M
    if clean_intra == CLEAN_INTRA_CAUSAL:
        clean_clean = kp <= qp
        clean_end = qp + 1
    elif clean_intra == CLEAN_INTRA_BLOCK:
        clean_clean = kb <= qb
        clean_end = (qb + 1) * M
    else:
        raise ValueError(f"unknown clean_intra {clean_intra}")
    corr_corr = kb == qb
    if clean_prefix is None:
        corr_clean = kb < qb
        corr_end = qb * M
    else:
        table = np.asarray(clean_prefix, dtype=np.int64)
        corr_end = table[np.minimum(qb, table.shape[0] - 1)]
        corr_clean = kp < corr_end
    if window:
        clean_clean = clean_clean & (kp >= clean_end - window)
        corr_clean = corr_clean & (kp >= corr_end - window)
    return np.where(
        qs == CLEAN,
        np.where(ks == CLEAN, clean_clean, False),
        np.where(ks == CORRUPTED, corr_corr, corr_clean),
    )


def attention_fwd_head(Q: np.ndarray, K: np.ndarray, V: np.ndarray, mask: np.ndarray, scale: float):
    """One head: ``O = softmax(scale * Q K^T + mask) V`` and its row log-sum-exp.

    ``Q`` is ``[n_q, d]``, ``K``/``V`` are ``[n_k, d]``, ``mask`` is ``[n_q, n_k]`` bool.
    Rows with no visible key return ``O = 0`` and ``LSE = -inf``.
    """
    S = scale * (Q @ K.T)
    S = np.where(mask, S, -np.inf)
    m = S.max(axis=1, initial=-np.inf)
    empty = ~np.isfinite(m)
    m_safe = np.where(empty, 0.0, m)
    P = np.exp(S - m_safe[:, None])  # exp(-inf) = 0 for masked keys
    l = P.sum(axis=1)
    l_safe = np.where(empty, 1.0, l)
    O = (P @ V) / l_safe[:, None]
    O[empty] = 0.0
    lse = np.where(empty, -np.inf, m_safe + np.log(l_safe))
    return O, lse


def attention_bwd_head(Q, K, V, O, lse, dO, mask, scale):
    """One head: gradients of ``sum(dO * O)`` w.r.t. Q, K and V, from the saved ``(O, LSE)``.

    With ``P = exp(S - LSE)`` (the softmax probabilities), ``dV = P^T dO``,
    ``dP = dO V^T``, ``D_i = sum_d dO_i O_i``, ``dS = P * (dP - D)``,
    ``dQ = scale * dS K`` and ``dK = scale * dS^T Q``.  Rows with LSE = -inf
    contribute nothing.
    """
    S = scale * (Q @ K.T)
    finite = np.isfinite(lse)
    lse_safe = np.where(finite, lse, 0.0)
    P = np.where(mask & finite[:, None], np.exp(S - lse_safe[:, None]), 0.0)
    dV = P.T @ dO
    dP = dO @ V.T
    D = np.sum(dO * O, axis=1)
    dS = P * (dP - D[:, None])
    dQ = scale * (dS @ K)
    dK = scale * (dS.T @ Q)
    return dQ, dK, dV


def _as64(x) -> np.ndarray:
    if hasattr(x, "detach"):  # torch tensor: upcast the values the GPU receives
        x = x.detach().cpu().double().numpy()
    return np.asarray(x, dtype=np.float64)


def _heads_arg(heads: Optional[Iterable[int]], Hq: int) -> List[int]:
    return list(range(Hq)) if heads is None else sorted(set(int(h) for h in heads))


def fwd(q, k, v, q_ranges, k_ranges, M: int, clean_intra: int = CLEAN_INTRA_CAUSAL,
        scale: Optional[float] = None, heads: Optional[Iterable[int]] = None,
        q_rows: Optional[np.ndarray] = None, chunk: int = 1024, window: int = 0,
        clean_prefix: Optional[Sequence[int]] = None):
    """Masked attention of the query rows over all key rows.

    ``q`` is ``[batch][n_q][Hq][d]`` holding ``q_ranges``; ``k``/``v`` are
    ``[batch][n_k][Hkv][d]`` holding ``k_ranges``.  ``heads`` restricts the
    query heads computed and ``q_rows`` the query rows (indices into ``q``).
    Returns ``O [batch][len(q_rows)][len(heads)][d]`` and
    ``LSE [batch][len(heads)][len(q_rows)]``.
    """
    q, k, v = _as64(q), _as64(k), _as64(v)
    B, nq, Hq, d = q.shape
    Hkv = k.shape[2]
    g = Hq // Hkv
    scale = 1.0 / math.sqrt(d) if scale is None else float(scale)
    hs = _heads_arg(heads, Hq)
    qs_all, qp_all = rows_of(q_ranges)
    ks, kp = rows_of(k_ranges)
    assert qs_all.shape[0] == nq and ks.shape[0] == k.shape[1]
    rows = np.arange(nq) if q_rows is None else np.asarray(q_rows)
    O = np.zeros((B, rows.shape[0], len(hs), d))
    LSE = np.full((B, len(hs), rows.shape[0]), -np.inf)
    for c0 in range(0, rows.shape[0], chunk):
        r = rows[c0:c0 + chunk]
        mask = visible(qs_all[r], qp_all[r], ks, kp, M, clean_intra, window, clean_prefix)
        for b in range(B):
            for hi, h in enumerate(hs):
                o, lse = attention_fwd_head(q[b, r, h], k[b, :, h // g], v[b, :, h // g], mask, scale)
                O[b, c0:c0 + r.shape[0], hi] = o
                LSE[b, hi, c0:c0 + r.shape[0]] = lse
    return O, LSE


def bwd(q, k, v, o, lse, do, q_ranges, k_ranges, M: int, clean_intra: int = CLEAN_INTRA_CAUSAL,
        scale: Optional[float] = None, heads: Optional[Iterable[int]] = None, chunk: int = 1024,
        window: int = 0, clean_prefix: Optional[Sequence[int]] = None):
    """Gradients of ``sum(dO * O)`` given the saved forward ``(O, LSE)``.

    ``o``/``do`` are ``[batch][n_q][len(heads)][d]`` and ``lse`` is
    ``[batch][len(heads)][n_q]`` for the query heads in ``heads`` (all heads
    by default).  Returns ``dQ`` for those heads and ``dK``/``dV`` summed over
    those heads (the full KV-head gradient when every head of a GQA group is
    included).
    """
    q, k, v, o, do = _as64(q), _as64(k), _as64(v), _as64(o), _as64(do)
    lse = _as64(lse)
    B, nq, Hq, d = q.shape
    Hkv = k.shape[2]
    g = Hq // Hkv
    scale = 1.0 / math.sqrt(d) if scale is None else float(scale)
    hs = _heads_arg(heads, Hq)
    qs_all, qp_all = rows_of(q_ranges)
    ks, kp = rows_of(k_ranges)
    dQ = np.zeros((B, nq, len(hs), d))
    dK = np.zeros(k.shape)
    dV = np.zeros(v.shape)
    for c0 in range(0, nq, chunk):
        r = slice(c0, min(nq, c0 + chunk))
        mask = visible(qs_all[r], qp_all[r], ks, kp, M, clean_intra, window, clean_prefix)
        for b in range(B):
            for hi, h in enumerate(hs):
                kv = h // g
                dq, dk, dv = attention_bwd_head(q[b, r, h], k[b, :, kv], v[b, :, kv], o[b, r, hi],
                                                lse[b, hi, r], do[b, r, hi], mask, scale)
                dQ[b, r, hi] = dq
                dK[b, :, kv] += dk
                dV[b, :, kv] += dv
    return dQ, dK, dV


def lse_merge(o_parts: Sequence[np.ndarray], lse_parts: Sequence[np.ndarray]):
    """J-way merge of normalised partial attentions over disjoint key sets.

    eq. ``eq:csbp-lse-merge`` generalised to J parts through
    eq. ``eq:correctness-online-softmax-merge``: ``m = max_j z_j``,
    ``w_j = exp(z_j - m)`` (0 when ``z_j = -inf``, the ``isfinite`` guard of
    the paper's merge kernel), ``O = sum_j w_j O_j / sum_j w_j`` and
    ``z = m + ln(sum_j w_j)``.  A row empty in every part gets ``O = 0`` and
    ``z = -inf``.

    ``o_parts[j]`` is ``[batch][rows][H][d]``, ``lse_parts[j]`` is ``[batch][H][rows]``.
    """
    O = [_as64(x) for x in o_parts]
    Z = [_as64(x) for x in lse_parts]
    z = np.stack(Z)  # [J][batch][H][rows]
    m = z.max(axis=0)
    empty = ~np.isfinite(m)
    m_safe = np.where(empty, 0.0, m)
    w = np.where(np.isfinite(z), np.exp(z - m_safe[None]), 0.0)
    den = w.sum(axis=0)
    num = np.zeros_like(O[0])
    for j in range(len(O)):
        num += np.transpose(w[j], (0, 2, 1))[..., None] * O[j]
    den_t = np.transpose(np.where(empty, 1.0, den), (0, 2, 1))[..., None]
    out = num / den_t
    out[np.transpose(empty, (0, 2, 1))] = 0.0
    lse = np.where(empty, -np.inf, m_safe + np.log(np.where(empty, 1.0, den)))
    return out, lse


def joint_fwd(q, k, v, L: int, M: int, **kw):
    """Fused forward over the packed ``[x_t ; x]`` rows of length 2L."""
    r = joint_ranges(L)
    return fwd(q, k, v, r, r, M, **kw)


def joint_bwd(q, k, v, o, lse, do, L: int, M: int, **kw):
    r = joint_ranges(L)
    return bwd(q, k, v, o, lse, do, r, r, M, **kw)


def count_visible_pairs(q_ranges, k_ranges, M: int, clean_intra: int = CLEAN_INTRA_CAUSAL, chunk: int = 4096,
                        window: int = 0, clean_prefix: Optional[Sequence[int]] = None) -> int:
    """Popcount of the explicit mask: the number of valid query-key pairs per (batch, head)."""
    qs, qp = rows_of(q_ranges)
    ks, kp = rows_of(k_ranges)
    total = 0
    for c0 in range(0, qs.shape[0], chunk):
        total += int(visible(qs[c0:c0 + chunk], qp[c0:c0 + chunk], ks, kp, M, clean_intra, window,
                             clean_prefix).sum())
    return total
