"""Attention over the selected blocks (float64), test infrastructure only.

For every query head h of execution group g and every chunk query t of
sequence b (absolute position p = cached_len_b + t):

1. gather: copy the K and V pages of every block j in T[b,g] out of the pool
   (``k_pool[page_table[b, kvh, j]]``), in table order, together with each
   key's absolute position 64*j + r -- an explicit gather, which is exactly
   the copy that zero-copy execution avoids (Sec. 3.3) and so an independent
   way of computing what the in-place kernel must produce.  Only keys at
   positions before the sequence end cached_len_b + C exist: the rows of the
   last page past it (a length that is not a multiple of 64) are not part of
   the sequence and are dropped, whatever they hold;
2. z = sm_scale * q . k for every gathered key, with z = -inf where the key
   position exceeds p (causal masking in absolute positions, App. B.2 last
   paragraph: positions come from the logical block id, never from a key's
   rank in the compacted list);
3. lse = m + log(sum exp(z - m)) with m = max z;  o = sum exp(z - lse) * v.

A query with no visible key gets o = 0 and lse = -inf.  The dense baseline
is the same computation over T[b,g] = all blocks of sequence b, which is what
the table definition gives for an all-ones mask (Sec. 3.2).

Parity: pinned by agreement with torch's fp64 scaled-dot-product attention on
contiguous, unpaged K/V (all-open tables and cached_len = 0), by the masked-
dense formulation, by page-permutation invariance and by a hand-worked
fixture (tests/test_oracle.py).
"""
from __future__ import annotations

from typing import Iterable, List, Optional, Sequence, Tuple

import numpy as np

from .bf16 import bf16_to_f64


def gather_selected(k_pool_bits, v_pool_bits, page_table, b: int, kvh: int,
                    table: Sequence[int],
                    seq_len: Optional[int] = None) -> Tuple[np.ndarray, np.ndarray, np.ndarray]:
    """Explicit copy of the selected pages: Ksel, Vsel [n, D] and key positions.

    Rows at positions >= ``seq_len`` (when given) are left out."""
    page = k_pool_bits.shape[1]
    ks, vs, pos = [], [], []
    for j in table:
        pid = page_table[b, kvh, j]
        rows = page if seq_len is None else max(0, min(page, int(seq_len) - page * int(j)))
        ks.append(bf16_to_f64(k_pool_bits[pid][:rows]))
        vs.append(bf16_to_f64(v_pool_bits[pid][:rows]))
        pos.append(page * int(j) + np.arange(rows))
    D = k_pool_bits.shape[2]
    if not ks:
        return np.zeros((0, D)), np.zeros((0, D)), np.zeros(0, dtype=np.int64)
    return np.concatenate(ks), np.concatenate(vs), np.concatenate(pos)


def attention_rows(q: np.ndarray, qpos: np.ndarray, ksel: np.ndarray,
                   vsel: np.ndarray, kpos: np.ndarray, sm_scale: float,
                   row_batch: int = 256) -> Tuple[np.ndarray, np.ndarray]:
    """Softmax attention of query rows q [n, D] over gathered keys, float64."""
    n, D = q.shape
    out = np.zeros((n, vsel.shape[1]))
    lse = np.full(n, -np.inf)
    for r0 in range(0, n, row_batch):
        r1 = min(n, r0 + row_batch)
        z = sm_scale * (q[r0:r1] @ ksel.T)
        z[kpos[None, :] > qpos[r0:r1, None]] = -np.inf
        m = z.max(axis=1) if z.shape[1] else np.full(r1 - r0, -np.inf)
        ok = np.isfinite(m)
        if not ok.any():
            continue
        zz = z[ok] - m[ok, None]
        l = np.exp(zz).sum(axis=1)
        lse_ok = m[ok] + np.log(l)
        p = np.exp(z[ok] - lse_ok[:, None])
        out[r0:r1][ok] = p @ vsel
        lse[r0:r1][ok] = lse_ok
    return out, lse


def dense_tables(n_blocks: Sequence[int], num_groups: int) -> List[List[List[int]]]:
    """T[b][g] = every block of sequence b (the all-ones mask); n_blocks[b] = nKB_b
    = ceil((cached_len_b + C) / 64)."""
    return [[list(range(int(n))) for _ in range(num_groups)] for n in n_blocks]


def chunk_attention(q_bits: np.ndarray, k_pool_bits: np.ndarray,
                    v_pool_bits: np.ndarray, page_table: np.ndarray,
                    cached_len: Sequence[int], tables, group_size: int,
                    sm_scale: float,
                    heads: Optional[Iterable[Tuple[int, int]]] = None,
                    queries: Optional[Sequence[int]] = None):
    """Chunk attention through per-group tables.

    ``tables`` is T[b][g] (lists) or a CSR pair (kv_indptr, kv_indices) with
    rows in (b-major, g-minor) order.  ``heads`` restricts the work to some
    (b, h) pairs and ``queries`` to some chunk positions (for sampled checks
    at full size).  Returns (out [B, C, Hq, D] float64, lse [B, Hq, C]);
    rows that were not computed are NaN.
    """
    B, C, Hq, D = q_bits.shape
    Hkv = page_table.shape[1]
    ratio = Hq // Hkv
    G = Hq // group_size
    if isinstance(tables, tuple):
        indptr, indices = tables
        tables = [[indices[indptr[b * G + g]:indptr[b * G + g + 1]].tolist()
                   for g in range(G)] for b in range(B)]
    if heads is None:
        heads = [(b, h) for b in range(B) for h in range(Hq)]
    t_idx = np.arange(C) if queries is None else np.asarray(queries)
    out = np.full((B, C, Hq, D), np.nan)
    lse = np.full((B, Hq, C), np.nan)
    by_group = {}
    for (b, h) in heads:
        by_group.setdefault((b, h // group_size), []).append(h)
    for (b, g), hs in by_group.items():
        kvh = (g * group_size) // ratio
        ksel, vsel, kpos = gather_selected(k_pool_bits, v_pool_bits, page_table,
                                           b, kvh, tables[b][g], int(cached_len[b]) + C)
        qpos = int(cached_len[b]) + t_idx
        for h in hs:
            q = bf16_to_f64(q_bits[b, t_idx, h, :])
            o, l = attention_rows(q, qpos, ksel, vsel, kpos, sm_scale)
            out[b, t_idx, h, :] = o
            lse[b, h, t_idx] = l
    return out, lse


def block_sparse_attention(q_bits: np.ndarray, k_pool_bits: np.ndarray,
                           v_pool_bits: np.ndarray, page_table: np.ndarray,
                           cached_len: Sequence[int], mask_bits: np.ndarray, q_block: int,
                           sm_scale: float,
                           heads: Optional[Iterable[Tuple[int, int]]] = None,
                           queries: Optional[Sequence[int]] = None):
    """Block-sparse execution of the 2D mask (the ablation arm of Sec. 4.4).

    Query t of Q-block i = t // q_block of head h attends to the blocks of its
    own mask row, T = {j < nKB_b : M[b, h, i, j]} (no union over Q-blocks or
    heads), through the same gather and softmax as ``chunk_attention``.
    ``mask_bits`` is the unpacked mask, bool [B, Hq, nQB, >= nKB_b].  Returns
    (out [B, C, Hq, D], lse [B, Hq, C]); rows not computed are NaN.
    """
    B, C, Hq, D = q_bits.shape
    Hkv = page_table.shape[1]
    ratio = Hq // Hkv
    page = k_pool_bits.shape[1]
    if heads is None:
        heads = [(b, h) for b in range(B) for h in range(Hq)]
    t_all = np.arange(C) if queries is None else np.asarray(queries)
    out = np.full((B, C, Hq, D), np.nan)
    lse = np.full((B, Hq, C), np.nan)
    for (b, h) in heads:
        nkb = -(-(int(cached_len[b]) + C) // page)
        kvh = h // ratio
        for i in sorted(set((t_all // q_block).tolist())):
            t_idx = t_all[t_all // q_block == i]
            table = [j for j in range(nkb) if mask_bits[b, h, i, j]]
            ksel, vsel, kpos = gather_selected(k_pool_bits, v_pool_bits, page_table,
                                               b, kvh, table, int(cached_len[b]) + C)
            q = bf16_to_f64(q_bits[b, t_idx, h, :])
            o, l = attention_rows(q, int(cached_len[b]) + t_idx, ksel, vsel, kpos, sm_scale)
            out[b, t_idx, h, :] = o
            lse[b, h, t_idx] = l
    return out, lse
