"""Block-union KV tables with set logic (float-free), test infrastructure only.

Follows Sec. 3.2 literally:

* Q-block union:     Mbar[b,h,j] = OR_i M[b,h,i,j]
* intra-group union: G[b,g,j]    = OR_{h in H(g)} Mbar[b,h,j]
* table:             T[b,g]      = { j : G[b,g,j] = 1 }

with H(g) = {g*s, ..., g*s + s - 1} for execution groups of s consecutive query
heads (the KV group by default, or 4-head sub-groups of a larger KV group,
App. B.1).  Only blocks j < nKB_b (cached + chunk blocks of sequence b) are
part of the domain; bits beyond it are ignored.  Tables are emitted as CSR
(``kv_indptr``, ``kv_indices``) with rows in (b-major, g-minor) order and
entries as ascending logical block ids (App. B.2 passes exactly this pair to
the paged kernel).

Parity: pinned by coverage + minimality (Sec. 3.2, the paragraph after the
table equation), by brute-force enumeration on tiny shapes against a bitwise
formulation, and by a hand-worked fixture.
"""
from __future__ import annotations

from typing import List, Sequence, Tuple

import numpy as np


def unpack_masks(masks: np.ndarray) -> np.ndarray:
    """uint64 [..., W] -> bool [..., 64*W]; column j is bit j&63 of word j>>6."""
    shifts = np.arange(64, dtype=np.uint64)
    bits = (masks[..., None] >> shifts) & np.uint64(1)
    return bits.reshape(masks.shape[:-1] + (masks.shape[-1] * 64,)).astype(bool)


def block_tables(masks: np.ndarray, group_size: int,
                 n_blocks: Sequence[int]) -> List[List[List[int]]]:
    """T[b][g] as sorted Python lists, from masks uint64 [B, Hq, nQB, W]."""
    B, Hq, nqb, _ = masks.shape
    if Hq % group_size:
        raise ValueError("group_size must divide the number of query heads")
    bits = unpack_masks(masks)
    G = Hq // group_size
    tables: List[List[List[int]]] = []
    for b in range(B):
        nkb = int(n_blocks[b])
        per_b = []
        for g in range(G):
            selected = set()
            for h in range(g * group_size, (g + 1) * group_size):   # h in H(g)
                for i in range(nqb):                                  # every Q-block
                    selected.update(np.nonzero(bits[b, h, i, :nkb])[0].tolist())
            per_b.append(sorted(selected))
        tables.append(per_b)
    return tables


def tables_to_csr(tables: List[List[List[int]]]) -> Tuple[np.ndarray, np.ndarray]:
    rows = [row for per_b in tables for row in per_b]
    indptr = np.zeros(len(rows) + 1, dtype=np.int32)
    for r, row in enumerate(rows):
        indptr[r + 1] = indptr[r] + len(row)
    indices = np.array([j for row in rows for j in row], dtype=np.int32)
    return indptr, indices


def union_densities(masks: np.ndarray, group_size: int,
                    n_cached: Sequence[int]) -> dict:
    """Mean fraction of *cached* blocks kept at each aggregation step.

    pre-union (per (h, i) row), after the Q-block union (per head) and after
    the intra-group union (per group) -- the quantities Table 2 reports as
    sparsity (1 - density).
    """
    bits = unpack_masks(masks)
    B, Hq, nqb, _ = masks.shape
    pre, qu, gu = [], [], []
    for b in range(B):
        nc = int(n_cached[b])
        if nc == 0:
            continue
        cb = bits[b, :, :, :nc]
        pre.append(cb.mean())
        mbar = cb.any(axis=1)
        qu.append(mbar.mean())
        gu.append(mbar.reshape(Hq // group_size, group_size, nc).any(axis=1).mean())
    f = lambda v: float(np.mean(v)) if v else 0.0
    return dict(pre_union=f(pre), q_union=f(qu), group_union=f(gu))
