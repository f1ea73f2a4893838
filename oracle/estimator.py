"""Mean-pooled block-score mask estimator (float64), test infrastructure only.

The paper accepts any lightweight block-level pattern search that yields the
2D mask M[b,h,i,j] (Sec. 3.1; Sec. 3.2 first paragraph; Sec. 2.1 "pattern
search overhead" on why it must be cheap per chunk).  It does not define this
particular selector; the reading implemented here is:

1. q_mean[b,h,i]   = mean of the query rows of Q-block i, head h (the last
   Q-block of a chunk whose length is not a multiple of q_block holds fewer
   rows, and its mean is over the rows it holds);
2. k_mean[b,kvh,j] = mean of the key rows of logical block j, found through
   the page table (KV-head-major pages, Sec. 3.3); a block is only pooled
   over its rows at positions before the sequence end cached_len + C;
3. s[b,h,i,j] = q_mean . k_mean[kvh(h)], for the full cached blocks
   j < nC_b = floor(cached_len_b / page) only;
4. keep the top k = ceil(top_frac * nC_b) cached blocks of each row, ranked by
   score descending then block index ascending; scores are compared in
   float32, the precision the GPU scores are produced in (the decision is
   taken in one precision on both sides), with -0.0 equal to +0.0;
5. OR in the sink blocks {0..sink-1}, the local window
   {nC-local .. nC-1} (the full cached blocks just before the chunk) and the
   chunk-causal blocks: every block from nC up to the block holding the last
   query of Q-block i, i.e. {nC .. floor((cached_len + min((i+1)*q_block, C)
   - 1) / page)}; the whole chunk is thereby open after the Q-block union
   (Sec. 3.1 last paragraph of the overview; App. B.2 last paragraph).  With
   aligned lengths this is {nC .. nC + (i+1)*q_block/page - 1}.  A block
   that holds both cached and chunk tokens (cached_len not a multiple of
   page) counts as a chunk block: it is open for every Q-block and never a
   top-k candidate.

Lengths: nQB = ceil(C / q_block) Q-blocks and nKB_b = ceil((cached_len_b + C)
/ page) blocks per sequence; any cached_len >= 0 and C >= 1.

When nC_b = 0 there is neither top-k nor local window.  The unscaled dot
product is used because a positive softmax scale does not change a ranking.

A second selection rule, the alpha-threshold ("max-threshold") reading of
the FlashPrefill-style selector the paper pairs with the union, keeps every
cached block whose score is within a margin of the row's best (see
``select_threshold_blocks``).

Parity: pinned (closed-form pooling, brute-force top-k with ties, needle
recall, popcount bounds; the threshold rule against top-k prefixes and its
limit cases) in tests/test_oracle.py.
"""
from __future__ import annotations

import math
from dataclasses import dataclass
from typing import List, Sequence

import numpy as np

from .bf16 import bf16_to_f64


@dataclass(frozen=True)
class EstimatorParams:
    top_frac: float
    sink_blocks: int = 1
    local_blocks: int = 4


def n_kv_blocks(cached_len: int, chunk_len: int, page: int) -> int:
    """nKB = ceil((cached_len + C) / page): every block holding a token."""
    return -(-(int(cached_len) + int(chunk_len)) // page)


def causal_block_end(cached_len: int, chunk_len: int, i: int, q_block: int,
                     page: int) -> int:
    """One past the block holding the last query of Q-block i (step 5)."""
    last = min((i + 1) * q_block, chunk_len) - 1
    return (int(cached_len) + last) // page + 1


def q_block_means(q_bits: np.ndarray, q_block: int) -> np.ndarray:
    """q [B, C, Hq, D] bf16 -> q_mean [B, Hq, nQB, D] float64, nQB = ceil(C/q_block)."""
    q = bf16_to_f64(q_bits)
    B, C, Hq, D = q.shape
    nqb = -(-C // q_block)
    out = np.zeros((B, Hq, nqb, D))
    for i in range(nqb):
        out[:, :, i, :] = q[:, i * q_block:min((i + 1) * q_block, C), :, :].mean(axis=1)
    return out


def k_block_means(k_pool_bits: np.ndarray, page_table: np.ndarray,
                  n_blocks: Sequence[int],
                  seq_len: Sequence[int] = None) -> np.ndarray:
    """Mean of each logical block's key rows, via the page table.

    Block j of sequence b is averaged over its rows r with page*j + r <
    seq_len[b] (all rows when ``seq_len`` is None).  Returns
    [B, Hkv, max_kv_blocks, D] float64; entries j >= n_blocks[b] are 0.
    """
    B, Hkv, maxkb = page_table.shape
    P, page_rows, D = k_pool_bits.shape
    out = np.zeros((B, Hkv, maxkb, D))
    for b in range(B):
        for h in range(Hkv):
            for j in range(int(n_blocks[b])):
                rows = page_rows if seq_len is None else \
                    min(page_rows, int(seq_len[b]) - page_rows * j)
                page = bf16_to_f64(k_pool_bits[page_table[b, h, j]][:rows])
                out[b, h, j] = page.mean(axis=0)
    return out


def block_scores(q_mean: np.ndarray, k_mean: np.ndarray,
                 n_cached: Sequence[int]) -> List[np.ndarray]:
    """s[b][h, i, j] = q_mean[b,h,i] . k_mean[b,kvh(h),j] for j < nC_b (float64)."""
    B, Hq, nqb, D = q_mean.shape
    Hkv = k_mean.shape[1]
    ratio = Hq // Hkv
    out = []
    for b in range(B):
        nc = int(n_cached[b])
        s = np.zeros((Hq, nqb, nc))
        for h in range(Hq):
            s[h] = q_mean[b, h] @ k_mean[b, h // ratio, :nc].T
        out.append(s)
    return out


def select_top_blocks(scores_row: np.ndarray, k: int) -> np.ndarray:
    """Indices of the k best blocks: score descending, then index ascending.

    ``scores_row`` is compared as given (callers pass float32 values).
    Numeric comparison makes -0.0 and +0.0 equal, so they tie and the
    smaller index wins.
    """
    n = scores_row.shape[0]
    idx = np.arange(n)
    order = np.lexsort((idx, -scores_row.astype(np.float64)))
    return np.sort(order[:k])


def n_selected(top_frac: float, n_cached: int) -> int:
    """k = ceil(top_frac * nC), computed in float32 like a kernel would."""
    if n_cached == 0:
        return 0
    return min(n_cached, int(math.ceil(float(np.float32(top_frac) * np.float32(n_cached)))))


def masks_from_scores(scores32: Sequence[np.ndarray], cached_len: Sequence[int],
                      chunk_len: int, page: int, q_block: int, words: int,
                      params: EstimatorParams) -> np.ndarray:
    """Step 4-5: float32 scores per sequence ([Hq, nQB, nC_b]) -> packed masks.

    Bit j&63 of word j>>6 of row (b,h,i) is M[b,h,i,j].
    """
    B = len(scores32)
    Hq, nqb = scores32[0].shape[:2]
    masks = np.zeros((B, Hq, nqb, words), dtype=np.uint64)
    for b in range(B):
        nc = int(cached_len[b]) // page
        k = n_selected(params.top_frac, nc)
        for h in range(Hq):
            for i in range(nqb):
                sel = set(select_top_blocks(scores32[b][h, i][:nc], k).tolist()) if k else set()
                sel |= set(range(min(params.sink_blocks, nc)))
                sel |= set(range(max(0, nc - params.local_blocks), nc))
                sel |= set(range(nc, causal_block_end(cached_len[b], chunk_len, i,
                                                      q_block, page)))
                for j in sel:
                    masks[b, h, i, j >> 6] |= np.uint64(1) << np.uint64(j & 63)
    return masks


def threshold_margin(alpha: float, temperature: float, sm_scale: float) -> np.float32:
    """The score margin of the alpha-threshold selector (a reading, below):
    ln(alpha) / (temperature * sm_scale) from the single-precision values of
    the three parameters, evaluated in double and rounded once to float32."""
    a, t, s = (float(np.float32(x)) for x in (alpha, temperature, sm_scale))
    return np.float32(math.log(a) / (t * s))


def select_threshold_blocks(scores_row: np.ndarray, margin: np.float32) -> np.ndarray:
    """Max-threshold selection (FlashPrefill-style, Sec. 4.1; the paper gives no
    formula, so this is a reading): keep block j when its estimated attention
    weight exp(temperature * sm_scale * (s_j - s_max)) is at least alpha, i.e.
    s_j >= s_max + margin with margin = ln(alpha) / (temperature * sm_scale).
    The sum s_max + margin is taken in float32, the precision the GPU scores
    are produced in, so both sides take the same decision."""
    s = np.asarray(scores_row, dtype=np.float32)
    if s.shape[0] == 0:
        return np.zeros(0, dtype=np.int64)
    thr = np.float32(s.max() + np.float32(margin))
    return np.nonzero(s >= thr)[0]


def masks_from_threshold(scores32: Sequence[np.ndarray], cached_len: Sequence[int],
                         chunk_len: int, page: int, q_block: int, words: int,
                         margin: np.float32, sink_blocks: int = 1,
                         local_blocks: int = 4) -> np.ndarray:
    """Like masks_from_scores, with the threshold selection of the cached blocks."""
    B = len(scores32)
    Hq, nqb = scores32[0].shape[:2]
    masks = np.zeros((B, Hq, nqb, words), dtype=np.uint64)
    for b in range(B):
        nc = int(cached_len[b]) // page
        for h in range(Hq):
            for i in range(nqb):
                sel = set(select_threshold_blocks(scores32[b][h, i][:nc], margin).tolist())
                sel |= set(range(min(sink_blocks, nc)))
                sel |= set(range(max(0, nc - local_blocks), nc))
                sel |= set(range(nc, causal_block_end(cached_len[b], chunk_len, i,
                                                      q_block, page)))
                for j in sel:
                    masks[b, h, i, j >> 6] |= np.uint64(1) << np.uint64(j & 63)
    return masks


def estimate_masks(q_bits: np.ndarray, k_pool_bits: np.ndarray,
                   page_table: np.ndarray, cached_len: Sequence[int],
                   page: int, q_block: int, chunk_len: int, words: int,
                   params: EstimatorParams, return_parts: bool = False,
                   k_mean: np.ndarray = None):
    """Full estimator -> packed masks uint64 [B, Hq, nQB, words].

    ``k_mean`` may carry block means pooled earlier (they do not depend on
    the chunk); blocks it does not cover must not be needed.
    """
    n_cached = [int(c) // page for c in cached_len]
    n_blocks = [n_kv_blocks(c, chunk_len, page) for c in cached_len]
    seq_len = [int(c) + chunk_len for c in cached_len]
    qm = q_block_means(q_bits, q_block)
    km = k_mean if k_mean is not None else k_block_means(k_pool_bits, page_table, n_blocks,
                                                         seq_len)
    sc = block_scores(qm, km, n_cached)
    masks = masks_from_scores([s.astype(np.float32) for s in sc], cached_len, chunk_len,
                              page, q_block, words, params)
    if return_parts:
        return masks, dict(q_mean=qm, k_mean=km, scores=sc)
    return masks
