"""Seeded generators.  See the package docstring for what they promise."""
from __future__ import annotations

import math
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass, replace
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

from .configs import Workload, SWEEP_CHUNKS, sweep_chunk

# stream tags for numpy.random.SeedSequence([seed, tag, ...])
_T_K, _T_V, _T_Q, _T_MU, _T_PERM, _T_NEEDLE, _T_MASK = 1, 2, 3, 4, 5, 6, 7

_POOL = None


def _pool() -> ThreadPoolExecutor:
    global _POOL
    if _POOL is None:
        _POOL = ThreadPoolExecutor(8)
    return _POOL


def _rng(*key: int) -> np.random.Generator:
    return np.random.default_rng(np.random.SeedSequence([int(k) for k in key]))


# ---------------------------------------------------------------------------
# bf16 bit patterns
# ---------------------------------------------------------------------------
def bf16_round(x: np.ndarray) -> np.ndarray:
    """float32 -> bf16 bits, round to nearest, ties to even (finite inputs)."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    lsb = (u >> np.uint32(16)) & np.uint32(1)
    r = u + np.uint32(0x7FFF)
    r += lsb
    r >>= np.uint32(16)
    return r.astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def _normal_bf16(shape, *key, scale: float = 1.0) -> np.ndarray:
    x = _rng(*key).standard_normal(shape, dtype=np.float32)
    if scale != 1.0:
        x *= np.float32(scale)
    return bf16_round(x)


# ---------------------------------------------------------------------------
# masks / tables / scores used directly as inputs by tests
# ---------------------------------------------------------------------------
def pack_bits(bits: np.ndarray, words: int) -> np.ndarray:
    """bool [..., n] -> uint64 [..., words]; bit j&63 of word j>>6 is column j."""
    n = bits.shape[-1]
    assert n <= words * 64
    pad = np.zeros(bits.shape[:-1] + (words * 64,), dtype=bool)
    pad[..., :n] = bits
    by = np.packbits(pad, axis=-1, bitorder="little")
    return np.ascontiguousarray(by).view("<u8").reshape(bits.shape[:-1] + (words,))


def random_masks(seed: int, batch: int, num_q_heads: int, n_qblocks: int,
                 q_block: int, page: int, cached_lens: Sequence[int],
                 chunk_len: int, words: int, p: float, sink_blocks: int = 1,
                 causal: bool = True) -> np.ndarray:
    """Bernoulli(p) bits over the full cached blocks, plus sink and chunk-causal bits.

    ``cached_lens`` are token counts.  The chunk-causal bits of Q-block i
    run from block cached_len // page up to the block holding the chunk's
    token min((i+1)*q_block, C) - 1.  Returns uint64 ``[B, Hq, nQB, words]``.
    This is the mask recipe of the tiny workload, and (with other ``p``) an
    input family for table tests.
    """
    rng = _rng(seed, _T_MASK)
    out = np.zeros((batch, num_q_heads, n_qblocks, words), dtype=np.uint64)
    for b in range(batch):
        cl = int(cached_lens[b])
        nc = cl // page
        nkb = -(-(cl + chunk_len) // page)
        bits = np.zeros((num_q_heads, n_qblocks, nkb), dtype=bool)
        if nc:
            bits[:, :, :nc] = rng.random((num_q_heads, n_qblocks, nc)) < p
            bits[:, :, :min(sink_blocks, nc)] = True
        if causal:
            for i in range(n_qblocks):
                last = cl + min((i + 1) * q_block, chunk_len) - 1
                bits[:, i, nc:last // page + 1] = True
        out[b] = pack_bits(bits, words)
    return out


def random_tables(seed: int, batch: int, num_groups: int,
                  cached_blocks: Sequence[int], chunk_blocks: int,
                  density: float) -> Tuple[np.ndarray, np.ndarray]:
    """CSR tables with a fixed fraction of cached blocks plus every chunk block.

    Rows are ordered (b-major, g-minor); entries are logical block ids in
    ascending order.  Used for matched-density attention runs.
    """
    rng = _rng(seed, _T_MASK, 99)
    rows: List[np.ndarray] = []
    for b in range(batch):
        nc = int(cached_blocks[b])
        for _ in range(num_groups):
            k = int(round(density * nc))
            sel = np.sort(rng.choice(nc, size=k, replace=False)) if k else np.zeros(0, np.int64)
            rows.append(np.concatenate([sel, np.arange(nc, nc + chunk_blocks)]).astype(np.int32))
    indptr = np.zeros(len(rows) + 1, dtype=np.int32)
    indptr[1:] = np.cumsum([len(r) for r in rows])
    return indptr, np.concatenate(rows).astype(np.int32)


def tied_scores(seed: int, rows: int, cols: int, n_distinct: int = 7) -> np.ndarray:
    """float32 scores drawn from a handful of values, so ranks tie constantly.

    Includes -0.0 and +0.0 among the values so that sign-of-zero handling is
    exercised as well as the index tie-break.
    """
    rng = _rng(seed, _T_MASK, 7)
    vals = np.concatenate([np.array([0.0, -0.0], np.float32),
                           rng.standard_normal(max(n_distinct - 2, 1)).astype(np.float32)])
    return vals[rng.integers(0, len(vals), size=(rows, cols))].astype(np.float32)


# ---------------------------------------------------------------------------
# workload inputs
# ---------------------------------------------------------------------------
def _page_assignment(w: Workload, nkb: Sequence[int]) -> Tuple[np.ndarray, int]:
    """page_table [B, Hkv, max_kv_blocks] (int32, -1 unused) and pool size."""
    B, Hkv = w.batch, w.num_kv_heads
    total = int(sum(Hkv * n for n in nkb))
    perm = _rng(w.seed, _T_PERM).permutation(total).astype(np.int32)
    pt = np.full((B, Hkv, w.max_kv_blocks), -1, dtype=np.int32)
    off = 0
    for b in range(B):
        for h in range(Hkv):
            pt[b, h, :nkb[b]] = perm[off:off + nkb[b]]
            off += nkb[b]
    return pt, total


def _gen_q(w: Workload, b: int, tag: int, mu: Optional[np.ndarray]) -> np.ndarray:
    """Q of one sequence/chunk, [C, Hq, D] bf16 bits."""
    C, Hq, D = w.chunk_len, w.num_q_heads, w.head_dim
    z = _rng(w.seed, _T_Q, b, tag).standard_normal((C, Hq, D), dtype=np.float32)
    if w.rho:
        ratio = w.ratio
        mu_h = np.repeat(mu, ratio, axis=0)          # [Hq, D]
        z *= np.float32(math.sqrt(1.0 - w.rho * w.rho))
        z += np.float32(w.rho) * mu_h[None, :, :]
    if w.q_prescale != 1.0:
        z *= np.float32(w.q_prescale)
    return bf16_round(z)


def _mu(w: Workload, b: int) -> np.ndarray:
    return _rng(w.seed, _T_MU, b).standard_normal((w.num_kv_heads, w.head_dim)).astype(np.float32)


def _needle_direction(q_bits: np.ndarray, h: int, i: int, q_block: int) -> np.ndarray:
    """Unit vector along the mean of the bf16 query rows of Q-block i, head h."""
    rows = bf16_bits_to_f32(q_bits[i * q_block:(i + 1) * q_block, h, :]).astype(np.float64)
    m = rows.mean(axis=0)
    return (m / np.linalg.norm(m)).astype(np.float32)


def _fill_kv(w: Workload, pt: np.ndarray, total: int, nkb: Sequence[int],
             needle_fn=None) -> Tuple[np.ndarray, np.ndarray]:
    """K/V pools, each [P, page, D] bf16 bits; K/V iid N(0,1)."""
    page, D = w.page_size, w.head_dim
    k_pool = np.empty((total, page, D), dtype=np.uint16)
    v_pool = np.empty((total, page, D), dtype=np.uint16)
    jobs = [(b, h) for b in range(w.batch) for h in range(w.num_kv_heads)]

    def one(job):
        b, h = job
        n = nkb[b]
        kb = _normal_bf16((n, page, D), w.seed, _T_K, b, h)
        vb = _normal_bf16((n, page, D), w.seed, _T_V, b, h)
        if needle_fn is not None:
            needle_fn(b, h, kb)
        ids = pt[b, h, :n]
        k_pool[ids] = kb
        v_pool[ids] = vb

    list(_pool().map(one, jobs))
    return k_pool, v_pool


def _apply_needle(kb: np.ndarray, j: int, u: np.ndarray, beta: float) -> None:
    blk = bf16_bits_to_f32(kb[j]) + np.float32(beta) * u[None, :]
    kb[j] = bf16_round(blk)


BF16_QNAN = np.uint16(0x7FC0)


def v_pages_transposed(v_pool: np.ndarray) -> np.ndarray:
    """The V pool with every page transposed to ``[D, page]`` (head dimension
    major, tokens contiguous), the same values: the library's optional
    transposed V layout.

    The seeded V data and the oracle use token-major pages ``[page, D]``, the
    paper's layout and the library's default; a caller that selects the
    transposed layout hands over this copy."""
    return np.ascontiguousarray(v_pool.transpose(0, 2, 1))


def poison_past_end(w: Workload, k_pool: np.ndarray, v_pool: np.ndarray,
                    pt: np.ndarray) -> None:
    """NaN in every K and V row of a sequence's last page past its end.

    Those rows are not part of the sequence (a paged cache leaves them
    unwritten); filling them with NaN makes any read that lets them into a
    result visible."""
    page = w.page_size
    for b in range(w.batch):
        n = w.n_kv_blocks(b)
        valid = w.seq_len(b) - page * (n - 1)
        if valid == page:
            continue
        for kvh in range(w.num_kv_heads):
            pid = pt[b, kvh, n - 1]
            k_pool[pid, valid:, :] = BF16_QNAN
            v_pool[pid, valid:, :] = BF16_QNAN


def make_inputs(w: Workload) -> Dict[str, object]:
    """All inputs of one chunk step of workload ``w`` (not the sweep)."""
    B, Hkv, ratio = w.batch, w.num_kv_heads, w.ratio
    nkb = [w.n_kv_blocks(b) for b in range(B)]
    ncb = [w.n_cached_blocks(b) for b in range(B)]
    pt, total = _page_assignment(w, nkb)
    mus = [_mu(w, b) if w.rho else None for b in range(B)]
    q = np.stack([_gen_q(w, b, 0, mus[b]) for b in range(B)])  # [B, C, Hq, D]

    needles: List[Tuple[int, int, int, int, int]] = []
    if w.needles_per_kv_head:
        rng = _rng(w.seed, _T_NEEDLE)
        for b in range(B):
            nc = ncb[b]
            lo, hi = w.sink_blocks, nc - w.local_blocks
            if hi - lo < w.needles_per_kv_head:
                continue                  # too short a cache for needles
            for kvh in range(Hkv):
                js = rng.choice(np.arange(lo, hi), size=w.needles_per_kv_head, replace=False)
                for j in np.sort(js):
                    h = kvh * ratio + int(rng.integers(ratio))
                    i = int(rng.integers(w.n_qblocks))
                    needles.append((b, kvh, int(j), h, i))

    by_bh: Dict[Tuple[int, int], list] = {}
    for (b, kvh, j, h, i) in needles:
        by_bh.setdefault((b, kvh), []).append((j, h, i))

    def needle_fn(b, kvh, kb):
        for (j, h, i) in by_bh.get((b, kvh), []):
            _apply_needle(kb, j, _needle_direction(q[b], h, i, w.q_block), w.needle_beta)

    k_pool, v_pool = _fill_kv(w, pt, total, nkb, needle_fn if needles else None)
    if w.poison_tail:
        poison_past_end(w, k_pool, v_pool, pt)

    masks = None
    if w.mask_kind == "bernoulli":
        masks = random_masks(w.seed, B, w.num_q_heads, w.n_qblocks, w.q_block,
                             w.page_size, w.cached_lens, w.chunk_len, w.words,
                             w.bernoulli_p, w.sink_blocks)
    return dict(workload=w, q=q, k_pool=k_pool, v_pool=v_pool, page_table=pt,
                cached_len=np.array(w.cached_lens, dtype=np.int32),
                masks=masks, needles=needles)


# ---------------------------------------------------------------------------
# the 64-chunk sweep: one pool for the whole sequence, Q generated per chunk
# ---------------------------------------------------------------------------
@dataclass
class SweepSequence:
    base: Workload
    k_pool: np.ndarray
    v_pool: np.ndarray
    page_table_full: np.ndarray       # [1, Hkv, 2048]
    needles: List[Tuple[int, int, int, int, int, int]]  # (b, kvh, j, h, target chunk, i)
    mu: Optional[np.ndarray]
    n_chunks: int = SWEEP_CHUNKS

    def q_chunk(self, c: int) -> np.ndarray:
        return _gen_q(self.base, 0, c, self.mu)[None]

    def inputs(self, c: int) -> Dict[str, object]:
        w = sweep_chunk(c, self.base)
        nkb = w.n_kv_blocks(0)
        pt = self.page_table_full.copy()
        pt[:, :, nkb:] = -1
        return dict(workload=w, q=self.q_chunk(c), k_pool=self.k_pool,
                    v_pool=self.v_pool, page_table=pt,
                    cached_len=np.array(w.cached_lens, dtype=np.int32), masks=None,
                    needles=[(b, kvh, j, h, i) for (b, kvh, j, h, tc, i) in self.needles if tc == c])


def make_sweep_sequence(w: Workload, n_chunks: int = SWEEP_CHUNKS) -> SweepSequence:
    """Whole-sequence K/V pool for a chunked prefill of ``n_chunks`` chunks.

    Needles: ``needles_per_kv_head`` blocks per KV head drawn without
    replacement from blocks [1, chunk_blocks * (n_chunks - 1)); each targets a
    (head of the group, Q-block) of a chunk strictly after its own.
    """
    assert w.batch == 1
    cb = w.chunk_len // w.page_size
    nkb_total = cb * n_chunks
    full = replace(w, cached_lens=(nkb_total * w.page_size - w.chunk_len,))
    pt, total = _page_assignment(full, [nkb_total])
    mu = _mu(w, 0) if w.rho else None
    rng = _rng(w.seed, _T_NEEDLE)
    needles = []
    for kvh in range(w.num_kv_heads):
        js = np.sort(rng.choice(np.arange(1, cb * (n_chunks - 1)),
                                size=w.needles_per_kv_head, replace=False))
        for j in js:
            own = int(j) // cb
            tc = int(rng.integers(own + 1, n_chunks))
            h = kvh * w.ratio + int(rng.integers(w.ratio))
            i = int(rng.integers(w.n_qblocks))
            needles.append((0, kvh, int(j), h, tc, i))
    # needle directions need the target chunk's Q; build them one chunk at a time
    dirs: Dict[Tuple[int, int], np.ndarray] = {}
    for tc in sorted({n[4] for n in needles}):
        qc = _gen_q(w, 0, tc, mu)
        for (_, kvh, j, h, t, i) in needles:
            if t == tc:
                dirs[(kvh, j)] = _needle_direction(qc, h, i, w.q_block)
        del qc

    def needle_fn(b, kvh, kb):
        for (_, nh, j, _h, _tc, _i) in needles:
            if nh == kvh:
                _apply_needle(kb, j, dirs[(kvh, j)], w.needle_beta)

    k_pool, v_pool = _fill_kv(full, pt, total, [nkb_total], needle_fn)
    return SweepSequence(base=w, k_pool=k_pool, v_pool=v_pool, page_table_full=pt,
                         needles=needles, mu=mu, n_chunks=n_chunks)
