"""The synthetic workloads, written as data.

Shapes follow the LLaMA-3.1-8B attention layer the paper measures on
(Sec. 4.1: 32 query heads, 8 KV heads, head_dim 128) with a 2048-token
chunk (the largest chunk of Table 5), plus one tiny GQA case that the CPU
oracle finishes in well under a second.

``rho`` is the weight of a seeded query direction shared by all tokens of a
(sequence, KV group): ``q = rho * mu + sqrt(1 - rho^2) * z`` with ``mu`` and
``z`` iid N(0, 1), so every element stays marginally N(0, 1).  With ``rho = 0``
the mean-pooled block scores are nearly independent across query blocks and
heads, and the two unions of Sec. 3.2 reopen ~95% of the cache at 128K; no
execution strategy can then be faster than dense.  The paper reports that
its masks keep 70.2% sparsity *after* both unions at RULER 128K (Sec. 4.4,
sparsity analysis), i.e. ~30% executed density.  ``rho`` below is the value
at which the 128K final chunk reaches that executed density (calibration
recorded in the design notes and checked by ``tests/test_synth.py``).
"""
from __future__ import annotations

import math
from dataclasses import dataclass, replace
from typing import Optional, Tuple

PAGE = 64  # KV block == page, tokens

# Query-direction weight that puts the 128K final chunk's executed cached
# density (after Q-block and intra-group union) at ~0.30.
RHO_CALIBRATED = 0.12


@dataclass(frozen=True)
class Workload:
    name: str
    seed: int
    batch: int
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    q_block: int
    chunk_len: int
    cached_lens: Tuple[int, ...]
    max_kv_blocks: int
    sm_scale: float
    page_size: int = PAGE
    mask_kind: str = "estimator"          # "estimator" | "bernoulli"
    top_frac: float = 0.0                  # estimator: keep ceil(top_frac * nC) blocks
    bernoulli_p: float = 0.0               # bernoulli: P(bit) over cached blocks
    sink_blocks: int = 1
    local_blocks: int = 4
    needles_per_kv_head: int = 0
    needle_beta: float = 2.0
    poison_tail: bool = False              # NaN in the rows of each last page past the end
    rho: float = 0.0
    q_prescale: float = 1.0
    group_size: int = 4                    # query heads per execution group
    description: str = ""

    # ---- derived -------------------------------------------------------
    @property
    def ratio(self) -> int:
        return self.num_q_heads // self.num_kv_heads

    @property
    def n_qblocks(self) -> int:
        return -(-self.chunk_len // self.q_block)

    @property
    def words(self) -> int:
        return (self.max_kv_blocks + 63) // 64

    def n_cached_blocks(self, b: int) -> int:
        return self.cached_lens[b] // self.page_size

    def n_kv_blocks(self, b: int) -> int:
        return -(-(self.cached_lens[b] + self.chunk_len) // self.page_size)

    def seq_len(self, b: int) -> int:
        return self.cached_lens[b] + self.chunk_len

    @property
    def num_groups(self) -> int:
        return self.num_q_heads // self.group_size

    def dense_flops(self) -> float:
        """Unmasked (query, key) pairs x 4*D, dense over the whole cache."""
        tot = 0.0
        C = self.chunk_len
        for b in range(self.batch):
            pairs = C * self.cached_lens[b] + C * (C + 1) / 2
            tot += self.num_q_heads * pairs * 4 * self.head_dim
        return tot


def _llama(name, seed, cached_lens, top_frac, needles, description, **kw):
    chunk = kw.pop("chunk_len", 2048)
    nkb_max = max(-(-(c + chunk) // PAGE) for c in cached_lens)
    return Workload(
        name=name, seed=seed, batch=len(cached_lens), num_q_heads=32,
        num_kv_heads=kw.pop("num_kv_heads", 8), head_dim=128, q_block=128, chunk_len=chunk,
        cached_lens=tuple(cached_lens), max_kv_blocks=kw.pop("max_kv_blocks", nkb_max),
        sm_scale=1.0 / math.sqrt(128.0), mask_kind="estimator",
        top_frac=top_frac, needles_per_kv_head=needles, rho=RHO_CALIBRATED,
        description=description, **kw)


WORKLOADS = {
    # batch 1, 4 query heads on 1 KV head, D=64, 1024 cached + 256-token chunk;
    # Bernoulli(0.25) masks over the 16 cached blocks + sink + chunk-causal.
    "tiny_gqa_1k": Workload(
        name="tiny_gqa_1k", seed=1, batch=1, num_q_heads=4, num_kv_heads=1,
        head_dim=64, q_block=64, chunk_len=256, cached_lens=(1024,),
        max_kv_blocks=20, sm_scale=1.0, mask_kind="bernoulli",
        bernoulli_p=0.25, rho=0.0, q_prescale=1.0 / 8.0,
        description="tiny GQA chunk, iid bf16, Q pre-scaled by 1/sqrt(64)"),
    "llama8b_32k": _llama(
        "llama8b_32k", 2, (30720,), 0.10, 8,
        "LLaMA-3.1-8B layer, 30720 cached + 2048 chunk, top 10%"),
    "llama8b_128k_final": _llama(
        "llama8b_128k_final", 3, (129024,), 0.05, 32,
        "LLaMA-3.1-8B layer, 128K final chunk: 129024 cached + 2048, top 5%"),
    "batched_ragged_4seq": _llama(
        "batched_ragged_4seq", 4, (16384, 32768, 65536, 126976), 0.08, 0,
        "4 sequences sharing one page pool, top 8%, ragged tables"),
    # Qwen3-30B-A3B-like attention layer (32 query heads on 4 KV heads, GQA 8:1):
    # execution groups of 4 heads are sub-groups of a KV group, so every KV
    # head has two tables (App. B.1).
    "qwen3_30b_128k_final": _llama(
        "qwen3_30b_128k_final", 6, (129024,), 0.05, 32,
        "Qwen3-30B-A3B-like layer (32/4 heads), 128K final chunk, top 5%, sub-groups of 4",
        num_kv_heads=4),
    # lengths that are not multiples of 64 or of q_block: a partial last
    # Q-block, a block holding both cached and chunk tokens, a partial last
    # page whose rows past the sequence end hold NaN, and a sequence with no
    # cached tokens.
    "tiny_unaligned": Workload(
        name="tiny_unaligned", seed=7, batch=3, num_q_heads=8, num_kv_heads=2,
        head_dim=64, q_block=64, chunk_len=200, cached_lens=(1000, 37, 0),
        max_kv_blocks=20, sm_scale=1.0 / 8.0, mask_kind="estimator", top_frac=0.25,
        poison_tail=True,
        description="unaligned lengths: 3 sequences (1000, 37, 0 cached) + 200-token chunk"),
    "llama8b_unaligned": _llama(
        "llama8b_unaligned", 8, (100001, 4999, 0), 0.05, 8,
        "LLaMA-3.1-8B layer, unaligned: 100001 / 4999 / 0 cached + 2000-token chunk",
        chunk_len=2000, poison_tail=True),
    "sweep_128k_64chunks": _llama(
        "sweep_128k_64chunks", 5, (129024,), 0.05, 64,
        "131072-token sequence prefilled in 64 chunks of 2048, top 5%",
        max_kv_blocks=2048),
}

SWEEP_CHUNKS = 64


def get_workload(name: str, **overrides) -> Workload:
    w = WORKLOADS[name]
    return replace(w, **overrides) if overrides else w


def sweep_chunk(c: int, base: Optional[Workload] = None) -> Workload:
    """The sweep workload as seen by chunk ``c`` (cached = 2048 * c)."""
    base = base or WORKLOADS["sweep_128k_64chunks"]
    return replace(base, cached_lens=(base.chunk_len * c,))
