"""Seeded synthetic inputs for the chunked-prefill block-union attention path.

This module only *generates* inputs.  It is shared by the CPU oracle's tests
and by the GPU path's tests and benchmark, so it deliberately contains none of
the method's arithmetic (no pooling of K blocks for scoring, no top-k, no
unions, no attention).  Everything it returns is a plain NumPy array:

* bf16 tensors are returned as ``uint16`` bit patterns (round-to-nearest-even
  from float32 draws of ``numpy.random.default_rng``, PCG64);
* the KV cache is KV-head-major and paged: logical block ``j`` of
  ``(sequence b, KV head kvh)`` lives in physical page
  ``page_table[b, kvh, j]`` of ``k_pool`` / ``v_pool`` (``[P, page, D]``),
  which is the layout of the paper's zero-copy execution (Sec. 3.3, Fig. 4
  and App. B.2: one contiguous ``[block, D]`` region per
  (batch, KV head, block) triple); the GPU library reads V pages in this
  layout by default, or transposed (``v_pages_transposed``: ``[P, D, page]``)
  when a caller selects that layout;
* physical page ids are a seeded permutation of all (b, kvh, j) triples, so
  the pool holds exactly the pages the workload needs.

Random choices that belong to the *workload* (Bernoulli masks of the tiny
case, needle positions and targets, the shared query direction) are drawn
here and handed to both sides as inputs.
"""
from .configs import Workload, WORKLOADS, get_workload, sweep_chunk  # noqa: F401
from .gen import (  # noqa: F401
    bf16_round,
    bf16_bits_to_f32,
    make_inputs,
    make_sweep_sequence,
    SweepSequence,
    random_masks,
    random_tables,
    tied_scores,
    v_pages_transposed,
)
