"""CPU reference ("oracle") for the chunked-prefill block-union attention path.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import, call or
link this package: only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` use it.  It shares no code with the HIP
library or its Python binding, and it never takes an input produced by them.

It is a plain, slow, float64 restatement of what the paper defines:

* ``estimator``  -- the mean-pooled block-score selector that stands in for
  the paper's pluggable pattern search (Sec. 3.1/3.2 only require *some*
  lightweight block-level selector; this one is a reading, see its header);
* ``tables``     -- Q-block union, intra-group union and the per-group table
  T[b,g] (Sec. 3.2, the three displayed equations), emitted as CSR
  ``kv_indptr`` / ``kv_indices`` (Sec. 3.3, App. B.2);
* ``attention``  -- attention of every chunk query over exactly the blocks of
  its group's table, after an explicit gather of those pages (the copy the
  zero-copy design avoids, Sec. 3.3), with causal masking in absolute
  positions (App. B.2, last paragraph); ``block_sparse_attention`` runs the
  same softmax per (head, Q-block) mask row without any union, the block-
  sparse execution the paper compares against (Sec. 4.4).

Parity status of each function is stated in its docstring; every function is
pinned by ``tests/test_oracle.py`` against properties that the paper or the
mathematics fix.
"""
from .bf16 import bf16_to_f64  # noqa: F401
from .estimator import (  # noqa: F401
    q_block_means, k_block_means, block_scores, select_top_blocks,
    masks_from_scores, n_selected, estimate_masks, EstimatorParams, threshold_margin,
    select_threshold_blocks, masks_from_threshold, n_kv_blocks, causal_block_end,
)
from .tables import unpack_masks, block_tables, tables_to_csr, union_densities  # noqa: F401
from .attention import (  # noqa: F401
    gather_selected, attention_rows, chunk_attention, dense_tables, block_sparse_attention,
)
