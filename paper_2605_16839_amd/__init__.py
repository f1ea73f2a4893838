"""MI355X-native chunked-prefill block-union attention (CompactAttention).

The compute path lives in ``libcompactattn.so`` (hand-written HIP for gfx950,
C ABI in ``include/compactattn.h``); this package is its Python binding.
"""
from .binding import (  # noqa: F401
    CAError, Problem, load, abi_version, check_problem, pool_q_blocks, pool_k_blocks,
    block_scores, select_blocks, estimate_masks, tables_workspace_bytes,
    build_block_tables, attention_workspace_bytes, chunk_attention,
    dense_paged_chunk_attention, validate_tables, block_sparse_tables_workspace_bytes,
    build_block_sparse_tables, block_sparse_chunk_attention, gather_selected_pages,
    packed_chunk_attention, estimate_masks_threshold, select_blocks_threshold, estimate_tables,
    build_block_tables_noalloc, check_tables_host,
    EXPORTED,
    LIB_PATH,
    DEBUG_LIB_PATH,
    V_TOKEN_MAJOR,
    V_TRANSPOSED,
)
