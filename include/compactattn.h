/*
 * compactattn.h -- C ABI of the chunked-prefill block-union attention path
 * (CompactAttention, arXiv 2605.16839) for AMD Instinct MI355X (gfx950).
 *
 * The path, per chunk of a chunked prefill:
 *
 *   1. estimate   2D block masks M[b,h,i,j] from mean-pooled Q and K blocks
 *                 (a lightweight block-level selector; the paper accepts any
 *                 such pattern search, Sec. 3.1 and Sec. 3.2 first paragraph);
 *   2. tables     Q-block union, intra-group union and the per-group table
 *                 T[b,g] = { j : exists h in H(g), exists i, M[b,h,i,j] = 1 }
 *                 (Sec. 3.2, the three displayed equations), as CSR
 *                 kv_indptr / kv_indices (Sec. 3.3, App. B.2);
 *   3. attention  dense attention of every chunk query over exactly the blocks
 *                 of its group's table, read in place from the paged pool
 *                 (zero-copy, Sec. 3.3), causal in absolute positions
 *                 (App. B.2, last paragraph);
 *   plus a dense paged baseline (every block of the sequence).
 *
 * Conventions shared by every call
 * --------------------------------
 * - All pointers are DEVICE memory unless the name ends in _host.  The
 *   caller allocates and owns every buffer; the library allocates nothing
 *   and keeps no state besides a thread-local error string, the scratch
 *   array of ca_build_block_tables_noalloc and a launch counter that tags
 *   the split attention launches.
 * - bf16 tensors are passed as uint16_t bit patterns.  All tensors are dense
 *   row-major (C order) with the shapes given below.  The bf16 and fp32
 *   tensors (q, k_pool, v_pool, out, q_mean, k_mean, scores, packed pools)
 *   must start on a 16-byte boundary (CA_ERR_UNALIGNED otherwise; any
 *   hipMalloc or torch allocation does), and so must the attention
 *   workspace (CA_ERR_WORKSPACE).
 * - KV cache: KV-head-major pages (Sec. 3.3, Fig. 4; App. B.2).  Logical
 *   block j of (sequence b, KV head kvh) is physical page
 *   page_table[b, kvh, j] of k_pool and v_pool; one page id addresses the K
 *   page and the V page.  k_pool is [P, page_size, head_dim] (token-major
 *   pages, one [block, D] region per page, as the paper's cache).  v_pool
 *   has the layout named by ca_problem.v_layout:
 *     CA_V_TOKEN_MAJOR (0, the default of a zeroed struct): [P, page_size,
 *       head_dim], the same token-major pages as K (the paper's layout; a
 *       cache writer appends a token's V as one contiguous row).  The kernel
 *       reads each V^T operand fragment with two gfx950 transpose reads;
 *     CA_V_TRANSPOSED (1): [P, head_dim, page_size], every V page stored
 *       dimension-major with the page's tokens contiguous (the layout of
 *       vLLM's original paged V cache); each V^T fragment is one 16-byte
 *       LDS read.
 *   Only the attention entry points read v_pool.  page_table is int32
 *   [B, Hkv, max_kv_blocks]; entries at j >= nKB_b are ignored.
 * - Per sequence b: cached_len[b] tokens are already in the cache and the
 *   chunk adds chunk_len tokens (any lengths).  Chunk token t sits at
 *   absolute position cached_len[b] + t, key r of block j at
 *   page_size * j + r.  nC_b = floor(cached_len[b] / page_size) blocks are
 *   full of cached tokens (the candidates of the selector); the sequence
 *   occupies nKB_b = ceil((cached_len[b] + chunk_len) / page_size) blocks.
 *   A block holding both cached and chunk tokens counts as a chunk block.
 *   The tokens of a sequence's last page past its end (cached_len[b] +
 *   chunk_len: K rows, V columns) are not part of it and may hold anything,
 *   NaN included: pooling does not read them and attention gives them no
 *   weight.  Every page of the pool is nevertheless read whole, so it must
 *   be allocated whole (page_size tokens).
 * - Query head h belongs to KV head h / (Hq / Hkv) and to execution group
 *   h / group_size (contiguous heads, Sec. 3.2 and App. B.1: the KV group by
 *   default, or 4-head sub-groups of a larger KV group).  group_size must
 *   divide Hq / Hkv.
 * - Masks are uint64 [B, Hq, nQB, W], W = ceil(max_kv_blocks / 64),
 *   nQB = ceil(chunk_len / q_block) (the last Q-block may hold fewer than
 *   q_block queries): bit (j & 63) of word (j >> 6) of row (b,h,i) is
 *   M[b,h,i,j].  Only blocks j < nKB_b are meaningful.
 * - Tables: kv_indptr int32 [B*G + 1] and kv_indices int32 (capacity
 *   B*G*max_kv_blocks); row r = b*G + g lists T[b,g] as ascending LOGICAL
 *   block ids in kv_indices[kv_indptr[r] .. kv_indptr[r+1]).
 * - `stream` is a hipStream_t (NULL = the default stream).  Every call only
 *   enqueues work on it and returns without synchronising, except
 *   ca_validate_tables (and the attention calls of the debug build, see
 *   ca_check_tables_host).
 * - Argument and shape errors are reported before anything is enqueued; a
 *   failed launch returns CA_ERR_HIP with the HIP error text available from
 *   ca_last_error_detail().
 */
#ifndef COMPACTATTN_H
#define COMPACTATTN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define CA_ABI_VERSION 6

typedef enum ca_status {
  CA_OK = 0,
  CA_ERR_NULL = 1,          /* a required pointer is NULL                       */
  CA_ERR_SHAPE = 2,         /* a size is out of range or inconsistent           */
  CA_ERR_UNALIGNED = 3,     /* a tensor pointer is not 16-byte aligned          */
  CA_ERR_GROUP = 4,         /* group_size does not divide Hq / Hkv              */
  CA_ERR_WORKSPACE = 5,     /* workspace missing or too small                   */
  CA_ERR_UNSUPPORTED = 6,   /* head_dim / page_size / q_block not built for     */
  CA_ERR_INVALID_TABLE = 7, /* a malformed table or page id (table checks)      */
  CA_ERR_HIP = 8            /* a HIP runtime call or kernel launch failed       */
} ca_status;

typedef struct ca_problem {
  int32_t batch;             /* B >= 1                                          */
  int32_t num_q_heads;       /* Hq                                              */
  int32_t num_kv_heads;      /* Hkv, divides Hq                                 */
  int32_t head_dim;          /* D, 64 or 128                                    */
  int32_t page_size;         /* tokens per KV block == page; must be 64         */
  int32_t q_block;           /* query block of the masks: 64 or 128             */
  int32_t chunk_len;         /* C >= 1, any length                              */
  int32_t max_kv_blocks;     /* row stride of page_table, >= max_b nKB_b, <= 16384 */
  const int32_t* cached_len_host; /* HOST [B]: >= 0, any length                 */
  const int32_t* cached_len;      /* DEVICE [B]: the same values                */
  int32_t v_layout;          /* CA_V_TOKEN_MAJOR or CA_V_TRANSPOSED (v_pool)   */
} ca_problem;

/* ca_problem.v_layout: layout of the V pages of v_pool (see the file header). */
#define CA_V_TOKEN_MAJOR 0   /* [P, page_size, head_dim], as the K pages        */
#define CA_V_TRANSPOSED 1    /* [P, head_dim, page_size]                         */

int ca_abi_version(void);
const char* ca_status_string(ca_status s);
/* Thread-local detail of the last error returned on this thread ("" if none). */
const char* ca_last_error_detail(void);

/* Host-only validation of a problem (and of group_size if > 0); enqueues
 * nothing and needs no GPU.  Every entry point below performs it first. */
ca_status ca_check_problem(const ca_problem* p, int32_t group_size);

/* ------------------------------------------------------------------------
 * 1. Estimator (the selector; see the file header).  Stage by stage:
 *    q_mean[b,h,i]   = mean of the query rows of Q-block i, head h (the
 *                      last Q-block's mean is over the rows it holds)
 *    k_mean[b,kvh,j] = mean of the key rows of block j before the sequence
 *                      end (all page_size rows but in a partial last block)
 *    scores[b,h,i,j] = q_mean[b,h,i] . k_mean[b,kvh(h),j], j < nC_b
 *    masks: top k = ceil(top_frac * nC_b) (float32 product, at most nC_b)
 *           cached blocks per row by score descending then j ascending
 *           (-0.0 ranks equal to +0.0), OR sink blocks {0..sink_blocks-1},
 *           OR the local window {nC_b-local_blocks .. nC_b-1}, OR the
 *           chunk-causal blocks {nC_b .. e_i - 1}, e_i = 1 + the block that
 *           holds the last query of Q-block i, i.e.
 *           e_i = (cached_len + min((i+1)*q_block, C) - 1) / page_size + 1
 *           (nC_b + (i+1)*q_block/page_size for aligned lengths), all
 *           clipped to [0, nKB_b); every other bit of the row is 0.
 * Pooling and scores accumulate in float32.
 * ---------------------------------------------------------------------- */

/* q bf16 [B, C, Hq, D] -> q_mean fp32 [B, Hq, nQB, D]. */
ca_status ca_pool_q_blocks(const ca_problem* p, const uint16_t* q, float* q_mean,
                           void* stream);

/* k_mean fp32 [B, Hkv, max_kv_blocks, D]: blocks j in [first_block, nKB_b) of
 * every sequence are (re)computed from k_pool; the others are left untouched,
 * so a caller that keeps k_mean across chunks passes first_block = the number
 * of blocks that were full when earlier chunks pooled them (a block pooled
 * while partial has to be pooled again; min_b nC_b is always safe). */
ca_status ca_pool_k_blocks(const ca_problem* p, const uint16_t* k_pool,
                           const int32_t* page_table, int32_t first_block,
                           float* k_mean, void* stream);

/* scores fp32 [B, Hq, nQB, max_kv_blocks]; only j < nC_b is written. */
ca_status ca_block_scores(const ca_problem* p, const float* q_mean,
                          const float* k_mean, float* scores, void* stream);

/* scores (as above, finite values) -> masks uint64 [B, Hq, nQB, W]. */
ca_status ca_select_blocks(const ca_problem* p, const float* scores, float top_frac,
                           int32_t sink_blocks, int32_t local_blocks,
                           uint64_t* masks, void* stream);

/* All four stages in order. */
ca_status ca_estimate_masks(const ca_problem* p, const uint16_t* q,
                            const uint16_t* k_pool, const int32_t* page_table,
                            float top_frac, int32_t sink_blocks, int32_t local_blocks,
                            int32_t k_mean_first_block, float* q_mean, float* k_mean,
                            float* scores, uint64_t* masks, void* stream);

/* 1b. Alpha-threshold selection (the FlashPrefill-style "max-threshold"
 *    selector the paper pairs with the union, Sec. 4.1; the paper gives no
 *    formula, so this is a reading).  Per mask row (b,h,i), a cached block j
 *    is kept when its estimated attention weight relative to the row's best,
 *    exp(temperature * sm_scale * (s_j - s_max)), is at least alpha:
 *        s_j >= s_max + margin,  margin = ln(alpha) / (temperature * sm_scale)
 *    with s = the block scores (ca_block_scores), margin computed in double from the
 *    single-precision parameters and rounded once to float, and the sum
 *    s_max + margin taken in float.  Sink, local and chunk-causal bits as in
 *    ca_select_blocks.  alpha in (0, 1], temperature > 0, sm_scale > 0 (else
 *    CA_ERR_SHAPE).  ca_estimate_masks_threshold = pooling + scores + this.
 * ---------------------------------------------------------------------- */
ca_status ca_select_blocks_threshold(const ca_problem* p, const float* scores, float alpha,
                                    float temperature, float sm_scale, int32_t sink_blocks,
                                    int32_t local_blocks, uint64_t* masks, void* stream);

ca_status ca_estimate_masks_threshold(const ca_problem* p, const uint16_t* q,
                                      const uint16_t* k_pool, const int32_t* page_table,
                                      float alpha, float temperature, float sm_scale,
                                      int32_t sink_blocks, int32_t local_blocks,
                                      int32_t k_mean_first_block, float* q_mean,
                                      float* k_mean, float* scores, uint64_t* masks,
                                      void* stream);

/* ------------------------------------------------------------------------
 * 2. Block tables (Sec. 3.2): bitwise OR over the nQB mask rows of every
 *    head of each group, compaction of the set bits j < nKB_b into the CSR
 *    pair.  Integer only; deterministic (no atomics on the output).
 *    Workspace: ca_tables_workspace_bytes(p, group_size) bytes of device
 *    memory, contents irrelevant on entry.
 * ---------------------------------------------------------------------- */
size_t ca_tables_workspace_bytes(const ca_problem* p, int32_t group_size);

ca_status ca_build_block_tables(const ca_problem* p, const uint64_t* masks,
                                int32_t group_size, int32_t* kv_indptr,
                                int32_t* kv_indices, void* ws, size_t ws_bytes,
                                void* stream);

/* 2a. Allocation-free ca_build_block_tables, for callers that cannot allocate
 *    device memory (code under HIP graph capture, tight serving loops,
 *    harnesses that forbid hipMalloc): the same kernels and the same tables,
 *    bit for bit, with the union words and row counts in a scratch array of
 *    CA_NOALLOC_SCRATCH_BYTES that the library holds on every GPU it runs on
 *    until the process ends (looked up on the first call on each device, with
 *    that device current; the stream must belong to the current device).  The
 *    call allocates nothing.  It needs ca_tables_workspace_bytes(p, group_size)
 *    <= CA_NOALLOC_SCRATCH_BYTES (B * G rows of ceil(max_kv_blocks / 64) 8-byte
 *    words + one int32 count each: 511 rows at max_kv_blocks = 16384), else
 *    CA_ERR_WORKSPACE before any launch.  Every call on one GPU uses that GPU's
 *    one scratch array: calls that overlap on one GPU (different streams or
 *    host threads without ordering) race and must not be issued. */
#define CA_NOALLOC_SCRATCH_BYTES (1u << 20)

ca_status ca_build_block_tables_noalloc(const ca_problem* p, const uint64_t* masks,
                                        int32_t group_size, int32_t* kv_indptr,
                                        int32_t* kv_indices, void* stream);

/* 2b. Fused estimator-to-union (Sec. 3.2: the selected blocks of every head
 *    and Q-block of a group only matter through their union): the four
 *    estimator stages of ca_estimate_masks, except that each selection row
 *    is ORed straight into the words of its (b, group) table row instead of
 *    being stored as a mask, then the words are compacted into the CSR pair.
 *    The tables are bit-identical to ca_build_block_tables(group_size) of
 *    the masks ca_estimate_masks produces from the same inputs; no per-row
 *    mask is written.  q_mean, k_mean and scores are written as by
 *    ca_estimate_masks (k_mean_first_block likewise).
 *    Workspace: at least B * (Hq / group_size) * W * 8 bytes of device memory,
 *    8-byte aligned (ca_tables_workspace_bytes(p, group_size) is enough);
 *    its contents on entry are irrelevant (it is cleared by the first
 *    stage).  Errors: CA_ERR_GROUP, CA_ERR_NULL, CA_ERR_SHAPE (top_frac,
 *    sink/local, first_block), CA_ERR_WORKSPACE, all before any launch. */
ca_status ca_estimate_tables(const ca_problem* p, const uint16_t* q, const uint16_t* k_pool,
                             const int32_t* page_table, float top_frac, int32_t sink_blocks,
                             int32_t local_blocks, int32_t k_mean_first_block,
                             int32_t group_size, float* q_mean, float* k_mean, float* scores,
                             int32_t* kv_indptr, int32_t* kv_indices, void* ws,
                             size_t ws_bytes, void* stream);

/* ------------------------------------------------------------------------
 * 3. Chunk attention over the tables (Sec. 3.3, App. B.2).
 *    q bf16 [B, C, Hq, D]; out bf16 [B, C, Hq, D]; lse fp32 [B, Hq, C]
 *    (natural-log log-sum-exp of the scaled scores, may be NULL).
 *    For query (b, h, t) and every key of every block j in T[b, h/group_size]
 *    with key position <= cached_len[b] + t:
 *        out = softmax(sm_scale * q.k) . v      (bf16 MFMA, fp32 softmax)
 *    Table entries must be ascending and < nKB_b; blocks are read in place
 *    through page_table (no gather).  A query that sees no key gets out = 0,
 *    lse = -inf.
 *    num_splits: 1 = one pass per query tile; > 1 = the table of each row is
 *    cut into that many consecutive pieces whose partial results are merged
 *    by log-sum-exp (needs workspace); 0 = let the library choose:
 *      - when the query tiles fill the GPU, B * G is a multiple of 8 and the
 *        workspace holds ca_attention_workspace_bytes(p, group_size, 0):
 *        every table row is cut in two at a point computed on the GPU from
 *        the table lengths, so that the 8 XCDs of the MI355X carry equal
 *        loads (rows r with r % 8 = x run on XCD x, which also runs the
 *        second pieces of XCD x-1's rows); the dense baseline does this only
 *        when the sequences differ in length;
 *      - otherwise splits only when the query tiles alone cannot fill the
 *        GPU and the workspace is large enough.
 *    The result does not depend on the choice beyond floating-point rounding.
 *    The XCD-balanced split merges its two pieces inside the same launch:
 *    the second piece of each query tile to finish reads the other's fp32
 *    partial result from the workspace and writes the tile's output rows.
 *    It learns that it is second from one counter per tile in the
 *    workspace, which each launch tags with its own 56-bit value.  Uniform
 *    splits (num_splits > 1) are merged by a second launch on the stream.
 *    Either way the workspace needs no clearing and may hold anything on
 *    entry (a launch leaves its counters at zero), and two launches that run
 *    at the same time must not share a workspace.
 *    Workspace: ca_attention_workspace_bytes(p, group_size, num_splits)
 *    bytes (0 when no split is needed; for num_splits = 0 it returns the
 *    size that lets the library pick freely).
 * ---------------------------------------------------------------------- */
size_t ca_attention_workspace_bytes(const ca_problem* p, int32_t group_size,
                                    int32_t num_splits);

ca_status ca_chunk_attention(const ca_problem* p, const uint16_t* q,
                             const uint16_t* k_pool, const uint16_t* v_pool,
                             const int32_t* page_table, const int32_t* kv_indptr,
                             const int32_t* kv_indices, int32_t group_size,
                             float sm_scale, int32_t num_splits, uint16_t* out,
                             float* lse, void* ws, size_t ws_bytes, void* stream);

/* Dense paged baseline: the same kernel with T[b,g] = every block 0..nKB_b-1
 * (the table an all-ones mask gives), without reading any table. */
ca_status ca_dense_paged_chunk_attention(const ca_problem* p, const uint16_t* q,
                                         const uint16_t* k_pool, const uint16_t* v_pool,
                                         const int32_t* page_table, float sm_scale,
                                         int32_t num_splits, uint16_t* out, float* lse,
                                         void* ws, size_t ws_bytes, void* stream);

/* ------------------------------------------------------------------------
 * 4. Execution-strategy arms at matched masks (Sec. 4.4, Fig. 7c; App. C
 *    Table 9).  They compute what the paper compares the zero-copy path
 *    against, with the same attention kernel, so that only the strategy
 *    differs.
 *
 * 4a. Block-sparse: every (sequence b, query head h, Q-block i) is its own
 *    tile with its own block list (no packing of the heads of a group; each
 *    tile reads its pages separately).
 *    ca_build_block_sparse_tables: CSR over rows (b*Hq + h)*nQB + i,
 *    kv_indptr int32 [B*Hq*nQB + 1], kv_indices capacity
 *    B*Hq*nQB*max_kv_blocks, entries ascending.  group_size = 0: row
 *    (b,h,i) = the set bits j < nKB_b of its own mask row M[b,h,i,:]
 *    (the raw mask executed directly); group_size > 0: row (b,h,i) = the
 *    union table T[b, h/group_size] of section 2, limited to the blocks
 *    Q-block i can see (j < e_i of section 1), which is the
 *    same unioned mask the zero-copy path executes (the matched-table
 *    ablation of Sec. 4.4).
 *    Workspace: ca_block_sparse_tables_workspace_bytes(p, group_size).
 *    ca_block_sparse_chunk_attention: for query t of Q-block i of head h,
 *    out = softmax over the keys of the blocks of row (b,h,i) with position
 *    <= cached_len[b] + t (as in section 3).  A query tile is one head x 128
 *    queries, so q_block must be 128 (else CA_ERR_UNSUPPORTED).  num_splits
 *    and workspace as in section 3 with group_size = 1
 *    (ca_attention_workspace_bytes(p, 1, num_splits)).
 * ---------------------------------------------------------------------- */
size_t ca_block_sparse_tables_workspace_bytes(const ca_problem* p, int32_t group_size);

ca_status ca_build_block_sparse_tables(const ca_problem* p, const uint64_t* masks,
                                       int32_t group_size, int32_t* kv_indptr,
                                       int32_t* kv_indices, void* ws, size_t ws_bytes,
                                       void* stream);

ca_status ca_block_sparse_chunk_attention(const ca_problem* p, const uint16_t* q,
                                          const uint16_t* k_pool, const uint16_t* v_pool,
                                          const int32_t* page_table,
                                          const int32_t* kv_indptr,
                                          const int32_t* kv_indices, float sm_scale,
                                          int32_t num_splits, uint16_t* out, float* lse,
                                          void* ws, size_t ws_bytes, void* stream);

/* 4b. Copy: the selected pages of every group table are first gathered into
 *    contiguous pools, then attention runs on them.
 *    ca_gather_selected_pages: packed page p (0 <= p < kv_indptr[B*G]) gets
 *    K_pool / V_pool page page_table[b, kvh, kv_indices[p]] of the row that
 *    owns entry p; k_packed is bf16 [capacity_pages, page, D] and v_packed
 *    has capacity_pages pages in the layout of v_pool (ca_problem.v_layout;
 *    pages are copied whole); capacity_pages must be >= kv_indptr[B*G]
 *    (B*G*max_kv_blocks always is; entries beyond the capacity are not
 *    copied).  Invalid entries (kv_indices outside [0, max_kv_blocks)) are
 *    skipped.
 *    ca_packed_chunk_attention: the section 3 result for the same tables,
 *    reading table entry p from packed page p (no page_table); the same
 *    kernel, so the output is bit-identical to ca_chunk_attention.
 * ---------------------------------------------------------------------- */
ca_status ca_gather_selected_pages(const ca_problem* p, const uint16_t* k_pool,
                                   const uint16_t* v_pool, const int32_t* page_table,
                                   const int32_t* kv_indptr, const int32_t* kv_indices,
                                   int32_t group_size, uint16_t* k_packed,
                                   uint16_t* v_packed, int64_t capacity_pages,
                                   void* stream);

ca_status ca_packed_chunk_attention(const ca_problem* p, const uint16_t* q,
                                    const uint16_t* k_packed, const uint16_t* v_packed,
                                    const int32_t* kv_indptr, const int32_t* kv_indices,
                                    int32_t group_size, float sm_scale, int32_t num_splits,
                                    int64_t capacity_pages, uint16_t* out, float* lse,
                                    void* ws, size_t ws_bytes, void* stream);

/* ------------------------------------------------------------------------
 * Debug helper: synchronises `stream`, copies the tables to the host and
 * checks kv_indptr[0] == 0, non-decreasing row bounds within capacity,
 * entries strictly ascending and < nKB_b, and (if require_chunk_open) that
 * every chunk block nC_b..nKB_b-1 is present (nC_b = floor(cached_len /
 * page_size), nKB_b = ceil((cached_len + chunk_len) / page_size)).  Returns CA_ERR_INVALID_TABLE
 * with a description in ca_last_error_detail() on the first violation.
 * ---------------------------------------------------------------------- */
ca_status ca_validate_tables(const ca_problem* p, int32_t group_size,
                             const int32_t* kv_indptr, const int32_t* kv_indices,
                             int32_t require_chunk_open, void* stream);

/* ------------------------------------------------------------------------
 * Host-only table check (no GPU, nothing enqueued): the checks of
 * ca_validate_tables on HOST copies of the tables and, when page_table is not
 * NULL (a HOST copy of the page table [B, Hkv, max_kv_blocks]), that the page
 * of every listed block is in [0, pool_pages).  group_size >= 1: one row per
 * (b, group), as ca_build_block_tables writes them; group_size == 0: one row
 * per (b, h, Q-block), the block-sparse layout of ca_build_block_sparse_tables.
 * Returns CA_ERR_INVALID_TABLE with a description in ca_last_error_detail()
 * on the first violation; the arrays are only read.
 *
 * Debug build.  libcompactattn_debug.so (the same sources compiled with
 * CA_DEBUG_CHECKS) runs this check before every attention launch
 * (ca_chunk_attention, ca_dense_paged_chunk_attention,
 * ca_block_sparse_chunk_attention, ca_packed_chunk_attention): it
 * synchronises the stream, copies the tables and the page table to the host,
 * takes pool_pages from the device allocations that hold k_pool and v_pool,
 * and returns CA_ERR_INVALID_TABLE instead of launching when a table entry or
 * a page id is out of range (for the packed pools: when the tables list more
 * pages than the pools hold).  Results are otherwise identical to the
 * release library's; every attention call then synchronises.
 * ---------------------------------------------------------------------- */
ca_status ca_check_tables_host(const ca_problem* p, int32_t group_size,
                               const int32_t* kv_indptr, const int32_t* kv_indices,
                               const int32_t* page_table, int64_t pool_pages,
                               int32_t require_chunk_open);

#ifdef __cplusplus
}
#endif
#endif /* COMPACTATTN_H */
