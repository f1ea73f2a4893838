// Internal launcher interface between the C ABI (api.hip) and the kernels.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ca {

// Validated problem sizes, derived once on the host.
struct Dims {
  int B, Hq, Hkv, D, page, q_block, C, max_kv_blocks;
  int nqb;           // ceil(C / q_block)
  int W;             // mask words per row
  int max_nc;        // max_b full cached blocks, floor(cached_len_b / page)
  int max_nkb;       // max_b blocks of the sequence, ceil((cached_len_b + C) / page)
};

// Q-block and K-block pooling in one launch (q or k_pool may be nullptr to
// skip that part); clear_words[0, n_clear) are zeroed by the same launch.
hipError_t launch_pool(const Dims& d, const uint16_t* q, float* q_mean, const uint16_t* k_pool,
                       const int32_t* page_table, const int32_t* cached_len, int first_block,
                       float* k_mean, hipStream_t st, uint64_t* clear_words = nullptr,
                       int n_clear = 0);
hipError_t launch_pool_q(const Dims& d, const uint16_t* q, float* q_mean, hipStream_t st,
                         uint64_t* clear_words = nullptr, int n_clear = 0);
hipError_t launch_pool_k(const Dims& d, const uint16_t* k_pool, const int32_t* page_table,
                         const int32_t* cached_len, int first_block, float* k_mean,
                         hipStream_t st);
hipError_t launch_scores(const Dims& d, const float* q_mean, const float* k_mean,
                         const int32_t* cached_len, float* scores, hipStream_t st);
// With group_words set, the selected rows are ORed into the (b, group) union
// words (cleared beforehand) instead of being stored as masks.
hipError_t launch_select(const Dims& d, const float* scores, const int32_t* cached_len,
                         float top_frac, int sink_blocks, int local_blocks, uint64_t* masks,
                         hipStream_t st, uint64_t* group_words = nullptr, int group_size = 1);
hipError_t raise_select_lds(int bytes);
hipError_t launch_threshold_select(const Dims& d, const float* scores, const int32_t* cached_len,
                                   float margin, int sink_blocks, int local_blocks,
                                   uint64_t* masks, hipStream_t st);

size_t tables_ws_bytes(const Dims& d, int group_size);
hipError_t launch_tables(const Dims& d, const uint64_t* masks, const int32_t* cached_len,
                         int group_size, int32_t* kv_indptr, int32_t* kv_indices, void* ws,
                         hipStream_t st);
// CSR from per-row union words (each row's count is its words' popcount).
hipError_t launch_compact_words(const Dims& d, int rows, const uint64_t* words,
                                int32_t* kv_indptr, int32_t* kv_indices, hipStream_t st);
// Block-sparse rows (b, h, Q-block i) holding the union of the group of h,
// causally limited to Q-block i (the block-sparse arm at matched tables).
size_t union_rows_ws_bytes(const Dims& d, int group_size);
hipError_t launch_union_rows(const Dims& d, const uint64_t* masks, const int32_t* cached_len,
                             int group_size, int32_t* kv_indptr, int32_t* kv_indices, void* ws,
                             hipStream_t st);

// Table layouts the attention kernel understands.
constexpr int kTablesPerGroup = 0;   // row b*G + g, entries translated by page_table
constexpr int kTablesPerQTile = 1;   // row (b*Hq + h)*n_qtiles + tile (block-sparse arm)
constexpr int kTablesPacked = 2;     // per-group rows; page of entry p is p (copy arm)

// V page layouts of the pool (ca_problem.v_layout).
constexpr int kVTokenMajor = 0;   // [P, page, D], like the K pages
constexpr int kVTransposed = 1;   // [P, D, page]

// Attention over per-group tables (dense = identity tables, no table read).
struct AttnLaunch {
  const uint16_t* q;
  const uint16_t* k_pool;
  const uint16_t* v_pool;
  const int32_t* page_table;
  const int32_t* kv_indptr;
  const int32_t* kv_indices;
  const int32_t* cached_len;
  uint16_t* out;
  float* lse;
  int group_size;
  float sm_scale;
  int splits;        // >= 1
  void* ws;          // partials when splits > 1 (+ cuts and counters: XCD split)
  bool dense;
  int table_mode = kTablesPerGroup;
  long long packed_pages = 0;
  // splits == 2 with the cut of every table row chosen so that the 8 XCDs
  // carry equal loads (needs B * G % 8 == 0 and attn_xcd_ws_bytes of ws)
  bool xcd_balanced = false;
  int v_layout = kVTokenMajor;
};
int attn_rows_per_workgroup(int table_mode);             // (head, query) rows per workgroup
int attn_query_tile(int group_size, int table_mode);     // chunk queries per workgroup
int attn_base_workgroups(const Dims& d, int group_size, int table_mode);
int attn_resident_workgroups(int table_mode);            // workgroups the GPU holds at once
size_t attn_ws_bytes(const Dims& d, int splits);
size_t attn_xcd_ws_bytes(const Dims& d, int group_size);
hipError_t launch_attention(const Dims& d, const AttnLaunch& a, hipStream_t st);
hipError_t launch_gather(const Dims& d, const uint16_t* k_pool, const uint16_t* v_pool,
                         const int32_t* page_table, const int32_t* kv_indptr,
                         const int32_t* kv_indices, int group_size, long long capacity_pages,
                         uint16_t* k_packed, uint16_t* v_packed, hipStream_t st);

}  // namespace ca
