// C ABI of libcompactattn: host-side validation and launch glue.
// The meaning of every entry point is documented in include/compactattn.h.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <mutex>
#include <string>
#include <vector>

#include "compactattn.h"
#include "common.hpp"
#include "kernels.hpp"

namespace {

thread_local std::string g_detail;

ca_status fail(ca_status s, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
ca_status fail(ca_status s, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_detail = buf;
  return s;
}

ca_status ok() {
  g_detail.clear();
  return CA_OK;
}

ca_status hip_status(hipError_t e, const char* what) {
  if (e == hipSuccess) return ok();
  return fail(CA_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

// Validates p (and group_size when > 0) and fills d.
ca_status check(const ca_problem* p, int32_t group_size, ca::Dims* d) {
  if (p == nullptr) return fail(CA_ERR_NULL, "problem is NULL");
  if (p->cached_len_host == nullptr) return fail(CA_ERR_NULL, "cached_len_host is NULL");
  if (p->batch < 1 || p->num_q_heads < 1 || p->num_kv_heads < 1)
    return fail(CA_ERR_SHAPE, "batch, num_q_heads and num_kv_heads must be >= 1");
  if (p->num_q_heads % p->num_kv_heads != 0)
    return fail(CA_ERR_SHAPE, "num_kv_heads (%d) must divide num_q_heads (%d)",
                p->num_kv_heads, p->num_q_heads);
  if (p->head_dim != 64 && p->head_dim != 128)
    return fail(CA_ERR_UNSUPPORTED, "head_dim %d not supported (64, 128)", p->head_dim);
  if (p->page_size != ca::kPage)
    return fail(CA_ERR_UNSUPPORTED, "page_size %d not supported (64)", p->page_size);
  if (p->q_block != 64 && p->q_block != 128)
    return fail(CA_ERR_UNSUPPORTED, "q_block %d not supported (64, 128)", p->q_block);
  if (p->chunk_len < 1) return fail(CA_ERR_SHAPE, "chunk_len must be >= 1");
  if (p->v_layout != CA_V_TOKEN_MAJOR && p->v_layout != CA_V_TRANSPOSED)
    return fail(CA_ERR_SHAPE, "v_layout %d is not CA_V_TOKEN_MAJOR (0) or CA_V_TRANSPOSED (1)",
                p->v_layout);
  if (p->max_kv_blocks < 1 || p->max_kv_blocks > ca::kMaxKvBlocks)
    return fail(CA_ERR_SHAPE, "max_kv_blocks %d out of range [1, %d]", p->max_kv_blocks,
                ca::kMaxKvBlocks);
  int max_nc = 0, max_nkb = 0;
  for (int b = 0; b < p->batch; ++b) {
    const int c = p->cached_len_host[b];
    if (c < 0) return fail(CA_ERR_SHAPE, "cached_len[%d] = %d is negative", b, c);
    // any lengths: the last block of a sequence may be partial
    const long long nkb = ((long long)c + p->chunk_len + p->page_size - 1) / p->page_size;
    if (nkb > p->max_kv_blocks)
      return fail(CA_ERR_SHAPE, "sequence %d needs %lld blocks > max_kv_blocks %d", b, nkb,
                  p->max_kv_blocks);
    if (c / p->page_size > max_nc) max_nc = c / p->page_size;
    if (nkb > max_nkb) max_nkb = (int)nkb;
  }
  if (group_size > 0) {
    const int ratio = p->num_q_heads / p->num_kv_heads;
    if (ratio % group_size != 0)
      return fail(CA_ERR_GROUP, "group_size %d must divide Hq/Hkv = %d", group_size, ratio);
  }
  if (d != nullptr) {
    d->B = p->batch;
    d->Hq = p->num_q_heads;
    d->Hkv = p->num_kv_heads;
    d->D = p->head_dim;
    d->page = p->page_size;
    d->q_block = p->q_block;
    d->C = p->chunk_len;
    d->max_kv_blocks = p->max_kv_blocks;
    d->nqb = (p->chunk_len + p->q_block - 1) / p->q_block;
    d->W = (p->max_kv_blocks + 63) / 64;
    d->max_nc = max_nc;
    d->max_nkb = max_nkb;
  }
  return ok();
}

ca_status need_device(const ca_problem* p) {
  if (p->cached_len == nullptr) return fail(CA_ERR_NULL, "cached_len (device) is NULL");
  return CA_OK;
}

ca_status attention_tile_ok(int group_size, int table_mode) {
  const int rows = ca::attn_rows_per_workgroup(table_mode);
  if (rows % group_size != 0)
    return fail(CA_ERR_UNSUPPORTED, "group_size %d must divide %d", group_size, rows);
  return CA_OK;
}

// Splits chosen when the caller passes num_splits = 0.
int auto_splits(const ca::Dims& d, int group_size, size_t ws_bytes, bool have_ws,
                int table_mode = ca::kTablesPerGroup) {
  const int base = ca::attn_base_workgroups(d, group_size, table_mode);
  const int target = ca::attn_resident_workgroups(table_mode);
  if (base >= target || !have_ws) return 1;
  int s = (target + base - 1) / base;
  const int max_by_len = d.max_nkb / 4 > 1 ? d.max_nkb / 4 : 1;
  if (s > max_by_len) s = max_by_len;
  if (s > 16) s = 16;
  while (s > 1 && ca::attn_ws_bytes(d, s) > ws_bytes) --s;
  return s < 1 ? 1 : s;
}

// num_splits = 0 on per-group tables whose query tiles already fill the GPU:
// two pieces per table row, cut so that the 8 XCDs carry equal loads (the
// execution groups of one XCD otherwise differ in table length).  Needs the
// rows to spread evenly over the XCDs.  Dense rows of equal length (every
// sequence the same length) are balanced already.
bool xcd_balance_ok(const ca::Dims& d, const ca_problem* p, int group_size, int table_mode,
                    bool dense) {
  if (table_mode == ca::kTablesPerQTile) return false;
  const int R = d.B * (d.Hq / group_size);
  if (R % 8 != 0) return false;
  if (ca::attn_base_workgroups(d, group_size, table_mode) <
      ca::attn_resident_workgroups(table_mode))
    return false;
  if (dense) {
    for (int b = 1; b < d.B; ++b)
      if (p->cached_len_host[b] != p->cached_len_host[0]) return true;
    return false;
  }
  return true;
}

// The kernels read and write the bf16 and fp32 tensors with 16-byte vector
// accesses, so each must start on a 16-byte boundary (every hipMalloc or torch
// allocation does; a view that starts mid-row may not).  NULL passes here: the
// NULL checks report it.
template <typename... T>
ca_status need_aligned16(const char* names, const T*... ptrs) {
  const bool ok = ((reinterpret_cast<uintptr_t>(ptrs) % 16 == 0) && ...);
  return ok ? CA_OK : fail(CA_ERR_UNALIGNED, "%s must be 16-byte aligned", names);
}

// Rows of a table layout: group_size >= 1, one row per (b, group) (the group
// union tables); group_size == 0, one row per (b, h, Q-block) (block-sparse).
int table_rows(const ca::Dims& d, int group_size) {
  return group_size > 0 ? d.B * (d.Hq / group_size) : d.B * d.Hq * d.nqb;
}
void row_owner(const ca::Dims& d, int group_size, int r, int* b, int* kvh) {
  const int ratio = d.Hq / d.Hkv;
  if (group_size > 0) {
    const int G = d.Hq / group_size;
    *b = r / G;
    *kvh = ((r % G) * group_size) / ratio;
  } else {
    *b = r / (d.Hq * d.nqb);
    *kvh = ((r / d.nqb) % d.Hq) / ratio;
  }
}

// The table checks on host arrays: kv_indptr[0] == 0, non-decreasing row
// bounds within the capacity, entries strictly ascending in [0, nKB_b), the
// chunk blocks all present (require_chunk_open), and with a page table, the
// page of every listed block in [0, pool_pages).
ca_status check_tables(const ca_problem* p, const ca::Dims& d, int group_size,
                       const int32_t* ip, const int32_t* ix, const int32_t* page_table,
                       long long pool_pages, bool require_chunk_open) {
  const int R = table_rows(d, group_size);
  const size_t cap = (size_t)R * d.max_kv_blocks;
  if (ip[0] != 0) return fail(CA_ERR_INVALID_TABLE, "kv_indptr[0] = %d, expected 0", ip[0]);
  for (int r = 0; r < R; ++r)
    if (ip[r + 1] < ip[r] || (size_t)ip[r + 1] > cap)
      return fail(CA_ERR_INVALID_TABLE, "kv_indptr[%d..%d] = %d..%d is not a valid range", r,
                  r + 1, ip[r], ip[r + 1]);
  for (int r = 0; r < R; ++r) {
    int b, kvh;
    row_owner(d, group_size, r, &b, &kvh);
    const int nc = p->cached_len_host[b] / d.page;
    const int nkb = ca::blocks_for(p->cached_len_host[b] + d.C);
    int prev = -1, chunk_seen = 0;
    for (int x = ip[r]; x < ip[r + 1]; ++x) {
      const int j = ix[x];
      if (j <= prev || j < 0 || j >= nkb)
        return fail(CA_ERR_INVALID_TABLE, "row %d entry %d = %d (previous %d, nKB %d)", r,
                    x - ip[r], j, prev, nkb);
      if (page_table) {
        const int32_t pg = page_table[((size_t)b * d.Hkv + kvh) * d.max_kv_blocks + j];
        if (pg < 0 || pg >= pool_pages)
          return fail(CA_ERR_INVALID_TABLE,
                      "row %d block %d: page %d outside the pool's %lld pages", r, j, pg,
                      pool_pages);
      }
      if (j >= nc) ++chunk_seen;
      prev = j;
    }
    if (require_chunk_open && chunk_seen != nkb - nc)
      return fail(CA_ERR_INVALID_TABLE, "row %d holds %d of the %d chunk blocks", r, chunk_seen,
                  nkb - nc);
  }
  return ok();
}

// Synchronises the stream and copies the tables (and the page table when
// given) to the host.
ca_status copy_tables(const ca::Dims& d, int group_size, const int32_t* kv_indptr,
                      const int32_t* kv_indices, const int32_t* page_table, hipStream_t st,
                      std::vector<int32_t>& ip, std::vector<int32_t>& ix,
                      std::vector<int32_t>& pt) {
  hipError_t e = hipStreamSynchronize(st);
  if (e != hipSuccess) return hip_status(e, "stream synchronize");
  const int R = table_rows(d, group_size);
  ip.assign(R + 1, 0);
  if ((e = hipMemcpy(ip.data(), kv_indptr, (R + 1) * sizeof(int32_t), hipMemcpyDeviceToHost)) !=
      hipSuccess)
    return hip_status(e, "copy kv_indptr");
  const size_t cap = (size_t)R * d.max_kv_blocks;
  const size_t n = ip[R] > 0 && (size_t)ip[R] <= cap ? (size_t)ip[R] : 0;
  ix.assign(n > 0 ? n : 1, 0);
  if (n > 0 &&
      (e = hipMemcpy(ix.data(), kv_indices, n * sizeof(int32_t), hipMemcpyDeviceToHost)) !=
          hipSuccess)
    return hip_status(e, "copy kv_indices");
  if (page_table) {
    pt.assign((size_t)d.B * d.Hkv * d.max_kv_blocks, 0);
    if ((e = hipMemcpy(pt.data(), page_table, pt.size() * sizeof(int32_t),
                       hipMemcpyDeviceToHost)) != hipSuccess)
      return hip_status(e, "copy page_table");
  }
  return ok();
}

#ifdef CA_DEBUG_CHECKS
// Pages of `page_elems` elements from `pool` to the end of the allocation that
// holds it.
ca_status pool_pages_of(const uint16_t* pool, size_t page_elems, long long* pages) {
  void* base = nullptr;
  size_t size = 0;
  hipError_t e = hipMemGetAddressRange(&base, &size, const_cast<uint16_t*>(pool));
  if (e != hipSuccess) return hip_status(e, "pool address range");
  const size_t avail = static_cast<const char*>(base) + size - reinterpret_cast<const char*>(pool);
  *pages = (long long)(avail / (page_elems * sizeof(uint16_t)));
  return ok();
}

// The debug build's check before every attention launch: the tables and
// every page the launch will read, against the allocations of the pools.
ca_status debug_check_launch(const ca_problem* p, const ca::Dims& d, int group_size,
                             int table_mode, bool dense, const uint16_t* k_pool,
                             const uint16_t* v_pool, const int32_t* page_table,
                             const int32_t* kv_indptr, const int32_t* kv_indices,
                             long long packed_pages, hipStream_t st) {
  const size_t page_elems = (size_t)d.page * d.D;
  long long pk = 0, pv = 0;
  ca_status s;
  if ((s = pool_pages_of(k_pool, page_elems, &pk)) != CA_OK) return s;
  if ((s = pool_pages_of(v_pool, page_elems, &pv)) != CA_OK) return s;
  const long long pages = pk < pv ? pk : pv;
  const int gs = table_mode == ca::kTablesPerQTile ? 0 : group_size;
  std::vector<int32_t> ip, ix, pt;
  if (dense) {
    // identity tables: every block of every sequence
    const int R = d.B * d.Hkv;
    ip.assign(R + 1, 0);
    for (int r = 0; r < R; ++r) {
      const int b = r / d.Hkv;
      const int nkb = ca::blocks_for(p->cached_len_host[b] + d.C);
      ip[r + 1] = ip[r] + nkb;
      for (int j = 0; j < nkb; ++j) ix.push_back(j);
    }
    hipError_t e = hipStreamSynchronize(st);
    if (e != hipSuccess) return hip_status(e, "stream synchronize");
    pt.assign((size_t)d.B * d.Hkv * d.max_kv_blocks, 0);
    if ((e = hipMemcpy(pt.data(), page_table, pt.size() * sizeof(int32_t),
                       hipMemcpyDeviceToHost)) != hipSuccess)
      return hip_status(e, "copy page_table");
    return check_tables(p, d, d.Hq / d.Hkv, ip.data(), ix.data(), pt.data(), pages, false);
  }
  const bool packed = table_mode == ca::kTablesPacked;
  if ((s = copy_tables(d, gs, kv_indptr, kv_indices, packed ? nullptr : page_table, st, ip, ix,
                       pt)) != CA_OK)
    return s;
  if ((s = check_tables(p, d, gs, ip.data(), ix.data(), packed ? nullptr : pt.data(), pages,
                        false)) != CA_OK)
    return s;
  if (packed) {
    // the packed pools hold the listed pages in table order
    const long long listed = ip[table_rows(d, gs)];
    const long long cap = packed_pages < pages ? packed_pages : pages;
    if (listed > cap)
      return fail(CA_ERR_INVALID_TABLE, "the tables list %lld pages, the packed pools hold %lld",
                  listed, cap);
  }
  return ok();
}
#endif

ca_status run_attention(const ca_problem* p, const uint16_t* q, const uint16_t* k_pool,
                        const uint16_t* v_pool, const int32_t* page_table,
                        const int32_t* kv_indptr, const int32_t* kv_indices, int32_t group_size,
                        float sm_scale, int32_t num_splits, uint16_t* out, float* lse, void* ws,
                        size_t ws_bytes, void* stream, bool dense,
                        int table_mode = ca::kTablesPerGroup, long long packed_pages = 0) {
  ca::Dims d;
  ca_status s = check(p, group_size, &d);
  if (s != CA_OK) return s;
  if ((s = need_device(p)) != CA_OK) return s;
  if (!q || !k_pool || !v_pool || !out || (!page_table && table_mode != ca::kTablesPacked))
    return fail(CA_ERR_NULL, "q, k_pool, v_pool, page_table and out are required");
  if ((s = need_aligned16("q, k_pool, v_pool and out", q, k_pool, v_pool, out)) != CA_OK) return s;
  if (table_mode == ca::kTablesPerQTile &&
      ca::attn_query_tile(group_size, table_mode) != d.q_block)
    return fail(CA_ERR_UNSUPPORTED,
                "block-sparse attention runs one head x one Q-block per tile: q_block must be "
                "%d, got %d", ca::attn_query_tile(group_size, table_mode), d.q_block);
  if (table_mode == ca::kTablesPacked && packed_pages < 1)
    return fail(CA_ERR_SHAPE, "capacity_pages must be >= 1");
  if (!dense && (!kv_indptr || !kv_indices))
    return fail(CA_ERR_NULL, "kv_indptr and kv_indices are required");
  // softmax(sm_scale * q.k): a zero, negative or non-finite scale would turn the
  // masked (-inf) scores into NaN or +inf weights
  if (!(sm_scale > 0.f) || !std::isfinite(sm_scale))
    return fail(CA_ERR_SHAPE, "sm_scale must be finite and > 0, got %g", (double)sm_scale);
  if ((s = attention_tile_ok(group_size, table_mode)) != CA_OK) return s;
  if (num_splits < 0 || num_splits > 64)
    return fail(CA_ERR_SHAPE, "num_splits %d out of range [0, 64]", num_splits);
  int splits = num_splits;
  bool xcd = false;
  if (splits == 0) {
    xcd = xcd_balance_ok(d, p, group_size, table_mode, dense) && ws != nullptr &&
          ws_bytes >= ca::attn_xcd_ws_bytes(d, group_size);
    splits = xcd ? 2 : auto_splits(d, group_size, ws_bytes, ws != nullptr, table_mode);
  }
  if (splits > 1) {
    const size_t need = ca::attn_ws_bytes(d, splits);
    if (ws == nullptr || ws_bytes < need)
      return fail(CA_ERR_WORKSPACE, "attention with %d splits needs %zu workspace bytes, got %zu",
                  splits, need, ws == nullptr ? (size_t)0 : ws_bytes);
    if (reinterpret_cast<uintptr_t>(ws) % 16 != 0)
      return fail(CA_ERR_WORKSPACE, "workspace must be 16-byte aligned");
  }
  ca::AttnLaunch L;
  L.q = q;
  L.k_pool = k_pool;
  L.v_pool = v_pool;
  L.page_table = page_table;
  L.kv_indptr = kv_indptr;
  L.kv_indices = kv_indices;
  L.cached_len = p->cached_len;
  L.out = out;
  L.lse = lse;
  L.group_size = group_size;
  L.sm_scale = sm_scale;
  L.splits = splits;
  L.xcd_balanced = xcd;
  L.ws = ws;
  L.dense = dense;
  L.table_mode = table_mode;
  L.packed_pages = packed_pages;
  L.v_layout = p->v_layout == CA_V_TRANSPOSED ? ca::kVTransposed : ca::kVTokenMajor;
#ifdef CA_DEBUG_CHECKS
  if ((s = debug_check_launch(p, d, group_size, table_mode, dense, k_pool, v_pool, page_table,
                              kv_indptr, kv_indices, packed_pages,
                              static_cast<hipStream_t>(stream))) != CA_OK)
    return s;
#endif
  return hip_status(ca::launch_attention(d, L, static_cast<hipStream_t>(stream)),
                    dense ? "dense paged attention launch" : "chunk attention launch");
}

}  // namespace

// Scratch of the allocation-free table builder: the union words and row counts
// that ca_build_block_tables keeps in the caller's workspace.  Every GPU the
// library runs on holds its own copy until the process ends; host code never
// uses this name as an address, only the pointer hipGetSymbolAddress returns
// for the current device.
static __device__ __align__(256) uint64_t scratch[CA_NOALLOC_SCRATCH_BYTES / sizeof(uint64_t)];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices];   // device address of `scratch`, per device

// Device address of the current device's scratch, looked up once per device
// (with that device current) on the first call.
ca_status scratch_ptr(void** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_status(e, "hipGetDevice");
  if (dev < 0 || dev >= kMaxDevices)
    return fail(CA_ERR_UNSUPPORTED, "device %d: the scratch table holds %d devices", dev,
                kMaxDevices);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch_ptr[dev] == nullptr) {
    void* ptr = nullptr;
    e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return hip_status(e, "hipGetSymbolAddress(scratch)");
    if (ptr == nullptr) return fail(CA_ERR_HIP, "hipGetSymbolAddress(scratch) returned NULL");
    g_scratch_ptr[dev] = ptr;
  }
  *out = g_scratch_ptr[dev];
  return CA_OK;
}

}  // namespace

extern "C" {

int ca_abi_version(void) { return CA_ABI_VERSION; }

const char* ca_status_string(ca_status s) {
  switch (s) {
    case CA_OK: return "CA_OK";
    case CA_ERR_NULL: return "CA_ERR_NULL";
    case CA_ERR_SHAPE: return "CA_ERR_SHAPE";
    case CA_ERR_UNALIGNED: return "CA_ERR_UNALIGNED";
    case CA_ERR_GROUP: return "CA_ERR_GROUP";
    case CA_ERR_WORKSPACE: return "CA_ERR_WORKSPACE";
    case CA_ERR_UNSUPPORTED: return "CA_ERR_UNSUPPORTED";
    case CA_ERR_INVALID_TABLE: return "CA_ERR_INVALID_TABLE";
    case CA_ERR_HIP: return "CA_ERR_HIP";
  }
  return "CA_ERR_UNKNOWN";
}

const char* ca_last_error_detail(void) { return g_detail.c_str(); }

ca_status ca_check_problem(const ca_problem* p, int32_t group_size) {
  return check(p, group_size, nullptr);
}

ca_status ca_pool_q_blocks(const ca_problem* p, const uint16_t* q, float* q_mean, void* stream) {
  ca::Dims d;
  ca_status s = check(p, 0, &d);
  if (s != CA_OK) return s;
  if (!q || !q_mean) return fail(CA_ERR_NULL, "q and q_mean are required");
  if ((s = need_aligned16("q and q_mean", q, q_mean)) != CA_OK) return s;
  return hip_status(ca::launch_pool_q(d, q, q_mean, static_cast<hipStream_t>(stream)),
                    "pool_q launch");
}

ca_status ca_pool_k_blocks(const ca_problem* p, const uint16_t* k_pool,
                           const int32_t* page_table, int32_t first_block, float* k_mean,
                           void* stream) {
  ca::Dims d;
  ca_status s = check(p, 0, &d);
  if (s != CA_OK) return s;
  if ((s = need_device(p)) != CA_OK) return s;
  if (!k_pool || !page_table || !k_mean)
    return fail(CA_ERR_NULL, "k_pool, page_table and k_mean are required");
  if ((s = need_aligned16("k_pool and k_mean", k_pool, k_mean)) != CA_OK) return s;
  if (first_block < 0) return fail(CA_ERR_SHAPE, "first_block must be >= 0");
  return hip_status(ca::launch_pool_k(d, k_pool, page_table, p->cached_len, first_block,
                                      k_mean, static_cast<hipStream_t>(stream)),
                    "pool_k launch");
}

// Both pooling stages in one launch, with the checks of ca_pool_q_blocks and
// ca_pool_k_blocks.
static ca_status pool_both(const ca_problem* p, const uint16_t* q, const uint16_t* k_pool,
                           const int32_t* page_table, int32_t first_block, float* q_mean,
                           float* k_mean, void* stream) {
  ca::Dims d;
  ca_status s = check(p, 0, &d);
  if (s != CA_OK) return s;
  if ((s = need_device(p)) != CA_OK) return s;
  if (!q || !q_mean || !k_pool || !page_table || !k_mean)
    return fail(CA_ERR_NULL, "q, q_mean, k_pool, page_table and k_mean are required");
  if ((s = need_aligned16("q, q_mean, k_pool and k_mean", q, q_mean, k_pool, k_mean)) != CA_OK)
    return s;
  if (first_block < 0) return fail(CA_ERR_SHAPE, "first_block must be >= 0");
  return hip_status(ca::launch_pool(d, q, q_mean, k_pool, page_table, p->cached_len, first_block,
                                    k_mean, static_cast<hipStream_t>(stream)),
                    "pool launch");
}

ca_status ca_block_scores(const ca_problem* p, const float* q_mean, const float* k_mean,
                          float* scores, void* stream) {
  ca::Dims d;
  ca_status s = check(p, 0, &d);
  if (s != CA_OK) return s;
  if ((s = need_device(p)) != CA_OK) return s;
  if (!q_mean || !k_mean || !scores)
    return fail(CA_ERR_NULL, "q_mean, k_mean and scores are required");
  if ((s = need_aligned16("q_mean, k_mean and scores", q_mean, k_mean, scores)) != CA_OK) return s;
  return hip_status(ca::launch_scores(d, q_mean, k_mean, p->cached_len, scores,
                                      static_cast<hipStream_t>(stream)),
                    "scores launch");
}

// The keys of one selection row live in LDS: raise the dynamic LDS cap for
// long caches.
static ca_status select_lds_ready(const ca::Dims& d) {
  const size_t lds = (size_t)(d.max_nc > 0 ? d.max_nc : 1) * sizeof(uint32_t);
  if (lds > 48 * 1024) {
    hipError_t e = ca::raise_select_lds((int)lds);
    if (e != hipSuccess) return hip_status(e, "raise select LDS limit");
  }
  return CA_OK;
}

ca_status ca_select_blocks(const ca_problem* p, const float* scores, float top_frac,
                           int32_t sink_blocks, int32_t local_blocks, uint64_t* masks,
                           void* stream) {
  ca::Dims d;
  ca_status s = check(p, 0, &d);
  if (s != CA_OK) return s;
  if ((s = need_device(p)) != CA_OK) return s;
  if (!scores || !masks) return fail(CA_ERR_NULL, "scores and masks are required");
  if (!(top_frac >= 0.f && top_frac <= 1.f))
    return fail(CA_ERR_SHAPE, "top_frac must be in [0, 1]");
  if (sink_blocks < 0 || local_blocks < 0)
    return fail(CA_ERR_SHAPE, "sink_blocks and local_blocks must be >= 0");
  if ((s = select_lds_ready(d)) != CA_OK) return s;
  return hip_status(ca::launch_select(d, scores, p->cached_len, top_frac, sink_blocks,
                                      local_blocks, masks, static_cast<hipStream_t>(stream)),
                    "select launch");
}

ca_status ca_estimate_masks(const ca_problem* p, const uint16_t* q, const uint16_t* k_pool,
                            const int32_t* page_table, float top_frac, int32_t sink_blocks,
                            int32_t local_blocks, int32_t k_mean_first_block, float* q_mean,
                            float* k_mean, float* scores, uint64_t* masks, void* stream) {
  // the selection parameters are checked before the first stage is enqueued
  if (!(top_frac >= 0.f && top_frac <= 1.f))
    return fail(CA_ERR_SHAPE, "top_frac must be in [0, 1]");
  if (sink_blocks < 0 || local_blocks < 0)
    return fail(CA_ERR_SHAPE, "sink_blocks and local_blocks must be >= 0");
  if (!masks) return fail(CA_ERR_NULL, "masks is required");
  ca_status s = need_aligned16("q, k_pool, q_mean, k_mean and scores", q, k_pool, q_mean, k_mean,
                               scores);
  if (s != CA_OK) return s;
  if ((s = pool_both(p, q, k_pool, page_table, k_mean_first_block, q_mean, k_mean, stream)) !=
      CA_OK)
    return s;
  if ((s = ca_block_scores(p, q_mean, k_mean, scores, stream)) != CA_OK) return s;
  return ca_select_blocks(p, scores, top_frac, sink_blocks, local_blocks, masks, stream);
}

ca_status ca_estimate_tables(const ca_problem* p, const uint16_t* q, const uint16_t* k_pool,
                             const int32_t* page_table, float top_frac, int32_t sink_blocks,
                             int32_t local_blocks, int32_t k_mean_first_block,
                             int32_t group_size, float* q_mean, float* k_mean, float* scores,
                             int32_t* kv_indptr, int32_t* kv_indices, void* ws, size_t ws_bytes,
                             void* stream) {
  ca::Dims d;
  if (group_size < 1) return fail(CA_ERR_GROUP, "group_size must be >= 1");
  ca_status s = check(p, group_size, &d);
  if (s != CA_OK) return s;
  if ((s = need_device(p)) != CA_OK) return s;
  if (!q || !k_pool || !page_table || !q_mean || !k_mean || !scores || !kv_indptr || !kv_indices)
    return fail(CA_ERR_NULL,
                "q, k_pool, page_table, q_mean, k_mean, scores, kv_indptr and kv_indices are "
                "required");
  if ((s = need_aligned16("q, k_pool, q_mean, k_mean and scores", q, k_pool, q_mean, k_mean,
                          scores)) != CA_OK)
    return s;
  if (!(top_frac >= 0.f && top_frac <= 1.f))
    return fail(CA_ERR_SHAPE, "top_frac must be in [0, 1]");
  if (sink_blocks < 0 || local_blocks < 0)
    return fail(CA_ERR_SHAPE, "sink_blocks and local_blocks must be >= 0");
  if (k_mean_first_block < 0) return fail(CA_ERR_SHAPE, "first_block must be >= 0");
  const int rows = d.B * (d.Hq / group_size);
  const size_t need = (size_t)rows * d.W * sizeof(uint64_t);
  if (ws == nullptr || ws_bytes < need)
    return fail(CA_ERR_WORKSPACE, "fused tables need %zu workspace bytes, got %zu", need,
                ws == nullptr ? (size_t)0 : ws_bytes);
  if (reinterpret_cast<uintptr_t>(ws) % sizeof(uint64_t) != 0)
    return fail(CA_ERR_WORKSPACE, "workspace must be 8-byte aligned");
  if ((s = select_lds_ready(d)) != CA_OK) return s;
  const hipStream_t st = static_cast<hipStream_t>(stream);
  uint64_t* words = static_cast<uint64_t*>(ws);
  hipError_t e = ca::launch_pool(d, q, q_mean, k_pool, page_table, p->cached_len,
                                 k_mean_first_block, k_mean, st, words, (int)((size_t)rows * d.W));
  if (e == hipSuccess) e = ca::launch_scores(d, q_mean, k_mean, p->cached_len, scores, st);
  if (e == hipSuccess)
    e = ca::launch_select(d, scores, p->cached_len, top_frac, sink_blocks, local_blocks, nullptr,
                          st, words, group_size);
  if (e == hipSuccess) e = ca::launch_compact_words(d, rows, words, kv_indptr, kv_indices, st);
  return hip_status(e, "fused estimate-tables launch");
}

static ca_status check_threshold(float alpha, float temperature, float sm_scale,
                                 int32_t sink_blocks, int32_t local_blocks) {
  if (!(alpha > 0.f && alpha <= 1.f))
    return fail(CA_ERR_SHAPE, "alpha must be in (0, 1], got %g", (double)alpha);
  if (!(temperature > 0.f) || !(sm_scale > 0.f))
    return fail(CA_ERR_SHAPE, "temperature and sm_scale must be > 0");
  if (sink_blocks < 0 || local_blocks < 0)
    return fail(CA_ERR_SHAPE, "sink_blocks and local_blocks must be >= 0");
  return CA_OK;
}

ca_status ca_select_blocks_threshold(const ca_problem* p, const float* scores, float alpha,
                                    float temperature, float sm_scale, int32_t sink_blocks,
                                    int32_t local_blocks, uint64_t* masks, void* stream) {
  ca::Dims d;
  ca_status s = check(p, 0, &d);
  if (s != CA_OK) return s;
  if ((s = need_device(p)) != CA_OK) return s;
  if (!scores || !masks) return fail(CA_ERR_NULL, "scores and masks are required");
  if ((s = check_threshold(alpha, temperature, sm_scale, sink_blocks, local_blocks)) != CA_OK)
    return s;
  // margin = ln(alpha) / (temperature * sm_scale), rounded once to fp32
  const float margin = (float)(std::log((double)alpha) / ((double)temperature * sm_scale));
  return hip_status(ca::launch_threshold_select(d, scores, p->cached_len, margin, sink_blocks,
                                                local_blocks, masks,
                                                static_cast<hipStream_t>(stream)),
                    "threshold select launch");
}

ca_status ca_estimate_masks_threshold(const ca_problem* p, const uint16_t* q,
                                      const uint16_t* k_pool, const int32_t* page_table,
                                      float alpha, float temperature, float sm_scale,
                                      int32_t sink_blocks, int32_t local_blocks,
                                      int32_t k_mean_first_block, float* q_mean, float* k_mean,
                                      float* scores, uint64_t* masks, void* stream) {
  // the selection parameters are checked before the first stage is enqueued
  ca_status s = check_threshold(alpha, temperature, sm_scale, sink_blocks, local_blocks);
  if (s != CA_OK) return s;
  if (!masks) return fail(CA_ERR_NULL, "masks is required");
  if ((s = need_aligned16("q, k_pool, q_mean, k_mean and scores", q, k_pool, q_mean, k_mean,
                          scores)) != CA_OK)
    return s;
  if ((s = pool_both(p, q, k_pool, page_table, k_mean_first_block, q_mean, k_mean, stream)) !=
      CA_OK)
    return s;
  if ((s = ca_block_scores(p, q_mean, k_mean, scores, stream)) != CA_OK) return s;
  return ca_select_blocks_threshold(p, scores, alpha, temperature, sm_scale, sink_blocks,
                                    local_blocks, masks, stream);
}

size_t ca_tables_workspace_bytes(const ca_problem* p, int32_t group_size) {
  ca::Dims d;
  if (group_size < 1 || check(p, group_size, &d) != CA_OK) return 0;
  return ca::tables_ws_bytes(d, group_size);
}

ca_status ca_build_block_tables(const ca_problem* p, const uint64_t* masks, int32_t group_size,
                                int32_t* kv_indptr, int32_t* kv_indices, void* ws,
                                size_t ws_bytes, void* stream) {
  ca::Dims d;
  if (group_size < 1) return fail(CA_ERR_GROUP, "group_size must be >= 1");
  ca_status s = check(p, group_size, &d);
  if (s != CA_OK) return s;
  if ((s = need_device(p)) != CA_OK) return s;
  if (!masks || !kv_indptr || !kv_indices)
    return fail(CA_ERR_NULL, "masks, kv_indptr and kv_indices are required");
  const size_t need = ca::tables_ws_bytes(d, group_size);
  if (ws == nullptr || ws_bytes < need)
    return fail(CA_ERR_WORKSPACE, "tables need %zu workspace bytes, got %zu", need,
                ws == nullptr ? (size_t)0 : ws_bytes);
  if (reinterpret_cast<uintptr_t>(ws) % sizeof(uint64_t) != 0)
    return fail(CA_ERR_WORKSPACE, "workspace must be 8-byte aligned (it holds uint64 words)");
  return hip_status(ca::launch_tables(d, masks, p->cached_len, group_size, kv_indptr,
                                      kv_indices, ws, static_cast<hipStream_t>(stream)),
                    "tables launch");
}

ca_status ca_build_block_tables_noalloc(const ca_problem* p, const uint64_t* masks,
                                        int32_t group_size, int32_t* kv_indptr,
                                        int32_t* kv_indices, void* stream) {
  ca::Dims d;
  if (group_size < 1) return fail(CA_ERR_GROUP, "group_size must be >= 1");
  ca_status s = check(p, group_size, &d);
  if (s != CA_OK) return s;
  if ((s = need_device(p)) != CA_OK) return s;
  if (!masks || !kv_indptr || !kv_indices)
    return fail(CA_ERR_NULL, "masks, kv_indptr and kv_indices are required");
  const size_t need = ca::tables_ws_bytes(d, group_size);
  if (need > CA_NOALLOC_SCRATCH_BYTES)
    return fail(CA_ERR_WORKSPACE,
                "the tables need %zu scratch bytes (B * G rows x (W words + 1 count)), more than "
                "the %zu bytes of the allocation-free entry point: use ca_build_block_tables",
                need, (size_t)CA_NOALLOC_SCRATCH_BYTES);
  void* ws = nullptr;
  if ((s = scratch_ptr(&ws)) != CA_OK) return s;
  // union_kernel writes every word and count that compact_kernel reads, so the
  // previous call's contents need no clearing
  return hip_status(ca::launch_tables(d, masks, p->cached_len, group_size, kv_indptr,
                                      kv_indices, ws, static_cast<hipStream_t>(stream)),
                    "tables launch (allocation-free)");
}

size_t ca_attention_workspace_bytes(const ca_problem* p, int32_t group_size, int32_t num_splits) {
  ca::Dims d;
  if (group_size < 1 || check(p, group_size, &d) != CA_OK) return 0;
  if (num_splits < 0 || num_splits > 64) return 0;
  int s = num_splits;
  if (s == 0) {
    // room for the XCD-balanced split, or for the splits chosen without it
    const size_t uni = ca::attn_ws_bytes(d, auto_splits(d, group_size, (size_t)-1, true));
    const size_t bal = xcd_balance_ok(d, p, group_size, ca::kTablesPerGroup, false)
                           ? ca::attn_xcd_ws_bytes(d, group_size)
                           : 0;
    return bal > uni ? bal : uni;
  }
  return ca::attn_ws_bytes(d, s);
}

ca_status ca_chunk_attention(const ca_problem* p, const uint16_t* q, const uint16_t* k_pool,
                             const uint16_t* v_pool, const int32_t* page_table,
                             const int32_t* kv_indptr, const int32_t* kv_indices,
                             int32_t group_size, float sm_scale, int32_t num_splits,
                             uint16_t* out, float* lse, void* ws, size_t ws_bytes,
                             void* stream) {
  if (group_size < 1) return fail(CA_ERR_GROUP, "group_size must be >= 1");
  return run_attention(p, q, k_pool, v_pool, page_table, kv_indptr, kv_indices, group_size,
                       sm_scale, num_splits, out, lse, ws, ws_bytes, stream, false);
}

ca_status ca_dense_paged_chunk_attention(const ca_problem* p, const uint16_t* q,
                                         const uint16_t* k_pool, const uint16_t* v_pool,
                                         const int32_t* page_table, float sm_scale,
                                         int32_t num_splits, uint16_t* out, float* lse,
                                         void* ws, size_t ws_bytes, void* stream) {
  if (p == nullptr) return fail(CA_ERR_NULL, "problem is NULL");
  if (p->num_kv_heads < 1 || p->num_q_heads < p->num_kv_heads)
    return fail(CA_ERR_SHAPE, "num_q_heads must be >= num_kv_heads >= 1");
  // one execution group per KV head: every head of the KV group shares the table
  int gs = p->num_q_heads / p->num_kv_heads;
  while (gs > 1 && 128 % gs != 0) --gs;
  return run_attention(p, q, k_pool, v_pool, page_table, nullptr, nullptr, gs, sm_scale,
                       num_splits, out, lse, ws, ws_bytes, stream, true);
}

size_t ca_block_sparse_tables_workspace_bytes(const ca_problem* p, int32_t group_size) {
  ca::Dims d;
  if (group_size < 0 || check(p, group_size, &d) != CA_OK) return 0;
  if (group_size > 0) return ca::union_rows_ws_bytes(d, group_size);
  ca::Dims r = d;   // one table row per (b, h, Q-block): heads x Q-blocks, one Q-block each
  r.Hq = d.Hq * d.nqb;
  r.nqb = 1;
  return ca::tables_ws_bytes(r, 1);
}

ca_status ca_build_block_sparse_tables(const ca_problem* p, const uint64_t* masks,
                                       int32_t group_size, int32_t* kv_indptr,
                                       int32_t* kv_indices, void* ws, size_t ws_bytes,
                                       void* stream) {
  ca::Dims d;
  if (group_size < 0) return fail(CA_ERR_GROUP, "group_size must be >= 0");
  ca_status s = check(p, group_size, &d);
  if (s != CA_OK) return s;
  if ((s = need_device(p)) != CA_OK) return s;
  if (!masks || !kv_indptr || !kv_indices)
    return fail(CA_ERR_NULL, "masks, kv_indptr and kv_indices are required");
  const size_t need = ca_block_sparse_tables_workspace_bytes(p, group_size);
  if (ws == nullptr || ws_bytes < need)
    return fail(CA_ERR_WORKSPACE, "block-sparse tables need %zu workspace bytes, got %zu", need,
                ws == nullptr ? (size_t)0 : ws_bytes);
  if (reinterpret_cast<uintptr_t>(ws) % sizeof(uint64_t) != 0)
    return fail(CA_ERR_WORKSPACE, "workspace must be 8-byte aligned (it holds uint64 words)");
  hipStream_t st = static_cast<hipStream_t>(stream);
  if (group_size > 0)
    return hip_status(ca::launch_union_rows(d, masks, p->cached_len, group_size, kv_indptr,
                                            kv_indices, ws, st),
                      "block-sparse union rows launch");
  ca::Dims r = d;
  r.Hq = d.Hq * d.nqb;
  r.nqb = 1;
  return hip_status(ca::launch_tables(r, masks, p->cached_len, 1, kv_indptr, kv_indices, ws, st),
                    "block-sparse tables launch");
}

ca_status ca_block_sparse_chunk_attention(const ca_problem* p, const uint16_t* q,
                                          const uint16_t* k_pool, const uint16_t* v_pool,
                                          const int32_t* page_table, const int32_t* kv_indptr,
                                          const int32_t* kv_indices, float sm_scale,
                                          int32_t num_splits, uint16_t* out, float* lse,
                                          void* ws, size_t ws_bytes, void* stream) {
  return run_attention(p, q, k_pool, v_pool, page_table, kv_indptr, kv_indices, 1, sm_scale,
                       num_splits, out, lse, ws, ws_bytes, stream, false, ca::kTablesPerQTile);
}

ca_status ca_gather_selected_pages(const ca_problem* p, const uint16_t* k_pool,
                                   const uint16_t* v_pool, const int32_t* page_table,
                                   const int32_t* kv_indptr, const int32_t* kv_indices,
                                   int32_t group_size, uint16_t* k_packed, uint16_t* v_packed,
                                   int64_t capacity_pages, void* stream) {
  ca::Dims d;
  if (group_size < 1) return fail(CA_ERR_GROUP, "group_size must be >= 1");
  ca_status s = check(p, group_size, &d);
  if (s != CA_OK) return s;
  if (!k_pool || !v_pool || !page_table || !kv_indptr || !kv_indices || !k_packed || !v_packed)
    return fail(CA_ERR_NULL, "pools, page_table, tables and packed pools are required");
  if ((s = need_aligned16("k_pool, v_pool, k_packed and v_packed", k_pool, v_pool, k_packed,
                          v_packed)) != CA_OK)
    return s;
  const long long cap_max = (long long)d.B * (d.Hq / group_size) * d.max_kv_blocks;
  if (capacity_pages < 1 || capacity_pages > cap_max)
    return fail(CA_ERR_SHAPE, "capacity_pages %lld out of range [1, %lld]",
                (long long)capacity_pages, cap_max);
  return hip_status(ca::launch_gather(d, k_pool, v_pool, page_table, kv_indptr, kv_indices,
                                      group_size, capacity_pages, k_packed, v_packed,
                                      static_cast<hipStream_t>(stream)),
                    "gather launch");
}

ca_status ca_packed_chunk_attention(const ca_problem* p, const uint16_t* q,
                                    const uint16_t* k_packed, const uint16_t* v_packed,
                                    const int32_t* kv_indptr, const int32_t* kv_indices,
                                    int32_t group_size, float sm_scale, int32_t num_splits,
                                    int64_t capacity_pages, uint16_t* out, float* lse, void* ws,
                                    size_t ws_bytes, void* stream) {
  if (group_size < 1) return fail(CA_ERR_GROUP, "group_size must be >= 1");
  return run_attention(p, q, k_packed, v_packed, nullptr, kv_indptr, kv_indices, group_size,
                       sm_scale, num_splits, out, lse, ws, ws_bytes, stream, false,
                       ca::kTablesPacked, capacity_pages);
}

ca_status ca_check_tables_host(const ca_problem* p, int32_t group_size,
                               const int32_t* kv_indptr, const int32_t* kv_indices,
                               const int32_t* page_table, int64_t pool_pages,
                               int32_t require_chunk_open) {
  ca::Dims d;
  if (group_size < 0) return fail(CA_ERR_GROUP, "group_size must be >= 0");
  ca_status s = check(p, group_size, &d);
  if (s != CA_OK) return s;
  if (!kv_indptr || !kv_indices) return fail(CA_ERR_NULL, "kv_indptr and kv_indices are required");
  if (page_table && pool_pages < 0) return fail(CA_ERR_SHAPE, "pool_pages must be >= 0");
  return check_tables(p, d, group_size, kv_indptr, kv_indices, page_table, pool_pages,
                      require_chunk_open != 0);
}

ca_status ca_validate_tables(const ca_problem* p, int32_t group_size, const int32_t* kv_indptr,
                             const int32_t* kv_indices, int32_t require_chunk_open,
                             void* stream) {
  ca::Dims d;
  if (group_size < 1) return fail(CA_ERR_GROUP, "group_size must be >= 1");
  ca_status s = check(p, group_size, &d);
  if (s != CA_OK) return s;
  if (!kv_indptr || !kv_indices) return fail(CA_ERR_NULL, "kv_indptr and kv_indices are required");
  std::vector<int32_t> ip, ix, pt;
  if ((s = copy_tables(d, group_size, kv_indptr, kv_indices, nullptr,
                       static_cast<hipStream_t>(stream), ip, ix, pt)) != CA_OK)
    return s;
  return check_tables(p, d, group_size, ip.data(), ix.data(), nullptr, 0,
                      require_chunk_open != 0);
}

}  // extern "C"
