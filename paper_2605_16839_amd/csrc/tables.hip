// Block-union tables: Q-block union + intra-group union (bitwise OR) and
// compaction of the union bitmask into CSR kv_indptr / kv_indices
// (Sec. 3.2 displayed equations; App. B.2 for the CSR pair).
//
// Two launches, both integer-only and deterministic:
//   union_kernel   one workgroup per table row r = b*G + g: OR the
//                  group_size*nQB mask rows of the group word by word in LDS
//                  (ds_or_b64), clip to nKB_b, store the row's union words and
//                  its popcount;
//   compact_kernel one workgroup per row: row offset = sum of the counts of
//                  earlier rows (no atomics), then 256-block slabs are
//                  compacted with wave ballots + a 4-wave prefix in LDS, which
//                  writes the set block ids in ascending order.
#include "common.hpp"
#include "kernels.hpp"

namespace ca {

constexpr int kMaxWords = kMaxKvBlocks / 64;

__global__ __launch_bounds__(256) void union_kernel(const uint64_t* __restrict__ masks,
                                                    const int32_t* __restrict__ cached_len,
                                                    uint64_t* __restrict__ gwords,
                                                    int32_t* __restrict__ counts, int Hq,
                                                    int nqb, int W, int group_size, int G,
                                                    int C) {
  __shared__ unsigned long long acc[kMaxWords];
  __shared__ int red[4];
  const int r = blockIdx.x;
  const int b = r / G, g = r % G;
  const int t = threadIdx.x;
  const int nkb = blocks_for(cached_len[b] + C);
  for (int w = t; w < W; w += 256) acc[w] = 0ull;
  __syncthreads();
  const int rows = group_size * nqb;
  const uint64_t* src = masks + ((size_t)b * Hq + (size_t)g * group_size) * nqb * W;
  if (W <= 256 && (256 % W) == 0) {
    // fixed word per thread: OR privately, then one LDS atomic
    // 8 loads per lane in flight per round
    const int w = t % W, step = 256 / W;
    unsigned long long v = 0ull;
    for (int row0 = t / W; row0 < rows; row0 += 8 * step) {
      unsigned long long x[8];
#pragma unroll
      for (int m = 0; m < 8; ++m) {
        const int row = row0 + m * step;
        x[m] = row < rows ? src[(size_t)row * W + w] : 0ull;
      }
#pragma unroll
      for (int m = 0; m < 8; ++m) v |= x[m];
    }
    if (v) atomicOr(&acc[w], v);
  } else {
    for (int x = t; x < rows * W; x += 256) {
      const unsigned long long v = src[x];
      if (v) atomicOr(&acc[x % W], v);
    }
  }
  __syncthreads();
  int cnt = 0;
  for (int w = t; w < W; w += 256) {
    unsigned long long v = acc[w];
    const int lo = w * 64;
    if (lo >= nkb) v = 0ull;
    else if (nkb - lo < 64) v &= (~0ull >> (64 - (nkb - lo)));
    gwords[(size_t)r * W + w] = v;
    cnt += __popcll(v);
  }
  cnt = wave_sum(cnt);
  if (lane_id() == 0) red[t >> 6] = cnt;
  __syncthreads();
  if (t == 0) counts[r] = red[0] + red[1] + red[2] + red[3];
}

// Writes the set bits of one row's words, ascending, from row_start on.
__device__ void compact_row(const uint64_t* __restrict__ gw, int row_start,
                            int32_t* __restrict__ kv_indices, int W, int* wave_tot) {
  const int t = threadIdx.x;
  const int wv = t >> 6;
  int carry = 0;
  for (int base = 0; base < W * 64; base += 256) {
    const int j = base + t;
    const int w = j >> 6;
    const bool bit = (w < W) && ((gw[w] >> (j & 63)) & 1ull);
    const uint64_t bal = __ballot(bit);
    if (lane_id() == 0) wave_tot[wv] = __popcll(bal);
    __syncthreads();
    int before = carry, total = 0;
    for (int x = 0; x < 4; ++x) {
      if (x < wv) before += wave_tot[x];
      total += wave_tot[x];
    }
    if (bit) kv_indices[row_start + before + lanes_below(bal)] = j;
    carry += total;
    __syncthreads();
  }
}

__global__ __launch_bounds__(256) void compact_kernel(const uint64_t* __restrict__ gwords,
                                                      const int32_t* __restrict__ counts,
                                                      int32_t* __restrict__ kv_indptr,
                                                      int32_t* __restrict__ kv_indices, int W) {
  __shared__ int red[4];
  __shared__ int wave_tot[4];
  const int r = blockIdx.x;
  const int t = threadIdx.x;
  int part = 0;
  for (int x = t; x < r; x += 256) part += counts[x];
  part = wave_sum(part);
  if (lane_id() == 0) red[t >> 6] = part;
  __syncthreads();
  const int row_start = red[0] + red[1] + red[2] + red[3];
  if (t == 0) {
    if (r == 0) kv_indptr[0] = 0;
    kv_indptr[r + 1] = row_start + counts[r];
  }
  compact_row(gwords + (size_t)r * W, row_start, kv_indices, W, wave_tot);
}

// Same, with the counts taken from the words themselves: row r starts after
// the set bits of rows 0..r-1 (the fused estimator-to-union path, whose
// words are complete only once every selection row has been ORed in).
__global__ __launch_bounds__(256) void compact_words_kernel(const uint64_t* __restrict__ gwords,
                                                            int32_t* __restrict__ kv_indptr,
                                                            int32_t* __restrict__ kv_indices,
                                                            int W) {
  __shared__ int red[8];
  __shared__ int wave_tot[4];
  const int r = blockIdx.x;
  const int t = threadIdx.x;
  int before = 0, own = 0;
  for (int x = t; x < (r + 1) * W; x += 256) {
    const int c = __popcll(gwords[x]);
    if (x < r * W) before += c;
    else own += c;
  }
  before = wave_sum(before);
  own = wave_sum(own);
  if (lane_id() == 0) {
    red[t >> 6] = before;
    red[4 + (t >> 6)] = own;
  }
  __syncthreads();
  const int row_start = red[0] + red[1] + red[2] + red[3];
  if (t == 0) {
    if (r == 0) kv_indptr[0] = 0;
    kv_indptr[r + 1] = row_start + red[4] + red[5] + red[6] + red[7];
  }
  compact_row(gwords + (size_t)r * W, row_start, kv_indices, W, wave_tot);
}

hipError_t launch_compact_words(const Dims& d, int rows, const uint64_t* words,
                                int32_t* kv_indptr, int32_t* kv_indices, hipStream_t st) {
  compact_words_kernel<<<rows, 256, 0, st>>>(words, kv_indptr, kv_indices, d.W);
  return hipGetLastError();
}

// Block-sparse arm at matched tables (Sec. 4.4): the union of execution group
// g(h) as the mask row of every (b, h, Q-block i), limited to the blocks that
// Q-block i can see causally (up to the block holding its last query).  One
// workgroup per (b, h, i) row; words from the group rows written by
// union_kernel.
__global__ __launch_bounds__(256) void expand_union_kernel(const uint64_t* __restrict__ gwords,
                                                           const int32_t* __restrict__ cached_len,
                                                           uint64_t* __restrict__ rwords,
                                                           int32_t* __restrict__ counts, int Hq,
                                                           int nqb, int W, int group_size,
                                                           int q_block, int C) {
  __shared__ int red[4];
  const int r = blockIdx.x;                 // (b*Hq + h)*nqb + i
  const int i = r % nqb;
  const int h = (r / nqb) % Hq;
  const int b = r / (nqb * Hq);
  const int G = Hq / group_size;
  const int t = threadIdx.x;
  const int lim = causal_block_end(cached_len[b], C, i, q_block);
  const uint64_t* src = gwords + ((size_t)b * G + h / group_size) * W;
  int cnt = 0;
  for (int w = t; w < W; w += 256) {
    unsigned long long v = src[w];
    const int lo = w * 64;
    if (lo >= lim) v = 0ull;
    else if (lim - lo < 64) v &= (~0ull >> (64 - (lim - lo)));
    rwords[(size_t)r * W + w] = v;
    cnt += __popcll(v);
  }
  cnt = wave_sum(cnt);
  if (lane_id() == 0) red[t >> 6] = cnt;
  __syncthreads();
  if (t == 0) counts[r] = red[0] + red[1] + red[2] + red[3];
}

// The per-row words follow the group-row workspace at the next 8-byte boundary
// (the group-row part ends with one int32 count per row).
static size_t union_rows_offset(const Dims& d, int group_size) {
  return (tables_ws_bytes(d, group_size) + 7) & ~(size_t)7;
}

size_t union_rows_ws_bytes(const Dims& d, int group_size) {
  const size_t R = (size_t)d.B * d.Hq * d.nqb;
  return union_rows_offset(d, group_size) + R * d.W * sizeof(uint64_t) + R * sizeof(int32_t);
}

hipError_t launch_union_rows(const Dims& d, const uint64_t* masks, const int32_t* cached_len,
                             int group_size, int32_t* kv_indptr, int32_t* kv_indices, void* ws,
                             hipStream_t st) {
  const int G = d.Hq / group_size;
  const int RG = d.B * G;
  const int R = d.B * d.Hq * d.nqb;
  uint64_t* gwords = static_cast<uint64_t*>(ws);
  int32_t* gcounts = reinterpret_cast<int32_t*>(gwords + (size_t)RG * d.W);
  uint64_t* rwords = reinterpret_cast<uint64_t*>(
      static_cast<char*>(ws) + union_rows_offset(d, group_size));
  int32_t* rcounts = reinterpret_cast<int32_t*>(rwords + (size_t)R * d.W);
  union_kernel<<<RG, 256, 0, st>>>(masks, cached_len, gwords, gcounts, d.Hq, d.nqb, d.W,
                                   group_size, G, d.C);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  expand_union_kernel<<<R, 256, 0, st>>>(gwords, cached_len, rwords, rcounts, d.Hq, d.nqb, d.W,
                                         group_size, d.q_block, d.C);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  compact_kernel<<<R, 256, 0, st>>>(rwords, rcounts, kv_indptr, kv_indices, d.W);
  return hipGetLastError();
}

size_t tables_ws_bytes(const Dims& d, int group_size) {
  const size_t R = (size_t)d.B * (d.Hq / group_size);
  return R * d.W * sizeof(uint64_t) + R * sizeof(int32_t);
}

hipError_t launch_tables(const Dims& d, const uint64_t* masks, const int32_t* cached_len,
                         int group_size, int32_t* kv_indptr, int32_t* kv_indices, void* ws,
                         hipStream_t st) {
  const int G = d.Hq / group_size;
  const int R = d.B * G;
  uint64_t* gwords = static_cast<uint64_t*>(ws);
  int32_t* counts = reinterpret_cast<int32_t*>(gwords + (size_t)R * d.W);
  union_kernel<<<R, 256, 0, st>>>(masks, cached_len, gwords, counts, d.Hq, d.nqb, d.W,
                                  group_size, G, d.C);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  compact_kernel<<<R, 256, 0, st>>>(gwords, counts, kv_indptr, kv_indices, d.W);
  return hipGetLastError();
}

}  // namespace ca
