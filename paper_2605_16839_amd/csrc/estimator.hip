// Mean-pooled block-score selector: Q/K block pooling, block scores and the
// exact top-k + sink + local + chunk-causal mask emission.
//
// The paper plugs any lightweight block-level pattern search in front of the
// block union (Sec. 3.1, Sec. 3.2 first paragraph); per-chunk search cost is
// first-order under chunked prefill (Sec. 2.1), so every stage here is a
// single streaming pass: pooling is HBM-bound, scores are a small fp32
// contraction on the matrix cores, selection is an in-LDS radix select per
// mask row.
#include "common.hpp"
#include "kernels.hpp"

namespace ca {

// ---------------------------------------------------------------------------
// Pooling: one wavefront reduces `rows` rows of D bf16 (row stride `stride`
// elements) to their fp32 mean.  Lane l reads 16 bytes of row (l / CPR) +
// k*RPI, so each load instruction covers RPI whole rows contiguously; the
// lane adds its rows in ascending k, then the lanes holding the same chunk
// meet in a butterfly.
// ---------------------------------------------------------------------------
__device__ __forceinline__ void add_bf16x8(float (&acc)[8], const uint4& v) {
  acc[0] += bf16_lo(v.x); acc[1] += bf16_hi(v.x);
  acc[2] += bf16_lo(v.y); acc[3] += bf16_hi(v.y);
  acc[4] += bf16_lo(v.z); acc[5] += bf16_hi(v.z);
  acc[6] += bf16_lo(v.w); acc[7] += bf16_hi(v.w);
}

template <int D>
__device__ __forceinline__ void pool_store(float (&acc)[8], float* __restrict__ out, float scale) {
  constexpr int CPR = D / 8;
  const int l = lane_id();
#pragma unroll
  for (int o = CPR; o < kWave; o <<= 1) {
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[e] += __shfl_xor(acc[e], o, kWave);
  }
  if (l < CPR) {
    float4* dst = reinterpret_cast<float4*>(out + (l % CPR) * 8);
    dst[0] = make_float4(acc[0] * scale, acc[1] * scale, acc[2] * scale, acc[3] * scale);
    dst[1] = make_float4(acc[4] * scale, acc[5] * scale, acc[6] * scale, acc[7] * scale);
  }
}

// Any row count: one load per step of the loop.
template <int D>
__device__ __forceinline__ void pool_rows(const uint16_t* __restrict__ base, size_t stride,
                                          int rows, float* __restrict__ out, float scale) {
  constexpr int CPR = D / 8;           // 16-byte chunks per row
  constexpr int RPI = kWave / CPR;     // rows per load instruction
  const int l = lane_id();
  const int chunk = l % CPR;
  float acc[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) acc[e] = 0.f;
  for (int r = l / CPR; r < rows; r += RPI)
    add_bf16x8(acc, *reinterpret_cast<const uint4*>(base + (size_t)r * stride + chunk * 8));
  pool_store<D>(acc, out, scale);
}

// Exactly N * RPI rows: all N loads are issued before the first add, so a
// wave keeps N 16-byte loads per lane in flight instead of one (same adds,
// same order as pool_rows).
template <int D, int N>
__device__ __forceinline__ void pool_rows_n(const uint16_t* __restrict__ base, size_t stride,
                                            float* __restrict__ out, float scale) {
  constexpr int CPR = D / 8;
  constexpr int RPI = kWave / CPR;
  const int l = lane_id();
  const uint16_t* src = base + (size_t)(l / CPR) * stride + (l % CPR) * 8;
  uint4 v[N];
#pragma unroll
  for (int k = 0; k < N; ++k) v[k] = *reinterpret_cast<const uint4*>(src + (size_t)k * RPI * stride);
  float acc[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) acc[e] = 0.f;
#pragma unroll
  for (int k = 0; k < N; ++k) add_bf16x8(acc, v[k]);
  pool_store<D>(acc, out, scale);
}

// One launch pools both operands of the scores:
//   * workgroups [0, n_q_wg): one per (b, h, i) Q-block; each wave sums a
//     quarter of the block's rows and the four partial sums meet in LDS (the
//     chunk's last Q-block may hold fewer rows; its mean is over those);
//   * the rest: 4 waves per workgroup, one K block (b, kvh, j) per wave, j in
//     [first_block, nKB_b); a sequence's last block is pooled over its rows
//     before the sequence end only.
// In the fused estimator-to-union path the launch also clears the group union
// words that the selection ORs into (clear_words, n_clear; none otherwise).
struct PoolArgs {
  const uint16_t* q;
  float* q_mean;
  int B, C, Hq, q_block, nqb, n_q_wg;
  uint64_t* clear_words;
  int n_clear;
  const uint16_t* k_pool;
  const int32_t* page_table;
  const int32_t* cached_len;
  float* k_mean;
  int Hkv, max_kv_blocks, first_block, k_tiles;   // k_tiles workgroups per (b, kvh)
};

template <int D>
__global__ __launch_bounds__(256) void pool_kernel(const PoolArgs a) {
  __shared__ __attribute__((aligned(16))) float part[4][D];
  constexpr int RPI = kWave / (D / 8);
  for (int x = blockIdx.x * 256 + threadIdx.x; x < a.n_clear; x += gridDim.x * 256)
    a.clear_words[x] = 0ull;
  const int wv = threadIdx.x >> 6;
  if ((int)blockIdx.x < a.n_q_wg) {
    const int w = blockIdx.x;
    const int i = w % a.nqb;
    const int h = (w / a.nqb) % a.Hq;
    const int b = w / (a.nqb * a.Hq);
    const int quarter = a.q_block / 4;
    const int n_valid = a.C - i * a.q_block < a.q_block ? a.C - i * a.q_block : a.q_block;
    int rows = n_valid - wv * quarter;
    rows = rows < 0 ? 0 : (rows > quarter ? quarter : rows);
    const uint16_t* base =
        a.q + (((size_t)b * a.C + (size_t)i * a.q_block + (size_t)wv * quarter) * a.Hq + h) * D;
    const size_t stride = (size_t)a.Hq * D;
    if (rows == 8 * RPI) pool_rows_n<D, 8>(base, stride, part[wv], 1.0f);
    else pool_rows<D>(base, stride, rows, part[wv], 1.0f);
    __syncthreads();
    const int t = threadIdx.x;
    if (t < D)
      a.q_mean[(size_t)w * D + t] = ((part[0][t] + part[1][t]) + (part[2][t] + part[3][t])) *
                                    (1.0f / (float)n_valid);
    return;
  }
  const int kw = blockIdx.x - a.n_q_wg;
  const int bk = kw / a.k_tiles;   // b * Hkv + kvh
  const int b = bk / a.Hkv;
  const int j = a.first_block + (kw % a.k_tiles) * 4 + wv;
  const int seq = a.cached_len[b] + a.C;
  if (j >= blocks_for(seq)) return;
  const int rows = seq - kPage * j < kPage ? seq - kPage * j : kPage;
  const int page = a.page_table[(size_t)bk * a.max_kv_blocks + j];
  const uint16_t* base = a.k_pool + (size_t)page * kPage * D;
  float* out = a.k_mean + ((size_t)bk * a.max_kv_blocks + j) * D;
  if (rows == kPage) pool_rows_n<D, kPage / RPI>(base, D, out, 1.0f / (float)kPage);
  else pool_rows<D>(base, D, rows, out, 1.0f / (float)rows);
}

// ---------------------------------------------------------------------------
// Scores: for one (b, kvh), the ratio*nQB pooled query rows are contiguous in
// q_mean and the matching score rows are contiguous too.  One wave computes a
// 32-row x 32-block tile with fp32 matrix instructions (v_mfma_f32_32x32x2_f32,
// fp32 products and sums), its operands loaded straight into registers: lane
// l holds row / block l % 32 and, for k-step (t, e), element
// d = 8t + 4(l / 32) + e of both operands (the contraction over d may take
// the d in any order as long as both operands share it), so each lane loads
// its two rows as D/8 float4 pairs.  Four waves per workgroup.
// ---------------------------------------------------------------------------
typedef float f32x16 __attribute__((ext_vector_type(16)));

template <int D>
__global__ __launch_bounds__(256) void scores_kernel(const float* __restrict__ q_mean,
                                                     const float* __restrict__ k_mean,
                                                     const int32_t* __restrict__ cached_len,
                                                     float* __restrict__ scores, int Hq, int Hkv,
                                                     int nqb, int max_kv_blocks, int n_jt) {
  constexpr int NT = D / 8;
  const int bk = blockIdx.y;
  const int b = bk / Hkv, kvh = bk % Hkv;
  const int ratio = Hq / Hkv;
  const int nrows = ratio * nqb;
  const int nc = cached_len[b] / kPage;
  const int l = threadIdx.x & 63;
  const int tile = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int n_rt = (nrows + 31) / 32;
  const int rt = tile % n_rt, jt = tile / n_rt;
  const int r0 = rt * 32, j0 = jt * 32;
  if (jt >= n_jt || j0 >= nc) return;   // whole wave
  const size_t row_base = ((size_t)b * Hq + (size_t)kvh * ratio) * nqb;
  const int i = l & 31, h = l >> 5;
  const bool q_ok = r0 + i < nrows, k_ok = j0 + i < nc;
  const float* qrow = q_mean + (row_base + (q_ok ? r0 + i : 0)) * D + 4 * h;
  const float* krow = k_mean + ((size_t)bk * max_kv_blocks + (k_ok ? j0 + i : 0)) * D + 4 * h;
  float4 qa[NT], kb[NT];
#pragma unroll
  for (int t = 0; t < NT; ++t) {
    qa[t] = q_ok ? *reinterpret_cast<const float4*>(qrow + 8 * t) : make_float4(0.f, 0.f, 0.f, 0.f);
    kb[t] = k_ok ? *reinterpret_cast<const float4*>(krow + 8 * t) : make_float4(0.f, 0.f, 0.f, 0.f);
  }
  f32x16 acc;
#pragma unroll
  for (int v = 0; v < 16; ++v) acc[v] = 0.f;
#pragma unroll
  for (int t = 0; t < NT; ++t) {
    acc = __builtin_amdgcn_mfma_f32_32x32x2f32(qa[t].x, kb[t].x, acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_32x32x2f32(qa[t].y, kb[t].y, acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_32x32x2f32(qa[t].z, kb[t].z, acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_32x32x2f32(qa[t].w, kb[t].w, acc, 0, 0, 0);
  }
  // result v of lane l: row 8(v/4) + 4(l/32) + v%4 of the tile, block l % 32
  const int j = j0 + i;
  if (j >= nc) return;
#pragma unroll
  for (int v = 0; v < 16; ++v) {
    const int r = r0 + 8 * (v / 4) + 4 * h + (v % 4);
    if (r < nrows) scores[(row_base + r) * max_kv_blocks + j] = acc[v];
  }
}

// ---------------------------------------------------------------------------
// Selection: one workgroup (4 waves) per mask row (b, h, i).
// Scores become order-preserving uint32 keys (-0.0 folded onto +0.0); a
// 4-pass, 8-bit radix select finds the k-th largest key T and how many keys
// equal to T still have to be taken; those are the ones with the smallest
// block index (ranked by a ballot/prefix count).  Words of the mask are then
// emitted directly from wave ballots: wave v of a 256-block slab owns word
// slab/64 + v.
// ---------------------------------------------------------------------------
__device__ __forceinline__ uint32_t order_key(float f) {
  uint32_t u = __float_as_uint(f);
  if (u == 0x80000000u) u = 0u;
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// Block-wide inclusive scan of one int per thread (256 threads).
__device__ __forceinline__ int block_scan_256(int v, int* wave_tot) {
  const int w = threadIdx.x >> 6;
  int incl = wave_inclusive_scan(v);
  if (lane_id() == 63) wave_tot[w] = incl;
  __syncthreads();
  int add = 0;
  for (int x = 0; x < w; ++x) add += wave_tot[x];
  __syncthreads();
  return incl + add;
}

__global__ __launch_bounds__(256) void select_kernel(const float* __restrict__ scores,
                                                     const int32_t* __restrict__ cached_len,
                                                     uint64_t* __restrict__ masks, int Hq,
                                                     int nqb, int max_kv_blocks, int W,
                                                     int C, int q_block,
                                                     float top_frac, int sink_blocks,
                                                     int local_blocks,
                                                     unsigned long long* __restrict__ gwords,
                                                     int group_size) {
  extern __shared__ uint32_t keys[];
  __shared__ int hist[256];
  __shared__ int wave_tot[4];
  __shared__ int sh_digit, sh_above;
  const int row = blockIdx.x;
  const int t = threadIdx.x;
  const int wv = t >> 6;
  const int i = row % nqb;
  const int b = row / (nqb * Hq);
  const int cl = cached_len[b];
  const int nc = cl / kPage;            // full cached blocks: the candidates
  const int nkb = blocks_for(cl + C);
  int k = 0;
  if (nc > 0) {
    k = (int)ceilf(top_frac * (float)nc);
    k = k < 0 ? 0 : (k > nc ? nc : k);
  }
  const float* s = scores + (size_t)row * max_kv_blocks;
  // 8 loads per lane in flight per round (2048 scores)
  for (int j0 = 0; j0 < nc; j0 += 8 * 256) {
    float v[8];
#pragma unroll
    for (int m = 0; m < 8; ++m) {
      const int j = j0 + t + 256 * m;
      v[m] = j < nc ? s[j] : 0.f;
    }
#pragma unroll
    for (int m = 0; m < 8; ++m) {
      const int j = j0 + t + 256 * m;
      if (j < nc) keys[j] = order_key(v[m]);
    }
  }
  __syncthreads();

  const bool take_all = (k == nc);
  uint32_t prefix = 0u, pmask = 0u;
  int remaining = k;
  if (k > 0 && !take_all) {
    for (int shift = 24; shift >= 0; shift -= 8) {
      hist[t] = 0;
      __syncthreads();
      for (int j = t; j < nc; j += 256) {
        const uint32_t key = keys[j];
        if ((key & pmask) == prefix) atomicAdd(&hist[(key >> shift) & 255u], 1);
      }
      __syncthreads();
      // thread t <-> digit 255 - t: the inclusive scan counts keys with digit >= d
      const int d = 255 - t;
      const int c = hist[d];
      const int incl = block_scan_256(c, wave_tot);
      const int excl = incl - c;
      if (excl < remaining && remaining <= incl) {
        sh_digit = d;
        sh_above = excl;
      }
      __syncthreads();
      prefix |= (uint32_t)sh_digit << shift;
      pmask |= 0xffu << shift;
      remaining -= sh_above;
      __syncthreads();
    }
  }
  const uint32_t T = prefix;

  const int causal_end = causal_block_end(cl, C, i, q_block);
  const int sink_end = sink_blocks < nc ? sink_blocks : nc;
  const int local_begin = nc - local_blocks;
  int carry = 0;  // keys equal to T already seen, in block order
  uint64_t* mrow = masks + (size_t)row * W;
  // fused path: OR the row straight into the words of its group's table row
  const int h = (row / nqb) % Hq;
  unsigned long long* grow =
      gwords ? gwords + ((size_t)b * (Hq / group_size) + h / group_size) * W : nullptr;
  for (int base = 0; base < W * 64; base += 256) {
    const int j = base + t;
    const bool cached = j < nc;
    const uint32_t key = cached ? keys[j] : 0u;
    const bool eq = cached && k > 0 && !take_all && key == T;
    const uint64_t bal = __ballot(eq);
    if (lane_id() == 0) wave_tot[wv] = __popcll(bal);
    __syncthreads();
    int before = carry, total = 0;
    for (int x = 0; x < 4; ++x) {
      if (x < wv) before += wave_tot[x];
      total += wave_tot[x];
    }
    const int rank = before + lanes_below(bal);
    const bool sel = cached && (take_all || (k > 0 && (key > T || (eq && rank < remaining))));
    const bool forced = j < nkb && ((j < sink_end) || (j >= local_begin && j < nc) ||
                                    (j >= nc && j < causal_end));
    const uint64_t word = __ballot(sel || forced);
    const int widx = j >> 6;
    if (lane_id() == 0 && widx < W) {
      if (grow == nullptr) mrow[widx] = word;
      else if (word) atomicOr(grow + widx, (unsigned long long)word);
    }
    carry += total;
    __syncthreads();
  }
}

// ---------------------------------------------------------------------------
// Threshold selection (the alpha / max-threshold reading): one workgroup per
// mask row keeps every cached block with s_j >= s_max + margin (the sum in
// fp32), plus the same sink, local and chunk-causal bits as select_kernel.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void threshold_select_kernel(
    const float* __restrict__ scores, const int32_t* __restrict__ cached_len,
    uint64_t* __restrict__ masks, int Hq, int nqb, int max_kv_blocks, int W, int C,
    int q_block, float margin, int sink_blocks, int local_blocks) {
  __shared__ float red[4];
  const int row = blockIdx.x;
  const int t = threadIdx.x;
  const int wv = t >> 6;
  const int i = row % nqb;
  const int b = row / (nqb * Hq);
  const int cl = cached_len[b];
  const int nc = cl / kPage;
  const int nkb = blocks_for(cl + C);
  const float* s = scores + (size_t)row * max_kv_blocks;
  float mx = -INFINITY;
  for (int j = t; j < nc; j += 256) mx = fmaxf(mx, s[j]);
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) mx = fmaxf(mx, __shfl_xor(mx, o, kWave));
  if (lane_id() == 0) red[wv] = mx;
  __syncthreads();
  mx = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
  const float thr = mx + margin;
  const int causal_end = causal_block_end(cl, C, i, q_block);
  const int sink_end = sink_blocks < nc ? sink_blocks : nc;
  const int local_begin = nc - local_blocks;
  uint64_t* mrow = masks + (size_t)row * W;
  for (int base = 0; base < W * 64; base += 256) {
    const int j = base + t;
    const bool sel = j < nc && s[j] >= thr;
    const bool forced = j < nkb && ((j < sink_end) || (j >= local_begin && j < nc) ||
                                    (j >= nc && j < causal_end));
    const uint64_t word = __ballot(sel || forced);
    const int widx = j >> 6;
    if (lane_id() == 0 && widx < W) mrow[widx] = word;
  }
}

// ---------------------------------------------------------------------------
// launchers
// ---------------------------------------------------------------------------
// q == nullptr: no Q pooling; k_pool == nullptr: no K pooling.
hipError_t launch_pool(const Dims& d, const uint16_t* q, float* q_mean, const uint16_t* k_pool,
                       const int32_t* page_table, const int32_t* cached_len, int first_block,
                       float* k_mean, hipStream_t st, uint64_t* clear_words, int n_clear) {
  PoolArgs a;
  a.q = q;
  a.q_mean = q_mean;
  a.B = d.B;
  a.C = d.C;
  a.Hq = d.Hq;
  a.q_block = d.q_block;
  a.nqb = d.nqb;
  a.n_q_wg = q != nullptr ? d.B * d.Hq * d.nqb : 0;
  a.clear_words = clear_words;
  a.n_clear = n_clear;
  a.k_pool = k_pool;
  a.page_table = page_table;
  a.cached_len = cached_len;
  a.k_mean = k_mean;
  a.Hkv = d.Hkv;
  a.max_kv_blocks = d.max_kv_blocks;
  a.first_block = first_block;
  const int span = d.max_nkb - first_block;
  a.k_tiles = k_pool != nullptr && span > 0 ? (span + 3) / 4 : 0;
  const long long nwg = (long long)a.n_q_wg + (long long)a.k_tiles * d.B * d.Hkv;
  if (nwg == 0) return hipSuccess;
  if (nwg > 0x7fffffffLL) return hipErrorInvalidConfiguration;
  if (d.D == 128) pool_kernel<128><<<(int)nwg, 256, 0, st>>>(a);
  else pool_kernel<64><<<(int)nwg, 256, 0, st>>>(a);
  return hipGetLastError();
}

hipError_t launch_pool_q(const Dims& d, const uint16_t* q, float* q_mean, hipStream_t st,
                         uint64_t* clear_words, int n_clear) {
  return launch_pool(d, q, q_mean, nullptr, nullptr, nullptr, 0, nullptr, st, clear_words,
                     n_clear);
}

hipError_t launch_pool_k(const Dims& d, const uint16_t* k_pool, const int32_t* page_table,
                         const int32_t* cached_len, int first_block, float* k_mean,
                         hipStream_t st) {
  return launch_pool(d, nullptr, nullptr, k_pool, page_table, cached_len, first_block, k_mean,
                     st, nullptr, 0);
}

hipError_t launch_scores(const Dims& d, const float* q_mean, const float* k_mean,
                         const int32_t* cached_len, float* scores, hipStream_t st) {
  if (d.max_nc <= 0) return hipSuccess;
  const int nrows = (d.Hq / d.Hkv) * d.nqb;
  const int n_jt = (d.max_nc + 31) / 32;
  const int tiles = ((nrows + 31) / 32) * n_jt;
  dim3 grid((tiles + 3) / 4, d.B * d.Hkv);
  if (d.D == 128)
    scores_kernel<128><<<grid, 256, 0, st>>>(q_mean, k_mean, cached_len, scores, d.Hq, d.Hkv,
                                             d.nqb, d.max_kv_blocks, n_jt);
  else
    scores_kernel<64><<<grid, 256, 0, st>>>(q_mean, k_mean, cached_len, scores, d.Hq, d.Hkv,
                                            d.nqb, d.max_kv_blocks, n_jt);
  return hipGetLastError();
}

hipError_t raise_select_lds(int bytes) {
  return hipFuncSetAttribute(reinterpret_cast<const void*>(&select_kernel),
                             hipFuncAttributeMaxDynamicSharedMemorySize, bytes);
}

hipError_t launch_select(const Dims& d, const float* scores, const int32_t* cached_len,
                         float top_frac, int sink_blocks, int local_blocks, uint64_t* masks,
                         hipStream_t st, uint64_t* group_words, int group_size) {
  dim3 grid(d.B * d.Hq * d.nqb);
  const size_t lds = (size_t)(d.max_nc > 0 ? d.max_nc : 1) * sizeof(uint32_t);
  select_kernel<<<grid, 256, lds, st>>>(scores, cached_len, masks, d.Hq, d.nqb,
                                        d.max_kv_blocks, d.W, d.C, d.q_block, top_frac,
                                        sink_blocks, local_blocks,
                                        reinterpret_cast<unsigned long long*>(group_words),
                                        group_size);
  return hipGetLastError();
}


hipError_t launch_threshold_select(const Dims& d, const float* scores, const int32_t* cached_len,
                                   float margin, int sink_blocks, int local_blocks,
                                   uint64_t* masks, hipStream_t st) {
  dim3 grid(d.B * d.Hq * d.nqb);
  threshold_select_kernel<<<grid, 256, 0, st>>>(scores, cached_len, masks, d.Hq, d.nqb,
                                                d.max_kv_blocks, d.W, d.C, d.q_block,
                                                margin, sink_blocks, local_blocks);
  return hipGetLastError();
}

}  // namespace ca
