// Mean-pooled block-score selector: Q/K block pooling, block scores and the
// exact top-k + sink + local + chunk-causal mask emission.
//
// The paper plugs any lightweight block-level pattern search in front of the
// block union (Sec. 3.1, Sec. 3.2 first paragraph); per-chunk search cost is
// first-order under chunked prefill (Sec. 2.1), so every stage here is a
// single streaming pass: pooling is HBM-bound, scores are a tiny fp32
// contraction, selection is an in-LDS radix select per mask row.
#include "common.hpp"
#include "kernels.hpp"

namespace ca {

// ---------------------------------------------------------------------------
// Pooling: one wavefront reduces `rows` rows of D bf16 (row stride `stride`
// elements) to their fp32 mean.  Lane l reads 16 bytes of row (l / CPR) +
// k*RPI, so each load instruction covers RPI whole rows contiguously.
// ---------------------------------------------------------------------------
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
  for (int r = l / CPR; r < rows; r += RPI) {
    const uint4 v = *reinterpret_cast<const uint4*>(base + (size_t)r * stride + chunk * 8);
    acc[0] += bf16_lo(v.x); acc[1] += bf16_hi(v.x);
    acc[2] += bf16_lo(v.y); acc[3] += bf16_hi(v.y);
    acc[4] += bf16_lo(v.z); acc[5] += bf16_hi(v.z);
    acc[6] += bf16_lo(v.w); acc[7] += bf16_hi(v.w);
  }
#pragma unroll
  for (int o = CPR; o < kWave; o <<= 1) {
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[e] += __shfl_xor(acc[e], o, kWave);
  }
  if (l < CPR) {
    float4* dst = reinterpret_cast<float4*>(out + chunk * 8);
    dst[0] = make_float4(acc[0] * scale, acc[1] * scale, acc[2] * scale, acc[3] * scale);
    dst[1] = make_float4(acc[4] * scale, acc[5] * scale, acc[6] * scale, acc[7] * scale);
  }
}

// One workgroup per (b, h, i): each wave sums a quarter of the Q-block's rows,
// the four partial sums meet in LDS.  In the fused estimator-to-union path
// this first stage also clears the group union words that the selection
// ORs into (clear_words, n_clear; none otherwise).
template <int D>
__global__ __launch_bounds__(256) void pool_q_kernel(const uint16_t* __restrict__ q,
                                                     float* __restrict__ q_mean, int B, int C,
                                                     int Hq, int q_block, int nqb,
                                                     uint64_t* __restrict__ clear_words,
                                                     int n_clear) {
  __shared__ __attribute__((aligned(16))) float part[4][D];
  for (int x = blockIdx.x * 256 + threadIdx.x; x < n_clear; x += gridDim.x * 256)
    clear_words[x] = 0ull;
  const int w = blockIdx.x;
  const int i = w % nqb;
  const int h = (w / nqb) % Hq;
  const int b = w / (nqb * Hq);
  const int wv = threadIdx.x >> 6;
  const int quarter = q_block / 4;
  // the chunk's last Q-block may hold fewer rows; its mean is over those
  const int n_valid = C - i * q_block < q_block ? C - i * q_block : q_block;
  int rows = n_valid - wv * quarter;
  rows = rows < 0 ? 0 : (rows > quarter ? quarter : rows);
  const uint16_t* base =
      q + (((size_t)b * C + (size_t)i * q_block + (size_t)wv * quarter) * Hq + h) * D;
  pool_rows<D>(base, (size_t)Hq * D, rows, part[wv], 1.0f);
  __syncthreads();
  const int t = threadIdx.x;
  if (t < D)
    q_mean[(size_t)w * D + t] = ((part[0][t] + part[1][t]) + (part[2][t] + part[3][t])) *
                                (1.0f / (float)n_valid);
}

// One wave per (b, kvh, j), j in [first_block, nKB_b).  A sequence's last
// block is pooled over its rows before the sequence end only.
template <int D>
__global__ __launch_bounds__(256) void pool_k_kernel(const uint16_t* __restrict__ k_pool,
                                                     const int32_t* __restrict__ page_table,
                                                     const int32_t* __restrict__ cached_len,
                                                     float* __restrict__ k_mean, int Hkv,
                                                     int max_kv_blocks, int C,
                                                     int first_block) {
  const int bk = blockIdx.y;  // b * Hkv + kvh
  const int b = bk / Hkv;
  const int j = first_block + blockIdx.x * 4 + (threadIdx.x >> 6);
  const int seq = cached_len[b] + C;
  if (j >= blocks_for(seq)) return;
  const int rows = seq - kPage * j < kPage ? seq - kPage * j : kPage;
  const int page = page_table[(size_t)bk * max_kv_blocks + j];
  pool_rows<D>(k_pool + (size_t)page * kPage * D, D, rows,
               k_mean + ((size_t)bk * max_kv_blocks + j) * D, 1.0f / (float)rows);
}

// ---------------------------------------------------------------------------
// Scores: for one (b, kvh), the ratio*nQB pooled query rows are contiguous in
// q_mean and the matching score rows are contiguous too.  A workgroup
// computes a 64-row x 32-block tile with fp32 FMAs (d ascending) from whole
// rows of both operands staged in LDS; lanes 0..15 of a row group own 16
// consecutive blocks, so the score stores are contiguous.
// ---------------------------------------------------------------------------
template <int D>
__global__ __launch_bounds__(256) void scores_kernel(const float* __restrict__ q_mean,
                                                     const float* __restrict__ k_mean,
                                                     const int32_t* __restrict__ cached_len,
                                                     float* __restrict__ scores, int Hq, int Hkv,
                                                     int nqb, int max_kv_blocks) {
  constexpr int TR = 64, TB = 32;
  __shared__ float qs[TR][D + 1];
  __shared__ float ks[TB][D + 1];
  const int bk = blockIdx.z;
  const int b = bk / Hkv, kvh = bk % Hkv;
  const int ratio = Hq / Hkv;
  const int nrows = ratio * nqb;
  const int nc = cached_len[b] / kPage;
  const int j0 = blockIdx.x * TB, r0 = blockIdx.y * TR;
  if (j0 >= nc) return;
  const size_t row_base = ((size_t)b * Hq + (size_t)kvh * ratio) * nqb;
  const float* qrow = q_mean + row_base * D;
  const float* krow = k_mean + ((size_t)bk * max_kv_blocks) * D;
  const int t = threadIdx.x;
  for (int x = t; x < TR * D / 4; x += 256) {
    const int r = x / (D / 4), d4 = x % (D / 4);
    const float4 v = (r0 + r < nrows)
                         ? *reinterpret_cast<const float4*>(qrow + (size_t)(r0 + r) * D + 4 * d4)
                         : make_float4(0.f, 0.f, 0.f, 0.f);
    qs[r][4 * d4 + 0] = v.x; qs[r][4 * d4 + 1] = v.y;
    qs[r][4 * d4 + 2] = v.z; qs[r][4 * d4 + 3] = v.w;
  }
  for (int x = t; x < TB * D / 4; x += 256) {
    const int r = x / (D / 4), d4 = x % (D / 4);
    const float4 v = (j0 + r < nc)
                         ? *reinterpret_cast<const float4*>(krow + (size_t)(j0 + r) * D + 4 * d4)
                         : make_float4(0.f, 0.f, 0.f, 0.f);
    ks[r][4 * d4 + 0] = v.x; ks[r][4 * d4 + 1] = v.y;
    ks[r][4 * d4 + 2] = v.z; ks[r][4 * d4 + 3] = v.w;
  }
  __syncthreads();
  const int bc = t & 15, rg = t >> 4;   // blocks bc, bc+16; rows rg + 16a
  float acc[4][2];
#pragma unroll
  for (int a = 0; a < 4; ++a) { acc[a][0] = 0.f; acc[a][1] = 0.f; }
#pragma unroll 8
  for (int d = 0; d < D; ++d) {
    const float k0 = ks[bc][d], k1 = ks[bc + 16][d];
#pragma unroll
    for (int a = 0; a < 4; ++a) {
      const float qv = qs[rg + 16 * a][d];
      acc[a][0] = fmaf(qv, k0, acc[a][0]);
      acc[a][1] = fmaf(qv, k1, acc[a][1]);
    }
  }
#pragma unroll
  for (int a = 0; a < 4; ++a) {
    const int r = r0 + rg + 16 * a;
    if (r >= nrows) continue;
#pragma unroll
    for (int c = 0; c < 2; ++c) {
      const int j = j0 + bc + 16 * c;
      if (j < nc) scores[(row_base + r) * max_kv_blocks + j] = acc[a][c];
    }
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
  for (int j = t; j < nc; j += 256) keys[j] = order_key(s[j]);
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
hipError_t launch_pool_q(const Dims& d, const uint16_t* q, float* q_mean, hipStream_t st,
                         uint64_t* clear_words, int n_clear) {
  dim3 grid(d.B * d.Hq * d.nqb);
  if (d.D == 128)
    pool_q_kernel<128><<<grid, 256, 0, st>>>(q, q_mean, d.B, d.C, d.Hq, d.q_block, d.nqb,
                                             clear_words, n_clear);
  else
    pool_q_kernel<64><<<grid, 256, 0, st>>>(q, q_mean, d.B, d.C, d.Hq, d.q_block, d.nqb,
                                            clear_words, n_clear);
  return hipGetLastError();
}

hipError_t launch_pool_k(const Dims& d, const uint16_t* k_pool, const int32_t* page_table,
                         const int32_t* cached_len, int first_block, float* k_mean,
                         hipStream_t st) {
  const int span = d.max_nkb - first_block;
  if (span <= 0) return hipSuccess;
  dim3 grid((span + 3) / 4, d.B * d.Hkv);
  if (d.D == 128)
    pool_k_kernel<128><<<grid, 256, 0, st>>>(k_pool, page_table, cached_len, k_mean, d.Hkv,
                                             d.max_kv_blocks, d.C, first_block);
  else
    pool_k_kernel<64><<<grid, 256, 0, st>>>(k_pool, page_table, cached_len, k_mean, d.Hkv,
                                            d.max_kv_blocks, d.C, first_block);
  return hipGetLastError();
}

hipError_t launch_scores(const Dims& d, const float* q_mean, const float* k_mean,
                         const int32_t* cached_len, float* scores, hipStream_t st) {
  if (d.max_nc <= 0) return hipSuccess;
  const int nrows = (d.Hq / d.Hkv) * d.nqb;
  dim3 grid((d.max_nc + 31) / 32, (nrows + 63) / 64, d.B * d.Hkv);
  if (d.D == 128)
    scores_kernel<128><<<grid, 256, 0, st>>>(q_mean, k_mean, cached_len, scores, d.Hq, d.Hkv,
                                             d.nqb, d.max_kv_blocks);
  else
    scores_kernel<64><<<grid, 256, 0, st>>>(q_mean, k_mean, cached_len, scores, d.Hq, d.Hkv,
                                            d.nqb, d.max_kv_blocks);
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
