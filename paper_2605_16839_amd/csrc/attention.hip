// Zero-copy paged chunk attention over per-group block tables (Sec. 3.3,
// App. B.2), bf16 MFMA with fp32 online softmax, and the split-KV
// log-sum-exp combine.
//
// Work decomposition (one workgroup = 4 wavefronts = 128 (head, query) rows):
//   * a table row r = b*G + g serves the group_size query heads of group g;
//     all of them read the same KV pages, so a workgroup packs rows of every
//     head of the group (group_size heads x 128/group_size chunk queries) and
//     each KV page staged in LDS feeds all 128 rows;
//   * wave w owns rows 32w..32w+31, one (head, query) pair per MFMA column;
//   * per table entry j the workgroup streams page page_table[b,kvh,j] (64
//     keys) of K and V from HBM into LDS (double buffered, one barrier per
//     page), then each wave computes S^T = K Q^T (keys x queries) with
//     v_mfma_f32_32x32x16_bf16, so that every lane holds one query column
//     and the softmax row statistics stay in-lane, and O^T += V^T P^T;
//   * V is stored transposed in LDS ([d][key]) with key order permuted
//     inside each 16-key group so that the P^T fragment produced by the QK
//     accumulator layout can be fed to the PV MFMA without any shuffle;
//   * causal masking is applied only to chunk blocks whose keys can be later
//     than the workgroup's first query, by absolute position 64*j + r versus
//     cached_len + t (positions from the logical block id, App. B.2);
//     entries past the workgroup's last visible block end the loop (tables
//     are ascending).
#include "common.hpp"
#include "kernels.hpp"

namespace ca {

constexpr int kRows = 128;   // (head, query) rows per workgroup
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

struct AttnArgs {
  const uint16_t* q;
  const uint16_t* k_pool;
  const uint16_t* v_pool;
  const int32_t* page_table;
  const int32_t* kv_indptr;
  const int32_t* kv_indices;
  const int32_t* cached_len;
  uint16_t* out;
  float* lse;
  float* part_o;     // [splits, B*Hq*C, D] when splits > 1
  float* part_lse;   // [splits, B*Hq*C]
  int B, Hq, Hkv, C, max_kv_blocks, group_size, G, n_qtiles, splits;
  float scale_log2;
};

// Position of key k (0..63) of a page inside the transposed V tile: bits 2
// and 3 of k are swapped, which makes the 8 keys that one lane contributes
// to a PV MFMA k-step contiguous.
__device__ __forceinline__ int vperm(int k) {
  return (k & ~12) | ((k & 4) << 1) | ((k & 8) >> 1);
}

template <int D, bool DENSE>
__global__ __launch_bounds__(256, 2) void paged_attention_kernel(const AttnArgs a) {
  constexpr int KS = D + 8;    // bf16 per K row in LDS (16-byte pad)
  constexpr int VS = 64 + 8;   // bf16 per V^T row in LDS
  constexpr int NKS = D / 16;  // k-steps of the QK contraction
  constexpr int NDT = D / 32;  // 32-row d tiles of O^T
  constexpr int KLD = (64 * D / 8) / 256;  // 16-byte K loads per thread per page
  __shared__ __attribute__((aligned(16))) uint16_t k_s[2][64 * KS];
  __shared__ __attribute__((aligned(16))) uint16_t vt_s[2][D * VS];

  const int t = threadIdx.x;
  const int wv = t >> 6;
  const int lane = t & 63;
  const int col = lane & 31;
  const int half = lane >> 5;

  // XCD-aware order: consecutive logical tiles (same table row) land on
  // the same XCD and share its L2.
  int bid = blockIdx.x;
  const int nwg = gridDim.x;
  if ((nwg & 7) == 0) bid = (bid & 7) * (nwg >> 3) + (bid >> 3);
  const int sp = bid % a.splits;
  const int qt = (bid / a.splits) % a.n_qtiles;
  const int rowid = bid / (a.splits * a.n_qtiles);
  const int b = rowid / a.G;
  const int g = rowid % a.G;
  const int gs = a.group_size;
  const int QT = kRows / gs;
  const int q0 = qt * QT;
  const int r = wv * 32 + col;
  const int head = g * gs + r / QT;
  const int tq = q0 + r % QT;
  const int kvh = (g * gs) / (a.Hq / a.Hkv);

  const int cl = a.cached_len[b];
  const int nc = cl / kPage;
  const int nkb = nc + a.C / kPage;
  const int qpos = cl + tq;
  const int j_last = (cl + q0 + QT - 1) / kPage;   // last block any row can see
  const int mask_from = cl + q0;                    // keys beyond this need masking

  int len, tbase = 0;
  if (DENSE) {
    len = nkb;
  } else {
    tbase = a.kv_indptr[rowid];
    len = a.kv_indptr[rowid + 1] - tbase;
  }
  const int e0 = (int)(((long long)len * sp) / a.splits);
  const int e1 = (int)(((long long)len * (sp + 1)) / a.splits);
  const int32_t* ptab = a.page_table + ((size_t)b * a.Hkv + kvh) * a.max_kv_blocks;

  // Q^T fragments: lane holds query column `col`, d = 16*ks + 8*half .. +7.
  bf16x8 qf[NKS];
  {
    const uint16_t* qrow = a.q + (((size_t)b * a.C + tq) * a.Hq + head) * D + 8 * half;
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks)
      qf[ks] = *reinterpret_cast<const bf16x8*>(qrow + 16 * ks);
  }

  f32x16 o[NDT];
#pragma unroll
  for (int x = 0; x < NDT; ++x)
#pragma unroll
    for (int v = 0; v < 16; ++v) o[x][v] = 0.f;
  float m_run = -INFINITY;   // running max, log2-scaled units
  float l_run = 0.f;         // partial row sum over this lane's keys

  uint4 kreg[KLD];
  uint4 vreg[4];
  const int vkb = t >> 4;          // V: 4-key block 0..15
  const int vd0 = (t & 15) * 8;    // V: first of 8 d values
  const bool v_active = vd0 < D;

  auto entry = [&](int e) -> int { return DENSE ? e : a.kv_indices[tbase + e]; };
  auto load_page = [&](int j) {
    const size_t page = (size_t)ptab[j];
    const uint16_t* kb = a.k_pool + page * (kPage * D);
    const uint16_t* vb = a.v_pool + page * (kPage * D);
#pragma unroll
    for (int x = 0; x < KLD; ++x) {
      const int c = t + 256 * x;
      kreg[x] = *reinterpret_cast<const uint4*>(kb + (size_t)c * 8);
    }
    if (v_active) {
#pragma unroll
      for (int rr = 0; rr < 4; ++rr)
        vreg[rr] = *reinterpret_cast<const uint4*>(vb + (size_t)(4 * vkb + rr) * D + vd0);
    }
  };
  auto store_page = [&](int st) {
    uint16_t* ks = k_s[st];
#pragma unroll
    for (int x = 0; x < KLD; ++x) {
      const int c = t + 256 * x;
      const int row = c / (D / 8), c8 = c % (D / 8);
      *reinterpret_cast<uint4*>(ks + row * KS + c8 * 8) = kreg[x];
    }
    if (v_active) {
      uint16_t* vt = vt_s[st];
      const int kpos = vperm(4 * vkb);
      const uint32_t* w0 = reinterpret_cast<const uint32_t*>(&vreg[0]);
      const uint32_t* w1 = reinterpret_cast<const uint32_t*>(&vreg[1]);
      const uint32_t* w2 = reinterpret_cast<const uint32_t*>(&vreg[2]);
      const uint32_t* w3 = reinterpret_cast<const uint32_t*>(&vreg[3]);
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int sh = (e & 1) * 16;
        const uint32_t x0 = (w0[e >> 1] >> sh) & 0xffffu;
        const uint32_t x1 = (w1[e >> 1] >> sh) & 0xffffu;
        const uint32_t x2 = (w2[e >> 1] >> sh) & 0xffffu;
        const uint32_t x3 = (w3[e >> 1] >> sh) & 0xffffu;
        uint2 pk;
        pk.x = x0 | (x1 << 16);
        pk.y = x2 | (x3 << 16);
        *reinterpret_cast<uint2*>(vt + (vd0 + e) * VS + kpos) = pk;
      }
    }
  };

  int e = e0;
  int j = (e < e1) ? entry(e) : 0;
  bool active = (e < e1) && (j <= j_last);
  if (active) {
    load_page(j);
    store_page(0);
  }
  __syncthreads();
  int stage = 0;
  while (active) {
    int jn = 0;
    const bool nxt = (e + 1 < e1) && ((jn = entry(e + 1)) <= j_last);
    if (nxt) load_page(jn);

    // ---- S^T = K Q^T for the 64 keys of block j (two 32-key tiles) ----
    const uint16_t* ks = k_s[stage];
    f32x16 s0, s1;
#pragma unroll
    for (int v = 0; v < 16; ++v) { s0[v] = 0.f; s1[v] = 0.f; }
#pragma unroll
    for (int x = 0; x < NKS; ++x) {
      const bf16x8 a0 = *reinterpret_cast<const bf16x8*>(ks + col * KS + 16 * x + 8 * half);
      const bf16x8 a1 = *reinterpret_cast<const bf16x8*>(ks + (32 + col) * KS + 16 * x + 8 * half);
      s0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a0, qf[x], s0, 0, 0, 0);
      s1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a1, qf[x], s1, 0, 0, 0);
    }
    // key index inside the page of accumulator slot v: 8*(v/4) + 4*half + v%4
    if (kPage * j + kPage - 1 > mask_from) {
      const int kb = kPage * j + 4 * half;
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int kp = kb + 8 * (v >> 2) + (v & 3);
        if (kp > qpos) s0[v] = -INFINITY;
        if (kp + 32 > qpos) s1[v] = -INFINITY;
      }
    }
    float mx = -INFINITY;
#pragma unroll
    for (int v = 0; v < 16; ++v) mx = fmaxf(mx, fmaxf(s0[v], s1[v]));
    mx = fmaxf(mx, __shfl_xor(mx, 32, kWave));
    const float m_new = fmaxf(m_run, mx * a.scale_log2);
    const float m_base = (m_new == -INFINITY) ? 0.f : m_new;
    const float alpha = exp2f(m_run - m_base);
    float psum = 0.f;
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      s0[v] = exp2f(fmaf(s0[v], a.scale_log2, -m_base));
      s1[v] = exp2f(fmaf(s1[v], a.scale_log2, -m_base));
      psum += s0[v] + s1[v];
    }
    l_run = fmaf(l_run, alpha, psum);
    m_run = m_new;
    if (__ballot(alpha != 1.0f)) {
#pragma unroll
      for (int x = 0; x < NDT; ++x)
#pragma unroll
        for (int v = 0; v < 16; ++v) o[x][v] *= alpha;
    }
    // ---- P^T fragments: k-step kk covers accumulator slots 8*(kk%2)..+7 ----
    bf16x8 pf[4];
#pragma unroll
    for (int x = 0; x < 8; ++x) {
      pf[0][x] = (__bf16)s0[x];
      pf[1][x] = (__bf16)s0[8 + x];
      pf[2][x] = (__bf16)s1[x];
      pf[3][x] = (__bf16)s1[8 + x];
    }
    // ---- O^T += V^T P^T ----
    const uint16_t* vt = vt_s[stage];
#pragma unroll
    for (int x = 0; x < NDT; ++x) {
#pragma unroll
      for (int kk = 0; kk < 4; ++kk) {
        const bf16x8 av =
            *reinterpret_cast<const bf16x8*>(vt + (32 * x + col) * VS + 16 * kk + 8 * half);
        o[x] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av, pf[kk], o[x], 0, 0, 0);
      }
    }
    if (nxt) store_page(stage ^ 1);
    __syncthreads();
    stage ^= 1;
    ++e;
    j = jn;
    active = nxt;
  }

  // ---- epilogue ----
  const float l_tot = l_run + __shfl_xor(l_run, 32, kWave);
  const float inv = l_tot > 0.f ? 1.0f / l_tot : 0.f;
  const float lse_val = l_tot > 0.f ? (m_run + log2f(l_tot)) * kLn2 : -INFINITY;
  const size_t qrow_idx = ((size_t)b * a.Hq + head) * a.C + tq;   // [B, Hq, C] order
  if (a.splits == 1) {
    uint16_t* orow = a.out + (((size_t)b * a.C + tq) * a.Hq + head) * D;
#pragma unroll
    for (int x = 0; x < NDT; ++x) {
#pragma unroll
      for (int q4 = 0; q4 < 4; ++q4) {
        const int d = 32 * x + 8 * q4 + 4 * half;
        uint2 pk;
        pk.x = pack_bf16x2(o[x][4 * q4 + 0] * inv, o[x][4 * q4 + 1] * inv);
        pk.y = pack_bf16x2(o[x][4 * q4 + 2] * inv, o[x][4 * q4 + 3] * inv);
        *reinterpret_cast<uint2*>(orow + d) = pk;
      }
    }
    if (a.lse != nullptr && half == 0) a.lse[qrow_idx] = lse_val;
  } else {
    const size_t prow = (size_t)sp * a.B * a.Hq * a.C + qrow_idx;
    float* po = a.part_o + prow * D;
#pragma unroll
    for (int x = 0; x < NDT; ++x) {
#pragma unroll
      for (int q4 = 0; q4 < 4; ++q4) {
        const int d = 32 * x + 8 * q4 + 4 * half;
        *reinterpret_cast<float4*>(po + d) =
            make_float4(o[x][4 * q4 + 0] * inv, o[x][4 * q4 + 1] * inv,
                        o[x][4 * q4 + 2] * inv, o[x][4 * q4 + 3] * inv);
      }
    }
    if (half == 0) a.part_lse[prow] = lse_val;
  }
}

// Split-KV merge: lse = log sum_i exp(lse_i), out = sum_i exp(lse_i - lse) o_i.
// One 32-lane half-wave per (b, h, t) row, 4 floats of d per lane (D = 128)
// or 2 (D = 64).
template <int D>
__global__ __launch_bounds__(256) void combine_kernel(const float* __restrict__ part_o,
                                                      const float* __restrict__ part_lse,
                                                      uint16_t* __restrict__ out,
                                                      float* __restrict__ lse, int B, int Hq,
                                                      int C, int splits) {
  constexpr int PER = D / 32;
  const size_t nrows = (size_t)B * Hq * C;
  const size_t row = (size_t)blockIdx.x * 8 + (threadIdx.x >> 5);
  if (row >= nrows) return;
  const int sub = threadIdx.x & 31;
  float mx = -INFINITY;
  for (int i = 0; i < splits; ++i) mx = fmaxf(mx, part_lse[(size_t)i * nrows + row]);
  float acc[PER];
#pragma unroll
  for (int x = 0; x < PER; ++x) acc[x] = 0.f;
  float wsum = 0.f;
  if (mx != -INFINITY) {
    for (int i = 0; i < splits; ++i) {
      const float li = part_lse[(size_t)i * nrows + row];
      if (li == -INFINITY) continue;
      const float wgt = expf(li - mx);
      wsum += wgt;
      const float* po = part_o + ((size_t)i * nrows + row) * D + sub * PER;
#pragma unroll
      for (int x = 0; x < PER; ++x) acc[x] = fmaf(wgt, po[x], acc[x]);
    }
  }
  const float inv = wsum > 0.f ? 1.0f / wsum : 0.f;
  // row is in [B, Hq, C] order; out is [B, C, Hq, D]
  const int tq = (int)(row % C);
  const int h = (int)((row / C) % Hq);
  const int b = (int)(row / ((size_t)C * Hq));
  uint16_t* orow = out + (((size_t)b * C + tq) * Hq + h) * D + sub * PER;
#pragma unroll
  for (int x = 0; x < PER; ++x) orow[x] = float_to_bf16_bits(acc[x] * inv);
  if (lse != nullptr && sub == 0) lse[row] = wsum > 0.f ? mx + logf(wsum) : -INFINITY;
}

int attn_query_tile(int group_size) { return kRows / group_size; }

int attn_base_workgroups(const Dims& d, int group_size) {
  return d.B * (d.Hq / group_size) * (d.C / attn_query_tile(group_size));
}

size_t attn_ws_bytes(const Dims& d, int splits) {
  if (splits <= 1) return 0;
  const size_t rows = (size_t)d.B * d.Hq * d.C;
  return (size_t)splits * rows * (d.D + 1) * sizeof(float);
}

hipError_t launch_attention(const Dims& d, const AttnLaunch& L, hipStream_t st) {
  AttnArgs a;
  a.q = L.q;
  a.k_pool = L.k_pool;
  a.v_pool = L.v_pool;
  a.page_table = L.page_table;
  a.kv_indptr = L.kv_indptr;
  a.kv_indices = L.kv_indices;
  a.cached_len = L.cached_len;
  a.out = L.out;
  a.lse = L.lse;
  const size_t rows = (size_t)d.B * d.Hq * d.C;
  a.part_o = L.splits > 1 ? static_cast<float*>(L.ws) : nullptr;
  a.part_lse = L.splits > 1 ? static_cast<float*>(L.ws) + (size_t)L.splits * rows * d.D : nullptr;
  a.B = d.B;
  a.Hq = d.Hq;
  a.Hkv = d.Hkv;
  a.C = d.C;
  a.max_kv_blocks = d.max_kv_blocks;
  a.group_size = L.group_size;
  a.G = d.Hq / L.group_size;
  a.n_qtiles = d.C / attn_query_tile(L.group_size);
  a.splits = L.splits;
  a.scale_log2 = L.sm_scale * kLog2e;
  const int nwg = attn_base_workgroups(d, L.group_size) * L.splits;
  if (d.D == 128) {
    if (L.dense) paged_attention_kernel<128, true><<<nwg, 256, 0, st>>>(a);
    else paged_attention_kernel<128, false><<<nwg, 256, 0, st>>>(a);
  } else {
    if (L.dense) paged_attention_kernel<64, true><<<nwg, 256, 0, st>>>(a);
    else paged_attention_kernel<64, false><<<nwg, 256, 0, st>>>(a);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || L.splits == 1) return e;
  const int cgrid = (int)((rows + 7) / 8);
  if (d.D == 128)
    combine_kernel<128><<<cgrid, 256, 0, st>>>(a.part_o, a.part_lse, L.out, L.lse, d.B, d.Hq,
                                               d.C, L.splits);
  else
    combine_kernel<64><<<cgrid, 256, 0, st>>>(a.part_o, a.part_lse, L.out, L.lse, d.B, d.Hq,
                                              d.C, L.splits);
  return hipGetLastError();
}

}  // namespace ca
