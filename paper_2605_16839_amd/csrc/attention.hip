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
//   * the pages of the table are copied from HBM straight into LDS with
//     16-byte direct-to-LDS loads (no register round trip); each lane picks
//     its source chunk so that the LDS image is XOR-swizzled and the MFMA
//     operand reads are bank-conflict free;
//   * each wave computes S^T = K Q^T (keys x queries) with
//     v_mfma_f32_32x32x16_bf16, so every lane holds one query column and the
//     softmax statistics stay in-lane, then O^T += V^T P^T, the V^T
//     fragments coming straight from the row-major V page through the gfx950
//     transpose read ds_read_b64_tr_b16;
//   * the copy of page i+1 is in flight while page i is processed (double
//     buffered tiles, one barrier per page); the MFMA and softmax phases of
//     the two workgroups resident on a CU overlap on each SIMD;
//   * causal masking is applied only to the trailing entries whose keys can
//     be later than the workgroup's first query, by absolute position
//     64*j + r versus cached_len + t (positions from the logical block id,
//     App. B.2); entries past the workgroup's last visible block are dropped
//     (tables are ascending).
#include <type_traits>

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
  int table_mode;          // kTablesPerGroup / kTablesPerQTile / kTablesPacked
  long long packed_pages;  // capacity of the packed pools (kTablesPacked)
  float scale_log2;
};

// Swizzled position (16-byte chunk) of chunk c of row r in an LDS page tile.
// gfx950 LDS has 64 banks of 4 bytes; a 16-byte read is served 16 lanes per
// cycle and an 8-byte read 32 lanes per cycle.
// K is read 16 bytes per lane by 16 consecutive rows at one chunk: the 16
// rows must land on 16 different 16-byte bank slots of the 256-byte bank
// window (a D = 64 row is half a window, so rows pair up).
// V is read 8 bytes per lane by the transpose read, 32 lanes covering 4
// consecutive rows x 4 chunks: each row's aligned group of 4 chunks must
// move to a different aligned group of the window.
template <int D>
__device__ __forceinline__ int k_swz(int r, int c) {
  return D == 128 ? (c ^ (r & 15)) : (c ^ ((r >> 1) & 7));
}
template <int D>
__device__ __forceinline__ int v_swz(int r, int c) {
  return D == 128 ? (c ^ ((r & 3) << 2)) : (c ^ (((r >> 1) & 1) << 2));
}

// 2^x with a single v_exp_f32 (results below the normal range flush to 0,
// which only affects softmax weights < 2^-126).
__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// o[x] *= alpha for every tile when `any` is non-zero.  The branch lives
// inside the asm so that the accumulators keep their registers on both paths
// (a compiler-level branch makes the register allocator copy all of them
// every step).  Only taken when the exponent base moves (lazy rescaling);
// the leading nops cover the MFMA-to-VALU and the trailing ones the
// VALU-to-MFMA dependency distances of the accumulators.
template <int NDT>
__device__ __forceinline__ void rescale_tiles(f32x16 (&o)[NDT], float alpha, uint64_t any) {
#pragma unroll
  for (int x = 0; x < NDT; ++x) {
    __asm__ volatile(
        "s_cmp_eq_u64 %16, 0\n"
        "s_cbranch_scc1 1f\n"
        "s_nop 7\n s_nop 7\n s_nop 7\n"
        "v_mul_f32 %0, %17, %0\n v_mul_f32 %1, %17, %1\n"
        "v_mul_f32 %2, %17, %2\n v_mul_f32 %3, %17, %3\n"
        "v_mul_f32 %4, %17, %4\n v_mul_f32 %5, %17, %5\n"
        "v_mul_f32 %6, %17, %6\n v_mul_f32 %7, %17, %7\n"
        "v_mul_f32 %8, %17, %8\n v_mul_f32 %9, %17, %9\n"
        "v_mul_f32 %10, %17, %10\n v_mul_f32 %11, %17, %11\n"
        "v_mul_f32 %12, %17, %12\n v_mul_f32 %13, %17, %13\n"
        "v_mul_f32 %14, %17, %14\n v_mul_f32 %15, %17, %15\n"
        "s_nop 7\n"
        "1:"
        : "+v"(o[x][0]), "+v"(o[x][1]), "+v"(o[x][2]), "+v"(o[x][3]), "+v"(o[x][4]),
          "+v"(o[x][5]), "+v"(o[x][6]), "+v"(o[x][7]), "+v"(o[x][8]), "+v"(o[x][9]),
          "+v"(o[x][10]), "+v"(o[x][11]), "+v"(o[x][12]), "+v"(o[x][13]), "+v"(o[x][14]),
          "+v"(o[x][15])
        : "s"(any), "v"(alpha)
        : "scc");
  }
}

template <bool DENSE>
__device__ __forceinline__ int table_entry(const int32_t* __restrict__ idx, int base, int e) {
  return DENSE ? e : idx[base + e];
}

typedef __attribute__((address_space(3))) void lds_void;
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) i16x4 lds_i16x4;

// Copy one page (64 rows x D bf16, contiguous in HBM) into an LDS tile with
// direct-to-LDS loads.  Each wave instruction fills 1 KB of the tile, lane l
// writing bytes [16l, 16l+16); the lane's source is the chunk that the
// swizzle maps there (the swizzles are involutions).
template <int D, bool IS_V>
__device__ __forceinline__ void page_to_lds(const uint16_t* __restrict__ src, uint16_t* tile,
                                            int wv, int lane) {
  constexpr int CPR = D / 8;                             // 16-byte chunks per row
  constexpr int ROWS_PER_INST = 64 / CPR;                // rows per 1 KB instruction
  constexpr int INST_PER_WAVE = (64 * D * 2) / 1024 / 4; // 4 waves share a page
#pragma unroll
  for (int m = 0; m < INST_PER_WAVE; ++m) {
    const int inst = wv * INST_PER_WAVE + m;
    const int r = inst * ROWS_PER_INST + lane / CPR;
    const int cpos = lane % CPR;
    const int c = IS_V ? v_swz<D>(r, cpos) : k_swz<D>(r, cpos);
    const uint32_t off = (uint32_t)(r * D + c * 8);   // unsigned: scalar base + 32-bit offset
    __builtin_amdgcn_global_load_lds(src + off, (lds_void*)(tile + inst * 512), 16, 0, 0);
  }
}

// Wait for this wave's direct-to-LDS copies and tell the compiler that the
// tiles behind p0/p1 changed (the copies write them outside its view).
__device__ __forceinline__ void copies_landed(void* p0, void* p1) {
  __builtin_amdgcn_s_waitcnt(0);
  __asm__ volatile("" : : "v"(p0), "v"(p1) : "memory");
}

// NaN-propagating maximum (v_maximum3_f32 on gfx950).  fmaxf would quiet
// each MFMA result with an extra v_max first (IEEE mode); the scores are
// never NaN, so the two agree.
__device__ __forceinline__ float max3(float a, float b, float c) {
  return __builtin_elementwise_maximum(__builtin_elementwise_maximum(a, b), c);
}

// Lazy rescaling threshold (log2 units): the running max used as the
// exponent base is only moved when a new score exceeds it by more than this,
// so the weights stay <= 2^kRescaleSlack and most pages skip the O rescale.
constexpr float kRescaleSlack = 8.0f;

// max / sum of a value and its partner in the other half of the wave
// (lanes l and l^32 hold the same query column).
__device__ __forceinline__ float halves_max(float x) {
  const uint32_t u = __float_as_uint(x);
  const auto r = __builtin_amdgcn_permlane32_swap(u, u, false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float halves_sum(float x) {
  const uint32_t u = __float_as_uint(x);
  const auto r = __builtin_amdgcn_permlane32_swap(u, u, false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// S^T tile of one page: keys 0..31 in .lo, 32..63 in .hi.
struct STile {
  f32x16 lo, hi;
};

// S^T = K Q^T over one page: A = K rows (32 keys x 16 d per k-step), B = Q^T.
template <int D>
__device__ __forceinline__ void qk_page(STile& st, const uint16_t* __restrict__ ks,
                                        const bf16x8 (&qf)[D / 16], int col, int half) {
#pragma unroll
  for (int v = 0; v < 16; ++v) { st.lo[v] = 0.f; st.hi[v] = 0.f; }
#pragma unroll
  for (int x = 0; x < D / 16; ++x) {
    const int c = 2 * x + half;
    const bf16x8 a0 = *reinterpret_cast<const bf16x8*>(ks + col * D + 8 * k_swz<D>(col, c));
    const bf16x8 a1 =
        *reinterpret_cast<const bf16x8*>(ks + (32 + col) * D + 8 * k_swz<D>(32 + col, c));
    st.lo = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a0, qf[x], st.lo, 0, 0, 0);
    st.hi = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a1, qf[x], st.hi, 0, 0, 0);
  }
}

// V^T fragment for PV k-step kk and d tile x.  Lane (d row `col`, half) needs
// the 8 keys 16kk + 4half + {0..3} and 16kk + 8 + 4half + {0..3}, the key
// order of the P^T fragment taken from the S^T accumulator layout.  In a
// 16-lane group, source lane 4m + q points at key row base + m, d columns
// 4q..4q+3 of the group's 16 d; the transpose read then hands lane i the
// four keys of d = group base + i.
template <int D>
__device__ __forceinline__ bf16x8 vt_frag(const uint16_t* __restrict__ vs, int lane, int x,
                                          int kk) {
  const int grp = lane >> 4, sl = lane & 15;
  const int m = sl >> 2, q = sl & 3;
  const int d = 32 * x + 16 * (grp & 1) + 4 * q;
  const int c = d >> 3, sub = d & 7;
  const int r0 = 16 * kk + 4 * (grp >> 1) + m;
  const int r1 = r0 + 8;
  const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (lds_i16x4*)(vs + r0 * D + 8 * v_swz<D>(r0, c) + sub));
  const i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (lds_i16x4*)(vs + r1 * D + 8 * v_swz<D>(r1, c) + sub));
  // whole-vector casts only: element-wise bf16 <-> i16 moves are not reliable
  const u32x2 l2 = __builtin_bit_cast(u32x2, lo), h2 = __builtin_bit_cast(u32x2, hi);
  const u32x4 w = {l2[0], l2[1], h2[0], h2[1]};
  return __builtin_bit_cast(bf16x8, w);
}

template <int D, bool DENSE>
__global__ __launch_bounds__(256, 2) void paged_attention_kernel(const AttnArgs a) {
  constexpr int NKS = D / 16;   // k-steps of the QK contraction
  constexpr int NDT = D / 32;   // 32-row d tiles of O^T
  constexpr int PAGE = 64 * D;  // bf16 per page tile
  constexpr int COPIES = 2 * (64 * D * 2) / 1024 / 4;   // copy instructions per wave per step
  // Separate buffers (not one array) so that the compiler can tell the copy
  // target of a step from the tiles that step reads.
  __shared__ __attribute__((aligned(1024))) uint16_t k_s0[PAGE];
  __shared__ __attribute__((aligned(1024))) uint16_t k_s1[PAGE];
  __shared__ __attribute__((aligned(1024))) uint16_t v_s0[PAGE];
  __shared__ __attribute__((aligned(1024))) uint16_t v_s1[PAGE];

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
    // per-group rows, or one row per (head, query tile) for the block-sparse arm
    const int trow = a.table_mode == kTablesPerQTile ? rowid * a.n_qtiles + qt : rowid;
    tbase = a.kv_indptr[trow];
    len = a.kv_indptr[trow + 1] - tbase;
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

  // Table entries e0 .. e_end-1 (entries past the last visible block are
  // dropped; tables are ascending).  Those whose keys can be later than the
  // first query of the tile need the causal mask and form a suffix.
  int e_end = e1;
  if (DENSE) {
    e_end = e1 < j_last + 1 ? e1 : j_last + 1;
  } else {
    while (e_end > e0 && table_entry<DENSE>(a.kv_indices, tbase, e_end - 1) > j_last) --e_end;
  }
  const int n = e_end - e0;
  int n_main = n;
  while (n_main > 0 &&
         kPage * table_entry<DENSE>(a.kv_indices, tbase, e0 + n_main - 1) + kPage - 1 > mask_from)
    --n_main;
  // Block and page ids of the entries, 64 at a time: lane l of blk_cur /
  // pg_cur holds entry e0 + base + l (clamped to the last entry), the *_nxt
  // pair the following 64; a step picks its ids with a scalar readlane.
  int base = 0, blk_cur = 0, pg_cur = 0, blk_nxt = 0, pg_nxt = 0;
  auto fetch = [&](int b0, int& blk, int& pg) {
    int idx = b0 + lane;
    idx = idx < n ? idx : n - 1;
    idx = idx < 0 ? 0 : idx;
    blk = (n > 0) ? table_entry<DENSE>(a.kv_indices, tbase, e0 + idx) : 0;
    if (!DENSE && a.table_mode == kTablesPacked) {
      // packed pools hold the selected pages in table order (copy arm)
      const long long pp = (long long)tbase + e0 + idx;
      pg = (n > 0) ? (int)(pp < a.packed_pages ? pp : a.packed_pages - 1) : 0;
    } else {
      pg = (n > 0) ? ptab[blk] : 0;
    }
  };
  fetch(0, blk_cur, pg_cur);
  fetch(64, blk_nxt, pg_nxt);
  auto advance = [&](int i) {   // make i - base < 64
    while (i - base >= 64) {
      base += 64;
      blk_cur = blk_nxt;
      pg_cur = pg_nxt;
      fetch(base + 64, blk_nxt, pg_nxt);
    }
  };
  auto id_of = [&](int cur, int nxt, int i) -> int {   // i - base in [0, 128)
    const int d = i - base;
    return d < 64 ? __builtin_amdgcn_readlane(cur, d) : __builtin_amdgcn_readlane(nxt, d - 64);
  };
  auto page_ptr = [&](const uint16_t* pool, int i) -> const uint16_t* {
    return pool + (size_t)id_of(pg_cur, pg_nxt, i) * (kPage * D);
  };

  // Prologue: K and V of page 0 in LDS.
  if (n > 0) {
    page_to_lds<D, false>(page_ptr(a.k_pool, 0), k_s0, wv, lane);
    page_to_lds<D, true>(page_ptr(a.v_pool, 0), v_s0, wv, lane);
  }
  copies_landed(k_s0, v_s0);
  __syncthreads();

  // Step i (page e0 + i, buffer parity S = i & 1 as a compile-time constant so
  // that the copy targets and the tiles read are distinct objects): the copy
  // of page i+1 into buffers S^1 goes out first and lands while page i is
  // processed from buffers S: S^T = K Q^T, online softmax, O^T += V^T P^T.
  auto step = [&](auto masked, auto stage, int i) __attribute__((always_inline)) {
    constexpr int S = decltype(stage)::value;
    uint16_t* const k_here = S ? k_s1 : k_s0;
    uint16_t* const k_next = S ? k_s0 : k_s1;
    uint16_t* const v_here = S ? v_s1 : v_s0;
    uint16_t* const v_next = S ? v_s0 : v_s1;
    const int i1 = i + 1 < n ? i + 1 : n - 1;   // clamped: the copy stays valid, unused
    page_to_lds<D, false>(page_ptr(a.k_pool, i1), k_next, wv, lane);
    page_to_lds<D, true>(page_ptr(a.v_pool, i1), v_next, wv, lane);
    STile st;
    qk_page<D>(st, k_here, qf, col, half);

    // ---- online softmax of page e0 + i ----
    if constexpr (decltype(masked)::value) {
      const int j = id_of(blk_cur, blk_nxt, i);
      // key of accumulator slot v: 64*j + 8*(v/4) + 4*half + v%4 (+32 in .hi)
      const int lim = qpos - kPage * j - 4 * half;
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int kp = 8 * (v >> 2) + (v & 3);
        if (kp > lim) st.lo[v] = -INFINITY;
        if (kp + 32 > lim) st.hi[v] = -INFINITY;
      }
    }
    float mx = max3(st.lo[0], st.hi[0], st.lo[1]);
    mx = max3(mx, st.hi[1], st.lo[2]);
#pragma unroll
    for (int v = 2; v < 15; ++v) mx = max3(mx, st.hi[v], st.lo[v + 1]);
    mx = max3(mx, st.hi[15], st.hi[15]);
    mx = halves_max(mx) * a.scale_log2;
    // move the base only when the page's max exceeds it by the slack
    // (-inf > -inf + slack is false: a fully masked row keeps its base)
    const bool rebase = mx > m_run + kRescaleSlack;
    const float alpha = rebase ? fast_exp2(m_run - mx) : 1.0f;
    m_run = rebase ? mx : m_run;
    l_run *= alpha;
    rescale_tiles<NDT>(o, alpha, __ballot(rebase));
    const float m_base = (m_run == -INFINITY) ? 0.f : m_run;
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      st.lo[v] = fast_exp2(fmaf(st.lo[v], a.scale_log2, -m_base));
      st.hi[v] = fast_exp2(fmaf(st.hi[v], a.scale_log2, -m_base));
    }
    float ps0 = st.lo[0], ps1 = st.hi[0];
#pragma unroll
    for (int v = 1; v < 16; ++v) { ps0 += st.lo[v]; ps1 += st.hi[v]; }
    l_run += ps0 + ps1;
    // P^T fragments: k-step kk covers accumulator slots 8*(kk%2)..+7
    bf16x8 pf[4];
#pragma unroll
    for (int x = 0; x < 8; ++x) {
      pf[0][x] = (__bf16)st.lo[x];
      pf[1][x] = (__bf16)st.lo[8 + x];
      pf[2][x] = (__bf16)st.hi[x];
      pf[3][x] = (__bf16)st.hi[8 + x];
    }

    // ---- O^T += V^T P^T ----
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) {
#pragma unroll
      for (int x = 0; x < NDT; ++x)
        o[x] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vt_frag<D>(v_here, lane, x, kk),
                                                       pf[kk], o[x], 0, 0, 0);
    }
    copies_landed(k_next, v_next);
    __syncthreads();
  };
  using Plain = std::integral_constant<bool, false>;
  using Masked = std::integral_constant<bool, true>;
  using S0 = std::integral_constant<int, 0>;
  using S1 = std::integral_constant<int, 1>;
  int i = 0;
  for (; i + 1 < n_main; i += 2) {
    advance(i);
    step(Plain{}, S0{}, i);
    step(Plain{}, S1{}, i + 1);
  }
  if (i < n_main) {             // i is even here
    advance(i);
    step(Plain{}, S0{}, i);
    ++i;
  }
  for (; i < n; ++i) {
    advance(i);
    if (i & 1) step(Masked{}, S1{}, i);
    else step(Masked{}, S0{}, i);
  }

  // ---- epilogue ----
  const float l_tot = halves_sum(l_run);
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


// Copy arm (Sec. 4.4): pack the selected K and V pages of every table row into
// contiguous pools in table order (packed page p = table entry p of the CSR),
// so that attention can run on contiguous KV.  One workgroup per packed page;
// the row of entry p is found by binary search in kv_indptr.
template <int D>
__global__ __launch_bounds__(256) void gather_kernel(
    const uint16_t* __restrict__ k_pool, const uint16_t* __restrict__ v_pool,
    const int32_t* __restrict__ page_table, const int32_t* __restrict__ kv_indptr,
    const int32_t* __restrict__ kv_indices, int R, int G, int group_size, int Hq, int Hkv,
    int max_kv_blocks, uint16_t* __restrict__ k_packed, uint16_t* __restrict__ v_packed) {
  const int p = blockIdx.x;
  if (p >= kv_indptr[R]) return;
  int lo = 0, hi = R;   // kv_indptr[lo] <= p < kv_indptr[hi]
  while (hi - lo > 1) {
    const int mid = (lo + hi) >> 1;
    if (kv_indptr[mid] <= p) lo = mid;
    else hi = mid;
  }
  const int b = lo / G, g = lo % G;
  const int kvh = (g * group_size) / (Hq / Hkv);
  const int j = kv_indices[p];
  if (j < 0 || j >= max_kv_blocks) return;
  const int pg = page_table[((size_t)b * Hkv + kvh) * max_kv_blocks + j];
  constexpr int N16 = kPage * D * 2 / 16;   // 16-byte pieces per page
  const uint4* ks = reinterpret_cast<const uint4*>(k_pool + (size_t)pg * kPage * D);
  const uint4* vs = reinterpret_cast<const uint4*>(v_pool + (size_t)pg * kPage * D);
  uint4* kd = reinterpret_cast<uint4*>(k_packed + (size_t)p * kPage * D);
  uint4* vd = reinterpret_cast<uint4*>(v_packed + (size_t)p * kPage * D);
#pragma unroll
  for (int i = threadIdx.x; i < N16; i += 256) {
    const uint4 kv = ks[i], vv = vs[i];
    kd[i] = kv;
    vd[i] = vv;
  }
}

hipError_t launch_gather(const Dims& d, const uint16_t* k_pool, const uint16_t* v_pool,
                         const int32_t* page_table, const int32_t* kv_indptr,
                         const int32_t* kv_indices, int group_size, long long capacity_pages,
                         uint16_t* k_packed, uint16_t* v_packed, hipStream_t st) {
  const int G = d.Hq / group_size;
  const int R = d.B * G;
  if (capacity_pages <= 0) return hipSuccess;
  const int grid = (int)capacity_pages;
  if (d.D == 128)
    gather_kernel<128><<<grid, 256, 0, st>>>(k_pool, v_pool, page_table, kv_indptr, kv_indices,
                                             R, G, group_size, d.Hq, d.Hkv, d.max_kv_blocks,
                                             k_packed, v_packed);
  else
    gather_kernel<64><<<grid, 256, 0, st>>>(k_pool, v_pool, page_table, kv_indptr, kv_indices,
                                            R, G, group_size, d.Hq, d.Hkv, d.max_kv_blocks,
                                            k_packed, v_packed);
  return hipGetLastError();
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
  a.table_mode = L.table_mode;
  a.packed_pages = L.packed_pages;
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
