// Zero-copy paged chunk attention over per-group block tables (Sec. 3.3,
// App. B.2), bf16 MFMA with fp32 online softmax, and the split-KV
// log-sum-exp combine.
//
// Work decomposition: one workgroup = NW wavefronts; a wave owns 32*CT
// (head, query) rows, CT 32-column MFMA tiles:
//   * a table row r = b*G + g serves the group_size query heads of group g;
//     all of them read the same KV pages, so a workgroup packs rows of every
//     head of the group (group_size heads x 32*CT*NW/group_size chunk
//     queries) and each KV page staged in LDS feeds all of them;
//   * the kernels run CT = 2: one wave per SIMD holding up to 512 registers
//     (the O^T accumulators and Q^T fragments in AGPRs), and every K and V
//     fragment a wave reads from LDS feeds two v_mfma_f32_32x32x16_bf16 (one
//     per column tile), half the LDS traffic per flop of a 32-column wave.
//     CT = 1 (two waves per SIMD, 32 columns and at most 256 registers each,
//     all VGPRs) also compiles: it keeps the matrix cores busier per cycle,
//     but doubles the LDS reads and per-page scalar work per flop, and on
//     MI355X it ran at a lower clock, for no gain in time;
//   * S^T = K Q^T (keys x queries): every lane holds one query column, so
//     the softmax statistics are in-lane plus one v_permlane32_swap; then
//     O^T += V^T P^T.  Lanes read the K rows in an order (key_of_row) that
//     gives every lane 8 consecutive keys of its P^T fragment, so the
//     matching V^T fragment is one 16-byte read of a transposed V page
//     ([D, 64], VL = kVTransposed) or two gfx950 transpose reads
//     (ds_read_b64_tr_b16) of a token-major page ([64, D], the paper's
//     layout, VL = kVTokenMajor);
//   * pages go from HBM into LDS with 16-byte direct-to-LDS buffer loads (no
//     register round trip) into XOR-swizzled tiles (conflict-free operand
//     reads);
//   * software pipeline: step i issues the copies of K(i+2) and V(i), the PV
//     MFMAs of page i-1 and the QK MFMAs of page i+1, and between them (one
//     MFMA per slot) the softmax of page i; one barrier per page;
//   * the causally masked diagonal pages (and an odd leftover page) run after
//     the pipeline, one at a time: their keys are compared by absolute
//     position 64*j + r against cached_len + t (positions from the logical
//     block id, App. B.2); entries past the tile's last visible block are
//     dropped (tables are ascending);
//   * the workgroups of one table row run on one of the 8 XCDs and share its
//     L2, so each page comes from HBM once; by default every row is cut in
//     two so that the XCDs carry equal loads (xcd_split_kernel), the two
//     pieces merged by combine_kernel.
#include <type_traits>
#include <utility>

#include "common.hpp"
#include "kernels.hpp"

namespace ca {

// Per-group tables: 4 waves of 64 columns (one wave per SIMD).  Block-sparse
// tiles (one head x 128 queries): 2 waves of 64 columns, two workgroups per CU.
constexpr int kWavesGroup = 4;
constexpr int kWavesQTile = 2;
constexpr int kColTiles = 2;     // 32-column MFMA tiles per wave
constexpr int kWavesPerCu = 4;   // resident waves per CU (1 per SIMD)
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
  // XCD-balanced two-piece split (splits == 2): table row r is cut at entry
  // split_at[r]; -1 = not cut, run whole as piece 0; -2 = not cut, run whole
  // as piece 1; nullptr = every row cut in the middle
  const int32_t* split_at;
  int rows_per_unit;   // table rows that read one KV head's pages together
};

constexpr int kXcds = 8;   // MI355X: 8 accelerator complex dies, 32 CUs and one L2 each

// LDS page tiles: K pages and token-major V pages are 64 key rows x D; a
// transposed V page is D rows x 64 keys.
constexpr int kTileK = 0;
constexpr int kTileVT = 1;   // transposed V page
constexpr int kTileVR = 2;   // token-major V page

// Swizzled position (16-byte chunk) of chunk c of row r in an LDS page tile.
// gfx950 LDS has 64 banks of 4 bytes; a 16-byte read is served 16 lanes per
// cycle and an 8-byte read 32 lanes per cycle.
// K tiles are read 16 bytes per lane by 16 rows at one chunk: the 16 rows
// must land on 16 different 16-byte bank slots of the 256-byte bank window
// (a D = 64 row is half a window, so rows pair up).
// Transposed V tiles (128-byte rows, two per window) are read the same way.
// Token-major V tiles are read 8 bytes per lane by the transpose read, 32
// lanes covering 4 consecutive rows x 64 bytes: each row's aligned group of
// 4 chunks must move to a different aligned group of the window.
// Every swizzle leaves a row's pattern unchanged under +32 rows (K also under
// +8 and +16, token-major V under +4 and +16), so the operand reads of one
// lane differ only by immediate offsets.
template <int D>
__device__ __forceinline__ int k_swz(int r, int c) {
  return D == 128 ? (c ^ (r & 15)) : (c ^ ((r >> 1) & 7));
}
__device__ __forceinline__ int vt_swz(int r, int c) { return c ^ ((r >> 1) & 7); }
template <int D>
__device__ __forceinline__ int vr_swz(int r, int c) {
  return D == 128 ? (c ^ ((r & 3) << 2)) : (c ^ (((r >> 1) & 1) << 2));
}
template <int D, int TILE>
__device__ __forceinline__ int tile_swz(int r, int c) {
  if constexpr (TILE == kTileVT) return vt_swz(r, c);
  else if constexpr (TILE == kTileVR) return vr_swz<D>(r, c);
  else return k_swz<D>(r, c);
}

// Key row that lane column `col` reads from a K tile: bits 2 and 3 of the
// key index swapped.  With it the S^T accumulator rows that one lane packs
// into a P^T fragment are 8 consecutive keys, so the matching V^T fragment
// is one contiguous run of keys.
__device__ __forceinline__ int key_of_row(int r) {
  return (r & ~12) | ((r & 4) << 1) | ((r & 8) >> 1);
}

// 2^x with a single v_exp_f32 (results below the normal range flush to 0,
// which only affects softmax weights < 2^-126).
__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

typedef __attribute__((address_space(3))) void lds_void;
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) i16x4 lds_i16x4;

// Raw buffer resource of one page (64 rows x D bf16).  The page copies use
// buffer loads to LDS rather than global_load_lds: while a global_load_lds is
// in flight the compiler cannot count LDS reads (it treats the copy as a flat
// access that may touch LDS) and makes every operand read wait for all
// outstanding LDS reads, which defeats the fragment prefetch.  Offsets past
// the page would read 0 instead of faulting.
constexpr int kRawBufferWord3 = 0x00020000;   // gfx9 raw buffer, 32-bit data format
#define CA_PAGE_RSRC(page, D)                                                              \
  __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(page), 0, kPage * (D) * 2,      \
                                    kRawBufferWord3)

// Copy one page (16 KB at D = 128, contiguous in HBM) into an LDS tile with
// direct-to-LDS loads.  Each wave instruction fills 1 KB of the tile, lane l
// writing bytes [16l, 16l+16); the lane's source is the chunk that the
// swizzle maps there (the swizzles are involutions).  NW waves share a page.
template <int D, int TILE>
__device__ __forceinline__ uint32_t copy_src_offset(int inst, int lane) {
  constexpr int RL = TILE == kTileVT ? kPage : D;   // elements per row
  constexpr int CPR = RL / 8;                       // 16-byte chunks per row
  constexpr int ROWS_PER_INST = 64 / CPR;
  const int r = inst * ROWS_PER_INST + lane / CPR;
  const int cpos = lane % CPR;
  const int c = tile_swz<D, TILE>(r, cpos);
  return (uint32_t)(r * RL + c * 8);   // unsigned: scalar base + 32-bit offset
}
template <int D, int NW, int TILE>
__device__ __forceinline__ void page_to_lds(const uint16_t* __restrict__ src, uint16_t* tile,
                                            int wv, int lane) {
  constexpr int INST_PER_WAVE = (64 * D * 2) / 1024 / NW;
#pragma unroll
  for (int m = 0; m < INST_PER_WAVE; ++m) {
    const int inst = wv * INST_PER_WAVE + m;
    const uint32_t off = copy_src_offset<D, TILE>(inst, lane);
    __builtin_amdgcn_raw_ptr_buffer_load_lds(CA_PAGE_RSRC(src, D), (lds_void*)(tile + inst * 512),
                                             16, 2 * off, 0, 0, 0);
  }
}

// One of the 1 KB copy instructions of page_to_lds (instruction m of this
// wave), so that a step can spread its copies between MFMAs.
template <int D, int NW, int TILE>
__device__ __forceinline__ void page_part_to_lds(const uint16_t* __restrict__ src, uint16_t* tile,
                                                 int wv, int lane, int m) {
  constexpr int INST_PER_WAVE = (64 * D * 2) / 1024 / NW;
  const int inst = wv * INST_PER_WAVE + m;
  const uint32_t off = copy_src_offset<D, TILE>(inst, lane);
  __builtin_amdgcn_raw_ptr_buffer_load_lds(CA_PAGE_RSRC(src, D), (lds_void*)(tile + inst * 512),
                                           16, 2 * off, 0, 0, 0);
}

// Wait for this wave's direct-to-LDS copies and tell the compiler that the
// tiles behind the pointers changed (the copies write them outside its view).
__device__ __forceinline__ void tile_written(const void* tile) {
  __asm__ volatile("" : : "v"(tile) : "memory");
}
template <typename... T>
__device__ __forceinline__ void copies_landed(const T*... tiles) {
  __builtin_amdgcn_s_waitcnt(0);
  (tile_written(tiles), ...);
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

// S^T tiles of one page for the wave's column tiles: s[c][h] holds keys
// 32h .. 32h+31 of column tile c; accumulator slot v of lane half hf is row
// 8*(v/4) + 4*hf + v%4 of the tile, i.e. key
// 32h + 16*(v/8) + 8*hf + 4*((v/4)%2) + v%4 (key_of_row).
template <int CT>
struct SPage {
  f32x16 s[CT][2];
};
// P^T fragments (bf16) of one page: p[c][kk] covers keys 16kk .. 16kk+15.
template <int CT>
struct PFrag {
  bf16x8 p[CT][4];
};

// ---- MFMAs with explicit register classes (inline asm) ----
// With one wave per SIMD (AG = true) the O^T accumulators and Q^T fragments
// live in AGPRs and the S^T tiles and P^T fragments in VGPRs; with two waves
// per SIMD everything is in VGPRs (a wave that uses AGPRs may only hold 128
// VGPRs).  The compiler cannot see the wait states these instructions need,
// so the kernel places explicit s_nop fences where an MFMA result is read by
// VALU code or a VALU result is read by an MFMA.
template <bool AG>
__device__ __forceinline__ void mfma_o(f32x16& o, const bf16x8& a, const bf16x8& b) {
  if constexpr (AG) asm volatile("v_mfma_f32_32x32x16_bf16 %0, %1, %2, %0" : "+a"(o) : "v"(a), "v"(b));
  else asm volatile("v_mfma_f32_32x32x16_bf16 %0, %1, %2, %0" : "+v"(o) : "v"(a), "v"(b));
}
template <bool AG>
__device__ __forceinline__ void mfma_s0(f32x16& s, const bf16x8& a, const bf16x8& b) {
  if constexpr (AG) asm volatile("v_mfma_f32_32x32x16_bf16 %0, %1, %2, 0" : "=&v"(s) : "v"(a), "a"(b));
  else asm volatile("v_mfma_f32_32x32x16_bf16 %0, %1, %2, 0" : "=&v"(s) : "v"(a), "v"(b));
}
template <bool AG>
__device__ __forceinline__ void mfma_s(f32x16& s, const bf16x8& a, const bf16x8& b) {
  if constexpr (AG) asm volatile("v_mfma_f32_32x32x16_bf16 %0, %1, %2, %0" : "+v"(s) : "v"(a), "a"(b));
  else asm volatile("v_mfma_f32_32x32x16_bf16 %0, %1, %2, %0" : "+v"(s) : "v"(a), "v"(b));
}

// Whole-tuple fence on the O^T accumulators: an MFMA result read or
// overwritten by VALU code, or a VALU result read by an MFMA, needs wait
// states the compiler cannot see through inline asm.
template <bool AG, int CT, int NDT>
__device__ __forceinline__ void fence_o(f32x16 (&o)[CT][NDT]) {
#pragma unroll
  for (int c = 0; c < CT; ++c)
#pragma unroll
    for (int x = 0; x < NDT; ++x) {
      if constexpr (AG) asm volatile("s_nop 7\n s_nop 7\n s_nop 7" : "+a"(o[c][x]));
      else asm volatile("s_nop 7\n s_nop 7\n s_nop 7" : "+v"(o[c][x]));
    }
}

// Fences on S^T tiles (MFMA results about to be read by the softmax) and on
// P^T fragments (VALU results about to be read by MFMAs).
template <int CT>
__device__ __forceinline__ void fence_sp(SPage<CT>& s, PFrag<CT>& p) {
  if constexpr (CT == 2)
    asm volatile("s_nop 7\n s_nop 7\n s_nop 4"
                 : "+v"(s.s[0][0]), "+v"(s.s[0][1]), "+v"(s.s[1][0]), "+v"(s.s[1][1]),
                   "+v"(p.p[0][0]), "+v"(p.p[0][1]), "+v"(p.p[0][2]), "+v"(p.p[0][3]),
                   "+v"(p.p[1][0]), "+v"(p.p[1][1]), "+v"(p.p[1][2]), "+v"(p.p[1][3]));
  else
    asm volatile("s_nop 7\n s_nop 7\n s_nop 4"
                 : "+v"(s.s[0][0]), "+v"(s.s[0][1]), "+v"(p.p[0][0]), "+v"(p.p[0][1]),
                   "+v"(p.p[0][2]), "+v"(p.p[0][3]));
}
template <int CT>
__device__ __forceinline__ void fence_s(SPage<CT>& s) {
  if constexpr (CT == 2)
    asm volatile("s_nop 7\n s_nop 7\n s_nop 5"
                 : "+v"(s.s[0][0]), "+v"(s.s[0][1]), "+v"(s.s[1][0]), "+v"(s.s[1][1]));
  else
    asm volatile("s_nop 7\n s_nop 7\n s_nop 5" : "+v"(s.s[0][0]), "+v"(s.s[0][1]));
}
template <int CT>
__device__ __forceinline__ void fence_p(PFrag<CT>& p) {
  if constexpr (CT == 2)
    asm volatile("s_nop 7\n s_nop 7\n s_nop 5"
                 : "+v"(p.p[0][0]), "+v"(p.p[0][1]), "+v"(p.p[0][2]), "+v"(p.p[0][3]),
                   "+v"(p.p[1][0]), "+v"(p.p[1][1]), "+v"(p.p[1][2]), "+v"(p.p[1][3]));
  else
    asm volatile("s_nop 7\n s_nop 7\n s_nop 5"
                 : "+v"(p.p[0][0]), "+v"(p.p[0][1]), "+v"(p.p[0][2]), "+v"(p.p[0][3]));
}

// Forces v to be computed at this point of the instruction stream (an empty
// volatile asm that reads it): keeps the softmax work of a slot from being
// moved to its uses by the compiler.
template <typename T>
__device__ __forceinline__ void pin(const T& v) {
  asm volatile("" : : "v"(v));
}

// Softmax schedule of one page for E weights per lane: E + 2 element ops
// (op j: score of element j, exp of element j-1, sum of element j-2) and
// E / 8 packs, the pack of unit u (elements 8u .. 8u+7) right after element
// op 8u+8.  soft_op(o, E) is j for an element op, -1-u for a pack.
constexpr int soft_ops(int E) { return E + 2 + E / 8; }
constexpr int soft_op(int o, int E) {
  int op = 0;
  for (int j = 0; j <= E + 1; ++j) {
    if (op++ == o) return j;
    if (j >= 8 && j <= E && (j - 8) % 8 == 0 && op++ == o) return -1 - (j - 8) / 8;
  }
  return 1 << 20;
}
static_assert(soft_op(soft_ops(64) - 1, 64) == 65 && soft_op(9, 64) == -1 &&
                  soft_op(soft_ops(64) - 2, 64) == -8 && soft_op(soft_ops(32) - 1, 32) == 33 &&
                  soft_op(soft_ops(32) - 2, 32) == -4,
              "softmax op table");

// Calls f(integral_constant<int, I>) for I = 0 .. N-1 (compile-time indices).
template <typename F, int... I>
__device__ __forceinline__ void static_for_impl(F& f, std::integer_sequence<int, I...>) {
  (f(std::integral_constant<int, I>{}), ...);
}
template <int N, typename F>
__device__ __forceinline__ void static_for(F&& f) {
  static_for_impl(f, std::make_integer_sequence<int, N>{});
}

template <int D, int NW, int CT, bool DENSE, int VL>
__global__ __launch_bounds__(64 * NW, CT == 1 ? 2 : 1) void paged_attention_kernel(const AttnArgs a) {
  constexpr bool AG = CT == 2;         // O^T and Q^T in AGPRs (one wave per SIMD)
  constexpr bool VTR = VL == kVTransposed;
  constexpr int VTILE = VTR ? kTileVT : kTileVR;
  constexpr int NKS = D / 16;          // QK k-steps
  constexpr int NDT = D / 32;          // O^T d tiles
  constexpr int PAGE = 64 * D;
  constexpr int ROWS = 32 * CT * NW;
  constexpr int NPV = 4 * NDT;         // V^T fragments per page
  constexpr int NQK = 2 * NKS;         // K fragments per page
  constexpr int NFRAG = NPV + NQK;
  constexpr int NSLOT = CT * NFRAG;    // one MFMA per slot
  constexpr int FD = CT == 1 ? 4 : 3;  // fragment prefetch distance (slots)
  constexpr int DMA_PER_STEP = 2 * (64 * D * 2) / 1024 / NW;   // copy instructions per wave
  constexpr int DMA_STRIDE = (NSLOT / 2) / DMA_PER_STEP > 0 ? (NSLOT / 2) / DMA_PER_STEP : 1;
  constexpr int MAXS = 5 * CT;         // slots holding the max / rebase work
  constexpr int NE = 32 * CT;          // softmax weights per lane per page
  constexpr int NSOFT = soft_ops(NE);
  __shared__ __attribute__((aligned(1024))) uint16_t k_s0[PAGE];
  __shared__ __attribute__((aligned(1024))) uint16_t k_s1[PAGE];
  __shared__ __attribute__((aligned(1024))) uint16_t v_s0[PAGE];
  __shared__ __attribute__((aligned(1024))) uint16_t v_s1[PAGE];

  const int t = threadIdx.x;
  const int wv = __builtin_amdgcn_readfirstlane(t >> 6);
  const int lane = t & 63;
  const int col = lane & 31;
  const int half = lane >> 5;

  int bid = blockIdx.x;
  const int nwg = gridDim.x;
  if ((nwg & 7) == 0) bid = (bid & 7) * (nwg >> 3) + (bid >> 3);
  int sp, qt, rowid;
  if (a.split_at != nullptr) {
    // XCD x (logical workgroups [x, x+1) * nwg/8) holds the rows r with
    // r % 8 = x (group x of every sequence when G = 8); it first runs piece 0
    // of its own rows' tiles, then piece 1 of the previous XCD's rows' tiles:
    // each piece is read by all tiles of its row on one XCD, in step, through
    // that XCD's L2
    const int per_xcd = nwg / kXcds, own = per_xcd / 2;
    const int x = bid / per_xcd;
    int j = bid % per_xcd;
    sp = j < own ? 0 : 1;
    if (sp) j -= own;
    rowid = (sp ? x + kXcds - 1 : x) % kXcds + kXcds * (j / a.n_qtiles);
    qt = j % a.n_qtiles;
    if (sp) qt = a.n_qtiles - 1 - qt;   // second pieces in mirrored tile order
  } else {
    // XCD x holds the units u with u % 8 = x when the units spread evenly (a
    // unit = the table rows that read one KV head's pages: one group row, or
    // the heads of one KV group in the per-(head, Q-block) layout), so that
    // sequences of different lengths share every XCD; otherwise rows in order
    const int per_row = a.splits * a.n_qtiles;
    const int U = a.rows_per_unit;
    const int units = nwg / per_row / U;
    int rest;
    if ((nwg & 7) == 0 && units % kXcds == 0) {
      const int per_xcd = nwg / kXcds, per_unit = U * per_row;
      const int x = bid / per_xcd, j = bid % per_xcd;
      rowid = (x + kXcds * (j / per_unit)) * U + (j % per_unit) / per_row;
      rest = j % per_row;
    } else {
      rowid = bid / per_row;
      rest = bid % per_row;
    }
    sp = rest % a.splits;
    qt = rest / a.splits;
  }
  const int b = rowid / a.G;
  const int g = rowid % a.G;
  const int gs = a.group_size;
  const int QT = ROWS / gs;            // chunk queries per tile
  const int q0 = qt * QT;
  const int q_end = q0 + QT < a.C ? q0 + QT : a.C;   // the last tile may be partial
  int head[CT], tq[CT];
  bool valid[CT];
#pragma unroll
  for (int c = 0; c < CT; ++c) {
    const int r = wv * 32 * CT + 32 * c + col;
    head[c] = g * gs + r / QT;
    tq[c] = q0 + r % QT;
    valid[c] = tq[c] < a.C;
    if (!valid[c]) tq[c] = a.C - 1;    // computes a copy of a real row, never stored
  }
  const int kvh = (g * gs) / (a.Hq / a.Hkv);
  const int cl = a.cached_len[b];
  const int nkb = blocks_for(cl + a.C);
  int qpos[CT];
#pragma unroll
  for (int c = 0; c < CT; ++c) qpos[c] = cl + tq[c];
  const int j_last = (cl + q_end - 1) / kPage;     // last block any row can see
  const int mask_from = cl + q0;                   // keys beyond this need masking

  int len, tbase = 0;
  if (DENSE) {
    len = nkb;
  } else {
    // per-group rows, or one row per (head, query tile) for the block-sparse arm
    const int trow = a.table_mode == kTablesPerQTile ? rowid * a.n_qtiles + qt : rowid;
    tbase = a.kv_indptr[trow];
    len = a.kv_indptr[trow + 1] - tbase;
  }
  int e0, e1;
  bool whole = a.splits == 1;   // the piece is the whole row: final output
  if (a.split_at != nullptr) {
    int cut = a.split_at[rowid];
    if (cut < 0) {              // the row is not cut: one piece runs it, the other nothing
      if (sp != (cut == -1 ? 0 : 1)) return;
      whole = true;
      cut = sp ? 0 : len;
    }
    if (!whole) {
      // Tile q sees the chunk's blocks up to j_last(q), so its second piece
      // (which holds them) is longer for later tiles.  The first piece of tile
      // q moves by (j_last(q) - j_last(mirror q)) / 4 entries: the CUs that
      // finish their first pieces early take the long second pieces (mirrored
      // order above), and with the chunk's evenly growing j_last every CU of
      // the XCD ends together.
      const int qm = a.n_qtiles - 1 - qt;
      const int qm_end = (qm + 1) * QT < a.C ? (qm + 1) * QT : a.C;
      cut += (j_last - (cl + qm_end - 1) / kPage) / 4;
      cut = cut < 0 ? 0 : cut;
    }
    cut = cut > len ? len : cut;
    e0 = sp ? cut : 0;
    e1 = sp ? len : cut;
  } else {
    e0 = (int)(((long long)len * sp) / a.splits);
    e1 = (int)(((long long)len * (sp + 1)) / a.splits);
  }
  const int32_t* ptab = a.page_table + ((size_t)b * a.Hkv + kvh) * a.max_kv_blocks;

  bf16x8 qf[CT][NKS];
#pragma unroll
  for (int c = 0; c < CT; ++c) {
    const uint16_t* qrow = a.q + (((size_t)b * a.C + tq[c]) * a.Hq + head[c]) * D + 8 * half;
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks) {
      qf[c][ks] = *reinterpret_cast<const bf16x8*>(qrow + 16 * ks);
      if constexpr (AG) asm volatile("s_nop 2" : "+a"(qf[c][ks]));   // into AGPRs
    }
  }

  f32x16 o[CT][NDT];
#pragma unroll
  for (int c = 0; c < CT; ++c)
#pragma unroll
    for (int x = 0; x < NDT; ++x)
#pragma unroll
      for (int v = 0; v < 16; ++v) o[c][x][v] = 0.f;
  fence_o<AG, CT, NDT>(o);
  float m_run[CT], l_run[CT];
#pragma unroll
  for (int c = 0; c < CT; ++c) {
    m_run[c] = -INFINITY;
    l_run[c] = 0.f;
  }

  int e_end = e1;
  if (DENSE) {
    // a split may start past the tile's last visible block: then it is empty
    e_end = e1 < j_last + 1 ? e1 : j_last + 1;
    e_end = e_end > e0 ? e_end : e0;
  } else {
    while (e_end > e0 && a.kv_indices[tbase + e_end - 1] > j_last) --e_end;
  }
  const int n = e_end - e0;
  int n_main = n;
  while (n_main > 0 &&
         kPage * (DENSE ? e0 + n_main - 1 : a.kv_indices[tbase + e0 + n_main - 1]) + kPage - 1 >
             mask_from)
    --n_main;
  // pages run by the software-pipelined loop: an even number of unmasked ones
  const int n_pipe = n_main & ~1;

  SPage<CT> SA, SB;
  PFrag<CT> PA, PB;
  int base = 0, blk_cur = 0, pg_cur = 0, blk_nxt = 0, pg_nxt = 0;
  auto fetch = [&](int b0, int& blk, int& pg) {
    int idx = b0 + lane;
    idx = idx < n ? idx : n - 1;
    idx = idx < 0 ? 0 : idx;
    blk = (n > 0) ? (DENSE ? e0 + idx : a.kv_indices[tbase + e0 + idx]) : 0;
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
  auto advance = [&](int i) {
    while (i - base >= 64) {
      base += 64;
      blk_cur = blk_nxt;
      pg_cur = pg_nxt;
      fetch(base + 64, blk_nxt, pg_nxt);
    }
  };
  auto id_of = [&](int cur, int nxt, int i) -> int {
    const int d = i - base;
    return d < 64 ? __builtin_amdgcn_readlane(cur, d) : __builtin_amdgcn_readlane(nxt, d - 64);
  };
  auto page_ptr = [&](const uint16_t* pool, int i) -> const uint16_t* {
    return pool + (size_t)id_of(pg_cur, pg_nxt, i) * (kPage * D);
  };

  // Per-lane byte offsets of the MFMA operand reads inside a page tile; the
  // buffer, the d tile or 16-key block of a PV step and the upper 32 keys of
  // a QK step are immediates.  Lane column col reads key row key_of_row(col)
  // of K, so its P^T fragment kk holds keys 16kk + 8*half .. +7: in a
  // transposed V tile one 16-byte chunk of V^T row 32x + col; in a
  // token-major tile two transpose reads (keys +0..3 and +4..7; the 16 lanes
  // of a transpose read address 4 key rows x 16 d and receive one d each).
  constexpr int NVOFS = VTR ? 4 : NDT;
  uint32_t kofs[NKS], vofs[NVOFS];
#pragma unroll
  for (int x = 0; x < NKS; ++x) {
    const int kr = key_of_row(col);
    kofs[x] = (uint32_t)(kr * D * 2 + 16 * k_swz<D>(kr, 2 * x + half));
  }
  if constexpr (VTR) {
#pragma unroll
    for (int kk = 0; kk < 4; ++kk)
      vofs[kk] = (uint32_t)(col * kPage * 2 + 16 * vt_swz(col, 2 * kk + half));
  } else {
    const int grp = lane >> 4, sl = lane & 15;
    const int r0 = 8 * (grp >> 1) + (sl >> 2);
#pragma unroll
    for (int x = 0; x < NDT; ++x) {
      const int d = 32 * x + 16 * (grp & 1) + 4 * (sl & 3);
      vofs[x] = (uint32_t)(r0 * D * 2 + 16 * vr_swz<D>(r0, d >> 3) + 2 * (d & 7));
    }
  }
  // fragment F of a step: F < NPV is V^T fragment (kk = F / NDT, d tile
  // x = F % NDT), otherwise K fragment (k-step (F - NPV) / 2, keys
  // 32 * ((F - NPV) % 2) ..)
  auto load_frag = [&](int F, const uint16_t* vt, const uint16_t* kt) -> bf16x8 {
    if (F < NPV) {
      const int kk = F / NDT, x = F % NDT;
      if constexpr (VTR) {
        const char* p = reinterpret_cast<const char*>(vt) + vofs[kk] + 32 * kPage * 2 * x;
        return *reinterpret_cast<const bf16x8*>(p);
      } else {
        const char* p = reinterpret_cast<const char*>(vt) + vofs[x] + 16 * kk * D * 2;
        const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)p);
        const i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(p + 4 * D * 2));
        const u32x2 l2 = __builtin_bit_cast(u32x2, lo), h2 = __builtin_bit_cast(u32x2, hi);
        const u32x4 w = {l2[0], l2[1], h2[0], h2[1]};
        return __builtin_bit_cast(bf16x8, w);
      }
    }
    const int G2 = F - NPV;
    const char* p = reinterpret_cast<const char*>(kt) + kofs[G2 / 2] + (G2 % 2) * 32 * D * 2;
    return *reinterpret_cast<const bf16x8*>(p);
  };

  // Whole-page contractions (outside the pipelined loop).
  auto qk_page = [&](SPage<CT>& st, const uint16_t* kt) __attribute__((always_inline)) {
    static_for<NQK>([&](auto gtag) __attribute__((always_inline)) {
      constexpr int G2 = decltype(gtag)::value, x = G2 / 2, h = G2 % 2;
      const bf16x8 kf = load_frag(NPV + G2, kt, kt);
#pragma unroll
      for (int c = 0; c < CT; ++c) {
        if constexpr (x == 0) mfma_s0<AG>(st.s[c][h], kf, qf[c][x]);
        else mfma_s<AG>(st.s[c][h], kf, qf[c][x]);
      }
    });
  };
  auto pv_page = [&](const PFrag<CT>& pf, const uint16_t* vt) __attribute__((always_inline)) {
    static_for<NPV>([&](auto ftag) __attribute__((always_inline)) {
      constexpr int F = decltype(ftag)::value;
      const bf16x8 vf = load_frag(F, vt, vt);
#pragma unroll
      for (int c = 0; c < CT; ++c) mfma_o<AG>(o[c][F % NDT], vf, pf.p[c][F / NDT]);
    });
  };

  // Prologue: K(0) -> k_s0, K(1) -> k_s1, and V(0) into the buffer the first
  // step's PV reads, with a zero P: that PV adds nothing and every tile read
  // is initialised.  Then S(0).
#pragma unroll
  for (int c = 0; c < CT; ++c)
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) PB.p[c][kk] = __builtin_bit_cast(bf16x8, u32x4{0u, 0u, 0u, 0u});
  if (n_pipe > 0) {
    page_to_lds<D, NW, kTileK>(page_ptr(a.k_pool, 0), k_s0, wv, lane);
    page_to_lds<D, NW, kTileK>(page_ptr(a.k_pool, 1), k_s1, wv, lane);
    page_to_lds<D, NW, VTILE>(page_ptr(a.v_pool, 0), v_s1, wv, lane);
    copies_landed(k_s0, k_s1, v_s1);
    __syncthreads();
    qk_page(SA, k_s0);
    __syncthreads();
    fence_sp<CT>(SA, PB);   // S(0) and the zero P are read by the first step's first slots
  }

  // Step i: DMA K(i+2) -> k[i%2], V(i) -> v[i%2]; PV(i-1) from v[(i-1)%2] and
  // P(i-1); QK(i+1) from k[(i+1)%2]; softmax(i) of S(i) into P(i).  One MFMA
  // per slot, the softmax work spread over the slots.
  auto step = [&](auto par, int i) __attribute__((always_inline)) {
    constexpr int P = decltype(par)::value;
    SPage<CT>& sc = P ? SB : SA;
    SPage<CT>& sn = P ? SA : SB;
    PFrag<CT>& pn = P ? PB : PA;
    PFrag<CT>& po = P ? PA : PB;
    uint16_t* const k_dma = P ? k_s1 : k_s0;
    const uint16_t* const k_rd = P ? k_s0 : k_s1;
    uint16_t* const v_dma = P ? v_s1 : v_s0;
    const uint16_t* const v_rd = P ? v_s0 : v_s1;
    const int i2 = i + 2 < n_pipe ? i + 2 : n_pipe - 1;
    const uint16_t* const k_src = page_ptr(a.k_pool, i2);
    const uint16_t* const v_src = page_ptr(a.v_pool, i);
    // No hazard fence here: the last MFMA writing S and the last pack writing
    // P come well before their first readers in this step (end of step,
    // barrier, page pointers); the hazard test checks the distance.
    float mx[CT][2], alpha[CT], nmb[CT], ps[CT];
#pragma unroll
    for (int c = 0; c < CT; ++c) {
      mx[c][0] = mx[c][1] = -INFINITY;
      alpha[c] = 1.f;
      nmb[c] = 0.f;
      ps[c] = 0.f;
    }
    bool rb_any = false;
    bf16x8 fr[NFRAG];
#pragma unroll
    for (int f = 0; f < FD; ++f) fr[f] = load_frag(f, v_rd, k_rd);
    static_for<NSLOT>([&](auto stag) __attribute__((always_inline)) {
      constexpr int s = decltype(stag)::value;
      constexpr int F = s / CT, c = s % CT;
      if constexpr (c == 0 && F + FD < NFRAG) fr[F + FD] = load_frag(F + FD, v_rd, k_rd);
      // the copies of K(i+2) and V(i), one instruction every DMA_STRIDE slots
      // over the first half of the step (issued all at once they queue in
      // the address unit and stall the wave)
      if constexpr (s % DMA_STRIDE == 0 && s / DMA_STRIDE < DMA_PER_STEP) {
        constexpr int m = s / DMA_STRIDE;
        if constexpr (m < DMA_PER_STEP / 2)
          page_part_to_lds<D, NW, kTileK>(k_src, k_dma, wv, lane, m);
        else
          page_part_to_lds<D, NW, VTILE>(v_src, v_dma, wv, lane, m - DMA_PER_STEP / 2);
      }
      if constexpr (F < NPV) {
        mfma_o<AG>(o[c][F % NDT], fr[F], po.p[c][F / NDT]);
      } else {
        constexpr int G2 = F - NPV, x = G2 / 2, h = G2 % 2;
        if constexpr (x == 0) mfma_s0<AG>(sn.s[c][h], fr[F], qf[c][x]);
        else mfma_s<AG>(sn.s[c][h], fr[F], qf[c][x]);
      }
      // softmax work of this slot
      if constexpr (s < 4 * CT) {
        // two independent max chains per column tile (half the dependent latency)
        constexpr int cc = s / 4, k0 = 4 * (s % 4);
        mx[cc][0] = max3(mx[cc][0], sc.s[cc][0][k0], sc.s[cc][1][k0]);
        mx[cc][1] = max3(mx[cc][1], sc.s[cc][0][k0 + 1], sc.s[cc][1][k0 + 1]);
        mx[cc][0] = max3(mx[cc][0], sc.s[cc][0][k0 + 2], sc.s[cc][1][k0 + 2]);
        mx[cc][1] = max3(mx[cc][1], sc.s[cc][0][k0 + 3], sc.s[cc][1][k0 + 3]);
        pin(mx[cc][0]);
        pin(mx[cc][1]);
      } else if constexpr (s < MAXS) {
        constexpr int cc = s - 4 * CT;
        const float m = halves_max(fmaxf(mx[cc][0], mx[cc][1])) * a.scale_log2;
        const bool rebase = m > m_run[cc] + kRescaleSlack;
        alpha[cc] = rebase ? fast_exp2(m_run[cc] - m) : 1.0f;
        m_run[cc] = rebase ? m : m_run[cc];
        rb_any |= rebase;
        nmb[cc] = (m_run[cc] == -INFINITY) ? 0.f : -m_run[cc];
        pin(nmb[cc]);
        pin(alpha[cc]);
      } else {
        // Weights of the page, software-pipelined over the remaining slots so
        // that no instruction waits on the one before it: element op j does
        // the scaled score of element j, the exp of element j-1 and the row
        // sum of element j-2 (elements in unit order, unit u = 8 weights of
        // one P^T fragment); unit u is packed to bf16 after element op 8u+8.
        constexpr int lo = ((s - MAXS) * NSOFT) / (NSLOT - MAXS);
        constexpr int hi = ((s - MAXS + 1) * NSOFT) / (NSLOT - MAXS);
        static_for<hi - lo>([&](auto otag) __attribute__((always_inline)) {
          constexpr int op = soft_op(lo + decltype(otag)::value, NE);
          if constexpr (op >= 0) {
            if constexpr (op < NE) {
              constexpr int u = op / 8, cc = u / 4, kk = u % 4, v = 8 * (kk % 2) + op % 8;
              f32x16& sv = sc.s[cc][kk / 2];
              sv[v] = fmaf(sv[v], a.scale_log2, nmb[cc]);
              pin(sv[v]);
            }
            if constexpr (op >= 1 && op <= NE) {
              constexpr int e = op - 1, u = e / 8, cc = u / 4, kk = u % 4, v = 8 * (kk % 2) + e % 8;
              f32x16& sv = sc.s[cc][kk / 2];
              sv[v] = fast_exp2(sv[v]);
              pin(sv[v]);
            }
            if constexpr (op >= 2) {
              constexpr int e = op - 2, u = e / 8, cc = u / 4, kk = u % 4, v = 8 * (kk % 2) + e % 8;
              ps[cc] += sc.s[cc][kk / 2][v];
              pin(ps[cc]);
            }
          } else {
            constexpr int u = -1 - op, cc = u / 4, kk = u % 4;
            const f32x16& sv = sc.s[cc][kk / 2];
#pragma unroll
            for (int x = 0; x < 8; ++x) pn.p[cc][kk][x] = (__bf16)sv[8 * (kk % 2) + x];
            pin(pn.p[cc][kk]);
          }
        });
      }
      __builtin_amdgcn_sched_barrier(0);
    });
#pragma unroll
    for (int c = 0; c < CT; ++c) l_run[c] = l_run[c] * alpha[c] + ps[c];
    const uint64_t any = __ballot(rb_any);
    if (any) {   // the exponent base moved on some lane: rescale O (rare)
      fence_o<AG, CT, NDT>(o);
#pragma unroll
      for (int c = 0; c < CT; ++c)
#pragma unroll
        for (int x = 0; x < NDT; ++x) o[c][x] *= alpha[c];
      fence_o<AG, CT, NDT>(o);
    }
    copies_landed(k_dma, v_dma);
    __syncthreads();
  };
  using P0 = std::integral_constant<int, 0>;
  using P1 = std::integral_constant<int, 1>;
  if (n_pipe > 0) {
    for (int i = 0; i < n_pipe; i += 2) {
      advance(i);
      step(P0{}, i);
      advance(i + 1);
      step(P1{}, i + 1);
    }
    // PV of page n_pipe - 1 (odd: its P is PB, its V in v_s1)
    fence_p<CT>(PB);
    pv_page(PB, v_s1);
    __syncthreads();
  }

  // Remaining pages (the causally masked diagonal ones and an odd leftover),
  // one at a time without overlap: K and V of the page to LDS, S = K Q^T,
  // mask, softmax, O += V^T P^T.
  for (int i = n_pipe; i < n; ++i) {
    advance(i);
    page_to_lds<D, NW, kTileK>(page_ptr(a.k_pool, i), k_s0, wv, lane);
    page_to_lds<D, NW, VTILE>(page_ptr(a.v_pool, i), v_s0, wv, lane);
    copies_landed(k_s0, v_s0);
    __syncthreads();
    if (i >= n_main) {
      // The tokens of a sequence's last page past its end are not part of it
      // and may hold anything: their weights are exactly 0, so their V
      // entries (the last `past` keys of the page) are zeroed to keep
      // 0 * NaN out of O (their K scores are masked).
      const int past = kPage * id_of(blk_cur, blk_nxt, i) + kPage - (cl + a.C);
      if (past > 0) {
        for (int x = t; x < past * D; x += 64 * NW) {
          const int r = x / past, key = kPage - past + x % past;   // r: the d index
          if constexpr (VTR) v_s0[r * kPage + 8 * vt_swz(r, key >> 3) + (key & 7)] = 0;
          else v_s0[key * D + 8 * vr_swz<D>(key, r >> 3) + (r & 7)] = 0;
        }
        __syncthreads();
      }
    }
    qk_page(SA, k_s0);
    fence_s<CT>(SA);
    if (i >= n_main) {
      const int j = id_of(blk_cur, blk_nxt, i);
#pragma unroll
      for (int c = 0; c < CT; ++c) {
        const int lim = qpos[c] - kPage * j - 8 * half;
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const int kp = 16 * (v >> 3) + 4 * ((v >> 2) & 1) + (v & 3);   // key - 8*half
          if (kp > lim) SA.s[c][0][v] = -INFINITY;
          if (kp + 32 > lim) SA.s[c][1][v] = -INFINITY;
        }
      }
    }
    float alpha[CT];
    bool rb_any = false;
#pragma unroll
    for (int c = 0; c < CT; ++c) {
      float mx = -INFINITY;
#pragma unroll
      for (int k = 0; k < 16; ++k) mx = max3(mx, SA.s[c][0][k], SA.s[c][1][k]);
      const float m = halves_max(mx) * a.scale_log2;
      const bool rebase = m > m_run[c] + kRescaleSlack;
      alpha[c] = rebase ? fast_exp2(m_run[c] - m) : 1.0f;
      m_run[c] = rebase ? m : m_run[c];
      rb_any |= rebase;
      const float nmb = (m_run[c] == -INFINITY) ? 0.f : -m_run[c];
      float ps = 0.f;
#pragma unroll
      for (int h = 0; h < 2; ++h)
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const float e = fast_exp2(fmaf(SA.s[c][h][v], a.scale_log2, nmb));
          SA.s[c][h][v] = e;
          ps += e;
        }
      l_run[c] = l_run[c] * alpha[c] + ps;
#pragma unroll
      for (int kk = 0; kk < 4; ++kk)
#pragma unroll
        for (int x = 0; x < 8; ++x) PA.p[c][kk][x] = (__bf16)SA.s[c][kk / 2][8 * (kk % 2) + x];
    }
    if (__ballot(rb_any)) {
      fence_o<AG, CT, NDT>(o);
#pragma unroll
      for (int c = 0; c < CT; ++c)
#pragma unroll
        for (int x = 0; x < NDT; ++x) o[c][x] *= alpha[c];
      fence_o<AG, CT, NDT>(o);
    }
    fence_p<CT>(PA);
    pv_page(PA, v_s0);
    __syncthreads();
  }
  fence_o<AG, CT, NDT>(o);

  // epilogue
#pragma unroll
  for (int c = 0; c < CT; ++c) {
    const float l_tot = halves_sum(l_run[c]);
    const float inv = l_tot > 0.f ? 1.0f / l_tot : 0.f;
    const float lse_val = l_tot > 0.f ? (m_run[c] + log2f(l_tot)) * kLn2 : -INFINITY;
    const size_t qrow_idx = ((size_t)b * a.Hq + head[c]) * a.C + tq[c];
    if (!valid[c]) continue;
    if (whole) {
      uint16_t* orow = a.out + (((size_t)b * a.C + tq[c]) * a.Hq + head[c]) * D;
#pragma unroll
      for (int x = 0; x < NDT; ++x) {
#pragma unroll
        for (int q4 = 0; q4 < 4; ++q4) {
          const int d = 32 * x + 8 * q4 + 4 * half;
          uint2 pk;
          pk.x = pack_bf16x2(o[c][x][4 * q4 + 0] * inv, o[c][x][4 * q4 + 1] * inv);
          pk.y = pack_bf16x2(o[c][x][4 * q4 + 2] * inv, o[c][x][4 * q4 + 3] * inv);
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
              make_float4(o[c][x][4 * q4 + 0] * inv, o[c][x][4 * q4 + 1] * inv,
                          o[c][x][4 * q4 + 2] * inv, o[c][x][4 * q4 + 3] * inv);
        }
      }
      if (half == 0) a.part_lse[prow] = lse_val;
    }
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
                                                      int C, int splits,
                                                      const int32_t* __restrict__ split_at,
                                                      int G, int group_size) {
  constexpr int PER = D / 32;
  const size_t nrows = (size_t)B * Hq * C;
  const size_t row = (size_t)blockIdx.x * 8 + (threadIdx.x >> 5);
  if (row >= nrows) return;
  const int sub = threadIdx.x & 31;
  auto load_part = [&](int i, float (&v)[PER]) {
    const float* po = part_o + ((size_t)i * nrows + row) * D + sub * PER;
    if constexpr (PER == 4) {
      const float4 f = *reinterpret_cast<const float4*>(po);
      v[0] = f.x, v[1] = f.y, v[2] = f.z, v[3] = f.w;
    } else {
      const float2 f = *reinterpret_cast<const float2*>(po);
      v[0] = f.x, v[1] = f.y;
    }
  };
  float acc[PER];
#pragma unroll
  for (int x = 0; x < PER; ++x) acc[x] = 0.f;
  float wsum = 0.f, mx = -INFINITY;
  if (splits == 2) {
    // Two pieces (the XCD-balanced split): every load is issued before any
    // result is needed, so the row costs one memory latency instead of three.
    // The slots of an uncut row are stale; they are loaded but never used.
    float v0[PER], v1[PER];
    const int cut = split_at != nullptr
        ? split_at[(int)(row / ((size_t)C * Hq)) * G + (int)((row / C) % Hq) / group_size]
        : 0;
    const float l0 = part_lse[row], l1 = part_lse[nrows + row];
    load_part(0, v0);
    load_part(1, v1);
    if (cut < 0) return;   // a table row that was not cut wrote its output already
    mx = fmaxf(l0, l1);
    if (mx != -INFINITY) {
      const float w0 = l0 == -INFINITY ? 0.f : expf(l0 - mx);
      const float w1 = l1 == -INFINITY ? 0.f : expf(l1 - mx);
      wsum = w0 + w1;
#pragma unroll
      for (int x = 0; x < PER; ++x)
        acc[x] = (w0 > 0.f ? w0 * v0[x] : 0.f) + (w1 > 0.f ? w1 * v1[x] : 0.f);
    }
  } else {
    if (split_at != nullptr) {   // a table row that was not cut wrote its output already
      const int hh = (int)((row / C) % Hq), bb = (int)(row / ((size_t)C * Hq));
      if (split_at[bb * G + hh / group_size] < 0) return;
    }
    for (int i = 0; i < splits; ++i) mx = fmaxf(mx, part_lse[(size_t)i * nrows + row]);
  }
  if (splits != 2 && mx != -INFINITY) {
    for (int i = 0; i < splits; ++i) {
      const float li = part_lse[(size_t)i * nrows + row];
      if (li == -INFINITY) continue;
      const float wgt = expf(li - mx);
      wsum += wgt;
      float v[PER];
      load_part(i, v);
#pragma unroll
      for (int x = 0; x < PER; ++x) acc[x] = fmaf(wgt, v[x], acc[x]);
    }
  }
  const float inv = wsum > 0.f ? 1.0f / wsum : 0.f;
  // row is in [B, Hq, C] order; out is [B, C, Hq, D]
  const int tq = (int)(row % C);
  const int h = (int)((row / C) % Hq);
  const int b = (int)(row / ((size_t)C * Hq));
  uint16_t* orow = out + (((size_t)b * C + tq) * Hq + h) * D + sub * PER;
  uint32_t pk[PER / 2];
#pragma unroll
  for (int x = 0; x < PER / 2; ++x) pk[x] = pack_bf16x2(acc[2 * x] * inv, acc[2 * x + 1] * inv);
  if constexpr (PER == 4) *reinterpret_cast<uint2*>(orow) = make_uint2(pk[0], pk[1]);
  else *reinterpret_cast<uint32_t*>(orow) = pk[0];
  if (lse != nullptr && sub == 0) lse[row] = wsum > 0.f ? mx + logf(wsum) : -INFINITY;
}

// Cut points of the XCD-balanced two-piece split.  The R = 8m table rows are
// spread over the 8 XCDs by r % 8 (XCD x holds rows x, x+8, ..; its load
// alone is L_x table entries).  XCD x runs the first C_x
// entries of its own rows and the remaining L_{x-1} - C_{x-1} of the previous
// XCD's rows, so its load is C_x + L_{x-1} - C_{x-1}; equal loads S = sum L / 8
// give C_x = C_{x-1} + S - L_{x-1}, fixed up to the choice of C_0, which is
// taken in the middle of the range that keeps every 0 <= C_x <= L_x (clamped
// when no such choice exists).  C_x is shared among the rows of XCD x in
// proportion to their lengths.  Dense tables: row r has nKB_b entries.
__global__ __launch_bounds__(256) void xcd_split_kernel(const int32_t* __restrict__ kv_indptr,
                                                        const int32_t* __restrict__ cached_len,
                                                        int32_t* __restrict__ split_at, int R,
                                                        int G, int C, int dense) {
  __shared__ long long L[kXcds], Cx[kXcds];
  const int m = R / kXcds;
  const int t = threadIdx.x;
  auto row_len = [&](int r) -> long long {
    return dense ? (long long)blocks_for(cached_len[r / G] + C)
                 : (long long)(kv_indptr[r + 1] - kv_indptr[r]);
  };
  if (t < kXcds) {   // L_x, one thread per XCD
    long long v = 0;
    for (int k = 0; k < m; ++k) v += row_len(t + kXcds * k);
    L[t] = v;
  }
  __syncthreads();
  if (t == 0) {
    long long total = 0;
    for (int x = 0; x < kXcds; ++x) total += L[x];
    // D_x = sum_{k=1..x} (S - L_{k-1}) in units of 1/8 entry (S = total / 8);
    // 8 C_0 is taken in the middle of the range keeping 0 <= C_x <= L_x
    long long D8[kXcds];
    D8[0] = 0;
    for (int x = 1; x < kXcds; ++x) D8[x] = D8[x - 1] + total - 8 * L[x - 1];
    long long lo = 0, hi = 8 * L[0];
    for (int x = 0; x < kXcds; ++x) {
      lo = lo > -D8[x] ? lo : -D8[x];
      hi = hi < 8 * L[x] - D8[x] ? hi : 8 * L[x] - D8[x];
    }
    // any feasible C_0 balances; the largest keeps the most entries on their
    // own XCD, and rows with C_x = L_x (or 0) are not cut at all
    const long long c0 = lo <= hi ? hi : (lo + hi) / 2;   // lo > hi: clamped below
    for (int x = 0; x < kXcds; ++x) {
      long long cx = (c0 + D8[x]) / 8;
      Cx[x] = cx < 0 ? 0 : (cx > L[x] ? L[x] : cx);
    }
  }
  __syncthreads();
  if (t < kXcds) {   // C_x over the rows of XCD x in proportion to their lengths
    long long before = 0;
    for (int k = 0; k < m; ++k) {
      const int r = t + kXcds * k;
      const long long len = row_len(r);
      const long long a0 = L[t] > 0 ? (before * Cx[t]) / L[t] : 0;
      const long long a1 = L[t] > 0 ? ((before + len) * Cx[t]) / L[t] : 0;
      const long long c = a1 - a0;
      split_at[r] = c >= len ? -1 : (c <= 0 ? -2 : (int32_t)c);
      before += len;
    }
  }
}

int attn_rows_per_workgroup(int table_mode) {
  return 32 * kColTiles * (table_mode == kTablesPerQTile ? kWavesQTile : kWavesGroup);
}

int attn_query_tile(int group_size, int table_mode) {
  return attn_rows_per_workgroup(table_mode) / group_size;
}

int attn_base_workgroups(const Dims& d, int group_size, int table_mode) {
  const int qt = attn_query_tile(group_size, table_mode);
  return d.B * (d.Hq / group_size) * ((d.C + qt - 1) / qt);
}

int attn_resident_workgroups(int table_mode) {
  // kWavesPerCu waves per CU on 256 CUs
  return 256 * kWavesPerCu / (table_mode == kTablesPerQTile ? kWavesQTile : kWavesGroup);
}

size_t attn_ws_bytes(const Dims& d, int splits) {
  if (splits <= 1) return 0;
  const size_t rows = (size_t)d.B * d.Hq * d.C;
  return (size_t)splits * rows * (d.D + 1) * sizeof(float);
}

size_t attn_xcd_ws_bytes(const Dims& d, int group_size) {
  return attn_ws_bytes(d, 2) + (size_t)d.B * (d.Hq / group_size) * sizeof(int32_t);
}

template <int D, int NW, int VL>
static void launch_kernel(const AttnArgs& a, bool dense, int nwg, hipStream_t st) {
  if (dense) paged_attention_kernel<D, NW, kColTiles, true, VL><<<nwg, 64 * NW, 0, st>>>(a);
  else paged_attention_kernel<D, NW, kColTiles, false, VL><<<nwg, 64 * NW, 0, st>>>(a);
}

template <int D, int NW>
static void launch_layout(const AttnArgs& a, bool dense, int v_layout, int nwg, hipStream_t st) {
  if (v_layout == kVTransposed) launch_kernel<D, NW, kVTransposed>(a, dense, nwg, st);
  else launch_kernel<D, NW, kVTokenMajor>(a, dense, nwg, st);
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
  const int qt = attn_query_tile(L.group_size, L.table_mode);
  a.n_qtiles = (d.C + qt - 1) / qt;
  a.splits = L.splits;
  a.table_mode = L.table_mode;
  a.packed_pages = L.packed_pages;
  a.scale_log2 = L.sm_scale * kLog2e;
  a.split_at = nullptr;
  a.rows_per_unit = L.table_mode == kTablesPerQTile ? d.Hq / d.Hkv : 1;
  if (L.xcd_balanced) {
    const int R = d.B * a.G;
    int32_t* cut = reinterpret_cast<int32_t*>(static_cast<char*>(L.ws) + attn_ws_bytes(d, 2));
    xcd_split_kernel<<<1, 256, 0, st>>>(L.kv_indptr, L.cached_len, cut, R, a.G, d.C,
                                        L.dense ? 1 : 0);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    a.split_at = cut;
  }
  const int nwg = attn_base_workgroups(d, L.group_size, L.table_mode) * L.splits;
  const bool qtile = L.table_mode == kTablesPerQTile;
  if (d.D == 128) {
    if (qtile) launch_layout<128, kWavesQTile>(a, L.dense, L.v_layout, nwg, st);
    else launch_layout<128, kWavesGroup>(a, L.dense, L.v_layout, nwg, st);
  } else {
    if (qtile) launch_layout<64, kWavesQTile>(a, L.dense, L.v_layout, nwg, st);
    else launch_layout<64, kWavesGroup>(a, L.dense, L.v_layout, nwg, st);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || L.splits == 1) return e;
  const int cgrid = (int)((rows + 7) / 8);
  if (d.D == 128)
    combine_kernel<128><<<cgrid, 256, 0, st>>>(a.part_o, a.part_lse, L.out, L.lse, d.B, d.Hq,
                                               d.C, L.splits, a.split_at, a.G, L.group_size);
  else
    combine_kernel<64><<<cgrid, 256, 0, st>>>(a.part_o, a.part_lse, L.out, L.lse, d.B, d.Hq,
                                              d.C, L.splits, a.split_at, a.G, L.group_size);
  return hipGetLastError();
}

}  // namespace ca
