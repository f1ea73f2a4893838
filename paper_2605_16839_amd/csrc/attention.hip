// Zero-copy paged chunk attention over per-group block tables (Sec. 3.3,
// App. B.2), bf16 MFMA with fp32 online softmax, and the split-KV
// log-sum-exp merge.
//
// Work decomposition: one workgroup = NW wavefronts, 16*NCT (head, query)
// rows per wave: NCT = 2 runs two waves per SIMD (256 registers each), NCT = 4
// one wave per SIMD (512 registers):
//   * a table row r = b*G + g serves the group_size query heads of group g;
//     all of them read the same KV pages, so a workgroup packs rows of every
//     head of the group (group_size heads x 16*NCT*NW/group_size chunk
//     queries) and each KV page staged in LDS feeds all of them;
//   * the contractions are v_mfma_f32_16x16x32_bf16: a wave's rows are NCT
//     16-column tiles and a page's 64 keys four 16-key tiles, so every K and
//     V fragment a wave reads from LDS feeds NCT MFMAs.  On MI355X this kernel
//     runs at the board's power limit, and the 16x16x32 form moves half the
//     accumulator data per flop of the 32x32x16 form: the same flops then
//     cost less energy and the clock stays higher;
//   * S^T = K Q^T (keys x queries): a lane holds one query column of each of
//     its NCT column tiles and 4 keys of each 16-key tile; the softmax
//     statistics are in-lane plus a reduction over the 4 lane groups
//     (v_permlane16_swap, v_permlane32_swap); then O^T += V^T P^T.  Lanes read
//     the K rows of a page in an order (key_of) that gives every lane 8
//     consecutive keys of each 32-key P^T fragment, so the matching V^T
//     fragment is one 16-byte read of a transposed V page ([D, 64],
//     VL = kVTransposed) or two gfx950 transpose reads (ds_read_b64_tr_b16)
//     of a token-major page ([64, D], the paper's layout, VL = kVTokenMajor);
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
//     two so that the XCDs carry equal loads (xcd_cut, computed by each
//     workgroup from the table lengths);
//   * the XCD-balanced split's two pieces are merged inside the kernel: the
//     second piece of a query tile to finish (an arrival counter per tile)
//     reads the other's partial result and writes the output rows; uniform
//     splits are merged by combine_kernel.
#include <atomic>
#include <chrono>
#include <random>
#include <type_traits>
#include <utility>

#include "common.hpp"
#include "kernels.hpp"

namespace ca {

#ifndef CA_COL_TILES
#define CA_COL_TILES 2
#endif
// 16-column MFMA tiles per wave: 4 (one wave per SIMD, 512 registers) or 2
// (two waves per SIMD, 256 registers each).  Per-group tables: 256 rows per
// workgroup; block-sparse tiles (one head x 128 queries): 128 rows.
constexpr int kColTiles = CA_COL_TILES;
constexpr int kWavesGroup = 16 / kColTiles;
constexpr int kWavesQTile = 8 / kColTiles;
constexpr int kWavesPerCu = 16 / kColTiles;   // resident waves per CU
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
  // XCD-balanced split: one arrival counter per query tile (rowid * n_qtiles
  // + qt), (tag << 8) | the number of the tile's pieces that stored their
  // partial; a value with another tag counts 0, and the merging piece leaves
  // 0 behind.  nullptr otherwise (uniform splits: combine_kernel merges)
  unsigned long long* arrive;
  unsigned long long tag;   // this launch's tag, < 2^56 and never 0
  int B, Hq, Hkv, C, max_kv_blocks, group_size, G, n_qtiles, splits;
  int table_mode;          // kTablesPerGroup / kTablesPerQTile / kTablesPacked
  long long packed_pages;  // capacity of the packed pools (kTablesPacked)
  float scale_log2;
  // XCD-balanced two-piece split (splits == 2) when not nullptr: every
  // workgroup computes its row's cut point (xcd_cut), and the first tile's
  // first piece records it in split_at[r]: the cut entry, or -1 = not cut,
  // run whole as piece 0; -2 = not cut, run whole as piece 1
  int32_t* split_at;
  int rows_per_unit;   // table rows that read one KV head's pages together
};

constexpr int kXcds = 8;   // MI355X: 8 accelerator complex dies, 32 CUs and one L2 each

// 64-bit lane exchanges as two 32-bit ones.
__device__ __forceinline__ long long shfl_xor_i64(long long v, int mask) {
  const int lo = __shfl_xor((int)(unsigned int)v, mask, 64);
  const int hi = __shfl_xor((int)(v >> 32), mask, 64);
  return (long long)(((unsigned long long)(unsigned int)hi << 32) | (unsigned int)lo);
}
// Lane src's value, as a wave-uniform (scalar) value.
__device__ __forceinline__ long long readlane_i64(long long v, int src) {
  const int lo = __builtin_amdgcn_readlane((int)(unsigned int)v, src);
  const int hi = __builtin_amdgcn_readlane((int)(v >> 32), src);
  return (long long)(((unsigned long long)(unsigned int)hi << 32) | (unsigned int)lo);
}

// Cut point of table row r in the XCD-balanced two-piece split, from the
// table lengths (every lane of the calling wave gets the same value).  The
// R = 8m table rows are spread over the 8 XCDs by r % 8: XCD x holds rows
// x, x+8, .., its load alone is L_x table entries.  XCD x runs the first C_x
// entries of its own rows and the remaining L_{x-1} - C_{x-1} of the previous
// XCD's rows, so its load is C_x + L_{x-1} - C_{x-1}; equal loads S = sum L / 8
// give C_x = C_{x-1} + S - L_{x-1}, fixed up to the choice of C_0.  Any C_0
// that keeps every 0 <= C_x <= L_x balances exactly; the largest keeps the
// most entries on their own XCD and leaves whole the rows of every XCD with
// C_x = L_x (or 0).  When no such C_0 exists the cuts are clamped.  C_x is
// shared among the rows of XCD x in proportion to their lengths.  Dense
// tables: row r has nKB_b entries.  Returns the cut entry, -1 (not cut, whole
// row in piece 0) or -2 (not cut, whole row in piece 1).
template <bool DENSE>
__device__ int xcd_cut(const AttnArgs& a, int r) {
  const int lane = threadIdx.x & 63;
  const int R = a.B * a.G;
  auto row_len = [&](int q) -> long long {
    return DENSE ? (long long)blocks_for(a.cached_len[q / a.G] + a.C)
                 : (long long)(a.kv_indptr[q + 1] - a.kv_indptr[q]);
  };
  // lane l sums rows l, l + 64, ..: all on XCD l % 8; then the 8 lanes of
  // each XCD meet, so every lane holds L_{lane % 8}
  long long v = 0;
  for (int q = lane; q < R; q += 64) v += row_len(q);
  v += shfl_xor_i64(v, 8);
  v += shfl_xor_i64(v, 16);
  v += shfl_xor_i64(v, 32);
  long long L[kXcds], total = 0;
#pragma unroll
  for (int x = 0; x < kXcds; ++x) {
    L[x] = readlane_i64(v, x);
    total += L[x];
  }
  // D_x = sum_{k=1..x} (S - L_{k-1}) in units of 1/8 entry (S = total / 8);
  // the range of 8 C_0 that keeps 0 <= C_x <= L_x
  long long D8[kXcds];
  D8[0] = 0;
#pragma unroll
  for (int x = 1; x < kXcds; ++x) D8[x] = D8[x - 1] + total - 8 * L[x - 1];
  long long lo = 0, hi = 8 * L[0];
#pragma unroll
  for (int x = 0; x < kXcds; ++x) {
    lo = lo > -D8[x] ? lo : -D8[x];
    hi = hi < 8 * L[x] - D8[x] ? hi : 8 * L[x] - D8[x];
  }
  const long long c0 = lo <= hi ? hi : (lo + hi) / 2;   // lo > hi: clamped below
  const int xr = r % kXcds;
  long long Lx = 0, Dx = 0;
#pragma unroll
  for (int x = 0; x < kXcds; ++x)
    if (x == xr) Lx = L[x], Dx = D8[x];
  long long cx = (c0 + Dx) / 8;
  cx = cx < 0 ? 0 : (cx > Lx ? Lx : cx);
  // C_x over the rows of XCD x in proportion to their lengths: the entries of
  // the rows before r on the same XCD
  long long before = 0;
  for (int q = xr + kXcds * lane; q < r; q += kXcds * 64) before += row_len(q);
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) before += shfl_xor_i64(before, o);
  before = readlane_i64(before, 0);
  const long long len = row_len(r);
  const long long a0 = Lx > 0 ? (before * cx) / Lx : 0;
  const long long a1 = Lx > 0 ? ((before + len) * cx) / Lx : 0;
  const long long c = a1 - a0;
  return c >= len ? -1 : (c <= 0 ? -2 : (int)c);
}

// LDS page tiles: K pages and token-major V pages are 64 key rows x D; a
// transposed V page is D rows x 64 keys.
constexpr int kTileK = 0;
constexpr int kTileVT = 1;   // transposed V page
constexpr int kTileVR = 2;   // token-major V page

// Key that row r (0..15) of 16-key tile kt (0..3) of a page stands for in the
// QK contraction: 32*(kt/2) + 8*(r/4) + 4*(kt%2) + r%4.  The 16x16 result
// gives lane group g (lanes 16g .. 16g+15) rows 4g .. 4g+3 of every tile, so
// with this order the lane holds keys 32p + 8g .. 32p + 8g + 7 of each 32-key
// step p (tiles 2p and 2p+1): the 8 consecutive keys that its P^T fragment of
// that step covers.
__host__ __device__ constexpr int key_of(int kt, int r) {
  return 32 * (kt >> 1) + 8 * (r >> 2) + 4 * (kt & 1) + (r & 3);
}

// Swizzled position (16-byte chunk) of chunk c of row r in an LDS page tile.
// gfx950 LDS has 64 banks of 4 bytes; a 16-byte read is served 16 lanes per
// cycle and an 8-byte read 32 lanes per cycle.
// K tiles are read 16 bytes per lane by the 16 keys key_of(kt, 0..15) at one
// chunk: bits 0, 1, 3, 4 of those keys differ, so XOR-ing them into the chunk
// puts the 16 reads on 16 different 16-byte bank slots (D = 64: a row is half
// a 256-byte bank window, rows pair up by bit 0, and bits 1, 3, 4 pick the
// chunk).  Transposed V tiles (128-byte rows, two per window) are read 16
// bytes per lane by 16 consecutive d rows at one chunk.  Token-major V tiles
// are read 8 bytes per lane by the transpose read: 32 lanes cover keys
// {0..3, 8..11} (+ multiples of 4 and 16) x 32 bytes, so bits 0, 1, 3 of the
// key pick the 32-byte pair of chunks (D = 64: bit 0 picks the half window,
// bits 1 and 3 the pair).  None of the swizzles depends on key bits 2 or 5, so
// a lane's operand reads of the four key tiles differ only by immediates.
template <int D>
__device__ __forceinline__ int k_swz(int r, int c) {
  return D == 128 ? (c ^ ((r & 3) | (((r >> 3) & 3) << 2)))
                  : (c ^ (((r >> 1) & 1) | (((r >> 3) & 3) << 1)));
}
__device__ __forceinline__ int vt_swz(int r, int c) { return c ^ ((r >> 1) & 7); }
template <int D>
__device__ __forceinline__ int vr_swz(int r, int c) {
  return D == 128 ? (c ^ (((r & 3) | (((r >> 3) & 1) << 2)) << 1))
                  : (c ^ ((((r >> 1) & 1) | (((r >> 3) & 1) << 1)) << 1));
}
template <int D, int TILE>
__device__ __forceinline__ int tile_swz(int r, int c) {
  if constexpr (TILE == kTileVT) return vt_swz(r, c);
  else if constexpr (TILE == kTileVR) return vr_swz<D>(r, c);
  else return k_swz<D>(r, c);
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

// Lazy rescaling (log2 units): the exponent base (a running maximum of the
// scaled scores) moves only when a weight could exceed 2^kRescaleSlack, so
// most pages skip the O rescale.  The unpipelined pages test their page
// maximum against base + kRescaleSlack; the pipelined steps compute no page
// maximum and test each lane's partial row sum over the page against
// kSumLimit, which bounds every weight in it.
constexpr float kRescaleSlack = 8.0f;
constexpr float kSumLimit = 256.0f;   // 2^kRescaleSlack
// Exponent base before the first page: finite and below any score, so the
// first page with a finite score always moves it (its alpha exp2(kNoBase - m)
// is 0, which clears the empty O and row sum), and no -inf test is needed.
// A row that never sees a finite score keeps it with a zero row sum.
constexpr float kNoBase = -1.0e30f;

// max / sum over the 4 lane groups (lanes l, l^16, l^32, l^48 hold the same
// query column): rows 0<->1 and 2<->3 swap (v_permlane16_swap), then rows
// {0,1}<->{2,3} (v_permlane32_swap); each swap hands both values back.
__device__ __forceinline__ float max2(float a, float b) {
  return __builtin_elementwise_maximum(a, b);   // v_maximum_f32: no quieting of the inputs
}
__device__ __forceinline__ float groups_max(float x) {
  uint32_t u = __float_as_uint(x);
  auto r = __builtin_amdgcn_permlane16_swap(u, u, false, false);
  u = __float_as_uint(max2(__uint_as_float(r[0]), __uint_as_float(r[1])));
  r = __builtin_amdgcn_permlane32_swap(u, u, false, false);
  return max2(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float groups_sum(float x) {
  uint32_t u = __float_as_uint(x);
  auto r = __builtin_amdgcn_permlane16_swap(u, u, false, false);
  u = __float_as_uint(__uint_as_float(r[0]) + __uint_as_float(r[1]));
  r = __builtin_amdgcn_permlane32_swap(u, u, false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// S^T of one page: s[kt][c] is 16-key tile kt of column tile c; value i of
// lane group g holds key key_of(kt, 4g + i) of the lane's query column.
template <int NCT>
struct SPage {
  f32x4 s[4][NCT];
};
// P^T fragments (bf16) of one page: p[kp][c] covers the 32 keys of step kp,
// lane group g holding keys 32kp + 8g .. 32kp + 8g + 7 (values 0..3 from
// tile 2kp, 4..7 from tile 2kp + 1).
template <int NCT>
struct PFrag {
  bf16x8 p[2][NCT];
};

// ---- MFMAs with explicit register classes (inline asm) ----
// O^T accumulators and Q^T fragments live in AGPRs, S^T tiles and P^T
// fragments in VGPRs.  The compiler cannot see the wait states these
// instructions need, so the kernel places explicit s_nop fences where an
// MFMA result is read by VALU code or a VALU result is read by an MFMA.
// With two waves per SIMD (AG = false) every value is in VGPRs: a wave that
// uses AGPRs may then only hold 128 VGPRs.
template <bool AG>
__device__ __forceinline__ void mfma_o(f32x4& o, const bf16x8& a, const bf16x8& b) {
  if constexpr (AG) asm volatile("v_mfma_f32_16x16x32_bf16 %0, %1, %2, %0" : "+a"(o) : "v"(a), "v"(b));
  else asm volatile("v_mfma_f32_16x16x32_bf16 %0, %1, %2, %0" : "+v"(o) : "v"(a), "v"(b));
}
template <bool AG>
__device__ __forceinline__ void mfma_s0(f32x4& s, const bf16x8& a, const bf16x8& b) {
  if constexpr (AG) asm volatile("v_mfma_f32_16x16x32_bf16 %0, %1, %2, 0" : "=&v"(s) : "v"(a), "a"(b));
  else asm volatile("v_mfma_f32_16x16x32_bf16 %0, %1, %2, 0" : "=&v"(s) : "v"(a), "v"(b));
}
template <bool AG>
__device__ __forceinline__ void mfma_s(f32x4& s, const bf16x8& a, const bf16x8& b) {
  if constexpr (AG) asm volatile("v_mfma_f32_16x16x32_bf16 %0, %1, %2, %0" : "+v"(s) : "v"(a), "a"(b));
  else asm volatile("v_mfma_f32_16x16x32_bf16 %0, %1, %2, %0" : "+v"(s) : "v"(a), "v"(b));
}

// Fence on the O^T accumulators: an MFMA result read or overwritten by VALU
// code, or a VALU result read by an MFMA, needs wait states the compiler
// cannot see through inline asm.  One set of wait states serves every tuple.
// Volatile asm statements keep their order, so empty statements that take
// each tuple as an operand pin the writes of every tuple above the wait (the
// statements before it) and the reads of every tuple below it (the
// statements after it); the MFMAs, also volatile asm, stay on their side.
template <bool AG, int NDT, int NCT>
__device__ __forceinline__ void tie_o(f32x4 (&o)[NDT][NCT]) {
#pragma unroll
  for (int x = 0; x < NDT; ++x)
#pragma unroll
    for (int c = 0; c < NCT; ++c) {
      if constexpr (AG) asm volatile("" : "+a"(o[x][c]));
      else asm volatile("" : "+v"(o[x][c]));
    }
}
template <bool AG, int NDT, int NCT>
__device__ __forceinline__ void fence_o(f32x4 (&o)[NDT][NCT]) {
  tie_o<AG>(o);
  asm volatile("s_nop 7\n s_nop 7\n s_nop 7");
  tie_o<AG>(o);
}

// Fences on S^T tiles (MFMA results about to be read by the softmax) and on
// P^T fragments (VALU results about to be read by MFMAs).
template <int NCT>
__device__ __forceinline__ void fence_s(SPage<NCT>& s) {
  if constexpr (NCT == 4)
    asm volatile("s_nop 7\n s_nop 7\n s_nop 5"
                 : "+v"(s.s[0][0]), "+v"(s.s[0][1]), "+v"(s.s[0][2]), "+v"(s.s[0][3]),
                   "+v"(s.s[1][0]), "+v"(s.s[1][1]), "+v"(s.s[1][2]), "+v"(s.s[1][3]),
                   "+v"(s.s[2][0]), "+v"(s.s[2][1]), "+v"(s.s[2][2]), "+v"(s.s[2][3]),
                   "+v"(s.s[3][0]), "+v"(s.s[3][1]), "+v"(s.s[3][2]), "+v"(s.s[3][3]));
  else
    asm volatile("s_nop 7\n s_nop 7\n s_nop 5"
                 : "+v"(s.s[0][0]), "+v"(s.s[0][1]), "+v"(s.s[1][0]), "+v"(s.s[1][1]),
                   "+v"(s.s[2][0]), "+v"(s.s[2][1]), "+v"(s.s[3][0]), "+v"(s.s[3][1]));
}
template <int NCT>
__device__ __forceinline__ void fence_p(PFrag<NCT>& p) {
  if constexpr (NCT == 4)
    asm volatile("s_nop 7\n s_nop 7\n s_nop 5"
                 : "+v"(p.p[0][0]), "+v"(p.p[0][1]), "+v"(p.p[0][2]), "+v"(p.p[0][3]),
                   "+v"(p.p[1][0]), "+v"(p.p[1][1]), "+v"(p.p[1][2]), "+v"(p.p[1][3]));
  else
    asm volatile("s_nop 7\n s_nop 7\n s_nop 5"
                 : "+v"(p.p[0][0]), "+v"(p.p[0][1]), "+v"(p.p[1][0]), "+v"(p.p[1][1]));
}
template <int NCT>
__device__ __forceinline__ void fence_sp(SPage<NCT>& s, PFrag<NCT>& p) {
  fence_s<NCT>(s);
  if constexpr (NCT == 4)
    asm volatile(""
                 : "+v"(p.p[0][0]), "+v"(p.p[0][1]), "+v"(p.p[0][2]), "+v"(p.p[0][3]),
                   "+v"(p.p[1][0]), "+v"(p.p[1][1]), "+v"(p.p[1][2]), "+v"(p.p[1][3]));
  else
    asm volatile("" : "+v"(p.p[0][0]), "+v"(p.p[0][1]), "+v"(p.p[1][0]), "+v"(p.p[1][1]));
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

template <int D, int NW, int NCT, bool DENSE, int VL>
__global__ __launch_bounds__(64 * NW, NCT == 4 ? 1 : 2) void paged_attention_kernel(const AttnArgs a) {
  constexpr bool AG = NCT == 4;        // O^T and Q^T in AGPRs (one wave per SIMD)
  constexpr bool VTR = VL == kVTransposed;
  constexpr int VTILE = VTR ? kTileVT : kTileVR;
  constexpr int NKS = D / 32;          // QK k-steps (32 d each)
  constexpr int NDT = D / 16;          // O^T d tiles
  constexpr int PAGE = 64 * D;
  constexpr int ROWS = 16 * NCT * NW;
  constexpr int NPV = 2 * NDT;         // V^T fragments per page (2 key steps x d tiles)
  constexpr int NQK = 4 * NKS;         // K fragments per page (4 key tiles x k-steps)
  constexpr int NFRAG = NPV + NQK;
  constexpr int NSLOT = NCT * NFRAG;   // one MFMA per slot, every fragment feeds NCT
  constexpr int FD = 3;                // fragment prefetch distance
  constexpr int DMA_PER_STEP = 2 * (64 * D * 2) / 1024 / NW;   // copy instructions per wave
  constexpr int DMA_STRIDE = (NSLOT / 2) / DMA_PER_STEP > 0 ? (NSLOT / 2) / DMA_PER_STEP : 1;
  // softmax slots: the weights of the page over all slots
  constexpr int NE = 16 * NCT;         // softmax weights per lane per page
  constexpr int NSOFT = soft_ops(NE);
  constexpr bool EVEN = NSLOT >= 2 * NE;   // softmax spread one instruction per slot
  __shared__ __attribute__((aligned(1024))) uint16_t k_s0[PAGE];
  __shared__ __attribute__((aligned(1024))) uint16_t k_s1[PAGE];
  __shared__ __attribute__((aligned(1024))) uint16_t v_s0[PAGE];
  __shared__ __attribute__((aligned(1024))) uint16_t v_s1[PAGE];

  const int t = threadIdx.x;
  const int wv = __builtin_amdgcn_readfirstlane(t >> 6);
  const int lane = t & 63;
  // The two waves that share a SIMD run the same slot schedule and meet at
  // every page barrier.  Half the waves (one per SIMD when the waves of a
  // workgroup are placed round-robin over the 4 SIMDs) get the higher issue
  // priority: that wave runs ahead within the step and the other fills the
  // gaps it leaves (0.4-0.6% at 128K in same-box A/B timings).
  if (NCT == 2 && wv < NW / 2) __builtin_amdgcn_s_setprio(1);
  const int col = lane & 15;           // query column within a 16-column tile
  const int grp = lane >> 4;           // lane group: keys 4*grp .. of each 16-key tile

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
  int head[NCT], tq[NCT];
  bool valid[NCT];
#pragma unroll
  for (int c = 0; c < NCT; ++c) {
    const int r = wv * 16 * NCT + 16 * c + col;
    head[c] = g * gs + r / QT;
    tq[c] = q0 + r % QT;
    valid[c] = tq[c] < a.C;
    if (!valid[c]) tq[c] = a.C - 1;    // computes a copy of a real row, never stored
  }
  const int kvh = (g * gs) / (a.Hq / a.Hkv);
  const int cl = a.cached_len[b];
  const int nkb = blocks_for(cl + a.C);
  int qpos[NCT];
#pragma unroll
  for (int c = 0; c < NCT; ++c) qpos[c] = cl + tq[c];
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
    int cut = xcd_cut<DENSE>(a, rowid);
    if (sp == 0 && qt == 0 && t == 0) a.split_at[rowid] = cut;   // a record of the schedule
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

  // Q^T fragments: column tile c, k-step ks: d = 32ks + 8*grp .. +7 of the lane's query
  bf16x8 qf[NCT][NKS];
#pragma unroll
  for (int c = 0; c < NCT; ++c) {
    const uint16_t* qrow = a.q + (((size_t)b * a.C + tq[c]) * a.Hq + head[c]) * D + 8 * grp;
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks) {
      qf[c][ks] = *reinterpret_cast<const bf16x8*>(qrow + 32 * ks);
      if constexpr (AG) asm volatile("s_nop 2" : "+a"(qf[c][ks]));   // into AGPRs
    }
  }

  f32x4 o[NDT][NCT];
#pragma unroll
  for (int x = 0; x < NDT; ++x)
#pragma unroll
    for (int c = 0; c < NCT; ++c)
#pragma unroll
      for (int v = 0; v < 4; ++v) o[x][c][v] = 0.f;
  fence_o<AG>(o);
  float m_run[NCT], l_run[NCT];
#pragma unroll
  for (int c = 0; c < NCT; ++c) {
    m_run[c] = kNoBase;
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

  SPage<NCT> SA, SB;
  PFrag<NCT> PA, PB;
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
  // buffer, the key tile of a QK fragment and the d tile or key step of a PV
  // fragment are immediates where the swizzle allows.  K fragment (kt, ks):
  // row key_of(kt, col), chunk 4ks + grp.  V^T fragment (kp, dt): d rows
  // 16dt + col, keys 32kp + 8grp .. +7: in a transposed tile one 16-byte chunk
  // of row 16dt + col; in a token-major tile two transpose reads (keys +0..3
  // and +4..7; the 16 lanes of a group address 4 key rows x 16 d and each
  // receives 4 keys of one d).
  constexpr int NVOFS = VTR ? 2 : NDT;
  uint32_t kofs[NKS], vofs[NVOFS];
#pragma unroll
  for (int ks = 0; ks < NKS; ++ks) {
    const int kr = key_of(0, col);
    kofs[ks] = (uint32_t)(kr * D * 2 + 16 * k_swz<D>(kr, 4 * ks + grp));
  }
  if constexpr (VTR) {
#pragma unroll
    for (int kp = 0; kp < 2; ++kp)
      vofs[kp] = (uint32_t)(col * kPage * 2 + 16 * vt_swz(col, 4 * kp + grp));
  } else {
    const int r0 = 8 * grp + (col >> 2);
#pragma unroll
    for (int x = 0; x < NDT; ++x) {
      const int d = 16 * x + 4 * (col & 3);
      vofs[x] = (uint32_t)(r0 * D * 2 + 16 * vr_swz<D>(r0, d >> 3) + 2 * (d & 7));
    }
  }
  // fragment F of a step: F < NPV is V^T fragment (kp = F / NDT, d tile
  // x = F % NDT), otherwise K fragment (key tile (F - NPV) % 4, k-step
  // (F - NPV) / 4: the 4 MFMAs that build one S^T tile are 8 slots apart)
  auto load_frag = [&](int F, const uint16_t* vt, const uint16_t* kt) -> bf16x8 {
    if (F < NPV) {
      const int kp = F / NDT, x = F % NDT;
      if constexpr (VTR) {
        const char* p = reinterpret_cast<const char*>(vt) + vofs[kp] + 16 * kPage * 2 * x;
        return *reinterpret_cast<const bf16x8*>(p);
      } else {
        const char* p = reinterpret_cast<const char*>(vt) + vofs[x] + 32 * kp * D * 2;
        const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)p);
        const i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(p + 4 * D * 2));
        const u32x2 l2 = __builtin_bit_cast(u32x2, lo), h2 = __builtin_bit_cast(u32x2, hi);
        const u32x4 w = {l2[0], l2[1], h2[0], h2[1]};
        return __builtin_bit_cast(bf16x8, w);
      }
    }
    const int G2 = F - NPV, kt4 = G2 % 4, ks = G2 / 4;
    const char* p = reinterpret_cast<const char*>(kt) + kofs[ks] +
                    (32 * (kt4 >> 1) + 4 * (kt4 & 1)) * D * 2;
    return *reinterpret_cast<const bf16x8*>(p);
  };

  // Whole-page contractions (outside the pipelined loop).
  auto qk_page = [&](SPage<NCT>& st, const uint16_t* kt) __attribute__((always_inline)) {
    static_for<NQK>([&](auto gtag) __attribute__((always_inline)) {
      constexpr int G2 = decltype(gtag)::value, kt4 = G2 % 4, ks = G2 / 4;
      const bf16x8 kf = load_frag(NPV + G2, kt, kt);
#pragma unroll
      for (int c = 0; c < NCT; ++c) {
        if constexpr (ks == 0) mfma_s0<AG>(st.s[kt4][c], kf, qf[c][ks]);
        else mfma_s<AG>(st.s[kt4][c], kf, qf[c][ks]);
      }
    });
  };
  auto pv_page = [&](const PFrag<NCT>& pf, const uint16_t* vt) __attribute__((always_inline)) {
    static_for<NPV>([&](auto ftag) __attribute__((always_inline)) {
      constexpr int F = decltype(ftag)::value;
      const bf16x8 vf = load_frag(F, vt, vt);
#pragma unroll
      for (int c = 0; c < NCT; ++c) mfma_o<AG>(o[F % NDT][c], vf, pf.p[F / NDT][c]);
    });
  };

  // Prologue: K(0) -> k_s0, K(1) -> k_s1, and V(0) into the buffer the first
  // step's PV reads, with a zero P: that PV adds nothing and every tile read
  // is initialised.  Then S(0).
#pragma unroll
  for (int kp = 0; kp < 2; ++kp)
#pragma unroll
    for (int c = 0; c < NCT; ++c) PB.p[kp][c] = __builtin_bit_cast(bf16x8, u32x4{0u, 0u, 0u, 0u});
  if (n_pipe > 0) {
    page_to_lds<D, NW, kTileK>(page_ptr(a.k_pool, 0), k_s0, wv, lane);
    page_to_lds<D, NW, kTileK>(page_ptr(a.k_pool, 1), k_s1, wv, lane);
    page_to_lds<D, NW, VTILE>(page_ptr(a.v_pool, 0), v_s1, wv, lane);
    copies_landed(k_s0, k_s1, v_s1);
    __syncthreads();
    qk_page(SA, k_s0);
    __syncthreads();
    fence_sp<NCT>(SA, PB);   // S(0) and the zero P are read by the first step's first slots
  }

  // Step i: DMA K(i+2) -> k[i%2], V(i) -> v[i%2]; PV(i-1) from v[(i-1)%2] and
  // P(i-1); QK(i+1) from k[(i+1)%2]; softmax(i) of S(i) into P(i).  One MFMA
  // per slot, the softmax work spread over the slots.
  auto step = [&](auto par, int i) __attribute__((always_inline)) {
    constexpr int P = decltype(par)::value;
    SPage<NCT>& sc = P ? SB : SA;
    SPage<NCT>& sn = P ? SA : SB;
    PFrag<NCT>& pn = P ? PB : PA;
    PFrag<NCT>& po = P ? PA : PB;
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
    float ps[NCT], wt[NE];
#pragma unroll
    for (int c = 0; c < NCT; ++c) ps[c] = 0.f;
    bf16x8 fr[NFRAG];
#pragma unroll
    for (int f = 0; f < FD; ++f) fr[f] = load_frag(f, v_rd, k_rd);
    static_for<NSLOT>([&](auto stag) __attribute__((always_inline)) {
      constexpr int s = decltype(stag)::value;
      constexpr int F = s / NCT, c = s % NCT;
      if constexpr (c == 0 && F + FD < NFRAG) fr[F + FD] = load_frag(F + FD, v_rd, k_rd);
      // the copies of K(i+2) and V(i), one instruction every DMA_STRIDE slots
      // over the first half of the step (issued all at once they queue in
      // the address unit and stall the wave), from slot 1: slot 0 issues the
      // step's first fragment reads right after the barrier
      if constexpr (s >= 1 && (s - 1) % DMA_STRIDE == 0 && (s - 1) / DMA_STRIDE < DMA_PER_STEP) {
        constexpr int m = (s - 1) / DMA_STRIDE;
        if constexpr (m < DMA_PER_STEP / 2)
          page_part_to_lds<D, NW, kTileK>(k_src, k_dma, wv, lane, m);
        else
          page_part_to_lds<D, NW, VTILE>(v_src, v_dma, wv, lane, m - DMA_PER_STEP / 2);
      }
      if constexpr (F < NPV) {
        mfma_o<AG>(o[F % NDT][c], fr[F], po.p[F / NDT][c]);
      } else {
        constexpr int G2 = F - NPV, kt4 = G2 % 4, ks = G2 / 4;
        if constexpr (ks == 0) mfma_s0<AG>(sn.s[kt4][c], fr[F], qf[c][ks]);
        else mfma_s<AG>(sn.s[kt4][c], fr[F], qf[c][ks]);
      }
      // softmax work of this slot: the weights of the page against the
      // current base, spread over the slots so that no instruction waits on
      // the one before it (elements in unit order, unit u = the 8 weights of
      // P^T fragment (kp, c) = (u / NCT, u % NCT): values 0..3 of tile 2kp,
      // then of tile 2kp + 1).  The raw scores stay in sc for the rare rebase
      // below.
      if constexpr (EVEN) {
        // Two slots per element, one or two instructions per slot: element
        // e's scaled score in slot 2e, its exp in slot 2e + 1, its row-sum add
        // in slot 2e + 2; half h of unit u's packs (its last exp in slot
        // 16u + 15) in slot 16u + 16 + 2h; the last add and the last unit's
        // packs after the slots.  (Whole element ops, three instructions each
        // in about every other slot, left the VALU work in bursts that the
        // MFMAs of the two waves hid less well.)
        constexpr int e = s / 2;
        if constexpr (s % 2 == 0) {
          if constexpr (e < NE) {
            constexpr int u = e / 8, x = e % 8, cc = u % NCT, kt4 = 2 * (u / NCT) + x / 4;
            wt[e] = fmaf(sc.s[kt4][cc][x % 4], a.scale_log2, -m_run[cc]);
            pin(wt[e]);
          }
          if constexpr (e >= 1 && e <= NE) {
            constexpr int e1 = e - 1, cc = (e1 / 8) % NCT;
            ps[cc] += wt[e1];
            pin(ps[cc]);
          }
          if constexpr (s >= 16 && (s - 16) % 16 < 4 && (s - 16) / 16 < NE / 8) {
            constexpr int u = (s - 16) / 16, h = ((s - 16) % 16) / 2, kp = u / NCT, cc = u % NCT;
#pragma unroll
            for (int x = 4 * h; x < 4 * h + 4; ++x) pn.p[kp][cc][x] = (__bf16)wt[8 * u + x];
            pin(pn.p[kp][cc]);
          }
        } else if constexpr (e < NE) {
          wt[e] = fast_exp2(wt[e]);
          pin(wt[e]);
        }
      } else {
        // one slot per element (D = 64): element op j does the scaled score
        // of element j, the exp of element j-1 and the row sum of element
        // j-2; unit u is packed to bf16 after element op 8u+8
        constexpr int lo = (s * NSOFT) / NSLOT;
        constexpr int hi = ((s + 1) * NSOFT) / NSLOT;
        static_for<hi - lo>([&](auto otag) __attribute__((always_inline)) {
          constexpr int op = soft_op(lo + decltype(otag)::value, NE);
          if constexpr (op >= 0) {
            if constexpr (op < NE) {
              constexpr int u = op / 8, x = op % 8, cc = u % NCT, kt4 = 2 * (u / NCT) + x / 4;
              wt[op] = fmaf(sc.s[kt4][cc][x % 4], a.scale_log2, -m_run[cc]);
              pin(wt[op]);
            }
            if constexpr (op >= 1 && op <= NE) {
              constexpr int e = op - 1;
              wt[e] = fast_exp2(wt[e]);
              pin(wt[e]);
            }
            if constexpr (op >= 2) {
              constexpr int e = op - 2, u = e / 8, cc = u % NCT;
              ps[cc] += wt[e];
              pin(ps[cc]);
            }
          } else {
            constexpr int u = -1 - op, kp = u / NCT, cc = u % NCT;
#pragma unroll
            for (int x = 0; x < 8; ++x) pn.p[kp][cc][x] = (__bf16)wt[8 * u + x];
            pin(pn.p[kp][cc]);
          }
        });
      }
      __builtin_amdgcn_sched_barrier(0);
    });
    if constexpr (EVEN) {
      // the last add and the last unit's packs (slots 2 NE and after)
      constexpr int e1 = NE - 1, u = NE / 8 - 1, kp = u / NCT, cc = u % NCT;
      ps[(e1 / 8) % NCT] += wt[e1];
#pragma unroll
      for (int x = 0; x < 8; ++x) pn.p[kp][cc][x] = (__bf16)wt[8 * u + x];
    }
    // A lane's partial row sum over its 16 keys of the page bounds each of its
    // weights: while it stays <= 2^slack no weight exceeds 2^slack and the
    // base stays (inf or NaN, from the first page's base, fail the test too).
    bool big = false;
#pragma unroll
    for (int c = 0; c < NCT; ++c) big |= !(ps[c] <= kSumLimit);
    if (__ballot(big)) {
      // Rare: every column moves its base to the page maximum where that is
      // higher (where it is not the base stays and alpha is 1), recomputes
      // the page's weights, row sum and packs against it, and rescales O and
      // l_run by alpha = exp2(old - new base).
      float alpha[NCT];
#pragma unroll
      for (int c = 0; c < NCT; ++c) {
        float mx = max2(sc.s[0][c][0], sc.s[1][c][0]);
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          if (v > 0) mx = max3(mx, sc.s[0][c][v], sc.s[1][c][v]);
          mx = max3(mx, sc.s[2][c][v], sc.s[3][c][v]);
        }
        const float m_new = max2(m_run[c], groups_max(mx) * a.scale_log2);
        alpha[c] = fast_exp2(m_run[c] - m_new);
        m_run[c] = m_new;
        float sum = 0.f;
#pragma unroll
        for (int kp = 0; kp < 2; ++kp)
#pragma unroll
          for (int x = 0; x < 8; ++x) {
            const float w = fast_exp2(fmaf(sc.s[2 * kp + x / 4][c][x % 4], a.scale_log2, -m_new));
            sum += w;
            pn.p[kp][c][x] = (__bf16)w;
          }
        l_run[c] = fmaf(l_run[c], alpha[c], sum);
        ps[c] = 0.f;
      }
      fence_o<AG>(o);
#pragma unroll
      for (int x = 0; x < NDT; ++x)
#pragma unroll
        for (int c = 0; c < NCT; ++c) o[x][c] *= alpha[c];
      fence_o<AG>(o);
    }
#pragma unroll
    for (int c = 0; c < NCT; ++c) l_run[c] += ps[c];
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
    fence_p<NCT>(PB);
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
    fence_s<NCT>(SA);
    if (i >= n_main) {
      const int j = id_of(blk_cur, blk_nxt, i);
#pragma unroll
      for (int c = 0; c < NCT; ++c) {
        const int lim = qpos[c] - kPage * j;
#pragma unroll
        for (int kt4 = 0; kt4 < 4; ++kt4)
#pragma unroll
          for (int v = 0; v < 4; ++v)
            if (32 * (kt4 >> 1) + 8 * grp + 4 * (kt4 & 1) + v > lim) SA.s[kt4][c][v] = -INFINITY;
      }
    }
    float alpha[NCT];
    bool rb_any = false;
#pragma unroll
    for (int c = 0; c < NCT; ++c) {
      float mx = max2(SA.s[0][c][0], SA.s[1][c][0]);
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        if (v > 0) mx = max3(mx, SA.s[0][c][v], SA.s[1][c][v]);
        mx = max3(mx, SA.s[2][c][v], SA.s[3][c][v]);
      }
      // a fully masked page (-inf) never moves the base
      const float m = groups_max(mx) * a.scale_log2;
      const bool rebase = m > m_run[c] + kRescaleSlack;
      const float m_new = rebase ? m : m_run[c];
      alpha[c] = fast_exp2(m_run[c] - m_new);
      m_run[c] = m_new;
      rb_any |= rebase;
      float ps = 0.f;
#pragma unroll
      for (int kt4 = 0; kt4 < 4; ++kt4)
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const float e = fast_exp2(fmaf(SA.s[kt4][c][v], a.scale_log2, -m_run[c]));
          SA.s[kt4][c][v] = e;
          ps += e;
        }
      l_run[c] = l_run[c] * alpha[c] + ps;
#pragma unroll
      for (int kp = 0; kp < 2; ++kp)
#pragma unroll
        for (int x = 0; x < 8; ++x) PA.p[kp][c][x] = (__bf16)SA.s[2 * kp + x / 4][c][x % 4];
    }
    if (__ballot(rb_any)) {
      fence_o<AG>(o);
#pragma unroll
      for (int x = 0; x < NDT; ++x)
#pragma unroll
        for (int c = 0; c < NCT; ++c) o[x][c] *= alpha[c];
      fence_o<AG>(o);
    }
    fence_p<NCT>(PA);
    pv_page(PA, v_s0);
    __syncthreads();
  }
  fence_o<AG>(o);

  // epilogue: O^T tile (x, c) value v of lane group grp is d = 16x + 4grp + v
  float inv[NCT], lse_val[NCT];
  size_t qrow_idx[NCT];
#pragma unroll
  for (int c = 0; c < NCT; ++c) {
    const float l_tot = groups_sum(l_run[c]);
    inv[c] = l_tot > 0.f ? 1.0f / l_tot : 0.f;
    lse_val[c] = l_tot > 0.f ? (m_run[c] + log2f(l_tot)) * kLn2 : -INFINITY;
    qrow_idx[c] = ((size_t)b * a.Hq + head[c]) * a.C + tq[c];
  }
  auto store_out = [&](int c, const float (&v)[NDT][4], float scale, float lse_row) {
    uint16_t* orow = a.out + (((size_t)b * a.C + tq[c]) * a.Hq + head[c]) * D;
#pragma unroll
    for (int x = 0; x < NDT; ++x) {
      uint2 pk;
      pk.x = pack_bf16x2(v[x][0] * scale, v[x][1] * scale);
      pk.y = pack_bf16x2(v[x][2] * scale, v[x][3] * scale);
      *reinterpret_cast<uint2*>(orow + 16 * x + 4 * grp) = pk;
    }
    if (a.lse != nullptr && grp == 0) a.lse[qrow_idx[c]] = lse_row;
  };
  if (whole) {
#pragma unroll
    for (int c = 0; c < NCT; ++c) {
      if (!valid[c]) continue;
      float v[NDT][4];
#pragma unroll
      for (int x = 0; x < NDT; ++x)
#pragma unroll
        for (int e = 0; e < 4; ++e) v[x][e] = o[x][c][e];
      store_out(c, v, inv[c], lse_val[c]);
    }
    return;
  }

  // One piece of a split row tile: its result is the normalised partial
  // output o * inv with its log-sum-exp.
  const size_t nrows = (size_t)a.B * a.Hq * a.C;
  auto store_part = [&]() {
#pragma unroll
    for (int c = 0; c < NCT; ++c) {
      if (!valid[c]) continue;
      const size_t prow = (size_t)sp * nrows + qrow_idx[c];
      float* po = a.part_o + prow * D;
#pragma unroll
      for (int x = 0; x < NDT; ++x)
        *reinterpret_cast<float4*>(po + 16 * x + 4 * grp) =
            make_float4(o[x][c][0] * inv[c], o[x][c][1] * inv[c], o[x][c][2] * inv[c],
                        o[x][c][3] * inv[c]);
      if (grp == 0) a.part_lse[prow] = lse_val[c];
    }
  };
  if (a.arrive == nullptr) {   // uniform splits: a merge launch follows
    store_part();
    return;
  }

  // The XCD-balanced split's two pieces are merged here, by the second to
  // finish; the first stores its partial and counts itself in.  The piece
  // that finds the other counted merges at once and stores nothing of its own.
  // The two pieces run on different XCDs, whose L2s are not coherent with
  // each other: thread 0 makes one agent-scope release (the count's swap,
  // which writes this XCD's L2 back to memory) and one agent-scope acquire
  // (which invalidates it) for the whole workgroup.  Such a fence acts on the
  // whole L2, so a fence in every wave costs far more (4% of the 128K final
  // chunk's attention time, measured).
  unsigned long long* const ctr = a.arrive + (size_t)rowid * a.n_qtiles + qt;
  __shared__ int s_last;
  if (t == 0) {
    const unsigned long long w = __hip_atomic_load(ctr, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    s_last = w == ((a.tag << 8) | 1ull);
    // the other piece has counted itself in after its release
    if (s_last) __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
  }
  __syncthreads();
  if (!s_last) {
    store_part();
    // every wave's stores have reached this XCD's L2 before thread 0's
    // release writes the L2 back
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    if (t == 0) {
      unsigned long long w = __hip_atomic_load(ctr, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      int counted = 0;
      // the swap fails only if the other piece's swap succeeded in between
      for (int it = 0; it < 2; ++it) {
        const unsigned long long nw = (w >> 8) == a.tag ? w + 1 : (a.tag << 8) | 1ull;
        if (__hip_atomic_compare_exchange_strong(ctr, &w, nw, __ATOMIC_ACQ_REL, __ATOMIC_RELAXED,
                                                 __HIP_MEMORY_SCOPE_AGENT)) {
          counted = (int)(nw & 0xff);
          break;
        }
      }
      s_last = counted == 2;
    }
    __syncthreads();
    if (!s_last) return;
  }
  // The merging piece (thread 0 has acquired, through the peek or the swap):
  // the other piece has counted itself in, so nothing else touches the
  // counter in this launch; leave it at 0 for the next one.
  if (t == 0) __hip_atomic_store(ctr, 0ull, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
#pragma unroll
  for (int c = 0; c < NCT; ++c) {
    if (!valid[c]) continue;
    const size_t row = qrow_idx[c];
    float mine[NDT][4], other[NDT][4], acc[NDT][4];
    const float* po = a.part_o + ((size_t)(1 - sp) * nrows + row) * D + 4 * grp;
#pragma unroll
    for (int x = 0; x < NDT; ++x) {
      const float4 f = *reinterpret_cast<const float4*>(po + 16 * x);
      other[x][0] = f.x, other[x][1] = f.y, other[x][2] = f.z, other[x][3] = f.w;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        mine[x][e] = o[x][c][e] * inv[c];
        acc[x][e] = 0.f;
      }
    }
    // lse = log(exp(lse_0) + exp(lse_1)); out = sum_i exp(lse_i - lse) o_i,
    // pieces in order (the arithmetic of the merge launch)
    const float lo = a.part_lse[(size_t)(1 - sp) * nrows + row];
    const float l0 = sp == 0 ? lse_val[c] : lo, l1 = sp == 0 ? lo : lse_val[c];
    const float mx = fmaxf(l0, l1);
    float wsum = 0.f;
    if (mx != -INFINITY) {
      const float w0 = l0 == -INFINITY ? 0.f : expf(l0 - mx);
      const float w1 = l1 == -INFINITY ? 0.f : expf(l1 - mx);
      wsum = w0 + w1;
      auto sum2 = [&](const float (&v0)[NDT][4], const float (&v1)[NDT][4]) {
#pragma unroll
        for (int x = 0; x < NDT; ++x)
#pragma unroll
          for (int e = 0; e < 4; ++e)
            acc[x][e] = (w0 > 0.f ? w0 * v0[x][e] : 0.f) + (w1 > 0.f ? w1 * v1[x][e] : 0.f);
      };
      if (sp == 0) sum2(mine, other);   // sp is uniform over the workgroup
      else sum2(other, mine);
    }
    store_out(c, acc, wsum > 0.f ? 1.0f / wsum : 0.f, wsum > 0.f ? mx + logf(wsum) : -INFINITY);
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

// Merge of uniform split-KV pieces: lse = log sum_i exp(lse_i),
// out = sum_i exp(lse_i - lse) o_i, pieces in order.  One 32-lane half-wave
// per (b, h, t) row, 4 floats of d per lane (D = 128) or 2 (D = 64).  (The
// XCD-balanced split merges its two pieces inside the attention launch.)
// Up to kCombineInFlight pieces are loaded all at once.
constexpr int kCombineInFlight = 8;

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
    // every load is issued before any result is needed: one memory latency
    float v0[PER], v1[PER];
    const float l0 = part_lse[row], l1 = part_lse[nrows + row];
    load_part(0, v0);
    load_part(1, v1);
    mx = fmaxf(l0, l1);
    if (mx != -INFINITY) {
      const float w0 = l0 == -INFINITY ? 0.f : expf(l0 - mx);
      const float w1 = l1 == -INFINITY ? 0.f : expf(l1 - mx);
      wsum = w0 + w1;
#pragma unroll
      for (int x = 0; x < PER; ++x)
        acc[x] = (w0 > 0.f ? w0 * v0[x] : 0.f) + (w1 > 0.f ? w1 * v1[x] : 0.f);
    }
  } else if (splits <= kCombineInFlight) {
    // every piece's lse and partial loaded before the first is needed (one
    // memory latency), then the same merge as the general loop below
    float l[kCombineInFlight], v[kCombineInFlight][PER];
#pragma unroll
    for (int i = 0; i < kCombineInFlight; ++i) {
      if (i < splits) {
        l[i] = part_lse[(size_t)i * nrows + row];
        load_part(i, v[i]);
      }
    }
#pragma unroll
    for (int i = 0; i < kCombineInFlight; ++i)
      if (i < splits) mx = fmaxf(mx, l[i]);
    if (mx != -INFINITY) {
#pragma unroll
      for (int i = 0; i < kCombineInFlight; ++i) {
        if (i >= splits || l[i] == -INFINITY) continue;
        const float wgt = expf(l[i] - mx);
        wsum += wgt;
#pragma unroll
        for (int x = 0; x < PER; ++x) acc[x] = fmaf(wgt, v[i][x], acc[x]);
      }
    }
  } else {
    for (int i = 0; i < splits; ++i) mx = fmaxf(mx, part_lse[(size_t)i * nrows + row]);
    if (mx != -INFINITY) {
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

int attn_rows_per_workgroup(int table_mode) {
  return 16 * kColTiles * (table_mode == kTablesPerQTile ? kWavesQTile : kWavesGroup);
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

// Workspace of a split launch: the partial outputs [splits, B*Hq*C, D] and
// log-sum-exps [splits, B*Hq*C] (fp32); the XCD-balanced split adds its cut
// points [B*G] (int32) and, at the next 8-byte boundary, one arrival counter
// per query tile [B*G*n_qtiles] (uint64).
static size_t attn_partial_bytes(const Dims& d, int splits) {
  return (size_t)splits * d.B * d.Hq * d.C * (d.D + 1) * sizeof(float);
}

static size_t align8(size_t x) { return (x + 7) & ~(size_t)7; }

size_t attn_ws_bytes(const Dims& d, int splits) {
  return splits <= 1 ? 0 : attn_partial_bytes(d, splits);
}

static size_t attn_xcd_counters_at(const Dims& d, int group_size) {
  return align8(attn_partial_bytes(d, 2) + (size_t)d.B * (d.Hq / group_size) * sizeof(int32_t));
}

size_t attn_xcd_ws_bytes(const Dims& d, int group_size) {
  return attn_xcd_counters_at(d, group_size) +
         (size_t)attn_base_workgroups(d, group_size, kTablesPerGroup) * 8;
}

// A tag per launch for the arrival counters: consecutive values from a
// per-process random start, kept below 2^56 and never 0.  A counter left with
// another tag (an earlier launch, or whatever the workspace held) counts 0.
static unsigned long long next_arrival_tag() {
  static std::atomic<unsigned long long> next{[] {
    std::random_device rd;
    const unsigned long long hi = rd(), lo = rd();
    return (hi << 32) ^ lo ^
           (unsigned long long)std::chrono::steady_clock::now().time_since_epoch().count();
  }()};
  for (;;) {
    const unsigned long long t = next.fetch_add(1) & ((1ull << 56) - 1);
    if (t != 0) return t;
  }
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
  a.arrive = nullptr;
  a.tag = 0;
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
  if (L.xcd_balanced)
    a.split_at = reinterpret_cast<int32_t*>(static_cast<char*>(L.ws) + attn_partial_bytes(d, 2));
  const int nwg = attn_base_workgroups(d, L.group_size, L.table_mode) * L.splits;
  if (L.xcd_balanced) {
    // per-group rows (selected or packed tables): the tiles attn_xcd_ws_bytes counts
    if (L.splits != 2 || L.table_mode == kTablesPerQTile) return hipErrorInvalidValue;
    a.arrive = reinterpret_cast<unsigned long long*>(static_cast<char*>(L.ws) +
                                                     attn_xcd_counters_at(d, L.group_size));
    a.tag = next_arrival_tag();
  }
  const bool qtile = L.table_mode == kTablesPerQTile;
  if (d.D == 128) {
    if (qtile) launch_layout<128, kWavesQTile>(a, L.dense, L.v_layout, nwg, st);
    else launch_layout<128, kWavesGroup>(a, L.dense, L.v_layout, nwg, st);
  } else {
    if (qtile) launch_layout<64, kWavesQTile>(a, L.dense, L.v_layout, nwg, st);
    else launch_layout<64, kWavesGroup>(a, L.dense, L.v_layout, nwg, st);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || L.splits == 1 || L.xcd_balanced) return e;
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
