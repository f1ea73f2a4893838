// Device-side helpers shared by the gfx950 kernels of libcompactattn.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ca {

constexpr int kWave = 64;          // CDNA wavefront
constexpr int kPage = 64;          // tokens per KV block / page
constexpr int kMaxKvBlocks = 16384;

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ float bf16_bits_to_float(uint32_t b) {
  return __uint_as_float(b << 16);
}

// Low / high bf16 of a packed 32-bit word, widened exactly.
__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// float -> bf16 bits, round to nearest even (v_cvt_pk_bf16_f32 on gfx950).
__device__ __forceinline__ uint16_t float_to_bf16_bits(float f) {
  __bf16 h = (__bf16)f;
  return __builtin_bit_cast(uint16_t, h);
}

__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  return (uint32_t)float_to_bf16_bits(lo) | ((uint32_t)float_to_bf16_bits(hi) << 16);
}

// Blocks holding at least one of `len` tokens (a sequence's last block may be
// partial).
__host__ __device__ __forceinline__ int blocks_for(int len) { return (len + kPage - 1) / kPage; }

// One past the last chunk-causal block of Q-block i: the block that holds the
// Q-block's last query (chunk token t sits at position cached_len + t; the
// last Q-block of a chunk may hold fewer than q_block queries).
__host__ __device__ __forceinline__ int causal_block_end(int cached_len, int C, int i,
                                                         int q_block) {
  const int last = (i + 1) * q_block < C ? (i + 1) * q_block - 1 : C - 1;
  return (cached_len + last) / kPage + 1;
}

__device__ __forceinline__ int lane_id() { return __lane_id(); }

template <typename T>
__device__ __forceinline__ T wave_sum(T v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, kWave);
  return v;
}

// Inclusive prefix sum across the 64 lanes of a wave.
__device__ __forceinline__ int wave_inclusive_scan(int v) {
  const int l = lane_id();
#pragma unroll
  for (int o = 1; o < kWave; o <<= 1) {
    int t = __shfl_up(v, o, kWave);
    if (l >= o) v += t;
  }
  return v;
}

// Number of set ballot bits in lanes below this one.
__device__ __forceinline__ int lanes_below(uint64_t ballot) {
  const int l = lane_id();
  const uint64_t below = (l == 0) ? 0ull : (~0ull >> (64 - l));
  return __popcll(ballot & below);
}

}  // namespace ca
