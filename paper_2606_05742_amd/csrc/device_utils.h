// Wave64 helpers used by the gfx950 kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace adapld {

constexpr int kWave = 64;

__device__ __forceinline__ int lane_id() { return threadIdx.x & (kWave - 1); }

// Lanes below the calling lane, as a 64-bit mask.
__device__ __forceinline__ uint64_t lanes_below() {
  const int l = lane_id();
  return l == 0 ? 0ull : (~0ull >> (64 - l));
}

__device__ __forceinline__ int wave_max_i32(int v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v = max(v, __shfl_xor(v, off, kWave));
  return v;
}

// Butterfly sum: every lane ends with the same value, and the order of the
// additions depends only on the lane layout, so equal inputs give equal sums.
__device__ __forceinline__ float wave_sum_f32(float v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off, kWave);
  return v;
}

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// fp32 -> bf16 bits, round to nearest even (finite inputs).
__device__ __forceinline__ uint32_t f32_to_bf16_bits(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7fffu + ((u >> 16) & 1u);
  return u >> 16;
}

// Ranking key of a scored row: larger key = higher score, then lower position.
// High word: the float's bits mapped to an unsigned order; low word: ~pos.
__device__ __forceinline__ uint64_t rank_key(float score, int pos) {
  uint32_t u = __float_as_uint(score);
  u = (u & 0x80000000u) ? ~u : (u | 0x80000000u);
  return ((uint64_t)u << 32) | (uint64_t)(0xffffffffu - (uint32_t)pos);
}
__device__ __forceinline__ int key_pos(uint64_t key) {
  return (int)(0xffffffffu - (uint32_t)(key & 0xffffffffu));
}
__device__ __forceinline__ float key_score(uint64_t key) {
  uint32_t u = (uint32_t)(key >> 32);
  u = (u & 0x80000000u) ? (u & 0x7fffffffu) : ~u;
  return __uint_as_float(u);
}

__device__ __forceinline__ uint64_t shfl_u64(uint64_t v, int src) {
  uint32_t lo = __shfl((uint32_t)v, src, kWave);
  uint32_t hi = __shfl((uint32_t)(v >> 32), src, kWave);
  return ((uint64_t)hi << 32) | lo;
}
__device__ __forceinline__ uint64_t shfl_xor_u64(uint64_t v, int m) {
  uint32_t lo = __shfl_xor((uint32_t)v, m, kWave);
  uint32_t hi = __shfl_xor((uint32_t)(v >> 32), m, kWave);
  return ((uint64_t)hi << 32) | lo;
}
__device__ __forceinline__ uint64_t shfl_up_u64(uint64_t v, int d) {
  uint32_t lo = __shfl_up((uint32_t)v, d, kWave);
  uint32_t hi = __shfl_up((uint32_t)(v >> 32), d, kWave);
  return ((uint64_t)hi << 32) | lo;
}

// A wave-wide top list: lane i holds the i-th largest key (0 = empty slot).
// Insert one key that every lane holds (uniform control flow).
__device__ __forceinline__ void topk_insert(uint64_t& mine, uint64_t key, int k) {
  const int lane = lane_id();
  const uint64_t last = shfl_u64(mine, k - 1);
  if (key <= last) return;                         // uniform: key is wave-uniform
  const uint64_t above = __ballot(lane < k && mine > key);
  const int p = __popcll(above);                   // insertion slot
  const uint64_t prev = shfl_up_u64(mine, 1);
  if (lane < k && lane > p) mine = prev;
  if (lane == p) mine = key;
}

// Merge two wave-wide lists sorted descending (64 slots each, empty = 0):
// the result holds the 64 largest of both, sorted descending.  The elementwise
// max against the reversed partner list is bitonic; half-cleaners sort it.
__device__ __forceinline__ uint64_t topk_merge(uint64_t mine, uint64_t other) {
  const int lane = lane_id();
  uint64_t rev = shfl_u64(other, 63 - lane);
  uint64_t c = mine > rev ? mine : rev;
#pragma unroll
  for (int s = 32; s >= 1; s >>= 1) {
    uint64_t p = shfl_xor_u64(c, s);
    const bool low = (lane & s) == 0;
    c = low ? (c > p ? c : p) : (c < p ? c : p);
  }
  return c;
}

}  // namespace adapld
