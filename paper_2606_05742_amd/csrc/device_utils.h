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

// Sum over the wave without LDS traffic: DPP butterflies inside each row of 16
// lanes (swap pairs, swap quads, half-row mirror, row mirror), then the four
// row sums combined through scalar reads.  The order of additions is fixed,
// so equal inputs give bit-equal sums; every lane returns the total.
template <int CTRL>
__device__ __forceinline__ float dpp_f32(float v) {
  return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), CTRL, 0xf, 0xf, false));
}
__device__ __forceinline__ float wave_sum_dpp(float v) {
  v += dpp_f32<0xb1>(v);   // quad_perm [1,0,3,2]
  v += dpp_f32<0x4e>(v);   // quad_perm [2,3,0,1]
  v += dpp_f32<0x141>(v);  // row_half_mirror
  v += dpp_f32<0x140>(v);  // row_mirror
  const float r0 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 0));
  const float r1 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 16));
  const float r2 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 32));
  const float r3 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 48));
  return (r0 + r1) + (r2 + r3);
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

// Sort a wave-wide list of 64 keys descending (bitonic network).
__device__ __forceinline__ uint64_t bitonic_sort_desc(uint64_t v) {
  const int lane = lane_id();
#pragma unroll
  for (int k = 2; k <= kWave; k <<= 1) {
#pragma unroll
    for (int j = k >> 1; j > 0; j >>= 1) {
      const uint64_t p = shfl_xor_u64(v, j);
      const bool keep_max = ((lane & j) == 0) == ((lane & k) == 0);
      v = keep_max ? (v > p ? v : p) : (v < p ? v : p);
    }
  }
  return v;
}

// s_waitcnt vmcnt(n) (gfx9 encoding, n < 64); lgkmcnt and expcnt unconstrained.
template <int N>
__device__ __forceinline__ void waitcnt_vm() {
  __builtin_amdgcn_s_waitcnt(0x0f70 | (N & 15) | ((N >> 4) << 14));
}

__device__ __forceinline__ uint32_t lds_addr(const void* p) {
  return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) uint8_t*)p;
}

// One wave-wide direct-to-LDS load: lane i's 16 bytes at gptr land at
// lds_base + 16*i.  Written as inline asm so that the compiler does not treat
// every later LDS read as possibly aliasing the in-flight load (it would wait
// for all outstanding loads there); callers wait explicitly with vmcnt.
__device__ __forceinline__ void dma16(const void* gptr, uint32_t lds_base) {
  asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off"
               :
               : "v"(gptr), "s"(lds_base)
               : "memory", "m0");
}

__device__ __forceinline__ uint64_t wave_max_u64(uint64_t v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    const uint64_t p = shfl_xor_u64(v, off);
    v = v > p ? v : p;
  }
  return v;
}

}  // namespace adapld
