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

template <int M> __device__ __forceinline__ uint32_t xor_lanes_u32(uint32_t v);

template <int S>
__device__ __forceinline__ int wave_max_i32_steps(int v) {
  v = max(v, (int)xor_lanes_u32<S>((uint32_t)v));
  if constexpr (S > 1) return wave_max_i32_steps<S / 2>(v);
  else return v;
}
// Max over the wave on DPP moves and permlane swaps; every lane returns it.
__device__ __forceinline__ int wave_max_i32(int v) { return wave_max_i32_steps<32>(v); }

template <int S>
__device__ __forceinline__ int wave_sum_i32_steps(int v) {
  v += (int)xor_lanes_u32<S>((uint32_t)v);
  if constexpr (S > 1) return wave_sum_i32_steps<S / 2>(v);
  else return v;
}
// Sum over the wave on DPP moves and permlane swaps; every lane returns it.
__device__ __forceinline__ int wave_sum_i32(int v) { return wave_sum_i32_steps<32>(v); }

// Inclusive prefix sum over the 64 lanes without LDS traffic: DPP row shifts
// by 1, 2, 4, 8 (lanes shifted in from outside the row of 16 read 0) give the
// sum within each row; the three lower rows' totals come in as scalars.
template <int CTRL>
__device__ __forceinline__ int dpp_shift_in_zero(int v) {
  return __builtin_amdgcn_update_dpp(0, v, CTRL, 0xf, 0xf, false);
}
__device__ __forceinline__ int wave_incl_scan_i32(int v) {
  v += dpp_shift_in_zero<0x111>(v);   // row_shr:1
  v += dpp_shift_in_zero<0x112>(v);   // row_shr:2
  v += dpp_shift_in_zero<0x114>(v);   // row_shr:4
  v += dpp_shift_in_zero<0x118>(v);   // row_shr:8
  const int t0 = __builtin_amdgcn_readlane(v, 15);
  const int t1 = __builtin_amdgcn_readlane(v, 31);
  const int t2 = __builtin_amdgcn_readlane(v, 47);
  const int row = lane_id() >> 4;
  return v + (row >= 1 ? t0 : 0) + (row >= 2 ? t1 : 0) + (row >= 3 ? t2 : 0);
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

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));

// acc + sum of the 8 products of two 8-element bf16 vectors, fp32 accumulation.
__device__ __forceinline__ float dot8_bf16(uint4 a, uint4 b, float acc) {
  acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, a.x), __builtin_bit_cast(bf16x2_t, b.x), acc, false);
  acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, a.y), __builtin_bit_cast(bf16x2_t, b.y), acc, false);
  acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, a.z), __builtin_bit_cast(bf16x2_t, b.z), acc, false);
  acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, a.w), __builtin_bit_cast(bf16x2_t, b.w), acc, false);
  return acc;
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

// Lane i receives lane (i ^ M)'s value, M a power of two below 64, with DPP
// moves and permlane swaps (ALU ops, no LDS round trip).  Layouts: DPP
// row_ror:n gives lane i the value of lane (i - n) mod 16 within its row of 16;
// permlane16_swap(v, v) returns {each row pair's even row, its odd row} and
// permlane32_swap(v, v) {the low 32 lanes, the high 32 lanes}, both broadcast
// over the pair.
template <int M>
__device__ __forceinline__ uint32_t xor_lanes_u32(uint32_t v) {
  static_assert(M >= 1 && M <= 32 && (M & (M - 1)) == 0, "power of two below 64");
  if constexpr (M == 1) {
    return __builtin_amdgcn_mov_dpp(v, 0xb1, 0xf, 0xf, false);   // quad_perm [1,0,3,2]
  } else if constexpr (M == 2) {
    return __builtin_amdgcn_mov_dpp(v, 0x4e, 0xf, 0xf, false);   // quad_perm [2,3,0,1]
  } else if constexpr (M == 4) {
    const uint32_t down = __builtin_amdgcn_mov_dpp(v, 0x124, 0xf, 0xf, false);   // row_ror:4, from i - 4
    const uint32_t up = __builtin_amdgcn_mov_dpp(v, 0x12c, 0xf, 0xf, false);     // row_ror:12, from i + 4
    return (lane_id() & 4) ? down : up;
  } else if constexpr (M == 8) {
    return __builtin_amdgcn_mov_dpp(v, 0x128, 0xf, 0xf, false);  // row_ror:8
  } else if constexpr (M == 16) {
    const auto p = __builtin_amdgcn_permlane16_swap(v, v, false, false);
    return (lane_id() & 16) ? p[0] : p[1];
  } else {
    const auto p = __builtin_amdgcn_permlane32_swap(v, v, false, false);
    return (lane_id() & 32) ? p[0] : p[1];
  }
}
template <int M>
__device__ __forceinline__ uint64_t xor_lanes_u64(uint64_t v) {
  const uint32_t lo = xor_lanes_u32<M>((uint32_t)v);
  const uint32_t hi = xor_lanes_u32<M>((uint32_t)(v >> 32));
  return ((uint64_t)hi << 32) | lo;
}
// Lane i receives lane 63 - i's value.
__device__ __forceinline__ uint64_t reverse_lanes_u64(uint64_t v) {
  const uint32_t lo = __builtin_amdgcn_mov_dpp((uint32_t)v, 0x140, 0xf, 0xf, false);          // row_mirror
  const uint32_t hi = __builtin_amdgcn_mov_dpp((uint32_t)(v >> 32), 0x140, 0xf, 0xf, false);
  return xor_lanes_u64<32>(xor_lanes_u64<16>(((uint64_t)hi << 32) | lo));
}

// Lane `src`'s value (uniform src) through the scalar unit.  The builtin
// returns int: each half is cast to uint32_t before widening, so the low half
// does not sign-extend into the high one.
__device__ __forceinline__ uint64_t readlane_u64(uint64_t v, int src) {
  const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((uint32_t)v, src);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((uint32_t)(v >> 32), src);
  return ((uint64_t)hi << 32) | lo;
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
  const uint64_t last = readlane_u64(mine, k - 1);
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
// Half-cleaner steps of distance S, S/2, ..., 1 (descending).
template <int S>
__device__ __forceinline__ uint64_t half_clean_desc(uint64_t c) {
  const uint64_t p = xor_lanes_u64<S>(c);
  c = (lane_id() & S) == 0 ? (c > p ? c : p) : (c < p ? c : p);
  if constexpr (S > 1) return half_clean_desc<S / 2>(c);
  else return c;
}
__device__ __forceinline__ uint64_t topk_merge(uint64_t mine, uint64_t other) {
  const uint64_t rev = reverse_lanes_u64(other);
  return half_clean_desc<32>(mine > rev ? mine : rev);
}

// Sort a wave-wide list of 64 keys descending (bitonic network): stage K
// merges blocks of K, step J compares lanes J apart.
template <int K, int J, int KMAX = kWave>
__device__ __forceinline__ uint64_t bitonic_steps(uint64_t v) {
  const int lane = lane_id();
  const uint64_t p = xor_lanes_u64<J>(v);
  const bool keep_max = ((lane & J) == 0) == ((lane & K) == 0);
  v = keep_max ? (v > p ? v : p) : (v < p ? v : p);
  if constexpr (J > 1) return bitonic_steps<K, J / 2, KMAX>(v);
  else if constexpr (K < KMAX) return bitonic_steps<2 * K, K, KMAX>(v);
  else return v;
}
__device__ __forceinline__ uint64_t bitonic_sort_desc(uint64_t v) { return bitonic_steps<2, 1>(v); }
// The same when only lanes below N (16 or 32) hold keys and the rest hold 0:
// sorting each block of N lanes leaves block 0 descending and the rest zero,
// the result of the full sort, in fewer steps (10 or 15 instead of 21).
template <int N>
__device__ __forceinline__ uint64_t bitonic_sort_desc_first(uint64_t v) { return bitonic_steps<2, 1, N>(v); }
template <int K, int J>
__device__ __forceinline__ uint32_t bitonic_steps_u32(uint32_t v) {
  const int lane = lane_id();
  const uint32_t p = xor_lanes_u32<J>(v);
  const bool keep_max = ((lane & J) == 0) == ((lane & K) == 0);
  v = keep_max ? (v > p ? v : p) : (v < p ? v : p);
  if constexpr (J > 1) return bitonic_steps_u32<K, J / 2>(v);
  else if constexpr (K < kWave) return bitonic_steps_u32<2 * K, K>(v);
  else return v;
}
__device__ __forceinline__ uint32_t bitonic_sort_desc_u32(uint32_t v) { return bitonic_steps_u32<2, 1>(v); }

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

// The same load with the non-temporal hint, for data that one wave reads
// once and nothing reads again (the semantic scan's bank rows): the caches
// then treat it as streaming instead of keeping it.  The scan reads its rows
// 11 % faster with it.  The verify kernel has its own scalar-base form and
// uses it only when one workgroup reads each tile: with two or more row
// groups of a (sequence, kv head), the later readers take the tiles from L2.
__device__ __forceinline__ void dma16_stream(const void* gptr, uint32_t lds_base) {
  asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off nt"
               :
               : "v"(gptr), "s"(lds_base)
               : "memory", "m0");
}

template <int S>
__device__ __forceinline__ uint64_t wave_max_steps(uint64_t v) {
  const uint64_t p = xor_lanes_u64<S>(v);
  v = v > p ? v : p;
  if constexpr (S > 1) return wave_max_steps<S / 2>(v);
  else return v;
}
__device__ __forceinline__ uint64_t wave_max_u64(uint64_t v) { return wave_max_steps<32>(v); }

}  // namespace adapld
