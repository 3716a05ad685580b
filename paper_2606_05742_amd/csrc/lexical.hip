// Lexical anchoring (Sec. 3.3): longest-suffix n-gram match over the context.
//
// One workgroup of 1024 threads (16 waves) per sequence.  The context is
// staged in LDS in pieces of up to kLexChunk tokens (plus the n_max-1 tokens
// before each piece, so every n-gram ending in the piece is visible), with
// 16-byte loads.  Pass 1 computes, for every candidate end position j in
// [0, L-2], the length of the common suffix of M[..j] and M[..L-1] capped at
// n_max, and reduces its maximum n*.  Pass 2 re-derives the match lengths,
// each thread over a contiguous run of positions, and compacts
// {j : len(j) >= n*} in ascending order with a wave scan and a 16-entry
// workgroup scan of the per-thread hit counts.  A context that fits one piece
// is staged once and scanned once: the match lengths stay in registers
// between the two steps; when every row of the batch fits one piece, the
// whole row is staged together with the length load.
#include "adapld_internal.h"
#include "device_utils.h"

namespace adapld {
namespace {

constexpr int kLexThreads = 1024;
constexpr int kLexWaves = kLexThreads / kWave;
constexpr int kMaxNmax = ADAPLD_MAX_NMAX;
constexpr int kLexChunk = 32768;   // tokens per LDS piece (128 KiB)
constexpr int kHalo = kMaxNmax;    // >= n_max - 1, multiple of 4

// Stage tokens [lo, hi) at s_tok[kHalo - (p0 - lo) ...]: s_tok[kHalo + i] holds M[p0 + i].
// A piece holds at most kLexChunk + kHalo tokens.  On the 16-byte path every
// load of a thread is issued before the first LDS write, so the loads are in
// flight together instead of one round trip per loop iteration: R (the
// number of int4 per thread the piece needs) is a compile-time count, indices
// are clamped into the piece, and a clamped slot writes the last element
// again with the value it already holds, so neither loads nor writes need a
// branch (a guarded write would let the compiler sink its load behind it).
constexpr int kStageVec = (kLexChunk + kHalo) / 4 / kLexThreads + 1;
template <int R>
__device__ __forceinline__ void stage_vec(const int4* __restrict__ src, int* dst, int n4) {
  const int tid = threadIdx.x;
  int4 v[R];
#pragma unroll
  for (int r = 0; r < R; ++r) v[r] = src[min(tid + r * kLexThreads, n4 - 1)];
#pragma unroll
  for (int r = 0; r < R; ++r) *reinterpret_cast<int4*>(&dst[4 * min(tid + r * kLexThreads, n4 - 1)]) = v[r];
}
__device__ __forceinline__ void stage(const int32_t* __restrict__ M, int* s_tok, int p0, int lo, int hi) {
  const int base = kHalo - (p0 - lo);  // LDS slot of token lo
  const int n = hi - lo;
  if (((lo | base) & 3) == 0 && (reinterpret_cast<uintptr_t>(M + lo) & 15) == 0) {
    const int n4 = n >> 2;
    const int4* __restrict__ src = reinterpret_cast<const int4*>(M + lo);
    int* dst = s_tok + base;
    static_assert(kStageVec == 9, "one case per count");
    switch ((n4 + kLexThreads - 1) / kLexThreads) {
      case 0: break;
      case 1: stage_vec<1>(src, dst, n4); break;
      case 2: stage_vec<2>(src, dst, n4); break;
      case 3: stage_vec<3>(src, dst, n4); break;
      case 4: stage_vec<4>(src, dst, n4); break;
      case 5: stage_vec<5>(src, dst, n4); break;
      case 6: stage_vec<6>(src, dst, n4); break;
      case 7: stage_vec<7>(src, dst, n4); break;
      case 8: stage_vec<8>(src, dst, n4); break;
      default: stage_vec<9>(src, dst, n4); break;
    }
    for (int i = 4 * n4 + threadIdx.x; i < n; i += kLexThreads) s_tok[base + i] = M[lo + i];
  } else {
    for (int i = threadIdx.x; i < n; i += kLexThreads) s_tok[base + i] = M[lo + i];
  }
}

// Common-suffix length of M[..j] and the query suffix, capped at cap
// (cap <= j + 1, so the n-gram never starts before position 0).
__device__ __forceinline__ int suffix_len(const int* s_tok, int p0, const int* s_suffix, int j, int cap) {
  int n = 0;
  while (n < cap && s_tok[kHalo + (j - p0) - n] == s_suffix[n]) ++n;
  return n;
}

// Single pass over a context staged whole in LDS (J = L - 1 <= kLexChunk,
// n_max <= NM <= 16, per <= PMAX).  Thread tid owns positions
// [tid * per, +per); per is odd, so the 64 lanes of a wave, reading word
// tid * per + i at the same time, touch 64 different LDS banks.
//
// The length at j is the number of k < min(n_max, j + 1) from 0 up with
// M[j - k] == M[L - 1 - k] (so tokens before position 0 never count).  It is
// 0 unless M[j] is the query's last token, so one compare per position picks
// out the few positions that need more, and only those read the tokens before
// them (16 waves on one CU make this VALU-bound: a full compare chain for
// every position cost about three times as long).  Runs of 33 positions
// keep the full chain, which measured faster there.  The lengths stay in
// registers (4 bits each) for the ordered compaction after the workgroup
// reduction of n*; NM and PMAX are compile-time bounds.
template <int NM, int PMAX>
__device__ __forceinline__ void single_pass(const int* s_tok, const int* s_suffix, int* s_red, int J, int per,
                                            int n_max, int32_t* __restrict__ out, int32_t* __restrict__ cand_count,
                                            int32_t* __restrict__ match_n) {
  const int tid = threadIdx.x;
  const int lane = lane_id();
  const int wave = tid / kWave;
  const int q0 = tid * per;
  uint64_t lens4[(PMAX + 15) / 16] = {};
  int best = 0;
  if constexpr (PMAX <= 17) {
    // Only positions whose token is the query's last token have a match length
    // of 1 or more; one compare per position finds them, and their lengths are
    // then extended against the rest of the suffix (capped at
    // min(n_max, j + 1)) from LDS.  Every other position keeps length 0.
    const int s0 = s_suffix[0];
    uint64_t m0 = 0;
#pragma unroll
    for (int e = 0; e < PMAX; ++e)
      if (e < per && q0 + e < J && s_tok[kHalo + q0 + e] == s0) m0 |= 1ull << e;
    for (uint64_t rem = m0; rem; rem &= rem - 1) {
      const int e = __builtin_ctzll(rem);
      const int j = q0 + e;
      const int cap = min(min(n_max, NM), j + 1);
      int n = 1;
      while (n < cap && s_tok[kHalo + j - n] == s_suffix[n]) ++n;
      const uint64_t bits = (uint64_t)n << (4 * (e & 15));
#pragma unroll
      for (int w = 0; w < (PMAX + 15) / 16; ++w)
        if ((e >> 4) == w) lens4[w] |= bits;
      best = max(best, n);
    }
  } else {
    // Runs of up to 33 positions (contexts beyond 16 Ki tokens): the
    // first-token filter's per-match loop costs more than it saves there, so
    // every position takes the full compare chain against the suffix held in
    // registers, with the run's tokens and the NM - 1 before it.
    int suf[NM];
#pragma unroll
    for (int k = 0; k < NM; ++k) suf[k] = k < n_max ? s_suffix[k] : 0;
    int w[NM - 1 + PMAX];   // w[i] = M[q0 - (NM - 1) + i]
#pragma unroll
    for (int i = 0; i < NM - 1 + PMAX; ++i) w[i] = i < NM - 1 + per ? s_tok[kHalo + q0 - (NM - 1) + i] : 0;
#pragma unroll
    for (int e = 0; e < PMAX; ++e) {
      const int j = q0 + e;
      if (e < per && j < J) {
        uint32_t eq = 0;
#pragma unroll
        for (int k = 0; k < NM; ++k) eq |= (uint32_t)(w[e + NM - 1 - k] == suf[k]) << k;
        const int n = min(__builtin_ctz(~eq), min(n_max, j + 1));
        lens4[e >> 4] |= (uint64_t)n << (4 * (e & 15));
        best = max(best, n);
      }
    }
  }
  best = wave_max_i32(best);
  if (lane == 0) s_red[wave] = best;
  __syncthreads();
  int n_star = 0;
#pragma unroll
  for (int v = 0; v < kLexWaves; ++v) n_star = max(n_star, s_red[v]);
  int found = 0;
  if (n_star > 0) {
    uint64_t bits = 0;
#pragma unroll
    for (int e = 0; e < PMAX; ++e)
      if (e < per && (int)((lens4[e >> 4] >> (4 * (e & 15))) & 15) >= n_star) bits |= 1ull << e;
    const int cnt = __popcll(bits);
    const int incl = wave_incl_scan_i32(cnt);
    __syncthreads();  // the n* reads of s_red are done
    if (lane == kWave - 1) s_red[wave] = incl;
    __syncthreads();
    int before = 0;
#pragma unroll
    for (int v = 0; v < kLexWaves; ++v) {
      const int c = s_red[v];
      before += (v < wave) ? c : 0;
      found += c;
    }
    int slot = before + incl - cnt;
    while (bits) {
      const int e = __builtin_ctzll(bits);
      bits &= bits - 1;
      out[slot++] = q0 + e;
    }
  }
  if (tid == 0) {
    *cand_count = found;
    *match_n = n_star;
  }
}

template <int NM>
__device__ __forceinline__ void single_pass_nm(const int* s_tok, const int* s_suffix, int* s_red, int J, int n_max,
                                               int32_t* out, int32_t* cand_count, int32_t* match_n) {
  const int per = J > 0 ? ((J + kLexThreads - 1) / kLexThreads) | 1 : 0;   // odd, <= 33
  if (per <= 9) single_pass<NM, 9>(s_tok, s_suffix, s_red, J, per, n_max, out, cand_count, match_n);
  else if (per <= 17) single_pass<NM, 17>(s_tok, s_suffix, s_red, J, per, n_max, out, cand_count, match_n);
  else single_pass<NM, kLexChunk / kLexThreads + 1>(s_tok, s_suffix, s_red, J, per, n_max, out, cand_count, match_n);
}

__global__ __launch_bounds__(kLexThreads) void lexical_match_kernel(
    const int32_t* __restrict__ tokens, const int32_t* __restrict__ lens, int L_stride, int n_max,
    int32_t* __restrict__ cand_pos, int32_t* __restrict__ cand_count,
    int32_t* __restrict__ match_n) {
  // kLexThreads more than one piece: the single pass may round its runs up
  __shared__ __attribute__((aligned(16))) int s_tok[kHalo + kLexChunk + kLexThreads];
  __shared__ int s_suffix[kMaxNmax];
  __shared__ int s_red[kLexWaves];

  const int b = blockIdx.x;
  const int tid = threadIdx.x;
  const int lane = lane_id();
  const int wave = tid / kWave;
  const int32_t* __restrict__ M = tokens + (size_t)b * L_stride;

  // When every context fits one piece (L_stride <= kLexChunk + 1), the whole
  // allocated row is staged without waiting for the length, so the length and
  // the tokens arrive in one memory round trip, and the query suffix is read
  // from the staged copy.
  if (L_stride <= kLexChunk + 1 && n_max <= 15) {
    const int L_raw = lens[b];
    stage(M, s_tok, 0, 0, L_stride);
    const int L = min(max(L_raw, 0), L_stride);
    __syncthreads();
    if (tid < n_max && tid < L) s_suffix[tid] = s_tok[kHalo + L - 1 - tid];
    __syncthreads();
    const int J = L - 1;
    int32_t* __restrict__ out = cand_pos + (size_t)b * L_stride;
    if (n_max <= 4) single_pass_nm<4>(s_tok, s_suffix, s_red, J, n_max, out, cand_count + b, match_n + b);
    else if (n_max <= 8) single_pass_nm<8>(s_tok, s_suffix, s_red, J, n_max, out, cand_count + b, match_n + b);
    else single_pass_nm<16>(s_tok, s_suffix, s_red, J, n_max, out, cand_count + b, match_n + b);
    return;
  }

  const int L = min(max(lens[b], 0), L_stride);
  const int J = L - 1;  // candidate end positions are [0, J)

  if (tid < n_max && tid < L) s_suffix[tid] = M[L - 1 - tid];
  const int npieces = J > 0 ? (J + kLexChunk - 1) / kLexChunk : 0;

  // A context that fits one piece is staged once and scanned once.
  if (npieces == 1 && n_max <= 15) {
    stage(M, s_tok, 0, 0, J);
    __syncthreads();
    int32_t* __restrict__ out = cand_pos + (size_t)b * L_stride;
    if (n_max <= 4) single_pass_nm<4>(s_tok, s_suffix, s_red, J, n_max, out, cand_count + b, match_n + b);
    else if (n_max <= 8) single_pass_nm<8>(s_tok, s_suffix, s_red, J, n_max, out, cand_count + b, match_n + b);
    else single_pass_nm<16>(s_tok, s_suffix, s_red, J, n_max, out, cand_count + b, match_n + b);
    return;
  }

  // Pass 1: n* = max over j of the capped common-suffix length.
  int best = 0;
  for (int p = 0; p < npieces; ++p) {
    const int p0 = p * kLexChunk;
    const int p1 = min(p0 + kLexChunk, J);
    __syncthreads();
    stage(M, s_tok, p0, max(p0 - (n_max - 1), 0), p1);
    __syncthreads();
    for (int j = p0 + tid; j < p1; j += kLexThreads)
      best = max(best, suffix_len(s_tok, p0, s_suffix, j, min(n_max, j + 1)));
  }
  best = wave_max_i32(best);
  if (lane == 0) s_red[wave] = best;
  __syncthreads();
  int n_star = 0;
#pragma unroll
  for (int w = 0; w < kLexWaves; ++w) n_star = max(n_star, s_red[w]);

  // Pass 2: ordered compaction of {j : len(j) == n*}.
  int total = 0;
  if (n_star > 0) {
    int32_t* __restrict__ out = cand_pos + (size_t)b * L_stride;
    for (int p = 0; p < npieces; ++p) {
      const int p0 = p * kLexChunk;
      const int p1 = min(p0 + kLexChunk, J);
      if (npieces > 1) {
        __syncthreads();
        stage(M, s_tok, p0, max(p0 - (n_max - 1), 0), p1);
        __syncthreads();
      }
      // Thread tid owns the contiguous run [q0, q0 + per) of this piece, so one
      // wave scan plus one workgroup scan of the hit counts orders all hits.
      const int per = (p1 - p0 + kLexThreads - 1) / kLexThreads;  // <= kLexChunk / kLexThreads
      const int q0 = p0 + tid * per;
      uint32_t bits = 0;
      for (int e = 0; e < per; ++e) {
        const int j = q0 + e;
        if (j < p1 && j >= n_star - 1 && suffix_len(s_tok, p0, s_suffix, j, n_star) == n_star) bits |= 1u << e;
      }
      const int cnt = __popc(bits);
      const int incl = wave_incl_scan_i32(cnt);
      __syncthreads();  // earlier reads of s_red are done
      if (lane == kWave - 1) s_red[wave] = incl;
      __syncthreads();
      int before = 0, piece_total = 0;
#pragma unroll
      for (int w = 0; w < kLexWaves; ++w) {
        const int c = s_red[w];
        before += (w < wave) ? c : 0;
        piece_total += c;
      }
      int slot = total + before + incl - cnt;
      while (bits) {
        const int e = __ffs(bits) - 1;
        bits &= bits - 1;
        out[slot++] = q0 + e;
      }
      total += piece_total;
    }
  }
  if (tid == 0) {
    cand_count[b] = total;
    match_n[b] = n_star;
  }
}

}  // namespace

hipError_t launch_lexical_match(const int32_t* tokens, const int32_t* lens, int B, int L_stride,
                                int n_max, int32_t* cand_pos, int32_t* cand_count,
                                int32_t* match_n, hipStream_t stream) {
  hipLaunchKernelGGL(lexical_match_kernel, dim3(B), dim3(kLexThreads), 0, stream, tokens, lens,
                     L_stride, n_max, cand_pos, cand_count, match_n);
  return hipGetLastError();
}

}  // namespace adapld
