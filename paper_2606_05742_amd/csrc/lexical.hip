// Lexical anchoring (Sec. 3.3): longest-suffix n-gram match over the context.
//
// One workgroup of 1024 threads (16 waves) per sequence.  Pass 1 computes, for
// every candidate end position j in [0, L-2], the length of the common suffix
// of M[..j] and M[..L-1] capped at n_max, and reduces its maximum n*.  Pass 2
// re-derives the match lengths and compacts {j : len(j) >= n*} in ascending
// order with wave ballots and a 16-entry workgroup scan.  The context is read
// twice from L2 (a few KiB to 128 KiB per sequence), so the kernel is
// latency-bound, not bandwidth-bound.
#include "adapld_internal.h"
#include "device_utils.h"

namespace adapld {
namespace {

constexpr int kLexThreads = 1024;
constexpr int kLexWaves = kLexThreads / kWave;
constexpr int kMaxNmax = 64;

__device__ __forceinline__ int suffix_len(const int32_t* __restrict__ M, const int* s_suffix,
                                          int j, int cap) {
  // cap = min(n_max, j + 1): the n-gram ending at j may not start before 0.
  int n = 0;
  while (n < cap && M[j - n] == s_suffix[n]) ++n;
  return n;
}

__global__ __launch_bounds__(kLexThreads) void lexical_match_kernel(
    const int32_t* __restrict__ tokens, const int32_t* __restrict__ lens, int L_stride, int n_max,
    int32_t* __restrict__ cand_pos, int32_t* __restrict__ cand_count,
    int32_t* __restrict__ match_n) {
  __shared__ int s_suffix[kMaxNmax];
  __shared__ int s_red[kLexWaves];
  __shared__ int s_base[kLexWaves];

  const int b = blockIdx.x;
  const int tid = threadIdx.x;
  const int lane = lane_id();
  const int wave = tid / kWave;
  const int32_t* __restrict__ M = tokens + (size_t)b * L_stride;
  const int L = min(max(lens[b], 0), L_stride);

  if (tid < n_max && tid < L) s_suffix[tid] = M[L - 1 - tid];
  __syncthreads();

  // Pass 1: n* = max over j of the capped common-suffix length.
  int best = 0;
  for (int j = tid; j < L - 1; j += kLexThreads) best = max(best, suffix_len(M, s_suffix, j, min(n_max, j + 1)));
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
    for (int base = 0; base < L - 1; base += kLexThreads) {
      const int j = base + tid;
      bool hit = false;
      if (j < L - 1 && j >= n_star - 1) hit = suffix_len(M, s_suffix, j, n_star) == n_star;
      const uint64_t ball = __ballot(hit);
      __syncthreads();  // previous round's s_base reads are done
      if (lane == 0) s_base[wave] = __popcll(ball);
      __syncthreads();
      int before = 0, round_total = 0;
#pragma unroll
      for (int w = 0; w < kLexWaves; ++w) {
        const int c = s_base[w];
        before += (w < wave) ? c : 0;
        round_total += c;
      }
      if (hit) out[total + before + __popcll(ball & lanes_below())] = j;
      total += round_total;
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
