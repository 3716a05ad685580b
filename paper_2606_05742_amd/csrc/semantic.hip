// Lexical/semantic backoff (Sec. 3.3) and hidden-state reranking (Sec. 3.4).
//
// scan kernel: grid (chunks, B), kScanWaves waves per workgroup.  A sequence
// with a lexical hit gathers its candidate rows; a sequence without one scans
// every row [0, L-2] (the fallback).  The decision is read on the device from
// cand_count, so no host synchronisation sits between the lexical match and
// this step; chunks past a sequence's row count exit at once.
//
// Each wave streams bank rows through 16-byte loads (lane l reads elements
// 8*(l + 64*i) .. +7 of a row), holds the query slice for those elements in
// registers, accumulates the dot product and the squared norm in fp32 with
// v_dot2c_f32_bf16 (two bf16 products per instruction) and
// reduces them with fixed DPP butterflies: identical rows produce bit-identical
// scores, so exact ties are broken only by position.  A wave keeps its top-k
// as one key per lane (key = ordered score bits : ~position); the waves of a
// workgroup merge their lists with a bitonic merge and write one list per
// chunk.
//
// merge kernel: one workgroup per sequence merges the chunk lists (see the
// kernel), applies tau to a fallback, decodes positions and scores and sets
// the kind.
#include "adapld_internal.h"
#include "device_utils.h"

namespace adapld {
namespace {

constexpr int kScanThreads = kScanWaves * kWave;

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));

// acc + sum of the 8 products of two 8-element bf16 vectors, fp32 accumulation.
__device__ __forceinline__ float dot8_bf16(uint4 a, uint4 b, float acc) {
  acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, a.x), __builtin_bit_cast(bf16x2_t, b.x), acc, false);
  acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, a.y), __builtin_bit_cast(bf16x2_t, b.y), acc, false);
  acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, a.z), __builtin_bit_cast(bf16x2_t, b.z), acc, false);
  acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, a.w), __builtin_bit_cast(bf16x2_t, b.w), acc, false);
  return acc;
}
// Rows whose loads are in flight together per wave (more for short rows).
template <int NIT>
struct RowsInFlight { static constexpr int value = NIT <= 4 ? 8 : (NIT <= 8 ? 4 : 2); };

struct ScanArgs {
  const uint16_t* bank;
  const uint16_t* query;
  const int32_t* lens;
  const int32_t* cand_pos;
  const int32_t* cand_count;
  int L_stride, d, k, nchunk;
  uint64_t* ws_keys;  // [B][nchunk][k]
};

__device__ __forceinline__ void seq_rows(const ScanArgs& a, int b, int& L, int& cc, int& nrows) {
  L = min(max(a.lens[b], 0), a.L_stride);
  cc = min(max(a.cand_count[b], 0), a.L_stride);
  nrows = cc > 0 ? cc : max(L - 1, 0);
}

template <int NIT>
__global__ __launch_bounds__(kScanThreads) void semantic_scan_kernel(const ScanArgs a) {
  __shared__ uint64_t s_keys[kScanWaves][kWave];
  const int b = blockIdx.y;
  const int chunk = blockIdx.x;
  int L, cc, nrows;
  seq_rows(a, b, L, cc, nrows);
  const int r0 = chunk * kRowsPerChunk;
  if (r0 >= nrows) return;
  const int r1 = min(r0 + kRowsPerChunk, nrows);
  const int lane = lane_id();
  const int wave = threadIdx.x / kWave;
  const int d = a.d;

  const uint16_t* __restrict__ qptr =
      a.query ? a.query + (size_t)b * d : a.bank + ((size_t)b * a.L_stride + (L - 1)) * d;
  uint4 qv[NIT];
  float qn = 0.f;
#pragma unroll
  for (int it = 0; it < NIT; ++it) {
    const int e = (it * kWave + lane) * 8;
    qv[it] = e < d ? *reinterpret_cast<const uint4*>(qptr + e) : make_uint4(0, 0, 0, 0);
    qn = dot8_bf16(qv[it], qv[it], qn);
  }
  qn = wave_sum_dpp(qn);
  const float qnorm = sqrtf(qn);

  const uint16_t* __restrict__ bank_b = a.bank + (size_t)b * a.L_stride * d;
  const int32_t* __restrict__ cands = a.cand_pos + (size_t)b * a.L_stride;
  uint64_t mine = 0;
  constexpr int kRowsInFlight = RowsInFlight<NIT>::value;
  for (int i0 = r0 + wave * kRowsInFlight; i0 < r1; i0 += kScanWaves * kRowsInFlight) {
    int pos[kRowsInFlight];
    bool ok[kRowsInFlight];
    uint4 hv[kRowsInFlight][NIT];
#pragma unroll
    for (int rr = 0; rr < kRowsInFlight; ++rr) {
      const int i = i0 + rr;
      int r = cc > 0 ? (i < r1 ? cands[i] : -1) : i;
      ok[rr] = i < r1 && r >= 0 && r < L;
      pos[rr] = r;
      const uint16_t* __restrict__ row = bank_b + (size_t)(ok[rr] ? r : 0) * d;
#pragma unroll
      for (int it = 0; it < NIT; ++it) {
        const int e = (it * kWave + lane) * 8;
        hv[rr][it] = (ok[rr] && e < d) ? *reinterpret_cast<const uint4*>(row + e)
                                       : make_uint4(0, 0, 0, 0);
      }
    }
#pragma unroll
    for (int rr = 0; rr < kRowsInFlight; ++rr) {
      float dot = 0.f, nn = 0.f;
#pragma unroll
      for (int it = 0; it < NIT; ++it) {
        dot = dot8_bf16(hv[rr][it], qv[it], dot);
        nn = dot8_bf16(hv[rr][it], hv[rr][it], nn);
      }
      dot = wave_sum_dpp(dot);
      nn = wave_sum_dpp(nn);
      if (ok[rr]) {  // wave-uniform
        const float den = sqrtf(nn) * qnorm;
        const float s = den > 0.f ? dot / den : 0.f;
        topk_insert(mine, rank_key(s, pos[rr]), a.k);
      }
    }
  }

  s_keys[wave][lane] = mine;
  __syncthreads();
  if (wave == 0) {
#pragma unroll
    for (int w = 1; w < kScanWaves; ++w) mine = topk_merge(mine, s_keys[w][lane]);
    if (lane < a.k) a.ws_keys[((size_t)b * a.nchunk + chunk) * a.k + lane] = mine;
  }
}

// Merge kernel.  Every chunk list holds its chunk's k largest keys, sorted.
// Only keys >= theta can rank, for any theta that at least k keys reach; two
// such bounds are combined: the largest k-th entry over the lists (that list
// alone has k keys above it) and the k-th largest list maximum (found by a
// ballot radix select on the score bits of up to 512 list heads).  The keys
// that pass are gathered into LDS in one coalesced pass and merged by one
// wave.  If the gather overflows (adversarial score layouts), the lists are
// merged one by one instead.
constexpr int kMaxCand = 2048;

__global__ __launch_bounds__(kScanThreads) void topk_merge_kernel(const ScanArgs a, float tau,
                                                                  int32_t* __restrict__ topk_pos,
                                                                  float* __restrict__ topk_score,
                                                                  int32_t* __restrict__ topk_count,
                                                                  int32_t* __restrict__ kind) {
  __shared__ uint64_t s_cand[kMaxCand];
  __shared__ uint64_t s_red[kScanWaves];
  __shared__ int s_ncand;
  const int b = blockIdx.x;
  const int lane = lane_id();
  const int wave = threadIdx.x / kWave;
  int L, cc, nrows;
  seq_rows(a, b, L, cc, nrows);
  const int nvalid = (nrows + kRowsPerChunk - 1) / kRowsPerChunk;
  const int k = a.k;
  const uint64_t* __restrict__ lists = a.ws_keys + (size_t)b * a.nchunk * k;

  uint64_t th = 0;
  for (int c = threadIdx.x; c < nvalid; c += kScanThreads) {
    const uint64_t v = lists[(size_t)c * k + (k - 1)];
    th = v > th ? v : th;
  }
  th = wave_max_u64(th);
  if (wave == 0 && nvalid >= k) {
    // k-th largest score among the heads of the first 512 lists (8 per lane).
    uint32_t hs[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int c = lane + kWave * i;
      hs[i] = c < nvalid ? (uint32_t)(lists[(size_t)c * k] >> 32) : 0u;
    }
    // Greedy MSB-first: the largest x with #{heads >= x} >= k is the k-th largest head.
    uint32_t prefix = 0;
    for (int bit = 31; bit >= 0; --bit) {
      const uint32_t cand = prefix | (1u << bit);
      int cnt = 0;
#pragma unroll
      for (int i = 0; i < 8; ++i) cnt += __popcll(__ballot(hs[i] >= cand));
      if (cnt >= k) prefix = cand;
    }
    const uint64_t thb = (uint64_t)prefix << 32;
    th = thb > th ? thb : th;
  }
  if (lane == 0) s_red[wave] = th;
  if (threadIdx.x == 0) s_ncand = 0;
  __syncthreads();
#pragma unroll
  for (int w = 0; w < kScanWaves; ++w) th = s_red[w] > th ? s_red[w] : th;
  const uint64_t floor_key = th > 0 ? th : 1;  // key 0 marks an empty slot
  for (int i = threadIdx.x; i < nvalid * k; i += kScanThreads) {
    const uint64_t v = lists[i];
    if (v >= floor_key) {
      const int slot = atomicAdd(&s_ncand, 1);
      if (slot < kMaxCand) s_cand[slot] = v;
    }
  }
  __syncthreads();
  if (wave != 0) return;
  const int ncand = s_ncand;
  uint64_t mine = 0;
  if (ncand <= kMaxCand) {
    for (int base = 0; base < ncand; base += kWave) {
      const uint64_t v = base + lane < ncand ? s_cand[base + lane] : 0ull;
      mine = topk_merge(mine, bitonic_sort_desc(v));
    }
  } else {
    for (int c = 0; c < nvalid; ++c) {
      const uint64_t other = lane < k ? lists[(size_t)c * k + lane] : 0ull;
      mine = topk_merge(mine, other);
    }
  }

  const float score = key_score(mine);
  bool keep = lane < k && mine != 0ull;
  if (cc == 0 && !isnan(tau)) keep = keep && score >= tau;  // tau filters the fallback only
  const int count = __popcll(__ballot(keep));                  // kept entries form a prefix
  if (keep) {
    topk_pos[(size_t)b * k + lane] = key_pos(mine);
    topk_score[(size_t)b * k + lane] = score;
  }
  if (lane == 0) {
    topk_count[b] = count;
    kind[b] = cc > 0 ? ADAPLD_KIND_LEX : (count > 0 ? ADAPLD_KIND_SEM : ADAPLD_KIND_NONE);
  }
}

template <int NIT>
void launch_scan(const ScanArgs& a, int B, hipStream_t stream) {
  hipLaunchKernelGGL(semantic_scan_kernel<NIT>, dim3(a.nchunk, B), dim3(kScanThreads), 0, stream, a);
}

}  // namespace

hipError_t launch_semantic_topk(const uint16_t* bank, const uint16_t* query, const int32_t* lens,
                                const int32_t* cand_pos, const int32_t* cand_count, int B,
                                int L_stride, int d, int k, float tau, int32_t* topk_pos,
                                float* topk_score, int32_t* topk_count, int32_t* kind,
                                uint64_t* ws_keys, hipStream_t stream) {
  ScanArgs a{bank, query, lens, cand_pos, cand_count, L_stride, d, k, scan_chunks(L_stride), ws_keys};
  const int nit = (d + 8 * kWave - 1) / (8 * kWave);
  switch (nit) {
#define ADAPLD_SCAN_CASE(n) \
  case n:                   \
    launch_scan<n>(a, B, stream); \
    break;
    ADAPLD_SCAN_CASE(1) ADAPLD_SCAN_CASE(2) ADAPLD_SCAN_CASE(3) ADAPLD_SCAN_CASE(4)
    ADAPLD_SCAN_CASE(5) ADAPLD_SCAN_CASE(6) ADAPLD_SCAN_CASE(7) ADAPLD_SCAN_CASE(8)
    ADAPLD_SCAN_CASE(9) ADAPLD_SCAN_CASE(10) ADAPLD_SCAN_CASE(11) ADAPLD_SCAN_CASE(12)
    ADAPLD_SCAN_CASE(13) ADAPLD_SCAN_CASE(14) ADAPLD_SCAN_CASE(15) ADAPLD_SCAN_CASE(16)
#undef ADAPLD_SCAN_CASE
    default:
      return hipErrorInvalidValue;
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(topk_merge_kernel, dim3(B), dim3(kScanThreads), 0, stream, a, tau, topk_pos,
                     topk_score, topk_count, kind);
  return hipGetLastError();
}

}  // namespace adapld
