// Lexical/semantic backoff (Sec. 3.3) and hidden-state reranking (Sec. 3.4).
//
// Scored rows.  Sequence b scores nrows_b bank rows: its lexical candidates
// when it has any (rerank), else every row [0, L-2] (the fallback).  The
// choice is read on the device from cand_count, so no host synchronisation
// sits between the lexical match and this step.  The scored rows of all
// sequences are laid end to end (sequence b starts at P_b, the sum of the
// earlier nrows) and cut into kScanWaveSlots equal contiguous ranges, one per
// wave of the scan grid: every wave streams the same number of rows, whatever
// the mix of fallbacks and hits.
//
// scan kernel: each wave streams its range from HBM into a private LDS ring
// with direct-to-LDS loads (global_load_lds_dwordx4 with the non-temporal
// hint, since every row is read once; up to kScanRingBytes in flight per
// wave, no register staging), reads each row back with 16-byte LDS
// reads (lane l holds elements 8*(l + 64*i) .. +7), holds the query slice for
// those elements in registers, accumulates the dot product and the squared
// norm in fp32 with v_dot2c_f32_bf16 and reduces them with fixed DPP
// butterflies: identical rows produce bit-identical scores, so exact ties are
// broken only by position.  The wave keeps a top-k as one key per lane (key =
// ordered score bits : ~position) and writes it out at the end of every
// sequence its range touches (a segment).
//
// merge kernel: one workgroup per sequence merges its segment lists (see the
// kernel), applies tau to a fallback, decodes positions and scores and sets
// the kind.
#include "adapld_internal.h"
#include "device_utils.h"
#include "tree_device.h"

namespace adapld {
namespace {

constexpr int kScanThreads = kScanWaves * kWave;
constexpr int kScanRingBytes = 32768;   // LDS ring per wave

typedef unsigned u32x4_t __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) u32x4_t lds_u32x4;

// Rows held by a wave's ring: a row occupies NIT KiB (one KiB per 16-byte
// load of the whole wave); 2 to 8 rows, at most 32 KiB.
template <int NIT>
struct RingRows {
  static constexpr int value = (32 / NIT) < 2 ? 2 : ((32 / NIT) > 8 ? 8 : (32 / NIT));
};

struct ScanArgs {
  const uint16_t* bank;
  const uint16_t* query;
  const int32_t* lens;
  const int32_t* cand_pos;
  const int32_t* cand_count;
  int B, L_stride, d, k, lists;   // lists = segment-list slots per sequence
  uint64_t* ws_keys;              // [B][lists][k]
  const int32_t* cand_kind;       // kind of a non-empty candidate set (NULL: LEX)
  int rerank_only;                // 1: an empty candidate set scores nothing (kind NONE)
  int seq_div;                    // list s reads the bank rows and query of sequence s / seq_div
  int pre;                        // 1: position j is scored by bank row j-1 and the default query
                                  // is row L-2 (Eq. (6)); position 0 is not scored
};

__device__ __forceinline__ void seq_rows(const ScanArgs& a, int b, int& L, int& cc, int& nrows) {
  L = min(max(a.lens[b], 0), a.L_stride);
  cc = min(max(a.cand_count[b], 0), a.L_stride);
  nrows = cc > 0 ? cc : (a.rerank_only ? 0 : max(L - 1, 0));
}

// Rows are split over W waves, wave w taking [floor(w total / W),
// floor((w+1) total / W)): never empty, so the waves that meet one sequence
// are consecutive and each writes one list.  Up to kScanWaveSlots rows, one
// row per wave (the scan is one memory round trip); beyond that at least
// kScanMinRows rows per wave, so a mid-sized scan's merge reads fewer, longer
// lists (b1_l4096: 512 lists instead of 1024, 49.5 -> 46.8 us per step).
constexpr int kScanMinRows = 8;
__device__ __forceinline__ int scan_waves(int total) {
  if (total <= kScanWaveSlots) return total;
  const int w = (total + kScanMinRows - 1) / kScanMinRows;
  return w < kScanWaveSlots ? w : kScanWaveSlots;
}
__device__ __forceinline__ int wave_of_row(int g, int total) {
  return (int)((((int64_t)g + 1) * scan_waves(total) - 1) / total);
}

// Wait until at most `later` rows issued after the oldest one are still in
// flight (NIT loads per row).
template <int NIT, int R>
__device__ __forceinline__ void wait_rows(int later) {
  static_assert((R - 1) * NIT < 64, "vmcnt holds 6 bits");
#define ADAPLD_WAIT_ROWS(n) \
  if (later == n) { asm volatile("s_waitcnt vmcnt(%0)" ::"n"(n * NIT) : "memory"); return; }
  ADAPLD_WAIT_ROWS(0)
  if constexpr (R > 1) { ADAPLD_WAIT_ROWS(1) }
  if constexpr (R > 2) { ADAPLD_WAIT_ROWS(2) }
  if constexpr (R > 3) { ADAPLD_WAIT_ROWS(3) }
  if constexpr (R > 4) { ADAPLD_WAIT_ROWS(4) }
  if constexpr (R > 5) { ADAPLD_WAIT_ROWS(5) }
  if constexpr (R > 6) { ADAPLD_WAIT_ROWS(6) }
  if constexpr (R > 7) { ADAPLD_WAIT_ROWS(7) }
#undef ADAPLD_WAIT_ROWS
}

template <int NIT>
__global__ __launch_bounds__(kScanThreads, 1) void semantic_scan_kernel(const ScanArgs a) {
  constexpr int R = RingRows<NIT>::value;
  constexpr int kSlotBytes = NIT * 1024;
  __shared__ __attribute__((aligned(1024))) uint8_t s_ring[kScanWaves][kScanRingBytes];
  __shared__ int s_start[kMaxScanSeqs + 1];   // P_b
  __shared__ int s_len[kMaxScanSeqs];         // clamped L
  __shared__ int s_cc[kMaxScanSeqs];          // clamped candidate count
  __shared__ int s_win[kScanWaves][kWave];    // bank rows of the wave's next 64 rows (-1: skip)
  __shared__ int s_pos[kScanWaves][8];
  __shared__ int s_red[kScanWaves];
  static_assert(R * kSlotBytes <= kScanRingBytes, "ring overflow");

  const int tid = threadIdx.x;
  const int lane = lane_id();
  const int wave = tid / kWave;
  const int B = a.B;
  const int d = a.d;

  // P_b for every sequence: a workgroup-wide exclusive scan of nrows_b.
  int carry = 0;
  for (int base = 0; base < B; base += kScanThreads) {
    const int b = base + tid;
    int n = 0;
    if (b < B) {
      int L, cc;
      seq_rows(a, b, L, cc, n);
      s_len[b] = L;
      s_cc[b] = cc;
    }
    const int incl = wave_incl_scan_i32(n);
    if (lane == kWave - 1) s_red[wave] = incl;
    __syncthreads();
    int before = 0, total = 0;
#pragma unroll
    for (int w = 0; w < kScanWaves; ++w) {
      before += w < wave ? s_red[w] : 0;
      total += s_red[w];
    }
    if (b < B) s_start[b] = carry + before + incl - n;
    carry += total;
    __syncthreads();
  }
  if (tid == 0) s_start[B] = carry;
  __syncthreads();
  const int rows_total = carry;

  // This wave's range of global rows; waves are independent from here on.
  const int w = __builtin_amdgcn_readfirstlane(blockIdx.x * kScanWaves + wave);
  const int nw = scan_waves(rows_total);
  if (w >= nw) return;
  const int g0 = (int)((int64_t)w * rows_total / nw);
  const int g1 = (int)((int64_t)(w + 1) * rows_total / nw);
  // Sequence holding g0: the last b with P_b <= g0 (empty sequences share P).
  auto seq_of = [&](int g) {
    int lo = 0, hi = B;   // P_lo <= g < P_hi
    while (hi - lo > 1) {
      const int mid = (lo + hi) >> 1;
      if (s_start[mid] <= g) lo = mid; else hi = mid;
    }
    return lo;
  };

  const uint32_t ring = __builtin_amdgcn_readfirstlane(lds_addr(&s_ring[wave][0]));
  const lds_u32x4* ring_p = (const lds_u32x4*)(&s_ring[wave][0]);

  // Producer: issues the loads of row g into ring slot (g - g0) % R.  The
  // bank rows of 64 rows at a time are resolved by the lanes together (one
  // candidate load per lane) into s_win.
  int pb = seq_of(g0);
  int p_start = s_start[pb], p_end = s_start[pb + 1];
  auto fill_window = [&](int gw) {
    const int gl = gw + lane;
    int r = -1;
    if (gl < g1) {
      const int b = seq_of(gl);
      const int i = gl - s_start[b];
      const int rr = s_cc[b] > 0 ? a.cand_pos[(size_t)b * a.L_stride + i] : i;
      r = rr >= a.pre && rr < s_len[b] ? rr : -1;   // positions outside [pre, L) are skipped
    }
    s_win[wave][lane] = r;
  };
  auto issue = [&](int g) {
    while (g >= p_end) {
      ++pb;
      p_start = p_end;
      p_end = s_start[pb + 1];
    }
    if (((g - g0) & (kWave - 1)) == 0) fill_window(g);
    const int r = s_win[wave][(g - g0) & (kWave - 1)];
    const int slot = (g - g0) % R;
    if (lane == 0) s_pos[wave][slot] = r;
    // A skipped row still loads (row 0 of its sequence) so that every row
    // counts NIT loads in vmcnt.
    const uint16_t* row = a.bank + ((size_t)(pb / a.seq_div) * a.L_stride + (r >= 0 ? r - a.pre : 0)) * d;
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");   // the slot's previous row has been read
#pragma unroll
    for (int it = 0; it < NIT; ++it) {
      const int e = (it * kWave + lane) * 8;
      dma16_stream(row + (e < d ? e : 0), ring + slot * kSlotBytes + it * 1024);
    }
  };

  // Consumer state: the current segment's sequence, query slice and list.
  int cb = -1, c_end = g0, list = 0;
  uint4 qv[NIT];
  float qnorm = 0.f;
  uint64_t mine = 0;
  auto flush = [&]() {
    if (cb >= 0 && lane < a.k) a.ws_keys[((size_t)cb * a.lists + list) * a.k + lane] = mine;
    mine = 0;
  };
  auto query_of = [&](int b) {
    return a.query ? a.query + (size_t)(b / a.seq_div) * d
                   : a.bank + ((size_t)(b / a.seq_div) * a.L_stride + max(s_len[b] - 1 - a.pre, 0)) * d;
  };
  auto begin_segment = [&](int g) {
    flush();
    cb = seq_of(g);
    c_end = s_start[cb + 1];
    list = w - wave_of_row(s_start[cb], rows_total);
  };
  auto set_norm = [&]() {
    float qn = 0.f;
#pragma unroll
    for (int it = 0; it < NIT; ++it) qn = dot8_bf16(qv[it], qv[it], qn);
    qnorm = sqrtf(wave_sum_dpp(qn));
  };
  // A later segment (a range crossing into the next sequence) loads its query
  // directly; the compiler's wait for it also drains the ring, which happens
  // at most a few times per wave.
  auto enter = [&](int g) {
    begin_segment(g);
    const uint16_t* qptr = query_of(cb);
#pragma unroll
    for (int it = 0; it < NIT; ++it) {
      const int e = (it * kWave + lane) * 8;
      qv[it] = e < d ? *reinterpret_cast<const uint4*>(qptr + e) : make_uint4(0, 0, 0, 0);
    }
    set_norm();
  };

  // The first segment's query goes into the ring's last slot by direct loads,
  // ahead of the first R-1 rows, so waiting for it leaves those rows in
  // flight; row R-1 takes the slot once the query is in registers.
  int gp = g0;
  {
    const uint16_t* qptr = query_of(seq_of(g0));
#pragma unroll
    for (int it = 0; it < NIT; ++it) {
      const int e = (it * kWave + lane) * 8;
      dma16(qptr + (e < d ? e : 0), ring + (R - 1) * kSlotBytes + it * 1024);
    }
  }
  for (; gp < g1 && gp - g0 < R - 1; ++gp) issue(gp);
  wait_rows<NIT, R>(gp - g0);
  begin_segment(g0);
#pragma unroll
  for (int it = 0; it < NIT; ++it) {
    const int e = (it * kWave + lane) * 8;
    const u32x4_t raw = ring_p[((R - 1) * kSlotBytes + it * 1024) / 16 + lane];
    qv[it] = e < d ? make_uint4(raw[0], raw[1], raw[2], raw[3]) : make_uint4(0, 0, 0, 0);
  }
  set_norm();
  if (gp < g1) issue(gp++);   // its wait for LDS reads covers the query's
  for (int g = g0; g < g1; ++g) {
    wait_rows<NIT, R>(min(gp - g - 1, R - 1));
    if (g >= c_end) enter(g);
    const int slot = (g - g0) % R;
    const int pos = s_pos[wave][slot];
    float dot = 0.f, nn = 0.f;
#pragma unroll
    for (int it = 0; it < NIT; ++it) {
      const int e = (it * kWave + lane) * 8;
      const u32x4_t raw = ring_p[(slot * kSlotBytes + it * 1024) / 16 + lane];
      const uint4 hv = e < d ? make_uint4(raw[0], raw[1], raw[2], raw[3]) : make_uint4(0, 0, 0, 0);
      dot = dot8_bf16(hv, qv[it], dot);
      nn = dot8_bf16(hv, hv, nn);
    }
    if (gp < g1) issue(gp++);   // refills this slot: its data is in registers
    dot = wave_sum_dpp(dot);
    nn = wave_sum_dpp(nn);
    if (pos >= 0) {  // wave-uniform
      const float den = sqrtf(nn) * qnorm;
      const float sc = den > 0.f ? dot / den : 0.f;
      topk_insert(mine, rank_key(sc, pos), a.k);
    }
  }
  flush();
}

// Merge kernel.  Every segment list holds its segment's k largest keys, sorted.
// Only keys >= theta can rank, for any theta that at least k keys reach; two
// such bounds are combined: the largest k-th entry over the lists (that list
// alone has k keys above it) and the k-th largest of 64 per-lane maxima of
// the list heads (a bitonic sort of one register per lane).  The keys
// that pass are gathered into LDS in one coalesced pass and merged by one
// wave.  If the gather overflows (adversarial score layouts), the lists are
// merged one by one instead.
constexpr int kMaxCand = 2048;

__global__ __launch_bounds__(kScanThreads) void topk_merge_kernel(const ScanArgs a, float tau,
                                                                  int32_t* __restrict__ topk_pos,
                                                                  float* __restrict__ topk_score,
                                                                  int32_t* __restrict__ topk_count,
                                                                  int32_t* __restrict__ kind,
                                                                  const TreeOut tree) {
  __shared__ uint64_t s_cand[kMaxCand];
  __shared__ __attribute__((aligned(8))) int s_start[2 * ADAPLD_MAX_TREE_NODES];
  __shared__ uint64_t s_red[kScanWaves];
  __shared__ int s_sum[kScanWaves][2];
  __shared__ int s_ncand;
  const int b = blockIdx.x;
  const int lane = lane_id();
  const int wave = threadIdx.x / kWave;
  int L, cc, nrows;
  seq_rows(a, b, L, cc, nrows);
  // P_b and the total row count locate this sequence's segment lists: one per
  // scan wave whose range meets rows [P_b, P_b + nrows).
  int before = 0, total = 0;
  for (int j = threadIdx.x; j < a.B; j += kScanThreads) {
    int Lj, ccj, nj;
    seq_rows(a, j, Lj, ccj, nj);
    before += j < b ? nj : 0;
    total += nj;
  }
  before = wave_sum_i32(before);
  total = wave_sum_i32(total);
  if (lane == 0) {
    s_sum[wave][0] = before;
    s_sum[wave][1] = total;
  }
  __syncthreads();
  before = total = 0;
#pragma unroll
  for (int w = 0; w < kScanWaves; ++w) {
    before += s_sum[w][0];
    total += s_sum[w][1];
  }
  const int nvalid = nrows > 0 ? wave_of_row(before + nrows - 1, total) - wave_of_row(before, total) + 1 : 0;
  const int k = a.k;
  const uint64_t* __restrict__ lists = a.ws_keys + (size_t)b * a.lists * k;

  // Two lower bounds on the final k-th key, whose loads go out together: the
  // largest k-th entry over the lists (that list alone has k keys above it),
  // and the k-th largest of 64 per-lane maxima of list heads in wave 0 (lane l
  // takes lists l, l+64, ..., l+448; at least k heads reach it).
  // Loads are batched and branch-free (indices clamped into the lists, the
  // excess masked afterwards), so a batch is one memory round trip.
  uint64_t th = 0, y = 0;
  const bool heads = wave == 0 && nvalid >= k;
  uint64_t h[8];
  if (heads) {
#pragma unroll
    for (int j = 0; j < 8; ++j) h[j] = lists[(size_t)min(lane + j * kWave, nvalid - 1) * k];
  }
  for (int c0 = threadIdx.x; c0 < nvalid; c0 += 4 * kScanThreads) {
    uint64_t v[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) v[j] = lists[(size_t)min(c0 + j * kScanThreads, nvalid - 1) * k + (k - 1)];
#pragma unroll
    for (int j = 0; j < 4; ++j) th = (c0 + j * kScanThreads < nvalid && v[j] > th) ? v[j] : th;
  }
  if (heads) {
#pragma unroll
    for (int j = 0; j < 8; ++j) y = (lane + j * kWave < nvalid && h[j] > y) ? h[j] : y;
  }
  th = wave_max_u64(th);
  if (wave == 0 && nvalid >= k) {
    // The bound needs only the score word: at least k heads have a score word
    // at or above the k-th largest one, so at least k keys reach it with a
    // zero position word.  Sorting 32-bit words halves the lane exchanges.
    const uint32_t ys = bitonic_sort_desc_u32((uint32_t)(y >> 32));
    const uint64_t thb = (uint64_t)(uint32_t)__builtin_amdgcn_readlane(ys, k - 1) << 32;
    th = thb > th ? thb : th;
  }
  if (lane == 0) s_red[wave] = th;
  if (threadIdx.x == 0) s_ncand = 0;
  __syncthreads();
#pragma unroll
  for (int w = 0; w < kScanWaves; ++w) th = s_red[w] > th ? s_red[w] : th;
  const uint64_t floor_key = th > 0 ? th : 1;  // key 0 marks an empty slot
  const int nkeys = nvalid * k;
  for (int i0 = threadIdx.x; i0 < nkeys; i0 += 8 * kScanThreads) {
    uint64_t v[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) v[j] = lists[min(i0 + j * kScanThreads, nkeys - 1)];
#pragma unroll
    for (int j = 0; j < 8; ++j)
      if (i0 + j * kScanThreads < nkeys && v[j] >= floor_key) {
        const int slot = atomicAdd(&s_ncand, 1);
        if (slot < kMaxCand) s_cand[slot] = v[j];
      }
  }
  __syncthreads();
  if (wave != 0) return;
  const int ncand = s_ncand;
  // The tree (step only) reads the tokens after the ranked rows.  Requesting
  // the lines after the first 64 gathered keys now, before the sort, lets the
  // tree's reads hit this CU's cache instead of waiting on memory afterwards.
  int pf0 = 0, pf1 = 0;
  const bool prefetch = tree.tokens != nullptr && lane < ncand && L >= 2;
  if (prefetch) {
    const int32_t* M = tree.tokens + (size_t)b * a.L_stride;
    const int p = min(max(key_pos(s_cand[lane]), 0), L - 2);
    pf0 = M[p + 1];
    pf1 = M[min(p + 1 + tree.S, L - 1)];
  }
  uint64_t mine = 0;
  if (ncand <= kMaxCand) {
    for (int base = 0; base < ncand; base += kWave) {
      const uint64_t v = base + lane < ncand ? s_cand[base + lane] : 0ull;
      const int n = ncand - base;   // keys in this batch (lanes below n)
      const uint64_t sorted = n <= 16 ? bitonic_sort_desc_first<16>(v)
                              : n <= 32 ? bitonic_sort_desc_first<32>(v) : bitonic_sort_desc(v);
      mine = base == 0 ? sorted : topk_merge(mine, sorted);   // the first batch needs no merge
    }
  } else {
    for (int c = 0; c < nvalid; ++c) {
      const uint64_t other = lane < k ? lists[(size_t)c * k + lane] : 0ull;
      mine = topk_merge(mine, other);
    }
  }

  // Consumes the prefetched tokens, which keeps the loads and places their
  // wait here (s_ncand is not read again, so the store is harmless).
  if (prefetch && (pf0 | pf1) == -1) s_ncand = -1;
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
    kind[b] = cc > 0 ? (a.cand_kind ? a.cand_kind[b] : ADAPLD_KIND_LEX)
                     : (count > 0 ? ADAPLD_KIND_SEM : ADAPLD_KIND_NONE);
  }
  // The step's tree, from the ranked list in registers (kind NONE has count 0).
  if (tree.tokens) build_tree_wave(tree, b, a.L_stride, L, keep ? key_pos(mine) : -1, count, s_start);
}

template <int NIT>
void launch_scan(const ScanArgs& a, hipStream_t stream) {
  hipLaunchKernelGGL(semantic_scan_kernel<NIT>, dim3(kScanWaveSlots / kScanWaves), dim3(kScanThreads), 0,
                     stream, a);
}

}  // namespace

hipError_t launch_semantic_topk(const uint16_t* bank, const uint16_t* query, const int32_t* lens,
                                const int32_t* cand_pos, const int32_t* cand_count, int B,
                                int L_stride, int d, int k, float tau, int32_t* topk_pos,
                                float* topk_score, int32_t* topk_count, int32_t* kind,
                                uint64_t* ws_keys, const int32_t* cand_kind, int rerank_only,
                                hipStream_t stream, int seq_div, const TreeOut* tree, int preceding) {
  ScanArgs a{bank, query, lens, cand_pos, cand_count, B, L_stride, d, k, scan_lists(L_stride), ws_keys,
             cand_kind, rerank_only, seq_div, preceding ? 1 : 0};
  const int nit = (d + 8 * kWave - 1) / (8 * kWave);
  switch (nit) {
#define ADAPLD_SCAN_CASE(n) \
  case n:                   \
    launch_scan<n>(a, stream); \
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
  const TreeOut t = tree ? *tree : TreeOut{};
  hipLaunchKernelGGL(topk_merge_kernel, dim3(B), dim3(kScanThreads), 0, stream, a, tau, topk_pos,
                     topk_score, topk_count, kind, t);
  return hipGetLastError();
}

}  // namespace adapld
