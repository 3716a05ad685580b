// Incremental device-resident n-gram index: the lexical match of Sec. 3.3
// (the longest-suffix generalisation of the exact-match set) answered from an
// index that is updated with each iteration's new tokens, instead of a scan
// of the whole context.
//
// Per sequence and n-gram length n (1 .. n_max) the index holds an
// open-addressing table of the distinct n-grams that end at a candidate
// position j in [n-1, L-2] (a slot keeps one such end position as its key,
// so keys are compared token by token against the context, never by hash
// alone), and for each n-gram an ascending array of all its end positions in
// a per-level pool.  Positions only grow, so arrays are append-only: a full
// array moves to one of twice the capacity (the pool never needs more than
// 12 ints per context token; see ngram_pool_ints).
//
// update kernel: one workgroup per (level, sequence).  The positions that
// became candidates since the last update (all of them for a build, or
// when the context shrank) are inserted in batches of 256 in ascending
// order: each batch is sorted by 64-bit n-gram hash, equal n-grams form
// contiguous groups (checked token by token; a hash collision inside a batch
// falls back to inserting that batch one position at a time), each group's
// first thread finds or creates its slot and reserves room, arrays that
// overflow are copied by the whole workgroup, and every thread writes its
// position at its rank inside its group, so every array stays ascending.
//
// append kernel: one workgroup per sequence, one wave per level, each wave
// inserting its level's new positions 64 at a time (a register bitonic sort
// of hash bits and index forms the groups; a batch holding two different
// n-grams with equal bits falls back to one position at a time); a level that
// was never built, or whose context shrank or pool overflowed, is rebuilt
// from scratch by its wave.  With the match fused in, the first
// wave then answers the lexical match from the levels just brought up to
// date, so an iteration costs one launch.
//
// match kernel: one workgroup per sequence; lane n-1 of the first wave looks
// up the last n tokens at level n, the longest level with a hit gives n*,
// and its array is copied out as C_lex: one contiguous read.
#include "adapld_internal.h"
#include "device_utils.h"

namespace adapld {
namespace {

constexpr int kNgThreads = 256;

struct NgSlot {
  int key_end;   // an end position of the slot's n-gram; -1: empty
  int off;       // its position array in the pool
  int count;
  int cap;
};

struct NgHeader {
  int pool_top;      // ints of the pool in use
  int indexed_len;   // context length the level reflects
  int overflow;      // nonzero: the pool overflowed (the level is unusable)
  int magic;         // kNgMagic once a build has initialised the level
};

constexpr int kNgMagic = 0x6e677231;

struct NgLevel {
  NgSlot* tab;
  int32_t* pool;
  NgHeader* hdr;
  size_t mask;
  int pool_ints;
};

__device__ __forceinline__ NgLevel ng_level(void* index, int b, int n, int n_max, int L_stride) {
  const size_t slots = ngram_slots(L_stride);
  const size_t lb = ngram_level_bytes(L_stride);
  char* base = static_cast<char*>(index) + ((size_t)b * n_max + (n - 1)) * lb;
  NgLevel l;
  l.tab = reinterpret_cast<NgSlot*>(base);
  l.pool = reinterpret_cast<int32_t*>(base + slots * sizeof(NgSlot));
  l.hdr = reinterpret_cast<NgHeader*>(base + slots * sizeof(NgSlot) + ngram_pool_ints(L_stride) * 4);
  l.mask = slots - 1;
  l.pool_ints = (int)ngram_pool_ints(L_stride);
  return l;
}

// 64-bit hash of the n tokens ending at j, newest first.
__device__ __forceinline__ uint64_t ng_hash(const int32_t* M, int j, int n) {
  uint64_t h = 0x243F6A8885A308D3ull ^ (uint64_t)n;
  for (int i = 0; i < n; ++i) {
    h ^= (uint32_t)M[j - i];
    h *= 0x100000001B3ull;
    h ^= h >> 29;
  }
  h ^= h >> 30;
  h *= 0xBF58476D1CE4E5B9ull;
  h ^= h >> 27;
  h *= 0x94D049BB133111EBull;
  h ^= h >> 31;
  return h;
}

__device__ __forceinline__ bool ng_equal(const int32_t* M, int j0, int j1, int n) {
  for (int i = 0; i < n; ++i)
    if (M[j0 - i] != M[j1 - i]) return false;
  return true;
}

// The slot of the n-gram ending at j (creating it when `insert`), or -1 when
// it is absent.  The table is at most half full, so an empty slot ends every
// probe; the loop is bounded by the table size all the same.
__device__ int ng_probe(const NgLevel& lv, const int32_t* M, int j, int n, uint64_t h, bool insert, bool& created) {
  created = false;
  size_t s = h & lv.mask;
  for (size_t step = 0; step <= lv.mask; ++step, s = (s + 1) & lv.mask) {
    int k = __hip_atomic_load(&lv.tab[s].key_end, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
    if (k < 0) {
      if (!insert) return -1;
      const int prev = atomicCAS(&lv.tab[s].key_end, -1, j);
      if (prev == -1) {
        created = true;
        return (int)s;
      }
      k = prev;
    }
    if (ng_equal(M, k, j, n)) return (int)s;
  }
  return -1;
}

__device__ __forceinline__ int pow2_at_least(int v) {
  int c = 4;
  while (c < v) c <<= 1;
  return c;
}

// Reserve `ints` of the pool; -1 (and the overflow flag) when it is full.
__device__ __forceinline__ int ng_reserve(int* s_top, int* s_over, int pool_ints, int ints) {
  const int off = atomicAdd(s_top, ints);
  if (off + ints > pool_ints) {
    atomicOr(s_over, 1);
    return -1;
  }
  return off;
}

// Insert [j_lo, j_lo + cnt) one position at a time (one thread): the path
// taken when a batch holds two different n-grams with equal hash bits.
__device__ void ng_insert_serial(const NgLevel& lv, const int32_t* M, int n, int j_lo, int cnt, int* top, int* over) {
  for (int i = 0; i < cnt; ++i) {
    const int j = j_lo + i;
    bool created;
    const int s = ng_probe(lv, M, j, n, ng_hash(M, j, n), true, created);
    if (s < 0) {
      *over = 1;
      continue;
    }
    NgSlot& sl = lv.tab[s];
    int c0 = created ? 0 : sl.count, cap = created ? 0 : sl.cap, off = created ? -1 : sl.off;
    if (c0 + 1 > cap) {
      const int ncap = pow2_at_least(c0 + 1);
      const int noff = *top;
      if (noff + ncap > lv.pool_ints) {
        *over = 1;
        continue;
      }
      *top = noff + ncap;
      for (int e = 0; e < c0; ++e) lv.pool[noff + e] = lv.pool[off + e];
      off = noff;
      cap = ncap;
    }
    lv.pool[off + c0] = j;
    sl.off = off;
    sl.count = c0 + 1;
    sl.cap = cap;
  }
}

// Insert [j_lo, j_lo + cnt) (cnt <= 64) with one wave and no barriers: the
// groups of ng_insert_batch, formed by a register bitonic sort of (hash bits,
// index).  The sort key keeps the hash's top 32 bits and its low 26 bits (the
// table index of every table this index can have: at most 2^26 slots), then
// the index, so equal n-grams are contiguous and in position order.  *top is
// the level's pool top, owned by this wave.
__device__ void ng_insert_wave(const NgLevel& lv, const int32_t* M, int n, int j_lo, int cnt, int* top, int* over) {
  const int lane = lane_id();
  const bool valid = lane < cnt;
  uint64_t key = 0;   // invalid lanes sort last
  if (valid) {
    const uint64_t h = ng_hash(M, j_lo + lane, n);
    key = ~((h & 0xffffffff00000000ull) | ((h & 0x3ffffffull) << 6) | (uint64_t)lane);
  }
  const uint64_t v = ~bitonic_sort_desc(key);   // ascending (hash bits, index)
  const int jt = j_lo + (int)(v & 63);
  const uint64_t gk = v >> 6;                    // the group key
  const uint64_t gprev = shfl_u64(gk, lane > 0 ? lane - 1 : 0);
  const int jprev = __shfl(jt, lane > 0 ? lane - 1 : 0, kWave);
  const bool head = valid && (lane == 0 || gprev != gk);
  const bool differs = valid && !head && !ng_equal(M, jprev, jt, n);
  if (__ballot(differs)) {
    if (lane == 0) ng_insert_serial(lv, M, n, j_lo, cnt, top, over);
    return;
  }
  const uint64_t heads = __ballot(head);
  const uint64_t upto = lane == 63 ? ~0ull : ((2ull << lane) - 1);   // lanes 0 .. lane
  const int hp = valid ? 63 - __builtin_clzll(heads & upto) : 0;      // this lane's group head
  const uint64_t after = heads & ~upto;
  const int gend = after ? __builtin_ctzll(after) : cnt;             // (head) end of its group
  int slot = -1, off = -1, c0 = 0, cap = 0, req = 0;
  if (head) {
    bool created;
    // the table index is the low bits of the hash (= key bits 6..31 here)
    slot = ng_probe(lv, M, jt, n, (gk & 0x3ffffffull), true, created);
    if (slot >= 0 && !created) {
      off = lv.tab[slot].off;
      c0 = lv.tab[slot].count;
      cap = lv.tab[slot].cap;
    }
    if (slot >= 0 && c0 + (gend - lane) > cap) req = pow2_at_least(c0 + (gend - lane));
  }
  // room for the groups that grow: a wave prefix sum of the requests
  const int incl = wave_incl_scan_i32(req);
  const int total = __builtin_amdgcn_readlane(incl, kWave - 1);
  const int top0 = *top;
  const bool fits = top0 + total <= lv.pool_ints;
  int noff = -1;
  if (req > 0 && fits) noff = top0 + incl - req;
  uint64_t moves = __ballot(req > 0 && fits && c0 > 0);
  if (lane == 0) {
    if (fits) *top = top0 + total;
    else if (total > 0) *over = 1;
  }
  while (moves) {   // the whole wave copies each array that moves
    const int h = __builtin_ctzll(moves);
    moves &= moves - 1;
    const int from = __shfl(off, h, kWave), to = __shfl(noff, h, kWave), len = __shfl(c0, h, kWave);
    for (int e = lane; e < len; e += kWave) lv.pool[to + e] = lv.pool[from + e];
  }
  if (req > 0) {
    off = noff;   // -1 when the pool is full
    cap = req;
  }
  if (head && slot >= 0 && off >= 0) {
    lv.tab[slot].off = off;
    lv.tab[slot].count = c0 + (gend - lane);
    lv.tab[slot].cap = cap;
  } else if (head) {
    *over = 1;
  }
  const int goff = __shfl(head ? off : 0, hp, kWave), gc0 = __shfl(c0, hp, kWave);
  if (valid && goff >= 0) lv.pool[goff + gc0 + (lane - hp)] = jt;
}

// Insert candidate end positions [j_lo, j_lo + cnt) (cnt <= kNgThreads) of
// one level, keeping every position array ascending.
__device__ void ng_insert_batch(const NgLevel& lv, const int32_t* M, int n, int j_lo, int cnt, int* s_top,
                                int* s_over) {
  __shared__ uint64_t s_key[kNgThreads];
  __shared__ int s_idx[kNgThreads];
  __shared__ int s_hp[kNgThreads];     // group head of each sorted element
  __shared__ int s_gend[kNgThreads];   // (head) end of its group
  __shared__ int s_goff[kNgThreads];   // (head) array offset after any move
  __shared__ int s_gc0[kNgThreads];    // (head) array length before the batch
  __shared__ int s_rel[kNgThreads][3]; // moves: old offset, new offset, length
  __shared__ int s_nrel, s_collide;
  const int tid = threadIdx.x;
  // 1. hash, then sort (hash, index) ascending; entries past cnt hash to ~0
  //    and keep their larger indices, so the cnt valid ones come first.
  const bool valid_in = tid < cnt;
  s_key[tid] = valid_in ? ng_hash(M, j_lo + tid, n) : ~0ull;
  s_idx[tid] = tid;
  if (tid == 0) {
    s_nrel = 0;
    s_collide = 0;
  }
  __syncthreads();
  for (int k = 2; k <= kNgThreads; k <<= 1) {
    for (int jj = k >> 1; jj > 0; jj >>= 1) {
      const int p = tid ^ jj;
      if (p > tid) {
        const uint64_t a = s_key[tid], c = s_key[p];
        const int ia = s_idx[tid], ic = s_idx[p];
        const bool gt = a > c || (a == c && ia > ic);
        const bool up = (tid & k) == 0;
        if (gt == up) {
          s_key[tid] = c;
          s_key[p] = a;
          s_idx[tid] = ic;
          s_idx[p] = ia;
        }
      }
      __syncthreads();
    }
  }
  // 2. groups of equal hash, checked token by token against the predecessor
  const bool valid = tid < cnt;
  const int jt = j_lo + s_idx[tid];
  const bool head = valid && (tid == 0 || s_key[tid - 1] != s_key[tid]);
  if (valid && !head && !ng_equal(M, j_lo + s_idx[tid - 1], jt, n)) s_collide = 1;
  s_hp[tid] = head ? tid : 0;
  __syncthreads();
  for (int off = 1; off < kNgThreads; off <<= 1) {   // inclusive max-scan: the head of every element
    const int v = tid >= off ? s_hp[tid - off] : 0;
    __syncthreads();
    s_hp[tid] = max(s_hp[tid], v);
    __syncthreads();
  }
  if (valid && (tid + 1 == cnt || s_key[tid + 1] != s_key[tid])) s_gend[s_hp[tid]] = tid + 1;
  __syncthreads();
  if (s_collide) {
    // A hash collision inside the batch: insert one position at a time.
    if (tid == 0) ng_insert_serial(lv, M, n, j_lo, cnt, s_top, s_over);
    __syncthreads();
    return;
  }
  // 3. each group's head finds or creates its slot and reserves room
  if (head) {
    bool created;
    const int s = ng_probe(lv, M, jt, n, s_key[tid], true, created);
    int off = -1, c0 = 0, cap = 0;
    if (s >= 0) {
      NgSlot& sl = lv.tab[s];
      if (!created) {
        off = sl.off;
        c0 = sl.count;
        cap = sl.cap;
      }
      const int nc = c0 + (s_gend[tid] - tid);
      if (nc > cap) {
        const int ncap = pow2_at_least(nc);
        const int noff = ng_reserve(s_top, s_over, lv.pool_ints, ncap);
        if (noff >= 0) {
          if (c0 > 0) {
            const int r = atomicAdd(&s_nrel, 1);
            s_rel[r][0] = off;
            s_rel[r][1] = noff;
            s_rel[r][2] = c0;
          }
          off = noff;
          cap = ncap;
        } else {
          off = -1;   // overflow: the level is marked unusable
        }
      }
      if (off >= 0) {
        sl.off = off;
        sl.count = nc;
        sl.cap = cap;
      }
    } else {
      *s_over = 1;
    }
    s_goff[tid] = off;
    s_gc0[tid] = c0;
  }
  __syncthreads();
  // 4. moved arrays are copied by the whole workgroup; new positions go to
  //    their rank inside their group (disjoint from the copies)
  for (int r = 0; r < s_nrel; ++r) {
    const int from = s_rel[r][0], to = s_rel[r][1], len = s_rel[r][2];
    for (int e = tid; e < len; e += kNgThreads) lv.pool[to + e] = lv.pool[from + e];
  }
  if (valid) {
    const int h = s_hp[tid];
    if (s_goff[h] >= 0) lv.pool[s_goff[h] + s_gc0[h] + (tid - h)] = jt;
  }
  __syncthreads();
}

struct NgArgs {
  const int32_t* tokens;
  const int32_t* lens;
  void* index;
  int B, L_stride, n_max;
  int rebuild;
};

__global__ __launch_bounds__(kNgThreads) void ngram_update_kernel(const NgArgs a) {
  __shared__ int s_top, s_over, s_start;
  const int n = blockIdx.x + 1;
  const int b = blockIdx.y;
  const NgLevel lv = ng_level(a.index, b, n, a.n_max, a.L_stride);
  const int32_t* M = a.tokens + (size_t)b * a.L_stride;
  const int L = min(max(a.lens[b], 0), a.L_stride);
  if (threadIdx.x == 0) {
    const NgHeader h = *lv.hdr;
    // A build, a context that shrank or an unusable level starts from scratch.
    const bool fresh = a.rebuild || h.magic != kNgMagic || L < h.indexed_len || h.indexed_len < 0 || h.overflow;
    s_top = fresh ? 0 : h.pool_top;
    s_over = 0;
    s_start = fresh ? -1 : max(n - 1, h.indexed_len - 1);
  }
  __syncthreads();
  int j0 = s_start;
  if (j0 < 0) {
    for (size_t s = threadIdx.x; s <= lv.mask; s += kNgThreads) lv.tab[s] = NgSlot{-1, 0, 0, 0};
    j0 = n - 1;
    __syncthreads();
  }
  // candidate end positions [j0, L-2], in batches, ascending
  for (int lo = j0; lo <= L - 2; lo += kNgThreads) ng_insert_batch(lv, M, n, lo, min(kNgThreads, L - 1 - lo), &s_top, &s_over);
  if (threadIdx.x == 0) *lv.hdr = NgHeader{s_top, L, s_over, kNgMagic};
}

// The lexical match of sequence b from its (up-to-date) index, by the first
// wave of the workgroup: lane n-1 looks up level n; writes the outputs.
__device__ void ng_match_seq(const NgArgs& a, int b, int32_t* __restrict__ cand_pos, int32_t* __restrict__ cand_count,
                             int32_t* __restrict__ match_n, int* s_n, int* s_off, int* s_cnt);

// Appending, one wave per level (n_max <= kNgAppendWaves), each inserting its
// level's new positions 64 at a time; with MATCH the first wave then answers
// the lexical match from the levels just brought up to date, so an iteration
// costs one launch.
constexpr int kNgAppendWaves = 16;

template <bool MATCH>
__global__ __launch_bounds__(kNgAppendWaves * kWave) void ngram_append_kernel(const NgArgs a, int32_t* __restrict__ cand_pos,
                                                                             int32_t* __restrict__ cand_count,
                                                                             int32_t* __restrict__ match_n) {
  __shared__ int s_top[kNgAppendWaves], s_over[kNgAppendWaves];
  __shared__ int s_n, s_off, s_cnt;
  const int b = blockIdx.x;
  const int wave = threadIdx.x / kWave;
  const int lane = lane_id();
  const int n = wave + 1;
  const int32_t* M = a.tokens + (size_t)b * a.L_stride;
  const int L = min(max(a.lens[b], 0), a.L_stride);
  if (n <= a.n_max) {
    const NgLevel lv = ng_level(a.index, b, n, a.n_max, a.L_stride);
    const NgHeader h = *lv.hdr;
    const bool fresh = h.magic != kNgMagic || L < h.indexed_len || h.indexed_len < 0 || h.overflow;
    int j0 = max(n - 1, h.indexed_len - 1);
    if (fresh) {   // a context that shrank, or a level never built: start from scratch
      for (size_t s = lane; s <= lv.mask; s += kWave) lv.tab[s] = NgSlot{-1, 0, 0, 0};
      j0 = n - 1;
    }
    if (lane == 0) {
      s_top[wave] = fresh ? 0 : h.pool_top;
      s_over[wave] = 0;
    }
    for (int lo = j0; lo <= L - 2; lo += kWave) ng_insert_wave(lv, M, n, lo, min(kWave, L - 1 - lo), &s_top[wave], &s_over[wave]);
    if (lane == 0) *lv.hdr = NgHeader{s_top[wave], L, s_over[wave], kNgMagic};
  }
  if constexpr (MATCH) {
    __syncthreads();   // every level of this sequence is up to date
    ng_match_seq(a, b, cand_pos, cand_count, match_n, &s_n, &s_off, &s_cnt);
  }
}

__global__ __launch_bounds__(kNgThreads) void ngram_match_kernel(const NgArgs a, int32_t* __restrict__ cand_pos,
                                                                 int32_t* __restrict__ cand_count,
                                                                 int32_t* __restrict__ match_n) {
  __shared__ int s_n, s_off, s_cnt;
  ng_match_seq(a, blockIdx.x, cand_pos, cand_count, match_n, &s_n, &s_off, &s_cnt);
}

__device__ void ng_match_seq(const NgArgs& a, int b, int32_t* __restrict__ cand_pos, int32_t* __restrict__ cand_count,
                             int32_t* __restrict__ match_n, int* s_n, int* s_off, int* s_cnt) {
  const int lane = lane_id();
  const int32_t* M = a.tokens + (size_t)b * a.L_stride;
  const int L = min(max(a.lens[b], 0), a.L_stride);
  if (threadIdx.x < kWave) {
    // lane n-1 looks up level n
    const int n = lane + 1;
    int cnt = 0, off = 0;
    bool stale = false;
    if (n <= a.n_max) {
      const NgLevel lv = ng_level(a.index, b, n, a.n_max, a.L_stride);
      const NgHeader h = *lv.hdr;
      stale = h.magic != kNgMagic || h.indexed_len != L || h.overflow != 0;
      if (!stale && L >= n + 1) {
        bool created;
        const int s = ng_probe(lv, M, L - 1, n, ng_hash(M, L - 1, n), false, created);
        if (s >= 0) {
          cnt = lv.tab[s].count;
          off = lv.tab[s].off;
        }
      }
    }
    const uint64_t hit = __ballot(cnt > 0);
    const bool any_stale = __ballot(stale) != 0;
    const int top = hit ? 63 - __builtin_clzll(hit) : -1;   // the longest level with a hit
    if (lane == 0) {
      *s_n = any_stale ? -1 : top + 1;
      *s_cnt = 0;
      *s_off = 0;
    }
    if (!any_stale && lane == top) {
      *s_cnt = cnt;
      *s_off = off;
    }
  }
  __syncthreads();
  const int nstar = *s_n, cnt = *s_cnt;
  if (cnt > 0) {
    const NgLevel lv = ng_level(a.index, b, nstar, a.n_max, a.L_stride);
    const int32_t* __restrict__ src = lv.pool + *s_off;
    int32_t* __restrict__ dst = cand_pos + (size_t)b * a.L_stride;
    for (int i = threadIdx.x; i < cnt; i += blockDim.x) dst[i] = src[i];
  }
  if (threadIdx.x == 0) {
    cand_count[b] = cnt;
    match_n[b] = nstar;
  }
}

}  // namespace

hipError_t launch_ngram_update(const int32_t* tokens, const int32_t* lens, int B, int L_stride, int n_max,
                               void* index, int rebuild, hipStream_t stream) {
  const NgArgs a{tokens, lens, index, B, L_stride, n_max, rebuild};
  hipLaunchKernelGGL(ngram_update_kernel, dim3(n_max, B), dim3(kNgThreads), 0, stream, a);
  return hipGetLastError();
}

hipError_t launch_ngram_append(const int32_t* tokens, const int32_t* lens, int B, int L_stride, int n_max, void* index,
                               int32_t* cand_pos, int32_t* cand_count, int32_t* match_n, hipStream_t stream) {
  const NgArgs a{tokens, lens, index, B, L_stride, n_max, 0};
  if (n_max > kNgAppendWaves) {   // more levels than one workgroup's waves: the build kernel's path
    hipLaunchKernelGGL(ngram_update_kernel, dim3(n_max, B), dim3(kNgThreads), 0, stream, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || !cand_pos) return e;
    hipLaunchKernelGGL(ngram_match_kernel, dim3(B), dim3(kNgThreads), 0, stream, a, cand_pos, cand_count, match_n);
    return hipGetLastError();
  }
  const dim3 block(n_max * kWave);
  if (cand_pos)
    hipLaunchKernelGGL(ngram_append_kernel<true>, dim3(B), block, 0, stream, a, cand_pos, cand_count, match_n);
  else
    hipLaunchKernelGGL(ngram_append_kernel<false>, dim3(B), block, 0, stream, a, cand_pos, cand_count, match_n);
  return hipGetLastError();
}

hipError_t launch_ngram_match(const int32_t* tokens, const int32_t* lens, const void* index, int B, int L_stride,
                              int n_max, int32_t* cand_pos, int32_t* cand_count, int32_t* match_n,
                              hipStream_t stream) {
  const NgArgs a{tokens, lens, const_cast<void*>(index), B, L_stride, n_max, 0};
  hipLaunchKernelGGL(ngram_match_kernel, dim3(B), dim3(kNgThreads), 0, stream, a, cand_pos, cand_count, match_n);
  return hipGetLastError();
}

}  // namespace adapld
