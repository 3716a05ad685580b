// The paper's own semantic fallback (Sec. 3.3, Eqs. (4)-(5)): when the lexical
// set of a sequence is empty, its candidates are the earlier positions j in
// [0, L-2] whose token embedding has cosine >= tau with the embedding of the
// last token; the hidden-state rerank of Sec. 3.4 then ranks them.
//
// The cosine of a position depends on its token only, so the test is taken
// once per distinct token of the context (a quarter of the positions at
// L = 8192 in Zipf-distributed text), in three kernels:
//
// set kernel: one workgroup per sequence whose lexical set is empty marks
// the tokens of its positions in a bitmap of the vocabulary held in LDS and
// writes the distinct tokens (into the space of the candidate list, which is
// written last).
//
// flags kernel: workgroups of 4 waves tile the distinct tokens, 4 per wave
// (each row is a first touch from HBM, so many waves share the latency).
// A wave holds the anchor embedding in registers, reads its token ids with
// one load, gathers each token's embedding row (two rows in flight,
// 16-byte coalesced loads), reduces the dot product and the squared norm
// with the same fixed DPP butterfly as the hidden-state scan, and writes one
// flag byte per distinct token.
//
// compact kernel: one workgroup per sequence turns the flags into a bitmap of
// the passing tokens in LDS, then writes the candidate set in ascending
// position order (a non-empty lexical set is copied through), its size and
// its kind, in rounds of 4 consecutive positions per thread with a wave +
// workgroup scan of the counts (as the lexical kernel orders its hits).
//
// A vocabulary too large for the LDS bitmap (more than kSetMaxV tokens) takes
// the same flags kernel over positions instead of distinct tokens (16 per
// wave), and a compaction of per-position flag bytes in runs of 32.
//
// The rerank is the hidden-state scan and merge kernels in rerank-only mode.
//
// The same kernels serve the successor retrieval of the paper's draft
// construction (Sec. 3.5): there a "list" is one branch token of one
// sequence, its query is the branch token's embedding, its positions are the
// occurrence candidates t in [1, L-2] (flag index t - 1, the rerank row of
// t), and a list is only scanned when the branch token never occurs.
#include <cmath>

#include "adapld_internal.h"
#include "device_utils.h"

namespace adapld {
namespace {

constexpr int kFlagWaves = 4;
constexpr int kPosPerWave = 16;                               // positions per wave
constexpr int kSetPerWave = 4;                                // distinct tokens per wave
constexpr int kCompactThreads = 1024;
constexpr int kCompactRun = 32;                               // flags per thread per piece
constexpr int kCompactPiece = kCompactThreads * kCompactRun;
constexpr int kSetMaxV = 1 << 20;                             // vocabulary bitmap: 128 KiB of LDS
constexpr int kSetBatch = 8;                                  // token loads in flight per thread
constexpr int kSetRun = 4;                                    // positions per thread per compaction round

struct EmbedArgs {
  const int32_t* tokens;
  const int32_t* lens;
  const int32_t* cand_pos;   // lexical lists, copied through a skipped list (NULL: leave it)
  const int32_t* skip;       // [lists] nonzero: the list takes no embedding set
  const int32_t* qtok;       // [lists] query token (NULL: the sequence's last token)
  const uint16_t* emb;
  int V, B, L_stride, d, flag_stride;
  int seq_div;               // list v belongs to sequence v / seq_div
  int pos_off;               // flag i stands for position i + pos_off
  float tau;
  uint8_t* flags;       // [lists][flag_stride]
  int32_t* out_pos;     // [lists][L_stride]
  int32_t* out_count;   // [lists]
  int32_t* out_kind;    // [lists] or NULL
};

// cos(emb[t], anchor) >= tau for one gathered row; a token outside [0, V) has
// a zero embedding (cosine 0).
// SET: the items are list v's distinct tokens (the set kernel's list and
// count); otherwise its positions [pos_off, L - 1).
template <int NIT, bool SET>
__global__ __launch_bounds__(kFlagWaves * kWave) void embed_flags_kernel(const EmbedArgs a) {
  const int v = blockIdx.y;
  const int b = v / a.seq_div;
  const int lane = lane_id();
  const int wave = threadIdx.x / kWave;
  if (a.skip[v] != 0) return;        // e.g. a lexical hit needs no flags
  const int L = min(max(a.lens[b], 0), a.L_stride);
  const int n_pos = L - 1 - a.pos_off;
  const int J = SET ? min(a.out_count[v], n_pos) : n_pos;   // flags [0, J)
  constexpr int kPer = SET ? kSetPerWave : kPosPerWave;
  const int j0 = (blockIdx.x * kFlagWaves + wave) * kPer;
  if (j0 >= J) return;
  const int32_t* __restrict__ M = a.tokens + (size_t)b * a.L_stride;
  const int32_t* __restrict__ items = SET ? a.out_pos + (size_t)v * a.L_stride : M + a.pos_off;
  const int d = a.d;

  const int at = a.qtok ? a.qtok[v] : M[L - 1];
  const bool a_ok = at >= 0 && at < a.V;
  const int my_tok = lane < kPer && j0 + lane < J ? items[j0 + lane] : -1;
  uint4 qv[NIT];
  float qn = 0.f;
#pragma unroll
  for (int it = 0; it < NIT; ++it) {
    const int e = (it * kWave + lane) * 8;
    qv[it] = a_ok && e < d ? *reinterpret_cast<const uint4*>(a.emb + (size_t)at * d + e) : make_uint4(0, 0, 0, 0);
    qn = dot8_bf16(qv[it], qv[it], qn);
  }
  const float qnorm = sqrtf(wave_sum_dpp(qn));

  auto score = [&](const uint4 (&rv)[NIT]) {
    float dot = 0.f, nn = 0.f;
#pragma unroll
    for (int it = 0; it < NIT; ++it) {
      dot = dot8_bf16(rv[it], qv[it], dot);
      nn = dot8_bf16(rv[it], rv[it], nn);
    }
    dot = wave_sum_dpp(dot);
    nn = wave_sum_dpp(nn);
    const float den = sqrtf(nn) * qnorm;
    return den > 0.f ? dot / den : 0.f;
  };
  auto load_row = [&](int t, uint4 (&rv)[NIT]) {
    const bool ok = t >= 0 && t < a.V;
#pragma unroll
    for (int it = 0; it < NIT; ++it) {
      const int e = (it * kWave + lane) * 8;
      rv[it] = ok && e < d ? *reinterpret_cast<const uint4*>(a.emb + (size_t)t * d + e) : make_uint4(0, 0, 0, 0);
    }
  };
  uint8_t* __restrict__ fl = a.flags + (size_t)v * a.flag_stride;
  const int n = min(kPer, J - j0);
  for (int i = 0; i < n; i += 2) {
    uint4 r0[NIT], r1[NIT];
    const int t0 = __builtin_amdgcn_readlane(my_tok, i);
    const int t1 = i + 1 < n ? __builtin_amdgcn_readlane(my_tok, i + 1) : -1;
    load_row(t0, r0);
    load_row(t1, r1);
    const float s0 = score(r0);
    const float s1 = score(r1);
    if (lane == 0) {
      fl[j0 + i] = s0 >= a.tau ? 1 : 0;
      if (i + 1 < n) fl[j0 + i + 1] = s1 >= a.tau ? 1 : 0;
    }
  }
}

__global__ __launch_bounds__(kCompactThreads) void embed_compact_kernel(const EmbedArgs a) {
  __shared__ int s_red[kCompactThreads / kWave];
  const int v = blockIdx.x;
  const int b = v / a.seq_div;
  const int tid = threadIdx.x;
  const int lane = lane_id();
  const int wave = tid / kWave;
  int32_t* __restrict__ out = a.out_pos + (size_t)v * a.L_stride;
  if (a.skip[v] != 0) {
    if (a.cand_pos) {   // the backoff rule: a lexical set is the result
      const int cc = min(max(a.skip[v], 0), a.L_stride);
      const int32_t* __restrict__ in = a.cand_pos + (size_t)v * a.L_stride;
      for (int i = tid; i < cc; i += kCompactThreads) out[i] = in[i];
      if (tid == 0) {
        a.out_count[v] = cc;
        if (a.out_kind) a.out_kind[v] = ADAPLD_KIND_LEX;
      }
    }
    return;
  }
  const int L = min(max(a.lens[b], 0), a.L_stride);
  const int J = max(L - 1 - a.pos_off, 0);
  const uint8_t* __restrict__ fl = a.flags + (size_t)v * a.flag_stride;
  int total = 0;
  for (int p0 = 0; p0 < J; p0 += kCompactPiece) {
    // Thread tid owns positions [q0, q0 + 32) of this piece (16-byte aligned).
    const int q0 = p0 + tid * kCompactRun;
    uint32_t bits = 0;
    if (q0 < J) {
      const uint4 f0 = *reinterpret_cast<const uint4*>(fl + q0);
      const uint4 f1 = *reinterpret_cast<const uint4*>(fl + q0 + 16);
      const uint32_t w[8] = {f0.x, f0.y, f0.z, f0.w, f1.x, f1.y, f1.z, f1.w};
#pragma unroll
      for (int e = 0; e < kCompactRun; ++e)
        if (((w[e >> 2] >> (8 * (e & 3))) & 0xffu) != 0u && q0 + e < J) bits |= 1u << e;
    }
    const int cnt = __popc(bits);
    const int incl = wave_incl_scan_i32(cnt);
    __syncthreads();   // earlier reads of s_red are done
    if (lane == kWave - 1) s_red[wave] = incl;
    __syncthreads();
    int before = 0, piece = 0;
#pragma unroll
    for (int w = 0; w < kCompactThreads / kWave; ++w) {
      const int c = s_red[w];
      before += w < wave ? c : 0;
      piece += c;
    }
    int slot = total + before + incl - cnt;
    while (bits) {
      const int e = __builtin_ctz(bits);
      bits &= bits - 1;
      out[slot++] = q0 + e;
    }
    total += piece;
  }
  if (tid == 0) {
    a.out_count[v] = total;
    if (a.out_kind) a.out_kind[v] = total > 0 ? ADAPLD_KIND_SEM : ADAPLD_KIND_NONE;
  }
}

// Exclusive prefix of cnt over the workgroup's threads in order; *total gets the sum.
__device__ __forceinline__ int block_excl_scan(int cnt, int* s_red, int* total) {
  const int lane = lane_id();
  const int wave = threadIdx.x / kWave;
  const int incl = wave_incl_scan_i32(cnt);
  __syncthreads();   // earlier reads of s_red are done
  if (lane == kWave - 1) s_red[wave] = incl;
  __syncthreads();
  int before = 0, sum = 0;
#pragma unroll
  for (int w = 0; w < kCompactThreads / kWave; ++w) {
    const int c = s_red[w];
    before += w < wave ? c : 0;
    sum += c;
  }
  *total = sum;
  return before + incl - cnt;
}

// The distinct tokens in [0, V) of list v's positions, in no particular
// order, into out_pos (row v) and their number into out_count[v].  The first batch of
// token loads is issued with the list's skip flag and length, before either
// is known (indices clamped to the row), so the kernel starts with one
// memory round trip.
__global__ __launch_bounds__(kCompactThreads) void embed_set_kernel(const EmbedArgs a) {
  __shared__ uint32_t s_bits[kSetMaxV / 32];
  __shared__ int s_count;
  const int v = blockIdx.x;
  const int b = v / a.seq_div;
  const int tid = threadIdx.x;
  // Position i's token is M[i]; M[min(i, last)] stays inside the row.
  const int32_t* __restrict__ M = a.tokens + (size_t)b * a.L_stride + a.pos_off;
  const int last = a.L_stride - 1 - a.pos_off;
  const int skip = a.skip[v];
  const int L = min(max(a.lens[b], 0), a.L_stride);
  int t[kSetBatch];
#pragma unroll
  for (int r = 0; r < kSetBatch; ++r) t[r] = M[min(r * kCompactThreads + tid, last)];
  if (skip != 0) return;
  const int J = max(L - 1 - a.pos_off, 0);
  const int nwords = (a.V + 31) >> 5;
  for (int i = tid; i < nwords; i += kCompactThreads) s_bits[i] = 0u;
  if (tid == 0) s_count = 0;
  __syncthreads();
  for (int i0 = 0; i0 < J; i0 += kSetBatch * kCompactThreads) {
    if (i0 > 0) {
#pragma unroll
      for (int r = 0; r < kSetBatch; ++r) t[r] = M[min(i0 + r * kCompactThreads + tid, last)];
    }
#pragma unroll
    for (int r = 0; r < kSetBatch; ++r) {
      const int x = t[r];
      if (i0 + r * kCompactThreads + tid < J && x >= 0 && x < a.V) {
        const uint32_t bit = 1u << (x & 31);
        if ((s_bits[x >> 5] & bit) == 0u) atomicOr(&s_bits[x >> 5], bit);
      }
    }
  }
  __syncthreads();
  // Rounds of one bitmap word per thread (frequent tokens have small ids, so
  // a thread owning a run of words could hold hundreds of tokens).  The list
  // is a set: a wave takes its slots with one LDS atomic, in whatever order
  // the waves arrive, and lanes write their tokens at the wave's prefix.
  int32_t* __restrict__ out = a.out_pos + (size_t)v * a.L_stride;
  const int lane = lane_id();
  for (int w0 = 0; w0 < nwords; w0 += kCompactThreads) {
    const int w = w0 + tid;
    uint32_t bits = w < nwords ? s_bits[w] : 0u;
    const int cnt = __popc(bits);
    const int incl = wave_incl_scan_i32(cnt);
    const int wave_cnt = __builtin_amdgcn_readlane(incl, kWave - 1);
    int base = 0;
    if (lane == 0 && wave_cnt > 0) base = atomicAdd(&s_count, wave_cnt);
    int slot = __builtin_amdgcn_readfirstlane(base) + incl - cnt;
    while (bits) {
      const int e = __builtin_ctz(bits);
      bits &= bits - 1;
      out[slot++] = (w << 5) + e;
    }
  }
  __syncthreads();
  if (tid == 0) a.out_count[v] = s_count;
}

// The candidate set from the flags of the distinct tokens: a bitmap of the
// tokens that pass, then the positions whose token is in it.  As in the set
// kernel, the first loads of the token list, the flags and the positions'
// tokens go out together with the list's skip flag, length and set size.
__global__ __launch_bounds__(kCompactThreads) void embed_compact_set_kernel(const EmbedArgs a) {
  __shared__ uint32_t s_bits[kSetMaxV / 32];
  __shared__ int s_red[kCompactThreads / kWave];
  const int v = blockIdx.x;
  const int b = v / a.seq_div;
  const int tid = threadIdx.x;
  int32_t* __restrict__ out = a.out_pos + (size_t)v * a.L_stride;
  const uint8_t* __restrict__ fl = a.flags + (size_t)v * a.flag_stride;
  const int32_t* __restrict__ M = a.tokens + (size_t)b * a.L_stride + a.pos_off;
  const int last = a.L_stride - 1 - a.pos_off;   // M[min(i, last)] stays inside the row
  const int skip = a.skip[v];
  const int L = min(max(a.lens[b], 0), a.L_stride);
  const int n_set = a.out_count[v];
  int st[kSetBatch];
  uint32_t sf[kSetBatch];
#pragma unroll
  for (int r = 0; r < kSetBatch; ++r) {
    const int i = min(r * kCompactThreads + tid, a.L_stride - 1);
    st[r] = out[i];
    sf[r] = fl[i];
  }
  int pt[kSetRun];   // the tokens of this thread's first positions
#pragma unroll
  for (int e = 0; e < kSetRun; ++e) pt[e] = M[min(tid * kSetRun + e, last)];
  if (skip != 0) {
    if (a.cand_pos) {   // the backoff rule: a lexical set is the result
      const int cc = min(max(skip, 0), a.L_stride);
      const int32_t* __restrict__ in = a.cand_pos + (size_t)v * a.L_stride;
      for (int i = tid; i < cc; i += kCompactThreads) out[i] = in[i];
      if (tid == 0) {
        a.out_count[v] = cc;
        if (a.out_kind) a.out_kind[v] = ADAPLD_KIND_LEX;
      }
    }
    return;
  }
  const int J = max(L - 1 - a.pos_off, 0);
  const int nwords = (a.V + 31) >> 5;
  const int D = min(max(n_set, 0), J);   // distinct tokens, listed in out
  for (int i = tid; i < nwords; i += kCompactThreads) s_bits[i] = 0u;
  __syncthreads();
  for (int i0 = 0; i0 < D; i0 += kSetBatch * kCompactThreads) {
    if (i0 > 0) {
#pragma unroll
      for (int r = 0; r < kSetBatch; ++r) {
        const int i = min(i0 + r * kCompactThreads + tid, D - 1);
        st[r] = out[i];
        sf[r] = fl[i];
      }
    }
#pragma unroll
    for (int r = 0; r < kSetBatch; ++r)
      if (i0 + r * kCompactThreads + tid < D && sf[r] != 0u) atomicOr(&s_bits[st[r] >> 5], 1u << (st[r] & 31));
  }
  __syncthreads();   // every read of the token list is done: out is rewritten below
  const bool zero_passes = 0.f >= a.tau;   // a token outside [0, V): zero embedding, cosine 0
  int total = 0;
  for (int p0 = 0; p0 < J; p0 += kSetRun * kCompactThreads) {
    // Thread tid owns positions [q0, q0 + kSetRun) of this round: neighbouring
    // lanes read neighbouring tokens.
    const int q0 = p0 + tid * kSetRun;
    if (p0 > 0) {
#pragma unroll
      for (int e = 0; e < kSetRun; ++e) pt[e] = M[min(q0 + e, last)];
    }
    uint32_t bits = 0;
#pragma unroll
    for (int e = 0; e < kSetRun; ++e) {
      const int x = pt[e];
      const bool pass = x >= 0 && x < a.V ? ((s_bits[x >> 5] >> (x & 31)) & 1u) != 0u : zero_passes;
      if (pass && q0 + e < J) bits |= 1u << e;
    }
    int round;
    int slot = total + block_excl_scan(__popc(bits), s_red, &round);
    while (bits) {
      const int e = __builtin_ctz(bits);
      bits &= bits - 1;
      out[slot++] = q0 + e;
    }
    total += round;
  }
  if (tid == 0) {
    a.out_count[v] = total;
    if (a.out_kind) a.out_kind[v] = total > 0 ? ADAPLD_KIND_SEM : ADAPLD_KIND_NONE;
  }
}

template <int NIT>
void launch_flags(const EmbedArgs& a, int B, bool set, hipStream_t stream) {
  const int per_wg = kFlagWaves * (set ? kSetPerWave : kPosPerWave);
  const dim3 grid((a.L_stride + per_wg - 1) / per_wg, B);
  if (set)
    hipLaunchKernelGGL((embed_flags_kernel<NIT, true>), grid, dim3(kFlagWaves * kWave), 0, stream, a);
  else
    hipLaunchKernelGGL((embed_flags_kernel<NIT, false>), grid, dim3(kFlagWaves * kWave), 0, stream, a);
}

size_t flag_stride_of(int L_stride) {
  return ((size_t)L_stride + kCompactRun - 1) / kCompactRun * kCompactRun;
}

// The set kernel (vocabularies of up to kSetMaxV tokens), the flags kernel
// (one instantiation per 512-element slice count of d), then the compaction.
hipError_t launch_embed_lists(const EmbedArgs& a, int lists, hipStream_t stream) {
  const int nit = (a.d + 8 * kWave - 1) / (8 * kWave);
  if (nit < 1 || nit > 16) return hipErrorInvalidValue;
  const bool set = a.V <= kSetMaxV;
  if (set) {
    hipLaunchKernelGGL(embed_set_kernel, dim3(lists), dim3(kCompactThreads), 0, stream, a);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  switch (nit) {
#define ADAPLD_FLAGS_CASE(n) \
  case n:                    \
    launch_flags<n>(a, lists, set, stream); \
    break;
    ADAPLD_FLAGS_CASE(1) ADAPLD_FLAGS_CASE(2) ADAPLD_FLAGS_CASE(3) ADAPLD_FLAGS_CASE(4)
    ADAPLD_FLAGS_CASE(5) ADAPLD_FLAGS_CASE(6) ADAPLD_FLAGS_CASE(7) ADAPLD_FLAGS_CASE(8)
    ADAPLD_FLAGS_CASE(9) ADAPLD_FLAGS_CASE(10) ADAPLD_FLAGS_CASE(11) ADAPLD_FLAGS_CASE(12)
    ADAPLD_FLAGS_CASE(13) ADAPLD_FLAGS_CASE(14) ADAPLD_FLAGS_CASE(15) ADAPLD_FLAGS_CASE(16)
#undef ADAPLD_FLAGS_CASE
    default:
      return hipErrorInvalidValue;
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (set)
    hipLaunchKernelGGL(embed_compact_set_kernel, dim3(lists), dim3(kCompactThreads), 0, stream, a);
  else
    hipLaunchKernelGGL(embed_compact_kernel, dim3(lists), dim3(kCompactThreads), 0, stream, a);
  return hipGetLastError();
}

}  // namespace

size_t embed_ws_bytes(int B, int L_stride) {
  // flags (rows padded to whole 32-flag runs of the compaction, 16-byte
  // aligned), then the candidate list, its size and its kind
  return (size_t)B * flag_stride_of(L_stride) + (size_t)B * L_stride * 4 + (size_t)B * 8;
}

size_t embed_flag_bytes(int lists, int L_stride) { return (size_t)lists * flag_stride_of(L_stride); }

hipError_t launch_embedding_fallback(const int32_t* tokens, const int32_t* lens, const int32_t* cand_pos,
                                     const int32_t* cand_count, const uint16_t* emb, int V, int B,
                                     int L_stride, int d, float tau, void* ws, int32_t** cands,
                                     int32_t** counts, int32_t** kinds, hipStream_t stream) {
  const size_t stride = flag_stride_of(L_stride);
  uint8_t* base = static_cast<uint8_t*>(ws);
  EmbedArgs a{};
  a.tokens = tokens; a.lens = lens; a.cand_pos = cand_pos; a.skip = cand_count; a.qtok = nullptr;
  a.emb = emb; a.V = V; a.B = B; a.L_stride = L_stride; a.d = d; a.flag_stride = (int)stride;
  a.seq_div = 1; a.pos_off = 0; a.tau = tau;
  a.flags = base;
  a.out_pos = reinterpret_cast<int32_t*>(base + (size_t)B * stride);
  a.out_count = a.out_pos + (size_t)B * L_stride;
  a.out_kind = a.out_count + B;
  *cands = a.out_pos;
  *counts = a.out_count;
  *kinds = a.out_kind;
  return launch_embed_lists(a, B, stream);
}

hipError_t launch_successor_embed(const int32_t* tokens, const int32_t* lens, const uint16_t* emb, int V,
                                  int B, int W, int L_stride, int d, float tau, const int32_t* skip,
                                  const int32_t* branch_tok, uint8_t* flags, int32_t* lists,
                                  int32_t* counts, hipStream_t stream) {
  EmbedArgs a{};
  a.tokens = tokens; a.lens = lens; a.cand_pos = nullptr; a.skip = skip; a.qtok = branch_tok;
  a.emb = emb; a.V = V; a.B = B * W; a.L_stride = L_stride; a.d = d;
  a.flag_stride = (int)flag_stride_of(L_stride); a.seq_div = W; a.pos_off = 1; a.tau = tau;
  a.flags = flags; a.out_pos = lists; a.out_count = counts; a.out_kind = nullptr;
  return launch_embed_lists(a, B * W, stream);
}

}  // namespace adapld
