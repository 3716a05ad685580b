// Tree-masked verify attention (Sec. 3.6: all draft paths scored in one
// target forward with tree attention).
//
// Work decomposition.  For one sequence b and kv head g, the T*G query rows
// (node u, query head g*G + i) are stacked row = u*G + i, so the G heads that
// share a kv head share every K/V byte read.  A workgroup owns up to
// waves*NB*32 stacked rows and one split of the context keys; the last split
// also takes the tree keys.  Grid = (splits, row groups, B*Hkv).
//
// Per 64-key tile the workgroup stages K (row-major) and V (transposed to
// [dim][key]) in LDS; each wave then computes S^T = K Q^T with
// v_mfma_f32_32x32x16_bf16 (A = K rows from LDS, B = the wave's Q block held
// in registers), so every lane owns one query column and 16 keys of it:
// softmax bookkeeping (running max, rescale) is lane-local except one swap
// with the lane 32 away.  P^T is fed straight back as the B operand of
// O^T = V^T P^T; the MFMA's k index is permuted consistently on both operands
// so no shuffle is needed.  Logits are fp32 in the log2 domain.
//
// Splits write unnormalised partial outputs with their running max and sum to
// the workspace; a combine kernel merges them with log-sum-exp weights.
#include <algorithm>

#include "adapld_internal.h"
#include "device_utils.h"

namespace adapld {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

constexpr int kD = ADAPLD_HEAD_DIM;
constexpr int kKsStride = kD + 8;         // bf16 per K row in LDS (pad against bank conflicts)
constexpr int kVsStride = kKeyTile + 4;   // bf16 per V^T row in LDS
constexpr int kMaxWaves = 8;
constexpr int kMaskWords = (ADAPLD_MAX_TREE_NODES + 63) / 64;
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

struct VerifyArgs {
  const uint16_t* q;
  const uint16_t* k_ctx;
  const uint16_t* v_ctx;
  const uint16_t* k_tree;
  const uint16_t* v_tree;
  const int32_t* lens;
  const int32_t* node_count;
  const uint64_t* tree_mask;
  int L_stride, T_max, Hq, Hkv, G, rows_max, nsplit, chunk, nw;
  float scale_log2;
  uint16_t* out;
  float* lse;
  float* ws_o;    // [B*Hkv][nsplit][rows_max][D]  unnormalised partial outputs
  float2* ws_ml;  // [B*Hkv][nsplit][rows_max]     (running max in log2 units, sum)
};

__device__ __forceinline__ bf16x8_t as_bf16x8(uint4 v) { return __builtin_bit_cast(bf16x8_t, v); }

// NB = 2 needs more than 256 VGPRs, so it runs one wave per SIMD (4 waves).
template <int NB>
__global__ __launch_bounds__((NB == 1 ? kMaxWaves : 4) * kWave) void tree_verify_kernel(const VerifyArgs a) {
  __shared__ __attribute__((aligned(16))) uint16_t Ks[kKeyTile * kKsStride];
  __shared__ __attribute__((aligned(16))) uint16_t Vs[kD * kVsStride];

  const int lane = lane_id();
  const int wave = threadIdx.x / kWave;
  const int nthreads = blockDim.x;
  const int split = blockIdx.x;
  const int bg = blockIdx.z;
  const int b = bg / a.Hkv;
  const int g = bg - b * a.Hkv;
  const int T = min(max(a.node_count[b], 0), a.T_max);
  const int L = min(max(a.lens[b], 0), a.L_stride);
  const int G = a.G;
  const int rows = T * G;
  const int rows_per_wg = (nthreads / kWave) * NB * 32;
  const int row_base = blockIdx.y * rows_per_wg;
  if (row_base >= rows) return;

  const int c0 = split * a.chunk;
  const int c1 = min(c0 + a.chunk, L);
  const bool do_tree = split == a.nsplit - 1;
  const int col = lane & 31;
  const int half = lane >> 5;

  // Query fragments (B operand): lane holds dims [16*ds + 8*half, +8) of its row.
  bf16x8_t qf[NB][kD / 16];
  uint64_t mk[NB][kMaskWords];
  int qrow[NB], qu[NB], qh[NB];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    const int qr = row_base + (wave * NB + nb) * 32 + col;
    const bool valid = qr < rows;
    const int u = valid ? qr / G : 0;
    const int h = g * G + (qr - u * G);
    qrow[nb] = qr;
    qu[nb] = u;
    qh[nb] = h;
    const uint16_t* qp = a.q + (((size_t)b * a.T_max + u) * a.Hq + h) * kD + 8 * half;
#pragma unroll
    for (int ds = 0; ds < kD / 16; ++ds)
      qf[nb][ds] = as_bf16x8(valid ? *reinterpret_cast<const uint4*>(qp + 16 * ds) : make_uint4(0, 0, 0, 0));
#pragma unroll
    for (int w = 0; w < kMaskWords; ++w)
      mk[nb][w] = (valid && w < a.nw) ? a.tree_mask[((size_t)b * a.T_max + u) * a.nw + w] : 0ull;
  }

  float m_run[NB], l_run[NB];
  f32x16_t o[NB][kD / 32];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    m_run[nb] = -INFINITY;
    l_run[nb] = 0.f;
#pragma unroll
    for (int db = 0; db < kD / 32; ++db) o[nb][db] = f32x16_t{};
  }

  const int n_ctx_tiles = c1 > c0 ? (c1 - c0 + kKeyTile - 1) / kKeyTile : 0;
  const int n_tree_tiles = do_tree ? (T + kKeyTile - 1) / kKeyTile : 0;
  const size_t ctx_base = (size_t)bg * a.L_stride * kD;
  const size_t tree_base = ((size_t)b * a.T_max * a.Hkv + g) * kD;
  const size_t tree_stride = (size_t)a.Hkv * kD;

  for (int t = 0; t < n_ctx_tiles + n_tree_tiles; ++t) {
    const bool is_tree = t >= n_ctx_tiles;
    const int k0 = is_tree ? (t - n_ctx_tiles) * kKeyTile : c0 + t * kKeyTile;
    const int kend = is_tree ? T : c1;
    const uint16_t* kb = is_tree ? a.k_tree + tree_base : a.k_ctx + ctx_base;
    const uint16_t* vb = is_tree ? a.v_tree + tree_base : a.v_ctx + ctx_base;
    const size_t kstride = is_tree ? tree_stride : (size_t)kD;

    // Stage the tile: 16 chunks of 8 dims per key; 16 consecutive threads read one 256-byte row.
    for (int c = threadIdx.x; c < kKeyTile * (kD / 8); c += nthreads) {
      const int kr = c >> 4;
      const int d0 = (c & 15) * 8;
      const int key = k0 + kr;
      uint4 kv = make_uint4(0, 0, 0, 0), vv = make_uint4(0, 0, 0, 0);
      if (key < kend) {
        kv = *reinterpret_cast<const uint4*>(kb + key * kstride + d0);
        vv = *reinterpret_cast<const uint4*>(vb + key * kstride + d0);
      }
      *reinterpret_cast<uint4*>(&Ks[kr * kKsStride + d0]) = kv;
      const uint32_t w[4] = {vv.x, vv.y, vv.z, vv.w};
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        Vs[(d0 + 2 * i) * kVsStride + kr] = (uint16_t)(w[i] & 0xffffu);
        Vs[(d0 + 2 * i + 1) * kVsStride + kr] = (uint16_t)(w[i] >> 16);
      }
    }
    __syncthreads();

#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      // S^T block per 32 keys: lane holds keys 8*(r/4) + 4*half + r%4 of its query column.
      f32x16_t s[kKeyTile / 32];
#pragma unroll
      for (int kb2 = 0; kb2 < kKeyTile / 32; ++kb2) {
        s[kb2] = f32x16_t{};
#pragma unroll
        for (int ds = 0; ds < kD / 16; ++ds) {
          const bf16x8_t ka =
              *reinterpret_cast<const bf16x8_t*>(&Ks[(kb2 * 32 + col) * kKsStride + 16 * ds + 8 * half]);
          s[kb2] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka, qf[nb][ds], s[kb2], 0, 0, 0);
        }
      }
      // Scale, mask, tile max.
      float mx = -INFINITY;
#pragma unroll
      for (int kb2 = 0; kb2 < kKeyTile / 32; ++kb2) {
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int key = k0 + kb2 * 32 + 8 * (r >> 2) + 4 * half + (r & 3);
          bool ok;
          if (is_tree) {
            ok = key < kend;
            uint64_t word = 0;
#pragma unroll
            for (int w = 0; w < kMaskWords; ++w) word = (w == (key >> 6)) ? mk[nb][w] : word;
            ok = ok && ((word >> (key & 63)) & 1ull);
          } else {
            ok = key < kend;
          }
          const float z = ok ? s[kb2][r] * a.scale_log2 : -INFINITY;
          s[kb2][r] = z;
          mx = fmaxf(mx, z);
        }
      }
      mx = fmaxf(mx, __shfl_xor(mx, 32, kWave));
      const float m_new = fmaxf(m_run[nb], mx);
      const float m_use = m_new == -INFINITY ? 0.f : m_new;
      const float alpha = exp2f(m_run[nb] - m_use);
      m_run[nb] = m_new;
      float psum = 0.f;
#pragma unroll
      for (int kb2 = 0; kb2 < kKeyTile / 32; ++kb2)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const float pv = exp2f(s[kb2][r] - m_use);
          s[kb2][r] = pv;
          psum += pv;
        }
      l_run[nb] = l_run[nb] * alpha + psum;
#pragma unroll
      for (int db = 0; db < kD / 32; ++db) o[nb][db] *= alpha;

      // O^T += V^T P^T, 16 keys per MFMA: B = P^T (regs 8*s2 .. 8*s2+7 of s[kb2]),
      // A = V^T with the same key order: keys {16*s2 + 4*half + 0..3, 16*s2 + 8 + 4*half + 0..3}.
#pragma unroll
      for (int kb2 = 0; kb2 < kKeyTile / 32; ++kb2) {
#pragma unroll
        for (int s2 = 0; s2 < 2; ++s2) {
          bf16x8_t pb;
#pragma unroll
          for (int i = 0; i < 8; ++i) pb[i] = (__bf16)s[kb2][8 * s2 + i];
          const int key_lo = kb2 * 32 + 16 * s2 + 4 * half;
#pragma unroll
          for (int db = 0; db < kD / 32; ++db) {
            const uint16_t* vrow = &Vs[(db * 32 + col) * kVsStride];
            const uint2 lo = *reinterpret_cast<const uint2*>(vrow + key_lo);
            const uint2 hi = *reinterpret_cast<const uint2*>(vrow + key_lo + 8);
            const bf16x8_t va = as_bf16x8(make_uint4(lo.x, lo.y, hi.x, hi.y));
            o[nb][db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va, pb, o[nb][db], 0, 0, 0);
          }
        }
      }
    }
    __syncthreads();
  }

  // Epilogue: lane holds dims db*32 + 8*(r/4) + 4*half + r%4 of its query row.
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    const int qr = qrow[nb];
    const float l_tot = l_run[nb] + __shfl_xor(l_run[nb], 32, kWave);
    if (qr >= rows) continue;
    const int u = qu[nb], h = qh[nb];
    if (a.nsplit == 1) {
      const float inv = 1.f / l_tot;
      uint16_t* op = a.out + (((size_t)b * a.T_max + u) * a.Hq + h) * kD;
#pragma unroll
      for (int db = 0; db < kD / 32; ++db)
#pragma unroll
        for (int r4 = 0; r4 < 4; ++r4) {
          const int dim = db * 32 + 8 * r4 + 4 * half;
          uint2 pk;
          pk.x = f32_to_bf16_bits(o[nb][db][4 * r4 + 0] * inv) | (f32_to_bf16_bits(o[nb][db][4 * r4 + 1] * inv) << 16);
          pk.y = f32_to_bf16_bits(o[nb][db][4 * r4 + 2] * inv) | (f32_to_bf16_bits(o[nb][db][4 * r4 + 3] * inv) << 16);
          *reinterpret_cast<uint2*>(op + dim) = pk;
        }
      if (half == 0 && a.lse) a.lse[((size_t)b * a.Hq + h) * a.T_max + u] = (m_run[nb] + log2f(l_tot)) * kLn2;
    } else {
      const size_t slot = ((size_t)bg * a.nsplit + split) * a.rows_max + qr;
      float* wp = a.ws_o + slot * kD;
#pragma unroll
      for (int db = 0; db < kD / 32; ++db)
#pragma unroll
        for (int r4 = 0; r4 < 4; ++r4) {
          const int dim = db * 32 + 8 * r4 + 4 * half;
          *reinterpret_cast<float4*>(wp + dim) =
              make_float4(o[nb][db][4 * r4 + 0], o[nb][db][4 * r4 + 1], o[nb][db][4 * r4 + 2], o[nb][db][4 * r4 + 3]);
        }
      if (half == 0) a.ws_ml[slot] = make_float2(m_run[nb], l_tot);
    }
  }
}

// One workgroup of D threads per stacked query row: merge the splits.
__global__ __launch_bounds__(kD) void verify_combine_kernel(const VerifyArgs a) {
  const int qr = blockIdx.x;
  const int bg = blockIdx.y;
  const int b = bg / a.Hkv;
  const int g = bg - b * a.Hkv;
  const int T = min(max(a.node_count[b], 0), a.T_max);
  if (qr >= T * a.G) return;
  const int u = qr / a.G;
  const int h = g * a.G + (qr - u * a.G);
  const int dim = threadIdx.x;
  float M = -INFINITY;
  for (int s = 0; s < a.nsplit; ++s) {
    const float2 ml = a.ws_ml[((size_t)bg * a.nsplit + s) * a.rows_max + qr];
    if (ml.y > 0.f) M = fmaxf(M, ml.x);
  }
  float num = 0.f, den = 0.f;
  for (int s = 0; s < a.nsplit; ++s) {
    const size_t slot = ((size_t)bg * a.nsplit + s) * a.rows_max + qr;
    const float2 ml = a.ws_ml[slot];
    if (ml.y > 0.f) {
      const float w = exp2f(ml.x - M);
      num += w * a.ws_o[slot * kD + dim];
      den += w * ml.y;
    }
  }
  a.out[(((size_t)b * a.T_max + u) * a.Hq + h) * kD + dim] = (uint16_t)f32_to_bf16_bits(num / den);
  if (dim == 0 && a.lse) a.lse[((size_t)b * a.Hq + h) * a.T_max + u] = (M + log2f(den)) * kLn2;
}

}  // namespace

VerifyPlan plan_verify(int B, int L_stride, int T_max, int Hq, int Hkv) {
  VerifyPlan p{};
  p.G = Hq / Hkv;
  p.rows_max = T_max * p.G;
  p.nb = 2;
  const int blocks = (p.rows_max + 31) / 32;
  p.waves = std::min(4, std::max(1, (blocks + p.nb - 1) / p.nb));
  if (blocks <= 4) {  // small trees: one block per wave keeps more waves busy
    p.nb = 1;
    p.waves = std::max(1, blocks);
  }
  p.rows_per_wg = p.waves * p.nb * 32;
  p.rowgroups = (p.rows_max + p.rows_per_wg - 1) / p.rows_per_wg;
  // Enough workgroups to cover 256 CUs twice, but splits no shorter than 512 keys.
  const int base = B * Hkv * p.rowgroups;
  const int want = std::max(1, (512 + base - 1) / std::max(base, 1));
  const int max_split = std::max(1, (L_stride + 511) / 512);
  p.nsplit = std::min(want, max_split);
  int chunk = (L_stride + p.nsplit - 1) / p.nsplit;
  chunk = ((chunk + kKeyTile - 1) / kKeyTile) * kKeyTile;
  p.chunk = std::max(chunk, kKeyTile);
  p.nsplit = std::max(1, (L_stride + p.chunk - 1) / p.chunk);
  return p;
}

size_t verify_ws_bytes(const VerifyPlan& p, int B, int Hkv) {
  if (p.nsplit <= 1) return 0;
  const size_t slots = (size_t)B * Hkv * p.nsplit * p.rows_max;
  return slots * kD * sizeof(float) + slots * sizeof(float2);
}

hipError_t launch_tree_verify_attn(const uint16_t* q, const uint16_t* k_ctx, const uint16_t* v_ctx,
                                   const uint16_t* k_tree, const uint16_t* v_tree,
                                   const int32_t* lens, const int32_t* node_count,
                                   const uint64_t* tree_mask, int B, int L_stride, int T_max,
                                   int Hq, int Hkv, float scale, uint16_t* out, float* lse,
                                   void* ws, const VerifyPlan& p, hipStream_t stream) {
  VerifyArgs a{};
  a.q = q; a.k_ctx = k_ctx; a.v_ctx = v_ctx; a.k_tree = k_tree; a.v_tree = v_tree;
  a.lens = lens; a.node_count = node_count; a.tree_mask = tree_mask;
  a.L_stride = L_stride; a.T_max = T_max; a.Hq = Hq; a.Hkv = Hkv; a.G = p.G;
  a.rows_max = p.rows_max; a.nsplit = p.nsplit; a.chunk = p.chunk; a.nw = (T_max + 63) / 64;
  a.scale_log2 = scale * kLog2e;
  a.out = out; a.lse = lse;
  const size_t slots = (size_t)B * Hkv * p.nsplit * p.rows_max;
  a.ws_o = static_cast<float*>(ws);
  a.ws_ml = ws ? reinterpret_cast<float2*>(static_cast<char*>(ws) + slots * kD * sizeof(float)) : nullptr;

  const dim3 grid(p.nsplit, p.rowgroups, B * Hkv);
  const dim3 block(p.waves * kWave);
  if (p.nb == 1)
    hipLaunchKernelGGL(tree_verify_kernel<1>, grid, block, 0, stream, a);
  else
    hipLaunchKernelGGL(tree_verify_kernel<2>, grid, block, 0, stream, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || p.nsplit == 1) return e;
  hipLaunchKernelGGL(verify_combine_kernel, dim3(p.rows_max, B * Hkv), dim3(kD), 0, stream, a);
  return hipGetLastError();
}

}  // namespace adapld
