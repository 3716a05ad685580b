// Tree-masked verify attention (Sec. 3.6: all draft paths are scored in one
// target forward with tree attention).
//
// Work decomposition.  For one sequence b and kv head g the T*G query rows
// (node u, query head g*G + i) are stacked as row = u*G + i, so the G heads
// that share a kv head share every K/V byte read from HBM.  A workgroup of 8
// waves owns a number of 32-row blocks and one split of the context
// keys; the last split also takes the tree keys.  Either every wave owns a
// row block and reads both 32-key halves of each tile (KH = 1), or the two
// waves that share a SIMD own the same row block and take one half of each
// tile each (KH = 2): then every tile is read from LDS once per row block,
// not once per wave, and the pair merges its two softmax states through LDS
// at the end, so a workgroup covers twice the keys without a second split.
// The grid is one-dimensional and XCD-aware (see the block index decode in
// the kernel).
//
// Memory pipeline.  K and V tiles of 64 keys stream through a 4-stage LDS ring
// with direct-to-LDS loads (global_load_lds_dwordx4): no VGPR staging, and up
// to three tiles are in flight.  The K tiles of all stages fill the first
// 64 KiB and the V tiles the next 64 KiB, so with the stage known at compile
// time (the main loop is unrolled over the ring) every fragment address is a
// per-lane offset plus an instruction immediate; full context tiles are
// loaded from a scalar base address.  Each 256-byte key row is stored with its
// 16-byte chunks XOR-swizzled by the row index, which keeps both LDS read
// patterns below free of bank conflicts.  One barrier per tile both publishes
// the next tile and frees the stage of the tile before the current one.
//
// Math.  S^T = K Q^T on v_mfma_f32_32x32x16_bf16 (A = K rows read from LDS,
// B = the wave's query block held in registers) leaves every lane owning one
// query column and 16 keys of it, so the online softmax is lane-local except
// for one v_permlane32_swap.  P^T goes straight back as the B operand of
// O^T = V^T P^T; the A operand V^T is read with ds_read_b64_tr_b16, which
// transposes 16-bit elements across lanes on the fly, so V stays row-major in
// LDS.  The MFMA k index of P and V is permuted identically, so no shuffle is
// needed.  Logits are fp32 in the log2 domain; the running max is only moved
// when it grows by more than 8 (a factor 256), which keeps the rescale of the
// output accumulators off the common path.
//
// Schedule.  The loop is software-pipelined over half tiles of 32 keys: the
// MFMAs of P V for half h-1 are issued beside the max of half h, and those of
// S for half h+1 beside the exponentials of half h, so each wave keeps its
// matrix core busy while its softmax runs on the VALU.  Tiles with a masked
// key (the ragged end of the context and the tree tiles) run the same
// pipeline with the mask applied.
//
// Splits write their normalised partial outputs O/l in bf16 (half the bytes of
// fp32; one more rounding of relative size 2^-9, the size of the final
// output's own) with the running max and sum in fp32; a combine kernel merges
// them with log-sum-exp weights.
#include <algorithm>
#include <type_traits>

#include "adapld_internal.h"
#include "device_utils.h"

namespace adapld {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef short s16x4_t __attribute__((ext_vector_type(4)));
typedef short s16x8_t __attribute__((ext_vector_type(8)));
typedef __attribute__((address_space(3))) void lds_void_t;
typedef __attribute__((address_space(3))) s16x4_t lds_s16x4_t;
typedef __attribute__((address_space(3))) uint8_t lds_u8;
typedef __attribute__((address_space(3))) bf16x8_t lds_bf16x8_t;

constexpr int kD = ADAPLD_HEAD_DIM;           // 128 bf16 = 256 bytes per key row
constexpr int kRowBytes = kD * 2;
constexpr int kStages = 4;  // power of two
constexpr int kTileBytes = kKeyTile * kRowBytes;  // 16 KiB for K (and for V)
constexpr int kMaskWords = (ADAPLD_MAX_TREE_NODES + 63) / 64;
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;
constexpr float kRescaleSlack = 8.0f;         // log2 units the running max may lag


struct VerifyArgs {
  const uint16_t* q;
  const uint16_t* k_ctx;
  const uint16_t* v_ctx;
  const uint16_t* k_tree;
  const uint16_t* v_tree;
  const int32_t* lens;
  const int32_t* node_count;
  const uint64_t* tree_mask;
  int L_stride, T_max, Hq, Hkv, G, rows_max, nsplit, chunk, nw, rowgroups, n_kvgroups;
  float scale_log2;
  uint16_t* out;
  float* lse;
  uint16_t* ws_o;  // [B*Hkv][nsplit][rows_max][D]  partial outputs O/l, bf16
  float2* ws_ml;   // [B*Hkv][nsplit][rows_max]     (running max in log2 units, sum)
};

__device__ __forceinline__ bf16x8_t as_bf16x8(uint4 v) { return __builtin_bit_cast(bf16x8_t, v); }

// Physical 16-byte chunk of logical chunk c in key row r is c ^ swz(r).  LDS
// has 64 four-byte banks (256 bytes per row of banks).  swz is a bijection on
// every 16 consecutive rows, so a K fragment read (16 lanes per cycle, one
// chunk of 16 different rows) touches 16 different chunk positions; and the
// four consecutive rows that 32 lanes of a transposed V read cover get
// different values of swz >> 2, so their 64-byte column blocks land in four
// different quarters of the bank row.  Both reads are free of bank conflicts.
__device__ __forceinline__ int swz(int r) { return ((r & 3) << 2) | ((r >> 2) & 3); }

// Issue this wave's share of one K/V tile: 64/WAVES key rows of K and of V,
// four rows (1 KiB) per instruction.  Keys past kend re-read key kend-1 (in
// bounds); their logits are masked.
template <int WAVES>
__device__ __forceinline__ void issue_tile(const uint16_t* kb, const uint16_t* vb, size_t stride,
                                           int k0, int kend, uint32_t lk, uint32_t lv, int wave,
                                           int lane) {
  constexpr int kRowsPerWave = kKeyTile / WAVES;
#pragma unroll
  for (int i = 0; i < kRowsPerWave / 4; ++i) {
    const int row0 = kRowsPerWave * wave + 4 * i;
    const int row = row0 + (lane >> 4);
    const int c = (lane & 15) ^ swz(row);
    const size_t key = (size_t)min(k0 + row, kend - 1);
    const uint32_t off = __builtin_amdgcn_readfirstlane(row0 * kRowBytes);
    dma16(kb + key * stride + c * 8, lk + off);
    dma16(vb + key * stride + c * 8, lv + off);
  }
}

// One wave-wide direct-to-LDS load with a scalar base: lane i's 16 bytes at
// gbase + voff land at lds_base + 16*i.
__device__ __forceinline__ void dma16_s(const void* gbase, uint32_t voff, uint32_t lds_base) {
  asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, %1"
               :
               : "v"(voff), "s"(gbase), "s"(lds_base)
               : "memory", "m0");
}
// The same with the non-temporal hint, for tiles that no other workgroup
// reads (one row group): the caches treat them as streaming.  With two or
// more row groups the tiles must stay in L2 for the other readers.
__device__ __forceinline__ void dma16_s_stream(const void* gbase, uint32_t voff, uint32_t lds_base) {
  asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, %1 nt"
               :
               : "v"(voff), "s"(gbase), "s"(lds_base)
               : "memory", "m0");
}

// The same share of a tile whose 64 keys are all below kend (no clamping):
// the row addresses are a scalar base plus lane offsets fixed per wave.
template <int WAVES, bool STREAM>
__device__ __forceinline__ void issue_tile_full(const uint16_t* kb, const uint16_t* vb, int k0, uint32_t lk,
                                                uint32_t lv, int wave, const uint32_t (&voff)[64 / WAVES / 4]) {
  constexpr int kRowsPerWave = kKeyTile / WAVES;
#pragma unroll
  for (int i = 0; i < kRowsPerWave / 4; ++i) {
    const int row0 = kRowsPerWave * wave + 4 * i;
    const size_t key0 = (size_t)(k0 + row0);
    if constexpr (STREAM) {
      dma16_s_stream(kb + key0 * kD, voff[i], lk + row0 * kRowBytes);
      dma16_s_stream(vb + key0 * kD, voff[i], lv + row0 * kRowBytes);
    } else {
      dma16_s(kb + key0 * kD, voff[i], lk + row0 * kRowBytes);
      dma16_s(vb + key0 * kD, voff[i], lv + row0 * kRowBytes);
    }
  }
}

// Wait for this wave's loads of the current tile, then for every wave's (the
// barrier).  LPW = loads per wave per tile; `later` tiles issued after the
// current one may stay in flight.  The asm memory clobber keeps LDS reads from
// moving above it.
template <int LPW>
__device__ __forceinline__ void wait_tile_and_sync(int later) {
  static_assert(2 * LPW < 64, "vmcnt holds 6 bits");
  if (later >= 2) asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)\n\ts_barrier" ::"n"(2 * LPW) : "memory");
  else if (later == 1) asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)\n\ts_barrier" ::"n"(LPW) : "memory");
  else asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

// STREAM: the context tiles are read by this workgroup alone (one row group)
// and are loaded with the non-temporal hint.
template <int NB, int WAVES, int KH, bool STREAM>
__global__ __launch_bounds__(WAVES * kWave, 1) void tree_verify_kernel(const VerifyArgs a) {
  static_assert(KH == 1 || (KH == 2 && WAVES == 8), "wave pairs share a SIMD: waves w and w + 4");
  constexpr int kThreads = WAVES * kWave;
  constexpr int kBlocks = WAVES / KH;   // 32-row blocks per workgroup
  constexpr int HP = 2 / KH;            // halves of each tile one wave consumes
  constexpr int kLoadsPerWave = 2 * kTileBytes / 1024 / WAVES;   // 1 KiB per wave-wide load
  __shared__ __attribute__((aligned(1024))) uint8_t smem[kStages * 2 * kTileBytes];
  __shared__ uint64_t s_mask[ADAPLD_MAX_TREE_NODES * kMaskWords];

  const int lane = lane_id();
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
  // Workgroups are dispatched round-robin over the 8 XCDs; the row groups of
  // one (kv head, split) get consecutive slots on the same XCD, so the second
  // reader of a K/V tile finds it in that XCD's L2.
  const int xcd = blockIdx.x & 7;
  const int slot = blockIdx.x >> 3;
  const int kvgroup = (slot / a.rowgroups) * 8 + xcd;   // = bg * nsplit + split
  const int rg = slot % a.rowgroups;
  if (kvgroup >= a.n_kvgroups) return;
  const int bg = kvgroup / a.nsplit;
  const int split = kvgroup - bg * a.nsplit;
  const int b = bg / a.Hkv;
  const int g = bg - b * a.Hkv;
  const int T = min(max(a.node_count[b], 0), a.T_max);
  const int L = min(max(a.lens[b], 0), a.L_stride);
  const int G = a.G;
  const int rows = T * G;
  const int row_base = rg * (kBlocks * NB * 32);
  if (row_base >= rows) return;
  // Row block of this wave, and (KH = 2) the half of every tile it takes.
  const int wrow = KH == 2 ? wave % kBlocks : wave;
  const int kh = KH == 2 ? wave / kBlocks : 0;

  const int c0 = split * a.chunk;
  const int c1 = min(c0 + a.chunk, L);
  const bool do_tree = split == a.nsplit - 1;
  const int col = lane & 31;
  const int half = lane >> 5;

  // Query fragments (B operand): lane holds dims [16*ds + 8*half, +8) of its row.
  bf16x8_t qf[NB][kD / 16];
  int qrow[NB], qu[NB], qh[NB];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    const int qr = row_base + (wrow * NB + nb) * 32 + col;
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
  }
  // The tree's mask rows go to registers here and to LDS once every load of
  // the prologue has landed (below), so they share one memory round trip with
  // the query loads and the first tiles.
  constexpr int kMaskRegs = (ADAPLD_MAX_TREE_NODES * kMaskWords + kThreads - 1) / kThreads;
  const int n_mask = do_tree ? T * a.nw : 0;
  uint64_t mw[kMaskRegs];
#pragma unroll
  for (int r = 0; r < kMaskRegs; ++r) {
    const int i = threadIdx.x + r * kThreads;
    mw[r] = i < n_mask ? a.tree_mask[(size_t)b * a.T_max * a.nw + i] : 0ull;
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

  const int n_ctx = c1 > c0 ? (c1 - c0 + kKeyTile - 1) / kKeyTile : 0;
  const int n_tiles = n_ctx + (do_tree ? (T + kKeyTile - 1) / kKeyTile : 0);
  const uint16_t* kc = a.k_ctx + (size_t)bg * a.L_stride * kD;
  const uint16_t* vc = a.v_ctx + (size_t)bg * a.L_stride * kD;
  const size_t tree_off = ((size_t)b * a.T_max * a.Hkv + g) * kD;
  const size_t tree_stride = (size_t)a.Hkv * kD;
  const uint32_t smem_base = lds_addr(smem);

  // The ring keeps the K tiles of the kStages stages in the first 64 KiB of
  // LDS and the V tiles in the next 64 KiB, so every fragment address below is
  // a lane offset plus an instruction immediate once the stage is known.
  constexpr int kVRegion = kStages * kTileBytes;
  constexpr int kRowsPerWave = kKeyTile / WAVES;
  uint32_t voff[kRowsPerWave / 4];
#pragma unroll
  for (int i = 0; i < kRowsPerWave / 4; ++i) {
    const int row = kRowsPerWave * wave + 4 * i + (lane >> 4);
    voff[i] = (lane >> 4) * kRowBytes + (((lane & 15) ^ swz(row)) << 4);
  }
  auto issue = [&](int t) {
    const uint32_t lk = smem_base + (t % kStages) * kTileBytes;
    const uint32_t lv = lk + kVRegion;
    if (t < n_ctx) {
      const int k0 = c0 + t * kKeyTile;
      if (k0 + kKeyTile <= c1)
        issue_tile_full<WAVES, STREAM>(kc, vc, k0, lk, lv, wave, voff);
      else
        issue_tile<WAVES>(kc, vc, kD, k0, c1, lk, lv, wave, lane);
    } else {
      issue_tile<WAVES>(a.k_tree + tree_off, a.v_tree + tree_off, tree_stride, (t - n_ctx) * kKeyTile, T,
                        lk, lv, wave, lane);
    }
  };
  // The first kStages - 1 tiles are requested together with the query and
  // mask loads above; all of them have landed after this wait (loads return
  // in order), and the barrier publishes the tiles and the mask table.
#pragma unroll
  for (int t = 0; t < kStages - 1; ++t)
    if (t < n_tiles) issue(t);
  waitcnt_vm<0>();
#pragma unroll
  for (int r = 0; r < kMaskRegs; ++r) {
    const int i = threadIdx.x + r * kThreads;
    if (i < n_mask) s_mask[i] = mw[r];
  }
  __syncthreads();

  // Lane-dependent LDS byte offsets within a stage.  K fragment for dims
  // [16*ds + 8*half, +8) of key row kb*32 + col sits at kofs[ds] + kb*32*kRowBytes.
  // Transposed V reads: each 16-lane group covers 4 keys x 16 dims; the key rows
  // are kb*32 + 16*s2 + vkey (+8), whose swizzle depends on vkey only.  vofs
  // include the offset of the V region.
  // With KH = 2 the offsets also hold the 32-row offset of the wave's half
  // of the tile (the swizzle has period 16 rows, so it is unchanged).
  const int half_off = kh * 32 * kRowBytes;
  int kofs[kD / 16];
#pragma unroll
  for (int ds = 0; ds < kD / 16; ++ds)
    kofs[ds] = half_off + col * kRowBytes + (((2 * ds + half) ^ swz(col)) << 4);
  const int vkey = 4 * half + ((lane & 15) >> 2);
  const int vdim = (lane & 16) + 4 * (lane & 3);
  int vofs[2][kD / 32];
#pragma unroll
  for (int db = 0; db < kD / 32; ++db) {
    const int cch = (db * 32 + vdim) >> 3;
    vofs[0][db] = half_off + kVRegion + vkey * kRowBytes + ((cch ^ swz(vkey)) << 4) + (vdim & 7) * 2;
    vofs[1][db] = half_off + kVRegion + (vkey + 8) * kRowBytes + ((cch ^ swz(vkey + 8)) << 4) + (vdim & 7) * 2;
  }
  const float sl2 = a.scale_log2;

  static_assert(NB == 1, "software-pipelined loop handles one 32-row block per wave");
  // The wave's half h lies in tile h / HP, which sits in stage (h / HP) % kStages.
  // With KH = 1 it covers keys [32*(h&1), +32) of that tile; with KH = 2 the
  // wave's own half, whose offset is already in kofs and vofs.
  auto kstage = [&](int h) {
    return (const lds_u8*)smem + ((h / HP) & (kStages - 1)) * kTileBytes + (HP == 2 ? (h & 1) : 0) * 32 * kRowBytes;
  };
  auto qk = [&](int h, f32x16_t& sacc) {
    const lds_u8* kbase = kstage(h);
    sacc = f32x16_t{};
#pragma unroll
    for (int ds = 0; ds < kD / 16; ++ds) {
      const bf16x8_t ka = *reinterpret_cast<const lds_bf16x8_t*>(kbase + kofs[ds]);
      sacc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka, qf[0][ds], sacc, 0, 0, 0);
    }
  };
  // Fixed-half variants: HS = half index modulo HP * kStages.
  auto half_base = [&](auto HS) {
    constexpr int hs = decltype(HS)::value;
    return (const lds_u8*)smem + ((hs / HP) & (kStages - 1)) * kTileBytes + (HP == 2 ? (hs & 1) : 0) * 32 * kRowBytes;
  };
  auto qk_c = [&](auto HS, f32x16_t& sacc) {
    const lds_u8* kbase = half_base(HS);
    sacc = f32x16_t{};
#pragma unroll
    for (int ds = 0; ds < kD / 16; ++ds) {
      const bf16x8_t ka = *reinterpret_cast<const lds_bf16x8_t*>(kbase + kofs[ds]);
      sacc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka, qf[0][ds], sacc, 0, 0, 0);
    }
  };
  auto pv_c = [&](auto HS, const bf16x8_t (&pbv)[2]) {
    const lds_u8* vbase = half_base(HS);
#pragma unroll
    for (int s2 = 0; s2 < 2; ++s2) {
#pragma unroll
      for (int db = 0; db < kD / 32; ++db) {
        const lds_u8* vb2 = vbase + 16 * s2 * kRowBytes;
        const s16x4_t lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4_t*)(vb2 + vofs[0][db]));
        const s16x4_t hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4_t*)(vb2 + vofs[1][db]));
        const s16x8_t vv = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
        o[0][db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, vv), pbv[s2], o[0][db], 0, 0, 0);
      }
    }
  };
  auto pv = [&](int h, const bf16x8_t (&pbv)[2]) {
    const lds_u8* vbase = kstage(h);   // vofs include the V region
#pragma unroll
    for (int s2 = 0; s2 < 2; ++s2) {
#pragma unroll
      for (int db = 0; db < kD / 32; ++db) {
        const lds_u8* vb2 = vbase + 16 * s2 * kRowBytes;
        const s16x4_t lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4_t*)(vb2 + vofs[0][db]));
        const s16x4_t hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4_t*)(vb2 + vofs[1][db]));
        const s16x8_t vv = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
        o[0][db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, vv), pbv[s2], o[0][db], 0, 0, 0);
      }
    }
  };
  // Mask (masked tiles only), row max, and the lazy rescale of the running state.
  auto max_rescale = [&](int h, f32x16_t& sv, auto masked) {
    if constexpr (decltype(masked)::value) {
      const int t = h / HP, kb = HP == 2 ? (h & 1) : kh;
      const bool is_tree = t >= n_ctx;
      const int k0 = is_tree ? (t - n_ctx) * kKeyTile : c0 + t * kKeyTile;
      const int kend = is_tree ? T : c1;
      const uint64_t mword = (is_tree && qrow[0] < rows) ? s_mask[qu[0] * a.nw + (k0 >> 6)] : 0ull;
      // Bit 8*(r/4) + r%4 of mbits is the mask bit of this lane's key r.
      const uint32_t mbits = (uint32_t)(mword >> (kb * 32 + 4 * half));
      const int kbase = k0 + kb * 32 + 4 * half;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int kr = 8 * (r >> 2) + (r & 3);   // key kbase + kr
        const bool ok = kbase + kr < kend && (!is_tree || ((mbits >> kr) & 1u));
        sv[r] = ok ? sv[r] : -INFINITY;
      }
    }
    float mx = fmaxf(fmaxf(sv[0], sv[1]), sv[2]);
#pragma unroll
    for (int r = 3; r < 15; r += 2) mx = fmaxf(fmaxf(mx, sv[r]), sv[r + 1]);
    mx = fmaxf(mx, sv[15]);
    {
      const auto sw2 = __builtin_amdgcn_permlane32_swap(__float_as_int(mx), __float_as_int(mx), false, false);
      mx = fmaxf(__int_as_float(sw2[0]), __int_as_float(sw2[1]));
    }
    const float mt = mx * sl2;  // scale > 0, so the max commutes with scaling
    if (__ballot(mt > m_run[0] + kRescaleSlack)) {
      const float m_new = fmaxf(m_run[0], mt);
      const float alpha = m_new == m_run[0] ? 1.f : __builtin_amdgcn_exp2f(m_run[0] - m_new);
      m_run[0] = m_new;
      l_run[0] *= alpha;
#pragma unroll
      for (int db = 0; db < kD / 32; ++db) o[0][db] *= alpha;
    }
  };
  // P = exp2(S*scale - m) packed to bf16 in MFMA B-operand order.
  auto exp_pack = [&](const f32x16_t& sv, bf16x8_t (&pbv)[2]) {
    const float m_use = m_run[0] == -INFINITY ? 0.f : m_run[0];
    float psum = 0.f;
#pragma unroll
    for (int s2 = 0; s2 < 2; ++s2) {
      bf16x8_t v;
#pragma unroll
      for (int i = 0; i < 8; i += 2) {
        const float p0 = __builtin_amdgcn_exp2f(fmaf(sv[8 * s2 + i], sl2, -m_use));
        const float p1 = __builtin_amdgcn_exp2f(fmaf(sv[8 * s2 + i + 1], sl2, -m_use));
        psum += p0 + p1;
        const bf16x2_t pk = __builtin_convertvector((f32x2_t){p0, p1}, bf16x2_t);
        v[i] = pk[0];
        v[i + 1] = pk[1];
      }
      pbv[s2] = v;
    }
    l_run[0] += psum;
  };
  // Pieces of the same two steps for the unrolled loop below: the row max in
  // log2 units, the rescale to a new max, and the exponentials of one 16-key
  // part (s2) of the half, adding to psum in the order exp_pack uses.
  auto row_max = [&](const f32x16_t& sv) {
    float mx = fmaxf(fmaxf(sv[0], sv[1]), sv[2]);
#pragma unroll
    for (int r = 3; r < 15; r += 2) mx = fmaxf(fmaxf(mx, sv[r]), sv[r + 1]);
    mx = fmaxf(mx, sv[15]);
    const auto sw2 = __builtin_amdgcn_permlane32_swap(__float_as_int(mx), __float_as_int(mx), false, false);
    mx = fmaxf(__int_as_float(sw2[0]), __int_as_float(sw2[1]));
    return mx * sl2;
  };
  auto rescale_to = [&](float mt) {
    const float m_new = fmaxf(m_run[0], mt);
    const float alpha = m_new == m_run[0] ? 1.f : __builtin_amdgcn_exp2f(m_run[0] - m_new);
    m_run[0] = m_new;
    l_run[0] *= alpha;
#pragma unroll
    for (int db = 0; db < kD / 32; ++db) o[0][db] *= alpha;
  };
  auto exp_part = [&](const f32x16_t& sv, int s2, float m_use, bf16x8_t& pbv, float& psum) {
    bf16x8_t v;
#pragma unroll
    for (int i = 0; i < 8; i += 2) {
      const float p0 = __builtin_amdgcn_exp2f(fmaf(sv[8 * s2 + i], sl2, -m_use));
      const float p1 = __builtin_amdgcn_exp2f(fmaf(sv[8 * s2 + i + 1], sl2, -m_use));
      psum += p0 + p1;
      const bf16x2_t pk = __builtin_convertvector((f32x2_t){p0, p1}, bf16x2_t);
      v[i] = pk[0];
      v[i + 1] = pk[1];
    }
    pbv = v;
  };
  // Before the first half of tile t+1: wait for its loads, then the barrier.
  // Every wave has passed the last read of tile t-1 by then, so its stage is
  // refilled with tile t+kStages-1.
  auto next_tile = [&](int t) {
    wait_tile_and_sync<kLoadsPerWave>(min(kStages - 3, n_tiles - 2 - t));
    if (t + kStages - 1 < n_tiles) issue(t + kStages - 1);
  };

  // Software pipeline over halves: while the softmax of half h runs on the
  // VALU, the MFMAs of PV(h-1) and of S(h+1) are in flight.
  const int H = HP * n_tiles;
  const int n_plain = max(c1 - c0, 0) / kKeyTile;   // leading context tiles with no masked key
  const int H_plain = HP * n_plain;
  // A wave whose row block holds no valid row (the tail of the last row
  // group) issues its share of every tile and takes every barrier, and does
  // no math: its MFMAs would only cost power.
  const bool idle = row_base + wrow * NB * 32 >= rows;
  if (idle && H > 0) {
    wait_tile_and_sync<kLoadsPerWave>(min(kStages - 2, n_tiles - 1));
    if (HP == 1 && H > 1) next_tile(0);
    for (int h = 1; h < H; ++h)
      if (h % HP == HP - 1 && h + 1 < H) next_tile(h / HP);
  } else if (H > 0) {
    f32x16_t s_cur, s_nxt;
    bf16x8_t pb[2];
    wait_tile_and_sync<kLoadsPerWave>(min(kStages - 2, n_tiles - 1));
    qk(0, s_cur);
    if (H_plain > 0) max_rescale(0, s_cur, std::false_type{});
    else max_rescale(0, s_cur, std::true_type{});
    if (HP == 1 && H > 1) next_tile(0);   // half 1 is in tile 1
    qk(1, s_nxt);
    exp_pack(s_cur, pb);
    s_cur = s_nxt;
    auto body = [&](int h, auto masked) {
      pv(h - 1, pb);
      max_rescale(h, s_cur, masked);
      if (h % HP == HP - 1 && h + 1 < H) next_tile(h / HP);
      qk(h + 1, s_nxt);        // past the last half this reads a stale stage; unused
      exp_pack(s_cur, pb);
      s_cur = s_nxt;
    };
    // The same step for an unmasked half whose index modulo kPeriod (HP
    // halves per stage, kStages stages) is the compile-time J: every LDS
    // address is then a lane offset plus an immediate.
    constexpr int kPeriod = HP * kStages;
    // Its softmax is split so that each side of the tile barrier pairs eight
    // MFMAs with about half of the VALU work: the exponentials of the first
    // 16 keys go beside the MFMAs of P V (h-1), those of the last 16 beside
    // the MFMAs of S (h+1).  They use the running max as it stands; the rare
    // half whose max outgrows it by more than kRescaleSlack is recomputed
    // after the check (the same values the check-first order gives).
    auto body_c = [&](auto J, int h) {
      constexpr int j = decltype(J)::value;
      pv_c(std::integral_constant<int, (j + kPeriod - 1) % kPeriod>{}, pb);
      const float mt = row_max(s_cur);
      const float m_use = m_run[0] == -INFINITY ? 0.f : m_run[0];
      float psum = 0.f;
      bf16x8_t pn[2];
      exp_part(s_cur, 0, m_use, pn[0], psum);
      // Empty asm statements that consume the values pin each part to its
      // side of the barrier: otherwise the compiler sinks both parts below
      // the rescale check, whose rare branch does not need them.
      asm volatile("" ::"v"(pn[0]), "v"(psum));
      if (j % HP == HP - 1 && h + 1 < H) next_tile(h / HP);
      qk_c(std::integral_constant<int, (j + 1) % kPeriod>{}, s_nxt);
      exp_part(s_cur, 1, m_use, pn[1], psum);
      asm volatile("" ::"v"(pn[1]), "v"(psum));
      if (__ballot(mt > m_run[0] + kRescaleSlack)) {
        rescale_to(mt);
        psum = 0.f;
        exp_part(s_cur, 0, m_run[0], pn[0], psum);
        exp_part(s_cur, 1, m_run[0], pn[1], psum);
      }
      l_run[0] += psum;
      pb[0] = pn[0];
      pb[1] = pn[1];
      s_cur = s_nxt;
    };
    using I1 = std::integral_constant<int, 1>;
    using I2 = std::integral_constant<int, 2>;
    using I3 = std::integral_constant<int, 3>;
    using I4 = std::integral_constant<int, 4>;
    using I5 = std::integral_constant<int, 5>;
    using I6 = std::integral_constant<int, 6>;
    using I7 = std::integral_constant<int, 7>;
    using I0 = std::integral_constant<int, 0>;
    int h = 1;
    if constexpr (kPeriod == 8) {
      for (; h + 8 <= H_plain; h += 8) {   // h = 1 (mod 8) here
        body_c(I1{}, h);
        body_c(I2{}, h + 1);
        body_c(I3{}, h + 2);
        body_c(I4{}, h + 3);
        body_c(I5{}, h + 4);
        body_c(I6{}, h + 5);
        body_c(I7{}, h + 6);
        body_c(I0{}, h + 7);
      }
    } else {
      static_assert(kPeriod == 4, "one or two halves per tile, four stages");
      for (; h + 4 <= H_plain; h += 4) {   // h = 1 (mod 4) here
        body_c(I1{}, h);
        body_c(I2{}, h + 1);
        body_c(I3{}, h + 2);
        body_c(I0{}, h + 3);
      }
    }
    for (; h < H_plain; ++h) body(h, std::false_type{});
    for (; h < H; ++h) body(h, std::true_type{});
    pv(H - 1, pb);
  }

  // Epilogue: lane holds dims db*32 + 8*(r/4) + 4*half + r%4 of its query row.
  float l_tot[NB];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) l_tot[nb] = l_run[nb] + __shfl_xor(l_run[nb], 32, kWave);
  if constexpr (KH == 2) {
    // The pair (wrow, kh = 1) hands its state to (wrow, kh = 0) through the
    // ring, which no wave reads any more after this barrier; lane i of both
    // waves holds the same query column.  Each state is relative to its own
    // running max: the merged one takes M = max(m0, m1) and weights 2^(m - M).
    static_assert(NB == 1, "one row block per wave");
    float4* xo = reinterpret_cast<float4*>(smem);                        // [kBlocks][16][64]
    float2* xml = reinterpret_cast<float2*>(smem + kBlocks * 16 * 64 * 16);   // [kBlocks][64]
    __syncthreads();
    if (kh == 1) {
#pragma unroll
      for (int db = 0; db < kD / 32; ++db)
#pragma unroll
        for (int r4 = 0; r4 < 4; ++r4)
          xo[(wrow * 16 + db * 4 + r4) * 64 + lane] =
              make_float4(o[0][db][4 * r4], o[0][db][4 * r4 + 1], o[0][db][4 * r4 + 2], o[0][db][4 * r4 + 3]);
      xml[wrow * 64 + lane] = make_float2(m_run[0], l_tot[0]);
    }
    __syncthreads();
    if (kh == 1) return;
    const float2 ml = xml[wrow * 64 + lane];
    const float M = fmaxf(m_run[0], ml.x);
    const float a0 = m_run[0] == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(m_run[0] - M);
    const float a1 = ml.x == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(ml.x - M);
#pragma unroll
    for (int db = 0; db < kD / 32; ++db)
#pragma unroll
      for (int r4 = 0; r4 < 4; ++r4) {
        const float4 v = xo[(wrow * 16 + db * 4 + r4) * 64 + lane];
        o[0][db][4 * r4 + 0] = a0 * o[0][db][4 * r4 + 0] + a1 * v.x;
        o[0][db][4 * r4 + 1] = a0 * o[0][db][4 * r4 + 1] + a1 * v.y;
        o[0][db][4 * r4 + 2] = a0 * o[0][db][4 * r4 + 2] + a1 * v.z;
        o[0][db][4 * r4 + 3] = a0 * o[0][db][4 * r4 + 3] + a1 * v.w;
      }
    l_tot[0] = a0 * l_tot[0] + a1 * ml.y;
    m_run[0] = M;
  }
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    const int qr = qrow[nb];
    if (qr >= rows) continue;
    const int u = qu[nb], h = qh[nb];
    if (a.nsplit == 1) {
      const float inv = 1.f / l_tot[nb];
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
      if (half == 0 && a.lse) a.lse[((size_t)b * a.Hq + h) * a.T_max + u] = (m_run[nb] + log2f(l_tot[nb])) * kLn2;
    } else {
      const size_t slot = ((size_t)bg * a.nsplit + split) * a.rows_max + qr;
      const float inv = l_tot[nb] > 0.f ? 1.f / l_tot[nb] : 0.f;
      uint16_t* wp = a.ws_o + slot * kD;
#pragma unroll
      for (int db = 0; db < kD / 32; ++db)
#pragma unroll
        for (int r4 = 0; r4 < 4; ++r4) {
          const int dim = db * 32 + 8 * r4 + 4 * half;
          uint2 pk;
          pk.x = f32_to_bf16_bits(o[nb][db][4 * r4 + 0] * inv) | (f32_to_bf16_bits(o[nb][db][4 * r4 + 1] * inv) << 16);
          pk.y = f32_to_bf16_bits(o[nb][db][4 * r4 + 2] * inv) | (f32_to_bf16_bits(o[nb][db][4 * r4 + 3] * inv) << 16);
          *reinterpret_cast<uint2*>(wp + dim) = pk;
        }
      if (half == 0) a.ws_ml[slot] = make_float2(m_run[nb], l_tot[nb]);
    }
  }
}

// Merge the splits: 8 stacked rows per workgroup, 16 threads x 8 dims (one
// 16-byte load per split) per row.
constexpr int kCombineRows = 8;
__global__ __launch_bounds__(kCombineRows * 16) void verify_combine_kernel(const VerifyArgs a) {
  const int qr = blockIdx.x * kCombineRows + (threadIdx.x >> 4);
  const int bg = blockIdx.y;
  if (qr >= a.rows_max) return;
  const int dim = (threadIdx.x & 15) * 8;
  const size_t row0 = (size_t)bg * a.nsplit * a.rows_max + qr;   // split 0 of this row
  const int b = bg / a.Hkv;
  const int T = min(max(a.node_count[b], 0), a.T_max);
  // One pass over the splits in index order, four at a time.  The maxima and
  // partials of a group are loaded together, and with node_count rather than
  // after it (every slot is in bounds; rows past the tree are dropped at the
  // end), so a call with up to four splits costs one memory round trip; the
  // running max moves online.  Split s carries O_s/l_s with weight
  // l_s 2^(m_s - M).
  float M = -INFINITY, den = 0.f;
  float num[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  for (int s0 = 0; s0 < a.nsplit; s0 += 4) {
    float2 ml[4];
    uint4 v[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const bool in = s0 + j < a.nsplit;
      const size_t slot = row0 + (size_t)(s0 + j) * a.rows_max;
      ml[j] = in ? a.ws_ml[slot] : make_float2(-INFINITY, 0.f);
      v[j] = in ? *reinterpret_cast<const uint4*>(a.ws_o + slot * kD + dim) : make_uint4(0u, 0u, 0u, 0u);
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      if (ml[j].y > 0.f) {
        const float m_new = fmaxf(M, ml[j].x);
        const float c = exp2f(M - m_new);   // 0 while nothing has been merged
        const float w = ml[j].y * exp2f(ml[j].x - m_new);
        const uint32_t wv[4] = {v[j].x, v[j].y, v[j].z, v[j].w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          num[2 * e] = num[2 * e] * c + w * bf16_lo(wv[e]);
          num[2 * e + 1] = num[2 * e + 1] * c + w * bf16_hi(wv[e]);
        }
        den = den * c + w;
        M = m_new;
      }
    }
  }
  if (qr >= T * a.G) return;
  const int g = bg - b * a.Hkv;
  const int u = qr / a.G;
  const int h = g * a.G + (qr - u * a.G);
  const float inv = 1.f / den;
  uint4 pk;
  pk.x = f32_to_bf16_bits(num[0] * inv) | (f32_to_bf16_bits(num[1] * inv) << 16);
  pk.y = f32_to_bf16_bits(num[2] * inv) | (f32_to_bf16_bits(num[3] * inv) << 16);
  pk.z = f32_to_bf16_bits(num[4] * inv) | (f32_to_bf16_bits(num[5] * inv) << 16);
  pk.w = f32_to_bf16_bits(num[6] * inv) | (f32_to_bf16_bits(num[7] * inv) << 16);
  *reinterpret_cast<uint4*>(a.out + (((size_t)b * a.T_max + u) * a.Hq + h) * kD + dim) = pk;
  if (dim == 0 && a.lse) a.lse[((size_t)b * a.Hq + h) * a.T_max + u] = (M + log2f(den)) * kLn2;
}

}  // namespace

VerifyPlan plan_verify(int B, int L_stride, int T_max, int Hq, int Hkv) {
  // Candidates: 8 waves each owning a 32-row block (256 rows per workgroup),
  // or 8 waves in SIMD pairs sharing a row block (128 rows, each wave half of
  // every tile).  Both keep two waves per SIMD, so one wave's softmax and LDS
  // waits overlap the other's MFMAs.  For each, and each number of context
  // splits, the estimated time is the
  // number of rounds of workgroups over the 256 CUs (one workgroup per CU:
  // the LDS ring takes 128 KiB) times one workgroup's time, which is its
  // per-SIMD share of row x key work plus a fixed start-up cost, plus the
  // combine kernel when the context is split.  The constants are in units of
  // one SIMD's time for 32 rows x 64 keys with two waves per SIMD.
  constexpr double kStartTiles = 12.0;    // start-up and drain of one workgroup
  constexpr double kCombineTiles = 6.0;   // the combine launch and its traffic
  // With more than one row group, every tile goes to LDS once per row group
  // (the second from L2) and must stay in L2 for it; with one row group the
  // tiles stream once, non-temporally (measured 4 % faster on 16 sequences of
  // 8192 keys with 32 query heads over 8 and 52-node trees).
  constexpr double kSharedTile = 0.1;
  struct Cand { int waves, kh; double per_tile; };   // per_tile: SIMD cost of one 64-key tile
  const Cand cands[] = {{8, 1, 2.0}, {8, 2, 1.0}};
  const int G = Hq / Hkv;
  const int rows_max = T_max * G;
  // A split holds at least one tile; small grids (one short sequence) gain
  // from splits of one or two tiles, since their time is mostly start-up.
  const int max_split = std::min(64, std::max(1, (L_stride + kKeyTile - 1) / kKeyTile));
  VerifyPlan best{};
  double best_cost = 0.0;
  for (const Cand& c : cands) {
    const int rows_per_wg = c.waves / c.kh * 32;
    const int rowgroups = (rows_max + rows_per_wg - 1) / rows_per_wg;
    for (int want = 1; want <= max_split; ++want) {
      int chunk = (L_stride + want - 1) / want;
      chunk = std::max(((chunk + kKeyTile - 1) / kKeyTile) * kKeyTile, kKeyTile);
      const int nsplit = std::max(1, (L_stride + chunk - 1) / chunk);
      if (nsplit != want) continue;   // the same split as a smaller count
      const long wgs = (long)B * Hkv * rowgroups * nsplit;
      const long rounds = (wgs + 255) / 256;
      const double tiles = (double)chunk / kKeyTile + (T_max + kKeyTile - 1) / kKeyTile;
      const double cost = rounds * ((c.per_tile + (rowgroups > 1 ? kSharedTile : 0.0)) * tiles + kStartTiles) +
                          (nsplit > 1 ? kCombineTiles : 0.0);
      if (best.waves == 0 || cost < best_cost) {
        best_cost = cost;
        best.G = G;
        best.rows_max = rows_max;
        best.nb = 1;
        best.waves = c.waves;
        best.kh = c.kh;
        best.rows_per_wg = rows_per_wg;
        best.rowgroups = rowgroups;
        best.nsplit = nsplit;
        best.chunk = chunk;
      }
    }
  }
  return best;
}

size_t verify_ws_bytes(const VerifyPlan& p, int B, int Hkv) {
  if (p.nsplit <= 1) return 0;
  const size_t slots = (size_t)B * Hkv * p.nsplit * p.rows_max;
  return slots * kD * sizeof(uint16_t) + slots * sizeof(float2);
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
  a.ws_o = static_cast<uint16_t*>(ws);
  a.ws_ml = ws ? reinterpret_cast<float2*>(static_cast<char*>(ws) + slots * kD * sizeof(uint16_t)) : nullptr;

  a.rowgroups = p.rowgroups;
  a.n_kvgroups = B * Hkv * p.nsplit;
  const dim3 grid(((a.n_kvgroups + 7) / 8) * 8 * p.rowgroups);
  // Streaming loads pay only with whole-workgroup row blocks over long chunks:
  // measured slower for the two-wave row blocks of short chunks.
  if (p.kh == 2)
    hipLaunchKernelGGL((tree_verify_kernel<1, 8, 2, false>), grid, dim3(8 * kWave), 0, stream, a);
  else if (p.rowgroups == 1)
    hipLaunchKernelGGL((tree_verify_kernel<1, 8, 1, true>), grid, dim3(8 * kWave), 0, stream, a);
  else
    hipLaunchKernelGGL((tree_verify_kernel<1, 8, 1, false>), grid, dim3(8 * kWave), 0, stream, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || p.nsplit == 1) return e;
  hipLaunchKernelGGL(verify_combine_kernel, dim3((p.rows_max + kCombineRows - 1) / kCombineRows, B * Hkv),
                     dim3(kCombineRows * 16), 0, stream, a);
  return hipGetLastError();
}

}  // namespace adapld
