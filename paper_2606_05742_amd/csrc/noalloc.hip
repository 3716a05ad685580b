// adapld_step_noalloc: one draft-and-verify step whose workspace is a device
// array of this library instead of caller memory, for callers that cannot
// allocate (code under HIP graph capture, serving loops that forbid
// allocation).  It validates and enqueues exactly what adapld_step does.
//
// `scratch` is file-scope device memory of kScratchBytes per GPU, held from
// the first call on that GPU until the process ends.  Host code never uses
// the array's name as an address: the first call on a device (with that
// device current) looks up the device's own copy with hipGetSymbolAddress,
// and every later call on that device passes the stored address.  Calls that
// overlap in time on one GPU share the array and race; the step needs no
// part of it cleared (every byte it reads was written earlier in the same
// call).
#include <mutex>

#include "adapld_internal.h"

namespace {

constexpr size_t kScratchBytes = ADAPLD_NOALLOC_SCRATCH_BYTES;
constexpr int kMaxDevices = 64;

static __device__ __align__(256) unsigned char scratch[kScratchBytes];

std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices];   // device address of scratch per device (set once, under the mutex)

// The current device's address of scratch, looked up on the first call.
hipError_t scratch_on_current_device(void** ptr) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    g_scratch_ptr[dev] = p;
  }
  *ptr = g_scratch_ptr[dev];
  return hipSuccess;
}

}  // namespace

extern "C" int adapld_step_noalloc(
    const int32_t* tokens, const int32_t* lens, const uint16_t* bank, const uint16_t* query, const uint16_t* q,
    const uint16_t* k_ctx, const uint16_t* v_ctx, const uint16_t* k_tree, const uint16_t* v_tree, int B,
    int L_stride, int d, int n_max, int k, int W, int S, int T_max, int Hq, int Hkv, int D, float tau,
    int preceding, float scale, int32_t* cand_pos, int32_t* cand_count, int32_t* match_n, int32_t* topk_pos,
    float* topk_score, int32_t* topk_count, int32_t* kind, int32_t* node_token, int32_t* node_parent,
    int32_t* node_depth, int32_t* node_src, int32_t* node_count, uint64_t* tree_mask, uint16_t* out,
    float* lse, hipStream_t stream) {
  if (B < 0) return ADAPLD_ERR_INVALID_ARG;
  if (B == 0) return ADAPLD_OK;
  // Sizes adapld_workspace_bytes rejects (0) are reported by adapld_step's
  // own checks below; a workspace beyond the array is refused here.
  if (adapld_workspace_bytes(ADAPLD_OP_STEP, B, L_stride, d, k, T_max, Hq, Hkv, D) > kScratchBytes)
    return ADAPLD_ERR_WORKSPACE_TOO_SMALL;
  void* ws = nullptr;
  const hipError_t e = scratch_on_current_device(&ws);
  if (e != hipSuccess) return adapld::record_hip_error(e);
  return adapld_step(tokens, lens, bank, query, q, k_ctx, v_ctx, k_tree, v_tree, B, L_stride, d, n_max, k, W,
                     S, T_max, Hq, Hkv, D, tau, preceding, scale, cand_pos, cand_count, match_n, topk_pos, topk_score,
                     topk_count, kind, node_token, node_parent, node_depth, node_src, node_count, tree_mask,
                     out, lse, ws, kScratchBytes, stream);
}
