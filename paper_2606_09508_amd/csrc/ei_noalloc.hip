// ei_entropy_guided_prefill_noalloc: the one-call layer path for callers that
// cannot allocate device memory.  The probe workspace lives in a file-scope
// device array instead of a caller's buffer.
//
// In host code `scratch` names a host-side stand-in, not the device array:
// its device address is looked up once per device with hipGetSymbolAddress
// (with that device current) and only that address is ever passed on.  Every
// call on a device shares the device's array; it keeps the previous call's
// contents, which the probe overwrites before reading (nothing in it needs to
// start at zero).  Calls that overlap on one device race on it.
#include "../../include/entropyinfer.h"
#include "ei_internal.h"

#include <mutex>

namespace {

constexpr size_t kScratchBytes = EI_NOALLOC_SCRATCH_BYTES;
constexpr int kMaxDevices = 64;

__device__ __align__(256) unsigned char scratch[kScratchBytes];

std::mutex g_mu;
void* g_addr[kMaxDevices] = {};

// The current device's copy of `scratch`, looked up on the first call on that
// device; nullptr if the lookup fails.
void* scratch_address() {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
  std::lock_guard<std::mutex> lock(g_mu);
  if (!g_addr[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return nullptr;
    g_addr[dev] = p;
  }
  return g_addr[dev];
}

}  // namespace

extern "C" ei_status ei_entropy_guided_prefill_noalloc(
    const uint16_t* q, const uint16_t* k, const uint16_t* v, ei_dims dims, ei_tiling tiling,
    double probe_scale, ei_budget_params params, int32_t mode, int32_t kmax, float softmax_scale,
    float* log_scores, float* entropy, uint8_t* head_is_rigid, int32_t* budget_blocks,
    int32_t* block_idx, int32_t* block_cnt, uint16_t* o, void* stream) {
  // Every argument check of the workspace entry point first, without a
  // workspace: a valid, non-empty problem then stops at the workspace check
  // (the last one) and nothing has been launched or looked up.
  ei_status st = ei_entropy_guided_prefill(
      q, k, v, dims, tiling, probe_scale, params, mode, kmax, softmax_scale, log_scores, entropy,
      head_is_rigid, budget_blocks, block_idx, block_cnt, o, nullptr, 0, stream);
  if (st != EI_ERR_WORKSPACE) return st;
  if (ei_prefill_workspace_bytes(dims, tiling) > kScratchBytes) return EI_ERR_WORKSPACE;
  void* ws = scratch_address();
  if (!ws) return EI_ERR_LAUNCH;
  return ei_entropy_guided_prefill(q, k, v, dims, tiling, probe_scale, params, mode, kmax,
                                   softmax_scale, log_scores, entropy, head_is_rigid,
                                   budget_blocks, block_idx, block_cnt, o, ws, kScratchBytes,
                                   stream);
}
