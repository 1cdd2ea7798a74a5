// noalloc.hip -- msa_forward_noalloc: msa_forward for callers that cannot
// allocate device memory (code under HIP graph capture, tight serving
// loops, harnesses that forbid hipMalloc).
//
// Its workspace is `scratch`, a file-scope device array of
// MSA_NOALLOC_WORKSPACE_BYTES: each device the library runs on holds its own
// copy until the process ends, shared by every such call on that device (so
// calls that overlap on one device race).  In host code `scratch` only
// stands for the symbol; its device address comes from hipGetSymbolAddress,
// looked up on the first call on each device with that device current and
// kept in g_scratch.  Nothing here allocates or frees memory.
#include <hip/hip_runtime.h>

#include <cstdint>
#include <mutex>
#include <string>

#include "errors.h"
#include "forward.h"
#include "msa.h"

namespace {

constexpr uint64_t kScratchBytes = MSA_NOALLOC_WORKSPACE_BYTES;
static __device__ __align__(256) char scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch[kMaxDevices] = {};

msa_status fail(msa_status st, const std::string& msg) {
  msa::set_last_error("msa_forward_noalloc: " + msg);
  return st;
}

// Device address of the current device's scratch array.
msa_status scratch_address(void** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) {
    (void)hipGetLastError();
    return fail(MSA_ERR_DEVICE, "no usable current device");
  }
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch[dev]) {
    void* ptr = nullptr;
    const hipError_t e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !ptr) {
      (void)hipGetLastError();
      return fail(MSA_ERR_DEVICE, std::string("hipGetSymbolAddress of the scratch array failed: ") +
                                      hipGetErrorString(e));
    }
    g_scratch[dev] = ptr;
  }
  *out = g_scratch[dev];
  return MSA_OK;
}

}  // namespace

extern "C" msa_status msa_forward_noalloc(msa_plan_t plan, const void* q, const void* k_cache,
                                          const void* v_cache, const int32_t* block_table, void* o,
                                          float* lse, void* hip_stream) {
  if (!plan) return fail(MSA_ERR_INVALID_ARG, "null plan");
  const int64_t need = msa::plan_workspace_bytes(plan);
  if ((uint64_t)need > kScratchBytes)
    return fail(MSA_ERR_UNSUPPORTED, "the plan needs " + std::to_string(need) +
                                         " bytes of workspace, more than the " +
                                         std::to_string(kScratchBytes) +
                                         " bytes of the library's scratch array (use msa_forward)");
  void* ws = nullptr;
  if (need > 0) {
    const msa_status st = scratch_address(&ws);
    if (st != MSA_OK) return st;
  }
  return msa::forward_impl("msa_forward_noalloc", plan, q, k_cache, v_cache, block_table, o, lse, ws,
                           ws ? (size_t)kScratchBytes : 0, hip_stream);
}
