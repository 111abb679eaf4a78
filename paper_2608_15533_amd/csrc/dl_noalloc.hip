// Allocation-free entry point: the split-replay value-tiled step with its replay
// coefficients in a fixed device-resident scratch array instead of a caller workspace.
//
// The array lives in this translation unit's code object, one copy per GPU, allocated
// by the HIP runtime when the code object is loaded and kept until the process ends.
// Host code never passes the array's name to a kernel (on the host it is only a
// stand-in for the symbol): its device address is looked up once per device with
// hipGetSymbolAddress, with that device current, and that address is what the kernels
// receive, exactly as they receive the caller's workspace in dl_append_step_tiled.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <mutex>

#include "deltalog.h"
#include "dl_internal.h"

namespace {

constexpr size_t kScratchBytes = DL_NOALLOC_SCRATCH_BYTES;
static_assert(kScratchBytes % 256 == 0, "whole 256-byte blocks");

static __device__ __align__(256) float scratch[kScratchBytes / sizeof(float)];

constexpr int kMaxDevices = 64;
std::mutex g_mu;
void* g_scratch[kMaxDevices] = {};   // device address of `scratch` on each device

// The current device's scratch address, looked up on the first call on that device.
int scratch_address(float** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess) return DL_E_HIP;
  if (dev < 0 || dev >= kMaxDevices) return DL_E_UNSUPPORTED;
  std::lock_guard<std::mutex> lock(g_mu);
  if (!g_scratch[dev]) {
    void* ptr = nullptr;
    const hipError_t e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !ptr) return DL_E_HIP;
    g_scratch[dev] = ptr;
  }
  *out = static_cast<float*>(g_scratch[dev]);
  return DL_OK;
}

}  // namespace

extern "C" int dl_append_step_tiled_noalloc(const dl_desc* desc, const dl_state* state,
                                            const dl_token* tok, float* o,
                                            const int32_t* slots, int32_t n,
                                            int32_t value_tiles, hipStream_t stream) {
  int rc = dl::tiled_check(desc, state, tok, o, slots, n, value_tiles);
  if (rc != DL_OK) return rc;
  if (n == 0) return DL_OK;
  size_t need = 0;
  rc = dl_tiled_workspace_bytes(desc, n, &need);
  if (rc != DL_OK) return rc;
  if (need > kScratchBytes) return DL_E_SCRATCH;
  float* coef = nullptr;
  if (need > 0) {                       // M == 1: no log, no coefficients, no scratch
    rc = scratch_address(&coef);
    if (rc != DL_OK) return rc;
  }
  // The prepare kernel writes the coefficients of every live entry before the tile
  // kernels (same stream) read exactly those entries: nothing needs clearing.
  return dl::tiled_launch(desc, state, tok, o, slots, n, value_tiles, /*split=*/true, coef,
                          stream);
}
