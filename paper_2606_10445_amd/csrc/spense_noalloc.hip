// spense_gemm_noalloc: spense_gemm for callers that cannot allocate device memory.
//
// The only device memory spense_gemm needs beyond its inputs and outputs is the fp32
// partial sums of K-sliced plans (S x M x N floats, added by the reduction kernel of the
// same call).  Here they live in a file-scope device array that every device the library
// runs on holds until the process ends, so the call takes no workspace argument and makes
// no allocation.  The plan, the kernels and therefore the results are spense_gemm's, bit
// for bit.
#include <hip/hip_runtime.h>

#include <mutex>

#include "spense.h"
#include "spense_internal.h"

namespace {

constexpr size_t kScratchBytes = SPENSE_NOALLOC_SCRATCH_BYTES;

// In host code `scratch` is a host-side stand-in for the array, not a device address:
// the device address comes from hipGetSymbolAddress, once per device with that device
// current, and only that address is handed to kernels.
__device__ __align__(256) uint8_t scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
std::once_flag g_once[kMaxDevices];
void* g_addr[kMaxDevices];
hipError_t g_rc[kMaxDevices];

// The device address of this device's scratch (looked up on the first call on it).
int scratch_address(void** out) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return spense::api_fail(SPENSE_ERR_HIP, "hipGetDevice failed");
  if (dev < 0 || dev >= kMaxDevices) return spense::api_fail(SPENSE_ERR_DEVICE, "device index %d out of range", dev);
  std::call_once(g_once[dev], [dev] { g_rc[dev] = hipGetSymbolAddress(&g_addr[dev], HIP_SYMBOL(scratch)); });
  if (g_rc[dev] != hipSuccess || !g_addr[dev])
    return spense::api_fail(SPENSE_ERR_HIP, "scratch address of device %d: %s", dev, hipGetErrorString(g_rc[dev]));
  *out = g_addr[dev];
  return SPENSE_OK;
}

}  // namespace

extern "C" int spense_gemm_noalloc(const void* X, int64_t M, int64_t ldx, const spense_packed_t* packed,
                                   const float* w_scale, const float* x_scale, void* Y, int64_t ldy,
                                   uint32_t out_flags, hipStream_t stream) {
  // spense_gemm_workspace_size is 0 for arguments spense_gemm rejects; it then reports them
  const size_t need = M > 0 ? spense_gemm_workspace_size(M, packed) : 0;
  if (need > kScratchBytes)
    return spense::api_fail(SPENSE_ERR_WS,
                            "this call needs %zu bytes of scratch; spense_gemm_noalloc holds %zu (call spense_gemm "
                            "with a workspace)",
                            need, kScratchBytes);
  void* ws = nullptr;
  size_t ws_bytes = 0;
  if (need > 0) {
    const int rc = scratch_address(&ws);
    if (rc) return rc;
    ws_bytes = kScratchBytes;
  }
  return spense_gemm(X, M, ldx, packed, w_scale, x_scale, Y, ldy, out_flags, ws, ws_bytes, stream);
}
