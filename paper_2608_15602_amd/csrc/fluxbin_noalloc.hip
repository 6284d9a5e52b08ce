// Batch-1 LUT-GEMV for callers that cannot allocate device memory (fluxbin_lut_gemv_noalloc): the split-tile
// workspace of fluxbin_lut_gemv (tile counters, then partial sums) lives in one file-scope device array of fixed size
// instead of a caller-provided buffer. Same launch plan and kernels as fluxbin_lut_gemv, so the result is bitwise the
// same.
//
// Every device the library runs on holds its own copy of the array until the process ends. Host code never passes the
// array's name to a kernel (on the host it is only a stand-in for the symbol): the device address of each device's
// copy is looked up once with hipGetSymbolAddress, with that device current, and kept per device.
#include <hip/hip_runtime.h>

#include <mutex>

#include "fluxbin_internal.h"

namespace fluxbin {

static __device__ __align__(256) uint8_t scratch[FLUXBIN_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
static std::mutex g_scratch_mu;
static void* g_scratch_ptr[kMaxDevices] = {};

// Device address of the current device's scratch array. On the first call for a device the address is looked up and
// the array is zero-filled on `stream` (by a kernel, stream-ordered before the caller's launch); afterwards every
// completed call leaves its tile counters at zero again.
static fluxbin_status scratch_for_current_device(hipStream_t stream, void** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  if (dev < 0 || dev >= kMaxDevices) return fail(FLUXBIN_ERR_UNSUPPORTED, "device index %d >= %d", dev, kMaxDevices);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p) return hip_fail(e, "hipGetSymbolAddress (static scratch)");
    const fluxbin_status st = launch_fill_zero(p, FLUXBIN_NOALLOC_SCRATCH_BYTES, stream);
    if (st != FLUXBIN_OK) return st;
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return FLUXBIN_OK;
}

fluxbin_status gemv_noalloc(const fluxbin_layer& L, const uint16_t* d_x, void* d_y, int y_fp32, hipStream_t stream) {
  if (L.shape.M > kNoallocMaxM)
    return fail(FLUXBIN_ERR_UNSUPPORTED, "M = %lld exceeds %lld rows, the most the static scratch's tile counters cover",
                (long long)L.shape.M, (long long)kNoallocMaxM);
  Plan p;
  fluxbin_status st = make_plan(L, 1, &p);
  if (st != FLUXBIN_OK) return st;
  // fixed counter region (room for the tile counters of any layer with M <= kNoallocMaxM), partial sums after it: no
  // layer's partial sums ever cover another layer's counters, so calls on different layers share the array
  const uint64_t partial_bytes = p.ws_bytes - p.ws_partials_off;
  p.ws_counters_off = 0;
  p.ws_partials_off = kNoallocCounterBytes;
  p.ws_bytes = kNoallocCounterBytes + partial_bytes;
  if (p.ws_bytes > FLUXBIN_NOALLOC_SCRATCH_BYTES)
    return fail(FLUXBIN_ERR_UNSUPPORTED, "launch plan needs %llu bytes of scratch, the static scratch holds %llu",
                (unsigned long long)p.ws_bytes, (unsigned long long)FLUXBIN_NOALLOC_SCRATCH_BYTES);
  void* ws = nullptr;
  st = scratch_for_current_device(stream, &ws);
  if (st != FLUXBIN_OK) return st;
  return launch_gemm(L, p, 1, d_x, L.shape.N, d_y, L.shape.M, y_fp32, ws, stream);
}

}  // namespace fluxbin
