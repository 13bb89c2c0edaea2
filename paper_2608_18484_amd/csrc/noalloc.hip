// Plans bound to a file-scope device array instead of a caller workspace,
// for callers that cannot allocate device memory (code under graph capture,
// serving loops, harnesses that forbid hipMalloc).
//
// The array is a static __device__ object of this translation unit: every
// device the library runs on holds one copy (kStaticScratchBytes) until the
// process ends.  Its host-side name is not a device address; the address on
// each device is looked up once, with that device current, by
// hipGetSymbolAddress, and only that pointer is handed to the kernels (as the
// workspace of an ordinary plan).
#include <hip/hip_runtime.h>

#include <mutex>
#include <string>

#include "sparsepr_internal.hpp"

namespace sparsepr {
namespace {

constexpr int kMaxDevices = 64;

static __device__ __align__(256) unsigned char scratch[kStaticScratchBytes];

std::mutex g_mu;
void* g_ptr[kMaxDevices];   // address of `scratch` on each device (null: not looked up yet)
bool g_busy[kMaxDevices];   // a live plan of this entry point holds that device's array

}  // namespace

void release_static_scratch(int dev) {
  std::lock_guard<std::mutex> lk(g_mu);
  if (dev >= 0 && dev < kMaxDevices) g_busy[dev] = false;
}

}  // namespace sparsepr

extern "C" sparsepr_status sparsepr_plan_create_static(const sparsepr_shape* shape,
                                                       const sparsepr_params* params,
                                                       sparsepr_plan_t* out) {
  using namespace sparsepr;
  if (!out) return set_error(SPARSEPR_ERR_INVALID_ARGUMENT, "out must not be NULL");
  size_t need = 0;
  sparsepr_status st = sparsepr_workspace_size(shape, params, &need);
  if (st != SPARSEPR_OK) return st;  // its message stands
  if (need > kStaticScratchBytes)
    return set_error(SPARSEPR_ERR_WORKSPACE_TOO_SMALL,
                     "sparsepr_plan_create_static: this shape needs " + std::to_string(need) +
                         " bytes of workspace, the static scratch array holds " +
                         std::to_string(kStaticScratchBytes) +
                         "; use sparsepr_plan_create with a caller workspace");
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) {
    (void)hipGetLastError();
    return set_error(SPARSEPR_ERR_HIP, std::string("hipGetDevice: ") + hipGetErrorString(e));
  }
  if (dev < 0 || dev >= kMaxDevices)
    return set_error(SPARSEPR_ERR_UNSUPPORTED, "sparsepr_plan_create_static: device index above 63");
  std::lock_guard<std::mutex> lk(g_mu);
  if (g_busy[dev])
    return set_error(SPARSEPR_ERR_INVALID_ARGUMENT,
                     "sparsepr_plan_create_static: a plan made by this entry point is alive on "
                     "this device; destroy it first (both would use the one scratch array)");
  if (!g_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p) {
      (void)hipGetLastError();
      return set_error(SPARSEPR_ERR_HIP, std::string("hipGetSymbolAddress(scratch): ") +
                                             hipGetErrorString(e));
    }
    g_ptr[dev] = p;
  }
  // an ordinary plan on the device's array; creating it clears the counters a
  // plan must start from (the array keeps whatever the last plan left)
  st = sparsepr_plan_create(shape, params, g_ptr[dev], kStaticScratchBytes, out);
  if (st != SPARSEPR_OK) return st;
  mark_static_plan(*out, dev);
  g_busy[dev] = true;
  return SPARSEPR_OK;
}
