// The fixed device scratch of hc_attention_static (the routed attention for
// callers that cannot allocate device memory) and the kernel that writes a
// layer's dense work list into it.
#include "hc_device.h"
#include "hc_plan.h"

#include <mutex>

namespace hc {
namespace {

// One array per GPU, loaded with the library's code object and held until the
// process ends.  Every hc_attention_static call on a GPU uses that GPU's copy.
static __device__ __align__(256) unsigned char scratch[kStaticScratchBytes];

// Device address of `scratch` on each GPU, resolved once per device.  In host
// code the array's name is not a device address, so only these are used.
constexpr int kMaxDevices = 64;
std::mutex g_mu;
void *g_ptr[kMaxDevices] = {};

// Unit i and merge item i of the layer's work list (closed forms of hc_plan.h).
__global__ __launch_bounds__(256) void static_plan_kernel(StaticPlan p, DenseUnit *units,
                                                          CombineItem *comb) {
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (i < static_n_units(p)) units[i] = static_dense_unit(p, i);
  if (i < static_n_comb(p)) comb[i] = static_comb_item(p, i);
}

}  // namespace

hipError_t static_scratch(int device, void **ptr) {
  *ptr = nullptr;
  if (device < 0 || device >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_mu);
  if (!g_ptr[device]) {
    // the caller has made `device` current
    void *p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    g_ptr[device] = p;
  }
  *ptr = g_ptr[device];
  return hipSuccess;
}

hipError_t launch_static_plan(const StaticPlan &p, DenseUnit *units, CombineItem *comb,
                              hipStream_t s) {
  const int n = static_n_units(p) > static_n_comb(p) ? static_n_units(p) : static_n_comb(p);
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(static_plan_kernel, dim3((n + 255) / 256), dim3(256), 0, s, p, units, comb);
  return hipGetLastError();
}

}  // namespace hc
