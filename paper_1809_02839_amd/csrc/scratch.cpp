// Device scratch for the allocation-free backward entry point: one file-scope
// device array per GPU, holding the split-K partial planes of the backward's
// GEMMs. Its device address is looked up once per device with
// hipGetSymbolAddress (the array's name in host code is only a host-side
// stand-in, never passed to a kernel) and cached; every later call on that
// device gets the cached address. All calls on one GPU share its array and
// its contents stay from the last call: calls that overlap on one GPU race.
#include <mutex>

#include "stage.hpp"

namespace spx {

namespace {

static __device__ __align__(256) unsigned char scratch[SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

}  // namespace

float* device_scratch(int device) {
  if (device < 0 || device >= kMaxDevices) throw StageError(SPECTRAIN_EINVAL, "device index outside the scratch table");
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[device]) {
    int current = -1;
    hip_check(hipGetDevice(&current), "hipGetDevice");
    if (current != device) hip_check(hipSetDevice(device), "hipSetDevice");
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (current != device) (void)hipSetDevice(current);
    hip_check(e, "hipGetSymbolAddress(scratch)");
    if (!p) throw StageError(SPECTRAIN_EHIP, "hipGetSymbolAddress(scratch) returned a null address");
    g_scratch_ptr[device] = p;
  }
  return static_cast<float*>(g_scratch_ptr[device]);
}

}  // namespace spx
