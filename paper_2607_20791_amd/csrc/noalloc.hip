// The min-p sampler entry point for callers that cannot allocate device
// memory (code under graph capture, serving loops, harnesses that forbid
// allocation): rgd_kernel_sample with its workspace taken from a fixed device
// array instead of a caller buffer.
//
// The array lives in this file.  In host code its name is only a host-side
// stand-in for the device symbol, so the kernels never receive it: the first
// call on a device (with that device current) looks up the array's device
// address with hipGetSymbolAddress and keeps it per device, and every launch
// passes that address.  Each device holds its own copy of the array for the
// life of the process.
#include <mutex>

#include "entry.hpp"
#include "kernels.hpp"
#include "rgd.h"

namespace {

constexpr size_t kScratchBytes = size_t(1) << 20;  // RGD_NOALLOC_SCRATCH_BYTES
static_assert(kScratchBytes == RGD_NOALLOC_SCRATCH_BYTES, "header and library disagree on the scratch size");

// Sampler workspace of every call on this device: the chunk kept-weight sums,
// chunk maxima and p-less statistics of rgd_sampler_workspace_bytes.  Every
// element a call reads is written earlier in the same call, so nothing needs
// clearing between calls.
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
std::once_flag g_once[kMaxDevices];
hipError_t g_lookup[kMaxDevices];
void* g_scratch[kMaxDevices];  // device address of `scratch` on each device

}  // namespace

extern "C" int32_t rgd_kernel_sample_noalloc(const float* z, int32_t R, int32_t V, float T, float min_p,
                                             const uint64_t* seeds, uint32_t ctr, uint32_t stream0,
                                             int32_t draws, int32_t* out, rgd_stream stream) {
  using namespace rgd;
  // the same checks as rgd_kernel_sample, before any HIP call
  if (!z || !seeds || !out) return set_error(RGD_E_INVALID_ARG, "null argument");
  if (R < 1 || V < 4 || V % 4 || (long long)V > 256LL * 4096 || draws < 1)
    return set_error(RGD_E_INVALID_ARG, "bad R/V/draws");
  if (!(T > 0.f)) return set_error(RGD_E_INVALID_ARG, "T must be > 0");
  if (!(min_p >= 0.f && min_p <= 1.f)) return set_error(RGD_E_INVALID_ARG, "min_p must be in [0,1]");
  const uint64_t need = rgd_sampler_workspace_bytes(R, V);
  if (need > kScratchBytes)
    return set_error(RGD_E_INVALID_ARG,
                     "R x V needs more sampler workspace than the library's fixed 1 MiB scratch "
                     "(rgd_sampler_workspace_bytes(R, V) must be <= RGD_NOALLOC_SCRATCH_BYTES)");
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess) return set_error(RGD_E_HIP, "hipGetDevice failed");
  if (dev < 0 || dev >= kMaxDevices) return set_error(RGD_E_UNSUPPORTED, "device index beyond 63");
  std::call_once(g_once[dev], [dev] {
    void* p = nullptr;
    g_lookup[dev] = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    g_scratch[dev] = g_lookup[dev] == hipSuccess ? p : nullptr;
  });
  if (g_lookup[dev] != hipSuccess || !g_scratch[dev])
    return set_error(RGD_E_HIP, "hipGetSymbolAddress of the sampler scratch failed");
  return kernel_sample(z, R, V, T, min_p, false, seeds, ctr, stream0, draws, g_scratch[dev], out, stream);
}
