// acid_l1_norms_noalloc: EasyCache's L1 sums (the same kernels as
// acid_l1_norms) with their partial sums in a file-scope device array, for
// callers that cannot allocate device memory and hold no model workspace.
//
// The array lives on every device the library runs on until the process
// ends.  Host code never passes the array's name to a kernel or a copy: in
// host code that name is only a stand-in, not a device address.  The device
// address is looked up once per device with hipGetSymbolAddress (with that
// device current) and cached; every launch and copy uses the cached address.
#include <mutex>

#include "common.h"

namespace acid {
namespace {

// Partial sums of at most kScratchGroups workgroups (one fp64 pair each),
// then the two final sums.  The grid of the L1 kernels never exceeds
// kScratchGroups, so every n fits.
constexpr int kScratchGroups = 1024;
constexpr int kScratchDoubles = 2 * kScratchGroups + 2;

static __device__ __align__(256) double scratch[kScratchDoubles];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
double* g_scratch_ptr[kMaxDevices] = {};

// The device address of `scratch` on device `dev`, looked up with that
// device current on first use and cached.
acid_status scratch_on(int dev, double** out) {
  if (dev < 0 || dev >= kMaxDevices)
    return set_error(ACID_ERR_UNSUPPORTED, "device ordinal %d beyond %d", dev, kMaxDevices);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    int cur = 0;
    ACID_HIP(hipGetDevice(&cur));
    if (cur != dev) ACID_HIP(hipSetDevice(dev));
    double* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(reinterpret_cast<void**>(&p), HIP_SYMBOL(scratch));
    if (cur != dev) ACID_HIP(hipSetDevice(cur));
    if (e != hipSuccess) return check_hip(e, "hipGetSymbolAddress(scratch)");
    if (!p) return set_error(ACID_ERR_HIP, "hipGetSymbolAddress(scratch) returned NULL");
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return ACID_OK;
}

}  // namespace
}  // namespace acid

using namespace acid;

extern "C" acid_status acid_l1_norms_noalloc(const float* a_dev, const float* b_dev,
                                             const float* c_dev, int64_t n, double* out_host,
                                             hipStream_t stream) {
  if (!out_host) return set_error(ACID_ERR_INVALID_ARG, "NULL argument");
  if (n < 0) return set_error(ACID_ERR_INVALID_ARG, "n %lld < 0", (long long)n);
  if (n == 0) {  // empty sums; the buffers are not touched
    out_host[0] = out_host[1] = 0.0;
    return ACID_OK;
  }
  if (!a_dev) return set_error(ACID_ERR_INVALID_ARG, "NULL argument");
  if (((uintptr_t)a_dev | (uintptr_t)b_dev | (uintptr_t)c_dev) % 16)
    return set_error(ACID_ERR_INVALID_ARG, "buffers must be 16-byte aligned");
  int dev = 0;
  if (stream)
    ACID_HIP(hipStreamGetDevice(stream, &dev));
  else
    ACID_HIP(hipGetDevice(&dev));
  double* ws = nullptr;
  ACID_TRY(scratch_on(dev, &ws));
  double* part = ws;
  double* res = ws + 2 * kScratchGroups;
  // Every partial the reduction reads is written by this call's first
  // kernel, and the result pair by its second: nothing needs clearing.
  hipError_t e = launch_l1_norms(a_dev, b_dev, c_dev, n, part, kScratchGroups, res, stream);
  if (e != hipSuccess) return check_hip(e, "l1 norms (no-alloc)");
  ACID_HIP(hipMemcpyAsync(out_host, res, 2 * sizeof(double), hipMemcpyDeviceToHost, stream));
  ACID_HIP(hipStreamSynchronize(stream));
  return ACID_OK;
}
