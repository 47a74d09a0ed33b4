// sn_project_weights_noalloc: the weight confinement W <- U (U^T W) with its
// workspace in a static device array instead of a caller buffer, for callers
// that cannot allocate device memory (code under stream capture, tight
// serving loops, harnesses that forbid allocation).
//
// The array `scratch` below is a file-scope __device__ symbol: every device
// the library runs on holds its own copy (kScratchBytes, allocated with the
// code object, kept until the process ends).  In host code its name is a
// host-side stand-in, never a device address, so its device address is looked
// up once per device with hipGetSymbolAddress (with that device current, on
// the first call there) and only that address is handed to the kernels.
//
// The kernels are those of sn_project_weights, called with the scratch
// address as their workspace; the projection's kernels write every workspace
// element they later read, so nothing needs clearing between calls.  Calls on
// one device share its scratch: two calls that overlap in time on that device
// (different streams, or different host threads without ordering) race.
#include <mutex>

#include "sn.h"
#include "sn_internal.h"

namespace {

constexpr size_t kScratchBytes = size_t(SN_PROJECT_NOALLOC_SCRATCH_BYTES);
constexpr int kMaxDevices = 64;

static __device__ __align__(256) unsigned char scratch[kScratchBytes];

std::mutex g_mu;
void *g_ptr[kMaxDevices] = {};

// Device address of this device's scratch (looked up on the first call made
// with the device current); nullptr with the HIP error in *err on failure.
void *scratch_ptr(int dev, hipError_t *err) {
  std::lock_guard<std::mutex> lock(g_mu);
  if (!g_ptr[dev]) {
    void *p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p) {
      *err = e != hipSuccess ? e : hipErrorInvalidSymbol;
      return nullptr;
    }
    g_ptr[dev] = p;
  }
  return g_ptr[dev];
}

}  // namespace

extern "C" int32_t sn_project_weights_noalloc(const void *basis, int64_t d, int64_t k, int32_t dt,
                                              void *W, int64_t m, int64_t ldw, sn_stream stream) {
  // every argument is checked before the device is touched
  int32_t st = sn::project_args_check(basis, d, k, dt, W, m, ldw);
  if (st || m == 0) return st;
  const size_t need = sn_project_weights_workspace_bytes(d, k, dt, m);
  if (need > kScratchBytes)
    return sn::set_error(SN_ERR_WORKSPACE,
                         "sn_project_weights_noalloc: a %lld x %lld matrix at k = %lld needs %zu "
                         "bytes of scratch; the static scratch holds %zu",
                         (long long)d, (long long)m, (long long)k, need, kScratchBytes);
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return sn::set_error(SN_ERR_HIP, "hipGetDevice: %s", hipGetErrorString(e));
  if (dev < 0 || dev >= kMaxDevices)
    return sn::set_error(SN_ERR_UNSUPPORTED, "device %d: at most %d devices", dev, kMaxDevices);
  void *ws = scratch_ptr(dev, &e);
  if (!ws)
    return sn::set_error(SN_ERR_HIP, "hipGetSymbolAddress(scratch): %s", hipGetErrorString(e));
  return sn_project_weights(basis, d, k, dt, W, m, ldw, ws, kScratchBytes, stream);
}
