// Scratch-free selection (phsa_select_noalloc): phsa_select with its bf16
// scratch in a static device array instead of a caller's workspace, for callers
// that cannot allocate.  The kernels are those of phsa_select; they receive the
// array's device address as their workspace argument.
#include <atomic>
#include <mutex>

#include "phsa.h"
#include "launch.h"

namespace phsa {

namespace {

constexpr size_t kScratchBytes = PHSA_NOALLOC_SCRATCH_BYTES;
constexpr int kMaxDevices = 64;

// One copy per GPU, from the first use on that GPU until the process ends.  In
// host code this name stands for the array, not its device address; the
// address comes from hipGetSymbolAddress.
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

// Device address of `scratch` on each GPU, looked up once per GPU.  Written
// under the mutex, read without it once set.
std::atomic<void *> g_scratch_ptr[kMaxDevices];
std::mutex g_scratch_mu;

// The array's device address on device `dev`, which must be current.
hipError_t scratch_address(int dev, void **out) {
  void *p = g_scratch_ptr[dev].load(std::memory_order_acquire);
  if (!p) {
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    p = g_scratch_ptr[dev].load(std::memory_order_relaxed);
    if (!p) {
      const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
      if (e != hipSuccess) return e;
      if (!p) return hipErrorInvalidSymbol;
      g_scratch_ptr[dev].store(p, std::memory_order_release);
    }
  }
  *out = p;
  return hipSuccess;
}

}  // namespace

}  // namespace phsa

using namespace phsa;

extern "C" phsa_status phsa_select_noalloc(const phsa_params *p, const void *Q, const float *K_comp, int32_t *sel,
                                           void *stream) {
  try {
    Geom g;
    const phsa_status st = validate(p, PHSA_OP_SELECT, &g);
    if (st != PHSA_OK) return st;
    if (!Q || !K_comp || !sel) return PHSA_ERR_NULL;
    const size_t need = select_split_bytes(g);
    if (need > kScratchBytes) return PHSA_ERR_SCRATCH_LIMIT;
    hipStream_t s = static_cast<hipStream_t>(stream);
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return PHSA_ERR_HIP;
    if (s) {
      hipDevice_t sdev = -1;
      if (hipStreamGetDevice(s, &sdev) != hipSuccess) return PHSA_ERR_INVALID_ARG;
      if (sdev != dev) return PHSA_ERR_INVALID_ARG;
    }
    void *ws = nullptr;
    if (need > 0 && scratch_address(dev, &ws) != hipSuccess) return PHSA_ERR_HIP;
    return launch_select(g, Q, K_comp, sel, ws, s) == hipSuccess ? PHSA_OK : PHSA_ERR_HIP;
  } catch (...) {
    return PHSA_ERR_HIP;
  }
}
