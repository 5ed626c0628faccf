// psattn_bwd_noalloc: the backward pass with its workspace in a file-scope device array, for
// callers that cannot allocate device memory (code under HIP graph capture, tight serving loops,
// harnesses that forbid allocation).  The kernels are those of psattn_bwd; only the origin of
// the workspace differs.
#include <hip/hip_runtime.h>

#include <cstdio>
#include <mutex>

#include "psattn.h"

namespace psattn {
psattn_status set_error(psattn_status st, const char* msg);
}

namespace {

constexpr size_t kScratchBytes = (size_t)PSATTN_NOALLOC_SCRATCH_MIB << 20;
constexpr int kMaxDevices = 64;

// The workspace of psattn_bwd_noalloc: one copy per GPU, held until the process ends.  Host code
// never passes this name to a kernel: it is a host-side stand-in, and the device address of each
// GPU's copy comes from hipGetSymbolAddress (scratch_ptr below).
static __device__ __align__(256) uint8_t scratch[kScratchBytes];

std::mutex g_mu;
void* g_scratch[kMaxDevices] = {};

// The device address of the current GPU's scratch array, looked up once per device.
psattn_status scratch_ptr(void** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return psattn::set_error(PSATTN_E_HIP, hipGetErrorString(e));
  if (dev < 0 || dev >= kMaxDevices) return psattn::set_error(PSATTN_E_UNSUPPORTED, "device index beyond 63");
  std::lock_guard<std::mutex> lk(g_mu);
  if (!g_scratch[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p) {
      char msg[256];
      snprintf(msg, sizeof msg, "hipGetSymbolAddress(scratch) on device %d failed: %s", dev, hipGetErrorString(e));
      return psattn::set_error(PSATTN_E_HIP, msg);
    }
    g_scratch[dev] = p;
  }
  *out = g_scratch[dev];
  return PSATTN_OK;
}

}  // namespace

extern "C" psattn_status psattn_bwd_noalloc(const psattn_tree* tree, const void* Q, const void* K, const void* V,
                                            const void* O, const float* LSE, const void* O_lo, const void* dO,
                                            float* dQ, float* dK, float* dV, void* stream) {
  size_t need = 0;
  psattn_status st = psattn_workspace_size(tree, 1, &need);
  if (st != PSATTN_OK) return st;
  if (need > kScratchBytes) {
    char msg[256];
    snprintf(msg, sizeof msg, "the backward pass of this tree needs %zu bytes of workspace; psattn_bwd_noalloc holds %zu",
             need, kScratchBytes);
    return psattn::set_error(PSATTN_E_WORKSPACE, msg);
  }
  void* ws = nullptr;
  st = scratch_ptr(&ws);
  if (st != PSATTN_OK) return st;
  return psattn_bwd(tree, Q, K, V, O, LSE, O_lo, dO, dQ, dK, dV, ws, kScratchBytes, stream);
}
