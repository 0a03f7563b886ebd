// hg_fake_quantize_noalloc: the one-pass simulated quantization for callers
// that cannot allocate device memory (code under HIP graph capture, serving
// loops, harnesses that forbid allocation).  It is hg_fake_quantize with the
// token-retention workspace taken from a fixed device array of this library
// instead of a caller buffer; the kernels and checks are the same.
//
// The array: file-scope device memory of HG_NOALLOC_SCRATCH_BYTES, one copy
// per GPU, held until the process ends.  Host code never uses the array's
// name as an address (on the host it names a stand-in, not device memory):
// the device address of the current GPU's copy is looked up once per device,
// on the entry point's first call on it, and kept.  Every call on one GPU
// shares that GPU's copy and leaves its contents behind; a call writes every
// byte it later reads (norms, token lists, saved rows), so nothing needs
// clearing.  Calls that overlap in time on one GPU (other streams, other host
// threads) race on the array and must be serialized by the caller.

#include <stdio.h>

#include <mutex>

#include "headguard.h"
#include "hg_kernels.h"

static __device__ __align__(256) unsigned char scratch[HG_NOALLOC_SCRATCH_BYTES];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_mutex;
void* g_scratch[kMaxDevices] = {};  // device address of each GPU's copy, once looked up

// Address of the current device's copy of the array (looked up once per
// device, with that device current).
int scratch_address(void** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess || dev < 0) {
    (void)hipGetLastError();
    return hg::set_error(HG_ERR_NO_DEVICE, "no current HIP device");
  }
  if (dev >= kMaxDevices) return hg::set_error(HG_ERR_NO_DEVICE, "device index beyond the supported 64");
  std::lock_guard<std::mutex> lock(g_mutex);
  if (!g_scratch[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p) {
      (void)hipGetLastError();
      char msg[160];
      snprintf(msg, sizeof msg, "scratch array address: %s", hipGetErrorString(e));
      return hg::set_error(HG_ERR_HIP, msg);
    }
    g_scratch[dev] = p;
  }
  *out = g_scratch[dev];
  return HG_OK;
}

}  // namespace

extern "C" int hg_fake_quantize_noalloc(const hg_config* cfg, const uint16_t* K, const uint16_t* V,
                                        const uint8_t* protect_mask, uint16_t* K_out, uint16_t* V_out,
                                        hipStream_t stream) {
  const hg::WorkspaceFn from_scratch = [](uint64_t need, hg::Workspace* ws) {
    if (need > (uint64_t)HG_NOALLOC_SCRATCH_BYTES) {
      char msg[200];
      snprintf(msg, sizeof msg, "the call needs a %llu-byte workspace; the library's array holds %llu",
               (unsigned long long)need, (unsigned long long)HG_NOALLOC_SCRATCH_BYTES);
      return hg::set_error(HG_ERR_SHAPE, msg);
    }
    int s = scratch_address(&ws->ptr);
    if (s) return s;
    ws->bytes = HG_NOALLOC_SCRATCH_BYTES;
    ws->caller = false;
    return (int)HG_OK;
  };
  return hg::fake_quantize(cfg, K, V, protect_mask, K_out, V_out, from_scratch, stream);
}
