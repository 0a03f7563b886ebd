// Exhaustive device-side checks of the arithmetic shortcuts the kernels take,
// run with the kernels' own helpers (paper_2609_35800_amd/csrc/hg_device.h):
//  - hgp_bf16_convert: the hardware fp32 -> BF16 conversion against round to
//    nearest even on the bit pattern, for every finite fp32 value;
//  - hgp_div_levels: the fma-corrected division by L = 3, 7, 15 against the
//    IEEE quotient, for every non-negative finite fp32 dividend;
//  - hgp_rcp_scale: the refined hardware reciprocal against the IEEE 1/S for
//    every BF16 value S in [2^-126, 2^101].
// Test infrastructure only: loaded by the GPU tests through ctypes.  Every
// kernel writes only into a small counter array.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "hg_device.h"

namespace {

constexpr uint64_t kPerThread = 256;

__global__ void bf16_convert_kernel(unsigned long long* cnt) {
  const uint64_t base = ((uint64_t)blockIdx.x * blockDim.x + threadIdx.x) * kPerThread;
  unsigned long long checked = 0, bad = 0;
  for (uint64_t k = 0; k < kPerThread; k += 2) {
    const uint32_t u0 = (uint32_t)(base + k), u1 = (uint32_t)(base + k + 1);
    const uint32_t hw = hg::pack_bf16x2_hw(__uint_as_float(u0), __uint_as_float(u1));
    const uint32_t sw = hg::pack_bf16x2(__uint_as_float(u0), __uint_as_float(u1));
    if (((u0 >> 23) & 0xFFu) != 0xFFu) { checked++; bad += (hw & 0xFFFFu) != (sw & 0xFFFFu); }
    if (((u1 >> 23) & 0xFFu) != 0xFFu) { checked++; bad += (hw >> 16) != (sw >> 16); }
  }
  atomicAdd(&cnt[0], checked);
  atomicAdd(&cnt[1], bad);
}

template <int L>
__global__ void div_levels_kernel(unsigned long long* cnt) {
  const uint64_t base = ((uint64_t)blockIdx.x * blockDim.x + threadIdx.x) * kPerThread;
  unsigned long long checked = 0, bad = 0;
  for (uint64_t k = 0; k < kPerThread; ++k) {
    const uint64_t u = base + k;
    if (u >= 0x7F800000ull) break;  // non-negative finite values only
    const float d = __uint_as_float((uint32_t)u);
    const float fast = hg::div_levels<L>(d);
    const float ieee = d / (float)L;
    checked++;
    bad += __float_as_uint(fast) != __float_as_uint(ieee);
  }
  atomicAdd(&cnt[0], checked);
  atomicAdd(&cnt[1], bad);
}

// One thread per BF16 pattern; counters[2] collects mismatches outside the
// documented range (reported, not asserted).
__global__ void rcp_scale_kernel(unsigned long long* cnt) {
  const uint32_t h = blockIdx.x * blockDim.x + threadIdx.x;  // 0 .. 0x7F7F
  if (h < 0x0080u || h > 0x7F7Fu) return;                     // positive normal finite
  const float S = __uint_as_float(h << 16);
  const bool in_range = S <= 0x1p101f;
  const bool bad = __float_as_uint(hg::rcp_scale(S)) != __float_as_uint(1.0f / S);
  if (in_range) {
    atomicAdd(&cnt[0], 1ull);
    if (bad) atomicAdd(&cnt[1], 1ull);
  } else if (bad) {
    atomicAdd(&cnt[2], 1ull);
  }
}

}  // namespace

extern "C" {

// counters[0] = values checked, counters[1] = mismatches (device memory, zeroed
// by the caller).  Returns a hipError_t.
int hgp_bf16_convert(unsigned long long* counters, void* stream) {
  // 2^32 patterns / 256 per thread / 256 threads per block
  hipLaunchKernelGGL(bf16_convert_kernel, dim3(65536), dim3(256), 0, (hipStream_t)stream, counters);
  return (int)hipGetLastError();
}

int hgp_div_levels(int levels, unsigned long long* counters, void* stream) {
  // 0x7F800000 non-negative finite patterns, 256 per thread, 256 threads per block
  const unsigned blocks = (unsigned)((0x7F800000ull + 256 * kPerThread - 1) / (256 * kPerThread));
  switch (levels) {
    case 3: hipLaunchKernelGGL(div_levels_kernel<3>, dim3(blocks), dim3(256), 0, (hipStream_t)stream, counters); break;
    case 7: hipLaunchKernelGGL(div_levels_kernel<7>, dim3(blocks), dim3(256), 0, (hipStream_t)stream, counters); break;
    case 15: hipLaunchKernelGGL(div_levels_kernel<15>, dim3(blocks), dim3(256), 0, (hipStream_t)stream, counters); break;
    default: return (int)hipErrorInvalidValue;
  }
  return (int)hipGetLastError();
}

// counters[0] = scales checked in range, [1] = mismatches in range,
// [2] = mismatches above 2^101 (outside the kernels' precondition).
int hgp_rcp_scale(unsigned long long* counters, void* stream) {
  hipLaunchKernelGGL(rcp_scale_kernel, dim3(128), dim3(256), 0, (hipStream_t)stream, counters);
  return (int)hipGetLastError();
}

}  // extern "C"
