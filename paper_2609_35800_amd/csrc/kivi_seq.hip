// KIVI-style keys with one range per channel over the whole supplied
// sequence, text included (HeadGuard §4, Quantization setup: the KIVI-style
// base recomputes key ranges over the supplied sequence, including text,
// while text KV stays BF16).  Selected by kivi_group = 0.
//
// A persistent grid of kSeqBlocksPerCU workgroups of kSeqThreads threads per
// compute unit walks the key slices (l, b, h); for each slice:
//  1. per-channel min / max over all T rows of the slice (the load layout
//     holds a token row across D/8 lanes, 8 channels per lane, so each lane
//     reduces its 8 channels over its rows in registers);
//  2. the four wavefronts' partial ranges are combined through LDS and every
//     lane forms the group scale of its 8 channels;
//  3. the image rows are read again and quantized with those scales (codes
//     and one metadata word per channel) or, for the one-pass simulated
//     quantization, reconstructed to BF16.
// Values, protected slices and the rest of the cache are handled by the
// regular kernels of the same call.
//
// The second read of a slice's image rows is what makes this mode costlier
// than the grouped one.  The grid is sized so that the slices in flight at
// once (one per workgroup, ~770 KB each for a 3000-token slice) stay well
// within the 256 MB Infinity Cache, so that read is served from it rather
// than from HBM; large workgroups keep enough loads in flight to stream the
// first pass at full HBM rate.

#include <algorithm>

#include "hg_device.h"
#include "hg_kernels.h"

namespace hg {

constexpr int kSeqThreads = 1024;
constexpr int kSeqBlocksPerCU = 2;
constexpr int kSeqUnroll1 = 4;  // rows in flight per lane, range pass
constexpr int kSeqUnroll2 = 4;  // rows in flight per lane, code pass

template <int D, int BITS, bool FAKE, int WAVES>
__device__ __forceinline__ void kivi_seq_slice(const Params& p, uint32_t s, const SliceRoute& route,
                                               float (&part)[2][WAVES][D]) {
  constexpr int CPT = D / 8;
  constexpr int RPL = 64 / CPT;
  constexpr int STEP = WAVES * RPL;
  constexpr int LEVELS = (1 << BITS) - 1;
  constexpr int ROW = D * BITS / 8;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int c8 = lane % CPT;
  const int r = lane / CPT;
  const uint16_t* slice = p.cache[0] + (size_t)s * p.T * D;

  // 1. ranges over all T rows
  float mn[8], mx[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    mn[e] = __builtin_inff();
    mx[e] = -__builtin_inff();
  }
  for (int t0 = wave * RPL + r; t0 < p.T; t0 += kSeqUnroll1 * STEP) {
    u32x4 v[kSeqUnroll1];
#pragma unroll
    for (int u = 0; u < kSeqUnroll1; ++u) v[u] = *(const u32x4*)(slice + (size_t)min(t0 + u * STEP, p.T - 1) * D + 8 * c8);
#pragma unroll
    for (int u = 0; u < kSeqUnroll1; ++u) {
      // rows past the end re-read the last row: the range is unchanged
      const float x[8] = {bf16_lo(v[u].x), bf16_hi(v[u].x), bf16_lo(v[u].y), bf16_hi(v[u].y),
                          bf16_lo(v[u].z), bf16_hi(v[u].z), bf16_lo(v[u].w), bf16_hi(v[u].w)};
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        mn[e] = fminf(mn[e], x[e]);
        mx[e] = fmaxf(mx[e], x[e]);
      }
    }
  }
#pragma unroll
  for (int e = 0; e < 8; ++e) {
#pragma unroll
    for (int off = CPT; off < 64; off *= 2) {
      mn[e] = fminf(mn[e], __shfl_xor(mn[e], off));
      mx[e] = fmaxf(mx[e], __shfl_xor(mx[e], off));
    }
  }

  // 2. combine the wavefronts and form the scales (the barrier first: the
  //    previous slice's readers of `part` are done)
  __syncthreads();
  if (r == 0) {
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      part[0][wave][8 * c8 + e] = mn[e];
      part[1][wave][8 * c8 + e] = mx[e];
    }
  }
  __syncthreads();
  GroupScale g[8];
  float S[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    float a = part[0][0][8 * c8 + e], b = part[1][0][8 * c8 + e];
#pragma unroll
    for (int w = 1; w < WAVES; ++w) {
      a = fminf(a, part[0][w][8 * c8 + e]);
      b = fmaxf(b, part[1][w][8 * c8 + e]);
    }
    g[e] = group_scale<LEVELS>(a, b);
    S[e] = bf16_as_float(g[e].meta & 0xFFFFu);
  }
  const size_t slab = (size_t)route.slot * p.B + route.b;
  if (!FAKE && wave == 0 && r == 0) {
    uint32_t* m = p.meta[0] + slab * D + 8 * c8;
    __builtin_nontemporal_store(u32x4{g[0].meta, g[1].meta, g[2].meta, g[3].meta}, (u32x4*)m);
    __builtin_nontemporal_store(u32x4{g[4].meta, g[5].meta, g[6].meta, g[7].meta}, (u32x4*)m + 1);
  }

  // 3. the image rows: codes, or their reconstruction
  const uint16_t* rows = slice + (size_t)p.s0 * D;
  uint8_t* codes = FAKE ? nullptr : p.codes[0] + slab * p.n * ROW;
  uint16_t* out = FAKE ? p.out[0] + (size_t)s * p.T * D + (size_t)p.s0 * D : nullptr;
  for (int t0 = wave * RPL + r; t0 < p.n; t0 += kSeqUnroll2 * STEP) {
    u32x4 v[kSeqUnroll2];
#pragma unroll
    for (int u = 0; u < kSeqUnroll2; ++u) v[u] = *(const u32x4*)(rows + (size_t)min(t0 + u * STEP, p.n - 1) * D + 8 * c8);
#pragma unroll
    for (int u = 0; u < kSeqUnroll2; ++u) {
      const int t = t0 + u * STEP;
      const float x[8] = {bf16_lo(v[u].x), bf16_hi(v[u].x), bf16_lo(v[u].y), bf16_hi(v[u].y),
                          bf16_lo(v[u].z), bf16_hi(v[u].z), bf16_lo(v[u].w), bf16_hi(v[u].w)};
      uint32_t cb[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) cb[e] = code_bits(x[e], g[e]);
      if constexpr (FAKE) {
        float y[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) y[e] = __builtin_fmaf((float)(cb[e] - kMagicBits), S[e], g[e].m);
        const u32x4 o = {pack_bf16x2_hw(y[0], y[1]), pack_bf16x2_hw(y[2], y[3]), pack_bf16x2_hw(y[4], y[5]),
                         pack_bf16x2_hw(y[6], y[7])};
        if (t < p.n) store_nt((u32x4*)(out + (size_t)t * D + 8 * c8), o);
      } else {
        const Packed<8, BITS> pk = pack_code_bits<8, BITS>(cb);
        if (t < p.n) store_packed<8, BITS>(codes + (size_t)t * ROW + c8 * BITS, pk);
      }
    }
  }
}

template <int D, int BITS, bool FAKE>
__global__ __launch_bounds__(kSeqThreads) void kivi_seq_kernel(const Params p) {
  constexpr int WAVES = kSeqThreads / 64;
  __shared__ float part[2][WAVES][D];
  const uint32_t slices = (uint32_t)p.L * p.B * p.H;
  for (uint32_t s = blockIdx.x; s < slices; s += gridDim.x) {  // key slice (l*B + b)*H + h
    const SliceRoute route = route_slice(p, 0, s);
    if (!route.kept) kivi_seq_slice<D, BITS, FAKE, WAVES>(p, s, route, part);  // kept: copied elsewhere
  }
}

template <int D, int BITS>
static hipError_t launch_k(const Params& p, bool fake, hipStream_t stream) {
  int dev = 0, cus = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e == hipSuccess) e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
  if (e != hipSuccess) return e;
  const uint32_t slices = (uint32_t)p.L * p.B * p.H;
  const uint32_t blocks = std::min<uint32_t>(slices, (uint32_t)std::max(cus, 1) * kSeqBlocksPerCU);
  if (fake)
    hipLaunchKernelGGL((kivi_seq_kernel<D, BITS, true>), dim3(blocks), dim3(kSeqThreads), 0, stream, p);
  else
    hipLaunchKernelGGL((kivi_seq_kernel<D, BITS, false>), dim3(blocks), dim3(kSeqThreads), 0, stream, p);
  return hipGetLastError();
}

template <int D>
static hipError_t launch_k_bits(const Params& p, int bits, bool fake, hipStream_t stream) {
  switch (bits) {
    case 2: return launch_k<D, 2>(p, fake, stream);
    case 3: return launch_k<D, 3>(p, fake, stream);
    case 4: return launch_k<D, 4>(p, fake, stream);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_kivi_seq(const Params& p, int D, int bits, bool fake, hipStream_t stream) {
  switch (D) {
    case 64: return launch_k_bits<64>(p, bits, fake, stream);
    case 128: return launch_k_bits<128>(p, bits, fake, stream);
    case 256: return launch_k_bits<256>(p, bits, fake, stream);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace hg
