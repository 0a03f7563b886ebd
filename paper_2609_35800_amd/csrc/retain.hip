// AKVQ-style token retention (HeadGuard §4, Quantization setup): in every KV
// head the keys and values of a nominal 2 % of the image tokens, those whose
// keys have the largest norms, stay in BF16, with or without head protection.
//
// The quantize kernel writes the squared key norm of every image token in the
// same pass that reads the keys (key_norm_kernel does it on its own for the
// one-pass simulated quantization, whose in-place outputs would otherwise
// overwrite the rows to keep).  Then, per (l, b, h):
//  - retain_select_kernel finds the k-th largest norm by a most-significant-
//    digit-first radix select over the fp32 bit patterns (non-negative, so they
//    order as unsigned integers), lists the retained tokens in ascending order
//    (all larger norms, then the lowest-index ties), and gathers their K and V
//    rows for each tensor the head does not keep in BF16;
//  - retain_scatter_kernel writes those rows back over the reconstruction.

#include "hg_device.h"
#include "hg_kernels.h"

namespace hg {

// ------------------------------------------------------------ key norms

// One workgroup per kBlockTokens tokens of one key slice; a token row is held
// by D/8 lanes, 8 channels each.
template <int D>
__global__ __launch_bounds__(kThreads) void key_norm_kernel(const Params p) {
  constexpr int R = D / 8;                // lanes per token row
  constexpr int RPL = 64 / R;             // token rows per load
  constexpr int NL = kWaveTokens / RPL;   // loads per lane
  const uint32_t s = blockIdx.x / (uint32_t)p.tiles;
  const int tile = (int)(blockIdx.x % (uint32_t)p.tiles);
  const int lane = threadIdx.x & 63;
  const int t_first = tile * kBlockTokens + (threadIdx.x >> 6) * kWaveTokens;
  if (t_first >= p.n) return;
  const int c = lane % R, r = lane / R;
  const uint16_t* rows = p.cache[0] + ((size_t)s * p.T + p.s0) * D;
  float* norm = p.norm + (size_t)s * p.n;
  u32x4 v[NL];
#pragma unroll
  for (int k = 0; k < NL; ++k) {
    const int t = min(t_first + r + RPL * k, p.n - 1);  // rows past the end: not stored
    v[k] = *(const u32x4*)(rows + (size_t)t * D + 8 * c);
  }
#pragma unroll
  for (int k = 0; k < NL; ++k) {
    const float sq = row_sqnorm<D>(v[k]);
    const int t = t_first + r + RPL * k;
    if (c == 0 && t < p.n) norm[t] = sq;
  }
}

// ------------------------------------------------------------ selection

// Copies rows sel[0..m) of one tensor's image span to rows base.. of dst.
template <int D>
__device__ __forceinline__ void gather_rows(const uint16_t* __restrict__ src, uint16_t* __restrict__ dst,
                                            const int32_t* sel, uint32_t m, uint32_t base) {
  constexpr int VPT = D / 8;
  for (uint32_t i = threadIdx.x; i < m * VPT; i += kThreads) {
    const uint32_t row = i / VPT, c = i % VPT;
    const u32x4 v = *(const u32x4*)(src + (size_t)sel[row] * D + 8 * c);
    store_nt((u32x4*)(dst + (size_t)(base + row) * D + 8 * c), v);
  }
}

// One workgroup per (l, b, h); requires 1 <= k <= n.
template <int D>
__global__ __launch_bounds__(kThreads) void retain_select_kernel(const Params p) {
  constexpr int WAVES = kThreads / 64;
  __shared__ uint32_t hist[256];
  __shared__ uint32_t pick[2];
  __shared__ uint32_t wcount[WAVES][2];
  __shared__ int32_t sel[kThreads];

  const uint32_t s = blockIdx.x;  // (l*B + b)*H + h
  const int n = p.n;
  const uint32_t k = (uint32_t)p.k;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const uint32_t* key = (const uint32_t*)(p.norm + (size_t)s * n);

  // 1. The k-th largest key: one 8-bit digit per pass from the top.  `want` is
  //    how many of the candidates sharing `prefix` are still to be taken.
  uint32_t prefix = 0, pmask = 0, want = k;
  for (int shift = 24; shift >= 0; shift -= 8) {
    hist[tid] = 0;
    __syncthreads();
    for (int t = tid; t < n; t += kThreads) {
      const uint32_t u = key[t];
      if ((u & pmask) == prefix) atomicAdd(&hist[(u >> shift) & 255u], 1u);
    }
    __syncthreads();
    if (wave == 0) {
      // lane covers digits 255 - 4*lane down to 252 - 4*lane
      uint32_t cnt[4], tot = 0;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        cnt[i] = hist[255 - 4 * lane - i];
        tot += cnt[i];
      }
      uint32_t incl = tot;
#pragma unroll
      for (int off = 1; off < 64; off *= 2) {
        const uint32_t y = __shfl_up(incl, off);
        if (lane >= off) incl += y;
      }
      uint32_t above = incl - tot;  // candidates with a larger digit
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        if (above < want && above + cnt[i] >= want) {
          pick[0] = 255u - 4u * lane - i;
          pick[1] = want - above;
        }
        above += cnt[i];
      }
    }
    __syncthreads();
    prefix |= pick[0] << shift;
    pmask |= 255u << shift;
    want = pick[1];
  }
  const uint32_t thr = prefix;  // the k-th largest key
  const uint32_t need = want;   // keys equal to thr that are retained (lowest indices)

  // 2. Retained tokens in ascending order: position of a retained token =
  //    (larger keys before it) + min(equal keys before it, need).
  const SliceRoute rk = route_slice(p, 0, s), rv = route_slice(p, 1, s);
  const uint16_t* src_k = p.cache[0] + ((size_t)s * p.T + p.s0) * D;
  const uint16_t* src_v = p.cache[1] + ((size_t)s * p.T + p.s0) * D;
  uint16_t* dst_k = rk.kept ? nullptr : p.ret[0] + ((size_t)rk.slot * p.B + rk.b) * k * D;
  uint16_t* dst_v = rv.kept ? nullptr : p.ret[1] + ((size_t)rv.slot * p.B + rv.b) * k * D;
  int32_t* idx = p.ret_idx + (size_t)s * k;
  const uint64_t below = (1ull << lane) - 1ull;
  uint32_t carry_gt = 0, carry_eq = 0;
  for (int c0 = 0; c0 < n; c0 += kThreads) {
    const int t = c0 + tid;
    const uint32_t u = t < n ? key[t] : 0u;
    const bool gt = t < n && u > thr;
    const bool eq = t < n && u == thr;
    const uint64_t bg = __ballot(gt), be = __ballot(eq);
    if (lane == 0) {
      wcount[wave][0] = (uint32_t)__popcll(bg);
      wcount[wave][1] = (uint32_t)__popcll(be);
    }
    __syncthreads();
    uint32_t pg = carry_gt + (uint32_t)__popcll(bg & below);
    uint32_t pe = carry_eq + (uint32_t)__popcll(be & below);
    uint32_t tg = 0, te = 0;
#pragma unroll
    for (int w = 0; w < WAVES; ++w) {
      if (w < wave) {
        pg += wcount[w][0];
        pe += wcount[w][1];
      }
      tg += wcount[w][0];
      te += wcount[w][1];
    }
    const uint32_t base = carry_gt + min(carry_eq, need);
    const uint32_t pos = pg + min(pe, need);
    if ((gt || (eq && pe < need)) && pos < k) {  // exactly k positions are taken
      idx[pos] = t;
      sel[pos - base] = t;
    }
    carry_gt += tg;
    carry_eq += te;
    // retained in this chunk (the bound only guards the buffers)
    const uint32_t m = min(carry_gt + min(carry_eq, need), k) - min(base, k);
    __syncthreads();
    if (m > 0) {
      if (dst_k) gather_rows<D>(src_k, dst_k, sel, m, base);
      if (dst_v) gather_rows<D>(src_v, dst_v, sel, m, base);
    }
  }
}

// ------------------------------------------------------------ write-back

// One workgroup per (l, b, h): the retained rows over p.out's image span.
template <int D>
__global__ __launch_bounds__(kThreads) void retain_scatter_kernel(const Params p) {
  constexpr int VPT = D / 8;
  const uint32_t s = blockIdx.x;
  const uint32_t k = (uint32_t)p.k;
  const int32_t* idx = p.ret_idx + (size_t)s * k;
#pragma unroll
  for (int X = 0; X < 2; ++X) {
    const SliceRoute r = route_slice(p, X, s);
    if (r.kept) continue;
    const uint16_t* src = p.ret[X] + ((size_t)r.slot * p.B + r.b) * k * D;
    uint16_t* dst = p.out[X] + ((size_t)s * p.T + p.s0) * D;
    for (uint32_t i = threadIdx.x; i < k * VPT; i += kThreads) {
      const uint32_t row = i / VPT, c = i % VPT;
      const uint32_t t = (uint32_t)idx[row];
      if (t >= (uint32_t)p.n) continue;  // not a token of the span: never written
      const u32x4 v = *(const u32x4*)(src + (size_t)row * D + 8 * c);
      store_nt((u32x4*)(dst + (size_t)t * D + 8 * c), v);
    }
  }
}

// ------------------------------------------------------------ launchers

hipError_t launch_key_norms(const Params& p, int D, hipStream_t stream) {
  const uint32_t blocks = (uint32_t)p.L * p.B * p.H * (uint32_t)p.tiles;
  if (D == 64)
    hipLaunchKernelGGL((key_norm_kernel<64>), dim3(blocks), dim3(kThreads), 0, stream, p);
  else if (D == 128)
    hipLaunchKernelGGL((key_norm_kernel<128>), dim3(blocks), dim3(kThreads), 0, stream, p);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

hipError_t launch_retain_select(const Params& p, int D, hipStream_t stream) {
  const uint32_t blocks = (uint32_t)p.L * p.B * p.H;
  if (D == 64)
    hipLaunchKernelGGL((retain_select_kernel<64>), dim3(blocks), dim3(kThreads), 0, stream, p);
  else if (D == 128)
    hipLaunchKernelGGL((retain_select_kernel<128>), dim3(blocks), dim3(kThreads), 0, stream, p);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

hipError_t launch_retain_scatter(const Params& p, int D, hipStream_t stream) {
  const uint32_t blocks = (uint32_t)p.L * p.B * p.H;
  if (D == 64)
    hipLaunchKernelGGL((retain_scatter_kernel<64>), dim3(blocks), dim3(kThreads), 0, stream, p);
  else if (D == 128)
    hipLaunchKernelGGL((retain_scatter_kernel<128>), dim3(blocks), dim3(kThreads), 0, stream, p);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

}  // namespace hg
