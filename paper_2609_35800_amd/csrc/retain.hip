// AKVQ-style token retention (HeadGuard §4, Quantization setup): in every KV
// head the keys and values of a nominal 2 % of the image tokens, those whose
// keys have the largest norms, stay in BF16, with or without head protection.
//
// The quantize kernel, and the one-pass simulated quantization out of place,
// write the squared key norm of every image token in the pass that reads the
// keys; key_norm_kernel computes them on their own for an in-place one-pass
// call, whose outputs would otherwise overwrite the rows to keep.  Then, per
// (l, b, h):
//  - retain_select_kernel (norms staged in LDS) finds the k-th largest norm by
//    a most-significant-digit-first radix select over the fp32 bit patterns
//    (non-negative, so they order as unsigned integers), starting below the
//    bits every norm of the head shares and stopping once the chosen digit's
//    candidates are all taken; lists the retained tokens in ascending order
//    (all larger norms, then the lowest-index ties); and, in the same
//    workgroup, gathers their K and V rows for each tensor the head does not
//    keep in BF16 (an out-of-place one-pass call, which computes the norms in
//    its own pass, copies them from the input straight to the output);
//  - retain_rows_kernel writes the gathered rows back over the
//    reconstruction.

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

// Keys held in LDS by the selection when the span fits this many tokens;
// longer spans read them from global memory (L2) in every pass.
constexpr int kResidentKeys = 12288;
constexpr int kRowsInFlight = 8;  // 16-byte row pieces in flight per thread when copying rows

// Copies the k retained rows of every tensor the head does not keep in BF16:
// kGather from p.cache into p.ret, kScatter from p.ret over p.out's image
// rows, kCacheToOut from p.cache straight into p.out.  `idx` lists the rows;
// an entry outside the span is not stored.
template <int D, RowCopy MODE>
__device__ __forceinline__ void copy_retained_rows(const Params& p, uint32_t s, const int32_t* idx) {
  constexpr int VPT = D / 8;  // 16-byte vectors per row
  constexpr int U = kRowsInFlight;
  const uint32_t k = (uint32_t)p.k;
  const size_t span = ((size_t)s * p.T + p.s0) * D;
  // sources and destinations of the tensors to copy: the first one not kept
  // in BF16, then V when both are copied
  const uint16_t* src[2];
  uint16_t* dst[2];
#pragma unroll
  for (int X = 0; X < 2; ++X) {
    const SliceRoute r = route_slice(p, X, s);
    uint16_t* ret = MODE == RowCopy::kCacheToOut ? nullptr : p.ret[X] + ((size_t)r.slot * p.B + r.b) * k * D;
    src[X] = MODE == RowCopy::kScatter ? ret : p.cache[X] + span;
    dst[X] = MODE == RowCopy::kGather ? ret : p.out[X] + span;
  }
  const bool k_kept = route_slice(p, 0, s).kept, v_kept = route_slice(p, 1, s).kept;
  const int nx = (k_kept ? 0 : 1) + (v_kept ? 0 : 1);
  if (k_kept) {
    src[0] = src[1];
    dst[0] = dst[1];
  }
  // row pieces of the first tensor, then of the second; retained-row buffers
  // are indexed by list position, image rows by token
  const uint32_t per = k * VPT, total = (uint32_t)nx * per;
  for (uint32_t i0 = threadIdx.x; i0 < total; i0 += U * kThreads) {
    u32x4 v[U];
    uint32_t tok[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const uint32_t i = min(i0 + u * kThreads, total - 1);
      const bool second = i >= per;
      const uint32_t e = second ? i - per : i, row = e / VPT, c = e % VPT;
      tok[u] = (uint32_t)idx[row];
      const uint32_t t = min(tok[u], (uint32_t)p.n - 1);
      const uint32_t at = MODE == RowCopy::kScatter ? row : t;
      v[u] = *(const u32x4*)((second ? src[1] : src[0]) + (size_t)at * D + 8 * c);
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const uint32_t i = i0 + u * kThreads;
      if (i >= total || tok[u] >= (uint32_t)p.n) continue;
      const bool second = i >= per;
      const uint32_t e = second ? i - per : i, row = e / VPT, c = e % VPT;
      const uint32_t at = MODE == RowCopy::kGather ? row : tok[u];
      store_nt((u32x4*)((second ? dst[1] : dst[0]) + (size_t)at * D + 8 * c), v[u]);
    }
  }
}

// One workgroup per (l, b, h); requires 1 <= k <= n.  Writes ret_idx, then
// copies the retained rows (kGather or kCacheToOut).
template <bool RESIDENT, int D, RowCopy MODE>
__global__ __launch_bounds__(kThreads) void retain_select_kernel(const Params p) {
  static_assert(kThreads == 256, "one histogram bin per thread");
  constexpr int WAVES = kThreads / 64;
  extern __shared__ uint32_t lds_keys[];  // n keys when RESIDENT
  __shared__ uint32_t hist[256];
  __shared__ uint32_t pick[3];
  __shared__ uint32_t wsum[WAVES][2];

  const uint32_t s = blockIdx.x;  // (l*B + b)*H + h
  const int n = p.n;
  const uint32_t k = (uint32_t)p.k;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const uint32_t* gkeys = (const uint32_t*)(p.norm + (size_t)s * n);
  uint32_t vmax = 0, vmin = ~0u;
  for (int t0 = tid; t0 < n; t0 += 4 * kThreads) {
    uint32_t u[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) u[i] = gkeys[min(t0 + i * kThreads, n - 1)];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      vmax = max(vmax, u[i]);  // clamped repeats of key n-1 change neither bound
      vmin = min(vmin, u[i]);
      if (RESIDENT && t0 + i * kThreads < n) lds_keys[t0 + i * kThreads] = u[i];
    }
  }
  const uint32_t* key = RESIDENT ? lds_keys : gkeys;

  // 0. Bounds of the keys: the bits above the highest bit in which the largest
  //    and smallest keys differ are common to every key, so the digits start
  //    below them.
#pragma unroll
  for (int off = 1; off < 64; off *= 2) {
    vmax = max(vmax, (uint32_t)__shfl_xor((int)vmax, off));
    vmin = min(vmin, (uint32_t)__shfl_xor((int)vmin, off));
  }
  if (lane == 0) {
    wsum[wave][0] = vmax;
    wsum[wave][1] = vmin;
  }
  __syncthreads();
#pragma unroll
  for (int w = 0; w < WAVES; ++w) {
    vmax = max(vmax, wsum[w][0]);
    vmin = min(vmin, wsum[w][1]);
  }
  const uint32_t diff = vmax ^ vmin;
  const int hb = diff ? 32 - __clz((int)diff) : 0;  // low bits that vary between keys
  uint32_t pmask = hb == 32 ? 0u : ~((1u << hb) - 1u);

  // 1. The k-th largest key, one 8-bit digit per pass from the top of the
  //    varying bits.  Candidates are the keys that match `prefix` under
  //    `pmask`; `want` of them are still to be taken.  The passes end once the
  //    digits are exhausted or every candidate of the chosen digit is taken
  //    (then no key outside the candidates ties with them).
  uint32_t prefix = vmax & pmask, want = k;
  bool done = hb == 0;  // all keys equal
  for (int shift = hb - 8; !done; shift -= 8) {
    shift = max(shift, 0);  // the last digit may repeat already fixed bits
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
          pick[2] = cnt[i];
        }
        above += cnt[i];
      }
    }
    __syncthreads();
    prefix |= pick[0] << shift;
    pmask |= 255u << shift;
    want = pick[1];
    done = shift == 0 || pick[1] == pick[2];
  }
  const uint32_t need = want;  // keys matching prefix that are retained (lowest indices)
  // Every wavefront has read the step-0 bounds from wsum before step 2 reuses
  // it; when all keys are equal the loop above ran no barrier.
  __syncthreads();

  // 2. Retained tokens in ascending order: every key above prefix under pmask,
  //    then the first `need` matching it.  Each thread owns a contiguous run of
  //    tokens; a block-wide exclusive scan of the per-run counts of larger and
  //    matching keys gives every run its starting counts, and the position of
  //    a retained token is (larger keys before it) + min(matching keys before
  //    it, need).
  const int run = (n + kThreads - 1) / kThreads;
  const int t_lo = min(tid * run, n), t_hi = min(t_lo + run, n);
  uint32_t cg = 0, ce = 0;
  for (int t = t_lo; t < t_hi; ++t) {
    const uint32_t u = key[t] & pmask;
    cg += u > prefix;
    ce += u == prefix;
  }
  uint32_t ig = cg, ie = ce;  // inclusive scans within the wavefront
#pragma unroll
  for (int off = 1; off < 64; off *= 2) {
    const uint32_t yg = __shfl_up(ig, off), ye = __shfl_up(ie, off);
    if (lane >= off) {
      ig += yg;
      ie += ye;
    }
  }
  if (lane == 63) {
    wsum[wave][0] = ig;
    wsum[wave][1] = ie;
  }
  __syncthreads();
  uint32_t pg = ig - cg, pe = ie - ce;
#pragma unroll
  for (int w = 0; w < WAVES; ++w) {
    if (w < wave) {
      pg += wsum[w][0];
      pe += wsum[w][1];
    }
  }
  int32_t* idx = p.ret_idx + (size_t)s * k;
  for (int t = t_lo; t < t_hi; ++t) {
    const uint32_t u = key[t] & pmask;
    const bool gt = u > prefix, eq = u == prefix;
    const uint32_t pos = pg + min(pe, need);
    if ((gt || (eq && pe < need)) && pos < k) idx[pos] = t;  // exactly k positions are taken
    pg += gt;
    pe += eq;
  }

  // 3. The retained rows, read back from the list just written (a workgroup
  //    barrier makes the global stores visible within the workgroup).
  __syncthreads();
  copy_retained_rows<D, MODE>(p, s, idx);
}

// ------------------------------------------------------------ retained rows

// Grid l*B*H: the retained rows of one (l, b, h) per workgroup, listed in
// p.ret_idx (the dequantize direction, and an in-place one-pass call).
template <int D, RowCopy MODE>
__global__ __launch_bounds__(kThreads) void retain_rows_kernel(const Params p) {
  copy_retained_rows<D, MODE>(p, blockIdx.x, p.ret_idx + (size_t)blockIdx.x * (uint32_t)p.k);
}

// ------------------------------------------------------------ launchers

hipError_t launch_key_norms(const Params& p, int D, hipStream_t stream) {
  const uint32_t blocks = (uint32_t)p.L * p.B * p.H * (uint32_t)p.tiles;
  if (D == 64)
    hipLaunchKernelGGL((key_norm_kernel<64>), dim3(blocks), dim3(kThreads), 0, stream, p);
  else if (D == 128)
    hipLaunchKernelGGL((key_norm_kernel<128>), dim3(blocks), dim3(kThreads), 0, stream, p);
  else if (D == 256)
    hipLaunchKernelGGL((key_norm_kernel<256>), dim3(blocks), dim3(kThreads), 0, stream, p);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

template <int D>
static hipError_t launch_rows_d(const Params& p, RowCopy mode, hipStream_t stream) {
  const dim3 grid((uint32_t)p.L * p.B * p.H);
  switch (mode) {
    case RowCopy::kGather:
      hipLaunchKernelGGL((retain_rows_kernel<D, RowCopy::kGather>), grid, dim3(kThreads), 0, stream, p);
      break;
    case RowCopy::kScatter:
      hipLaunchKernelGGL((retain_rows_kernel<D, RowCopy::kScatter>), grid, dim3(kThreads), 0, stream, p);
      break;
    default:
      hipLaunchKernelGGL((retain_rows_kernel<D, RowCopy::kCacheToOut>), grid, dim3(kThreads), 0, stream, p);
      break;
  }
  return hipGetLastError();
}

hipError_t launch_retain_rows(const Params& p, int D, RowCopy mode, hipStream_t stream) {
  if (D == 64) return launch_rows_d<64>(p, mode, stream);
  if (D == 128) return launch_rows_d<128>(p, mode, stream);
  if (D == 256) return launch_rows_d<256>(p, mode, stream);
  return hipErrorInvalidValue;
}

template <bool RESIDENT, int D>
static void launch_select_r(const Params& p, RowCopy mode, dim3 grid, size_t lds, hipStream_t stream) {
  if (mode == RowCopy::kGather)
    hipLaunchKernelGGL((retain_select_kernel<RESIDENT, D, RowCopy::kGather>), grid, dim3(kThreads), lds, stream, p);
  else
    hipLaunchKernelGGL((retain_select_kernel<RESIDENT, D, RowCopy::kCacheToOut>), grid, dim3(kThreads), lds,
                       stream, p);
}

template <int D>
static void launch_select_d(const Params& p, RowCopy mode, hipStream_t stream) {
  const dim3 grid((uint32_t)p.L * p.B * p.H);
  if (p.n <= kResidentKeys)
    launch_select_r<true, D>(p, mode, grid, (size_t)p.n * sizeof(uint32_t), stream);
  else
    launch_select_r<false, D>(p, mode, grid, 0, stream);
}

hipError_t launch_retain_select(const Params& p, int D, RowCopy mode, hipStream_t stream) {
  if (mode == RowCopy::kScatter) return hipErrorInvalidValue;
  if (D == 64)
    launch_select_d<64>(p, mode, stream);
  else if (D == 128)
    launch_select_d<128>(p, mode, stream);
  else if (D == 256)
    launch_select_d<256>(p, mode, stream);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

}  // namespace hg
