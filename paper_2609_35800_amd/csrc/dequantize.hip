// Dequantize kernels for gfx950, one instantiation per (base, head_dim,
// bits): the reconstruction of simulated quantization (HeadGuard §4,
// Quantization setup: entries are rounded to the base's levels and rebuilt as
// floating-point values for attention).  x^ = bf16_rne(q*S + m); q*S is exact
// (q < 16, S has 8 significant bits), so the fma equals the separate multiply
// and add; the BF16 rounding is the hardware conversion (round to nearest
// even, subnormals kept).  AKVQ keys are rotated back in fp32 before the BF16 rounding.
// Protected rows come back from the side store; text rows are not written.
//
// A workgroup owns one (tensor, l, b, h) slice and 4 wavefront tiles of
// consecutive image tokens (kDequantTokens per wavefront), and every path
// holds a token row across D/8 lanes so that stores are whole contiguous rows.

#include "hg_device.h"
#include "hg_kernels.h"

namespace hg {

// Tokens per wavefront tile.  Stores are 80 % of the traffic, and write
// throughput falls with the store instructions a wavefront issues back to
// back (measured write-only: one 1 KiB store per wavefront 6.8 TB/s, two
// 6.1-6.4, eight 5.5-5.8), so the min-max and KIVI-style paths at head_dim
// 128 take 16 tokens (four stores of whole rows).  The rotated AKVQ keys and
// head_dim 256 measured slower with the shorter tile and keep 32.
template <int BASE, int D>
constexpr int kDequantTokens = (D == 128 && BASE != HG_BASE_AKVQ) ? 16 : kWaveTokens;

// Per-token groups.  A token row is held by D/8 lanes, lane c holding
// channels [8c, 8c + 8), so each 16-byte store instruction of the wavefront
// writes 64/(D/8) whole consecutive token rows (one contiguous 1 KiB run for
// D = 128; two 512-byte rows at 256).  AKVQ keys are rotated back across the
// row's lanes first.
template <int D, int BITS, bool ROTATE, int TOKENS>
__device__ __forceinline__ void dequantize_tokens(const uint8_t* __restrict__ codes,
                                                  const uint32_t* __restrict__ meta,
                                                  uint16_t* __restrict__ rows,
                                                  int t_first, int n, int lane) {
  constexpr int LPT = D / 8;               // lanes per token row
  constexpr int TPI = 64 / LPT;            // token rows per instruction
  constexpr int NP = TOKENS / TPI;         // instructions per wavefront tile
  constexpr int ROW = D * BITS / 8;
  constexpr uint32_t kMask = (1u << BITS) - 1u;
  const int c = lane % LPT;
  const int r = lane / LPT;

  // Past-the-end tokens read the last token (not stored): loads unconditional.
  uint32_t pc[NP], mw[NP];
#pragma unroll
  for (int k = 0; k < NP; ++k) {
    const int t = min(t_first + r + TPI * k, n - 1);
    pc[k] = load_piece8<BITS, ROW>(codes + (size_t)t * ROW, c);
    mw[k] = meta[t];
  }
#pragma unroll
  for (int k = 0; k < NP; ++k) {
    const int t = t_first + r + TPI * k;
    const float S = bf16_as_float(mw[k] & 0xFFFFu);
    const float m = bf16_as_float(mw[k] >> 16);
    float y[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) y[e] = __builtin_fmaf((float)((pc[k] >> (BITS * e)) & kMask), S, m);
    if constexpr (ROTATE) fwht_row<D>(y, c);
    if (t < n) {
      u32x4 v = {pack_bf16x2_hw(y[0], y[1]), pack_bf16x2_hw(y[2], y[3]), pack_bf16x2_hw(y[4], y[5]),
                 pack_bf16x2_hw(y[6], y[7])};
      store_nt((u32x4*)(rows + (size_t)t * D + 8 * c), v);
    }
  }
}

template <int D, int BITS, int TOKENS>
__device__ __forceinline__ void dequantize_kivi_keys(const uint8_t* __restrict__ codes,
                                                     const uint32_t* __restrict__ meta,
                                                     uint16_t* __restrict__ rows,
                                                     int g_first, int group, int n, int lane) {
  constexpr int DH = D < 128 ? D : 128;  // channels per pass (head_dim 256: two passes)
  constexpr int LPR = DH / 8;
  constexpr int RPL = 64 / LPR;
  constexpr int NL = TOKENS / RPL;
  constexpr int ROW = D * BITS / 8;
  const int r = lane / LPR;

#pragma unroll
  for (int h = 0; h < D / DH; ++h) {
    const int c8 = h * LPR + lane % LPR;

    const u32x4* mp = (const u32x4*)(meta + (size_t)group * D + 8 * c8);
    const u32x4 m0 = mp[0], m1 = mp[1];
    const uint32_t mw[8] = {m0.x, m0.y, m0.z, m0.w, m1.x, m1.y, m1.z, m1.w};
    float S[8], m[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      S[e] = bf16_as_float(mw[e] & 0xFFFFu);
      m[e] = bf16_as_float(mw[e] >> 16);
    }

    constexpr uint32_t kMask = (1u << BITS) - 1u;
    uint32_t pc[NL];
#pragma unroll
    for (int k = 0; k < NL; ++k) {
      const int t = min(g_first + r + RPL * k, n - 1);
      pc[k] = load_piece8<BITS, ROW>(codes + (size_t)t * ROW, c8);
    }
#pragma unroll
    for (int k = 0; k < NL; ++k) {
      const int t = g_first + r + RPL * k;
      float y[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) y[e] = __builtin_fmaf((float)((pc[k] >> (BITS * e)) & kMask), S[e], m[e]);
      if (t < n) {
        u32x4 v = {pack_bf16x2_hw(y[0], y[1]), pack_bf16x2_hw(y[2], y[3]), pack_bf16x2_hw(y[4], y[5]),
                   pack_bf16x2_hw(y[6], y[7])};
        store_nt((u32x4*)(rows + (size_t)t * D + 8 * c8), v);
      }
    }
  }
}

template <int BASE, int D, int BITS>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(kMinWaves))) void dequantize_kernel(const Params p) {
  const Slice sl = decode_block(p, blockIdx.x);
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  constexpr int kTokens = kDequantTokens<BASE, D>;
  const int t_first = sl.tile * (kThreads / 64) * kTokens + wave * kTokens;
  if (t_first >= p.n) return;

  uint16_t* rows = const_cast<uint16_t*>(p.cache[sl.X]) + ((size_t)sl.s * p.T + p.s0) * D;
  const size_t slab = (size_t)sl.slot * p.B + sl.b;

  if (sl.kept) {
    copy_wave_rows<D, kTokens>(p.side[sl.X] + slab * p.n * D, rows, nullptr, t_first, p.n, lane);
    return;
  }
  const uint8_t* codes = p.codes[sl.X] + slab * p.n * (D * BITS / 8);
  if (BASE == HG_BASE_KIVI && sl.X == 0) {
    const int group = p.kivi_whole ? 0 : t_first / kWaveTokens;  // 32-token key groups
    dequantize_kivi_keys<D, BITS, kTokens>(codes, p.meta[0] + slab * p.ngroups * D, rows, t_first, group, p.n, lane);
  } else {
    const uint32_t* meta = p.meta[sl.X] + slab * p.n;
    if (BASE == HG_BASE_AKVQ && sl.X == 0)
      dequantize_tokens<D, BITS, true, kTokens>(codes, meta, rows, t_first, p.n, lane);
    else
      dequantize_tokens<D, BITS, false, kTokens>(codes, meta, rows, t_first, p.n, lane);
  }
}

// Launches of the min-max instantiation that write less than this many bytes
// of rows keep kDequantizeWaves per SIMD (Qwen-shaped cache 130.7 -> 127 us,
// one GPU's share of the 72B-shaped cache split 8 ways 116.8 -> 112.6 us;
// the larger caches unchanged at the min-max cap).
constexpr uint64_t kDequantizeSmallBytes = 1ull << 30;

// The workgroup tiles of the launch follow this kernel's tile size.
template <int BASE, int D, int BITS>
static hipError_t launch_d(const Params& p, Tensors which, hipStream_t stream) {
  constexpr int kTile = (kThreads / 64) * kDequantTokens<BASE, D>;
  static_assert(kTile >= kMinBlockTokens, "the host's grid check assumes this tile at least");
  Params pd = p;
  pd.tiles = (p.n + kTile - 1) / kTile;
  const uint64_t per_tensor = (uint64_t)p.L * p.B * p.H * (uint64_t)pd.tiles;
  const uint64_t blocks = which == Tensors::kBoth ? 2 * per_tensor : per_tensor;
  if (blocks > 0x7FFFFFFFull) return hipErrorInvalidConfiguration;
  pd.blocks_k = which == Tensors::kValues ? 0u : (uint32_t)per_tensor;
  const uint64_t row_bytes = blocks / (uint64_t)pd.tiles * (uint64_t)p.n * D * 2;  // rows the launch writes
  const int waves =
      BASE == HG_BASE_MINMAX && row_bytes >= kDequantizeSmallBytes ? kDequantizeWavesMinMax : kDequantizeWaves;
  hipLaunchKernelGGL((dequantize_kernel<BASE, D, BITS>), dim3((uint32_t)blocks), dim3(kThreads),
                     occupancy_lds(waves), stream, pd);
  return hipGetLastError();
}

template <int BASE, int D>
static hipError_t launch_d_bits(const Params& p, int bits, Tensors which, hipStream_t stream) {
  switch (bits) {
    case 2: return launch_d<BASE, D, 2>(p, which, stream);
    case 3: return launch_d<BASE, D, 3>(p, which, stream);
    case 4: return launch_d<BASE, D, 4>(p, which, stream);
    default: return hipErrorInvalidValue;
  }
}

template <int BASE>
static hipError_t launch_d_dim(const Params& p, int D, int bits, Tensors which, hipStream_t stream) {
  switch (D) {
    case 64: return launch_d_bits<BASE, 64>(p, bits, which, stream);
    case 128: return launch_d_bits<BASE, 128>(p, bits, which, stream);
    case 256: return launch_d_bits<BASE, 256>(p, bits, which, stream);
    default: return hipErrorInvalidValue;
  }
}

// KIVI-style and AKVQ-style values are dequantized per token exactly as
// min-max ones, so they run as a second launch of the min-max instantiation,
// with its shorter tiles and occupancy rule (the KIVI-style values in it:
// LLaVA-NeXT-shaped dequantize 1252 -> 1239 us at 2 bits, 1359 -> 1305 at 4).
hipError_t launch_dequantize(const Params& p, int base, int D, int bits, hipStream_t stream) {
  if (base == HG_BASE_MINMAX) return launch_d_dim<HG_BASE_MINMAX>(p, D, bits, Tensors::kBoth, stream);
  if (base != HG_BASE_KIVI && base != HG_BASE_AKVQ) return hipErrorInvalidValue;
  const hipError_t e = base == HG_BASE_KIVI ? launch_d_dim<HG_BASE_KIVI>(p, D, bits, Tensors::kKeys, stream)
                                            : launch_d_dim<HG_BASE_AKVQ>(p, D, bits, Tensors::kKeys, stream);
  return e != hipSuccess ? e : launch_d_dim<HG_BASE_MINMAX>(p, D, bits, Tensors::kValues, stream);
}

}  // namespace hg
