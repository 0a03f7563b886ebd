// Fused simulated quantization for gfx950: the image rows of every
// unprotected head are quantized by the base and reconstructed to BF16 in
// registers, in one pass over the cache (HeadGuard §4, Quantization setup:
// entries assigned low precision are rounded to the base quantizer's levels and
// reconstructed as floating-point values).  The result is bit-identical to
// hg_quantize followed by hg_dequantize, without the packed buffers: 4 bytes
// of traffic per element instead of about 4.6.  Protected rows are copied
// (or left alone when the output is the input); text rows are not written.
//
// Work decomposition as in quantize.hip (a workgroup per slice and four
// wavefront tiles of 32 image tokens; 16 in the min-max instantiation at
// head_dim 128, see kFakeTokens).  Per-token groups are computed with a lane quad
// per token and the reconstructed rows are transposed through LDS so that
// every store instruction writes whole consecutive token rows; KIVI keys are
// computed and stored in the whole-row load layout directly.

#include "hg_device.h"
#include "hg_kernels.h"

namespace hg {

// Tokens per wavefront tile.  Half of the traffic is stores, and write
// throughput falls with the store instructions a wavefront issues back to
// back, so the min-max instantiation at head_dim 128 (min-max caches, and
// the value tiles of the other bases) takes 16 tokens, one pass.  KIVI key
// groups need their 32 tokens in one wavefront.
template <int BASE, int D>
constexpr int kFakeTokens = (D == 128 && BASE == HG_BASE_MINMAX) ? 16 : kWaveTokens;


template <int D, int BITS, bool ROTATE, bool NORM, int TOKENS>
// rows and out may be the same memory (in place): no restrict qualifiers.
__device__ __forceinline__ void fake_tokens(const uint16_t* rows, uint16_t* out, float* norm,
                                            int t_first, int n, int lane, u32x4* __restrict__ stage) {
  constexpr int G = kTokenLanes<D>;     // lanes per token
  constexpr int E = D / G;             // elements per lane
  constexpr int NV = E / 8;            // 16-byte chunks per lane
  constexpr int TPP = 64 / G;          // tokens per pass
  constexpr int PASSES = TOKENS / TPP;
  constexpr int PB = PASSES < 2 ? PASSES : 2;  // passes whose loads are issued together
  constexpr int CPT = D / 8;           // chunks per token row
  constexpr int RPL = 64 / CPT;        // token rows per store instruction
  constexpr int NSP = TPP / RPL;       // store instructions per pass
  constexpr int LEVELS = (1 << BITS) - 1;
  const int j = lane % G;
  const int q = lane / G;
  // Head_dim 256: whole-row streaming loads moved into the quad layout through
  // the stage, as in the quantize kernel.
  constexpr bool kStaged = D == 256;
  constexpr int LPR = D / 8;           // staged loads: lanes per token row,
  constexpr int RPI = 64 / LPR;        // token rows per load instruction,
  constexpr int IPP = TPP / RPI;       // load instructions per pass

#pragma unroll
  for (int p0 = 0; p0 < PASSES; p0 += PB) {
    // Tokens past the span's end load the last token (never stored).
    u32x4 raw[PB][NV];
    u32x4 whole[kStaged ? PB * IPP : 1];
    if constexpr (kStaged) {
#pragma unroll
      for (int i = 0; i < PB * IPP; ++i) {
        const int t = min(t_first + p0 * TPP + i * RPI + lane / LPR, n - 1);
        whole[i] = __builtin_nontemporal_load((const u32x4*)(rows + (size_t)t * D) + lane % LPR);
      }
    } else {
#pragma unroll
      for (int b = 0; b < PB; ++b) {
        const int t = min(t_first + (p0 + b) * TPP + q, n - 1);
        const u32x4* src = (const u32x4*)(rows + (size_t)t * D + j * E);
#pragma unroll
        for (int k = 0; k < NV; ++k) raw[b][k] = src[k];
      }
    }

    // Rotated keys (and the staged loads) unroll both passes: rolled, their
    // per-pass register arrays went to scratch memory.  The plain path is
    // faster rolled (measured).
    constexpr int kUnrolledPasses = ROTATE || kStaged ? PB : 1;
#pragma unroll kUnrolledPasses
    for (int pass = 0; pass < PB; ++pass) {
      if constexpr (kStaged) {
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
#pragma unroll
        for (int i = 0; i < IPP; ++i) stage[stage_slot<D>(i * RPI + lane / LPR, lane % LPR)] = whole[pass * IPP + i];
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
#pragma unroll
        for (int k = 0; k < NV; ++k) raw[pass][k] = stage[stage_slot<D>(q, j * NV + k)];
      }
      float x[E];
#pragma unroll
      for (int k = 0; k < NV; ++k) {
        x[8 * k + 0] = bf16_lo(raw[pass][k].x);
        x[8 * k + 1] = bf16_hi(raw[pass][k].x);
        x[8 * k + 2] = bf16_lo(raw[pass][k].y);
        x[8 * k + 3] = bf16_hi(raw[pass][k].y);
        x[8 * k + 4] = bf16_lo(raw[pass][k].z);
        x[8 * k + 5] = bf16_hi(raw[pass][k].z);
        x[8 * k + 6] = bf16_lo(raw[pass][k].w);
        x[8 * k + 7] = bf16_hi(raw[pass][k].w);
      }
      if constexpr (NORM) {  // squared key norm for token retention, before the rotation
        const float sq = quad_sqnorm<E, G>(x);
        const int t = t_first + (p0 + pass) * TPP + q;
        if (t < n && j == 0) norm[t] = sq;
      }
      if constexpr (ROTATE) fwht_quad<E, G>(x, j, fwht_scale<D>());

      float mn = x[0], mx = x[0];
#pragma unroll
      for (int e = 1; e < E; ++e) {
        mn = fminf(mn, x[e]);
        mx = fmaxf(mx, x[e]);
      }
      mn = group_min<G>(mn);
      mx = group_max<G>(mx);
      const GroupScale g = group_scale<LEVELS>(mn, mx);
      const float S = bf16_as_float(g.meta & 0xFFFFu);

      // Level of each code, q*S + m (q*S exact, one rounding), then the inverse
      // rotation for AKVQ keys, then BF16.
#pragma unroll
      for (int e = 0; e < E; ++e) {
        x[e] = __builtin_fmaf(__builtin_rintf(code_scaled(x[e], g)), S, g.m);
      }
      if constexpr (ROTATE) fwht_quad<E, G>(x, j, fwht_scale<D>());

      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
#pragma unroll
      for (int k = 0; k < NV; ++k) {
        const u32x4 v = {pack_bf16x2_hw(x[8 * k + 0], x[8 * k + 1]), pack_bf16x2_hw(x[8 * k + 2], x[8 * k + 3]),
                         pack_bf16x2_hw(x[8 * k + 4], x[8 * k + 5]), pack_bf16x2_hw(x[8 * k + 6], x[8 * k + 7])};
        stage[stage_slot<D>(q, j * NV + k)] = v;
      }
      // LDS operations of one wavefront execute in order; the fences keep the
      // compiler from moving the accesses across each other.
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
      const int c = lane % CPT;
      const int r = lane / CPT;
#pragma unroll
      for (int k = 0; k < NSP; ++k) {
        const int tl = r + RPL * k;
        const int t = t_first + (p0 + pass) * TPP + tl;
        const u32x4 v = stage[stage_slot<D>(tl, c)];
        if (t < n) store_nt((u32x4*)(out + (size_t)t * D + 8 * c), v);
      }
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    }
  }
}

template <int D, int BITS>
__device__ __forceinline__ void fake_kivi_keys(const uint16_t* rows, uint16_t* out,
                                               int g_first, int n, int lane) {
  constexpr int DH = D < 128 ? D : 128;  // channels per pass (head_dim 256: two passes)
  constexpr int LPR = DH / 8;            // lanes per token row (8 channels each)
  constexpr int RPL = 64 / LPR;          // token rows per load
  constexpr int NL = kWaveTokens / RPL;  // loads per lane
  constexpr int LEVELS = (1 << BITS) - 1;
  const int r = lane / LPR;

#pragma unroll
  for (int h = 0; h < D / DH; ++h) {
    const int c8 = h * LPR + lane % LPR;

    u32x4 raw[NL];
#pragma unroll
    for (int k = 0; k < NL; ++k) {
      const int t = min(g_first + r + RPL * k, n - 1);  // past-the-end rows: excluded below
      raw[k] = __builtin_nontemporal_load((const u32x4*)(rows + (size_t)t * D + 8 * c8));  // whole rows: streaming
    }
    float x[NL][8];
#pragma unroll
    for (int k = 0; k < NL; ++k) {
      x[k][0] = bf16_lo(raw[k].x); x[k][1] = bf16_hi(raw[k].x);
      x[k][2] = bf16_lo(raw[k].y); x[k][3] = bf16_hi(raw[k].y);
      x[k][4] = bf16_lo(raw[k].z); x[k][5] = bf16_hi(raw[k].z);
      x[k][6] = bf16_lo(raw[k].w); x[k][7] = bf16_hi(raw[k].w);
    }
    GroupScale g[8];
    float S[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      float mn = __builtin_inff(), mx = -__builtin_inff();
#pragma unroll
      for (int k = 0; k < NL; ++k) {
        const bool ok = g_first + r + RPL * k < n;
        mn = fminf(mn, ok ? x[k][e] : __builtin_inff());
        mx = fmaxf(mx, ok ? x[k][e] : -__builtin_inff());
      }
#pragma unroll
      for (int off = LPR; off < 64; off *= 2) {
        mn = fminf(mn, __shfl_xor(mn, off));
        mx = fmaxf(mx, __shfl_xor(mx, off));
      }
      g[e] = group_scale<LEVELS>(mn, mx);
      S[e] = bf16_as_float(g[e].meta & 0xFFFFu);
    }
#pragma unroll
    for (int k = 0; k < NL; ++k) {
      const int t = g_first + r + RPL * k;
      float y[8];
#pragma unroll
      for (int e = 0; e < 8; ++e)
        y[e] = __builtin_fmaf(__builtin_rintf(code_scaled(x[k][e], g[e])), S[e], g[e].m);
      const u32x4 v = {pack_bf16x2_hw(y[0], y[1]), pack_bf16x2_hw(y[2], y[3]), pack_bf16x2_hw(y[4], y[5]),
                       pack_bf16x2_hw(y[6], y[7])};
      if (t < n) store_nt((u32x4*)(out + (size_t)t * D + 8 * c8), v);
    }
  }
}

// NORM (AKVQ keys, out of place only): also write every image key's squared
// norm for token retention, from the rows this pass reads anyway.
template <int BASE, int D, int BITS, bool NORM>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(kMinWaves)))
void fake_quantize_kernel(const Params p) {
  clear_words_share(p);
  const Slice sl = decode_launch_block(p, blockIdx.x);
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  constexpr int kTokens = kFakeTokens<BASE, D>;
  const int t_first = sl.tile * (kThreads / 64) * kTokens + wave * kTokens;
  if (t_first >= p.n) return;

  const size_t base = ((size_t)sl.s * p.T + p.s0) * D;
  const uint16_t* rows = p.cache[sl.X] + base;
  uint16_t* out = p.out[sl.X] + base;
  float* norm = NORM ? p.norm + (size_t)sl.s * p.n : nullptr;  // used for K only
  if (sl.kept) {
    if (NORM && sl.X == 0)
      copy_wave_rows<D, kTokens, NORM, false, true>(rows, out, norm, t_first, p.n, lane);
    else if (out != rows)
      copy_wave_rows<D, kTokens, false, true, true>(rows, out, nullptr, t_first, p.n, lane);
    return;
  }
  if (sl.X == 0 && p.kivi_whole) return;  // whole-sequence KIVI key ranges: kivi_seq.hip
  if (BASE == HG_BASE_KIVI && sl.X == 0) {
    static_assert(BASE != HG_BASE_KIVI || kTokens == kWaveTokens, "a wavefront holds a whole key group");
    fake_kivi_keys<D, BITS>(rows, out, t_first, p.n, lane);
  } else {
    __shared__ u32x4 stage_all[kThreads / 64][(64 / kTokenLanes<D>) * (D / 8)];  // one pass of tokens
    if (BASE == HG_BASE_AKVQ && sl.X == 0)
      fake_tokens<D, BITS, true, NORM, kTokens>(rows, out, norm, t_first, p.n, lane, stage_all[wave]);
    else
      fake_tokens<D, BITS, false, false, kTokens>(rows, out, nullptr, t_first, p.n, lane, stage_all[wave]);
  }
}

// Dynamic LDS of a one-pass launch: the occupancy cap's reservation, less the
// static stage of the per-token path.
template <int D>
constexpr size_t fake_lds() {
  return occupancy_lds(kFakeQuantizeWaves) - (kThreads / 64) * (64 / kTokenLanes<D>) * (D / 8) * 16;
}

// The workgroup tiles of a launch follow its kernel's tile size.
template <int BASE, int D, int BITS>
static hipError_t launch_f(const Params& p, Tensors which, bool norms, hipStream_t stream) {
  constexpr int kTile = (kThreads / 64) * kFakeTokens<BASE, D>;
  static_assert(kTile >= kMinBlockTokens, "the host's grid check assumes this tile at least");
  Params pf = p;
  pf.tiles = (p.n + kTile - 1) / kTile;
  const uint64_t per_tensor = (uint64_t)p.L * p.B * p.H * (uint64_t)pf.tiles;
  const bool kept = which == Tensors::kKeptKeysAndValues;
  const uint64_t blocks_k = which == Tensors::kValues ? 0
                            : kept ? (uint64_t)(p.L * p.H - p.n_unprot_k) * p.B * pf.tiles : per_tensor;
  const uint64_t blocks = which == Tensors::kKeys ? per_tensor : blocks_k + per_tensor;
  if (blocks > 0x7FFFFFFFull) return hipErrorInvalidConfiguration;
  pf.blocks_k = (uint32_t)blocks_k;
  pf.kept_keys = kept;
  if constexpr (BASE == HG_BASE_AKVQ) {
    if (norms) {
      hipLaunchKernelGGL((fake_quantize_kernel<BASE, D, BITS, true>), dim3((uint32_t)blocks), dim3(kThreads), fake_lds<D>(),
                         stream, pf);
      return hipGetLastError();
    }
  }
  if (norms) return hipErrorInvalidValue;  // key norms belong to the AKVQ base
  hipLaunchKernelGGL((fake_quantize_kernel<BASE, D, BITS, false>), dim3((uint32_t)blocks), dim3(kThreads), fake_lds<D>(),
                     stream, pf);
  return hipGetLastError();
}

template <int BASE, int D>
static hipError_t launch_f_bits(const Params& p, int bits, Tensors which, bool norms, hipStream_t stream) {
  switch (bits) {
    case 2: return launch_f<BASE, D, 2>(p, which, norms, stream);
    case 3: return launch_f<BASE, D, 3>(p, which, norms, stream);
    case 4: return launch_f<BASE, D, 4>(p, which, norms, stream);
    default: return hipErrorInvalidValue;
  }
}

template <int BASE>
static hipError_t launch_f_dim(const Params& p, int D, int bits, Tensors which, bool norms, hipStream_t stream) {
  switch (D) {
    case 64: return launch_f_bits<BASE, 64>(p, bits, which, norms, stream);
    case 128: return launch_f_bits<BASE, 128>(p, bits, which, norms, stream);
    case 256: return launch_f_bits<BASE, 256>(p, bits, which, norms, stream);
    default: return hipErrorInvalidValue;
  }
}

// Value tiles of the KIVI-style and AKVQ-style bases run as a launch of the
// min-max instantiation, which needs fewer registers than their key paths
// (as in launch_quantize); with KIVI keys over the whole sequence the whole
// launch does, its key blocks listing the protected key slices alone (out of
// place they are copied; in place they need nothing, and the launch takes the
// values only).
hipError_t launch_fake_quantize(const Params& p, int base, int D, int bits, bool norms, hipStream_t stream) {
  if (base == HG_BASE_KIVI && p.kivi_whole) {
    const bool in_place = p.out[0] == p.cache[0];
    return launch_f_dim<HG_BASE_MINMAX>(p, D, bits, in_place ? Tensors::kValues : Tensors::kKeptKeysAndValues,
                                        norms, stream);
  }
  if (base == HG_BASE_MINMAX) return launch_f_dim<HG_BASE_MINMAX>(p, D, bits, Tensors::kBoth, norms, stream);
  if (base != HG_BASE_KIVI && base != HG_BASE_AKVQ) return hipErrorInvalidValue;
  hipError_t e = base == HG_BASE_KIVI ? launch_f_dim<HG_BASE_KIVI>(p, D, bits, Tensors::kKeys, norms, stream)
                                      : launch_f_dim<HG_BASE_AKVQ>(p, D, bits, Tensors::kKeys, norms, stream);
  if (e != hipSuccess) return e;
  return launch_f_dim<HG_BASE_MINMAX>(p, D, bits, Tensors::kValues, false, stream);
}

}  // namespace hg
