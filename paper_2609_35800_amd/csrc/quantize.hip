// Fused quantize + pack kernels for gfx950, one instantiation per
// (base, head_dim, bits).  HeadGuard §3 (Applying protection) and §4
// (Quantization setup): every image-token K/V vector of an unprotected head
// goes through the base quantizer, protected heads' image rows are copied to
// the BF16 side store, text rows are never read.
//
// Work decomposition: a 256-thread workgroup owns one (tensor, l, b, h) slice
// and 128 consecutive image tokens of it; each wavefront owns 32 tokens.
//  - Per-token groups (min-max K and V, KIVI V, AKVQ K and V): a lane quad
//    (eight lanes at head_dim 256) holds one token vector, lane j the E
//    contiguous elements [j*E, (j+1)*E) loaded with 16-byte loads (head_dim
//    256: whole rows are loaded and moved into this layout through LDS); the
//    range is reduced with two (three) DPP exchanges; a lane's codes form one
//    contiguous piece of the packed row.  A wavefront covers 16 (8) tokens per
//    pass, two (four) passes.
//  - KIVI keys: the wavefront holds one 32-token group; lanes cover D/8
//    channel octets per token row (head_dim 256: one half of the channels at
//    a time) and 64/(D/8) token rows per load, so the per-channel range over
//    tokens is an in-register reduction plus cross-row shuffles.
//  - AKVQ keys: the normalized Walsh-Hadamard rotation runs on the token's
//    lanes before the range reduction: spans 1..E/2 in registers, the rest
//    by DPP exchanges.
//  - Protected slices: 16-byte copies of the image rows to the side store.
//  - AKVQ-style token retention: the same pass also writes the squared norm of
//    every image key (quad or row tree, see tree_sqnorm), before any rotation.
// All per-group arithmetic is IEEE fp32 (no contraction), the same operations
// in the same order as the reference definition.

#include "hg_device.h"
#include "hg_kernels.h"

namespace hg {

// ---------------------------------------------------------- per-token path

// Head_dim 256 loads the token rows whole (each instruction reads two
// complete 512-byte rows, streaming) and moves each pass into the quad layout
// through the wavefront's LDS stage: 3 % faster there than loading the quad
// layout directly.  At 64 and 128 the direct loads measured faster.
template <int D>
constexpr bool kStagedLoads = D == 256;

template <int D, int BITS, bool ROTATE, bool NORM>
__device__ __forceinline__ void quantize_tokens(const uint16_t* __restrict__ rows,
                                                uint8_t* __restrict__ codes,
                                                uint32_t* __restrict__ meta,
                                                float* __restrict__ norm,
                                                int t_first, int n, int lane, u32x4* __restrict__ stage) {
  constexpr int G = kTokenLanes<D>;     // lanes per token
  constexpr int E = D / G;             // elements per lane
  constexpr int NV = E / 8;            // 16-byte loads per lane per token
  constexpr int TPP = 64 / G;          // tokens per pass of the wavefront
  constexpr int PASSES = kWaveTokens / TPP;
  constexpr int LEVELS = (1 << BITS) - 1;
  constexpr int ROW = D * BITS / 8;    // packed bytes per token
  constexpr int PIECE = E * BITS / 8;  // packed bytes per lane
  const int j = lane % G;
  const int q = lane / G;
  constexpr int LPR = D / 8;            // staged loads: lanes per token row,
  constexpr int RPI = 64 / LPR;         // token rows per load instruction,
  constexpr int IPP = TPP / RPI;        // load instructions per pass
  uint32_t mw[PASSES];  // metadata word of this lane's token in each pass
  float nw[PASSES];     // its squared key norm (token retention)

#pragma unroll
  for (int p0 = 0; p0 < PASSES; p0 += 2) {
    // Two passes' loads are issued together.  Tokens past the span's end load
    // the last token instead (their results are not stored), so every load is
    // unconditional.
    u32x4 raw[2][NV];
    u32x4 whole[kStagedLoads<D> ? 2 * IPP : 1];
    if constexpr (kStagedLoads<D>) {
#pragma unroll
      for (int i = 0; i < 2 * IPP; ++i) {
        const int t = min(t_first + p0 * TPP + i * RPI + lane / LPR, n - 1);
        whole[i] = __builtin_nontemporal_load((const u32x4*)(rows + (size_t)t * D) + lane % LPR);
      }
    } else {
#pragma unroll
      for (int b = 0; b < 2; ++b) {
        const int t = min(t_first + (p0 + b) * TPP + q, n - 1);
        const u32x4* src = (const u32x4*)(rows + (size_t)t * D + j * E);
#pragma unroll
        for (int k = 0; k < NV; ++k) raw[b][k] = src[k];
      }
    }

#pragma unroll
    for (int pass = 0; pass < 2; ++pass) {
      const int t = t_first + (p0 + pass) * TPP + q;
      if constexpr (kStagedLoads<D>) {
        // LDS operations of one wavefront execute in order; the fences keep
        // the compiler from moving the accesses across each other.
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
      if constexpr (NORM) nw[p0 + pass] = quad_sqnorm<E, G>(x);
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

      uint32_t c[E];
#pragma unroll
      for (int e = 0; e < E; ++e) c[e] = code_bits(x[e], g);
      const Packed<E, BITS> pk = pack_code_bits<E, BITS>(c);
      if (t < n) store_packed<E, BITS>(codes + (size_t)t * ROW + j * PIECE, pk);
      mw[p0 + pass] = g.meta;
    }
  }
  // The wave's 32 metadata words (and squared norms) in one instruction each,
  // one whole 128-byte line: lane j of token group q writes the word of pass
  // j, token j*TPP + q.  Every lane of a group holds the group's word and
  // norm, so no exchange is needed.
  static_assert(PASSES <= G, "a lane per pass");
  if (j < PASSES) {
    uint32_t w = mw[0];
    float sq = NORM ? nw[0] : 0.0f;
#pragma unroll
    for (int i = 1; i < PASSES; ++i) {
      w = j == i ? mw[i] : w;
      if constexpr (NORM) sq = j == i ? nw[i] : sq;
    }
    const int t = t_first + j * TPP + q;
    if (t < n) {
      __builtin_nontemporal_store(w, meta + t);
      if constexpr (NORM) __builtin_nontemporal_store(sq, norm + t);
    }
  }
}

// ---------------------------------------------------------- KIVI key groups

template <int D, int BITS>
__device__ __forceinline__ void quantize_kivi_keys(const uint16_t* __restrict__ rows,
                                                   uint8_t* __restrict__ codes,
                                                   uint32_t* __restrict__ meta,
                                                   int g_first, int n, int lane) {
  constexpr int DH = D < 128 ? D : 128;      // channels per pass (head_dim 256: two passes)
  constexpr int LPR = DH / 8;                // lanes per token row (8 channels each)
  constexpr int RPL = 64 / LPR;              // token rows per load
  constexpr int NL = kWaveTokens / RPL;      // loads per lane
  constexpr int LEVELS = (1 << BITS) - 1;
  constexpr int ROW = D * BITS / 8;
  const int r = lane / LPR;                  // token row within a load

#pragma unroll
  for (int h = 0; h < D / DH; ++h) {
    const int c8 = h * LPR + lane % LPR;       // channel octet

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
    }

#pragma unroll
    for (int k = 0; k < NL; ++k) {
      const int t = g_first + r + RPL * k;
      uint32_t cq[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) cq[e] = code_bits(x[k][e], g[e]);
      const Packed<8, BITS> pk = pack_code_bits<8, BITS>(cq);
      if (t < n) store_packed<8, BITS>(codes + (size_t)t * ROW + c8 * BITS, pk);
    }
    // The group's DH metadata words in one instruction of whole lines: rows 0
    // and 1 (every row holds the reduced ranges) write the low and high four
    // words of each channel octet.
    if (r < 2) {
      uint32_t* m = meta + (size_t)(g_first / kWaveTokens) * D + 8 * c8 + 4 * r;
      const u32x4 lo = {g[0].meta, g[1].meta, g[2].meta, g[3].meta};
      const u32x4 hi = {g[4].meta, g[5].meta, g[6].meta, g[7].meta};
      __builtin_nontemporal_store(r ? hi : lo, (u32x4*)m);
    }
  }
}

// ---------------------------------------------------------------- kernel

template <int BASE, int D, int BITS, bool NORM>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(kMinWaves))) void quantize_kernel(const Params p) {
  clear_words_share(p);
  const Slice sl = decode_launch_block(p, blockIdx.x);
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int t_first = sl.tile * kBlockTokens + wave * kWaveTokens;
  if (t_first >= p.n) return;

  const uint16_t* rows = p.cache[sl.X] + ((size_t)sl.s * p.T + p.s0) * D;
  const size_t slab = (size_t)sl.slot * p.B + sl.b;  // [slot][B]

  float* norm = NORM ? p.norm + (size_t)sl.s * p.n : nullptr;  // used for K only
  if (sl.kept) {
    if (NORM && sl.X == 0)
      copy_wave_rows<D, kWaveTokens, NORM, true, true>(rows, p.side[0] + slab * p.n * D, norm, t_first, p.n, lane);
    else
      copy_wave_rows<D, kWaveTokens, false, true, true>(rows, p.side[sl.X] + slab * p.n * D, nullptr, t_first, p.n,
                                                        lane);
    return;
  }
  if (sl.X == 0 && p.kivi_whole) return;  // whole-sequence KIVI key ranges: kivi_seq.hip
  uint8_t* codes = p.codes[sl.X] + slab * p.n * (D * BITS / 8);
  if (BASE == HG_BASE_KIVI && sl.X == 0) {
    uint32_t* meta = p.meta[0] + slab * p.ngroups * D;
    quantize_kivi_keys<D, BITS>(rows, codes, meta, t_first, p.n, lane);
  } else {
    uint32_t* meta = p.meta[sl.X] + slab * p.n;
    u32x4* stage = nullptr;
    if constexpr (kStagedLoads<D>) {
      __shared__ u32x4 stage_all[kThreads / 64][(64 / kTokenLanes<D>) * (D / 8)];  // one pass of tokens
      stage = stage_all[wave];
    }
    if (BASE == HG_BASE_AKVQ && sl.X == 0)
      quantize_tokens<D, BITS, true, NORM>(rows, codes, meta, norm, t_first, p.n, lane, stage);
    else
      quantize_tokens<D, BITS, false, false>(rows, codes, meta, nullptr, t_first, p.n, lane, stage);
  }
}

// Wavefronts per SIMD of a quantize launch (each measured against 6 on the
// caches shaped like the workloads):
//  - 4 for 4-bit codes, whose stores are twice the 2-bit share of the traffic
//    (68 bytes per 256 read): 2-3 % faster everywhere (72B-shaped 996 -> 972
//    us, Qwen-shaped 138.3 -> 133.7);
//  - 4 at head_dim 256 (staged loads; its registers allow 5): Gemma-shaped
//    705 -> 694 us;
//  - 4 for the rotated AKVQ-style keys: InternVL-shaped 384 -> 381 us (3
//    bits: 395 -> 385); with the key norms of token retention, 4 measured
//    slower (399 -> 407), so those keep the rule by width;
//  - 5 for 3-bit codes: 0.5-0.7 %;
//  - else kQuantizeWaves.
// Launches whose registers already allow fewer (KIVI-style key groups at 4)
// are unaffected.
template <int BASE, int D, int BITS, bool NORM>
constexpr int kQuantizeWavesOf =
    BITS == 4 || D == 256 || (BASE == HG_BASE_AKVQ && !NORM) ? 4 : BITS == 3 ? 5 : kQuantizeWaves;

// Dynamic LDS of a quantize launch: the occupancy cap's reservation, less
// the static stage of the staged-load path.
template <int BASE, int D, int BITS, bool NORM>
constexpr size_t quantize_lds() {
  constexpr size_t stage = kStagedLoads<D> ? (kThreads / 64) * (64 / kTokenLanes<D>) * (D / 8) * 16 : 0;
  constexpr int waves = kQuantizeWavesOf<BASE, D, BITS, NORM>;
  static_assert(occupancy_lds(waves) > stage, "the stage fits the reservation");
  return occupancy_lds(waves) - stage;
}

// The workgroup tiles of a launch: kBlockTokens tokens each.
template <int BASE, int D, int BITS>
static hipError_t launch_q(const Params& p, Tensors which, bool norms, hipStream_t stream) {
  Params pq = p;
  pq.tiles = (p.n + kBlockTokens - 1) / kBlockTokens;
  const uint64_t per_tensor = (uint64_t)p.L * p.B * p.H * (uint64_t)pq.tiles;
  const bool kept = which == Tensors::kKeptKeysAndValues;
  const uint64_t blocks_k = which == Tensors::kValues ? 0
                            : kept ? (uint64_t)(p.L * p.H - p.n_unprot_k) * p.B * pq.tiles : per_tensor;
  const uint64_t blocks = which == Tensors::kKeys ? per_tensor : blocks_k + per_tensor;
  if (blocks > 0x7FFFFFFFull) return hipErrorInvalidConfiguration;
  pq.blocks_k = (uint32_t)blocks_k;
  pq.kept_keys = kept;
  if constexpr (BASE == HG_BASE_AKVQ) {
    if (norms) {
      constexpr size_t kLdsNorm = quantize_lds<BASE, D, BITS, true>();
      hipLaunchKernelGGL((quantize_kernel<BASE, D, BITS, true>), dim3((uint32_t)blocks), dim3(kThreads),
                         kLdsNorm, stream, pq);
      return hipGetLastError();
    }
  }
  if (norms) return hipErrorInvalidValue;  // key norms belong to the AKVQ base
  constexpr size_t kLds = quantize_lds<BASE, D, BITS, false>();
  hipLaunchKernelGGL((quantize_kernel<BASE, D, BITS, false>), dim3((uint32_t)blocks), dim3(kThreads),
                     kLds, stream, pq);
  return hipGetLastError();
}

template <int BASE, int D>
static hipError_t launch_q_bits(const Params& p, int bits, Tensors which, bool norms, hipStream_t stream) {
  switch (bits) {
    case 2: return launch_q<BASE, D, 2>(p, which, norms, stream);
    case 3: return launch_q<BASE, D, 3>(p, which, norms, stream);
    case 4: return launch_q<BASE, D, 4>(p, which, norms, stream);
    default: return hipErrorInvalidValue;
  }
}

template <int BASE>
static hipError_t launch_q_dim(const Params& p, int D, int bits, Tensors which, bool norms, hipStream_t stream) {
  switch (D) {
    case 64: return launch_q_bits<BASE, 64>(p, bits, which, norms, stream);
    case 128: return launch_q_bits<BASE, 128>(p, bits, which, norms, stream);
    case 256: return launch_q_bits<BASE, 256>(p, bits, which, norms, stream);
    default: return hipErrorInvalidValue;
  }
}

// The KIVI-style and AKVQ-style bases quantize values exactly as min-max
// does (per token, unrotated), so their value tiles run as a launch of the
// min-max instantiation: a kernel holds the registers of its largest path,
// and the key paths (KIVI groups, rotation) need more than the per-token
// path, which would leave the value tiles with fewer waves per SIMD.  With
// KIVI keys over the whole sequence this launch only copies protected keys
// and quantizes values, so all of it runs as the min-max instantiation, its
// key blocks listing the protected key slices alone (with every key slice
// listed, the 7/8 that exit at once cost 36 us on the LLaVA-NeXT-shaped
// cache).
hipError_t launch_quantize(const Params& p, int base, int D, int bits, bool norms, hipStream_t stream) {
  if (base == HG_BASE_KIVI && p.kivi_whole)
    return launch_q_dim<HG_BASE_MINMAX>(p, D, bits, Tensors::kKeptKeysAndValues, norms, stream);
  if (base == HG_BASE_MINMAX) return launch_q_dim<HG_BASE_MINMAX>(p, D, bits, Tensors::kBoth, norms, stream);
  if (base != HG_BASE_KIVI && base != HG_BASE_AKVQ) return hipErrorInvalidValue;
  hipError_t e = base == HG_BASE_KIVI ? launch_q_dim<HG_BASE_KIVI>(p, D, bits, Tensors::kKeys, norms, stream)
                                      : launch_q_dim<HG_BASE_AKVQ>(p, D, bits, Tensors::kKeys, norms, stream);
  if (e != hipSuccess) return e;
  return launch_q_dim<HG_BASE_MINMAX>(p, D, bits, Tensors::kValues, false, stream);
}

}  // namespace hg
