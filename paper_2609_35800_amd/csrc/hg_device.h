// Device helpers for the gfx950 quantizer kernels: BF16 conversions with
// directed rounding, quad-level DPP exchanges, the per-group scale rule, the
// in-register/quad Walsh-Hadamard transform and LSB-first bit packing.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace hg {

// Native clang vectors: nontemporal builtins and wide loads/stores need them.
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
// 12-byte pieces sit at 4-byte aligned offsets: declare that alignment.
typedef uint32_t u32x3 __attribute__((ext_vector_type(3), aligned(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// ------------------------------------------------------------------ BF16

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }
__device__ __forceinline__ float bf16_as_float(uint32_t h) { return __uint_as_float(h << 16); }

// Round toward -inf / +inf to a BF16 bit pattern (finite inputs).  Truncating
// the low half rounds toward zero; a value with a nonzero low half on the far
// side of zero then moves one BF16 unit away from zero.
__device__ __forceinline__ uint32_t bf16_round_down(float x) {
  uint32_t u = __float_as_uint(x);
  uint32_t step = ((u & 0xFFFFu) != 0u) & (u >> 31);
  return (u >> 16) + step;
}
__device__ __forceinline__ uint32_t bf16_round_up(float x) {
  uint32_t u = __float_as_uint(x);
  uint32_t step = ((u & 0xFFFFu) != 0u) & ((u >> 31) ^ 1u);
  return (u >> 16) + step;
}
// Round to nearest, ties to even: adding 0x7FFF plus the kept LSB carries into
// the kept half exactly when the dropped half is above one half, or equal to
// one half with an odd kept half.
__device__ __forceinline__ uint32_t bf16_round_nearest(float x) {
  uint32_t u = __float_as_uint(x);
  return (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;
}
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  return bf16_round_nearest(lo) | (bf16_round_nearest(hi) << 16);
}

// ------------------------------------------------------- quad DPP exchange

// quad_perm controls: lane i of each group of four reads lane i^1 / i^2.
constexpr int kQuadXor1 = 0xB1;  // [1,0,3,2]
constexpr int kQuadXor2 = 0x4E;  // [2,3,0,1]

template <int CTRL>
__device__ __forceinline__ float quad_swap(float v) {
  return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), CTRL, 0xF, 0xF, false));
}

__device__ __forceinline__ float quad_min(float v) {
  v = fminf(v, quad_swap<kQuadXor1>(v));
  return fminf(v, quad_swap<kQuadXor2>(v));
}
__device__ __forceinline__ float quad_max(float v) {
  v = fmaxf(v, quad_swap<kQuadXor1>(v));
  return fmaxf(v, quad_swap<kQuadXor2>(v));
}

// Row-level exchanges for a token held by a row of R = D/8 lanes (8 channels
// per lane): partner lane = lane ^ m for m = 1, 2, 4, 8, all within one
// 16-lane DPP row.  xor 4 composes quad reverse (lane ^ 3) with the
// half-row mirror (lane ^ 7); xor 8 is a rotation of the row by 8.  xor 16
// (head_dim 256) crosses DPP rows and goes through the LDS crossbar.
constexpr int kQuadRev = 0x1B;       // quad_perm [3,2,1,0]
constexpr int kRowHalfMirror = 0x141;
constexpr int kRowRor8 = 0x128;

template <int M>
__device__ __forceinline__ float row_xor(float v) {
  if constexpr (M == 1) return quad_swap<kQuadXor1>(v);
  else if constexpr (M == 2) return quad_swap<kQuadXor2>(v);
  else if constexpr (M == 4) return quad_swap<kRowHalfMirror>(quad_swap<kQuadRev>(v));
  else if constexpr (M == 8) return quad_swap<kRowRor8>(v);
  else {
    static_assert(M == 16, "row exchange");
    return __shfl_xor(v, 16);
  }
}

// Minimum / maximum over the G = 4 or 8 lanes holding one token.
template <int G>
__device__ __forceinline__ float group_min(float v) {
  v = quad_min(v);
  if constexpr (G == 8) v = fminf(v, row_xor<4>(v));
  return v;
}
template <int G>
__device__ __forceinline__ float group_max(float v) {
  v = quad_max(v);
  if constexpr (G == 8) v = fmaxf(v, row_xor<4>(v));
  return v;
}

// Lanes per token in the per-token compute layout: a quad up to head_dim 128
// (D/4 elements per lane), eight lanes at 256 (32 per lane), so a lane never
// holds more than 32 elements.
template <int D>
constexpr int kTokenLanes = D == 256 ? 8 : 4;

// --------------------------------------------------------- group scale rule

// fp32 RN(1/L) for L = 2^b - 1.
template <int LEVELS>
__device__ __forceinline__ constexpr float inv_levels() {
  static_assert(LEVELS == 3 || LEVELS == 7 || LEVELS == 15, "bits");
  return LEVELS == 3 ? 0x1.555556p-2f : LEVELS == 7 ? 0x1.24924ap-3f : 0x1.111112p-4f;
}

// Correctly rounded d / L for finite d >= 0: the product with RN(1/L) is off by
// at most one unit, and one fma residual step corrects it.  Equal to the IEEE
// quotient for every non-negative finite fp32 d at L = 3, 7 and 15 (checked
// exhaustively); three operations instead of a full division sequence.
template <int LEVELS>
__device__ __forceinline__ float div_levels(float d) {
  const float y = inv_levels<LEVELS>();
  const float q0 = d * y;
  const float r = __builtin_fmaf(-q0, (float)LEVELS, d);
  return __builtin_fmaf(r, y, q0);
}

// Correctly rounded 1/S for a BF16 scale S in [2^-126, 2^101]: the hardware
// reciprocal (within one unit) refined by one fma Newton step.  Equal to the
// IEEE quotient 1/S for every such S (checked exhaustively over all BF16
// values in the range).
__device__ __forceinline__ float rcp_scale(float S) {
  const float r0 = __builtin_amdgcn_rcpf(S);
  const float e = __builtin_fmaf(-S, r0, 1.0f);
  return __builtin_fmaf(r0, e, r0);
}

// Metadata of a group with range [mn, mx] at LEVELS = 2^b - 1:
// m = BF16 round-down of mn, S = BF16 round-up of (mx - m)/LEVELS, zeros
// stored as +0, a positive S raised to at least 2^-126 (BF16 0x0080) so that
// 1/S stays finite.  `inv` is the correctly rounded 1/S, or 0 when S == 0.
struct GroupScale {
  float m, inv;
  uint32_t meta;
};

template <int LEVELS>
__device__ __forceinline__ GroupScale group_scale(float mn, float mx) {
  uint32_t m16 = bf16_round_down(mn);
  m16 = (m16 == 0x8000u) ? 0u : m16;
  const float m = bf16_as_float(m16);
  const float s = div_levels<LEVELS>(mx - m);
  uint32_t s16 = bf16_round_up(s);
  s16 = (s16 == 0x8000u) ? 0u : s16;
  s16 = (s16 != 0u && s16 < 0x0080u) ? 0x0080u : s16;
  const float S = bf16_as_float(s16);
  const float inv = rcp_scale(s16 ? S : 1.0f);  // correctly rounded 1/S
  GroupScale g;
  g.m = m;
  g.inv = s16 ? inv : 0.0f;
  g.meta = s16 | (m16 << 16);
  return g;
}

// Code of one element, returned as the bit pattern of fl(t + 1.5*2^23) with
// t = (v - m) * inv (two roundings, no contraction): for 0 <= t < 2^22 that
// sum holds rint(t), ties to even, in its low bits above 0x4B400000.  Because
// m <= v <= max, 1/S and (max - m)/L are correctly rounded and S >= that
// quotient, 0 <= t <= L*(1 + 3*2^-24) < L + 1/2: rint(t) already lies in
// [0, L], so the clamp of the definition never changes it.
constexpr uint32_t kMagicBits = 0x4B400000u;

__device__ __forceinline__ uint32_t code_bits(float v, const GroupScale& g) {
  const float t = (v - g.m) * g.inv;
  return __float_as_uint(t + 0x1.8p23f);
}

// The scaled value of one element, t = (v - m) * inv (two roundings, no
// contraction), whose rint is its code (see code_bits: 0 <= t < L + 1/2).
// The one-pass reconstruction takes rint(t) directly (v_rndne_f32).
__device__ __forceinline__ float code_scaled(float v, const GroupScale& g) { return (v - g.m) * g.inv; }

// ------------------------------------------------- Walsh-Hadamard transform

// fp32(1/sqrt(D)) for the supported power-of-two head dims: 1/8 and 1/16
// exactly, and 1/sqrt(128) = 0.08838834764... rounded to nearest fp32.
template <int D>
__device__ __forceinline__ constexpr float fwht_scale() {
  static_assert(D == 64 || D == 128 || D == 256, "head_dim");
  return D == 64 ? 0.125f : D == 128 ? 0x1.6a09e6p-4f : 0.0625f;
}

// Butterflies of spans 1 .. E/2 inside one lane's E contiguous elements.
template <int E>
__device__ __forceinline__ void fwht_lane(float (&x)[E]) {
#pragma unroll
  for (int h = 1; h < E; h *= 2) {
#pragma unroll
    for (int i = 0; i < E; i += 2 * h) {
#pragma unroll
      for (int k = i; k < i + h; ++k) {
        float p = x[k], q = x[k + h];
        x[k] = p + q;
        x[k + h] = p - q;
      }
    }
  }
}

// Cross-lane butterfly stages carry a per-lane sign so that each stage is one
// fma with a DPP operand.  Pairs are (lane, lane ^ M); the lower lane must
// end with p + q and the upper with p - q (p the lower's value).  Each lane
// computes v' = fma(partner, s, v) with s = +1 in the lower and -1 in the
// upper lane: the lower gets p + q, the upper q - p = -(p - q).  The upper
// lane thus holds its value negated; as stages use distinct lane bits, a lane
// ends holding (-1)^popcount(lane & stage bits) times its value, and the final
// multiply by c uses c with that sign.  Negation is exact and round to nearest
// is symmetric, so every nonzero value equals the plain butterfly's bit for
// bit.  An exact-zero difference is +0 in either operand order, so a carried
// lane can end with -0 where the plain transform has +0; the final scale is
// therefore fma(v, c*sign, +0), which turns -0 into +0 and leaves every other
// product as the plain multiply rounds it.  The plain transform never yields
// -0 from inputs without -0 (dequantized levels q*S + m are never -0); in the
// quantizer the sign of a zero changes neither the range (its min is stored
// as +0 when zero) nor any code.
template <int CTRL>
__device__ __forceinline__ float butterfly_fma(float v, float s) {
  return __builtin_fmaf(quad_swap<CTRL>(v), s, v);
}

// Eight butterflies of one stage, each a single v_fmac_f32 whose first source
// is read through the DPP swizzle PERM: x = dpp(x) * s + x, one rounding, as
// butterfly_fma (the compiler keeps a separate DPP move otherwise).  A DPP
// read of a register needs two wait states after the VALU write of it, so the
// block starts and ends with s_nop 1; inside, each instruction reads only its
// own register, written before the block.
#define HG_BUTTERFLY8(PERM, x, s)                                                              \
  asm("s_nop 1\n"                                                                              \
      "v_fmac_f32_dpp %0, %0, %8 " PERM " row_mask:0xf bank_mask:0xf\n"                         \
      "v_fmac_f32_dpp %1, %1, %8 " PERM " row_mask:0xf bank_mask:0xf\n"                         \
      "v_fmac_f32_dpp %2, %2, %8 " PERM " row_mask:0xf bank_mask:0xf\n"                         \
      "v_fmac_f32_dpp %3, %3, %8 " PERM " row_mask:0xf bank_mask:0xf\n"                         \
      "v_fmac_f32_dpp %4, %4, %8 " PERM " row_mask:0xf bank_mask:0xf\n"                         \
      "v_fmac_f32_dpp %5, %5, %8 " PERM " row_mask:0xf bank_mask:0xf\n"                         \
      "v_fmac_f32_dpp %6, %6, %8 " PERM " row_mask:0xf bank_mask:0xf\n"                         \
      "v_fmac_f32_dpp %7, %7, %8 " PERM " row_mask:0xf bank_mask:0xf\n"                         \
      "s_nop 1"                                                                                \
      : "+v"((x)[0]), "+v"((x)[1]), "+v"((x)[2]), "+v"((x)[3]), "+v"((x)[4]), "+v"((x)[5]),    \
        "+v"((x)[6]), "+v"((x)[7])                                                             \
      : "v"(s))

// Full transform over D = G*E elements held by G = 4 or 8 consecutive lanes
// (lane j of the group holds elements [E*j, E*j + E)): spans 1..E/2 in
// registers, then E (lane ^ 1), 2E (lane ^ 2) and, for G = 8, 4E (lane ^ 4),
// then the scale c.  Same butterfly order as spans 1..D/2.
template <int E, int G = 4>
__device__ __forceinline__ void fwht_quad(float (&x)[E], int j, float c) {
  static_assert(E % 8 == 0 && (G == 4 || G == 8), "whole blocks of eight; quad or octet");
  fwht_lane<E>(x);
  const float s1 = (j & 1) ? -1.0f : 1.0f;
  const float s2 = (j & 2) ? -1.0f : 1.0f;
#pragma unroll
  for (int e = 0; e < E; e += 8) HG_BUTTERFLY8("quad_perm:[1,0,3,2]", x + e, s1);
#pragma unroll
  for (int e = 0; e < E; e += 8) HG_BUTTERFLY8("quad_perm:[2,3,0,1]", x + e, s2);
  float cs = c * s1 * s2;  // c with the carried sign, exact
  if constexpr (G == 8) {
    const float s4 = (j & 4) ? -1.0f : 1.0f;
#pragma unroll
    for (int e = 0; e < E; ++e) x[e] = __builtin_fmaf(row_xor<4>(x[e]), s4, x[e]);
    cs = cs * s4;
  }
#pragma unroll
  for (int e = 0; e < E; ++e) x[e] = __builtin_fmaf(x[e], cs, 0.0f);
}

// Full transform over D = 8R elements held by a row of R lanes (lane c holds
// elements [8c, 8c + 8)): spans 1, 2, 4 in registers, then 8, 16, ... by
// exchanges with lanes c ^ 1, c ^ 2, ..., each a sign-carrying fma stage (see
// fwht_quad), then the scale.  Same butterfly order as spans 1..D/2.
template <int M>
__device__ __forceinline__ void fwht_row_stage(float (&x)[8], float s) {
#pragma unroll
  for (int e = 0; e < 8; ++e) x[e] = __builtin_fmaf(row_xor<M>(x[e]), s, x[e]);
}

template <int D>
__device__ __forceinline__ void fwht_row(float (&x)[8], int c) {
  static_assert(D == 64 || D == 128 || D == 256, "head_dim");
  fwht_lane<8>(x);
  const float s1 = (c & 1) ? -1.0f : 1.0f, s2 = (c & 2) ? -1.0f : 1.0f;
  const float s4 = (c & 4) ? -1.0f : 1.0f;
  fwht_row_stage<1>(x, s1);
  fwht_row_stage<2>(x, s2);
  fwht_row_stage<4>(x, s4);
  float cs = fwht_scale<D>() * s1 * s2 * s4;
  if constexpr (D >= 128) {
    const float s8 = (c & 8) ? -1.0f : 1.0f;
    fwht_row_stage<8>(x, s8);
    cs = cs * s8;
  }
  if constexpr (D == 256) {
    const float s16 = (c & 16) ? -1.0f : 1.0f;
    fwht_row_stage<16>(x, s16);
    cs = cs * s16;
  }
#pragma unroll
  for (int e = 0; e < 8; ++e) x[e] = __builtin_fmaf(x[e], cs, 0.0f);
}

// ------------------------------------------------------ squared key norms

// Squared L2 norm in fp32 as a balanced tree over channel index: the squares,
// then sums of adjacent pairs, of adjacent pairs of those, and so on.  A lane
// reduces its own aligned block of N channels in registers; lanes holding
// adjacent blocks then combine through exchanges with lane ^ 1, lane ^ 2, ...,
// so every node is the sum of the same two halves as in the plain tree.  IEEE
// addition commutes, so both partners of an exchange hold the same sum.
template <int N>
__device__ __forceinline__ float tree_sqnorm(const float (&x)[N]) {
  float a[N];
#pragma unroll
  for (int e = 0; e < N; ++e) a[e] = x[e] * x[e];
#pragma unroll
  for (int w = N / 2; w >= 1; w /= 2) {
#pragma unroll
    for (int i = 0; i < w; ++i) a[i] = a[2 * i] + a[2 * i + 1];
  }
  return a[0];
}

// A token held by G = 4 or 8 lanes, lane j holding channels [j*E, (j+1)*E).
template <int E, int G = 4>
__device__ __forceinline__ float quad_sqnorm(const float (&x)[E]) {
  float s = tree_sqnorm<E>(x);
  s = s + quad_swap<kQuadXor1>(s);
  s = s + quad_swap<kQuadXor2>(s);
  if constexpr (G == 8) s = s + row_xor<4>(s);
  return s;
}

// A token held by a row of D/8 lanes, lane c holding channels [8c, 8c + 8)
// as one 16-byte vector of BF16.
template <int D>
__device__ __forceinline__ float row_sqnorm(u32x4 v) {
  const float x[8] = {bf16_lo(v.x), bf16_hi(v.x), bf16_lo(v.y), bf16_hi(v.y),
                      bf16_lo(v.z), bf16_hi(v.z), bf16_lo(v.w), bf16_hi(v.w)};
  float s = tree_sqnorm<8>(x);
  s = s + row_xor<1>(s);
  s = s + row_xor<2>(s);
  s = s + row_xor<4>(s);
  if constexpr (D >= 128) s = s + row_xor<8>(s);
  if constexpr (D == 256) s = s + row_xor<16>(s);
  return s;
}

// BF16 round-to-nearest-even of two fp32 values, packed low/high, by the
// hardware conversion (v_cvt_pk_bf16_f32).
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t pack_bf16x2_hw(float lo, float hi) {
  f32x2_t v = {lo, hi};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2_t));
}

// ------------------------------------------------------------ bit packing

// The packed bits of N codes of BITS bits each, LSB-first, in W = ceil(N*BITS/32) words.
template <int N, int BITS>
struct Packed {
  static constexpr int kBits = N * BITS;
  static constexpr int W = (kBits + 31) / 32;
  uint32_t w[W];
};

// Sum of the magic offsets (kMagicBits << s) that the whole-word codes of each
// word carry, modulo 2^32.
template <int N, int BITS>
struct MagicBias {
  uint32_t w[(N * BITS + 31) / 32];
  constexpr MagicBias() : w() {
    for (int e = 0; e < N; ++e) {
      const int pos = e * BITS;
      if ((pos % 32) + BITS <= 32) w[pos / 32] += kMagicBits << (pos % 32);
    }
  }
};

// Packs N codes given as magic bit patterns (kMagicBits + q).  Codes occupy
// disjoint bits, so packing by addition equals packing by OR; each word starts
// at minus the magic offsets it will receive, leaving one shift-add per code.
// A code that straddles two words is reduced to q first.
template <int N, int BITS>
__device__ __forceinline__ Packed<N, BITS> pack_code_bits(const uint32_t (&cb)[N]) {
  constexpr MagicBias<N, BITS> kBias{};
  Packed<N, BITS> p;
#pragma unroll
  for (int i = 0; i < Packed<N, BITS>::W; ++i) p.w[i] = 0u - kBias.w[i];
#pragma unroll
  for (int e = 0; e < N; ++e) {
    const int pos = e * BITS;
    const int sh = pos % 32;
    if (sh + BITS <= 32) {
      p.w[pos / 32] += cb[e] << sh;
    } else {
      const uint32_t q = cb[e] - kMagicBits;
      p.w[pos / 32] += q << sh;
      p.w[pos / 32 + 1] += q >> (32 - sh);
    }
  }
  return p;
}

// Store of a lane's packed piece at a byte address whose alignment is
// that of the piece: whole dwords for 32/64/96/128-bit pieces, 16-bit halves
// for 48-bit pieces.
template <int N, int BITS>
__device__ __forceinline__ void store_packed(uint8_t* dst, const Packed<N, BITS>& p) {
  constexpr int kBits = N * BITS;
  if constexpr (kBits == 16) {
    __builtin_nontemporal_store((uint16_t)p.w[0], (uint16_t*)dst);
  } else if constexpr (kBits == 24) {
    dst[0] = (uint8_t)p.w[0];
    dst[1] = (uint8_t)(p.w[0] >> 8);
    dst[2] = (uint8_t)(p.w[0] >> 16);
  } else if constexpr (kBits == 32) {
    __builtin_nontemporal_store(p.w[0], (uint32_t*)dst);
  } else if constexpr (kBits == 48) {
    uint16_t* d = (uint16_t*)dst;
    __builtin_nontemporal_store((uint16_t)p.w[0], d);
    __builtin_nontemporal_store((uint16_t)(p.w[0] >> 16), d + 1);
    __builtin_nontemporal_store((uint16_t)p.w[1], d + 2);
  } else if constexpr (kBits == 64) {
    u32x2 v = {p.w[0], p.w[1]};
    __builtin_nontemporal_store(v, (u32x2*)dst);
  } else if constexpr (kBits == 96) {
    u32x3 v = {p.w[0], p.w[1], p.w[2]};
    __builtin_nontemporal_store(v, (u32x3*)dst);
  } else {
    static_assert(kBits == 128, "unsupported packed piece");
    u32x4 v = {p.w[0], p.w[1], p.w[2], p.w[3]};
    __builtin_nontemporal_store(v, (u32x4*)dst);
  }
}

// The 8 codes of channels [8c, 8c + 8) of a packed token row: BITS bytes at
// byte offset BITS*c.  Three-byte pieces are read as the two aligned dwords
// around them (the second clamped to the row) and funnel-shifted.
template <int BITS, int ROW>
__device__ __forceinline__ uint32_t load_piece8(const uint8_t* row, int c) {
  if constexpr (BITS == 2) {
    return *(const uint16_t*)(row + 2 * c);
  } else if constexpr (BITS == 4) {
    return *(const uint32_t*)(row + 4 * c);
  } else {
    static_assert(BITS == 3 && ROW % 4 == 0, "piece");
    const int o = 3 * c;
    const uint32_t* w = (const uint32_t*)row;
    const uint32_t lo = w[o >> 2];
    const uint32_t hi = w[min((o >> 2) + 1, ROW / 4 - 1)];
    return __builtin_amdgcn_alignbyte(hi, lo, (uint32_t)(o & 3)) & 0xFFFFFFu;
  }
}

// Slot of 16-byte chunk c of token t in a wavefront's LDS stage of D/8
// chunks per token, XOR-swizzled so that the row layout (a token row across
// D/8 lanes) and the quad layout (a token across 4 or 8 lanes, 4 chunks per
// lane) both read and write it without bank conflicts.  Measured on gfx950
// with 16-byte accesses: a write conflicts when two of 8 consecutive lanes
// hit equal slots modulo 8, a read when two of 16 consecutive lanes hit
// equal slots modulo 16; the XOR terms below keep both apart for each head
// dim (quad-layout writes took 8 (head_dim 128) and 24 (256) extra cycles
// per instruction with a plain token XOR).
template <int D>
__device__ __forceinline__ constexpr int stage_slot(int t, int c) {
  if constexpr (D == 64) return t * 8 + (c ^ ((t & 1) + ((t >> 1) & 1)));
  else if constexpr (D == 128) return t * 16 + (c ^ ((((c >> 3) << 1) | (t & 1)) ^ (((t >> 1) & 1) << 1)));
  else return t * 32 + (c ^ ((c >> 3) | ((t & 1) << 3)));
}

__device__ __forceinline__ void store_nt(u32x4* dst, u32x4 v) {
  __builtin_nontemporal_store(v, dst);
}

// Bit-exact copy of a wavefront's token rows [t_first, t_first + TOKENS),
// clipped to n, from src to dst (rows of D BF16 at the same offsets): 16-byte
// vectors, vector i of the tile on lane i % 64, all loads issued before the
// streaming stores; with NT_LOADS the loads stream too (the rows are read
// once: the input cache; dequantize's side-store reads measured faster plain).  With NORM, every row's squared norm (row tree,
// row_sqnorm) also goes to norm[t], by a streaming store if NORM_NT.
// (Copying a head_dim-256 tile in two rounds of 8 vectors per lane lowers the
// kernels' register counts from 88-90 to 64-70, but measured no faster for
// quantize and 2 % slower for dequantize at the higher occupancy.)
template <int D, int TOKENS, bool NORM = false, bool NORM_NT = true, bool NT_LOADS = false>
__device__ __forceinline__ void copy_wave_rows(const uint16_t* __restrict__ src, uint16_t* __restrict__ dst,
                                               float* __restrict__ norm, int t_first, int n, int lane) {
  constexpr int VPT = D / 8;                // 16-byte vectors per row
  constexpr int kVec = TOKENS * VPT / 64;   // vectors per lane
  const int nvec = min(TOKENS, n - t_first) * VPT;
  const u32x4* s = (const u32x4*)(src + (size_t)t_first * D);
  u32x4* d = (u32x4*)(dst + (size_t)t_first * D);
  u32x4 v[kVec];
#pragma unroll
  for (int k = 0; k < kVec; ++k) {
    const u32x4* a = s + min(lane + 64 * k, nvec - 1);
    v[k] = NT_LOADS ? __builtin_nontemporal_load(a) : *a;
  }
#pragma unroll
  for (int k = 0; k < kVec; ++k) {
    const int i = lane + 64 * k;
    if (i < nvec) store_nt(d + i, v[k]);
  }
  if constexpr (NORM) {
    // vector i holds channels [8c, 8c + 8) of row i / VPT, c = i % VPT
#pragma unroll
    for (int k = 0; k < kVec; ++k) {
      const float sq = row_sqnorm<D>(v[k]);
      const int i = lane + 64 * k;
      if (i < nvec && i % VPT == 0) {
        if constexpr (NORM_NT)
          __builtin_nontemporal_store(sq, norm + t_first + i / VPT);
        else
          norm[t_first + i / VPT] = sq;
      }
    }
  }
}

}  // namespace hg
