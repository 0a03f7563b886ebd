// KIVI-style keys with one range per channel over the whole supplied
// sequence, text included (HeadGuard §4, Quantization setup: the KIVI-style
// base recomputes key ranges over the supplied sequence, including text,
// while text KV stays BF16).  Selected by kivi_group = 0.
//
// Every code depends on the range of its channel over all T rows of the
// slice, so a slice must be fully read before any of its codes is formed.
// Three forms:
//
// Partitioned resident kernel (T at most 32 workgroups' capacity): a
// persistent grid of 1024-thread workgroups, one per compute unit.  A group of
// P workgroups (past 8, rounded up to 16 or 32, so that the groups fill every
// compute unit) takes one key slice (l, b, h) at a time; workgroup q of the
// group holds rows [q R, (q + 1) R) of the slice, every channel, on chip (9
// row slots in LDS filled by buffer loads that write LDS directly, 15 in
// registers), so each slice is read from HBM exactly once:
//  1. per-channel min / max over the workgroup's rows, reduced across the
//     rows a wavefront holds by shuffles and across wavefronts by LDS
//     atomics;
//  2. with P > 1, the group's partial ranges are combined through a caller
//     workspace: each workgroup publishes its range of each channel as one
//     64-bit word, the BF16 minimum and maximum tagged with the slice's
//     sequence number in the group (relaxed device-scope atomics; a tagged
//     word carries its own values, so no fence is needed); every thread
//     polls some partners' words of one channel (1024 / D threads per
//     channel share the partners), a bounded number of times, until they
//     carry that tag, and folds them into the workgroup's range in LDS; two
//     buffers alternate between consecutive slices,
//     and the words start at zero (cleared by the call's first kernel, the
//     values' quantize or one-pass launch, or else by a kernel of their own);
//  3. codes (or, for the one-pass simulated quantization, the BF16
//     reconstruction) of the workgroup's image rows: whole packed rows, so
//     every stored line is complete; as the row slots are consumed, the
//     loads of the workgroup's rows of the next slice are issued into them.
// The grid never exceeds the number of workgroups the device holds at once,
// so every partner of a group is resident; a wait that runs out of polls
// (only if another kernel held the device's resources) ends anyway and is
// counted in the workspace's first word.  (Two 512-thread workgroups per
// compute unit, each holding half as many rows, measured 1 % slower.)
//
// Split kernels (longer slices, or too few compute units for a group of
// eight): a range launch over chunks of every slice, whose per-channel ranges
// are merged into the workspace by atomic maxima, then a code launch over
// chunks of the image rows; each slice is read twice, but every compute unit
// works on it.
//
// Two-pass kernel (a slice one workgroup holds, with no workspace, on a
// device of fewer than 8 compute units): a persistent grid of
// kSeqBlocksPerCU workgroups of kSeqThreads threads per compute unit walks
// the key slices; per slice a range pass over all T rows, the wavefronts'
// partial ranges combined through LDS, then a second pass over the image rows
// for the codes.
//
// Values, protected slices and the rest of the cache are handled by the
// regular kernels of the same call.

#include <stdlib.h>

#include <algorithm>

#include "hg_device.h"
#include "hg_kernels.h"

namespace hg {

constexpr int kSeqThreads = 1024;
constexpr int kSeqBlocksPerCU = 2;
constexpr int kSeqUnroll1 = 4;  // rows in flight per lane, range pass
constexpr int kSeqUnroll2 = 4;  // rows in flight per lane, code pass

// Per-channel range, over rows [t_begin, t_end) of a slice, of the 8
// channels this lane loads (lane i: channels 8 (i % (D/8)) on, row i / (D/8)
// of each WAVES * 64 / (D/8) rows), reduced over the wavefront's rows by
// shuffles; rows past the end re-read the last row, which leaves the range
// unchanged.  t_end > t_begin.  Streaming loads, here and in code_rows (9 %
// and 3 % faster launches than cached loads).
template <int D, int WAVES, int U = kSeqUnroll1>
__device__ __forceinline__ void range_rows(const uint16_t* __restrict__ slice, int t_begin, int t_end, float (&mn)[8],
                                           float (&mx)[8]) {
  constexpr int CPT = D / 8;
  constexpr int RPL = 64 / CPT;
  constexpr int STEP = WAVES * RPL;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int c8 = lane % CPT;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    mn[e] = __builtin_inff();
    mx[e] = -__builtin_inff();
  }
  for (int t0 = t_begin + wave * RPL + lane / CPT; t0 < t_end; t0 += U * STEP) {
    u32x4 v[U];
#pragma unroll
    for (int u = 0; u < U; ++u)
      v[u] = __builtin_nontemporal_load((const u32x4*)(slice + (size_t)min(t0 + u * STEP, t_end - 1) * D + 8 * c8));
#pragma unroll
    for (int u = 0; u < U; ++u) {
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
}

// Codes (or, FAKE, the BF16 reconstruction) of image rows [t_begin, t_end)
// of a slice (`rows`: its first image row; `codes` / `out`: the slice's
// packed rows / reconstructed image rows), this lane's 8 channels with
// scales g (S: the scales as floats).  t_end > t_begin.
template <int D, int BITS, bool FAKE, int WAVES, int U = kSeqUnroll2>
__device__ __forceinline__ void code_rows(const uint16_t* __restrict__ rows, uint8_t* codes, uint16_t* out,
                                          int t_begin, int t_end, const GroupScale (&g)[8], const float (&S)[8]) {
  constexpr int CPT = D / 8;
  constexpr int RPL = 64 / CPT;
  constexpr int STEP = WAVES * RPL;
  constexpr int ROW = D * BITS / 8;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int c8 = lane % CPT;
  for (int t0 = t_begin + wave * RPL + lane / CPT; t0 < t_end; t0 += U * STEP) {
    u32x4 v[U];
#pragma unroll
    for (int u = 0; u < U; ++u)
      v[u] = __builtin_nontemporal_load((const u32x4*)(rows + (size_t)min(t0 + u * STEP, t_end - 1) * D + 8 * c8));
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int t = t0 + u * STEP;
      const float x[8] = {bf16_lo(v[u].x), bf16_hi(v[u].x), bf16_lo(v[u].y), bf16_hi(v[u].y),
                          bf16_lo(v[u].z), bf16_hi(v[u].z), bf16_lo(v[u].w), bf16_hi(v[u].w)};
      if constexpr (FAKE) {
        float y[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) y[e] = __builtin_fmaf(__builtin_rintf(code_scaled(x[e], g[e])), S[e], g[e].m);
        const u32x4 o = {pack_bf16x2_hw(y[0], y[1]), pack_bf16x2_hw(y[2], y[3]), pack_bf16x2_hw(y[4], y[5]),
                         pack_bf16x2_hw(y[6], y[7])};
        if (t < t_end) store_nt((u32x4*)(out + (size_t)t * D + 8 * c8), o);
      } else {
        uint32_t cq[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) cq[e] = code_bits(x[e], g[e]);
        const Packed<8, BITS> pk = pack_code_bits<8, BITS>(cq);
        if (t < t_end) store_packed<8, BITS>(codes + (size_t)t * ROW + c8 * BITS, pk);
      }
    }
  }
}

template <int D, int BITS, bool FAKE, int WAVES>
__device__ __forceinline__ void kivi_seq_slice(const Params& p, uint32_t s, const SliceRoute& route,
                                               float (&part)[2][WAVES][D]) {
  constexpr int CPT = D / 8;
  constexpr int LEVELS = (1 << BITS) - 1;
  constexpr int ROW = D * BITS / 8;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int c8 = lane % CPT;
  const int r = lane / CPT;
  const uint16_t* slice = p.cache[0] + (size_t)s * p.T * D;

  // 1. ranges over all T rows
  float mn[8], mx[8];
  range_rows<D, WAVES>(slice, 0, p.T, mn, mx);

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
  if (p.n > 0)
    code_rows<D, BITS, FAKE, WAVES>(slice + (size_t)p.s0 * D, FAKE ? nullptr : p.codes[0] + slab * p.n * ROW,
                                    FAKE ? p.out[0] + (size_t)s * p.T * D + (size_t)p.s0 * D : nullptr, 0, p.n, g, S);
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

// ------------------------------------------------- partitioned resident kernel

constexpr int kPartThreads = 1024;
constexpr int kPartWaves = kPartThreads / 64;
constexpr int kPartLdsSlots = 9;
constexpr int kPartRegSlots = 15;
constexpr int kPartSlots = kPartLdsSlots + kPartRegSlots;
constexpr int kMaxPartners = 32;    // a group's partners share one XCD's 32 compute units
constexpr int kSerialPartners = 8;  // up to this many, one thread per channel polls every partner
// Exchange area (u64 words): a header (word 0 counts waits that ran out of
// polls), then [group][2 buffers][partner][D] tagged words for at most
// kExMaxWgs workgroups.
constexpr int kExHeader = 64;
constexpr int kExMaxWgs = 1024;
constexpr uint32_t kSpinLimit = 1u << 20;

typedef __attribute__((address_space(3))) void* lds_ptr;

// s_waitcnt immediates (gfx9 encoding): every vector memory operation done;
// every LDS operation done.
constexpr int kWaitVmem0 = 0x0F70;
constexpr int kWaitLds0 = 0xC07F;

// Work item i: the i-th (unprotected key head, batch row) pair, heads in
// row-major (l, h) order.  Its slab in the packed key buffers is i itself
// (slot u = i / B is the head's rank among quantized key heads).  Scalar work.
struct ResItem {
  uint32_t s;  // slice (l*B + b)*H + h
  bool valid;
};

__device__ __forceinline__ ResItem res_item(const Params& p, uint32_t item, uint32_t n_items) {
  ResItem it;
  it.valid = item < n_items;
  it.s = 0;
  if (!it.valid) return it;
  const uint32_t u = item / (uint32_t)p.B;
  const uint32_t b = item % (uint32_t)p.B;
  // Word holding the u-th unprotected head: the last word with fewer than
  // u + 1 unprotected heads before it (unprotected before word w:
  // 32w - prefix[w], non-decreasing in w), i.e. the number of words with at
  // most u of them, minus one.  The lanes test 64 words at a time (at most
  // four rounds), so the search is one round of loads, not a chain of
  // dependent ones.
  const uint32_t words = ((uint32_t)p.L * p.H + 31u) / 32u;
  uint32_t lane = threadIdx.x & 63u;
  asm volatile("" : "+v"(lane));  // keeps the lanes' word addresses in the call (not hoisted and spilled)
  uint32_t count = 0;
#pragma unroll
  for (uint32_t w0 = 0; w0 < (uint32_t)kMaskWords; w0 += 64u) {
    if (w0 >= words) break;
    const uint32_t w = min(w0 + lane, words - 1u);
    const bool le = w0 + lane < words && 32u * w - p.route.prefix[w] <= u;
    count += (uint32_t)__popcll(__ballot(le));
  }
  const uint32_t lo = count - 1u;
  uint32_t zeros = ~p.route.mask[lo];  // unprotected heads of word lo (bits past L*H never reached)
  for (uint32_t k = u - (32u * lo - p.route.prefix[lo]); k > 0; --k) zeros &= zeros - 1u;
  const uint32_t i = 32u * lo + (uint32_t)__builtin_ctz(zeros);
  const uint32_t l = i / (uint32_t)p.H, h = i % (uint32_t)p.H;
  it.s = (l * p.B + b) * p.H + h;
  return it;
}

// Buffer resource over `bytes` bytes at `base` (gfx9 raw buffer, no swizzle):
// an access whose offset is at or past `bytes` is dropped by the hardware.
constexpr uint32_t kRawBufferWord3 = 0x00020000u;
constexpr int kNonTemporal = 2;  // buffer instruction cache policy: streaming (nt)
constexpr uint32_t kDropped = 0x80000000u;  // an offset past every resource of this kernel

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc((void*)base, 0, bytes, kRawBufferWord3);
}

// 16-byte streaming load at byte `off` of a buffer resource, into registers
// or, for the whole wavefront, into 64 consecutive 16-byte LDS slots at `dst`
// (lane i at dst + 16 i).  (Device functions: called from the kernel's
// lambdas, the builtins would leave the kernel uninstantiated on the host.)
__device__ __forceinline__ u32x4 buffer_load16(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  return __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, kNonTemporal);
}
__device__ __forceinline__ void buffer_load16_lds(__amdgpu_buffer_rsrc_t r, lds_ptr dst, uint32_t off) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, dst, 16, off, 0, 0, kNonTemporal);
}

// Stores the packed codes of a lane quad's 32 consecutive channels: each lane
// holds the BITS bytes of its 8 channels in the low bits of `piece`; the
// quad's first lane gathers the other three (quad_perm broadcasts, executed
// by every lane) and writes the 4*BITS contiguous bytes at byte `off`.
template <int BITS>
__device__ __forceinline__ void store_quad_codes(__amdgpu_buffer_rsrc_t r, uint32_t off, uint32_t piece,
                                                 bool leader) {
  const uint32_t p1 = (uint32_t)__builtin_amdgcn_mov_dpp((int)piece, 0x55, 0xF, 0xF, false);  // [1,1,1,1]
  const uint32_t p2 = (uint32_t)__builtin_amdgcn_mov_dpp((int)piece, 0xAA, 0xF, 0xF, false);  // [2,2,2,2]
  const uint32_t p3 = (uint32_t)__builtin_amdgcn_mov_dpp((int)piece, 0xFF, 0xF, 0xF, false);  // [3,3,3,3]
  if (!leader) return;
  if constexpr (BITS == 2) {
    const u32x2 w = {piece | (p1 << 16), p2 | (p3 << 16)};
    __builtin_amdgcn_raw_buffer_store_b64(w, r, off, 0, kNonTemporal);
  } else if constexpr (BITS == 3) {
    const u32x3 w = {piece | (p1 << 24), (p1 >> 8) | (p2 << 16), (p2 >> 16) | (p3 << 8)};
    __builtin_amdgcn_raw_buffer_store_b96(w, r, off, 0, kNonTemporal);
  } else {
    static_assert(BITS == 4, "bits");
    const u32x4 w = {piece, p1, p2, p3};
    __builtin_amdgcn_raw_buffer_store_b128(w, r, off, 0, kNonTemporal);
  }
}

// A channel's range in one 64-bit exchange word: the sequence tag in the high
// half, then the maximum's and the minimum's BF16 bits (both are BF16 values:
// the range is taken over BF16 inputs, odd channels masked to their high
// halves), so one relaxed 64-bit store publishes the whole range and a reader
// that sees the tag sees the values with it.
__device__ __forceinline__ uint64_t tagged_range(float lo, float hi, uint32_t gen) {
  return ((uint64_t)gen << 32) | (__float_as_uint(hi) & 0xFFFF0000u) | (__float_as_uint(lo) >> 16);
}

// Folds partner r's range of one channel into [a, b]: `w` is the partner's
// word of the channel, loaded again, with a short sleep, until it carries
// tag `gen` or kSpinLimit polls have passed (then counted).  One word per
// partner and round trip: the minimum and the maximum arrive together.
__device__ __forceinline__ void fold_partner(const uint64_t* w, uint32_t gen, float& a, float& b,
                                             uint32_t& timeouts) {
  uint64_t v = __hip_atomic_load(w, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  for (uint32_t spin = 0; (uint32_t)(v >> 32) != gen; ++spin) {
    if (spin == kSpinLimit) {
      ++timeouts;
      return;
    }
    __builtin_amdgcn_s_sleep(2);
    v = __hip_atomic_load(w, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
  a = fminf(a, __uint_as_float((uint32_t)v << 16));
  b = fmaxf(b, __uint_as_float((uint32_t)v & 0xFFFF0000u));
}

// WIDE (more than kSerialPartners partners): every thread of the workgroup
// polls partners; else one thread per channel polls them all (its own
// instantiation, so the common case keeps the smaller register footprint).
template <int D, int BITS, bool FAKE, bool WIDE>
__global__ __launch_bounds__(kPartThreads) __attribute__((amdgpu_waves_per_eu(4)))
void kivi_part_kernel(const Params p, uint32_t n_items, uint32_t groups, uint32_t parts, uint32_t rows_per_part,
                      uint64_t* __restrict__ ex) {
  constexpr int LEVELS = (1 << BITS) - 1;
  constexpr int ROW = D * BITS / 8;
  constexpr int LR = D / 8;                  // lanes per row (8 channels each)
  constexpr int RPW = 64 / LR;               // rows per wavefront per slot
  constexpr int RS = kPartWaves * RPW;       // rows per slot
  __shared__ u32x4 rows_lds[kPartLdsSlots][kPartThreads];
  __shared__ float red[2 * D];               // per-channel min | max of the workgroup's rows
  __shared__ __attribute__((aligned(16))) uint32_t g_meta[D];
  __shared__ float g_inv[D];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int c = lane % LR;
  const int rw = lane / LR;
  // workgroup -> (group, partner); a group's partners are 8 workgroups apart
  const uint32_t bx = blockIdx.x;
  const uint32_t q = (bx / 8u) % parts;
  const uint32_t g = (bx / (8u * parts)) * 8u + bx % 8u;
  const int T = p.T;
  const int t_lo = (int)(q * rows_per_part);
  const int t_hi = min(t_lo + (int)rows_per_part, T);  // t_hi > t_lo (host)
  const int ch = 8 * c;

  if (tid < D) {
    red[tid] = __builtin_inff();
    red[D + tid] = -__builtin_inff();
  }
  __syncthreads();

  uint32_t item = g;
  ResItem cur = res_item(p, item, n_items);
  if (!cur.valid) return;  // every partner of the group takes the same items

  // First slice row of a slot for this lane (relative to t_lo): made opaque
  // once per slice so that the slots' row offsets are formed where they are
  // used (hoisted, they would all stay live and spill the resident rows).
  const int row0 = wave * RPW + rw;
  int rowb = row0;
  auto slice_rsrc = [&](uint32_t s) { return make_rsrc(p.cache[0] + (size_t)s * T * D, (uint32_t)T * D * 2); };
  auto src_off = [&](int slot) {
    return (uint32_t)min(t_lo + slot * RS + rowb, t_hi - 1) * (D * 2) + (uint32_t)ch * 2;
  };
  auto load_reg = [&](__amdgpu_buffer_rsrc_t r, int slot) { return buffer_load16(r, src_off(slot)); };
  auto load_lds = [&](__amdgpu_buffer_rsrc_t r, int j) {
    buffer_load16_lds(r, (lds_ptr)&rows_lds[j][wave * 64], src_off(j));
  };

  u32x4 v[kPartRegSlots];
  float mn[8], mx[8];
  // The odd channels (high halves) enter the range as the raw 32-bit words:
  // finite BF16 high halves with any low bits order exactly as the BF16
  // values (ties only between equal high halves), so the minimum and maximum
  // words carry the exact BF16 extremes, recovered by masking once per slice.
  auto range8 = [&](const u32x4 w) {
    const float x[8] = {bf16_lo(w.x), __uint_as_float(w.x), bf16_lo(w.y), __uint_as_float(w.y),
                        bf16_lo(w.z), __uint_as_float(w.z), bf16_lo(w.w), __uint_as_float(w.w)};
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      mn[e] = fminf(mn[e], x[e]);
      mx[e] = fmaxf(mx[e], x[e]);
    }
  };
  // Per-channel range over the workgroup's rows (slot rows past t_hi repeat
  // row t_hi - 1): the register slots (the compiler waits for their loads),
  // then, after every vector memory operation has completed (the scheduling
  // barrier keeps the LDS reads behind the wait), the LDS slots.
  auto range_pass = [&]() {
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      mn[e] = __builtin_inff();
      mx[e] = -__builtin_inff();
    }
#pragma unroll
    for (int k = 0; k < kPartRegSlots; ++k) range8(v[k]);
    __builtin_amdgcn_s_waitcnt(kWaitVmem0);
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int j = 0; j < kPartLdsSlots; ++j) range8(rows_lds[j][tid]);
  };

  {
    const __amdgpu_buffer_rsrc_t r = slice_rsrc(cur.s);
#pragma unroll
    for (int j = 0; j < kPartLdsSlots; ++j) load_lds(r, j);
#pragma unroll
    for (int k = 0; k < kPartRegSlots; ++k) v[k] = load_reg(r, kPartLdsSlots + k);
  }
  range_pass();

  uint32_t seq = 0;
  for (;;) {
    const ResItem nxt = res_item(p, item + groups, n_items);

    // 1. the workgroup's range: rows of the wavefront by shuffles, the
    //    wavefronts by LDS atomics
#pragma unroll
    for (int e = 1; e < 8; e += 2) {
      mn[e] = __uint_as_float(__float_as_uint(mn[e]) & 0xFFFF0000u);
      mx[e] = __uint_as_float(__float_as_uint(mx[e]) & 0xFFFF0000u);
    }
#pragma unroll
    for (int e = 0; e < 8; ++e) {
#pragma unroll
      for (int off = LR; off < 64; off *= 2) {
        mn[e] = fminf(mn[e], __shfl_xor(mn[e], off));
        mx[e] = fmaxf(mx[e], __shfl_xor(mx[e], off));
      }
    }
    if (rw == 0) {
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        atomicMin(&red[ch + e], mn[e]);
        atomicMax(&red[D + ch + e], mx[e]);
      }
    }
    __syncthreads();
    // 2. the slice's range from the partners' partial ranges, and its scales
    const size_t slab = (size_t)item;  // [slot][B] with slot = item / B
    if constexpr (WIDE) {
      // Each thread polls every (kPartThreads / D)-th partner for one channel
      // and folds what it found into the workgroup's range in LDS (min and
      // max are idempotent, so a published range that already holds some
      // partners' values is still exact).
      const uint32_t gen = seq + 1;
      uint64_t* buf = ex + kExHeader + ((size_t)g * 2u + (seq & 1u)) * parts * D;
      if (tid < D)
        __hip_atomic_store(buf + (size_t)q * D + tid, tagged_range(red[tid], red[D + tid], gen), __ATOMIC_RELAXED,
                           __HIP_MEMORY_SCOPE_AGENT);
      const int chx = tid % D;
      float a = __builtin_inff(), b = -__builtin_inff();
      uint32_t timeouts = 0;
      for (uint32_t r = (uint32_t)tid / D; r < parts; r += kPartThreads / D)
        if (r != q) fold_partner(buf + (size_t)r * D + chx, gen, a, b, timeouts);
      if (timeouts) __hip_atomic_fetch_add(ex, (uint64_t)timeouts, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      if (a <= b) {
        atomicMin(&red[chx], a);
        atomicMax(&red[D + chx], b);
      }
      __syncthreads();
    }
    if (tid < D) {
      float a = red[tid], b = red[D + tid];
      red[tid] = __builtin_inff();  // reset for the next slice (several barriers away)
      red[D + tid] = -__builtin_inff();
      if (!WIDE && parts > 1) {
        const uint32_t gen = seq + 1;
        uint64_t* buf = ex + kExHeader + ((size_t)g * 2u + (seq & 1u)) * parts * D;
        __hip_atomic_store(buf + (size_t)q * D + tid, tagged_range(a, b, gen), __ATOMIC_RELAXED,
                           __HIP_MEMORY_SCOPE_AGENT);
        uint32_t timeouts = 0;
        for (uint32_t r = 0; r < parts; ++r)
          if (r != q) fold_partner(buf + (size_t)r * D + tid, gen, a, b, timeouts);
        if (timeouts) __hip_atomic_fetch_add(ex, (uint64_t)timeouts, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      }
      const GroupScale gs = group_scale<LEVELS>(a, b);
      g_meta[tid] = gs.meta;
      g_inv[tid] = gs.inv;
      if (!FAKE && q == 0) __builtin_nontemporal_store(gs.meta, p.meta[0] + slab * D + tid);
    }
    __syncthreads();
    ++seq;
    GroupScale gsc[8];  // .meta unused below; one-pass: .m read in emit
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      gsc[e].meta = 0;
      gsc[e].m = FAKE ? 0.0f : bf16_as_float(g_meta[ch + e] >> 16);
      gsc[e].inv = g_inv[ch + e];
    }

    // 3. codes (or the reconstruction) of the workgroup's image rows through a
    //    resource over this slice's outputs; a row outside the image span, or
    //    a slot row past t_hi (the next partner's), gets an offset outside it
    rowb = row0;
    asm volatile("" : "+v"(rowb));
    const __amdgpu_buffer_rsrc_t res =
        FAKE ? make_rsrc(p.out[0] + ((size_t)cur.s * T + p.s0) * D, (uint32_t)p.n * D * 2)
             : make_rsrc(p.codes[0] + slab * p.n * ROW, (uint32_t)p.n * ROW);
    constexpr uint32_t kStride = FAKE ? D * 2 : ROW;
    const uint32_t lane_off = FAKE ? (uint32_t)ch * 2 : (uint32_t)c * BITS;
    const bool leader = (c & 3) == 0;
    auto emit = [&](u32x4 w, int slot) {
      asm volatile("" : "+v"(w));  // convert here, not reuse the range pass's values
      const int r = t_lo + slot * RS + rowb;
      const uint32_t off = r < t_hi ? (uint32_t)(r - p.s0) * kStride + lane_off : kDropped;
      const float x[8] = {bf16_lo(w.x), bf16_hi(w.x), bf16_lo(w.y), bf16_hi(w.y),
                          bf16_lo(w.z), bf16_hi(w.z), bf16_lo(w.w), bf16_hi(w.w)};
      if constexpr (FAKE) {
        // the metadata words (min and scale) are read back from LDS here
        // (held in registers with the rest, they would spill)
        const u32x4 m0 = *(const u32x4*)&g_meta[ch], m1 = *(const u32x4*)&g_meta[ch + 4];
        const uint32_t mw[8] = {m0.x, m0.y, m0.z, m0.w, m1.x, m1.y, m1.z, m1.w};
        float y[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          GroupScale ge;
          ge.m = bf16_as_float(mw[e] >> 16);
          ge.inv = gsc[e].inv;
          y[e] = __builtin_fmaf(__builtin_rintf(code_scaled(x[e], ge)), bf16_as_float(mw[e] & 0xFFFFu), ge.m);
        }
        const u32x4 o = {pack_bf16x2_hw(y[0], y[1]), pack_bf16x2_hw(y[2], y[3]), pack_bf16x2_hw(y[4], y[5]),
                         pack_bf16x2_hw(y[6], y[7])};
        __builtin_amdgcn_raw_buffer_store_b128(o, res, off, 0, kNonTemporal);
      } else {
        uint32_t cb[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) cb[e] = code_bits(x[e], gsc[e]);
        store_quad_codes<BITS>(res, off, pack_code_bits<8, BITS>(cb).w[0], leader);
      }
    };
    // The register slots come first, each refilled as soon as it is coded
    // (scheduling barriers keep each refill after the slot's use), so the
    // next slice's loads start at once.  The LDS slots are then all read
    // before any of them is refilled: an LDS read issued after a pending
    // direct-to-LDS load would wait for that load.
    auto code_pass = [&](bool refill) {
      const __amdgpu_buffer_rsrc_t r = slice_rsrc(nxt.s);
#pragma unroll
      for (int k = 0; k < kPartRegSlots; ++k) {
        emit(v[k], kPartLdsSlots + k);
        __builtin_amdgcn_sched_barrier(0);
        if (refill) v[k] = load_reg(r, kPartLdsSlots + k);
      }
#pragma unroll
      for (int j = 0; j < kPartLdsSlots; ++j) {
        emit(rows_lds[j][tid], j);
        __builtin_amdgcn_sched_barrier(0);
      }
      if (refill) {
        __builtin_amdgcn_s_waitcnt(kWaitLds0);  // every slot read before it is refilled
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int j = 0; j < kPartLdsSlots; ++j) load_lds(r, j);
      }
    };
    if (!nxt.valid) {
      code_pass(false);
      break;
    }
    code_pass(true);
    range_pass();
    cur = nxt;
    item += groups;
  }
}

// ------------------------------------------------------------ split kernels
//
// Slices too long for the resident kernel (or a device with too few compute
// units for a group): every slice is cut into chunks of kSplitRows rows, so
// all compute units share even a few long slices.  A range launch takes one
// (slice, chunk) per workgroup and merges the chunk's per-channel minimum and
// maximum into two words per channel of the workspace with device-scope
// atomic maxima on order-preserving images of the floats (the minimum as the
// complement of its image), so zero is the identity of both and the order of
// the merges cannot change the result; a code launch then takes one (slice,
// image chunk) per workgroup, forms the scales from the words and writes its
// rows' codes (its first chunk also the metadata).  Work items are taken in
// batches of kSplitBatch slices, whose words are cleared before their range
// launch.

constexpr int kSplitThreads = 512;
constexpr int kSplitWaves = kSplitThreads / 64;
constexpr int kSplitRows = 2048;
constexpr int kSplitRangeUnroll = 8;  // rows in flight per lane
constexpr int kSplitCodeUnroll = 16;
constexpr uint32_t kSplitBatch = 2 * kExMaxWgs;  // slices of 2D 32-bit words in the exchange area

// Order-preserving unsigned image of a float (finite or infinite): a < b
// implies ord(a) < ord(b), and every image is above 0.
__device__ __forceinline__ uint32_t ord_image(float f) {
  const uint32_t u = __float_as_uint(f);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}
__device__ __forceinline__ float from_ord_image(uint32_t o) {
  return __uint_as_float((o & 0x80000000u) ? (o & 0x7FFFFFFFu) : ~o);
}

template <int D>
__global__ __launch_bounds__(kSplitThreads) void kivi_split_range_kernel(const Params p, uint32_t item0,
                                                                         uint32_t n_items, uint32_t chunks,
                                                                         uint32_t* __restrict__ words) {
  constexpr int CPT = D / 8;
  __shared__ float red[2 * D];
  const int tid = threadIdx.x;
  const uint32_t local = blockIdx.x / chunks, chunk = blockIdx.x % chunks;
  const ResItem it = res_item(p, item0 + local, n_items);  // valid: the grid covers the batch exactly
  for (int i = tid; i < 2 * D; i += kSplitThreads) red[i] = i < D ? __builtin_inff() : -__builtin_inff();
  __syncthreads();
  const int t_begin = (int)chunk * kSplitRows;
  const int t_end = min(p.T, t_begin + kSplitRows);
  float mn[8], mx[8];
  range_rows<D, kSplitWaves, kSplitRangeUnroll>(p.cache[0] + (size_t)it.s * p.T * D, t_begin, t_end, mn, mx);
  const int lane = tid & 63;
  if (lane < CPT) {
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      atomicMin(&red[8 * lane + e], mn[e]);
      atomicMax(&red[D + 8 * lane + e], mx[e]);
    }
  }
  __syncthreads();
  if (tid < D) {
    uint32_t* w = words + (size_t)local * 2 * D;
    __hip_atomic_fetch_max(w + tid, ~ord_image(red[tid]), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __hip_atomic_fetch_max(w + D + tid, ord_image(red[D + tid]), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
}

template <int D, int BITS, bool FAKE>
__global__ __launch_bounds__(kSplitThreads) void kivi_split_code_kernel(const Params p, uint32_t item0,
                                                                        uint32_t n_items, uint32_t chunks,
                                                                        const uint32_t* __restrict__ words) {
  constexpr int CPT = D / 8;
  constexpr int LEVELS = (1 << BITS) - 1;
  constexpr int ROW = D * BITS / 8;
  __shared__ uint32_t g_meta[D];
  __shared__ float g_inv[D];
  const int tid = threadIdx.x;
  const uint32_t local = blockIdx.x / chunks, chunk = blockIdx.x % chunks;
  const uint32_t item = item0 + local;
  const ResItem it = res_item(p, item, n_items);
  const size_t slab = (size_t)item;  // [slot][B] with slot = item / B
  if (tid < D) {
    const uint32_t* w = words + (size_t)local * 2 * D;
    const GroupScale gs = group_scale<LEVELS>(from_ord_image(~w[tid]), from_ord_image(w[D + tid]));
    g_meta[tid] = gs.meta;
    g_inv[tid] = gs.inv;
    if (!FAKE && chunk == 0) __builtin_nontemporal_store(gs.meta, p.meta[0] + slab * D + tid);
  }
  __syncthreads();
  const int c8 = (tid & 63) % CPT;
  GroupScale g[8];
  float S[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    g[e].meta = g_meta[8 * c8 + e];
    g[e].m = bf16_as_float(g[e].meta >> 16);
    g[e].inv = g_inv[8 * c8 + e];
    S[e] = bf16_as_float(g[e].meta & 0xFFFFu);
  }
  const int t_begin = (int)chunk * kSplitRows;
  const int t_end = min(p.n, t_begin + kSplitRows);
  code_rows<D, BITS, FAKE, kSplitWaves, kSplitCodeUnroll>(p.cache[0] + ((size_t)it.s * p.T + p.s0) * D,
                                        FAKE ? nullptr : p.codes[0] + slab * p.n * ROW,
                                        FAKE ? p.out[0] + ((size_t)it.s * p.T + p.s0) * D : nullptr, t_begin, t_end,
                                        g, S);
}

// Zeroes the exchange words a launch uses (a kernel rather than a memset, so
// the call can be captured in a graph).
__global__ void zero_words_kernel(uint64_t* w, uint32_t n) {
  for (uint32_t i = blockIdx.x * blockDim.x + threadIdx.x; i < n; i += gridDim.x * blockDim.x) w[i] = 0;
}

// ---------------------------------------------------------------- host side

int kivi_part_capacity(int D) { return kPartSlots * kPartWaves * (512 / D); }

// Workgroups per slice of the resident kernel, 0 for the split kernels.  A
// grid holds 8 groups per 8 P workgroups, so past 8 partners P is rounded up
// to 16 or 32, which fill every compute unit; each partner keeps at least one
// row ((P - 1) ceil(T / P) < T holds for T > (P - 1)^2).
int kivi_partners(int T, int D) {
  const int cap = kivi_part_capacity(D);
  int parts = (T + cap - 1) / cap;
  if (parts > kMaxPartners || (uint64_t)T * D * 2 >= (1ull << 31)) return 0;  // split kernels
  if (parts > kSerialPartners) parts = parts <= 16 ? 16 : 32;
  if ((uint64_t)(parts - 1) * (uint64_t)((T + parts - 1) / parts) >= (uint64_t)T) return 0;
  return parts;
}

// The exchange area: the resident kernel's partial ranges when several
// workgroups hold a slice, else (longer slices) the split kernels' range
// words; a slice that one workgroup holds needs none.
uint64_t kivi_workspace_bytes(int T, int D) {
  return T > kivi_part_capacity(D) ? ((uint64_t)kExHeader + (uint64_t)kExMaxWgs * 2 * D) * 8 : 0;
}

// Compute units the persistent grids are sized for: the device's, or fewer
// with HG_TEST_CUS=n in the environment (a test hook: results must not
// depend on the grid).
static hipError_t grid_cus(int* cus) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e == hipSuccess) e = hipDeviceGetAttribute(cus, hipDeviceAttributeMultiprocessorCount, dev);
  if (e != hipSuccess) return e;
  const char* s = getenv("HG_TEST_CUS");
  if (s && *s) *cus = std::max(1, std::min(*cus, atoi(s)));
  return hipSuccess;
}

// Launch plan of one call's key kernels: the resident kernel when every
// workgroup of its grid can be resident at once (and, with several per slice,
// an exchange workspace is given), else, with a workspace, the split range
// and code kernels, and without one (a slice one workgroup holds, on a device
// with fewer than 8 compute units) the two-pass kernel; and the leading
// workspace words to clear before it (the exchange words the resident grid
// uses, or the header and the first batch's range words: the split kernels
// wait for nothing, so the header's first word then reads 0).
struct KiviPlan {
  bool resident = false;
  bool split = false;
  int parts = 0;
  uint32_t n_items = 0, groups = 0, rows_per_part = 0;
  uint32_t clear_words = 0;
};

template <int D, int BITS, bool FAKE>
static hipError_t plan_k(const Params& p, bool has_ws, KiviPlan* pl) {
  *pl = KiviPlan();
  pl->n_items = (uint32_t)p.n_unprot_k * (uint32_t)p.B;
  if (pl->n_items == 0) return hipSuccess;  // every key head kept in BF16: nothing to quantize here
  int cus = 0;
  hipError_t e = grid_cus(&cus);
  if (e != hipSuccess) return e;
  const int parts = kivi_partners(p.T, D);
  if (parts > 0 && (parts == 1 || has_ws)) {
    int per_cu = 0;
    e = parts > kSerialPartners
            ? hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kivi_part_kernel<D, BITS, FAKE, true>, kPartThreads, 0)
            : hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kivi_part_kernel<D, BITS, FAKE, false>, kPartThreads,
                                                           0);
    if (e != hipSuccess) return e;
    const uint32_t resident = (uint32_t)std::max(per_cu, 0) * (uint32_t)cus;  // workgroups held at once
    uint32_t cap = resident / (uint32_t)parts;
    if (parts > 1) cap = std::min(cap, (uint32_t)(kExMaxWgs / parts));
    cap = cap / 8u * 8u;
    const uint32_t rows_per_part = (uint32_t)((p.T + parts - 1) / parts);
    if (cap > 0 && rows_per_part <= (uint32_t)kivi_part_capacity(D)) {  // every row fits a slot
      pl->resident = true;
      pl->parts = parts;
      pl->groups = std::min((pl->n_items + 7u) / 8u * 8u, cap);
      pl->rows_per_part = rows_per_part;
      if (parts > 1) pl->clear_words = (uint32_t)(kExHeader + (uint64_t)pl->groups * 2 * parts * D);
      return hipSuccess;
    }
  }
  if (has_ws) {
    pl->split = true;
    pl->clear_words = (uint32_t)(kExHeader + (uint64_t)std::min(pl->n_items, kSplitBatch) * D);
  }
  return hipSuccess;
}

template <int D, int BITS, bool FAKE>
static hipError_t launch_k(const Params& p, void* ws, bool cleared, hipStream_t stream) {
  KiviPlan pl;
  hipError_t e = plan_k<D, BITS, FAKE>(p, ws != nullptr, &pl);
  if (e != hipSuccess || pl.n_items == 0) return e;
  if (pl.clear_words > 0 && !cleared) {
    hipLaunchKernelGGL(zero_words_kernel, dim3(std::min<uint32_t>((pl.clear_words + 255) / 256, 1024)), dim3(256),
                       0, stream, (uint64_t*)ws, pl.clear_words);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  if (pl.resident) {
    const dim3 grid(pl.groups * (uint32_t)pl.parts);
    if (pl.parts > kSerialPartners)
      hipLaunchKernelGGL((kivi_part_kernel<D, BITS, FAKE, true>), grid, dim3(kPartThreads), 0, stream, p, pl.n_items,
                         pl.groups, (uint32_t)pl.parts, pl.rows_per_part, (uint64_t*)ws);
    else
      hipLaunchKernelGGL((kivi_part_kernel<D, BITS, FAKE, false>), grid, dim3(kPartThreads), 0, stream, p, pl.n_items,
                         pl.groups, (uint32_t)pl.parts, pl.rows_per_part, (uint64_t*)ws);
    return hipGetLastError();
  }
  if (pl.split) {
    uint32_t* words = (uint32_t*)((uint64_t*)ws + kExHeader);
    const uint32_t range_chunks = (uint32_t)((p.T + kSplitRows - 1) / kSplitRows);
    const uint32_t code_chunks = (uint32_t)((p.n + kSplitRows - 1) / kSplitRows);
    // slices per launch pair: the words area's, and few enough that a launch
    // stays under 2^32 work-items
    const uint64_t chunks = std::max(range_chunks, code_chunks);
    const uint32_t batch = (uint32_t)std::max<uint64_t>(
        1, std::min<uint64_t>(kSplitBatch, (0xFFFFFFFFull / kSplitThreads) / chunks));
    for (uint32_t i0 = 0; i0 < pl.n_items; i0 += batch) {
      const uint32_t nb = std::min(batch, pl.n_items - i0);
      if (i0 > 0) {  // the first batch's words were cleared with the header
        const uint32_t n64 = nb * (uint32_t)D;  // 2D 32-bit words per slice
        hipLaunchKernelGGL(zero_words_kernel, dim3(std::min<uint32_t>((n64 + 255) / 256, 1024)), dim3(256), 0, stream,
                           (uint64_t*)words, n64);
      }
      hipLaunchKernelGGL((kivi_split_range_kernel<D>), dim3(nb * range_chunks), dim3(kSplitThreads), 0, stream, p, i0,
                         pl.n_items, range_chunks, words);
      hipLaunchKernelGGL((kivi_split_code_kernel<D, BITS, FAKE>), dim3(nb * code_chunks), dim3(kSplitThreads), 0,
                         stream, p, i0, pl.n_items, code_chunks, (const uint32_t*)words);
      e = hipGetLastError();
      if (e != hipSuccess) return e;
    }
    return hipSuccess;
  }
  int cus = 0;
  e = grid_cus(&cus);
  if (e != hipSuccess) return e;
  const uint32_t slices = (uint32_t)p.L * p.B * p.H;
  const uint32_t blocks = std::min<uint32_t>(slices, (uint32_t)std::max(cus, 1) * kSeqBlocksPerCU);
  hipLaunchKernelGGL((kivi_seq_kernel<D, BITS, FAKE>), dim3(blocks), dim3(kSeqThreads), 0, stream, p);
  return hipGetLastError();
}

template <int D, int BITS, bool FAKE>
static hipError_t plan_words(const Params& p, void* ws, uint32_t* clear_words) {
  KiviPlan pl;
  const hipError_t e = plan_k<D, BITS, FAKE>(p, ws != nullptr, &pl);
  *clear_words = pl.clear_words;
  return e;
}

// With clear_words: only the number of workspace words the launch needs
// cleared; else the launch.
template <int D, bool FAKE>
static hipError_t kivi_d(const Params& p, int bits, void* ws, bool cleared, uint32_t* clear_words,
                         hipStream_t stream) {
  switch (bits) {
    case 2: return clear_words ? plan_words<D, 2, FAKE>(p, ws, clear_words) : launch_k<D, 2, FAKE>(p, ws, cleared, stream);
    case 3: return clear_words ? plan_words<D, 3, FAKE>(p, ws, clear_words) : launch_k<D, 3, FAKE>(p, ws, cleared, stream);
    case 4: return clear_words ? plan_words<D, 4, FAKE>(p, ws, clear_words) : launch_k<D, 4, FAKE>(p, ws, cleared, stream);
    default: return hipErrorInvalidValue;
  }
}

static hipError_t kivi_dispatch(const Params& p, int D, int bits, bool fake, void* ws, bool cleared,
                                uint32_t* clear_words, hipStream_t stream) {
  switch (D) {
    case 64: return fake ? kivi_d<64, true>(p, bits, ws, cleared, clear_words, stream)
                         : kivi_d<64, false>(p, bits, ws, cleared, clear_words, stream);
    case 128: return fake ? kivi_d<128, true>(p, bits, ws, cleared, clear_words, stream)
                          : kivi_d<128, false>(p, bits, ws, cleared, clear_words, stream);
    case 256: return fake ? kivi_d<256, true>(p, bits, ws, cleared, clear_words, stream)
                          : kivi_d<256, false>(p, bits, ws, cleared, clear_words, stream);
    default: return hipErrorInvalidValue;
  }
}

hipError_t kivi_seq_clear_words(const Params& p, int D, int bits, bool fake, void* ws, uint32_t* words) {
  *words = 0;
  return kivi_dispatch(p, D, bits, fake, ws, false, words, nullptr);
}

hipError_t launch_kivi_seq(const Params& p, int D, int bits, bool fake, void* ws, bool cleared, hipStream_t stream) {
  return kivi_dispatch(p, D, bits, fake, ws, cleared, nullptr, stream);
}

}  // namespace hg
