// KIVI-style keys with one range per channel over the whole supplied
// sequence, text included (HeadGuard §4, Quantization setup: the KIVI-style
// base recomputes key ranges over the supplied sequence, including text,
// while text KV stays BF16).  Selected by kivi_group = 0.
//
// Every code depends on the range of its channel over all T rows of the
// slice, so a slice must be fully read before any of its codes is formed.
// Two kernels:
//
// Resident (T <= kResRows): a persistent grid, one 1024-thread workgroup per
// compute unit.  A workgroup takes one 64-channel part of a key slice (l, b, h)
// and holds all T rows of that part on chip — 9 row slots in LDS, filled by
// buffer loads that write LDS directly, and 15 in registers, 128 rows per
// slot — so each slice is read from HBM exactly once:
//  1. per-channel min / max over the resident rows (each lane holds 8
//     channels of one row per slot), reduced across the wavefront's rows by
//     shuffles and across the 16 wavefronts through LDS; 64 lanes form the
//     part's group scales and write its metadata words;
//  2. codes (or, for the one-pass simulated quantization, the BF16
//     reconstruction) of the image rows from the resident copy; as the slots
//     are consumed, the loads of the workgroup's next slice are issued into
//     them, so the next slice streams in while this one is coded.
// The parts of one slice go to workgroups whose indices differ by multiples
// of 8 (the dispatcher places those on the same XCD), so a slice's parts are
// processed at the same time.
//
// Two-pass (longer slices): a persistent grid of kSeqBlocksPerCU workgroups
// of kSeqThreads threads per compute unit walks the key slices; per slice a
// range pass over all T rows, the wavefronts' partial ranges combined through
// LDS, then a second pass over the image rows for the codes.  The grid is
// sized so that the slices in flight at once stay within the 256 MB Infinity
// Cache, which then serves much of the second read.
//
// Values, protected slices and the rest of the cache are handled by the
// regular kernels of the same call.

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

// ------------------------------------------------------ resident variant

constexpr int kResThreads = 1024;
constexpr int kResWaves = kResThreads / 64;
constexpr int kResPart = 64;                                  // channels per workgroup part
constexpr int kResLanesPerRow = kResPart / 8;                 // 8 channels per lane
constexpr int kResRowsPerWave = 64 / kResLanesPerRow;         // rows per load instruction
constexpr int kResRowsPerSlot = kResWaves * kResRowsPerWave;  // 128
constexpr int kResLdsSlots = 9;
constexpr int kResRegSlots = 15;
constexpr int kResSlots = kResLdsSlots + kResRegSlots;
constexpr int kResRows = kResSlots * kResRowsPerSlot;         // 3072

typedef __attribute__((address_space(3))) void* lds_ptr;

// s_waitcnt immediates (gfx9 encoding): every vector memory operation done;
// every LDS operation done.
constexpr int kWaitVmem0 = 0x0F70;
constexpr int kWaitLds0 = 0xC07F;

// Work item i of the resident kernel: the i-th (unprotected key head, batch
// row) pair, heads in row-major (l, h) order.  Its slab in the packed key
// buffers is i itself (slot u = i / B is the head's rank among quantized key
// heads).  Scalar work.
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
// a store whose offset is at or past `bytes` is dropped by the hardware.
constexpr uint32_t kRawBufferWord3 = 0x00020000u;
constexpr int kNonTemporal = 2;  // buffer instruction cache policy: streaming (nt)

__device__ __forceinline__ __amdgpu_buffer_rsrc_t out_rsrc(void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(base, 0, bytes, kRawBufferWord3);
}

// 16-byte load at byte `off` of a buffer resource, into registers or, for
// the whole wavefront, into 64 consecutive 16-byte LDS slots at `dst` (lane i
// at dst + 16 i).
__device__ __forceinline__ u32x4 buffer_load16(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  return __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, kNonTemporal);
}
__device__ __forceinline__ void buffer_load16_lds(__amdgpu_buffer_rsrc_t r, lds_ptr dst, uint32_t off) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, dst, 16, off, 0, 0, kNonTemporal);
}

// Store of one lane's 8 codes (BITS bytes) at byte `off` of the resource,
// with the default (write-back) cache policy, which measured faster than
// streaming stores for these small pieces (the parts of a packed code row are
// written by different workgroups, so every store covers part of a line).
template <int BITS>
__device__ __forceinline__ void store_codes8(__amdgpu_buffer_rsrc_t r, uint32_t off, uint32_t w) {
  if constexpr (BITS == 2) {
    __builtin_amdgcn_raw_buffer_store_b16((uint16_t)w, r, off, 0, 0);
  } else if constexpr (BITS == 4) {
    __builtin_amdgcn_raw_buffer_store_b32(w, r, off, 0, 0);
  } else {
    static_assert(BITS == 3, "bits");
    __builtin_amdgcn_raw_buffer_store_b8((uint8_t)w, r, off, 0, 0);
    __builtin_amdgcn_raw_buffer_store_b8((uint8_t)(w >> 8), r, off + 1, 0, 0);
    __builtin_amdgcn_raw_buffer_store_b8((uint8_t)(w >> 16), r, off + 2, 0, 0);
  }
}

template <int D, int BITS, bool FAKE>
__global__ __launch_bounds__(kResThreads) void kivi_res_kernel(const Params p, uint32_t n_items,
                                                               uint32_t streams) {
  constexpr int PARTS = D / kResPart;
  constexpr int LEVELS = (1 << BITS) - 1;
  constexpr int ROW = D * BITS / 8;
  __shared__ u32x4 rows_lds[kResLdsSlots][kResThreads];
  __shared__ float part_rng[2][kResWaves][kResPart];
  __shared__ uint32_t g_meta[kResPart];
  __shared__ float g_inv[kResPart];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int c = lane % kResLanesPerRow;
  const int r = lane / kResLanesPerRow;
  const int row0 = wave * kResRowsPerWave + r;  // row of slot 0 held by this lane
  // workgroup -> (stream, part); the parts of a stream are 8 workgroups apart
  const uint32_t bx = blockIdx.x;
  const int part = (int)((bx / 8u) % PARTS);
  const uint32_t stream = (bx / (8u * PARTS)) * 8u + bx % 8u;
  const int ch = part * kResPart + 8 * c;       // first of this lane's 8 channels
  const int T = p.T;

  uint32_t item = stream;
  ResItem cur = res_item(p, item, n_items);
  if (!cur.valid) return;

  // Row of a slot for this lane: `rowb` is row0, made opaque to the compiler
  // once per slice so that the 24 slots' row offsets are formed where they
  // are used instead of being hoisted out of the slice loop (which keeps them
  // all live and spills the resident rows).
  int rowb = row0;
  // Loads go through a buffer resource over the slice (wave-uniform), with a
  // 32-bit per-lane byte offset: rows past T repeat row T-1.
  auto slice_rsrc = [&](uint32_t s) {
    return __builtin_amdgcn_make_buffer_rsrc((void*)(p.cache[0] + (size_t)s * T * D), 0,
                                             (uint32_t)T * D * 2, kRawBufferWord3);
  };
  auto src_off = [&](int slot) {
    return (uint32_t)min(slot * kResRowsPerSlot + rowb, T - 1) * (D * 2) + (uint32_t)ch * 2;
  };
  auto load_reg = [&](__amdgpu_buffer_rsrc_t r, int slot) { return buffer_load16(r, src_off(slot)); };
  auto load_lds = [&](__amdgpu_buffer_rsrc_t r, int j) {
    buffer_load16_lds(r, (lds_ptr)&rows_lds[j][wave * 64], src_off(j));
  };

  u32x4 v[kResRegSlots];
  float mn[8], mx[8];
  auto range8 = [&](const u32x4 w) {
    const float x[8] = {bf16_lo(w.x), bf16_hi(w.x), bf16_lo(w.y), bf16_hi(w.y),
                        bf16_lo(w.z), bf16_hi(w.z), bf16_lo(w.w), bf16_hi(w.w)};
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      mn[e] = fminf(mn[e], x[e]);
      mx[e] = fmaxf(mx[e], x[e]);
    }
  };
  // Per-channel range over all T rows of the slice (slot rows past T repeat
  // row T-1): the register slots (the compiler waits for their loads), then,
  // after every vector memory operation has completed (the fence keeps the
  // LDS reads behind the wait), the LDS slots.
  auto range_pass = [&]() {
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      mn[e] = __builtin_inff();
      mx[e] = -__builtin_inff();
    }
#pragma unroll
    for (int k = 0; k < kResRegSlots; ++k) range8(v[k]);
    __builtin_amdgcn_s_waitcnt(kWaitVmem0);
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int j = 0; j < kResLdsSlots; ++j) range8(rows_lds[j][tid]);
  };

  // prologue: the first slice's loads and its range pass
  {
    const __amdgpu_buffer_rsrc_t r = slice_rsrc(cur.s);
#pragma unroll
    for (int j = 0; j < kResLdsSlots; ++j) load_lds(r, j);
#pragma unroll
    for (int k = 0; k < kResRegSlots; ++k) v[k] = load_reg(r, kResLdsSlots + k);
  }
  range_pass();

  for (;;) {
    const ResItem nxt = res_item(p, item + streams, n_items);

    // scales: the wavefront's rows by shuffles, the 16 wavefronts through LDS
#pragma unroll
    for (int e = 0; e < 8; ++e) {
#pragma unroll
      for (int off = kResLanesPerRow; off < 64; off *= 2) {
        mn[e] = fminf(mn[e], __shfl_xor(mn[e], off));
        mx[e] = fmaxf(mx[e], __shfl_xor(mx[e], off));
      }
    }
    if (r == 0) {
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        part_rng[0][wave][8 * c + e] = mn[e];
        part_rng[1][wave][8 * c + e] = mx[e];
      }
    }
    __syncthreads();
    const size_t slab = (size_t)item;  // [slot][B] with slot = item / B
    if (tid < kResPart) {
      float a = part_rng[0][0][tid], b = part_rng[1][0][tid];
#pragma unroll
      for (int w = 1; w < kResWaves; ++w) {
        a = fminf(a, part_rng[0][w][tid]);
        b = fmaxf(b, part_rng[1][w][tid]);
      }
      const GroupScale g = group_scale<LEVELS>(a, b);
      g_meta[tid] = g.meta;
      g_inv[tid] = g.inv;
      if (!FAKE) __builtin_nontemporal_store(g.meta, p.meta[0] + slab * D + part * kResPart + tid);
    }
    __syncthreads();
    GroupScale g[8];  // .meta unused below
    float S[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const uint32_t w = g_meta[8 * c + e];
      g[e].meta = 0;
      g[e].m = bf16_as_float(w >> 16);
      g[e].inv = g_inv[8 * c + e];
      S[e] = FAKE ? bf16_as_float(w & 0xFFFFu) : 0.0f;
    }

    // Codes (or the reconstruction) of the image rows, through buffer
    // resources over this slice's outputs: a text row, or a slot row past T,
    // has an offset outside the resource and its store is dropped, so the
    // code pass has no branches.
    rowb = row0;
    asm volatile("" : "+v"(rowb));
    // (the resource is wave-uniform, the slice's image rows; the lane's
    // channels are part of its offset)
    const __amdgpu_buffer_rsrc_t res =
        FAKE ? out_rsrc(p.out[0] + ((size_t)cur.s * T + p.s0) * D, (uint32_t)p.n * D * 2)
             : out_rsrc(p.codes[0] + slab * p.n * ROW, (uint32_t)p.n * ROW);
    // Byte offset of a slot row's piece: rows before the span wrap to huge
    // offsets and rows at or past its end (slot rows past T included, as
    // s0 + n <= T) land at or past n rows; both fall outside the resource.
    constexpr uint32_t kStride = FAKE ? D * 2 : ROW;
    const uint32_t lane_off = (FAKE ? (uint32_t)ch * 2 : (uint32_t)(ch / 8) * BITS) - (uint32_t)p.s0 * kStride;
    auto emit = [&](u32x4 w, int slot) {
      asm volatile("" : "+v"(w));  // convert here, not reuse the range pass's values
      const uint32_t off = (uint32_t)(slot * kResRowsPerSlot + rowb) * kStride + lane_off;
      const float x[8] = {bf16_lo(w.x), bf16_hi(w.x), bf16_lo(w.y), bf16_hi(w.y),
                          bf16_lo(w.z), bf16_hi(w.z), bf16_lo(w.w), bf16_hi(w.w)};
      uint32_t cb[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) cb[e] = code_bits(x[e], g[e]);
      if constexpr (FAKE) {
        float y[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) y[e] = __builtin_fmaf((float)(cb[e] - kMagicBits), S[e], g[e].m);
        const u32x4 o = {pack_bf16x2_hw(y[0], y[1]), pack_bf16x2_hw(y[2], y[3]), pack_bf16x2_hw(y[4], y[5]),
                         pack_bf16x2_hw(y[6], y[7])};
        __builtin_amdgcn_raw_buffer_store_b128(o, res, off, 0, kNonTemporal);
      } else {
        store_codes8<BITS>(res, off, pack_code_bits<8, BITS>(cb).w[0]);
      }
    };
    // The register slots come first, each refilled as soon as it is coded
    // (scheduling barriers keep each refill after the slot's use: hoisted
    // refills would need a second copy of the rows), so the next slice's
    // loads start at once.  The LDS slots are then all read before any of
    // them is refilled: the compiler cannot tell the slots apart, and an LDS
    // read issued after a pending direct-to-LDS load makes it wait for that
    // load.
    auto code_pass = [&](bool refill) {
      const __amdgpu_buffer_rsrc_t r = slice_rsrc(nxt.s);
#pragma unroll
      for (int k = 0; k < kResRegSlots; ++k) {
        emit(v[k], kResLdsSlots + k);
        __builtin_amdgcn_sched_barrier(0);
        if (refill) v[k] = load_reg(r, kResLdsSlots + k);
      }
#pragma unroll
      for (int j = 0; j < kResLdsSlots; ++j) {
        emit(rows_lds[j][tid], j);
        __builtin_amdgcn_sched_barrier(0);
      }
      if (refill) {
        __builtin_amdgcn_s_waitcnt(kWaitLds0);  // every slot read before it is refilled
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int j = 0; j < kResLdsSlots; ++j) load_lds(r, j);
      }
    };
    if (!nxt.valid) {
      code_pass(false);
      break;
    }
    code_pass(true);
    range_pass();
    cur = nxt;
    item += streams;
  }
}

template <int D, int BITS>
static hipError_t launch_k(const Params& p, bool fake, hipStream_t stream) {
  int dev = 0, cus = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e == hipSuccess) e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
  if (e != hipSuccess) return e;
  const uint32_t slices = (uint32_t)p.L * p.B * p.H;
  if (p.T <= kResRows) {
    // one workgroup per compute unit, in whole groups of 8 * PARTS (a stream's parts 8 apart)
    constexpr uint32_t PARTS = D / kResPart;
    const uint32_t unit = 8u * PARTS;
    const uint32_t n_items = (uint32_t)p.n_unprot_k * (uint32_t)p.B;
    const uint32_t want = (n_items + 7u) / 8u * unit;  // no more streams than items (rounded up)
    const uint32_t blocks = std::max(unit, std::min((uint32_t)std::max(cus, 1) / unit * unit, want));
    const uint32_t streams = blocks / PARTS;
    if (fake)
      hipLaunchKernelGGL((kivi_res_kernel<D, BITS, true>), dim3(blocks), dim3(kResThreads), 0, stream, p,
                         n_items, streams);
    else
      hipLaunchKernelGGL((kivi_res_kernel<D, BITS, false>), dim3(blocks), dim3(kResThreads), 0, stream, p,
                         n_items, streams);
    return hipGetLastError();
  }
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
