// Kernel parameter block and launchers shared by the host API and the
// quantize / dequantize kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <functional>

#include "headguard.h"

namespace hg {

constexpr int kThreads = 256;        // 4 wavefronts of 64
constexpr int kWaveTokens = 32;      // tokens per wavefront tile
constexpr int kBlockTokens = 128;    // tokens per workgroup tile (4 x 32)
constexpr int kMinBlockTokens = 64;  // smallest workgroup tile of any launch (dequantize, one-pass)
// Register budget: at least this many wavefronts per SIMD, so enough 16-byte
// loads are in flight per CU to cover HBM latency.
constexpr int kMinWaves = 4;
constexpr int kMaskWords = HG_MAX_HEADS / 32;

// Occupancy cap through a launch-time LDS reservation: gfx950 has 160 KiB of
// LDS per compute unit, and a workgroup that reserves just over 1/(w + 1) of
// it leaves room for w workgroups per compute unit but not w + 1 — for a
// 4-wavefront workgroup, w wavefronts per SIMD.  0: no cap.
constexpr size_t kLdsPerCU = 160 * 1024;
constexpr size_t occupancy_lds(int waves) { return waves > 0 ? kLdsPerCU / (waves + 1) + 512 : 0; }
// Wavefronts per SIMD of the quantize and dequantize kernels: at the 8 their
// registers allow, the memory system is oversubscribed (6 measured faster
// than 8, 5 and 4 over the workloads at 2 bits; quantize kernels whose
// registers already allow fewer, such as KIVI key groups at 4, are not
// affected).  Quantize lowers it for some launches (kQuantizeWavesOf).
constexpr int kQuantizeWaves = 6;
constexpr int kDequantizeWaves = 6;
// The min-max dequantize instantiation (per-token groups only: min-max keys
// and values, AKVQ-style values): 4 (kernel time 1095 -> 1053 us on the
// LLaVA-1.5-shaped cache, 872 -> 854 on the 72B-shaped one, 711 -> 698 at
// head_dim 256, 363 -> 351 for InternVL-shaped values) when a launch writes
// at least 1 GiB of rows; smaller launches keep 6 (dequantize.hip).  The
// KIVI-style and AKVQ-style key instantiations keep 6 (4: 6 % slower).
constexpr int kDequantizeWavesMinMax = 4;
// The one-pass kernels: 4 (0.3-1 % faster than uncapped or 6 on the Qwen-,
// 72B- and LLaVA-NeXT-shaped caches, InternVL-shaped unchanged).
constexpr int kFakeQuantizeWaves = 4;

// Mask routing in kernel arguments: bit i of `mask` marks protected head
// i = l*H + h; `prefix[w]` counts protected heads in words before w, so the
// rank of i among protected heads is prefix[i/32] + popcount of the lower
// bits of word i/32 (§3: a base must be able to skip individual heads).
struct Route {
  uint32_t mask[kMaskWords];
  uint32_t prefix[kMaskWords];  // 32-bit so the kernels read it with scalar loads
};

// A tiled launch covers K (tensor 0) and V (tensor 1), or one of them: blocks
// [0, blocks_k) take K tiles, the rest V tiles.  Each block takes one
// (tensor, l, b, h) slice and one of its `tiles` runs of consecutive image
// tokens.  The host sets tiles for kBlockTokens (the key-norm pass uses
// them); each quantize, dequantize and one-pass launcher sets tiles and
// blocks_k for its kernel's tile size.
struct Params {
  const uint16_t* cache[2];  // quantize, fake quantize: K, V input; dequantize: K_out, V_out
  uint16_t* out[2];          // fake quantize: K_out, V_out (may equal the input)
  uint8_t* codes[2];
  uint32_t* meta[2];
  uint16_t* side[2];
  int32_t L, B, H, T;
  int32_t s0, n;             // image span
  int32_t keys_only;
  int32_t kivi_whole;        // KIVI keys: one range over the whole sequence (kivi_seq.hip)
  int32_t ngroups;           // KIVI key groups per slice
  int32_t tiles;             // workgroup tiles per slice
  int32_t n_unprot_k;        // heads (l, h) whose keys are quantized
  uint32_t blocks_k;         // blocks of tensor K
  // AKVQ-style token retention
  float* norm;               // [L][B][H][n] squared key norms
  int32_t* ret_idx;          // [L][B][H][k] retained tokens, ascending
  uint16_t* ret[2];          // [slot][B][k][D] retained rows of K, V
  int32_t k;                 // retained tokens per (l, b, h)
  // words the first workgroups of this launch set to zero (the exchange area
  // of the whole-sequence KIVI key kernel that follows in the same call)
  uint64_t* clear;
  uint32_t clear_words;
  // 1: blocks [0, blocks_k) take only the protected key slices (k-th
  // protected head, batch row, tile), so a launch that has nothing to do for
  // the other key slices starts no workgroup for them
  int32_t kept_keys = 0;
  Route route;
};

// Tensors a launch covers: K and V, or one of them.
// kKeptKeysAndValues: the protected key slices, listed compactly (see
// decode_launch_block), then every value slice.
enum class Tensors { kBoth, kKeys, kValues, kKeptKeysAndValues };

// Dispatch over (base, D, bits); return hipSuccess or the launch error.
// With `norms`, the quantize kernel also writes the squared key norms (AKVQ).
hipError_t launch_quantize(const Params& p, int base, int D, int bits, bool norms, hipStream_t stream);
hipError_t launch_dequantize(const Params& p, int base, int D, int bits, hipStream_t stream);
hipError_t launch_fake_quantize(const Params& p, int base, int D, int bits, bool norms, hipStream_t stream);
// KIVI keys over the whole sequence: a persistent grid over the quantized key
// slices; each slice is held on chip by a group of workgroups (each a run of
// its rows, every channel) that combine their partial ranges through the
// exchange workspace `ws` (kivi_workspace_bytes; unused with one workgroup
// per slice), or, for longer slices, a range launch over chunks of every
// slice merging into `ws` and a code launch (without `ws`: a range pass and a
// code pass per slice by one workgroup).
// `cleared`: the words kivi_seq_clear_words gives were set to zero by an
// earlier launch of the call (else the launch clears them itself).
hipError_t launch_kivi_seq(const Params& p, int D, int bits, bool fake, void* ws, bool cleared, hipStream_t stream);
hipError_t kivi_seq_clear_words(const Params& p, int D, int bits, bool fake, void* ws, uint32_t* words);
// Workgroups per slice of the resident kernel (0: the split kernels), and
// the exchange workspace bytes a call with T rows per slice needs (0: none).
int kivi_partners(int T, int D);
uint64_t kivi_workspace_bytes(int T, int D);
// Token retention: squared key norms of every image token (p.norm); the k
// largest per (l, b, h) into p.ret_idx; their rows gathered from p.cache into
// p.ret, written back from p.ret into p.out, or copied from p.cache straight
// into p.out.  The selection copies the rows it selects (kGather or
// kCacheToOut) in the same launch.
hipError_t launch_key_norms(const Params& p, int D, hipStream_t stream);
enum class RowCopy { kGather, kScatter, kCacheToOut };
hipError_t launch_retain_select(const Params& p, int D, RowCopy mode, hipStream_t stream);
hipError_t launch_retain_rows(const Params& p, int D, RowCopy mode, hipStream_t stream);

// Host side: the one-pass call (api.hip) with its token-retention workspace
// supplied by `get_ws(need, &ws)` after the host-side argument checks, only
// when the call needs one: the caller's buffer (checked like every other
// argument) or library memory (`caller` false).  get_ws returns HG_OK or an
// error status, with the detail recorded by set_error.
struct Workspace {
  void* ptr = nullptr;
  uint64_t bytes = 0;
  bool caller = true;
};
typedef std::function<int(uint64_t need, Workspace* ws)> WorkspaceFn;
int fake_quantize(const hg_config* cfg, const uint16_t* K, const uint16_t* V, const uint8_t* mask,
                  uint16_t* K_out, uint16_t* V_out, const WorkspaceFn& get_ws, hipStream_t stream);
int set_error(int status, const char* msg);

// Routing of one (tensor, slice): whether it is kept in BF16 and its slot in
// the packed buffers (rank among kept heads if kept, else among quantized
// heads).  Wave-uniform scalar work.
struct SliceRoute {
  int b;
  bool kept;
  uint32_t slot;
};

__device__ __forceinline__ SliceRoute route_slice(const Params& p, int X, uint32_t s) {
  SliceRoute r;
  const uint32_t h = s % (uint32_t)p.H;
  const uint32_t lb = s / (uint32_t)p.H;
  r.b = (int)(lb % (uint32_t)p.B);
  const uint32_t l = lb / (uint32_t)p.B;
  const uint32_t i = l * (uint32_t)p.H + h;
  const uint32_t w = p.route.mask[i >> 5];
  const bool masked = (w >> (i & 31u)) & 1u;
  const uint32_t rank = (uint32_t)p.route.prefix[i >> 5] +
                        (uint32_t)__builtin_popcount(w & ((1u << (i & 31u)) - 1u));
  r.kept = masked && (X == 0 || !p.keys_only);
  if (r.kept) {
    r.slot = rank;
  } else if (X == 1 && p.keys_only) {
    r.slot = i;  // K-only mode: every V head is quantized
  } else {
    r.slot = i - rank;
  }
  return r;
}

// The first kClearBlocks workgroups of a launch set the p.clear_words words
// at p.clear to zero (a share each), before anything else.
constexpr uint32_t kClearBlocks = 64;
__device__ __forceinline__ void clear_words_share(const Params& p) {
  if (p.clear_words == 0 || blockIdx.x >= kClearBlocks) return;
  const uint32_t nb = min(gridDim.x, kClearBlocks);
  for (uint32_t i = blockIdx.x * blockDim.x + threadIdx.x; i < p.clear_words; i += nb * blockDim.x) p.clear[i] = 0;
}

// Block decoding: tensor, slice, token tile and routing of a workgroup.
struct Slice {
  int X;            // 0 = K, 1 = V
  int tile;         // token tile within the slice
  uint32_t s;       // (l*B + b)*H + h
  int b;
  bool kept;
  uint32_t slot;
};

__device__ __forceinline__ Slice decode_block(const Params& p, uint32_t bid) {
  Slice r;
  r.X = bid >= p.blocks_k ? 1 : 0;
  const uint32_t rel = bid - (r.X ? p.blocks_k : 0u);
  r.tile = (int)(rel % (uint32_t)p.tiles);
  r.s = rel / (uint32_t)p.tiles;
  const SliceRoute sr = route_slice(p, r.X, r.s);
  r.b = sr.b;
  r.kept = sr.kept;
  r.slot = sr.slot;
  return r;
}

// (l*H + h) of the k-th protected head (k < the number of protected heads):
// the word holding it is the last one with at most k protected heads before
// it (prefix[w], non-decreasing in w), so the number of words with
// prefix[w] <= k, minus one; the lanes test 64 words at a time.
__device__ __forceinline__ uint32_t kth_protected_head(const Params& p, uint32_t k) {
  const uint32_t words = ((uint32_t)p.L * p.H + 31u) / 32u;
  const uint32_t lane = threadIdx.x & 63u;
  uint32_t count = 0;
#pragma unroll
  for (uint32_t w0 = 0; w0 < (uint32_t)kMaskWords; w0 += 64u) {
    if (w0 >= words) break;
    const uint32_t w = min(w0 + lane, words - 1u);
    const bool le = w0 + lane < words && p.route.prefix[w] <= k;
    count += (uint32_t)__popcll(__ballot(le));
  }
  const uint32_t lo = count - 1u;
  uint32_t ones = p.route.mask[lo];
  for (uint32_t j = k - p.route.prefix[lo]; j > 0; --j) ones &= ones - 1u;
  return 32u * lo + (uint32_t)__builtin_ctz(ones);
}

// A block of a launch: with kept_keys, blocks [0, blocks_k) are the protected
// key slices in (protected head, batch row, tile) order, and the rest are
// value slices as in decode_block.
__device__ __forceinline__ Slice decode_launch_block(const Params& p, uint32_t bid) {
  if (!p.kept_keys || bid >= p.blocks_k) return decode_block(p, bid);
  Slice r;
  r.X = 0;
  r.tile = (int)(bid % (uint32_t)p.tiles);
  const uint32_t q = bid / (uint32_t)p.tiles;
  r.b = (int)(q % (uint32_t)p.B);
  const uint32_t k = q / (uint32_t)p.B;
  const uint32_t i = kth_protected_head(p, k);
  const uint32_t l = i / (uint32_t)p.H, h = i % (uint32_t)p.H;
  r.s = (l * (uint32_t)p.B + (uint32_t)r.b) * (uint32_t)p.H + h;
  r.kept = true;
  r.slot = k;
  return r;
}

}  // namespace hg
