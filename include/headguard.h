/*
 * headguard.h -- C ABI of libheadguard, the MI355X (gfx950) head-masked
 * low-bit image-KV quantizer of HeadGuard (arXiv 2609.35800).
 *
 * The operation (§3 "HeadGuard" and "Applying protection"; §4 "Quantization
 * setup"): given a model's KV cache, the positions of its image tokens, a fixed
 * protection mask over physical KV heads and a base quantizer, every image-token
 * key/value vector of an unprotected head is quantized by the base to b bits;
 * the protected heads keep their image keys (and values, in K+V mode) in BF16;
 * text KV is left alone.  A compatible base must be able to skip individual
 * heads (§3), which is what the mask routing does.
 *
 * Bases (§2 "KV-cache quantization", §4 "Quantization setup"):
 *   HG_BASE_MINMAX  per-token min-max round-to-nearest for keys and values;
 *   HG_BASE_KIVI    keys per channel over groups of `kivi_group` (32)
 *                   consecutive image tokens, or with kivi_group = 0 over the
 *                   whole supplied sequence of T tokens, text included (the
 *                   paper's KIVI-style harness; text still stays BF16);
 *                   values per token;
 *   HG_BASE_AKVQ    keys rotated by the normalized Walsh-Hadamard matrix over
 *                   head_dim, then per token; values per token, unrotated;
 *                   optionally (retain_permille > 0) the keys and values of
 *                   the image tokens with the largest key norms stay in BF16
 *                   in every head (§4: a nominal 2 %, retain_permille = 20).
 *
 * Quantizer of one group of values v (a token vector, or one channel of a
 * KIVI key group), all in IEEE fp32 with round-to-nearest-even:
 *   m = BF16 rounded toward -inf of min(v)     (a zero is stored as +0)
 *   s = (max(v) - m) / (2^b - 1)               (correctly rounded)
 *   S = BF16 rounded toward +inf of s          (+0 if zero; at least 2^-126)
 *   q = clamp(rint((v - m) * (1/S)), 0, 2^b-1) (rint ties to even; q = 0 if S = 0)
 *   metadata word = bits(S) | bits(m) << 16    (32 bits per group, §5.4)
 * Reconstruction: x^ = bf16_rne(q*S + m); for AKVQ keys the fp32 values
 * q*S + m are rotated back (the transform is its own inverse) before the BF16
 * rounding.  The rotation is the fast transform in fp32, butterfly spans
 * 1, 2, ..., D/2, then one multiply by fp32(1/sqrt(D)).
 *
 * Layouts (little-endian, row-major, n = img_len):
 *   K, V      BF16 [L][B][H][T][D], contiguous
 *   codes_X   [slot][B][n][D*bits/8]  token-major, code of channel d at bits
 *             [bits*d, bits*d + bits) of the token's row, least significant first
 *   meta_X    u32 [slot][B][n]                 per-token groups
 *             u32 [slot][B][ceil(n/G)][D]      KIVI keys, G = kivi_group
 *             u32 [slot][B][1][D]              KIVI keys, kivi_group = 0
 *   side_X    BF16 [p][B][n][D]  image rows of protected heads, bit-identical
 * slot = rank of (l, h) in row-major order among the heads whose X is
 * quantized; p = rank among the heads whose X is kept in BF16.  V is kept iff
 * the head is protected and keys_only == 0.
 *
 * Token retention (AKVQ, retain_permille > 0; §4 Quantization setup).  Per
 * (l, b, h), k = round(n * retain_permille / 1000) (halves up) image tokens
 * are retained: those whose keys, as stored (before the rotation), have the
 * largest squared norm, computed in fp32 as the squares summed pairwise over
 * adjacent blocks of 1, 2, 4, ... channels; equal norms go to the lower
 * token.  Every token is still quantized; a retained token's BF16 row
 * replaces its reconstruction, for each tensor the head does not keep:
 *   norm_k    fp32 [L][B][H][n]      squared key norm of every image token
 *   ret_idx   int32 [L][B][H][k]     retained tokens (0-based in the span), ascending
 *   ret_X     BF16 [slot][B][k][D]   their rows, for the quantized slots of X
 *
 * Ownership and synchronisation: the caller allocates every buffer, the
 * one-pass call's workspace included.  Device buffers are device memory of
 * the current HIP device; the mask is host memory read during the call only.
 * The library allocates no memory, keeps no state between calls and never
 * synchronises: HG_OK means the work is enqueued on `stream`; device faults
 * surface at the caller's next synchronisation.  The calls only launch
 * kernels on `stream`, so they can be captured in a HIP graph.  Every
 * argument check runs before any launch, so on an argument error no output is
 * touched.  A launch error (HG_ERR_HIP) at the call's first kernel leaves
 * every output untouched too; at a later kernel of the same call, the
 * kernels before it are enqueued and may write their outputs.  Calls are
 * thread-safe; the error detail is per thread.
 *
 * KIVI keys over the whole sequence (kivi_group = 0): when a key slice is
 * longer than one workgroup holds on chip, several co-resident workgroups
 * hold it together and exchange partial ranges through the caller's
 * workspace, waiting for one another (a bounded number of polls); past 32
 * workgroups' rows, chunks of each slice merge their ranges into the same
 * workspace with atomics and a second launch writes the codes.  The
 * kernel is sized to be resident on an otherwise idle device: a kernel
 * running concurrently on another stream can delay it, and one that keeps
 * compute units busy long enough makes waits run out (the workspace's first
 * word then counts them and the codes of the slices affected are wrong).
 *
 * Every buffer a call writes must be disjoint from every other buffer of the
 * call (HG_ERR_POINTER, checked on the host from the pointers and the sizes
 * hg_packed_sizes reports).  Preconditions not checked: inputs finite with
 * |x| < 2^96 (so every range and rotated value, at most sqrt(D) |x|, keeps its
 * scale below 2^101); buffers at least the sizes hg_packed_sizes reports.
 */
#ifndef HEADGUARD_H
#define HEADGUARD_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum { HG_BASE_MINMAX = 0, HG_BASE_KIVI = 1, HG_BASE_AKVQ = 2 } hg_base;

enum {
  HG_OK = 0,
  HG_ERR_NULL = 1,      /* a required pointer is NULL                          */
  HG_ERR_SHAPE = 2,     /* L, B, H, T not positive, L*H > HG_MAX_HEADS,
                           keys_only not 0 or 1, (quantize, dequantize,
                           one-pass) 2*L*B*H*ceil(img_len/64) > 2^31 - 1
                           workgroups, a workspace too small, or a head
                           budget fraction out of range                      */
  HG_ERR_SPAN = 3,      /* image span outside [0, T]                           */
  HG_ERR_BITS = 4,      /* bits not in {2, 3, 4}                               */
  HG_ERR_BASE = 5,      /* unknown base, kivi_group not 32 or 0, retain_permille
                           outside [0, 1000] or set with a base other than AKVQ */
  HG_ERR_HEADDIM = 6,   /* D not in {64, 128, 256}                             */
  HG_ERR_ALIGN = 7,     /* a device pointer is not 16-byte aligned (the
                           one-pass workspace: 256-byte)                     */
  HG_ERR_MASK = 8,      /* a mask entry is neither 0 nor 1                     */
  HG_ERR_NO_DEVICE = 9, /* no usable HIP device                                */
  HG_ERR_HIP = 10,      /* the HIP runtime reported an error (launch, pointer) */
  HG_ERR_POINTER = 11,  /* a buffer argument is not device memory              */
  HG_ERR_VALUE = 12     /* a head score is not finite                          */
};

/* Largest L*H the mask routing holds in kernel arguments. */
#define HG_MAX_HEADS 8192

typedef struct {
  int32_t L, B, H, T, D;       /* cache shape [L][B][H][T][D]                      */
  int32_t img_start, img_len;  /* image span [img_start, img_start + img_len),
                                  shared by every batch row; img_len may be 0      */
  int32_t bits;                /* 2, 3 or 4                                        */
  int32_t base;                /* hg_base                                          */
  int32_t keys_only;           /* 1: protect K only; 0: protect K and V            */
  int32_t kivi_group;          /* KIVI key group: 32 tokens, or 0 = whole sequence */
  int32_t retain_permille;     /* AKVQ token retention per mille (20 = 2 %), 0 = off */
} hg_config;

typedef struct {
  uint64_t codes_k, meta_k, side_k, codes_v, meta_v, side_v; /* bytes          */
  uint64_t norm_k, ret_idx, ret_k, ret_v;  /* bytes; 0 without token retention    */
  uint64_t workspace;          /* bytes of hg_quantize's workspace: the exchange
                                  area of KIVI keys over the whole sequence when
                                  a slice is longer than one workgroup holds
                                  (3072 / 1536 / 768 rows at D = 64 / 128 /
                                  256) and some key is quantized; else 0      */
  uint64_t fake_workspace;     /* bytes of hg_fake_quantize's workspace: the key
                                  norms, token lists and (in place) saved rows
                                  of token retention, or the same exchange area
                                  as `workspace`; else 0                        */
  int32_t n_protected;         /* heads with mask = 1                             */
  int32_t n_unprot_k, n_unprot_v; /* heads whose K / V are quantized              */
  int32_t retain_count;        /* k, retained tokens per (l, b, h)                */
} hg_sizes;

typedef struct {
  void *codes_k, *meta_k, *side_k, *codes_v, *meta_v, *side_v; /* device */
  void *norm_k, *ret_idx, *ret_k, *ret_v;                      /* device */
  void *workspace;  /* device, hg_sizes.workspace bytes, 256-byte aligned;
                       scratch for hg_quantize (contents on entry do not
                       matter; after the call its first 8 bytes count waits
                       that ran out of polls, 0 normally); unused by
                       hg_dequantize; may be NULL when its size is 0     */
} hg_packed;

/* Byte sizes of the packed buffers (the storage model of §5.4).  Pure
 * host computation; needs no device.  `protect_mask` is host uint8 [L*H],
 * row-major (l, h), entries 0 or 1. */
int hg_packed_sizes(const hg_config* cfg, const uint8_t* protect_mask, hg_sizes* out);

/* Quantize and pack the image KV of the whole cache (§3, §4).
 * K, V: device BF16 bit patterns, layout above.  `out` buffers: device memory
 * of at least the hg_packed_sizes sizes; a buffer whose size is 0 may be NULL.
 * Every device pointer must be 16-byte aligned (torch allocations are). */
int hg_quantize(const hg_config* cfg, const uint16_t* K, const uint16_t* V,
                const uint8_t* protect_mask, const hg_packed* out, hipStream_t stream);

/* Reconstruct the image rows of K_out, V_out (device BF16, same layout and
 * shape as K, V) from the packed buffers (simulated quantization's
 * reconstruction, §4).  Protected rows are copied back from the side store,
 * retained rows from ret_k / ret_v; text rows of K_out, V_out are not
 * written.  norm_k is not read. */
int hg_dequantize(const hg_config* cfg, const uint8_t* protect_mask, const hg_packed* in,
                  uint16_t* K_out, uint16_t* V_out, hipStream_t stream);

/* Head selection (§3 "Selecting physical KV heads", Eq. 2): the protection
 * mask from offline sensitivity scores.  g and o are host fp64 arrays
 * [L][Hq] of per-query-head image- and output-sensitivity scores (Eq. 1);
 * query heads h*(Hq/Hkv) .. h*(Hq/Hkv) + Hq/Hkv - 1 share KV head h.  Each
 * KV head's scores are the means over its query heads; each score is
 * standardized over all L*Hkv KV heads (population deviation; a constant
 * score gives 0); s = z(g) + z(o); the K heads with the largest s are marked
 * in mask_out (host uint8 [L*Hkv], row-major (l, h)), ties to the lower index.
 * The paper's main budget is K = round(L*Hkv/8).  Pure host computation. */
int hg_select_heads(const double* g, const double* o, int32_t L, int32_t Hq, int32_t Hkv,
                    int32_t K, uint8_t* mask_out);

/* Simulated quantization in one pass (§4 Quantization setup: low-precision
 * entries are rounded to the base's levels and reconstructed as floating-point
 * values): writes to the image rows of K_out, V_out exactly what hg_quantize
 * followed by hg_dequantize would, without packed buffers.  K_out may be K
 * (in place) and V_out may be V; otherwise an output must not overlap its
 * input, and no output may overlap the other tensor's input or the other
 * output (HG_ERR_POINTER, checked before any device work).  Kept
 * rows are copied (left alone in place); text rows are not written.  Device
 * pointers 16-byte aligned.
 * `workspace`: device memory of `workspace_bytes` bytes, 256-byte aligned,
 * owned by the caller, disjoint from K, V, K_out and V_out; with token
 * retention it holds the key norms, the retained token lists and, in place,
 * the saved retained rows, and must be at least hg_sizes.fake_workspace
 * bytes (out of place it needs only the norms and lists, about 4n + 4k bytes
 * per (l, b, h)); with KIVI keys over the whole sequence it is the exchange
 * area described above (hg_sizes.fake_workspace = hg_sizes.workspace); its
 * contents on entry do not matter and are overwritten.  When
 * hg_sizes.fake_workspace is 0 it is not used and may be NULL.  Errors: HG_ERR_NULL if it
 * is NULL but needed, HG_ERR_SHAPE if workspace_bytes is too small,
 * HG_ERR_ALIGN, HG_ERR_POINTER (overlap, or not device memory). */
int hg_fake_quantize(const hg_config* cfg, const uint16_t* K, const uint16_t* V,
                     const uint8_t* protect_mask, uint16_t* K_out, uint16_t* V_out,
                     void* workspace, uint64_t workspace_bytes, hipStream_t stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, serving loops, harnesses that forbid allocation): hg_fake_quantize
 * with its workspace (token retention's lists, or the whole-sequence KIVI key
 * exchange area) taken from a device array inside the
 * library, HG_NOALLOC_SCRATCH_BYTES per GPU, held until the process ends,
 * instead of a caller buffer.  Same arguments, results and errors as
 * hg_fake_quantize otherwise; a call whose workspace would exceed the array
 * (hg_sizes.fake_workspace in place, about 4n + 4k bytes per (l, b, h) out of
 * place) returns HG_ERR_SHAPE before any device work.  Allocates nothing.
 * Every call on one GPU shares that GPU's array: calls that overlap in time on
 * one GPU (on other streams or host threads) race on it and must be
 * serialized by the caller; nothing in it needs clearing between calls. */
#define HG_NOALLOC_SCRATCH_BYTES (96u << 20)
int hg_fake_quantize_noalloc(const hg_config* cfg, const uint16_t* K, const uint16_t* V,
                             const uint8_t* protect_mask, uint16_t* K_out, uint16_t* V_out,
                             hipStream_t stream);

/* Head budget (§3, "Selecting physical KV heads"): K = round(n_kv_heads *
 * num / den), halves rounded up, in exact integer arithmetic; the paper's
 * main budget is 1/8 of the physical KV heads, its sweeps 1/16 to 1/4.
 * Requires n_kv_heads >= 1, den >= 1 and 0 <= num <= den (else
 * HG_ERR_SHAPE); writes K to *K_out.  Pure host computation. */
int hg_head_budget(int32_t n_kv_heads, int32_t num, int32_t den, int32_t* K_out);

/* Static name of a status code. */
const char* hg_status_string(int status);

/* Detail of the last non-OK status returned on the calling thread ("" if none). */
const char* hg_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* HEADGUARD_H */
