/*
 * HeadGuard CPU oracle -- TEST INFRASTRUCTURE ONLY.
 *
 * A plain, slow, scalar C implementation of the head-masked image-KV quantizer
 * (HeadGuard, arXiv 2609.35800, §3 "Applying protection" and §4 "Quantization
 * setup"), used only to check the HIP library.  Only the tests, the smoke entry
 * and the bench's CPU-baseline leg may load it.  It shares no code with the
 * HIP path and includes nothing from it.
 *
 * Arithmetic: IEEE-754 binary32, round-to-nearest-even, no FMA contraction,
 * no flush-to-zero, correctly rounded division (build with
 * -O2 -fno-fast-math -ffp-contract=off).  The paper leaves the precision open;
 * the quantizer's per-group math is defined in fp32 (see the readings listed
 * in the design notes).
 *
 * Layouts (all little-endian, all row-major):
 *   K, V          BF16 bits [L][B][H][T][D]
 *   codes_X       [slot][B][n][D*bits/8]   LSB-first bitstream per token row
 *   meta_X        u32 [slot][B][n]           per-token groups
 *                 u32 [slot][B][ceil(n/G)][D] KIVI-style keys, G = kivi_group
 *                 u32 [slot][B][1][D]         KIVI-style keys, kivi_group = 0
 *                                             (range over the whole sequence)
 *                 each word = bf16(scale) | bf16(min) << 16
 *   side_X        BF16 bits [p][B][n][D]     protected heads' image rows
 * AKVQ-style token retention (retain_permille > 0, §4):
 *   norm_k        fp32 [L][B][H][n]          squared norm of every image key
 *   ret_idx       int32 [L][B][H][k]         retained image tokens, ascending
 *   ret_X         BF16 bits [slot][B][k][D]  their rows, for quantized slots
 * where n = img_len, slot = rank of (l,h) among the heads whose tensor X is
 * quantized, p = rank of (l,h) among protected heads (row-major (l,h) order),
 * k = the retained count per head.
 */
#ifndef HG_ORACLE_H
#define HG_ORACLE_H
#include <stdint.h>
#include <stddef.h>

#ifdef __cplusplus
extern "C" {
#endif

enum { HGO_MINMAX = 0, HGO_KIVI = 1, HGO_AKVQ = 2 };

typedef struct {
  int32_t L, B, H, T, D;
  int32_t img_start, img_len;
  int32_t bits;
  int32_t base;
  int32_t keys_only;
  int32_t kivi_group;
  int32_t retain_permille; /* AKVQ-style retention, per mille of image tokens; 0 = off */
} hgo_config;

typedef struct {
  uint64_t codes_k, meta_k, side_k, codes_v, meta_v, side_v; /* bytes */
  uint64_t norm_k, ret_idx, ret_k, ret_v;                    /* bytes */
  int32_t n_protected, n_unprot_k, n_unprot_v;
  int32_t retain_count;
} hgo_sizes_t;

/* BF16 <-> fp32 helpers (exposed so the tests can pin them). */
float    hgo_bf16_to_f32(uint16_t h);
uint16_t hgo_bf16_rne(float x);
uint16_t hgo_bf16_rd(float x);
uint16_t hgo_bf16_ru(float x);

/* Min-max quantization of one group of m fp32 values read at v[i*stride]:
 * codes q[i*qstride] in [0, 2^bits-1], returns the metadata word. */
uint32_t hgo_quantize_group(const float* v, int m, int stride, int bits,
                            uint8_t* q, int qstride);
/* Reconstruction of one element in fp32: q*S + m. */
float hgo_level(uint32_t meta, unsigned q);

/* Normalized Walsh-Hadamard transform in place, fp32, D a power of two. */
void hgo_fwht_norm(float* a, int D);
/* Same butterflies without the final 1/sqrt(D) scale. */
void hgo_fwht_raw(float* a, int D);
float hgo_fwht_scale(int D);

/* Routing of (tensor X in {0:K,1:V}, layer l, head h): *is_protected and the
 * slot index into the matching buffer.  Returns 0, or -1 on a bad argument. */
int hgo_route(const hgo_config* c, const uint8_t* mask, int X, int l, int h,
              int* is_protected, int* slot);

int hgo_sizes(const hgo_config* c, const uint8_t* mask, hgo_sizes_t* out);

/* One unprotected slice: rows = the n image rows (n*D BF16) of one (l,b,h).
 * codes receives n*D*bits/8 bytes, meta n words (or ceil(n/G)*D words for
 * KIVI-style keys). */
int hgo_quantize_slice(const hgo_config* c, int X, const uint16_t* rows,
                       uint8_t* codes, uint32_t* meta);
/* The same from the whole slice (T*D BF16, text rows included), as needed by
 * KIVI-style keys with kivi_group == 0: one range per channel over all T
 * tokens, meta D words, codes for the n image tokens only. */
int hgo_quantize_slice_seq(const hgo_config* c, int X, const uint16_t* slice,
                           uint8_t* codes, uint32_t* meta);
int hgo_dequantize_slice(const hgo_config* c, int X, const uint8_t* codes,
                         const uint32_t* meta, uint16_t* rows_out);

/* Whole cache.  Buffers are host memory sized by hgo_sizes; unused ones
 * (side_v with keys_only) may be NULL.  Dequant writes only the image rows of
 * K_out / V_out.  threads >= 1 splits the slices over POSIX threads. */
int hgo_quantize(const hgo_config* c, const uint16_t* K, const uint16_t* V,
                 const uint8_t* mask,
                 uint8_t* codes_k, uint32_t* meta_k, uint16_t* side_k,
                 uint8_t* codes_v, uint32_t* meta_v, uint16_t* side_v,
                 int threads);
int hgo_dequantize(const hgo_config* c, const uint8_t* mask,
                   const uint8_t* codes_k, const uint32_t* meta_k,
                   const uint16_t* side_k,
                   const uint8_t* codes_v, const uint32_t* meta_v,
                   const uint16_t* side_v,
                   uint16_t* K_out, uint16_t* V_out, int threads);

/* AKVQ-style token retention (§4 Quantization setup): in every KV head the
 * keys and values of the k image tokens whose keys have the largest norms stay
 * in BF16, with or without head protection. */
/* k = round(n * retain_permille / 1000), halves rounded up. */
int hgo_retain_count(const hgo_config* c);
/* Squared L2 norm of one BF16 key of D (a power of two) entries in fp32:
 * squares, then pairwise sums over adjacent blocks of 1, 2, 4, ... entries. */
float hgo_key_sqnorm(const uint16_t* key, int D);
/* The k largest of n values (lower index first among equals), written to
 * idx[k] in ascending index order. */
int hgo_retain_select(const float* sqnorm, int n, int k, int32_t* idx);
/* Whole cache: norm_k, ret_idx and the retained rows of the quantized slots
 * (layouts above).  ret_k / ret_v may be NULL when they hold no slot. */
int hgo_retain(const hgo_config* c, const uint16_t* K, const uint16_t* V,
               const uint8_t* mask, float* norm_k, int32_t* ret_idx,
               uint16_t* ret_k, uint16_t* ret_v, int threads);
/* After hgo_dequantize: the retained rows of the quantized slots are written
 * back bit-identical into K_out / V_out. */
int hgo_restore_retained(const hgo_config* c, const uint8_t* mask,
                         const int32_t* ret_idx, const uint16_t* ret_k,
                         const uint16_t* ret_v, uint16_t* K_out, uint16_t* V_out);

/* Head selection (§3 Eq. 2): g, o are per-query-head scores [L][Hq] (fp64);
 * query head hq belongs to KV head hq / (Hq/Hkv).  Writes mask[L*Hkv] with
 * the K heads of largest s = z(mean g) + z(mean o) set (ties: lower index).
 * Returns 0, or -1 on a bad argument. */
int hgo_select_heads(const double* g, const double* o, int L, int Hq, int Hkv, int K,
                     uint8_t* mask);

#ifdef __cplusplus
}
#endif
#endif
