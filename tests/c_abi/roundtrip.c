/*
 * The C ABI of libheadguard used from plain C (no C++, no Python): a small
 * cache is quantized, dequantized and quantized-and-reconstructed in one pass
 * through include/headguard.h, and the results are checked for what holds
 * without an oracle: every call succeeds; protected image rows come back
 * bit-identical and text rows are never written (§3 Applying protection); the
 * one-pass form writes the same bytes as quantize then dequantize (§4
 * Quantization setup); a second call writes the same bytes; and a bad
 * configuration is refused with its status and a detail message, before any
 * device work.  Prints "ok" and exits 0 on success.
 */
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "headguard.h"

#define CHECK_HIP(x)                                                     \
  do {                                                                   \
    hipError_t e_ = (x);                                                 \
    if (e_ != hipSuccess) {                                              \
      fprintf(stderr, "%s:%d: HIP error %d\n", __FILE__, __LINE__, e_);  \
      return 2;                                                          \
    }                                                                    \
  } while (0)

#define CHECK_HG(x)                                                                    \
  do {                                                                                 \
    int s_ = (x);                                                                      \
    if (s_ != HG_OK) {                                                                 \
      fprintf(stderr, "%s:%d: %s: %s\n", __FILE__, __LINE__, hg_status_string(s_),     \
              hg_last_error());                                                        \
      return 3;                                                                        \
    }                                                                                  \
  } while (0)

enum { L = 2, B = 2, H = 4, T = 48, D = 64, S0 = 5, N = 37 };
static const uint16_t kSentinel = 0x7FBF;

/* BF16 bit patterns of a simple seeded sequence: sign, exponent near 1, mantissa */
static uint16_t next_bf16(uint32_t* state) {
  *state = *state * 1664525u + 1013904223u;
  uint32_t r = *state >> 8;
  return (uint16_t)(((r & 1u) << 15) | ((123u + (r >> 1) % 8u) << 7) | ((r >> 4) & 0x7Fu));
}

int main(void) {
  const size_t elems = (size_t)L * B * H * T * D, bytes = elems * 2;
  hg_config cfg = {L, B, H, T, D, S0, N, 2, HG_BASE_AKVQ, 0, 32, 0};
  uint8_t mask[L * H] = {0};
  mask[1] = 1;
  mask[6] = 1;

  /* a bad bit width is refused before any device work */
  hg_config bad = cfg;
  bad.bits = 7;
  hg_sizes z;
  if (hg_packed_sizes(&bad, mask, &z) != HG_ERR_BITS || strlen(hg_last_error()) == 0) {
    fprintf(stderr, "bad config not refused\n");
    return 4;
  }
  CHECK_HG(hg_packed_sizes(&cfg, mask, &z));

  uint16_t* hK = malloc(bytes);
  uint16_t* hV = malloc(bytes);
  uint16_t* hKo = malloc(bytes);
  uint16_t* hVo = malloc(bytes);
  uint16_t* hKf = malloc(bytes);
  uint16_t* hVf = malloc(bytes);
  if (!hK || !hV || !hKo || !hVo || !hKf || !hVf) return 5;
  uint32_t state = 12345u;
  for (size_t i = 0; i < elems; ++i) hK[i] = next_bf16(&state);
  for (size_t i = 0; i < elems; ++i) hV[i] = next_bf16(&state);
  for (size_t i = 0; i < elems; ++i) hKo[i] = hVo[i] = kSentinel;

  uint16_t *K, *V, *Ko, *Vo, *Kf, *Vf;
  CHECK_HIP(hipMalloc((void**)&K, bytes));
  CHECK_HIP(hipMalloc((void**)&V, bytes));
  CHECK_HIP(hipMalloc((void**)&Ko, bytes));
  CHECK_HIP(hipMalloc((void**)&Vo, bytes));
  CHECK_HIP(hipMalloc((void**)&Kf, bytes));
  CHECK_HIP(hipMalloc((void**)&Vf, bytes));
  CHECK_HIP(hipMemcpy(K, hK, bytes, hipMemcpyHostToDevice));
  CHECK_HIP(hipMemcpy(V, hV, bytes, hipMemcpyHostToDevice));
  CHECK_HIP(hipMemcpy(Ko, hKo, bytes, hipMemcpyHostToDevice));
  CHECK_HIP(hipMemcpy(Vo, hVo, bytes, hipMemcpyHostToDevice));
  CHECK_HIP(hipMemcpy(Kf, hKo, bytes, hipMemcpyHostToDevice));
  CHECK_HIP(hipMemcpy(Vf, hVo, bytes, hipMemcpyHostToDevice));

  /* every packed buffer, 16-byte aligned device memory (hipMalloc is) */
  hg_packed pk;
  void** slots[] = {&pk.codes_k, &pk.meta_k, &pk.side_k, &pk.codes_v, &pk.meta_v,
                    &pk.side_v, &pk.norm_k, &pk.ret_idx, &pk.ret_k, &pk.ret_v};
  const uint64_t sizes[] = {z.codes_k, z.meta_k, z.side_k, z.codes_v, z.meta_v,
                            z.side_v, z.norm_k, z.ret_idx, z.ret_k, z.ret_v};
  for (int i = 0; i < 10; ++i) {
    *slots[i] = NULL;
    if (sizes[i]) CHECK_HIP(hipMalloc(slots[i], sizes[i]));
  }
  uint8_t* codes1 = malloc(z.codes_k ? z.codes_k : 1);
  uint8_t* codes2 = malloc(z.codes_k ? z.codes_k : 1);
  if (!codes1 || !codes2) return 5;

  hipStream_t stream;
  CHECK_HIP(hipStreamCreate(&stream));
  CHECK_HG(hg_quantize(&cfg, K, V, mask, &pk, stream));
  CHECK_HIP(hipStreamSynchronize(stream));
  CHECK_HIP(hipMemcpy(codes1, pk.codes_k, z.codes_k, hipMemcpyDeviceToHost));
  CHECK_HG(hg_quantize(&cfg, K, V, mask, &pk, stream));
  CHECK_HG(hg_dequantize(&cfg, mask, &pk, Ko, Vo, stream));
  CHECK_HG(hg_fake_quantize(&cfg, K, V, mask, Kf, Vf, NULL, 0, stream));
  CHECK_HIP(hipStreamSynchronize(stream));
  CHECK_HIP(hipMemcpy(codes2, pk.codes_k, z.codes_k, hipMemcpyDeviceToHost));
  CHECK_HIP(hipMemcpy(hKo, Ko, bytes, hipMemcpyDeviceToHost));
  CHECK_HIP(hipMemcpy(hVo, Vo, bytes, hipMemcpyDeviceToHost));
  CHECK_HIP(hipMemcpy(hKf, Kf, bytes, hipMemcpyDeviceToHost));
  CHECK_HIP(hipMemcpy(hVf, Vf, bytes, hipMemcpyDeviceToHost));

  int failures = 0;
  if (memcmp(codes1, codes2, z.codes_k) != 0) {
    fprintf(stderr, "second quantize wrote different codes\n");
    ++failures;
  }
  if (memcmp(hKo, hKf, bytes) != 0 || memcmp(hVo, hVf, bytes) != 0) {
    fprintf(stderr, "one-pass result differs from quantize then dequantize\n");
    ++failures;
  }
  size_t changed = 0;
  for (int l = 0; l < L; ++l)
    for (int b = 0; b < B; ++b)
      for (int h = 0; h < H; ++h)
        for (int t = 0; t < T; ++t)
          for (int d = 0; d < D; ++d) {
            const size_t i = ((((size_t)l * B + b) * H + h) * T + t) * D + d;
            const int image = t >= S0 && t < S0 + N;
            if (!image) {
              if (hKo[i] != kSentinel || hVo[i] != kSentinel) ++failures;
            } else if (mask[l * H + h]) {
              if (hKo[i] != hK[i] || hVo[i] != hV[i]) ++failures;
            } else {
              changed += (hKo[i] != hK[i]) + (hVo[i] != hV[i]);
            }
          }
  if (changed == 0) {
    fprintf(stderr, "2-bit reconstruction left every unprotected entry unchanged\n");
    ++failures;
  }

  for (int i = 0; i < 10; ++i)
    if (*slots[i]) CHECK_HIP(hipFree(*slots[i]));
  CHECK_HIP(hipFree(K));
  CHECK_HIP(hipFree(V));
  CHECK_HIP(hipFree(Ko));
  CHECK_HIP(hipFree(Vo));
  CHECK_HIP(hipFree(Kf));
  CHECK_HIP(hipFree(Vf));
  CHECK_HIP(hipStreamDestroy(stream));
  free(hK), free(hV), free(hKo), free(hVo), free(hKf), free(hVf), free(codes1), free(codes2);
  if (failures) {
    fprintf(stderr, "%d check(s) failed\n", failures);
    return 1;
  }
  printf("ok\n");
  return 0;
}
