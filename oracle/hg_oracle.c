/*
 * HeadGuard CPU oracle -- TEST INFRASTRUCTURE ONLY (see hg_oracle.h).
 *
 * Plain scalar loops, one step per line of the method, in the order the paper
 * describes it:
 *   - per-token min-max: each token's range is its own minimum and maximum and
 *     every entry rounds to the nearest of the 2^b evenly spaced levels
 *     (§1, first paragraph; §4 "Quantization setup");
 *   - KIVI-style: keys per channel, values per token (§2 "KV-cache
 *     quantization"; §4);
 *   - AKVQ-style: Hadamard rotation of the keys, then per-token (§2; §4);
 *   - protection: selected heads keep their image keys (and values in K+V
 *     mode) in BF16, text KV is never touched (§3 "Applying protection");
 *   - 32 bits of metadata per quantized vector (§5.4, storage estimate).
 * Where the paper is silent the readings are the ones stated in the header
 * comment of each function.
 *
 * Build: gcc -O2 -fno-fast-math -ffp-contract=off -fPIC -shared -pthread
 */
#include "hg_oracle.h"

#include <math.h>
#include <pthread.h>
#include <stdlib.h>
#include <string.h>

/* ------------------------------------------------------------------ BF16 */

static uint32_t f2u(float x) { uint32_t u; memcpy(&u, &x, 4); return u; }
static float u2f(uint32_t u) { float x; memcpy(&x, &u, 4); return x; }

float hgo_bf16_to_f32(uint16_t h) { return u2f((uint32_t)h << 16); }

/* Round to nearest, ties to even, on the fp32 bit pattern (finite inputs). */
uint16_t hgo_bf16_rne(float x) {
  uint32_t u = f2u(x);
  uint32_t hi = u >> 16, lo = u & 0xFFFFu;
  if (lo > 0x8000u || (lo == 0x8000u && (hi & 1u))) hi += 1; /* magnitude up */
  return (uint16_t)hi;
}

/* Round toward -infinity: drop the low half, then for a negative value with
 * a nonzero dropped part step one BF16 unit further from zero. */
uint16_t hgo_bf16_rd(float x) {
  uint32_t u = f2u(x);
  uint32_t hi = u >> 16, lo = u & 0xFFFFu;
  if (lo != 0 && (u >> 31)) hi += 1;
  return (uint16_t)hi;
}

/* Round toward +infinity: the mirror of hgo_bf16_rd. */
uint16_t hgo_bf16_ru(float x) {
  uint32_t u = f2u(x);
  uint32_t hi = u >> 16, lo = u & 0xFFFFu;
  if (lo != 0 && !(u >> 31)) hi += 1;
  return (uint16_t)hi;
}

/* ------------------------------------------------------- the base quantizer
 *
 * Readings (the paper fixes none of these):
 *  - levels: 2^b values m + k*S, k = 0..2^b-1, spanning the group's range;
 *  - metadata: min stored as BF16 rounded down, scale as BF16 rounded up, so
 *    the stored grid still covers [min, max]; 16 + 16 = 32 bits per group;
 *    a zero of either sign is stored as +0;
 *  - a positive scale below 2^-126 is raised to 2^-126 so 1/S is finite;
 *  - zero range (S == 0): every code is 0 and the group reconstructs to m;
 *  - code = clamp(rint((v - m) * (1/S)), 0, 2^b-1), rint ties to even, with
 *    one correctly rounded reciprocal per group and no fused multiply-add.
 */
uint32_t hgo_quantize_group(const float* v, int m, int stride, int bits,
                            uint8_t* q, int qstride) {
  float mn = v[0], mx = v[0];
  for (int i = 1; i < m; ++i) {
    float x = v[(size_t)i * stride];
    if (x < mn) mn = x;
    if (x > mx) mx = x;
  }
  uint16_t m16 = hgo_bf16_rd(mn);
  if (m16 == 0x8000u) m16 = 0;
  float mf = hgo_bf16_to_f32(m16);

  int levels = (1 << bits) - 1;
  float s = (mx - mf) / (float)levels;
  uint16_t s16 = hgo_bf16_ru(s);
  if (s16 == 0x8000u) s16 = 0;
  if (s16 != 0 && hgo_bf16_to_f32(s16) < 0x1p-126f) s16 = 0x0080u; /* 2^-126 */
  float S = hgo_bf16_to_f32(s16);

  if (s16 == 0) {
    for (int i = 0; i < m; ++i) q[(size_t)i * qstride] = 0;
  } else {
    float inv = 1.0f / S;
    for (int i = 0; i < m; ++i) {
      float t = (v[(size_t)i * stride] - mf) * inv;
      float r = rintf(t);
      if (r < 0.0f) r = 0.0f;
      if (r > (float)levels) r = (float)levels;
      q[(size_t)i * qstride] = (uint8_t)(unsigned)r;
    }
  }
  return (uint32_t)s16 | ((uint32_t)m16 << 16);
}

float hgo_level(uint32_t meta, unsigned q) {
  float S = hgo_bf16_to_f32((uint16_t)(meta & 0xFFFFu));
  float m = hgo_bf16_to_f32((uint16_t)(meta >> 16));
  float p = (float)q * S; /* exact: q < 2^8, S has 8 significant bits */
  return p + m;
}

/* ------------------------------------------------- Walsh-Hadamard rotation
 *
 * Reading: the rotation is the normalized Walsh-Hadamard matrix in natural
 * (Sylvester) order, H[i][j] = (-1)^popcount(i & j) / sqrt(D), applied as the
 * fast transform in fp32 with butterfly spans 1, 2, 4, ..., D/2 (each
 * butterfly rounds once), followed by one multiply by fp32(1/sqrt(D)).
 */
void hgo_fwht_raw(float* a, int D) {
  for (int h = 1; h < D; h *= 2) {
    for (int i = 0; i < D; i += 2 * h) {
      for (int j = i; j < i + h; ++j) {
        float p = a[j], q = a[j + h];
        a[j] = p + q;
        a[j + h] = p - q;
      }
    }
  }
}

float hgo_fwht_scale(int D) { return (float)(1.0 / sqrt((double)D)); }

void hgo_fwht_norm(float* a, int D) {
  hgo_fwht_raw(a, D);
  float c = hgo_fwht_scale(D);
  for (int j = 0; j < D; ++j) a[j] = a[j] * c;
}

/* ------------------------------------------------------------------ routing */

static int cfg_ok(const hgo_config* c) {
  if (!c) return 0;
  if (c->L <= 0 || c->B <= 0 || c->H <= 0 || c->T <= 0 || c->D <= 0) return 0;
  if (c->img_start < 0 || c->img_len < 0 || c->img_start + c->img_len > c->T) return 0;
  if (c->bits < 1 || c->bits > 8) return 0;
  if ((c->D * c->bits) % 8 != 0) return 0;
  if (c->base < HGO_MINMAX || c->base > HGO_AKVQ) return 0;
  if (c->base == HGO_KIVI && c->kivi_group < 0) return 0;
  if (c->base == HGO_AKVQ && (c->D & (c->D - 1)) != 0) return 0;
  if (c->retain_permille < 0 || c->retain_permille > 1000) return 0;
  if (c->retain_permille > 0 && c->base != HGO_AKVQ) return 0;
  return 1;
}

/* Protection (§3): K of a selected head is kept; V of a selected head is kept
 * only in K+V mode.  Slots are ranks in row-major (l, h) order. */
static int is_kept(const hgo_config* c, const uint8_t* mask, int X, int i) {
  if (!mask[i]) return 0;
  return X == 0 ? 1 : !c->keys_only;
}

int hgo_route(const hgo_config* c, const uint8_t* mask, int X, int l, int h,
              int* is_protected, int* slot) {
  if (!cfg_ok(c) || !mask || X < 0 || X > 1 || l < 0 || l >= c->L || h < 0 || h >= c->H)
    return -1;
  int i = l * c->H + h;
  int kept = is_kept(c, mask, X, i);
  int rank = 0;
  for (int j = 0; j < i; ++j)
    if (is_kept(c, mask, X, j) == kept) rank++;
  *is_protected = kept;
  *slot = rank;
  return 0;
}

static int kivi_keys(const hgo_config* c, int X) { return c->base == HGO_KIVI && X == 0; }

/* KIVI-style keys: kivi_group > 0 tiles the image span into groups of that
 * many tokens; kivi_group == 0 is one group per slice whose range covers the
 * whole supplied sequence, text included (§4 Quantization setup). */
static int kivi_whole(const hgo_config* c) { return c->kivi_group == 0; }

static uint64_t meta_words_per_slice(const hgo_config* c, int X) {
  if (kivi_keys(c, X)) {
    uint64_t ng = kivi_whole(c) ? (c->img_len > 0 ? 1 : 0)
                                : ((uint64_t)c->img_len + c->kivi_group - 1) / c->kivi_group;
    return ng * (uint64_t)c->D;
  }
  return (uint64_t)c->img_len;
}

int hgo_sizes(const hgo_config* c, const uint8_t* mask, hgo_sizes_t* out) {
  if (!cfg_ok(c) || !mask || !out) return -1;
  int LH = c->L * c->H, P = 0;
  for (int i = 0; i < LH; ++i) P += mask[i] ? 1 : 0;
  int uk = LH - P;
  int uv = c->keys_only ? LH : LH - P;
  int pv = c->keys_only ? 0 : P;
  uint64_t n = (uint64_t)c->img_len, B = (uint64_t)c->B, D = (uint64_t)c->D;
  uint64_t row = D * (uint64_t)c->bits / 8;
  out->n_protected = P;
  out->n_unprot_k = uk;
  out->n_unprot_v = uv;
  out->codes_k = (uint64_t)uk * B * n * row;
  out->codes_v = (uint64_t)uv * B * n * row;
  out->meta_k = (uint64_t)uk * B * meta_words_per_slice(c, 0) * 4;
  out->meta_v = (uint64_t)uv * B * meta_words_per_slice(c, 1) * 4;
  out->side_k = (uint64_t)P * B * n * D * 2;
  out->side_v = (uint64_t)pv * B * n * D * 2;
  uint64_t k = (uint64_t)hgo_retain_count(c);
  out->retain_count = (int32_t)k;
  out->norm_k = c->retain_permille > 0 ? (uint64_t)LH * B * n * 4 : 0;
  out->ret_idx = (uint64_t)LH * B * k * 4;
  out->ret_k = (uint64_t)uk * B * k * D * 2;
  out->ret_v = (uint64_t)uv * B * k * D * 2;
  return 0;
}

/* ------------------------------------------------------ bit packing (LSB-first) */

static void put_code(uint8_t* row, int bits, int i, unsigned q) {
  for (int k = 0; k < bits; ++k) {
    int pos = bits * i + k;
    if ((q >> k) & 1u) row[pos / 8] |= (uint8_t)(1u << (pos % 8));
  }
}

static unsigned get_code(const uint8_t* row, int bits, int i) {
  unsigned q = 0;
  for (int k = 0; k < bits; ++k) {
    int pos = bits * i + k;
    if ((row[pos / 8] >> (pos % 8)) & 1u) q |= 1u << k;
  }
  return q;
}

/* ------------------------------------------------------------ one slice */

int hgo_quantize_slice(const hgo_config* c, int X, const uint16_t* rows,
                       uint8_t* codes, uint32_t* meta) {
  if (!cfg_ok(c) || X < 0 || X > 1) return -1;
  if (kivi_keys(c, X) && kivi_whole(c)) return -1; /* needs the whole slice */
  int n = c->img_len, D = c->D, b = c->bits;
  size_t row_bytes = (size_t)D * b / 8;
  memset(codes, 0, (size_t)n * row_bytes);

  float* v = (float*)malloc(sizeof(float) * (size_t)D * (kivi_keys(c, X) ? c->kivi_group : 1));
  uint8_t* q = (uint8_t*)malloc((size_t)D * (kivi_keys(c, X) ? c->kivi_group : 1));
  if (!v || !q) { free(v); free(q); return -1; }

  if (kivi_keys(c, X)) {
    /* Keys per channel: each channel's range over a group of G consecutive
     * image tokens (the last group may be shorter). */
    int G = c->kivi_group;
    for (int g0 = 0, g = 0; g0 < n; g0 += G, ++g) {
      int m = (n - g0 < G) ? n - g0 : G;
      for (int d = 0; d < D; ++d) {
        for (int t = 0; t < m; ++t) v[t] = hgo_bf16_to_f32(rows[(size_t)(g0 + t) * D + d]);
        meta[(size_t)g * D + d] = hgo_quantize_group(v, m, 1, b, q, 1);
        for (int t = 0; t < m; ++t) put_code(codes + (size_t)(g0 + t) * row_bytes, b, d, q[t]);
      }
    }
  } else {
    /* One group per token vector; AKVQ-style keys are rotated first. */
    for (int t = 0; t < n; ++t) {
      for (int d = 0; d < D; ++d) v[d] = hgo_bf16_to_f32(rows[(size_t)t * D + d]);
      if (c->base == HGO_AKVQ && X == 0) hgo_fwht_norm(v, D);
      meta[t] = hgo_quantize_group(v, D, 1, b, q, 1);
      for (int d = 0; d < D; ++d) put_code(codes + (size_t)t * row_bytes, b, d, q[d]);
    }
  }
  free(v);
  free(q);
  return 0;
}

int hgo_quantize_slice_seq(const hgo_config* c, int X, const uint16_t* slice,
                           uint8_t* codes, uint32_t* meta) {
  if (!cfg_ok(c) || X < 0 || X > 1) return -1;
  if (!(kivi_keys(c, X) && kivi_whole(c)))
    return hgo_quantize_slice(c, X, slice + (size_t)c->img_start * c->D, codes, meta);
  /* Keys per channel, one range over all T tokens of the slice (text
   * included); only the image tokens' codes are kept. */
  int T = c->T, n = c->img_len, D = c->D, b = c->bits, s0 = c->img_start;
  size_t row_bytes = (size_t)D * b / 8;
  memset(codes, 0, (size_t)n * row_bytes);
  if (n == 0) return 0;
  float* v = (float*)malloc(sizeof(float) * (size_t)T);
  uint8_t* q = (uint8_t*)malloc((size_t)T);
  if (!v || !q) { free(v); free(q); return -1; }
  for (int d = 0; d < D; ++d) {
    for (int t = 0; t < T; ++t) v[t] = hgo_bf16_to_f32(slice[(size_t)t * D + d]);
    meta[d] = hgo_quantize_group(v, T, 1, b, q, 1);
    for (int t = 0; t < n; ++t) put_code(codes + (size_t)t * row_bytes, b, d, q[s0 + t]);
  }
  free(v);
  free(q);
  return 0;
}

int hgo_dequantize_slice(const hgo_config* c, int X, const uint8_t* codes,
                         const uint32_t* meta, uint16_t* rows_out) {
  if (!cfg_ok(c) || X < 0 || X > 1) return -1;
  int n = c->img_len, D = c->D, b = c->bits;
  size_t row_bytes = (size_t)D * b / 8;
  float* y = (float*)malloc(sizeof(float) * (size_t)D);
  if (!y) return -1;
  for (int t = 0; t < n; ++t) {
    const uint8_t* row = codes + (size_t)t * row_bytes;
    for (int d = 0; d < D; ++d) {
      uint32_t w = !kivi_keys(c, X) ? meta[t]
                   : meta[(size_t)(kivi_whole(c) ? 0 : t / c->kivi_group) * D + d];
      y[d] = hgo_level(w, get_code(row, b, d));
    }
    /* AKVQ-style keys come back to the original basis: H is symmetric and
     * orthonormal, so the inverse rotation is the same transform. */
    if (c->base == HGO_AKVQ && X == 0) hgo_fwht_norm(y, D);
    for (int d = 0; d < D; ++d) rows_out[(size_t)t * D + d] = hgo_bf16_rne(y[d]);
  }
  free(y);
  return 0;
}

/* ------------------------------------------------------------ whole cache */

typedef struct {
  const hgo_config* c;
  const uint8_t* mask;
  const uint16_t* in[2];
  uint8_t* codes[2];
  uint32_t* meta[2];
  uint16_t* side[2];
  uint16_t* out[2];
  int dequant;
  int tid, nthreads;
  int status;
} job_t;

static void* run_slices(void* arg) {
  job_t* j = (job_t*)arg;
  const hgo_config* c = j->c;
  int n = c->img_len, D = c->D;
  size_t row_bytes = (size_t)D * c->bits / 8;
  long nslices = 2L * c->L * c->B * c->H;
  for (long s = j->tid; s < nslices; s += j->nthreads) {
    int X = (int)(s / ((long)c->L * c->B * c->H));
    long r = s % ((long)c->L * c->B * c->H);
    int l = (int)(r / ((long)c->B * c->H));
    int b = (int)((r / c->H) % c->B);
    int h = (int)(r % c->H);
    int prot, slot;
    if (hgo_route(c, j->mask, X, l, h, &prot, &slot) != 0) { j->status = -1; return NULL; }
    size_t slice_off = (((size_t)l * c->B + b) * c->H + h) * c->T * D;
    size_t cache_off = slice_off + (size_t)c->img_start * D;
    size_t slab = (size_t)slot * c->B + b; /* [slot][B] */
    uint16_t* side = j->side[X] ? j->side[X] + slab * n * D : NULL;
    if (!j->dequant) {
      const uint16_t* rows = j->in[X] + cache_off;
      if (prot) {
        memcpy(side, rows, (size_t)n * D * 2);
      } else if (hgo_quantize_slice_seq(c, X, j->in[X] + slice_off, j->codes[X] + slab * n * row_bytes,
                                        j->meta[X] + slab * meta_words_per_slice(c, X)) != 0) {
        j->status = -1;
        return NULL;
      }
    } else {
      uint16_t* rows = j->out[X] + cache_off;
      if (prot) {
        memcpy(rows, side, (size_t)n * D * 2);
      } else if (hgo_dequantize_slice(c, X, j->codes[X] + slab * n * row_bytes,
                                      j->meta[X] + slab * meta_words_per_slice(c, X), rows) != 0) {
        j->status = -1;
        return NULL;
      }
    }
  }
  return NULL;
}

static int run_all(job_t* proto, int threads) {
  if (threads < 1) threads = 1;
  job_t* jobs = (job_t*)calloc((size_t)threads, sizeof(job_t));
  pthread_t* th = (pthread_t*)calloc((size_t)threads, sizeof(pthread_t));
  if (!jobs || !th) { free(jobs); free(th); return -1; }
  for (int t = 0; t < threads; ++t) {
    jobs[t] = *proto;
    jobs[t].tid = t;
    jobs[t].nthreads = threads;
    jobs[t].status = 0;
  }
  int started = 0;
  for (int t = 1; t < threads; ++t)
    if (pthread_create(&th[t], NULL, run_slices, &jobs[t]) == 0) started = t; else break;
  int status = 0;
  if (started != threads - 1) {
    /* Could not start every worker: fall back to doing all slices here. */
    for (int t = 1; t <= started; ++t) pthread_join(th[t], NULL);
    jobs[0].nthreads = 1;
    run_slices(&jobs[0]);
    status = jobs[0].status;
  } else {
    run_slices(&jobs[0]);
    for (int t = 1; t < threads; ++t) pthread_join(th[t], NULL);
    for (int t = 0; t < threads; ++t) if (jobs[t].status) status = -1;
  }
  free(jobs);
  free(th);
  return status;
}

int hgo_quantize(const hgo_config* c, const uint16_t* K, const uint16_t* V,
                 const uint8_t* mask,
                 uint8_t* codes_k, uint32_t* meta_k, uint16_t* side_k,
                 uint8_t* codes_v, uint32_t* meta_v, uint16_t* side_v,
                 int threads) {
  if (!cfg_ok(c) || !K || !V || !mask) return -1;
  job_t j;
  memset(&j, 0, sizeof j);
  j.c = c; j.mask = mask;
  j.in[0] = K; j.in[1] = V;
  j.codes[0] = codes_k; j.codes[1] = codes_v;
  j.meta[0] = meta_k; j.meta[1] = meta_v;
  j.side[0] = side_k; j.side[1] = side_v;
  return run_all(&j, threads);
}

int hgo_dequantize(const hgo_config* c, const uint8_t* mask,
                   const uint8_t* codes_k, const uint32_t* meta_k,
                   const uint16_t* side_k,
                   const uint8_t* codes_v, const uint32_t* meta_v,
                   const uint16_t* side_v,
                   uint16_t* K_out, uint16_t* V_out, int threads) {
  if (!cfg_ok(c) || !mask || !K_out || !V_out) return -1;
  job_t j;
  memset(&j, 0, sizeof j);
  j.c = c; j.mask = mask; j.dequant = 1;
  j.codes[0] = (uint8_t*)codes_k; j.codes[1] = (uint8_t*)codes_v;
  j.meta[0] = (uint32_t*)meta_k; j.meta[1] = (uint32_t*)meta_v;
  j.side[0] = (uint16_t*)side_k; j.side[1] = (uint16_t*)side_v;
  j.out[0] = K_out; j.out[1] = V_out;
  return run_all(&j, threads);
}

/* ---------------------------------------------------- AKVQ-style retention
 *
 * §4 Quantization setup: in each KV head the AKVQ-style base also keeps the
 * keys and values of a nominal 2 % of the image tokens in BF16, the tokens
 * whose keys have the largest norms, whether or not HeadGuard protects heads.
 * Readings (the paper fixes none of these):
 *  - the fraction is retain_permille / 1000 of the n image tokens of the head
 *    (20 for the paper's 2 %), k = round(n * fraction) with halves rounded up;
 *  - the norm is that of the key as stored (before the rotation, which keeps
 *    norms), computed as its square in fp32: each entry squared, then summed
 *    pairwise (adjacent entries, then adjacent pairs, ...), and tokens are
 *    ranked by that fp32 value, equal values to the lower token index;
 *  - a retained token is still quantized like every other (per-token groups do
 *    not interact); its BF16 row replaces the reconstruction;
 *  - per batch row and head the retained tokens are the same for K and V, and
 *    a row is stored only where that tensor is quantized (a protected head's
 *    BF16 rows already hold it).
 */
int hgo_retain_count(const hgo_config* c) {
  if (c->retain_permille <= 0) return 0;
  int64_t num = (int64_t)c->img_len * c->retain_permille;
  return (int)((num + 500) / 1000);
}

float hgo_key_sqnorm(const uint16_t* key, int D) {
  float a[D];
  for (int d = 0; d < D; ++d) {
    float x = hgo_bf16_to_f32(key[d]);
    a[d] = x * x;
  }
  for (int w = D / 2; w >= 1; w /= 2)
    for (int i = 0; i < w; ++i) a[i] = a[2 * i] + a[2 * i + 1];
  return a[0];
}

int hgo_retain_select(const float* sqnorm, int n, int k, int32_t* idx) {
  if (n < 0 || k < 0 || k > n) return -1;
  uint8_t* taken = (uint8_t*)calloc((size_t)n + 1, 1);
  if (!taken) return -1;
  /* k times: the largest remaining value, the lowest index among equals */
  for (int r = 0; r < k; ++r) {
    int best = -1;
    for (int i = 0; i < n; ++i)
      if (!taken[i] && (best < 0 || sqnorm[i] > sqnorm[best])) best = i;
    taken[best] = 1;
  }
  int m = 0;
  for (int i = 0; i < n; ++i)
    if (taken[i]) idx[m++] = i;
  free(taken);
  return 0;
}

typedef struct {
  const hgo_config* c;
  const uint8_t* mask;
  const uint16_t* in[2];
  float* norm_k;
  int32_t* ret_idx;
  uint16_t* ret[2];
  int tid, nthreads, status;
} retain_job_t;

static void* retain_heads(void* arg) {
  retain_job_t* j = (retain_job_t*)arg;
  const hgo_config* c = j->c;
  int n = c->img_len, D = c->D, k = hgo_retain_count(c);
  long nslices = (long)c->L * c->B * c->H;
  for (long s = j->tid; s < nslices; s += j->nthreads) {
    int l = (int)(s / ((long)c->B * c->H));
    int b = (int)((s / c->H) % c->B);
    int h = (int)(s % c->H);
    const uint16_t* keys = j->in[0] + ((size_t)s * c->T + c->img_start) * D;
    float* nrm = j->norm_k + (size_t)s * n;
    for (int t = 0; t < n; ++t) nrm[t] = hgo_key_sqnorm(keys + (size_t)t * D, D);
    int32_t* idx = j->ret_idx + (size_t)s * k;
    if (k == 0) continue;
    if (hgo_retain_select(nrm, n, k, idx) != 0) { j->status = -1; return NULL; }
    for (int X = 0; X < 2; ++X) {
      int prot, slot;
      if (hgo_route(c, j->mask, X, l, h, &prot, &slot) != 0) { j->status = -1; return NULL; }
      if (prot) continue;
      const uint16_t* rows = j->in[X] + ((size_t)s * c->T + c->img_start) * D;
      uint16_t* dst = j->ret[X] + ((size_t)slot * c->B + b) * k * D;
      for (int r = 0; r < k; ++r) memcpy(dst + (size_t)r * D, rows + (size_t)idx[r] * D, (size_t)D * 2);
    }
  }
  return NULL;
}

int hgo_retain(const hgo_config* c, const uint16_t* K, const uint16_t* V,
               const uint8_t* mask, float* norm_k, int32_t* ret_idx,
               uint16_t* ret_k, uint16_t* ret_v, int threads) {
  if (!cfg_ok(c) || c->retain_permille <= 0 || !K || !V || !mask) return -1;
  if (c->img_len == 0) return 0; /* no image tokens: nothing to rank or keep */
  if (!norm_k || (hgo_retain_count(c) > 0 && !ret_idx)) return -1;
  if (threads < 1) threads = 1;
  retain_job_t* jobs = (retain_job_t*)calloc((size_t)threads, sizeof(retain_job_t));
  pthread_t* th = (pthread_t*)calloc((size_t)threads, sizeof(pthread_t));
  if (!jobs || !th) { free(jobs); free(th); return -1; }
  for (int t = 0; t < threads; ++t) {
    retain_job_t* j = &jobs[t];
    j->c = c; j->mask = mask;
    j->in[0] = K; j->in[1] = V;
    j->norm_k = norm_k; j->ret_idx = ret_idx;
    j->ret[0] = ret_k; j->ret[1] = ret_v;
    j->tid = t; j->nthreads = threads;
  }
  int started = 0;
  for (int t = 1; t < threads; ++t)
    if (pthread_create(&th[t], NULL, retain_heads, &jobs[t]) == 0) started = t; else break;
  if (started != threads - 1) {
    for (int t = 1; t <= started; ++t) pthread_join(th[t], NULL);
    for (int t = 0; t < threads; ++t) jobs[t].status = 0;
    jobs[0].nthreads = 1;
    retain_heads(&jobs[0]);
  } else {
    retain_heads(&jobs[0]);
    for (int t = 1; t < threads; ++t) pthread_join(th[t], NULL);
  }
  int status = 0;
  for (int t = 0; t < threads; ++t) if (jobs[t].status) status = -1;
  free(jobs);
  free(th);
  return status;
}

int hgo_restore_retained(const hgo_config* c, const uint8_t* mask,
                         const int32_t* ret_idx, const uint16_t* ret_k,
                         const uint16_t* ret_v, uint16_t* K_out, uint16_t* V_out) {
  if (!cfg_ok(c) || c->retain_permille <= 0 || !mask || !K_out || !V_out) return -1;
  int D = c->D, k = hgo_retain_count(c);
  if (k == 0) return 0;
  const uint16_t* ret[2] = {ret_k, ret_v};
  uint16_t* out[2] = {K_out, V_out};
  for (long s = 0; s < (long)c->L * c->B * c->H; ++s) {
    int l = (int)(s / ((long)c->B * c->H));
    int b = (int)((s / c->H) % c->B);
    int h = (int)(s % c->H);
    const int32_t* idx = ret_idx + (size_t)s * k;
    for (int X = 0; X < 2; ++X) {
      int prot, slot;
      if (hgo_route(c, mask, X, l, h, &prot, &slot) != 0) return -1;
      if (prot) continue;
      uint16_t* rows = out[X] + ((size_t)s * c->T + c->img_start) * D;
      const uint16_t* src = ret[X] + ((size_t)slot * c->B + b) * k * D;
      for (int r = 0; r < k; ++r) memcpy(rows + (size_t)idx[r] * D, src + (size_t)r * D, (size_t)D * 2);
    }
  }
  return 0;
}

/* ------------------------------------------------------------ head selection
 *
 * §3 "Selecting physical KV heads", Eq. 2.  Readings: a query head hq belongs
 * to the KV head hq / (Hq/Hkv) (consecutive query heads share a KV head);
 * z() uses the population standard deviation over all L*Hkv KV heads, and a
 * zero deviation gives z = 0; TopK breaks ties toward the lower head index.
 */
static void zscore(double* x, int n) {
  double mean = 0.0, var = 0.0;
  for (int i = 0; i < n; ++i) mean += x[i];
  mean /= n;
  for (int i = 0; i < n; ++i) var += (x[i] - mean) * (x[i] - mean);
  var /= n;
  double sd = sqrt(var);
  for (int i = 0; i < n; ++i) x[i] = sd > 0.0 ? (x[i] - mean) / sd : 0.0;
}

int hgo_select_heads(const double* g, const double* o, int L, int Hq, int Hkv, int K,
                     uint8_t* mask) {
  if (!g || !o || !mask || L <= 0 || Hkv <= 0 || Hq <= 0 || Hq % Hkv != 0 || K < 0) return -1;
  int n = L * Hkv, rep = Hq / Hkv;
  double* gb = (double*)calloc((size_t)n, sizeof(double));
  double* ob = (double*)calloc((size_t)n, sizeof(double));
  double* sc = (double*)calloc((size_t)n, sizeof(double));
  if (!gb || !ob || !sc) { free(gb); free(ob); free(sc); return -1; }
  /* GQA average of the query heads of each physical KV head */
  for (int l = 0; l < L; ++l)
    for (int hq = 0; hq < Hq; ++hq) {
      int i = l * Hkv + hq / rep;
      gb[i] += g[(size_t)l * Hq + hq];
      ob[i] += o[(size_t)l * Hq + hq];
    }
  for (int i = 0; i < n; ++i) {
    gb[i] /= rep;
    ob[i] /= rep;
  }
  zscore(gb, n);
  zscore(ob, n);
  for (int i = 0; i < n; ++i) sc[i] = gb[i] + ob[i];
  /* TopK: K times, take the largest remaining score (lowest index on ties) */
  for (int i = 0; i < n; ++i) mask[i] = 0;
  for (int k = 0; k < K && k < n; ++k) {
    int best = -1;
    for (int i = 0; i < n; ++i)
      if (!mask[i] && (best < 0 || sc[i] > sc[best])) best = i;
    mask[best] = 1;
  }
  free(gb);
  free(ob);
  free(sc);
  return 0;
}
