// Host side of libheadguard: argument checks, the packed-size closed form,
// mask routing into kernel arguments, and kernel launch.  Declarations and
// the contract of every entry point are in include/headguard.h.

#include <stdarg.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <string>

#include "headguard.h"
#include "hg_kernels.h"

namespace {

thread_local std::string g_last_error;

int fail(int status, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
int fail(int status, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return status;
}

int ok() {
  g_last_error.clear();
  return HG_OK;
}

// Shape, span, bits, base and mask checks shared by every entry point.
int check_config(const hg_config* c, const uint8_t* mask) {
  if (!c) return fail(HG_ERR_NULL, "cfg is NULL");
  if (!mask) return fail(HG_ERR_NULL, "protect_mask is NULL");
  if (c->L <= 0 || c->B <= 0 || c->H <= 0 || c->T <= 0)
    return fail(HG_ERR_SHAPE, "L, B, H, T must be positive (got %d, %d, %d, %d)", c->L, c->B, c->H, c->T);
  if ((int64_t)c->L * c->H > HG_MAX_HEADS)
    return fail(HG_ERR_SHAPE, "L*H = %lld exceeds %d", (long long)c->L * c->H, HG_MAX_HEADS);
  if (c->D != 64 && c->D != 128 && c->D != 256)
    return fail(HG_ERR_HEADDIM, "head_dim %d not in {64, 128, 256}", c->D);
  if (c->img_start < 0 || c->img_len < 0 || (int64_t)c->img_start + c->img_len > c->T)
    return fail(HG_ERR_SPAN, "image span [%d, %d + %d) outside [0, %d]", c->img_start, c->img_start,
                c->img_len, c->T);
  if (c->bits < 2 || c->bits > 4) return fail(HG_ERR_BITS, "bits %d not in {2, 3, 4}", c->bits);
  if (c->base != HG_BASE_MINMAX && c->base != HG_BASE_KIVI && c->base != HG_BASE_AKVQ)
    return fail(HG_ERR_BASE, "unknown base %d", c->base);
  if (c->base == HG_BASE_KIVI && c->kivi_group != hg::kWaveTokens && c->kivi_group != 0)
    return fail(HG_ERR_BASE, "kivi_group %d unsupported (32, or 0 for the whole sequence)", c->kivi_group);
  if (c->keys_only != 0 && c->keys_only != 1) return fail(HG_ERR_SHAPE, "keys_only must be 0 or 1");
  if (c->retain_permille < 0 || c->retain_permille > 1000)
    return fail(HG_ERR_BASE, "retain_permille %d outside [0, 1000]", c->retain_permille);
  if (c->retain_permille > 0 && c->base != HG_BASE_AKVQ)
    return fail(HG_ERR_BASE, "token retention belongs to the AKVQ base (base %d)", c->base);
  const int LH = c->L * c->H;
  for (int i = 0; i < LH; ++i)
    if (mask[i] > 1) return fail(HG_ERR_MASK, "protect_mask[%d] = %u is neither 0 nor 1", i, mask[i]);
  return HG_OK;
}

struct Counts {
  int P, uk, uv, pv;
  uint64_t n, row, meta_k_words, meta_v_words;
  uint64_t k;  // retained tokens per (l, b, h)
};

Counts counts(const hg_config* c, const uint8_t* mask) {
  Counts k;
  const int LH = c->L * c->H;
  k.P = 0;
  for (int i = 0; i < LH; ++i) k.P += mask[i];
  k.uk = LH - k.P;
  k.uv = c->keys_only ? LH : LH - k.P;
  k.pv = c->keys_only ? 0 : k.P;
  k.n = (uint64_t)c->img_len;
  k.row = (uint64_t)c->D * c->bits / 8;
  const uint64_t groups = c->kivi_group == 0 ? (k.n > 0 ? 1 : 0) : (k.n + hg::kWaveTokens - 1) / hg::kWaveTokens;
  k.meta_k_words = c->base == HG_BASE_KIVI ? groups * c->D : k.n;
  k.meta_v_words = k.n;
  // round(n * permille / 1000), halves up
  k.k = c->retain_permille > 0 ? (k.n * (uint64_t)c->retain_permille + 500) / 1000 : 0;
  return k;
}

bool aligned(const void* p, uintptr_t a) { return ((uintptr_t)p % a) == 0; }

int check_device_ptr(const void* p, const char* name) {
  hipPointerAttribute_t attr;
  hipError_t e = hipPointerGetAttributes(&attr, p);
  if (e != hipSuccess) {
    (void)hipGetLastError();
    return fail(HG_ERR_POINTER, "%s is not device memory (%s)", name, hipGetErrorString(e));
  }
  if (attr.type != hipMemoryTypeDevice && attr.type != hipMemoryTypeManaged)
    return fail(HG_ERR_POINTER, "%s is not device memory (memory type %d)", name, (int)attr.type);
  return HG_OK;
}

// Checks that a HIP device is present.
int check_device() {
  int n = 0;
  hipError_t e = hipGetDeviceCount(&n);
  if (e != hipSuccess || n <= 0) {
    (void)hipGetLastError();
    return fail(HG_ERR_NO_DEVICE, "no HIP device (%s)", hipGetErrorString(e));
  }
  return HG_OK;
}

// Buffers the call reads or writes, with their sizes, for NULL, alignment and
// device-memory checks.
struct Buf {
  const void* p;
  uint64_t bytes;
  uintptr_t align;
  const char* name;
};

int check_buffers(const Buf* bufs, int nb) {
  for (int i = 0; i < nb; ++i) {
    if (bufs[i].bytes == 0) continue;
    if (!bufs[i].p) return fail(HG_ERR_NULL, "%s is NULL but %llu bytes are needed", bufs[i].name,
                                (unsigned long long)bufs[i].bytes);
    if (!aligned(bufs[i].p, bufs[i].align))
      return fail(HG_ERR_ALIGN, "%s is not %u-byte aligned", bufs[i].name, (unsigned)bufs[i].align);
  }
  for (int i = 0; i < nb; ++i) {
    if (bufs[i].bytes == 0) continue;
    int s = check_device_ptr(bufs[i].p, bufs[i].name);
    if (s) return s;
  }
  return HG_OK;
}

// The call's largest tiled grid (K and V, workgroup tiles of as few as
// kMinBlockTokens tokens) must fit the launch limit; checked before any launch.
int check_grid(const hg_config* c) {
  const uint64_t tiles = ((uint64_t)c->img_len + hg::kMinBlockTokens - 1) / hg::kMinBlockTokens;
  const uint64_t blocks = 2 * (uint64_t)c->L * c->B * c->H * tiles;
  if (blocks > 0x7FFFFFFFull)
    return fail(HG_ERR_SHAPE, "grid of %llu workgroups too large", (unsigned long long)blocks);
  return HG_OK;
}

// Launch steps of one call.  Test hook: with HG_FAIL_LAUNCH=i in the
// environment, step i (0-based) of every call reports hipErrorLaunchFailure
// without enqueuing anything, so the mapping of a launch error to HG_ERR_HIP
// can be exercised on a working device.  Step 0 failing leaves every output
// untouched; a later step failing leaves the earlier steps enqueued.
struct LaunchSteps {
  int fail_at = -1;
  int next = 0;
  LaunchSteps() {
    const char* s = getenv("HG_FAIL_LAUNCH");
    if (s && *s) fail_at = atoi(s);
  }
  template <class F>
  hipError_t operator()(F&& launch) {
    if (next++ == fail_at) return hipErrorLaunchFailure;
    return launch();
  }
};

// Workspace of the one-pass call with token retention, 256-byte aligned
// parts: the key norms, the retained token lists, then (in place only) the
// saved retained rows of K and V.
struct FakeWorkspace {
  uint64_t o_idx, o_k, o_v;
  uint64_t out_of_place, in_place;  // bytes each form needs
};

FakeWorkspace fake_workspace(const hg_sizes& z) {
  auto up = [](uint64_t b) { return (b + 255) & ~(uint64_t)255; };
  FakeWorkspace w;
  w.o_idx = up(z.norm_k);
  w.o_k = w.o_idx + up(z.ret_idx);
  w.o_v = w.o_k + up(z.ret_k);
  w.out_of_place = z.retain_count > 0 ? w.o_k : 0;
  w.in_place = z.retain_count > 0 ? w.o_v + up(z.ret_v) : 0;
  return w;
}

// Exchange workspace of KIVI-style keys over the whole sequence: needed when
// a key slice is held by several workgroups and some key slice is quantized.
uint64_t kivi_exchange_bytes(const hg_config* c, const Counts& k) {
  if (c->base != HG_BASE_KIVI || c->kivi_group != 0 || k.n == 0 || k.uk == 0) return 0;
  return hg::kivi_workspace_bytes(c->T, c->D);
}

void fill_params(hg::Params& p, const hg_config* c, const uint8_t* mask) {
  memset(&p, 0, sizeof p);
  p.L = c->L;
  p.B = c->B;
  p.H = c->H;
  p.T = c->T;
  p.s0 = c->img_start;
  p.n = c->img_len;
  p.keys_only = c->keys_only;
  p.kivi_whole = c->base == HG_BASE_KIVI && c->kivi_group == 0;
  p.ngroups = p.kivi_whole ? 1 : (c->img_len + hg::kWaveTokens - 1) / hg::kWaveTokens;
  p.tiles = (c->img_len + hg::kBlockTokens - 1) / hg::kBlockTokens;
  const int LH = c->L * c->H;
  uint32_t running = 0;
  for (int w = 0; w < (LH + 31) / 32; ++w) {
    uint32_t word = 0;
    for (int b = 0; b < 32 && 32 * w + b < LH; ++b) word |= (uint32_t)(mask[32 * w + b] & 1u) << b;
    p.route.mask[w] = word;
    p.route.prefix[w] = running;
    running += (uint32_t)__builtin_popcount(word);
  }
  p.n_unprot_k = LH - (int32_t)running;
}

}  // namespace

namespace hg {
// Records the detail of a status for hg_last_error (used by the other host
// sources of the library).
int set_error(int status, const char* msg) {
  g_last_error = status == HG_OK ? "" : msg;
  return status;
}
}  // namespace hg

extern "C" {

const char* hg_status_string(int s) {
  switch (s) {
    case HG_OK: return "HG_OK";
    case HG_ERR_NULL: return "HG_ERR_NULL";
    case HG_ERR_SHAPE: return "HG_ERR_SHAPE";
    case HG_ERR_SPAN: return "HG_ERR_SPAN";
    case HG_ERR_BITS: return "HG_ERR_BITS";
    case HG_ERR_BASE: return "HG_ERR_BASE";
    case HG_ERR_HEADDIM: return "HG_ERR_HEADDIM";
    case HG_ERR_ALIGN: return "HG_ERR_ALIGN";
    case HG_ERR_MASK: return "HG_ERR_MASK";
    case HG_ERR_NO_DEVICE: return "HG_ERR_NO_DEVICE";
    case HG_ERR_HIP: return "HG_ERR_HIP";
    case HG_ERR_POINTER: return "HG_ERR_POINTER";
    case HG_ERR_VALUE: return "HG_ERR_VALUE";
    default: return "HG_ERR_UNKNOWN";
  }
}

const char* hg_last_error(void) { return g_last_error.c_str(); }

int hg_packed_sizes(const hg_config* cfg, const uint8_t* mask, hg_sizes* out) {
  if (!out) return fail(HG_ERR_NULL, "out is NULL");
  int s = check_config(cfg, mask);
  if (s) return s;
  const Counts k = counts(cfg, mask);
  const uint64_t B = (uint64_t)cfg->B, D = (uint64_t)cfg->D;
  out->n_protected = k.P;
  out->n_unprot_k = k.uk;
  out->n_unprot_v = k.uv;
  out->codes_k = (uint64_t)k.uk * B * k.n * k.row;
  out->codes_v = (uint64_t)k.uv * B * k.n * k.row;
  out->meta_k = (uint64_t)k.uk * B * k.meta_k_words * 4;
  out->meta_v = (uint64_t)k.uv * B * k.meta_v_words * 4;
  out->side_k = (uint64_t)k.P * B * k.n * D * 2;
  out->side_v = (uint64_t)k.pv * B * k.n * D * 2;
  const uint64_t LHB = (uint64_t)cfg->L * cfg->H * B;
  out->retain_count = (int32_t)k.k;
  out->norm_k = cfg->retain_permille > 0 ? LHB * k.n * 4 : 0;
  out->ret_idx = LHB * k.k * 4;
  out->ret_k = (uint64_t)k.uk * B * k.k * D * 2;
  out->ret_v = (uint64_t)k.uv * B * k.k * D * 2;
  out->workspace = kivi_exchange_bytes(cfg, k);
  out->fake_workspace = cfg->retain_permille > 0 ? fake_workspace(*out).in_place : out->workspace;
  return ok();
}

static int run(bool quantize, const hg_config* cfg, const uint16_t* K, const uint16_t* V,
               const uint8_t* mask, const hg_packed* pk, hipStream_t stream) {
  int s = check_config(cfg, mask);
  if (!s) s = check_grid(cfg);
  if (s) return s;
  if (!pk) return fail(HG_ERR_NULL, "packed buffer descriptor is NULL");
  hg_sizes z;
  hg_packed_sizes(cfg, mask, &z);
  const uint64_t cache_bytes = (uint64_t)cfg->L * cfg->B * cfg->H * cfg->T * cfg->D * 2;
  const uint64_t need = cfg->img_len > 0 ? cache_bytes : 0;
  const Buf bufs[] = {
      {K, need, 16, quantize ? "K" : "K_out"},
      {V, need, 16, quantize ? "V" : "V_out"},
      {pk->codes_k, z.codes_k, 16, "codes_k"},
      {pk->meta_k, z.meta_k, 16, "meta_k"},
      {pk->side_k, z.side_k, 16, "side_k"},
      {pk->codes_v, z.codes_v, 16, "codes_v"},
      {pk->meta_v, z.meta_v, 16, "meta_v"},
      {pk->side_v, z.side_v, 16, "side_v"},
      {pk->norm_k, quantize ? z.norm_k : 0, 16, "norm_k"},  // dequantize does not read it
      {pk->ret_idx, z.ret_idx, 16, "ret_idx"},
      {pk->ret_k, z.ret_k, 16, "ret_k"},
      {pk->ret_v, z.ret_v, 16, "ret_v"},
      {pk->workspace, quantize ? z.workspace : 0, 256, "workspace"},  // dequantize does not use it
  };
  const int nb = (int)(sizeof bufs / sizeof bufs[0]);
  // Every buffer the call writes (quantize: the packed ones; dequantize: K_out,
  // V_out) must be disjoint from every other buffer of the call.
  for (int i = 0; i < nb; ++i) {
    const bool written = quantize ? i >= 2 : i < 2;
    if (!written || bufs[i].bytes == 0) continue;
    for (int j = 0; j < nb; ++j) {
      if (j == i || bufs[j].bytes == 0) continue;
      const uintptr_t a = (uintptr_t)bufs[i].p, b = (uintptr_t)bufs[j].p;
      if (a < b + bufs[j].bytes && b < a + bufs[i].bytes)
        return fail(HG_ERR_POINTER, "%s overlaps %s", bufs[i].name, bufs[j].name);
    }
  }
  s = check_device();
  if (s) return s;
  s = check_buffers(bufs, nb);
  if (s) return s;
  if (cfg->img_len == 0) return ok();

  hg::Params p;
  fill_params(p, cfg, mask);
  p.cache[0] = K;
  p.cache[1] = V;
  p.codes[0] = (uint8_t*)pk->codes_k;
  p.codes[1] = (uint8_t*)pk->codes_v;
  p.meta[0] = (uint32_t*)pk->meta_k;
  p.meta[1] = (uint32_t*)pk->meta_v;
  p.side[0] = (uint16_t*)pk->side_k;
  p.side[1] = (uint16_t*)pk->side_v;
  const bool retain = cfg->retain_permille > 0;
  p.norm = retain && quantize ? (float*)pk->norm_k : nullptr;
  p.ret_idx = (int32_t*)pk->ret_idx;
  p.ret[0] = (uint16_t*)pk->ret_k;
  p.ret[1] = (uint16_t*)pk->ret_v;
  p.k = z.retain_count;
  p.out[0] = quantize ? nullptr : (uint16_t*)K;
  p.out[1] = quantize ? nullptr : (uint16_t*)V;
  // whole-sequence KIVI keys: the first kernel of the call clears the key
  // kernel's exchange words (one launch fewer)
  void* kivi_ws = z.workspace ? pk->workspace : nullptr;
  if (quantize && p.kivi_whole && kivi_ws) {
    const hipError_t pe = hg::kivi_seq_clear_words(p, cfg->D, cfg->bits, false, kivi_ws, &p.clear_words);
    if (pe != hipSuccess) return fail(HG_ERR_HIP, "KIVI key kernel plan failed: %s", hipGetErrorString(pe));
    p.clear = (uint64_t*)kivi_ws;
  }
  LaunchSteps step;
  hipError_t e = step([&] {
    return quantize ? hg::launch_quantize(p, cfg->base, cfg->D, cfg->bits, retain, stream)
                    : hg::launch_dequantize(p, cfg->base, cfg->D, cfg->bits, stream);
  });
  p.clear_words = 0;
  if (e == hipSuccess && quantize && p.kivi_whole)
    e = step([&] { return hg::launch_kivi_seq(p, cfg->D, cfg->bits, false, kivi_ws, true, stream); });
  if (e == hipSuccess && p.k > 0 && quantize)
    e = step([&] { return hg::launch_retain_select(p, cfg->D, hg::RowCopy::kGather, stream); });
  if (e == hipSuccess && p.k > 0 && !quantize)
    e = step([&] { return hg::launch_retain_rows(p, cfg->D, hg::RowCopy::kScatter, stream); });
  if (e != hipSuccess) return fail(HG_ERR_HIP, "kernel launch failed: %s", hipGetErrorString(e));
  return ok();
}

}  // extern "C"

namespace hg {

// The one-pass simulated quantization.  `get_ws` supplies the token-retention
// workspace once the call's host-side argument checks have passed and its
// size is known (it is not called without retention).
int fake_quantize(const hg_config* cfg, const uint16_t* K, const uint16_t* V, const uint8_t* mask,
                  uint16_t* K_out, uint16_t* V_out, const WorkspaceFn& get_ws, hipStream_t stream) {
  int s = check_config(cfg, mask);
  if (!s) s = check_grid(cfg);
  if (s) return s;
  const uint64_t cache_bytes = (uint64_t)cfg->L * cfg->B * cfg->H * cfg->T * cfg->D * 2;
  const uint64_t need = cfg->img_len > 0 ? cache_bytes : 0;
  if (need && (!K || !V || !K_out || !V_out)) return fail(HG_ERR_NULL, "K, V, K_out and V_out are required");
  // Each output is its own input or disjoint from it; no output may overlap
  // the other tensor's input or the other output.
  auto overlap = [](const void* x, uint64_t nx, const void* y, uint64_t ny) {
    const uintptr_t a = (uintptr_t)x, b = (uintptr_t)y;
    return nx && ny && a < b + ny && b < a + nx;
  };
  for (int X = 0; X < 2; ++X) {
    const void* in = X ? (const void*)V : (const void*)K;
    const void* out = X ? (const void*)V_out : (const void*)K_out;
    const void* other_in = X ? (const void*)K : (const void*)V;
    const char* nm = X ? "V" : "K";
    if (out != in && overlap(in, need, out, need))
      return fail(HG_ERR_POINTER, "%s_out partially overlaps %s (must be the same buffer or disjoint)", nm, nm);
    if (overlap(out, need, other_in, need))
      return fail(HG_ERR_POINTER, "%s_out overlaps %s", nm, X ? "K" : "V");
  }
  if (overlap(K_out, need, V_out, need)) return fail(HG_ERR_POINTER, "K_out and V_out overlap");

  // Token retention: the workspace holds the norms and the selection.  Out of
  // place, the one-pass kernel writes the key norms from the rows it reads,
  // and the retained rows are then copied from the inputs to the outputs.  In
  // place (either tensor), the outputs would overwrite the rows to keep: the
  // norms come from a pass of their own, and the retained rows are saved to
  // the workspace first and written back last.
  hg_sizes z;
  hg_packed_sizes(cfg, mask, &z);
  const bool retain = need && z.retain_count > 0;
  const bool fused = retain && K_out != K && V_out != V;
  const FakeWorkspace lay = fake_workspace(z);
  // retention (AKVQ) or the exchange of whole-sequence KIVI key ranges
  const uint64_t ws_need = retain ? (fused ? lay.out_of_place : lay.in_place) : need ? z.workspace : 0;
  Workspace wsp;
  if (ws_need) {
    s = get_ws(ws_need, &wsp);
    if (s) return s;
    if (!wsp.ptr)
      return fail(HG_ERR_NULL, "workspace is NULL but the call needs %llu bytes", (unsigned long long)ws_need);
    if (ws_need > wsp.bytes)
      return fail(HG_ERR_SHAPE, "the call needs a %llu-byte workspace (%llu bytes available)",
                  (unsigned long long)ws_need, (unsigned long long)wsp.bytes);
    if (!aligned(wsp.ptr, 256)) return fail(HG_ERR_ALIGN, "workspace is not 256-byte aligned");
    const void* ins[4] = {K, V, K_out, V_out};
    const char* names[4] = {"K", "V", "K_out", "V_out"};
    for (int i = 0; i < 4; ++i)
      if (overlap(wsp.ptr, ws_need, ins[i], need)) return fail(HG_ERR_POINTER, "workspace overlaps %s", names[i]);
  }
  void* const ws = wsp.ptr;
  const Buf bufs[] = {{K, need, 16, "K"},
                      {V, need, 16, "V"},
                      {K_out, need, 16, "K_out"},
                      {V_out, need, 16, "V_out"},
                      {ws, wsp.caller ? ws_need : 0, 256, "workspace"}};
  s = check_device();
  if (s) return s;
  s = check_buffers(bufs, 5);
  if (s) return s;
  if (cfg->img_len == 0) return ok();
  hg::Params p;
  fill_params(p, cfg, mask);
  p.cache[0] = K;
  p.cache[1] = V;
  p.out[0] = K_out;
  p.out[1] = V_out;
  if (retain) {
    char* w = (char*)ws;
    p.norm = (float*)w;
    p.ret_idx = (int32_t*)(w + lay.o_idx);
    p.ret[0] = fused ? nullptr : (uint16_t*)(w + lay.o_k);
    p.ret[1] = fused ? nullptr : (uint16_t*)(w + lay.o_v);
    p.k = z.retain_count;
  }
  LaunchSteps step;
  hipError_t e = hipSuccess;
  if (retain && !fused) {
    e = step([&] { return hg::launch_key_norms(p, cfg->D, stream); });
    if (e == hipSuccess)
      e = step([&] { return hg::launch_retain_select(p, cfg->D, hg::RowCopy::kGather, stream); });
  }
  if (e == hipSuccess && p.kivi_whole && ws) {  // the one-pass kernel clears the key kernel's exchange words
    e = hg::kivi_seq_clear_words(p, cfg->D, cfg->bits, true, ws, &p.clear_words);
    p.clear = (uint64_t*)ws;
  }
  if (e == hipSuccess)
    e = step([&] { return hg::launch_fake_quantize(p, cfg->base, cfg->D, cfg->bits, fused, stream); });
  p.clear_words = 0;
  if (e == hipSuccess && p.kivi_whole)
    e = step([&] { return hg::launch_kivi_seq(p, cfg->D, cfg->bits, true, ws, true, stream); });
  if (e == hipSuccess && fused) {
    e = step([&] { return hg::launch_retain_select(p, cfg->D, hg::RowCopy::kCacheToOut, stream); });
  } else if (e == hipSuccess && retain) {
    e = step([&] { return hg::launch_retain_rows(p, cfg->D, hg::RowCopy::kScatter, stream); });
  }
  if (e != hipSuccess) return fail(HG_ERR_HIP, "kernel launch failed: %s", hipGetErrorString(e));
  return ok();
}

}  // namespace hg

extern "C" {

int hg_fake_quantize(const hg_config* cfg, const uint16_t* K, const uint16_t* V, const uint8_t* mask,
                     uint16_t* K_out, uint16_t* V_out, void* workspace, uint64_t workspace_bytes,
                     hipStream_t stream) {
  const hg::WorkspaceFn caller = [&](uint64_t, hg::Workspace* ws) {
    ws->ptr = workspace;
    ws->bytes = workspace ? workspace_bytes : 0;
    ws->caller = true;
    return (int)HG_OK;
  };
  return hg::fake_quantize(cfg, K, V, mask, K_out, V_out, caller, stream);
}

int hg_quantize(const hg_config* cfg, const uint16_t* K, const uint16_t* V, const uint8_t* mask,
                const hg_packed* out, hipStream_t stream) {
  if (!K || !V) {
    if (cfg && cfg->img_len != 0) return fail(HG_ERR_NULL, "K or V is NULL");
  }
  return run(true, cfg, K, V, mask, out, stream);
}

int hg_dequantize(const hg_config* cfg, const uint8_t* mask, const hg_packed* in, uint16_t* K_out,
                  uint16_t* V_out, hipStream_t stream) {
  if (!K_out || !V_out) {
    if (cfg && cfg->img_len != 0) return fail(HG_ERR_NULL, "K_out or V_out is NULL");
  }
  return run(false, cfg, K_out, V_out, mask, in, stream);
}

}  // extern "C"
