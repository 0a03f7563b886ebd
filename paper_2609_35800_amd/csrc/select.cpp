// Head selection (HeadGuard §3 "Selecting physical KV heads", Eq. 2), host
// side of libheadguard: average the per-query-head image and output
// sensitivity scores within each physical KV group, standardize each over all
// KV heads, and mark the K heads with the largest sum; and the head budget
// K = round(N_KV * f) of §3.  Declared in include/headguard.h.

#include <math.h>
#include <stdint.h>
#include <string.h>

#include <algorithm>
#include <numeric>
#include <vector>

#include "headguard.h"

namespace hg {
int set_error(int status, const char* msg);  // api.hip
}

namespace {

// z-score with the population deviation; a constant score gives z = 0.
void standardize(std::vector<double>& x) {
  const double n = (double)x.size();
  double sum = 0.0;
  for (double v : x) sum += v;
  const double mean = sum / n;
  double ss = 0.0;
  for (double v : x) ss += (v - mean) * (v - mean);
  const double sd = std::sqrt(ss / n);
  for (double& v : x) v = sd > 0.0 ? (v - mean) / sd : 0.0;
}

}  // namespace

extern "C" int hg_select_heads(const double* g, const double* o, int32_t L, int32_t Hq, int32_t Hkv,
                               int32_t K, uint8_t* mask) {
  if (!g || !o || !mask) return hg::set_error(HG_ERR_NULL, "g, o and mask must not be NULL");
  if (L <= 0 || Hq <= 0 || Hkv <= 0 || Hq % Hkv != 0 || (int64_t)L * Hkv > HG_MAX_HEADS || K < 0)
    return hg::set_error(HG_ERR_SHAPE, "need L, Hq, Hkv > 0, Hq a multiple of Hkv, L*Hkv <= HG_MAX_HEADS, K >= 0");
  const int n = L * Hkv, rep = Hq / Hkv;
  for (int64_t i = 0; i < (int64_t)L * Hq; ++i)
    if (!std::isfinite(g[i]) || !std::isfinite(o[i]))
      return hg::set_error(HG_ERR_VALUE, "scores must be finite");

  std::vector<double> gbar(n, 0.0), obar(n, 0.0);
  for (int l = 0; l < L; ++l)
    for (int h = 0; h < Hkv; ++h) {
      double sg = 0.0, so = 0.0;
      for (int r = 0; r < rep; ++r) {  // query heads h*rep .. h*rep + rep - 1 share KV head h
        sg += g[(size_t)l * Hq + (size_t)h * rep + r];
        so += o[(size_t)l * Hq + (size_t)h * rep + r];
      }
      gbar[(size_t)l * Hkv + h] = sg / rep;
      obar[(size_t)l * Hkv + h] = so / rep;
    }
  standardize(gbar);
  standardize(obar);

  std::vector<int> order(n);
  std::iota(order.begin(), order.end(), 0);
  std::vector<double> s(n);
  for (int i = 0; i < n; ++i) s[i] = gbar[i] + obar[i];
  std::stable_sort(order.begin(), order.end(), [&](int a, int b) { return s[a] > s[b]; });
  memset(mask, 0, (size_t)n);
  for (int k = 0; k < std::min(K, n); ++k) mask[order[k]] = 1;
  return hg::set_error(HG_OK, "");
}

extern "C" int hg_head_budget(int32_t n_kv_heads, int32_t num, int32_t den, int32_t* K_out) {
  if (!K_out) return hg::set_error(HG_ERR_NULL, "K_out must not be NULL");
  if (n_kv_heads < 1 || den < 1 || num < 0 || num > den)
    return hg::set_error(HG_ERR_SHAPE, "need n_kv_heads >= 1, den >= 1 and 0 <= num <= den");
  // round(n * num / den), halves up: floor((2 n num + den) / (2 den)), exact in 64 bits
  const int64_t q = (2 * (int64_t)n_kv_heads * num + den) / (2 * (int64_t)den);
  *K_out = (int32_t)q;
  return hg::set_error(HG_OK, "");
}
