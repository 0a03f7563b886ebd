"""The oracle's pins must catch plausible slips.  Each case plants one mistake
in a copy of the oracle source (on the CPU, in a temporary directory), builds
it, and runs the pin suites against the mutant: at least one pin must fail.
The planted mistakes cover each step of the method: rounding directions and
tie rules, the range, the scale and its levels, reconstruction, the
Walsh-Hadamard butterflies and scale, routing ranks and K-only protection,
KIVI-style group indexing, bit packing, the image-span offset, the buffer
sizes, the head selection's sum, grouping, standardization and ties, and the
token retention's count, norm, ranking, ties and row routing."""
import concurrent.futures as cf
import os
import shutil
import subprocess
import sys
import tempfile

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "hg_oracle.c")

MUTANTS = [
    ("rint_ties_away", "float r = rintf(t);", "float r = roundf(t);"),
    ("rd_wrong_direction", "if (lo != 0 && (u >> 31)) hi += 1;", "if (lo != 0 && !(u >> 31)) hi += 1;"),
    ("ru_truncates", "if (lo != 0 && !(u >> 31)) hi += 1;", "if (0) hi += 1;"),
    ("rne_ties_away", "(lo == 0x8000u && (hi & 1u))", "(lo == 0x8000u)"),
    ("min_sign", "if (x < mn) mn = x;", "if (x > mn) mn = x;"),
    ("max_init", "float mn = v[0], mx = v[0];", "float mn = v[0], mx = 0.0f;"),
    ("scale_uses_raw_min", "float s = (mx - mf) / (float)levels;", "float s = (mx - mn) / (float)levels;"),
    ("levels_off_by_one", "int levels = (1 << bits) - 1;", "int levels = (1 << bits);"),
    ("scale_round_nearest", "uint16_t s16 = hgo_bf16_ru(s);", "uint16_t s16 = hgo_bf16_rne(s);"),
    ("min_round_nearest", "uint16_t m16 = hgo_bf16_rd(mn);", "uint16_t m16 = hgo_bf16_rne(mn);"),
    ("clamp_off_by_one", "if (r > (float)levels) r = (float)levels;",
     "if (r > (float)levels - 1) r = (float)levels - 1;"),
    ("recon_sign", "return p + m;", "return p - m;"),
    ("recon_meta_halves_swapped",
     "float S = hgo_bf16_to_f32((uint16_t)(meta & 0xFFFFu));\n  float m = hgo_bf16_to_f32((uint16_t)(meta >> 16));",
     "float S = hgo_bf16_to_f32((uint16_t)(meta >> 16));\n  float m = hgo_bf16_to_f32((uint16_t)(meta & 0xFFFFu));"),
    ("fwht_sign", "a[j + h] = p - q;", "a[j + h] = q - p;"),
    ("fwht_missing_stage", "for (int h = 1; h < D; h *= 2)", "for (int h = 1; h < D / 2; h *= 2)"),
    ("fwht_reversed_stages", "for (int h = 1; h < D; h *= 2)", "for (int h = D / 2; h >= 1; h /= 2)"),
    ("fwht_missing_scale", "for (int j = 0; j < D; ++j) a[j] = a[j] * c;", "(void)c;"),
    ("route_rank_counts_all", "if (is_kept(c, mask, X, j) == kept) rank++;", "rank++;"),
    ("k_only_protects_values", "return X == 0 ? 1 : !c->keys_only;", "return 1;"),
    ("kivi_meta_transposed", "meta[(size_t)g * D + d] = hgo_quantize_group(v, m, 1, b, q, 1);",
     "meta[(size_t)d * ((n + G - 1) / G) + g] = hgo_quantize_group(v, m, 1, b, q, 1);"),
    ("kivi_group_offset_dropped", "v[t] = hgo_bf16_to_f32(rows[(size_t)(g0 + t) * D + d]);",
     "v[t] = hgo_bf16_to_f32(rows[(size_t)t * D + d]);"),
    ("pack_msb_first", "if ((q >> k) & 1u) row[pos / 8] |= (uint8_t)(1u << (pos % 8));",
     "if ((q >> k) & 1u) row[pos / 8] |= (uint8_t)(1u << (7 - pos % 8));"),
    ("span_offset_dropped", "size_t cache_off = slice_off + (size_t)c->img_start * D;",
     "size_t cache_off = slice_off;"),
    ("span_offset_dropped_in_quantize",
     "return hgo_quantize_slice(c, X, slice + (size_t)c->img_start * c->D, codes, meta);",
     "return hgo_quantize_slice(c, X, slice, codes, meta);"),
    ("akvq_no_inverse_rotation", "if (c->base == HGO_AKVQ && X == 0) hgo_fwht_norm(y, D);", "(void)0;"),
    ("akvq_rotates_values", "if (c->base == HGO_AKVQ && X == 0) hgo_fwht_norm(v, D);",
     "if (c->base == HGO_AKVQ) hgo_fwht_norm(v, D);"),
    ("kivi_meta_size_per_token", "return ng * (uint64_t)c->D;", "return ng;"),
    ("k_only_side_v_sized", "int pv = c->keys_only ? 0 : P;", "int pv = P;"),
    ("negative_zero_min_kept", "if (m16 == 0x8000u) m16 = 0;", ""),
    ("no_scale_floor", "if (s16 != 0 && hgo_bf16_to_f32(s16) < 0x1p-126f) s16 = 0x0080u; /* 2^-126 */", ""),
    ("zero_range_not_special", "if (s16 == 0) {", "if (s16 == 0 && 0) {"),
    ("kivi_whole_image_only", "for (int t = 0; t < T; ++t) v[t] = hgo_bf16_to_f32(slice[(size_t)t * D + d]);",
     "for (int t = 0; t < n; ++t) v[t] = hgo_bf16_to_f32(slice[(size_t)(s0 + t) * D + d]);"),
    ("kivi_whole_codes_unshifted", "put_code(codes + (size_t)t * row_bytes, b, d, q[s0 + t]);",
     "put_code(codes + (size_t)t * row_bytes, b, d, q[t]);"),
    ("select_difference", "sc[i] = gb[i] + ob[i];", "sc[i] = gb[i] - ob[i];"),
    ("select_interleaved_groups", "int i = l * Hkv + hq / rep;", "int i = l * Hkv + hq % Hkv;"),
    ("select_g_not_standardized", "zscore(gb, n);", ""),
    ("select_ties_to_upper", "if (!mask[i] && (best < 0 || sc[i] > sc[best])) best = i;",
     "if (!mask[i] && (best < 0 || sc[i] >= sc[best])) best = i;"),
    ("select_mean_off_by_one", "  mean /= n;", "  mean /= n + 1;"),
    ("retain_count_floor", "return (int)((num + 500) / 1000);", "return (int)(num / 1000);"),
    ("retain_smallest", "if (!taken[i] && (best < 0 || sqnorm[i] > sqnorm[best])) best = i;",
     "if (!taken[i] && (best < 0 || sqnorm[i] < sqnorm[best])) best = i;"),
    ("retain_ties_upper", "if (!taken[i] && (best < 0 || sqnorm[i] > sqnorm[best])) best = i;",
     "if (!taken[i] && (best < 0 || sqnorm[i] >= sqnorm[best])) best = i;"),
    ("sqnorm_running_sum", "for (int i = 0; i < w; ++i) a[i] = a[2 * i] + a[2 * i + 1];",
     "if (w == 1) for (int d = 1; d < D; ++d) a[0] = a[0] + a[d];"),
    ("sqnorm_l1", "    a[d] = x * x;", "    a[d] = fabsf(x);"),
    ("sqnorm_of_rotated_key", "    a[d] = x * x;\n  }",
     "    a[d] = x;\n  }\n  hgo_fwht_norm(a, D);\n  for (int d = 0; d < D; ++d) a[d] = a[d] * a[d];"),
    ("retain_norm_span_offset_dropped",
     "const uint16_t* keys = j->in[0] + ((size_t)s * c->T + c->img_start) * D;",
     "const uint16_t* keys = j->in[0] + (size_t)s * c->T * D;"),
    ("retain_values_from_keys",
     "const uint16_t* rows = j->in[X] + ((size_t)s * c->T + c->img_start) * D;",
     "const uint16_t* rows = j->in[0] + ((size_t)s * c->T + c->img_start) * D;"),
    ("restore_skips_values", "      uint16_t* rows = out[X] + ((size_t)s * c->T + c->img_start) * D;",
     "      if (X == 1) continue;\n      uint16_t* rows = out[X] + ((size_t)s * c->T + c->img_start) * D;"),
    ("retain_ret_sized_for_all_heads", "out->ret_k = (uint64_t)uk * B * k * D * 2;",
     "out->ret_k = (uint64_t)LH * B * k * D * 2;"),
]


def _run_mutant(name, old, new, tmp):
    src = open(SRC).read()
    assert src.count(old) == 1, f"{name}: pattern must occur exactly once"
    d = os.path.join(tmp, name)
    os.makedirs(d)
    shutil.copy(os.path.join(ROOT, "oracle", "hg_oracle.h"), d)
    with open(os.path.join(d, "hg_oracle.c"), "w") as f:
        f.write(src.replace(old, new))
    so = os.path.join(d, "lib.so")
    subprocess.check_call(["gcc", "-O2", "-fno-fast-math", "-ffp-contract=off", "-fPIC",
                           "-shared", "-pthread", "-w", "-o", so,
                           os.path.join(d, "hg_oracle.c"), "-lm"])
    env = dict(os.environ, HG_ORACLE_LIB=so, OMP_NUM_THREADS="1")
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
                        os.path.join(ROOT, "tests", "test_oracle_pins.py"),
                        os.path.join(ROOT, "tests", "test_oracle_cache.py"),
                        os.path.join(ROOT, "tests", "test_select_pins.py"),
                        os.path.join(ROOT, "tests", "test_oracle_retain.py")],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    return name, r.returncode


def test_every_planted_mistake_fails_a_pin():
    tmp = tempfile.mkdtemp(prefix="hg_mutants_")
    try:
        workers = max(1, min(8, (os.cpu_count() or 2)))
        with cf.ThreadPoolExecutor(workers) as ex:
            results = list(ex.map(lambda m: _run_mutant(*m, tmp), MUTANTS))
    finally:
        shutil.rmtree(tmp, ignore_errors=True)
    survivors = [n for n, rc in results if rc == 0]
    assert not survivors, f"mutants not caught by any pin: {survivors}"
