"""Host-side pieces of bench.py that run without a GPU: the byte accounting the
roofline figures divide by, the oracle baseline leg on every option, and the
rows of the measured-results table."""
import ast
import os

import numpy as np
import pytest

import bench
import oracle
import synthkv

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.mark.parametrize("over", [{}, {"base": "kivi", "kivi_group": 0}, {"base": "akvq", "retain_permille": 20},
                                  {"keys_only": 1}, {"img_len": 0}])
def test_algorithmic_bytes_by_hand(over):
    """Quantize bytes: BF16 image rows of K and V read once, every packed
    buffer written once; whole-sequence KIVI keys add the text rows of each
    quantized key slice; retention adds the norms (written and read), the
    token list and the retained rows (read and written)."""
    w = synthkv.WORKLOADS["tiny"].with_(**over)
    cfg = oracle.make_config(**w.config_fields())
    sz = oracle.sizes(cfg, synthkv.protect_mask(w))
    img = w.L * w.B * w.H * w.img_len * w.D * 2
    packed = sum(sz[n] for n in ("codes_k", "meta_k", "side_k", "codes_v", "meta_v", "side_v"))
    text = sz["n_unprot_k"] * w.B * (w.T - w.img_len) * w.D * 2 if over.get("kivi_group") == 0 and w.img_len else 0
    rows = sz["ret_k"] + sz["ret_v"]
    ab = bench.algorithmic_bytes(w, sz)
    assert ab["quant"] == 2 * img + text + packed + 2 * sz["norm_k"] + sz["ret_idx"] + 2 * rows
    assert ab["dequant"] == 2 * img + packed + sz["ret_idx"] + 2 * rows
    assert bench.fake_quantize_bytes(w, sz) == 4 * img + text + 2 * sz["norm_k"] + sz["ret_idx"] + 2 * rows


@pytest.mark.parametrize("over", [{}, {"base": "kivi", "kivi_group": 0}, {"base": "akvq", "retain_permille": 20}])
def test_cpu_baseline_every_option(over):
    """The oracle leg runs on every option the table uses, and reports the
    rate over the step's algorithmic bytes."""
    w = synthkv.WORKLOADS["tiny"].with_(**over)
    K, V = synthkv.gen_kv(w)
    r = bench.cpu_baseline(w, K, V, synthkv.protect_mask(w), 0.05, threads=1)
    assert r["kind"] == "oracle" and r["cores"] == 1 and r["value"] > 0
    assert np.isfinite(r["image_tokens_per_s"]) and r["image_tokens_per_s"] > 0


def _test_functions(path: str) -> set:
    with open(os.path.join(ROOT, path)) as f:
        tree = ast.parse(f.read())
    return {n.name for n in tree.body if isinstance(n, ast.FunctionDef) and n.name.startswith("test_")}


def test_table_rows():
    """Every table row names a distinct configuration, a workload that exists
    and a GPU parity test that exists."""
    labels = [bench.table_label(*r) for r in bench.TABLE_ROWS]
    assert len(set(labels)) == len(labels)
    for name, over, op in bench.TABLE_ROWS:
        assert name in synthkv.WORKLOADS and op in ("step", "fakequant")
        synthkv.WORKLOADS[name].with_(**over)
        path, test = bench.table_parity_test(name, over, op).split("::")
        assert test.split("[")[0] in _test_functions(path), (name, over, op)
