"""Bench: one step = quantize+pack and dequantize of a whole synthetic KV cache
(every layer, batch row and KV head; K and V) through libheadguard on one
MI355X.  Prints one JSON line.

Default workload: the LLaVA-NeXT-7B-shaped cache, the largest of the five
single-GPU workloads (32 layers x 4 rows x 32 KV heads x 3008 tokens x
head_dim 128, 2880 image tokens, KIVI-style 2-bit: keys per channel over
groups of 32 image tokens, values per token; 128 of 1024 heads protected,
keys only), inputs resident in HBM.

Algorithmic bytes per call: every image row of K and V is read once
(2 bytes per element) and the packed outputs (codes, metadata, BF16 side
store) are written once; dequantize moves the same bytes in the other
direction.  Text rows are never written; they are read only where the
method needs them, by KIVI-style keys with one range over the whole sequence.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
HBM_PEAK_GBPS = 8000.0  # MI355X HBM3E, vendor figure
QUANT_KERNEL = "quantize_kernel"
DEQUANT_KERNEL = "dequantize_kernel"
FAKE_KERNEL = "fake_quantize_kernel"
_CSRC = "paper_2609_35800_amd/csrc/"
# the device sources that decide what each timed call reads and writes; a
# counter measurement is reported only while their text is unchanged.  The
# whole-sequence KIVI key kernels and the token-retention kernels count only
# for the workloads whose calls launch them.
KERNEL_SOURCES = {
    QUANT_KERNEL: tuple(_CSRC + f for f in ("quantize.hip", "hg_device.h", "hg_kernels.h")),
    DEQUANT_KERNEL: tuple(_CSRC + f for f in ("dequantize.hip", "hg_device.h", "hg_kernels.h")),
    FAKE_KERNEL: tuple(_CSRC + f for f in ("fakequant.hip", "hg_device.h", "hg_kernels.h")),
}
KIVI_WHOLE_SOURCE = _CSRC + "kivi_seq.hip"
RETAIN_SOURCE = _CSRC + "retain.hip"
# The measured-results table: the five workloads (the 72B-shaped one at each
# bit width), the whole-sequence KIVI keys, the 2 % token retention and a
# 128K-token context with whole-sequence keys, each as a quantize + dequantize
# step, and the one-pass mode on three of them: (workload, option overrides,
# op).
TABLE_ROWS = (
    ("tiny", {}, "step"), ("qwen2.5-vl-7b", {}, "step"), ("llava-next-7b", {}, "step"),
    ("internvl-8b", {}, "step"), ("72b-long", {"bits": 2}, "step"), ("72b-long", {"bits": 3}, "step"),
    ("72b-long", {"bits": 4}, "step"), ("llava-next-7b", {"kivi_group": 0}, "step"),
    ("internvl-8b", {"retain_permille": 20}, "step"), ("qwen2.5-vl-7b-128k", {}, "step"),
    ("qwen2.5-vl-7b", {}, "fakequant"), ("llava-next-7b", {"kivi_group": 0}, "fakequant"),
    ("internvl-8b", {"retain_permille": 20}, "fakequant"),
)


def table_label(name: str, over: dict, op: str) -> str:
    parts = [name]
    if "bits" in over:
        parts.append(f"{over['bits']}-bit")
    if over.get("kivi_group") == 0:
        parts.append("whole-sequence keys")
    if over.get("retain_permille"):
        parts.append(f"{over['retain_permille'] / 10:g} % retention")
    if op == "fakequant":
        parts.append("one-pass")
    return ", ".join(parts)


def table_parity_test(name: str, over: dict, op: str) -> str:
    """The full-size GPU test that compares every slice of the row's call
    with the oracle."""
    if over.get("kivi_group") == 0:
        return ("tests/test_gpu_kivi_whole.py::test_full_size_llava_one_pass[False]" if op == "fakequant"
                else "tests/test_gpu_kivi_whole.py::test_full_size_llava")
    if over.get("retain_permille"):
        return ("tests/test_gpu_retain.py::test_full_size_internvl_two_percent_one_pass[False]" if op == "fakequant"
                else "tests/test_gpu_retain.py::test_full_size_internvl_two_percent")
    if op == "fakequant":
        return f"tests/test_gpu_workloads.py::test_one_pass_out_of_place[{name}]"
    if name == "72b-long":
        return f"tests/test_gpu_workloads.py::test_72b_long_bit_sweep[{over['bits']}]"
    return f"tests/test_gpu_workloads.py::test_workload[{name}]"


RESULTS_DOC = "BASELINE.md"  # the document whose results section --fill-baseline writes
RESULTS_HEADER = "## 4. Measured results"


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="llava-next-7b")
    ap.add_argument("--bits", type=int, default=None, help="override the workload's bit width")
    ap.add_argument("--kivi-group", type=int, default=None,
                    help="override the KIVI key group (0: one range over the whole sequence)")
    ap.add_argument("--retain-permille", type=int, default=None,
                    help="AKVQ-style token retention per mille (20 = the paper's 2 %%)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=10.0,
                    help="approximate CPU time budget of the oracle sample")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="accepted for recorded profiling commands; the 1 GiB device copy "
                         "that scales the counters now always runs")
    ap.add_argument("--quant-only", action="store_true",
                    help="time only the quantize launches (for profiling that kernel)")
    ap.add_argument("--table", metavar="JSON",
                    help="measure every workload of the measured-results table (quantize and "
                         "dequantize median times, oracle on the host cores) into JSON")
    ap.add_argument("--fill-baseline", metavar="JSON",
                    help="(no GPU) write the rows of a --table run as the results document's "
                         "measured-results section")
    ap.add_argument("--op", default="step", choices=["step", "fakequant"],
                    help="step: quantize+pack then dequantize (the default line); "
                         "fakequant: the one-pass simulated quantization alone")
    return ap.parse_args()


def _code_only(text: str) -> str:
    """C++ source without its comments and blank lines (string and character
    literals kept): what decides the compiled kernels."""
    out, i, n = [], 0, len(text)
    while i < n:
        c = text[i]
        if c in "\"'":
            j = i + 1
            while j < n and text[j] != c:
                j += 2 if text[j] == "\\" else 1
            out.append(text[i:j + 1])
            i = j + 1
        elif text.startswith("//", i):
            while i < n and text[i] != "\n":
                i += 1
        elif text.startswith("/*", i):
            k = text.find("*/", i + 2)
            i = n if k < 0 else k + 2
        else:
            out.append(c)
            i += 1
    return "\n".join(line.rstrip() for line in "".join(out).splitlines() if line.strip())


def kernel_sources(kernel: str, w=None) -> tuple:
    """Device sources of a call on workload w (without w: every source the
    call can launch)."""
    srcs = list(KERNEL_SOURCES[kernel])
    kivi_whole = w is None or (w.base == "kivi" and w.kivi_group == 0)
    if kernel in (QUANT_KERNEL, FAKE_KERNEL) and kivi_whole:
        srcs.append(KIVI_WHOLE_SOURCE)
    if w is None or w.retain_permille:
        srcs.append(RETAIN_SOURCE)
    return tuple(srcs)


def kernel_source_hash(kernel: str = QUANT_KERNEL, w=None) -> str:
    """Hash of the code (comments and blank lines removed) of the device
    sources of a call on workload w; a traffic record is reported only while
    it matches."""
    h = hashlib.sha256()
    for p in kernel_sources(kernel, w):
        with open(os.path.join(ROOT, p), encoding="utf-8") as f:
            h.update(_code_only(f.read()).encode())
    return h.hexdigest()[:16]


def variant_name(w) -> str:
    """Workload name plus the options that change which kernels run:
    e.g. qwen2.5-vl-7b_b2, llava-next-7b_kivi-whole_b2, internvl-8b_retain20_b2."""
    name = w.name
    if w.base == "kivi" and w.kivi_group == 0:
        name += "_kivi-whole"
    if w.retain_permille:
        name += f"_retain{w.retain_permille}"
    return f"{name}_b{w.bits}"


def traffic_record(w, kernel: str = QUANT_KERNEL):
    """The committed rocprofv3 FETCH_SIZE / WRITE_SIZE record of this workload
    variant's call, if one exists and was taken on the current sources."""
    path = os.path.join(ROOT, "profiles", f"traffic_{kernel}_{variant_name(w)}.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        rec = json.load(f)
    if rec.get("kernel_source_hash") != kernel_source_hash(kernel, w):
        return None
    return rec


def traffic_from_profile(w, kernel: str = QUANT_KERNEL):
    """HBM bytes per call (all kernels of the timed call) measured by the
    rocprofv3 FETCH_SIZE and WRITE_SIZE counters, if a committed measurement
    of this workload variant exists and was taken on the current sources."""
    rec = traffic_record(w, kernel)
    return rec.get("hbm_bytes_per_launch") if rec else None


def algorithmic_bytes(w, sizes) -> dict:
    """Bytes each call must move at least.  Quantize: the image rows of K and V
    read once, every packed buffer written once; KIVI-style keys with one range
    over the whole sequence (kivi_group 0) also read the text rows of every
    quantized key slice, whose values enter the range; with token retention
    also the key norms read back by the selection and the retained rows read
    again (the selection needs every norm first).  Dequantize: the packed
    buffers read, the image rows written; with retention the retained rows are
    written over the reconstruction."""
    img_elems = w.L * w.B * w.H * w.img_len * w.D
    read = 2 * img_elems * 2  # K and V image rows, BF16
    if w.base == "kivi" and w.kivi_group == 0 and w.img_len > 0:
        read += sizes["n_unprot_k"] * w.B * (w.T - w.img_len) * w.D * 2
    write = sum(sizes[n] for n in ("codes_k", "meta_k", "side_k", "codes_v", "meta_v", "side_v"))
    rows = sizes.get("ret_k", 0) + sizes.get("ret_v", 0)
    quant_extra = 2 * sizes.get("norm_k", 0) + sizes.get("ret_idx", 0) + 2 * rows
    dequant_extra = sizes.get("ret_idx", 0) + 2 * rows
    text = read - 2 * img_elems * 2  # text rows the range reads (quantize only)
    return {"quant": read + write + quant_extra, "dequant": read - text + write + dequant_extra,
            "read": read, "write": write}


def fake_quantize_bytes(w, sizes) -> int:
    """Bytes the out-of-place one-pass call must move: every image row of K
    and V read once and written once, plus the text rows of quantized key
    slices that KIVI-style keys over the whole sequence read for the range;
    with token retention also the key norms written and read back by the
    selection, the token lists written, and the retained rows read from the
    input again and written over their simulated reconstruction (the
    selection needs every norm, so it follows the pass that writes them)."""
    ab = algorithmic_bytes(w, sizes)
    img = 2 * w.L * w.B * w.H * w.img_len * w.D * 2
    rows = sizes.get("ret_k", 0) + sizes.get("ret_v", 0)
    retain = 2 * sizes.get("norm_k", 0) + sizes.get("ret_idx", 0) + 2 * rows
    return img + ab["read"] + retain


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(w, K, V, mask, budget_s: float, threads: int = 0):
    """The CPU oracle on a bounded sample of the same workload, quantize then
    dequantize: whole passes over the cache, repeated to fill about budget_s
    of wall time, or its first layers (all rows, heads, K and V) when one pass
    would exceed the budget.  threads = 0: one per host core, at most 16."""
    import oracle  # test infrastructure: the CPU baseline leg only
    import synthkv
    threads = threads or max(1, min(os.cpu_count() or 1, 16))

    def prepare(nl):
        sub = w.with_(L=nl)
        cfg = oracle.make_config(**sub.config_fields())
        m = np.ascontiguousarray(mask[: nl * w.H])
        return sub, cfg, m, synthkv.bf16_bits(K[:nl]), synthkv.bf16_bits(V[:nl])

    def one_pass(cfg, m, Kb, Vb, Ko, Vo):
        t0 = time.perf_counter()
        pk = oracle.quantize(cfg, Kb, Vb, m, threads=threads)
        oracle.dequantize(cfg, m, pk, Ko, Vo, threads=threads)
        return time.perf_counter() - t0

    sub, cfg, m, Kb, Vb = prepare(1)
    dt1 = one_pass(cfg, m, Kb, Vb, np.zeros_like(Kb), np.zeros_like(Vb))
    nl = int(max(1, min(w.L, budget_s / max(dt1, 1e-6))))
    sub, cfg, m, Kb, Vb = prepare(nl)
    Ko, Vo = np.zeros_like(Kb), np.zeros_like(Vb)
    total, passes = 0.0, 0
    while passes == 0 or total < budget_s:
        dt = one_pass(cfg, m, Kb, Vb, Ko, Vo)
        total += dt
        passes += 1
    ab = algorithmic_bytes(sub, oracle.sizes(cfg, m))
    per_pass = total / passes
    return {"value": round((ab["quant"] + ab["dequant"]) / per_pass / 1e9, 4), "unit": "GB/s",
            "cores": threads, "kind": "oracle", "cpu_model": cpu_model(),
            "host_cores": os.cpu_count(),
            "sample": f"{nl} of {w.L} layers of the same workload (all rows, heads, K and V), "
                      f"quantize+dequantize, {passes} pass(es), {total:.2f} s wall",
            # image tokens of the whole cache, scaled by the fraction of layers in the sample
            "image_tokens_per_s": round(w.B * w.img_len * nl / w.L / per_pass, 1)}


def host_call_us(hg, cfg, K, V, mask, packed, stream, calls: int = 50) -> float:
    """Host time of one hg_quantize call: argument and pointer checks, mask
    routing and the kernel launches, through ctypes with the arguments
    prepared once; median over `calls` calls (their GPU work is drained
    afterwards)."""
    import ctypes as C
    import torch
    lib = hg.library()
    m = np.ascontiguousarray(mask, dtype=np.uint8)
    pk = hg.hg_packed(**{n: (t.data_ptr() if t.numel() else None) for n, t in packed.items()})
    args = (C.byref(cfg), K.data_ptr(), V.data_ptr(), m.ctypes.data_as(C.c_void_p), C.byref(pk),
            stream.cuda_stream)
    ts = []
    for _ in range(calls):
        t0 = time.perf_counter_ns()
        rc = lib.hg_quantize(*args)
        ts.append(time.perf_counter_ns() - t0)
        if rc:
            raise RuntimeError(hg.hg_last_error())
    torch.cuda.synchronize()
    return float(np.median(ts)) / 1e3


def device_copy_gbps(stream) -> float:
    """A plain device-to-device copy of 1 GiB on the same stream: the practical
    bandwidth the kernels are compared with besides the vendor peak (its
    rocprofv3 counters also scale FETCH_SIZE and WRITE_SIZE to bytes)."""
    import torch
    n = 1 << 30
    a = torch.empty(n, dtype=torch.uint8, device="cuda")
    b = torch.empty_like(a)
    b.copy_(a)
    cev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(5)]
    for e0, e1 in cev:
        e0.record(stream)
        b.copy_(a)
        e1.record(stream)
    torch.cuda.synchronize()
    ms = float(np.mean([e0.elapsed_time(e1) for e0, e1 in cev]))
    del a, b
    return 2 * n / (ms * 1e-3) / 1e9


def bench_fakequant(args, hg, w, cfg, mask, K, V):
    """One-pass simulated quantization, out of place: every image row of K and
    V is read once and written once (protected rows copied); see
    fake_quantize_bytes."""
    import torch
    Ko, Vo = torch.empty_like(K), torch.empty_like(V)
    ws = hg.alloc_fake_workspace(cfg, mask)
    stream = torch.cuda.current_stream()
    for _ in range(args.warmup):
        hg.hg_fake_quantize(cfg, K, V, mask, Ko, Vo, ws, stream=stream)
    torch.cuda.synchronize()
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(args.steps)]
    t0 = time.perf_counter()
    for e0, e1 in ev:
        e0.record(stream)
        hg.hg_fake_quantize(cfg, K, V, mask, Ko, Vo, ws, stream=stream)
        e1.record(stream)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    ms = float(np.mean([a.elapsed_time(b) for a, b in ev]))
    nbytes = fake_quantize_bytes(w, hg.hg_packed_sizes(cfg, mask))
    gbps = nbytes / (ms * 1e-3) / 1e9
    copy_gbps = device_copy_gbps(stream)
    print(json.dumps({
        "metric": "fake-quantize (one-pass simulated quantization) HBM GB/s",
        "value": round(nbytes * args.steps / elapsed / 1e9, 2), "unit": "GB/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(elapsed / args.steps * 1e3, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f32",
        "data": "synthetic (seeded N(0,1) BF16 KV with outlier key channels; no model weights)",
        "config": {"workload": w.name, "bits": w.bits, "base": w.base, "keys_only": w.keys_only,
                   **({"kivi_group": w.kivi_group} if w.base == "kivi" else {}),
                   **({"retain_permille": w.retain_permille} if w.retain_permille else {})},
        "image_tokens_per_s": round(w.B * w.img_len / (ms * 1e-3), 1),
        "device_copy_GBps": round(copy_gbps, 1),
        "pct_of_device_copy": round(100 * gbps / copy_gbps, 1),
        "roofline": {"bound": "hbm", "kernel": FAKE_KERNEL, "achieved": round(gbps, 1),
                     "peak": HBM_PEAK_GBPS, "unit": "GB/s", "frac": round(gbps / HBM_PEAK_GBPS, 4),
                     "bytes_per_launch": nbytes, "ms": round(ms, 4),
                     "traffic": traffic_from_profile(w, FAKE_KERNEL)},
    }), flush=True)


def measure_table(args) -> None:
    """The measured-results table: for each row, the median quantize and
    dequantize call times (or the one-pass call's, out of place) over `steps`
    calls (HIP events on the launch stream, inputs resident in HBM), the GB/s
    and image tokens/s they give, the committed counter ratios, and the oracle
    on the host cores (one thread and all of them, quantize + dequantize, which
    is also what the one-pass mode computes)."""
    import torch
    import paper_2609_35800_amd as hg
    import synthkv
    stream = torch.cuda.current_stream()
    rows, oracle_runs = [], {}
    for name, over, op in TABLE_ROWS:
        w = synthkv.WORKLOADS[name].with_(**over)
        mask = synthkv.protect_mask(w)
        cfg = hg.make_config(**w.config_fields())
        sizes = hg.hg_packed_sizes(cfg, mask)
        K, V = synthkv.gen_kv(w, device="cuda")
        Ko, Vo = torch.empty_like(K), torch.empty_like(V)
        if op == "fakequant":  # out of place, as bench_fakequant
            ws = hg.alloc_fake_workspace(cfg, mask)
            run = lambda: hg.hg_fake_quantize(cfg, K, V, mask, Ko, Vo, ws, stream=stream)  # noqa: E731
            calls = (("hg_fake_quantize", fake_quantize_bytes(w, sizes), FAKE_KERNEL),)
        else:
            ab = algorithmic_bytes(w, sizes)
            packed = hg.alloc_packed(cfg, mask)
            q = lambda: hg.hg_quantize(cfg, K, V, mask, packed, stream=stream)  # noqa: E731
            d = lambda: hg.hg_dequantize(cfg, mask, packed, Ko, Vo, stream=stream)  # noqa: E731
            calls = (("hg_quantize", ab["quant"], QUANT_KERNEL), ("hg_dequantize", ab["dequant"], DEQUANT_KERNEL))
        ev = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(args.steps)]
        for _ in range(args.warmup):
            if op == "fakequant":
                run()
            else:
                q()
                d()
        for e0, e1, e2 in ev:
            e0.record(stream)
            if op == "fakequant":
                run()
            else:
                q()
            e1.record(stream)
            if op != "fakequant":
                d()
            e2.record(stream)
        torch.cuda.synchronize()
        times = [float(np.median([a.elapsed_time(b) for a, b, _ in ev])),
                 float(np.median([b.elapsed_time(c) for _, b, c in ev]))]
        key = (name, tuple(sorted(over.items())))
        if key not in oracle_runs:  # the one-pass rows reuse their step row's oracle timing
            oracle_runs[key] = (cpu_baseline(w, K, V, mask, args.cpu_seconds / 2),
                                cpu_baseline(w, K, V, mask, args.cpu_seconds / 4, threads=1))
        cb_n, cb_1 = oracle_runs[key]
        label = table_label(name, over, op)
        for (call, nbytes, kernel), ms in zip(calls, times):
            rec = traffic_record(w, kernel)
            rows.append({
                "config": label, "workload": w.name, "bits": w.bits, "overrides": over, "op": op, "call": call,
                "median_ms": round(ms, 4), "GBps": round(nbytes / (ms * 1e-3) / 1e9, 1),
                "pct_of_peak": round(100 * nbytes / (ms * 1e-3) / 1e9 / HBM_PEAK_GBPS, 1),
                "bytes": nbytes, "traffic_ratio": rec.get("ratio_to_algorithmic") if rec else None,
                "image_tokens_per_s": round(w.B * w.img_len / (ms * 1e-3), 1),
                "oracle_1_thread_GBps": cb_1["value"], "oracle_n_thread_GBps": cb_n["value"],
                "oracle_threads": cb_n["cores"], "oracle_sample": cb_n["sample"],
                "parity_test": table_parity_test(name, over, op),
            })
            print(json.dumps(rows[-1]), flush=True)
        del K, V, Ko, Vo
        torch.cuda.empty_cache()
    out = {"rows": rows, "steps": args.steps, "warmup": args.warmup, "cpu_model": cpu_model(),
           "host_cores": os.cpu_count(), "date": time.strftime("%Y-%m-%d")}
    with open(args.table, "w") as f:
        json.dump(out, f, indent=1)


def fill_baseline(path: str) -> None:
    """Writes the rows of a --table run as the results document's
    measured-results section (everything from its header to the next section
    is replaced)."""
    with open(path) as f:
        t = json.load(f)
    fmt = lambda v, spec: "—" if v is None else format(v, spec)  # noqa: E731
    lines = [RESULTS_HEADER, "",
             f"Written by `python bench.py --fill-baseline` from a `python bench.py --table` run on one MI355X "
             f"({t['date']}; median of {t['steps']} calls after {t['warmup']} warm-up steps, HIP events on the "
             "launch stream, inputs resident in HBM; bytes are the algorithmic bytes of `bench.py`). Counter "
             "ratios come from the committed rocprofv3 records under `profiles/` when they were taken on the "
             "current kernel sources. The oracle columns time the CPU oracle (quantize + dequantize, the "
             "step's byte count; for the one-pass rows too, since that mode computes the dequantize of the "
             f"quantize) on the box's host ({t['cpu_model']}): one thread, and one per core "
             f"(N = {t['rows'][0]['oracle_threads']}). Parity: every slice compared with the oracle, bit for "
             "bit, by the GPU test named.", "",
             "| Config | Call | Median time | GB/s | % of 8 TB/s | rocprof bytes ÷ algorithmic bytes | "
             "Image tokens/s | Oracle 1-thread | Oracle N-thread | Parity |",
             "|---|---|---|---|---|---|---|---|---|---|"]
    import synthkv
    kernels = {"hg_quantize": QUANT_KERNEL, "hg_dequantize": DEQUANT_KERNEL, "hg_fake_quantize": FAKE_KERNEL}
    for r in t["rows"]:
        # counter ratios from the records committed now (taken on the current sources)
        w = synthkv.WORKLOADS[r["workload"]].with_(**r.get("overrides", {"bits": r["bits"]}))
        rec = traffic_record(w, kernels[r["call"]])
        r["traffic_ratio"] = rec.get("ratio_to_algorithmic") if rec else None
        lines.append(f"| {r['config']} | `{r['call']}` | {r['median_ms'] * 1e3:.1f} µs | {r['GBps']:,.0f} | "
                     f"{r['pct_of_peak']:.1f} | {fmt(r['traffic_ratio'], '.4f')} | "
                     f"{r['image_tokens_per_s']:.3g} | {r['oracle_1_thread_GBps']:.3f} GB/s | "
                     f"{r['oracle_n_thread_GBps']:.2f} GB/s | bit-exact, `{r['parity_test']}` |")
    base = os.path.join(ROOT, RESULTS_DOC)
    with open(base) as f:
        text = f.read()
    i = text.index(RESULTS_HEADER)
    j = text.find("\n## ", i + len(RESULTS_HEADER))
    text = text[:i] + "\n".join(lines) + "\n" + (text[j:] if j >= 0 else "")
    with open(base, "w") as f:
        f.write(text)


def main():
    args = parse()
    if args.fill_baseline:
        return fill_baseline(args.fill_baseline)
    if args.gpus != 1:
        print(f"bench.py measures one GPU only: --gpus {args.gpus} is not supported "
              "(the quantizer's slices are independent; sharding is by KV head, layer or "
              "batch row with no communication).", file=sys.stderr)
        sys.exit(2)

    if args.table:
        return measure_table(args)

    import torch
    import paper_2609_35800_amd as hg
    import synthkv

    w = synthkv.WORKLOADS[args.workload]
    if args.bits is not None:
        w = w.with_(bits=args.bits)
    if args.kivi_group is not None:
        w = w.with_(kivi_group=args.kivi_group)
    if args.retain_permille is not None:
        w = w.with_(retain_permille=args.retain_permille)
    mask = synthkv.protect_mask(w)
    cfg = hg.make_config(**w.config_fields())
    sizes = hg.hg_packed_sizes(cfg, mask)
    ab = algorithmic_bytes(w, sizes)

    K, V = synthkv.gen_kv(w, device="cuda")
    if args.op == "fakequant":
        return bench_fakequant(args, hg, w, cfg, mask, K, V)
    packed = hg.alloc_packed(cfg, mask)
    Ko = torch.empty_like(K)
    Vo = torch.empty_like(V)
    stream = torch.cuda.current_stream()

    # Step i's calls are timed between events bound[i] (recorded before its
    # quantize: the end of step i-1), mid[i] (between quantize and dequantize)
    # and bound[i+1]: two event records per step.
    def step(mid=None, end=None):
        hg.hg_quantize(cfg, K, V, mask, packed, stream=stream)
        if mid is not None and not args.quant_only:
            mid.record(stream)
        if not args.quant_only:
            hg.hg_dequantize(cfg, mask, packed, Ko, Vo, stream=stream)
        if end is not None:
            end.record(stream)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()

    new_ev = lambda: torch.cuda.Event(enable_timing=True)  # noqa: E731
    bound = [new_ev() for _ in range(args.steps + 1)]
    mid = [new_ev() for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    bound[0].record(stream)
    for i in range(args.steps):
        step(mid[i], bound[i + 1])
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0

    if args.quant_only:
        q_ms = [bound[i].elapsed_time(bound[i + 1]) for i in range(args.steps)]
        d_ms = [0.0]
    else:
        q_ms = [bound[i].elapsed_time(mid[i]) for i in range(args.steps)]
        d_ms = [mid[i].elapsed_time(bound[i + 1]) for i in range(args.steps)]
    q_avg = float(np.mean(q_ms))
    d_avg = float(np.mean(d_ms))
    step_bytes = ab["quant"] + (0 if args.quant_only else ab["dequant"])
    value = step_bytes * args.steps / elapsed / 1e9
    q_gbps = ab["quant"] / (q_avg * 1e-3) / 1e9
    d_gbps = ab["dequant"] / (d_avg * 1e-3) / 1e9 if not args.quant_only else None
    traffic = traffic_from_profile(w)

    host_us = host_call_us(hg, cfg, K, V, mask, packed, stream)
    copy_gbps = device_copy_gbps(stream)

    out = {
        "metric": "quantize+pack+dequant HBM GB/s (% of MI355X peak); image KV tokens/s",
        "value": round(value, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(elapsed / args.steps * 1e3, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic (seeded N(0,1) BF16 KV with outlier key channels; no model weights)",
        "config": {"workload": w.name, "L": w.L, "B": w.B, "H_kv": w.H, "T": w.T, "D": w.D,
                   "img_start": w.img_start, "img_len": w.img_len, "bits": w.bits,
                   "base": w.base, "keys_only": w.keys_only, "protected_heads": int(mask.sum()),
                   **({"kivi_group": w.kivi_group} if w.base == "kivi" else {}),
                   **({"retain_permille": w.retain_permille} if w.retain_permille else {}),
                   "parallelism": "single GPU"},
        "pct_of_hbm_peak": round(100 * value / HBM_PEAK_GBPS, 2),
        "device_copy_GBps": round(copy_gbps, 1),
        "quantize_pct_of_device_copy": round(100 * q_gbps / copy_gbps, 1),
        "image_tokens_per_s": round(w.B * w.img_len * args.steps / elapsed, 1),
        "host_us_per_quantize_call": round(host_us, 2),
        "quantize": {"ms": round(q_avg, 4), "median_ms": round(float(np.median(q_ms)), 4),
                     "min_ms": round(float(np.min(q_ms)), 4), "GBps": round(q_gbps, 1),
                     "bytes": ab["quant"], "image_tokens_per_s": round(w.B * w.img_len / (q_avg * 1e-3), 1),
                     "token_vectors_per_s": round(2 * w.L * w.B * w.H * w.img_len / (q_avg * 1e-3), 1)},
        "dequantize": None if args.quant_only else
                      {"ms": round(d_avg, 4), "median_ms": round(float(np.median(d_ms)), 4),
                       "min_ms": round(float(np.min(d_ms)), 4), "GBps": round(d_gbps, 1),
                       "bytes": ab["dequant"]},
        "roofline": {"bound": "hbm", "kernel": QUANT_KERNEL, "achieved": round(q_gbps, 1),
                     "peak": HBM_PEAK_GBPS, "unit": "GB/s", "frac": round(q_gbps / HBM_PEAK_GBPS, 4),
                     "traffic": traffic},
    }
    if not args.no_cpu_baseline:
        cb = cpu_baseline(w, K, V, mask, args.cpu_seconds)
        one = cpu_baseline(w, K, V, mask, args.cpu_seconds / 2, threads=1)
        cb["single_thread"] = {"value": one["value"], "unit": one["unit"], "sample": one["sample"]}
        cb["gpu_speedup"] = round(value / cb["value"], 1)
        cb["gpu_speedup_vs_single_thread"] = round(value / one["value"], 1)
        out["cpu_baseline"] = cb
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
