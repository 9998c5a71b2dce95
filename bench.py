"""Throughput of the LM-operator row evaluation on one MI355X.

A step is one lmop_eval_rows call over the whole table: early dedup, the
batched prefill of every row's suffix against the shared prefix's KV
(W4A16 GEMMs, attention, norms), the constrained LM head, and (integer
types) the decode steps.  The shared prefix is computed once before the
timed region (lmop_set_prefix), weights and prefix KV are resident in HBM.

Default workload: the 8B-shape LM filter (32 layers, d 4096, 32/8 heads,
SwiGLU 14336, vocab 128256, int4 g32 weights; 10,000 rows, shared prefix 512,
suffix lognormal mean 60 clipped to [8, 512]; enum over 24 tokens).
Prints one JSON line.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_F16_TFLOPS = 2500.0   # MI355X dense fp16/bf16 MFMA
PEAK_HBM_GBS = 8000.0      # MI355X HBM3E
GEMM_SRC = os.path.join(ROOT, "paper_2606_31808_amd", "csrc", "gemm.hip")
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "gemm_w4a16_hbm_traffic.json")
COPY_BYTES = 1 << 30       # plain copy used to calibrate the HBM byte counters
# Kernel durations in the timed region come from HIP events around every
# PROF_PERIOD-th launch of each kernel: events around all ~8,500 launches of
# an 8B step add ~0.9% to it.  5 shares no factor with 16 or 32 layers, so
# every layer (the last one's short launches included) is in the sample.
PROF_PERIOD = 5


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def gemm_roofline(stats):
    """Dominant kernel family: the weight GEMMs (all four projections), W4A16
    or, with FP8 weights, W8A16."""
    fp8 = any(n.startswith("gemm_w8a16") for n in stats)
    fam = "gemm_w8a16" if fp8 else "gemm_w4a16"
    names = [n for n in stats if n.startswith(fam)]
    ms = sum(stats[n]["ms"] for n in names)
    fl = sum(stats[n]["flops"] for n in names)
    timed = sum(stats[n]["timed"] for n in names)
    if ms <= 0 or timed == 0:
        return None
    ach = fl / (ms * 1e-3) / 1e12
    algo_bytes = sum(stats[n]["bytes"] for n in names) / timed
    return {"bound": "mfma", "kernel": f"{fam} (qkv, o, gate/up, down)", "achieved": ach,
            "peak": PEAK_F16_TFLOPS, "unit": "TFLOP/s", "frac": ach / PEAK_F16_TFLOPS,
            "traffic": None if fp8 else measured_traffic(),
            "algorithmic_bytes_per_launch": algo_bytes,
            "launches": sum(stats[n]["launches"] for n in names), "timed_launches": timed,
            "avg_launch_ms": ms / timed, "flops_per_launch": fl / timed}


def _src_hash():
    """SHA-256 prefix of the GEMM source's code: // comments, trailing blanks
    and empty lines are dropped, so that a comment edit does not void the
    recorded traffic counters while any change to the code does."""
    import hashlib
    import re
    with open(GEMM_SRC) as f:
        lines = [re.sub(r"\s*//.*$", "", l).rstrip() for l in f]
    code = "\n".join(l for l in lines if l)
    return hashlib.sha256(code.encode()).hexdigest()[:16]


def measured_traffic():
    """HBM bytes per W4A16 GEMM launch from the committed PMC summary, if it was
    taken on the current kernel source; otherwise None."""
    try:
        with open(TRAFFIC_FILE) as f:
            t = json.load(f)
    except (OSError, ValueError):
        return None
    return t["bytes_per_launch"] if t.get("gemm_src_sha256_16") == _src_hash() else None


def _bench_line(log_path):
    """The JSON line a bench run printed (its stdout went to log_path)."""
    with open(log_path) as f:
        lines = [l for l in f if l.startswith("{")]
    return json.loads(lines[-1])


def _is_w4_gemm(name):
    # gemm_kernel<MI, weight format, epilogue, waves>; format 1 = int4
    if "gemm_kernel<" not in name:
        return False
    args = name.split("gemm_kernel<")[1].split(">")[0].split(",")
    return len(args) >= 2 and args[1].strip() in ("1", "true")


def _timed_gemm_rows(rows, n_timed):
    """The last n_timed W4A16 GEMM dispatches: the timed steps come after the
    shared-prefix pass and the warmup, so these are exactly the timed launches."""
    g = sorted((r for r in rows if _is_w4_gemm(r["Kernel_Name"])), key=lambda r: int(r["Dispatch_Id"]))
    return g[-n_timed:]


def pmc_summary(root):
    """Turns four rocprofv3 --pmc runs (GEMM FETCH_SIZE / WRITE_SIZE over one
    timed step, plain copy FETCH_SIZE / WRITE_SIZE, under `root`) into the
    traffic summary."""
    import csv
    import glob

    def rows(d):
        out = []
        for fn in glob.glob(os.path.join(root, d, "*counter_collection.csv")):
            out.extend(csv.DictReader(open(fn)))
        return out

    def gemm_mean(d, counter):
        n = _bench_line(os.path.join(root, d + ".log"))["roofline"]["launches"]
        sel = _timed_gemm_rows([r for r in rows(d) if r["Counter_Name"] == counter], n)
        assert len(sel) == n, (d, len(sel), n)
        return sum(float(r["Counter_Value"]) for r in sel) / n, n

    def copy_mean(d, counter):
        v = [float(r["Counter_Value"]) for r in rows(d)
             if r["Counter_Name"] == counter and "copy" in r["Kernel_Name"].lower()]
        return sum(v) / len(v)

    f_kib, f_n = gemm_mean("pmc_fetch", "FETCH_SIZE")
    w_kib, _ = gemm_mean("pmc_write", "WRITE_SIZE")
    cf = copy_mean("pmc_copy_fetch", "FETCH_SIZE")
    cw = copy_mean("pmc_copy_write", "WRITE_SIZE")
    # KiB as counted for a copy that moves COPY_BYTES each way -> bytes per counted KiB
    kf = COPY_BYTES / (cf * 1024.0)
    kw = COPY_BYTES / (cw * 1024.0)
    fetch_b = f_kib * 1024.0 * kf
    write_b = w_kib * 1024.0 * kw
    out = {"gemm_src_sha256_16": _src_hash(), "launches": f_n, "fetch_bytes_per_launch": fetch_b,
           "write_bytes_per_launch": write_b, "bytes_per_launch": fetch_b + write_b,
           "copy_scale_fetch": kf, "copy_scale_write": kw,
           "copy_fetch_kib": cf, "copy_write_kib": cw}
    with open(TRAFFIC_FILE, "w") as f:
        json.dump(out, f, indent=1)
    print(json.dumps(out))


def mfma_summary(root):
    """MFMA utilisation of the timed step's kernels from one rocprofv3 --pmc
    run of the bench (SQ_VALU_MFMA_BUSY_CYCLES, GRBM_GUI_ACTIVE; under
    root/pmc_mfma, the bench line in root/pmc_mfma.log).  Utilisation = MFMA
    busy cycles summed over all SIMDs / (GPU busy cycles of one XCD x 1024
    SIMDs); GRBM_GUI_ACTIVE comes summed over the 8 XCDs."""
    import csv
    import glob
    xcds, simds = 8, 1024
    rows = []
    for fn in glob.glob(os.path.join(root, "pmc_mfma", "*counter_collection.csv")):
        rows.extend(csv.DictReader(open(fn)))
    n = _bench_line(os.path.join(root, "pmc_mfma.log"))["roofline"]["launches"]
    by_id = {}
    for r in rows:
        d = by_id.setdefault(int(r["Dispatch_Id"]), {"name": r["Kernel_Name"]})
        d[r["Counter_Name"]] = d.get(r["Counter_Name"], 0.0) + float(r["Counter_Value"])
    gemm_ids = sorted(i for i, d in by_id.items() if _is_w4_gemm(d["name"]))[-n:]
    first = gemm_ids[0]

    def family(name):
        if _is_w4_gemm(name):
            epi = name.split("gemm_kernel<")[1].split(",")[2].strip()
            return {"1": "W4A16 GEMM, residual add (o, down)", "2": "W4A16 GEMM, SwiGLU (gate/up)",
                    "4": "W4A16 GEMM, QKV + RoPE (qkv)", "0": "W4A16 GEMM, fp16 store"}.get(epi, epi)
        if "gemm_kernel<" in name:
            return "W8A16 GEMM (FP8 weights)"
        if "head2_kernel" in name or "head_kernel" in name:
            return "LM head GEMM"
        if "attn_kernel" in name:
            return "attention"
        return None

    agg = {}
    for i, d in by_id.items():
        if i < first:
            continue
        fam = family(d["name"])
        if fam is None:
            continue
        a = agg.setdefault(fam, [0, 0.0, 0.0, 0.0])
        a[0] += 1
        a[1] += d.get("SQ_VALU_MFMA_BUSY_CYCLES", 0.0)
        a[2] += d.get("GRBM_GUI_ACTIVE", 0.0) / xcds * simds
        a[3] += d.get("SQ_INSTS_MFMA", 0.0)
    print(f"timed step: {n} W4A16 GEMM dispatches (bench: {n})")
    print("| kernel family | dispatches | MFMA instructions | MFMA busy (of all SIMD cycles) |")
    print("|---|---|---|---|")
    tot = [0, 0.0, 0.0, 0.0]
    for fam in sorted(agg):
        a = agg[fam]
        print(f"| {fam} | {a[0]} | {a[3]:.4g} | {100.0 * a[1] / a[2]:.1f}% |")
        if fam.startswith("W4A16"):
            for k in range(4):
                tot[k] += a[k]
    print(f"| all W4A16 GEMMs | {tot[0]} | {tot[3]:.4g} | {100.0 * tot[1] / tot[2]:.1f}% |")


def trace_summary(root):
    """Per-kernel durations of the timed W4A16 GEMM launches from a
    `rocprofv3 --kernel-trace` run of the default bench command (trace under
    root/prof_full, the bench line in root/prof_full.json)."""
    import csv
    import glob
    res = _bench_line(os.path.join(root, "prof_full.json"))
    n = res["roofline"]["launches"]
    rows = []
    for fn in glob.glob(os.path.join(root, "prof_full", "*kernel_trace.csv")):
        rows.extend(csv.DictReader(open(fn)))
    sel = _timed_gemm_rows(rows, n)
    dur = lambda r: (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) * 1e-6
    by = {}
    for r in sel:
        by.setdefault(r["Kernel_Name"], []).append(dur(r))
    total = sum(sum(v) for v in by.values())
    print(f"timed W4A16 GEMM launches: {len(sel)} (bench: {n})")
    for k, v in sorted(by.items()):
        print(f"  {k}: {len(v)} launches, avg {sum(v) / len(v):.4f} ms")
    print(f"family average: trace {total / len(sel):.4f} ms, bench HIP events "
          f"{res['roofline']['avg_launch_ms']:.4f} ms")


def head_roofline(stats):
    """The logit pass: the full-vocabulary head GEMM (streams the 1.05 GB head
    weight per launch), or with --head-restricted the allowed-token dot
    products (hidden rows + |A| weight rows per launch)."""
    name = "head_gemm" if "head_gemm" in stats else "head_restricted"
    s = stats.get(name)
    if not s or s["ms"] <= 0 or s["timed"] == 0:
        return None
    gbs = s["bytes"] / (s["ms"] * 1e-3) / 1e9
    tfl = s["flops"] / (s["ms"] * 1e-3) / 1e12
    return {"kernel": name, "bound": "hbm", "achieved": gbs, "peak": PEAK_HBM_GBS, "unit": "GB/s",
            "frac": gbs / PEAK_HBM_GBS, "tflops": tfl, "launches": s["launches"],
            "timed_launches": s["timed"], "avg_launch_ms": s["ms"] / s["timed"],
            "bytes_per_launch": s["bytes"] / s["timed"]}


DECODE_TRAFFIC_FILE = os.path.join(ROOT, "profiles", "decode_gemm_map_int_8b_traffic.json")


def decode_roofline(stats):
    """Integer/automaton decode steps: one forward over every live row of a
    decode group per step, so each decode-step GEMM streams all its weights
    for the few thousand rows still decoding.  The bound is whichever roof
    the launch's algorithmic intensity (FLOP per algorithmic byte: the
    weights at 0.5625 B per int4 parameter with its scale, plus activations
    in and out) puts it under: MFMA above the ridge (2.5 PFLOP/s over
    8 TB/s = 312.5 FLOP/B), HBM below it.  Both rates are reported, with the
    counter-measured bytes per launch when the committed PMC summary was
    taken on the current GEMM source."""
    names = [n for n in stats if n.startswith("decode_gemm_")]
    ms = sum(stats[n]["ms"] for n in names)
    timed = sum(stats[n]["timed"] for n in names)
    if ms <= 0 or timed == 0:
        return None
    by = sum(stats[n]["bytes"] for n in names)
    fl = sum(stats[n]["flops"] for n in names)
    gbs = by / (ms * 1e-3) / 1e9
    tfl = fl / (ms * 1e-3) / 1e12
    ridge = PEAK_F16_TFLOPS * 1e12 / (PEAK_HBM_GBS * 1e9)
    mfma = fl / by > ridge
    traffic = None
    try:
        with open(DECODE_TRAFFIC_FILE) as f:
            t = json.load(f)
        if t.get("gemm_src_sha256_16") == _src_hash():
            traffic = t["bytes_per_launch"]
    except (OSError, ValueError):
        pass
    ach, peak, unit = (tfl, PEAK_F16_TFLOPS, "TFLOP/s") if mfma else (gbs, PEAK_HBM_GBS, "GB/s")
    return {"kernel": "decode-step W4A16 GEMMs (qkv, o, gate/up, down)",
            "bound": "mfma" if mfma else "hbm", "achieved": ach, "peak": peak, "unit": unit,
            "frac": ach / peak, "flop_per_byte": fl / by, "tflops": tfl, "gbs": gbs,
            "launches": sum(stats[n]["launches"] for n in names),
            "timed_launches": timed, "avg_launch_ms": ms / timed,
            "algorithmic_bytes_per_launch": by / timed, "traffic": traffic}


def decode_pmc_summary(root):
    """HBM bytes per decode-step GEMM launch of map_int_8b from two rocprofv3
    --pmc runs of one step (FETCH_SIZE under root/pmc_dec_fetch, WRITE_SIZE
    under root/pmc_dec_write, bench lines in their .log) and the plain-copy
    calibration runs (root/pmc_copy_fetch, root/pmc_copy_write).  The decode
    steps of one decode group follow all of its prefill batches, so with one
    group (the default memory budget) the decode launches are the last
    W4A16 GEMM dispatches of the step."""
    import csv
    import glob

    def rows(d):
        out = []
        for fn in glob.glob(os.path.join(root, d, "*counter_collection.csv")):
            out.extend(csv.DictReader(open(fn)))
        return out

    def dec_mean(d, counter):
        line = _bench_line(os.path.join(root, d + ".log"))
        n = line["decode_roofline"]["launches"]
        sel = _timed_gemm_rows([r for r in rows(d) if r["Counter_Name"] == counter], n)
        assert len(sel) == n, (d, len(sel), n)
        return sum(float(r["Counter_Value"]) for r in sel) / n, n, line

    def copy_mean(d, counter):
        v = [float(r["Counter_Value"]) for r in rows(d)
             if r["Counter_Name"] == counter and "copy" in r["Kernel_Name"].lower()]
        return sum(v) / len(v)

    f_kib, n, line = dec_mean("pmc_dec_fetch", "FETCH_SIZE")
    w_kib, _, _ = dec_mean("pmc_dec_write", "WRITE_SIZE")
    kf = COPY_BYTES / (copy_mean("pmc_copy_fetch", "FETCH_SIZE") * 1024.0)
    kw = COPY_BYTES / (copy_mean("pmc_copy_write", "WRITE_SIZE") * 1024.0)
    out = {"gemm_src_sha256_16": _src_hash(), "workload": "map_int_8b", "launches": n,
           "fetch_bytes_per_launch": f_kib * 1024.0 * kf, "write_bytes_per_launch": w_kib * 1024.0 * kw,
           "bytes_per_launch": f_kib * 1024.0 * kf + w_kib * 1024.0 * kw,
           "algorithmic_bytes_per_launch": line["decode_roofline"]["algorithmic_bytes_per_launch"],
           "avg_launch_ms_under_counters": line["decode_roofline"]["avg_launch_ms"]}
    with open(DECODE_TRAFFIC_FILE, "w") as f:
        json.dump(out, f, indent=1)
    print(json.dumps(out))


def pass_rooflines(stats):
    """The other passes of a step: attention against MFMA (its FLOPs are the
    visible query-key pairs the host counts), RMSNorm against HBM (fp32 in,
    fp16 out)."""
    out = {}
    a = stats.get("attention")
    if a and a["ms"] > 0 and a["flops"] > 0 and a["timed"] > 0:
        t = a["flops"] / (a["ms"] * 1e-3) / 1e12
        out["attention"] = {"bound": "mfma", "achieved": t, "peak": PEAK_F16_TFLOPS,
                            "unit": "TFLOP/s", "frac": t / PEAK_F16_TFLOPS,
                            "avg_launch_ms": a["ms"] / a["timed"]}
    r = stats.get("rmsnorm")
    if r and r["ms"] > 0 and r["timed"] > 0:
        g = r["bytes"] / (r["ms"] * 1e-3) / 1e9
        out["rmsnorm"] = {"bound": "hbm", "achieved": g, "peak": PEAK_HBM_GBS, "unit": "GB/s",
                          "frac": g / PEAK_HBM_GBS, "avg_launch_ms": r["ms"] / r["timed"]}
    return out


def _blas_info():
    """The BLAS numpy's matmuls run on, and the threads it uses."""
    try:
        from threadpoolctl import threadpool_info
        for i in threadpool_info():
            if i.get("user_api") == "blas":
                return {"blas": f"{i.get('internal_api')} {i.get('version')}",
                        "threads": int(i.get("num_threads", 0))}
    except Exception:  # threadpoolctl missing or unreadable: report what numpy says
        pass
    return {"blas": "unknown", "threads": int(os.environ.get("OMP_NUM_THREADS", os.cpu_count() or 1))}


def cpu_baseline(weights, shape, wl, n_rows, seed=2):
    """The oracle (fp32 numpy, as it stands) on the host cores, timed like the
    GPU leg: the per-layer int4 dequantisation (kept for later calls) and the
    shared prefix are timed apart from the rows, as the GPU side loads weights
    and computes the prefix outside its timed region.  The rows are n_rows of
    the parity sample (the longest, the shortest, the first, the last and
    seeded others); rows time = (prefix + rows) - prefix alone."""
    import numpy as np
    from oracle import OracleLM
    from synth import parity_rows
    orc = OracleLM(weights, shape, dtype=np.float32, cache_dequant=True)
    t0 = time.perf_counter()
    for l in range(shape.n_layers):
        orc.layer_weights(l)
    orc.head_weights()
    t_deq = time.perf_counter() - t0
    allowed = wl.automaton if getattr(wl, "automaton", None) is not None else wl.allowed
    t0 = time.perf_counter()
    orc.eval_rows(wl.prefix, [], wl.kind, allowed, eos=wl.eos, max_tokens=wl.max_tokens)
    t_pre = time.perf_counter() - t0
    rows = parity_rows(wl, n_rows, seed)
    sub = wl.subset(rows)
    t0 = time.perf_counter()
    orc.eval_workload(sub)
    t_all = time.perf_counter() - t0
    t_rows = max(t_all - t_pre, 1e-9)
    rps = len(rows) / t_rows
    info = _blas_info()
    return {"value": rps, "unit": "rows/s", "cores": info["threads"], "kind": "oracle",
            "sample": f"{len(rows)} rows of the parity sample ({sub.n_suffix_tokens} suffix "
                      f"tokens) against a {len(wl.prefix)}-token shared prefix, fp32 numpy; "
                      f"rows {t_rows:.1f} s = prefix + rows {t_all:.1f} s - prefix alone "
                      f"{t_pre:.1f} s; int4 dequantisation {t_deq:.1f} s, once",
            "suffix_tokens_per_s": sub.n_suffix_tokens / t_rows,
            "prefix_s": t_pre, "dequant_s": t_deq,
            "full_table_s_extrapolated": t_deq + t_pre + wl.n_rows / rps,
            "blas": info["blas"], "blas_threads": info["threads"],
            "host_cpus": os.cpu_count()}


def device_peaks(dev_index=0):
    """MFMA peak re-derived from the clock the device reports (f16 dense:
    4,096 FLOP per CU per clock on gfx950), and the HBM copy bandwidth a
    plain device copy reaches, beside the published figures."""
    import ctypes
    import torch
    out = {"mfma_f16_spec_tflops": PEAK_F16_TFLOPS, "hbm_spec_gbs": PEAK_HBM_GBS}
    try:
        hip = ctypes.CDLL("libamdhip64.so")
        clk, ncu = ctypes.c_int(), ctypes.c_int()
        # hipDeviceAttributeClockRate (kHz) = 5, hipDeviceAttributeMultiprocessorCount = 63
        if hip.hipDeviceGetAttribute(ctypes.byref(clk), 5, dev_index) == 0 and \
                hip.hipDeviceGetAttribute(ctypes.byref(ncu), 63, dev_index) == 0:
            out["clock_mhz"] = clk.value / 1e3
            out["compute_units"] = ncu.value
            out["mfma_f16_derived_tflops"] = ncu.value * 4096 * clk.value * 1e3 / 1e12
    except OSError:
        pass
    n = COPY_BYTES // 4
    src = torch.ones(n, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    best = None
    for _ in range(5):
        a.record()
        dst.copy_(src)
        b.record()
        b.synchronize()
        ms = a.elapsed_time(b)
        best = ms if best is None else min(best, ms)
    out["hbm_copy_gbs"] = 2 * COPY_BYTES / (best * 1e-3) / 1e9
    del src, dst
    torch.cuda.empty_cache()
    return out


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=2)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--workload", default="filter_8b")
    ap.add_argument("--rows", type=int, default=None, help="truncate the table")
    ap.add_argument("--batch-tokens", type=int, default=0)
    ap.add_argument("--limit", type=int, default=0,
                    help="LIMIT k early exit: stop once k rows have value --limit-value")
    ap.add_argument("--limit-value", type=int, default=1)
    ap.add_argument("--weights", default="int4_g32", choices=["int4_g32", "fp8_e4m3"],
                    help="weight format of the linear maps")
    ap.add_argument("--cascade", action="store_true",
                    help="cascade filtering: a bool predicate first, the workload on its survivors")
    ap.add_argument("--cascade-model", default="",
                    help="model shape of the cascade's first predicate (default: the workload's)")
    ap.add_argument("--head-restricted", action="store_true",
                    help="compute only the allowed tokens' logits (logprob_full is NaN)")
    ap.add_argument("--cpu-rows", type=int, default=32,
                    help="rows of the parity sample the oracle baseline evaluates")
    ap.add_argument("--workspace-gb", type=float, default=0.0,
                    help="carve the library's scratch from a torch allocation of this size")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="only run one plain 1 GiB device copy (counter calibration)")
    ap.add_argument("--pmc-summary", metavar="DIR",
                    help="summarise the rocprofv3 --pmc runs under DIR and exit")
    ap.add_argument("--mfma-summary", metavar="DIR",
                    help="summarise an SQ_VALU_MFMA_BUSY_CYCLES pass under DIR/pmc_mfma and exit")
    ap.add_argument("--decode-pmc-summary", metavar="DIR",
                    help="summarise the decode-step GEMM counter runs under DIR and exit")
    ap.add_argument("--trace-summary", metavar="DIR",
                    help="summarise the rocprofv3 --kernel-trace run under DIR and exit")
    args = ap.parse_args()
    if args.pmc_summary:
        pmc_summary(args.pmc_summary)
        return
    if args.decode_pmc_summary:
        decode_pmc_summary(args.decode_pmc_summary)
        return
    if args.trace_summary:
        trace_summary(args.trace_summary)
        return
    if args.mfma_summary:
        mfma_summary(args.mfma_summary)
        return
    if args.calibrate_copy:
        import torch
        src = torch.ones(COPY_BYTES // 4, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copied_bytes": COPY_BYTES}))
        return
    if args.gpus != 1:
        print(json.dumps({"error": "the library runs on one GPU; --gpus must be 1"}))
        sys.exit(2)

    import numpy as np
    import torch
    from paper_2606_31808_amd import lmop as L
    from synth import make_weights, make_workload

    wl = make_workload(args.workload, n_rows=args.rows)
    # the first predicate of a cascade: a yes/no choice between two seeded tokens
    wl.cascade_allowed = np.random.default_rng(99).choice(wl.shape.vocab, 2, replace=False)
    shape = wl.shape
    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream(dev).cuda_stream
    log(f"[bench] generating {shape.name} weights on the GPU")
    t0 = time.perf_counter()
    w = make_weights(shape, seed=1234, device=dev, fmt=args.weights)
    torch.cuda.synchronize()
    log(f"[bench] weights {time.perf_counter() - t0:.1f} s; loading into the library")
    # room for the longest sequence (LLMQA prompts run past the default 4,096)
    longest = len(wl.prefix) + int(np.diff(wl.offsets).max()) + wl.max_tokens
    if wl.children is not None:
        longest += max(len(c) for c in wl.children)
    max_seq = 0 if longest <= 4096 else -(-longest // 1024) * 1024
    ctx = L.Context(shape, device=0, stream=stream, max_seq=max_seq)
    t0 = time.perf_counter()
    ctx.load_weights(w)
    t_load = time.perf_counter() - t0
    # the library holds its own repacked copy: keep the inputs on the host
    # only (the oracle baseline reads them there)
    w = w.to("cpu")
    torch.cuda.empty_cache()
    ws_buf = None
    if args.workspace_gb > 0:
        ws_buf = torch.empty(int(args.workspace_gb * (1 << 30)), dtype=torch.uint8, device=dev)
        ctx.set_workspace(ws_buf.data_ptr(), ws_buf.numel())
    t0 = time.perf_counter()
    root = ctx.set_prefix(wl.prefix)
    kids = None
    row_prefix = None
    if wl.children is not None:
        kids = ctx.set_prefixes(wl.children, parent=root)
        row_prefix = [kids[int(i)] for i in wl.row_child]
    t_prefix = time.perf_counter() - t0
    log(f"[bench] load {t_load:.2f} s, prefix {t_prefix * 1e3:.1f} ms")

    cascade = {}
    first_ctx, first_root = ctx, root
    if args.cascade and args.cascade_model:
        # the first predicate on a smaller model of the same vocabulary
        from synth import SHAPES
        s1 = SHAPES[args.cascade_model]
        w1 = make_weights(s1, seed=4321, device=dev)
        first_ctx = L.Context(s1, device=0, stream=stream, max_seq=max_seq)
        first_ctx.load_weights(w1)
        del w1
        torch.cuda.empty_cache()
        first_root = first_ctx.set_prefix(wl.prefix)
        if row_prefix:
            raise SystemExit("--cascade-model supports tables without child prefixes")

    def step():
        mask = None
        if args.cascade:
            # cascade filtering: a yes/no predicate on every row first, then
            # the workload's own predicate on the rows it kept
            t0 = time.perf_counter()
            first, _ = first_ctx.eval_rows(wl.tokens, wl.offsets, 0, wl.cascade_allowed,
                                           prefix=None if row_prefix else first_root,
                                           row_prefix=row_prefix,
                                           max_batch_tokens=args.batch_tokens)
            mask = first["value"] == 1
            cascade.update(first_ms=(time.perf_counter() - t0) * 1e3, kept=int(mask.sum()))
        t0 = time.perf_counter()
        out, _ = ctx.eval_rows(wl.tokens, wl.offsets, wl.kind, wl.type_spec, eos=wl.eos,
                               max_tokens=wl.max_tokens, prefix=None if row_prefix else root,
                               row_prefix=row_prefix, max_batch_tokens=args.batch_tokens,
                               head_restricted=args.head_restricted, limit=args.limit,
                               limit_value=args.limit_value, row_mask=mask)
        cascade.update(second_ms=(time.perf_counter() - t0) * 1e3)
        return out

    for i in range(args.warmup):
        t0 = time.perf_counter()
        step()
        log(f"[bench] warmup {i}: {time.perf_counter() - t0:.2f} s")
    # every PROF_PERIOD-th launch of each kernel is timed with HIP events
    ctx.set_profiling(PROF_PERIOD)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        out = step()
        log(f"[bench] step {i} done")
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    stats = ctx.kernel_stats()
    ctx.set_profiling(False)
    ms_step = elapsed * 1e3 / args.steps
    rows = wl.n_rows
    n_tok = wl.n_suffix_tokens
    if args.limit:
        # a LIMIT query: the rows it evaluated (the rest were skipped)
        rows = int(np.sum(out["n_tokens"] > 0))
        n_tok = int(sum(wl.offsets[r + 1] - wl.offsets[r] for r in range(wl.n_rows)
                        if out["n_tokens"][r] > 0))
    value = rows / (ms_step * 1e-3)
    rep, n_unique = L.lmop_dedup_rows(wl.tokens, wl.offsets,
                                      None if wl.row_child is None else wl.row_child)
    wdesc = "int4-g32" if args.weights == "int4_g32" else "fp8-e4m3 per-channel"
    res = {
        "metric": "rows/sec, 8B-shape W4 LM filter (10k rows); MFMA util %, HBM GB/s",
        "value": value, "unit": "rows/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": ms_step, "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": f"f16 ({wdesc} weights, fp32 accum)",
        "data": f"synthetic (seeded uniform token ids, random-init N(0,0.02) {wdesc} weights)",
        "config": {"workload": wl.name, "model_shape": shape.name, "rows": rows,
                   "unique_rows": n_unique, "unique_rows_per_s": n_unique / (ms_step * 1e-3),
                   "prefix_tokens": len(wl.prefix),
                   "suffix_tokens": n_tok, "suffix_tokens_per_s": n_tok / (ms_step * 1e-3),
                   "batch_tokens": args.batch_tokens or 16384, "parallelism": "single GPU",
                   "head": "restricted" if args.head_restricted else "full vocabulary",
                   "weights": args.weights},
        **({"limit": {"k": args.limit, "value": args.limit_value, "rows_in_table": wl.n_rows,
                      "rows_evaluated": rows, "ms_per_query": ms_step}} if args.limit else {}),
        **({"cascade": {"first_model": args.cascade_model or shape.name,
                        "rows": wl.n_rows, "kept_by_first": cascade.get("kept"),
                        "first_ms": cascade.get("first_ms"),
                        "second_ms": cascade.get("second_ms")}} if args.cascade else {}),
        "roofline": gemm_roofline(stats),
        "head_roofline": head_roofline(stats),
        **({"decode_roofline": dec} if (dec := decode_roofline(stats)) else {}),
        "pass_rooflines": pass_rooflines(stats),
        "load_weights_s": t_load, "set_prefix_ms": t_prefix * 1e3,
        # device memory: what the library held at most (weights, prefix KV,
        # scratch; with a workspace its scratch is the workspace), against the
        # paper's 16 GB GPU
        "memory": {**{k: v for k, v in ctx.memory().items()},
                   "library_peak_gb": (ctx.memory()["device_peak"]
                                       + ctx.memory()["workspace_bytes"]) / 1e9,
                   "torch_peak_gb": torch.cuda.max_memory_allocated() / 1e9},
        "device": device_peaks(),
        # mean timed duration x all launches, per step
        "kernels_ms_per_step": {k: v["ms"] / max(v["timed"], 1) * v["launches"] / args.steps
                                for k, v in sorted(stats.items())},
        "profiling_period": PROF_PERIOD,
    }
    if not args.no_cpu_baseline:
        log("[bench] oracle CPU baseline")
        res["cpu_baseline"] = cpu_baseline(w, shape, wl, args.cpu_rows)
    print(json.dumps(res), flush=True)
    ctx.close()


if __name__ == "__main__":
    main()
