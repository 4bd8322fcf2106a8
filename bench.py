#!/usr/bin/env python3
"""Throughput of the Cross-Request State Packed Forward on one MI355X.

Workload (default): the steady-state cross-request pipeline of a 32-layer Llama-2-7B-shape
decoder in bf16 (d 4096, 32 heads x 128, SwiGLU 11008, vocab 32000), action length K = 7:
every step packs one new 276-row prefill (256 N(0,1) "vision" rows + 20 instruction token
ids) with the 6 single decode rows of the requests in flight (M = 282 rows), runs all 32
layers over a ring of 8 slots x 288 positions (slots wrap every 8 steps), and emits 7 greedy
tokens through the LM head.  Weights are random N(0, 0.02) (seeded draws on the GPU).

One "step" is one packed forward (af_packed_forward) plus its host bookkeeping; W warm-up
steps (>= K - 1 so every timed step is a full M = 282 step), then K timed steps bracketed by
device synchronizations.  A second pass over the same number of steps records HIP events
around every kernel launch (on the launch stream) for the per-kernel roofline figures.

Prints one JSON line (stdout); progress goes to stderr.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "packed tokens/s + packed steps/s at 7B shape; % MFMA bf16 peak, % HBM BW"
PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0       # MI355X HBM3E


def log(*a):
    print("[bench]", *a, file=sys.stderr, flush=True)


EXTRAS = ("sequential", "attention_stress", "sweep", "stress", "k_sweep", "copy_shift", "naive_pipe")


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=30)
    p.add_argument("--warmup", type=int, default=10)
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--cpu-steps", type=int, default=2, help="whole 32-layer steps of the CPU oracle sample")
    p.add_argument("--no-timing-pass", action="store_true")
    p.add_argument("--no-extra", action="store_true",
                   help="skip the measurements beside the packed step (baseline, attention, sweeps, ablations)")
    p.add_argument("--extra", action="append", choices=EXTRAS, default=None,
                   help="run only these measurements beside the packed step (repeatable; default: all)")
    p.add_argument("--copy-calibration", action="store_true",
                   help="before warm-up, run one streaming copy of COPY_BYTES (read once, written once) "
                        "whose hardware-counter readings scale the FETCH_SIZE / WRITE_SIZE of the others")
    p.add_argument("--summarize-pmc", nargs=2, metavar=("FETCH_CSV", "WRITE_CSV"),
                   help="print the traffic summary of two rocprofv3 --pmc runs (FETCH_SIZE, WRITE_SIZE "
                        "counter_collection.csv files of a --copy-calibration run) and exit")
    p.add_argument("--summarize-mfma", nargs=2, metavar=("COUNTER_CSV", "KERNEL_STATS_CSV"),
                   help="print MFMA work per kernel class from a rocprofv3 --pmc SQ_INSTS_VALU_MFMA_MOPS_BF16 "
                        "SQ_VALU_MFMA_BUSY_CYCLES run and a --kernel-trace --stats run of the same command, and exit")
    p.add_argument("--summarize-stats", metavar="KERNEL_STATS_CSV",
                   help="print a per-kernel table of a rocprofv3 --kernel-trace --stats kernel_stats.csv and exit")
    p.add_argument("--summarize-stalls", nargs=4, metavar=("SQ_CSV", "LDS_CSV", "TCP_CSV", "KERNEL_STATS_CSV"),
                   help="print wait, MFMA, LDS and L1/L2 request figures per kernel class from three rocprofv3 "
                        "--pmc runs (the counter sets of the profiling recipe) and a --kernel-trace --stats run, "
                        "and exit")
    return p.parse_args()


COPY_BYTES = 1 << 30        # calibration copy: 1 GiB read + 1 GiB written, far beyond the 256 MB last-level cache
KERNELS_SRC = os.path.join(ROOT, "paper_2512_20276_amd", "csrc", "af_gemm.hip")
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic_gemm_gateup_7b_m282.md")


def kernels_sha256():
    import hashlib
    with open(KERNELS_SRC, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()


def measured_traffic():
    """HBM bytes per gate/up launch from the committed counter summary, or None when the kernel
    source has changed since the counters were taken."""
    try:
        kv = dict(l.split(":", 1) for l in open(TRAFFIC_FILE).read().splitlines() if l.startswith("- ") and ":" in l)
    except OSError:
        return None
    kv = {k[2:].strip(): v.strip().strip("`") for k, v in kv.items()}
    if kv.get("kernel_source_sha256") != kernels_sha256():
        return None
    return int(kv["traffic_bytes_per_launch"])


def _kernel_class(name: str) -> str:
    """Maps a kernel name (mangled or demangled) to the label used in the summaries."""
    import re
    if any(k in name for k in ("gemm_kernel", "gemm32_kernel", "gemm32x2_kernel", "gemm32c_kernel",
                               "gemm32w_kernel")):
        epi = (re.search(r"gemm32(?:x2|c|w)?_kernelI(?:Li\d+E)*Li(\d+)EEEv", name)    # bf16, mangled
               or re.search(r"gemm32(?:x2|c|w)?_kernel<[^>]*?(\d+)>", name)            # bf16, demangled
               or re.search(r",\s*(\d)>\s*\(", name) or re.search(r",\s*\(af::Epi\)(\d)>", name)
               or re.search(r"GemmCfgI(?:Li\d+E)+EELi(\d)E", name))                  # fp32 kernel
        e = int(epi.group(1)) if epi else -1
        if "gemm32c_kernel" in name and e == 0:  # its split-K instance: partial sums only
            return "gemm (split-K partials: QKV / O / down)"
        return {0: "gemm (store)", 1: "gemm (f32 store, LM head)", 2: "gemm (+residual: O / down)",
                3: "gemm (gate/up + SwiGLU)", 4: "gemm (QKV + RoPE + ring write)"}.get(e, "gemm")
    for key in ("splitk_reduce", "resid_norm_kernel", "attention_kernel", "rmsnorm_kernel", "embed_kernel",
                "argmax_kernel", "frag_pack_kernel"):
        if key in name:
            return key
    if "neg" in name.lower():
        return "calibration copy (torch.neg, out=)"
    return name[:60]


def summarize_stats(path):
    import csv
    rows = list(csv.DictReader(open(path)))
    print("| kernel | calls | avg us | min us | max us | total ms | % |")
    print("|---|---:|---:|---:|---:|---:|---:|")
    for r in sorted(rows, key=lambda r: -float(r["TotalDurationNs"])):
        print(f"| `{_kernel_class(r['Name'])}`: `{r['Name'][:100]}` | {r['Calls']} | {float(r['AverageNs']) / 1e3:.2f} | "
              f"{float(r['MinNs']) / 1e3:.2f} | {float(r['MaxNs']) / 1e3:.2f} | "
              f"{float(r['TotalDurationNs']) / 1e6:.3f} | {float(r['Percentage']):.2f} |")


def summarize_pmc(fetch_csv, write_csv):
    """Average FETCH_SIZE / WRITE_SIZE (KiB per dispatch) per kernel class, scaled by the readings
    of the calibration copy, which fetches and writes COPY_BYTES."""
    import csv
    from collections import defaultdict

    def per_class(path, counter):
        acc = defaultdict(lambda: [0.0, 0])
        for r in csv.DictReader(open(path)):
            if r["Counter_Name"] != counter:
                continue
            a = acc[_kernel_class(r["Kernel_Name"])]
            a[0] += float(r["Counter_Value"])
            a[1] += 1
        return {k: (v / n, n) for k, (v, n) in acc.items()}

    f, w = per_class(fetch_csv, "FETCH_SIZE"), per_class(write_csv, "WRITE_SIZE")
    cal = "calibration copy (torch.neg, out=)"
    fs = COPY_BYTES / (f[cal][0] * 1024)
    ws = COPY_BYTES / (w[cal][0] * 1024)
    print(f"calibration: copy of {COPY_BYTES} B reads FETCH_SIZE {f[cal][0]:.0f} KiB, WRITE_SIZE {w[cal][0]:.0f} KiB "
          f"-> scale fetch x{fs:.4f}, write x{ws:.4f}\n")
    print("| kernel class | dispatches | FETCH KiB/dispatch | WRITE KiB/dispatch | HBM bytes/dispatch (scaled) |")
    print("|---|---:|---:|---:|---:|")
    for k in sorted(f, key=lambda k: -f[k][0] * f[k][1]):
        wk = w.get(k, (0.0, 0))[0]
        tb = f[k][0] * 1024 * fs + wk * 1024 * ws
        print(f"| {k} | {f[k][1]} | {f[k][0]:.0f} | {wk:.0f} | {tb:.4g} |")
    # attention launches by instance and grid (the decode-only instance at a given grid is one
    # workload, e.g. the 56 decode rows x 32 heads of the stress mix)
    def per_grid(path, counter):
        acc = defaultdict(lambda: [0.0, 0])
        for r in csv.DictReader(open(path)):
            if r["Counter_Name"] != counter or "attention_kernel" not in r["Kernel_Name"]:
                continue
            name = r["Kernel_Name"]
            inst = ("decode-only" if "Lb0E" in name else
                    "four-wave: query tiles + decode rows" if "attention_kernel4" in name else
                    "eight-wave: query tiles + decode-row pairs")
            a = acc[(inst, int(r["Grid_Size"]), int(r["Workgroup_Size"]))]
            a[0] += float(r["Counter_Value"])
            a[1] += 1
        return {k: (v / n, n) for k, (v, n) in acc.items()}
    fa, wa = per_grid(fetch_csv, "FETCH_SIZE"), per_grid(write_csv, "WRITE_SIZE")
    if fa:
        print("\n| attention instance | workgroups | dispatches | FETCH KiB | WRITE KiB | HBM bytes (scaled) |")
        print("|---|---:|---:|---:|---:|---:|")
        for k in sorted(fa, key=lambda k: -fa[k][0]):
            wk = wa.get(k, (0.0, 0))[0]
            print(f"| {k[0]} | {k[1] // k[2]} | {fa[k][1]} | {fa[k][0]:.0f} | {wk:.0f} | "
                  f"{fa[k][0] * 1024 * fs + wk * 1024 * ws:.4g} |")
    g = "gemm (gate/up + SwiGLU)"
    if g in f:
        tb = int(round(f[g][0] * 1024 * fs + w[g][0] * 1024 * ws))
        print(f"\n- traffic_bytes_per_launch: {tb}")
        print(f"- kernel_source_sha256: `{kernels_sha256()}`")


def summarize_mfma(counter_csv, stats_csv):
    """MFMA work per kernel class from SQ_INSTS_VALU_MFMA_MOPS_BF16 (units of 512 flops) and
    SQ_VALU_MFMA_BUSY_CYCLES (matrix-core cycles summed over every SIMD), against the average
    duration of the same class in a --kernel-trace --stats run: busy fraction = busy cycles /
    (duration x 2.4 GHz x 256 CUs x 4 SIMDs)."""
    import csv
    from collections import defaultdict
    acc = defaultdict(lambda: defaultdict(lambda: [0.0, 0]))
    for r in csv.DictReader(open(counter_csv)):
        a = acc[_kernel_class(r["Kernel_Name"])][r["Counter_Name"]]
        a[0] += float(r["Counter_Value"])
        a[1] += 1
    dur = defaultdict(lambda: [0.0, 0])
    for r in csv.DictReader(open(stats_csv)):
        d = dur[_kernel_class(r["Name"])]
        d[0] += float(r["TotalDurationNs"])
        d[1] += int(r["Calls"])
    print("| kernel class | dispatches | MFMA GFLOP/dispatch (counter) | MFMA busy cycles/dispatch | avg us | "
          "counter TFLOP/s | MFMA busy fraction |")
    print("|---|---:|---:|---:|---:|---:|---:|")
    for k, cs in sorted(acc.items(), key=lambda kv: -kv[1].get("SQ_VALU_MFMA_BUSY_CYCLES", [0, 1])[0]):
        mops = cs.get("SQ_INSTS_VALU_MFMA_MOPS_BF16", [0.0, 1])
        busy = cs.get("SQ_VALU_MFMA_BUSY_CYCLES", [0.0, 1])
        n = max(mops[1], 1)
        fl = mops[0] / n * 512
        bc = busy[0] / max(busy[1], 1)
        if fl == 0 and bc == 0:
            continue
        us = dur[k][0] / dur[k][1] / 1e3 if dur[k][1] else float("nan")
        print(f"| {k} | {n} | {fl / 1e9:.3f} | {bc:.4g} | {us:.2f} | {fl / (us * 1e-6) / 1e12:.1f} | "
              f"{bc / (us * 1e-6 * 2.4e9 * 256 * 4):.4f} |")


def summarize_stalls(sq_csv, lds_csv, tcp_csv, stats_csv):
    """Where the waves of each kernel class spend their time, and the L1's outstanding L2 reads.
    Counters (averaged per dispatch, summed over the chip): SQ_WAVE_CYCLES, SQ_WAIT_ANY,
    SQ_WAIT_INST_ANY, SQ_WAIT_INST_LDS, SQ_VALU_MFMA_BUSY_CYCLES; SQ_INSTS_LDS, SQ_LDS_BANK_CONFLICT;
    TCP_TCC_READ_REQ_sum (128-byte L2 reads), TCP_TCC_READ_REQ_LATENCY_sum (their summed latency,
    cycles), TCP_PENDING_STALL_CYCLES_sum.  Reads in flight per CU = summed latency / (duration x
    2.4 GHz x 256 CUs): by Little's law the number of L2 reads each CU keeps outstanding."""
    import csv
    from collections import defaultdict
    acc = defaultdict(lambda: defaultdict(lambda: [0.0, 0]))
    for path in (sq_csv, lds_csv, tcp_csv):
        for r in csv.DictReader(open(path)):
            a = acc[_kernel_class(r["Kernel_Name"])][r["Counter_Name"]]
            a[0] += float(r["Counter_Value"])
            a[1] += 1
    dur = defaultdict(lambda: [0.0, 0])
    for r in csv.DictReader(open(stats_csv)):
        d = dur[_kernel_class(r["Name"])]
        d[0] += float(r["TotalDurationNs"])
        d[1] += int(r["Calls"])
    g = lambda cs, k: cs[k][0] / cs[k][1] if cs.get(k) and cs[k][1] else float("nan")
    print("| kernel class | avg us | waves waiting (any) | waiting on a dependency | on LDS | MFMA busy per SIMD | "
          "LDS bank-conflict cycles / LDS instr | L2 reads / dispatch | avg L2 read latency (cycles) | "
          "L2 reads in flight per CU | L1 pending-stall share |")
    print("|---|---:|---:|---:|---:|---:|---:|---:|---:|---:|---:|")
    for k, cs in sorted(acc.items(), key=lambda kv: -(dur[kv[0]][0] if dur[kv[0]][1] else 0)):
        if not dur[k][1] or "SQ_WAVE_CYCLES" not in cs:
            continue
        us = dur[k][0] / dur[k][1] / 1e3
        cyc = us * 1e-6 * 2.4e9
        wave = g(cs, "SQ_WAVE_CYCLES")
        req, lat = g(cs, "TCP_TCC_READ_REQ_sum"), g(cs, "TCP_TCC_READ_REQ_LATENCY_sum")
        if not (wave > 0 and req > 0):
            continue
        print(f"| {k} | {us:.2f} | {g(cs, 'SQ_WAIT_ANY') / wave:.2f} | {g(cs, 'SQ_WAIT_INST_ANY') / wave:.2f} | "
              f"{g(cs, 'SQ_WAIT_INST_LDS') / wave:.3f} | {g(cs, 'SQ_VALU_MFMA_BUSY_CYCLES') / (cyc * 1024):.3f} | "
              f"{g(cs, 'SQ_LDS_BANK_CONFLICT') / max(g(cs, 'SQ_INSTS_LDS'), 1):.3f} | {req:.4g} | {lat / req:.0f} | "
              f"{lat / (cyc * 256):.1f} | {g(cs, 'TCP_PENDING_STALL_CYCLES_sum') / (cyc * 256):.2f} |")


# ----------------------------------------------------------------------------- algorithmic work
def gemm_work(M, D, F, V, n_emit):
    """Per-launch algorithmic flops and bytes (weights once, activations in and out, bf16)."""
    b = 2
    w = {
        "gemm_qkv": (2 * M * D * 3 * D, b * (3 * D * D + M * D + 3 * M * D)),
        "gemm_o": (2 * M * D * D, b * (D * D + M * D + 2 * M * D)),
        "gemm_gateup": (2 * M * D * 2 * F, b * (2 * F * D + M * D + M * F)),
        "gemm_down": (2 * M * F * D, b * (D * F + M * F + 2 * M * D)),
        "lm_head": (2 * n_emit * D * V, b * (V * D + n_emit * D) + 4 * n_emit * V),
    }
    return w


def attention_bytes(segs, H, hd):
    """Keys and values each row's segment reads (its slot, positions 0..kv_len-1), plus Q in and O out."""
    b = 2
    kv = sum((s[3] + s[1]) * H * hd * 2 * b for s in segs)
    M = sum(s[1] for s in segs)
    return kv + 2 * M * H * hd * b


# ----------------------------------------------------------------------------- extra measurements
def sequential_baseline(af, w, shape, pids, pool, K, n_req=6, warm=2):
    """The plain per-request schedule on the same kernels (the paper's baseline): each request
    alone, a 276-row prefill then K - 1 single-row decode forwards through all layers, with the
    greedy token fed back on the device.  Returns ms per request (one action chunk)."""
    import torch
    L_P = int(pids.numel())
    ring = af.Ring(shape.n_layers, 2, L_P + K, shape.n_heads, shape.head_dim, dtype=torch.bfloat16)
    hidden = torch.empty((L_P, shape.d_model), dtype=torch.bfloat16, device="cuda")
    toks = torch.zeros(K, dtype=torch.int32, device="cuda")
    times = []
    for r in range(warm + n_req):
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        s = ring.append(r, L_P)
        s.flags = af.AF_SEG_EMIT
        af.packed_forward(w, pids, pool[r % len(pool)][:L_P], [s], ring, hidden, None, toks[0:1])
        for k in range(1, K):
            s = ring.append(r, 1)
            s.flags = af.AF_SEG_EMIT
            af.packed_forward(w, toks[k - 1:k], None, [s], ring, hidden[:1], None, toks[k:k + 1])
        ring.release(r)
        torch.cuda.synchronize()
        if r >= warm:
            times.append(time.perf_counter() - t0)
    ring.close()
    return sorted(times)[len(times) // 2] * 1e3


def decode_heavy_attention(af, w, shape, n_pipe=8, K=8, L_P=276, reps=10):
    """Attention of the multi-pipeline stress step (n_pipe pipelines x (L_P prefill + K - 1
    decode rows), pipeline-major, one slot per request: 64 slots x 288), timed by the library's
    per-kernel HIP events inside one layer forward (layer 0 of the loaded model); also the
    decode rows alone.  Ring history is seeded N(0, 1)."""
    import torch
    import workload as wl
    H, hd, D = shape.n_heads, shape.head_dim, shape.d_model
    n_slots, max_pos = n_pipe * K, 288
    ring = af.Ring(1, n_slots, max_pos, H, hd, dtype=torch.bfloat16)
    segs_all, segs_dec, row, row_d = [], [], 0, 0
    for p in range(n_pipe):
        rid0 = 10_000 + p * K
        s = ring.append(rid0, L_P)
        segs_all.append((row, L_P, s.slot, 0, rid0, af.AF_SEG_EMIT))
        row += L_P
        for st in range(1, K):
            rid = rid0 + st
            ring.append(rid, L_P + st - 1)
            s = ring.append(rid, 1)
            segs_all.append((row, 1, s.slot, s.pos0, rid, af.AF_SEG_EMIT))
            segs_dec.append((row_d, 1, s.slot, s.pos0, rid, af.AF_SEG_EMIT))
            row += 1
            row_d += 1
    for sl in range(n_slots):
        kv = wl.draw(("ring history", sl), (2, max_pos, H, hd), device="cuda", dtype=torch.bfloat16)
        ring.write_kv(0, sl, 0, kv[0], kv[1])
    out = {}
    for name, segs, M in (("stress_step", segs_all, row), ("decode_rows_only", segs_dec, row_d)):
        hid = wl.draw(("stress hidden", name), (M, D), device="cuda", dtype=torch.bfloat16)
        af.packed_layer_forward(w, 0, hid.clone(), segs, ring)
        torch.cuda.synchronize()
        w.timing_enable((1 << af.AF_K_COUNT) - 1)
        for _ in range(reps):
            af.packed_layer_forward(w, 0, hid.clone(), segs, ring)
        torch.cuda.synchronize()
        tm = w.timing_read()
        w.timing_enable(0)
        at_ms = tm["attention"][0] / tm["attention"][1]
        nbytes = attention_bytes(segs, H, hd)
        layer_ms = sum(ms for ms, n in tm.values()) / reps
        out[name] = {"M": M, "attention_us": round(at_ms * 1e3, 2), "bytes": nbytes,
                     "GB/s": round(nbytes / (at_ms * 1e-3) / 1e9, 1),
                     "frac_hbm": round(nbytes / (at_ms * 1e-3) / 1e9 / PEAK_HBM_GBS, 4),
                     "layer_kernels_ms": round(layer_ms, 4)}
    ring.close()
    return out


def _reserve(af, ring, specs):
    """Ring reservation of one packed step: specs (request_id, pos0, q_len) in packing order; a
    request not yet resident first gets pos0 positions of history.  Returns segment tuples."""
    segs, row = [], 0
    for rid, pos0, q_len in specs:
        if pos0 > 0:
            ring.append(rid, pos0)
        s = ring.append(rid, q_len)
        segs.append((row, q_len, s.slot, s.pos0, rid, af.AF_SEG_EMIT))
        row += q_len
    return segs


def layer_roofline(M, D, F):
    """Algorithmic GEMM flops and weight bytes of one layer at M rows (bf16 weights)."""
    flops = 2 * M * (4 * D * D + 3 * D * F)
    wbytes = 2 * (4 * D * D + 3 * D * F)
    return flops, wbytes


def sweep(af, w, shape, reps=4, n_layers=4):
    """The packed-mix sweep: one layer forward per point (a prefill of P rows + d decode rows
    with contexts uniform in {max(1, P), .., P + 7}; ring 16 slots x 544 with N(0, 1) history),
    timed per kernel class with HIP events.  Successive runs rotate over n_layers weight layers
    (1.6 GB for 4), so the 256 MB last-level cache does not hold the weights between runs."""
    import torch
    import workload as wl
    H, hd, D, F = shape.n_heads, shape.head_dim, shape.d_model, shape.d_ff
    n_slots, max_pos = wl.SWEEP_RING
    ring = af.Ring(n_layers, n_slots, max_pos, H, hd, dtype=torch.bfloat16)
    for l in range(n_layers):
        kv = wl.draw(("sweep ring", l), (2, n_slots, max_pos, H, hd), device="cuda")
        for sl in range(n_slots):
            ring.write_kv(l, sl, 0, kv[0, sl], kv[1, sl])
    del kv
    points = []
    for P in wl.SWEEP_PREFILL:
        for d in wl.SWEEP_DECODE:
            specs = wl.sweep_point_specs(P, d)
            segs = _reserve(af, ring, specs)
            M = sum(sg[1] for sg in segs)
            x = wl.draw(("sweep rows", P, d), (M, D), device="cuda")
            xs = [x.clone() for _ in range(n_layers)]
            for l in range(n_layers):
                af.packed_layer_forward(w, l, xs[l], segs, ring)
            torch.cuda.synchronize()
            w.timing_enable((1 << af.AF_K_COUNT) - 1)
            for _ in range(reps):
                for l in range(n_layers):
                    af.packed_layer_forward(w, l, xs[l], segs, ring)
            torch.cuda.synchronize()
            tm = w.timing_read()
            w.timing_enable(0)
            n = reps * n_layers
            gemm_us = sum(tm[k][0] for k in ("gemm_qkv", "gemm_o", "gemm_gateup", "gemm_down")) / n * 1e3
            at_us = tm["attention"][0] / n * 1e3
            norm_us = tm["rmsnorm"][0] / n * 1e3
            flops, wbytes = layer_roofline(M, D, F)
            at_bytes = attention_bytes(segs, H, hd)
            points.append({"P": P, "d": d, "M": M, "gemm_us": round(gemm_us, 2), "attention_us": round(at_us, 2),
                           "rmsnorm_us": round(norm_us, 2),
                           "gemm_frac_mfma": round(flops / (gemm_us * 1e-6) / (PEAK_BF16_TFLOPS * 1e12), 4),
                           "gemm_frac_hbm": round(wbytes / (gemm_us * 1e-6) / (PEAK_HBM_GBS * 1e9), 4),
                           "attention_frac_hbm": round(at_bytes / (at_us * 1e-6) / (PEAK_HBM_GBS * 1e9), 4)})
            for sg in segs:
                ring.release(sg[4])
    ring.close()
    return points


def stress(af, w, shape, steps=8):
    """The multi-pipeline stress workload: 8 pipelines of depth 8 (276-row prefill + 7 decode
    rows each) packed into every 32-layer forward, M = 2264 rows in steady state, ring 64 slots x
    288.  Warm-up until every step is full, then `steps` timed steps and a per-kernel pass."""
    import torch
    import workload as wl
    from paper_2512_20276_amd.pipeline import Pipeline
    st = wl.STRESS
    P, K, L_V, L_T = st["n_pipes"], st["K"], st["n_vision"], st["n_text"]
    L_P, D, F = L_V + L_T, shape.d_model, shape.d_ff
    ring = af.Ring(shape.n_layers, st["n_slots"], st["max_pos"], shape.n_heads, shape.head_dim, dtype=torch.bfloat16)
    text = wl.draw_ids(("instruction", 0), L_T, shape.vocab, device="cuda")
    pids = torch.cat([torch.full((L_V,), -1, dtype=torch.int32, device="cuda"), text])
    pool = []
    for i in range(4):   # four distinct sets of camera frames, reused cyclically
        e = torch.zeros((P * (L_P + K - 1), D), dtype=torch.bfloat16, device="cuda")
        for p in range(P):
            e[p * L_P:p * L_P + L_V] = wl.draw(("stress vision", i, p), (L_V, D), device="cuda")
        pool.append(e)
    pipe = Pipeline(w, ring, K, pids, lambda t: pool[t % len(pool)], keep_history=False, n_pipes=P)
    for _ in range(K):
        pipe.step()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        M = pipe.step().M
    torch.cuda.synchronize()
    dt = (time.perf_counter() - t0) / steps
    w.timing_enable((1 << af.AF_K_COUNT) - 1)
    for _ in range(steps):
        pipe.step()
    torch.cuda.synchronize()
    tm = w.timing_read()
    w.timing_enable(0)
    ring.close()
    flops, _ = layer_roofline(M, D, F)
    gemm_s = sum(tm[k][0] for k in ("gemm_qkv", "gemm_o", "gemm_gateup", "gemm_down")) / steps * 1e-3
    return {"M": M, "pipelines": P, "K": K, "ms_per_step": round(dt * 1e3, 3),
            "packed_steps_per_s": round(1 / dt, 3), "packed_tokens_per_s": round(M / dt, 1),
            "action_tokens_per_s": round(P * K / dt, 1),
            "mfma_frac_projection_gemms": round(flops * shape.n_layers / gemm_s / (PEAK_BF16_TFLOPS * 1e12), 4),
            "kernel_ms_per_step": {k: round(ms / steps, 4) for k, (ms, n) in tm.items()}}


def k_sweep(af, w, shape, Ks=(7, 16, 24, 32), text_rows=(20, 64, 256), steps=10):
    """Action length K crossed with the prefill length, as in the paper's K experiment (a
    prefill of 256 vision rows plus an instruction of 20, 64 or 256 token ids: L_P = 276, 320,
    512): the 32-layer pipeline at each point (one L_P-row prefill + K - 1 decode rows per step,
    ring K + 1 slots), against the plain per-request schedule on the same kernels (prefill,
    then K - 1 single-row decodes)."""
    import torch
    import workload as wl
    from paper_2512_20276_amd.pipeline import Pipeline
    D, L_V = shape.d_model, 256
    out = []
    for L_T in text_rows:
        text = wl.draw_ids(("instruction", 0, L_T), L_T, shape.vocab, device="cuda")
        pids = torch.cat([torch.full((L_V,), -1, dtype=torch.int32, device="cuda"), text])
        L_P = L_V + L_T
        for K in Ks:
            max_pos = (L_P + K + 31) // 32 * 32
            ring = af.Ring(shape.n_layers, K + 1, max_pos, shape.n_heads, shape.head_dim, dtype=torch.bfloat16)
            pool = []
            for i in range(4):
                e = torch.zeros((L_P + K - 1, D), dtype=torch.bfloat16, device="cuda")
                e[:L_V] = wl.draw(("vision", 0, i), (L_V, D), device="cuda")
                pool.append(e)
            pipe = Pipeline(w, ring, K, pids, lambda t: pool[t % len(pool)], keep_history=False)
            for _ in range(K + 1):
                pipe.step()
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            for _ in range(steps):
                M = pipe.step().M
            torch.cuda.synchronize()
            dt = (time.perf_counter() - t0) / steps
            ring.close()
            seq_ms = sequential_baseline(af, w, shape, pids, pool, K, n_req=2, warm=1)
            out.append({"K": K, "L_P": L_P, "M": M, "ms_per_step": round(dt * 1e3, 3),
                        "packed_steps_per_s": round(1 / dt, 2), "packed_tokens_per_s": round(M / dt, 1),
                        "action_tokens_per_s": round(K / dt, 1), "sequential_ms_per_request": round(seq_ms, 3),
                        "speedup_vs_sequential": round(seq_ms / (dt * 1e3), 3)})
            log(f"K={K} L_P={L_P}: {dt * 1e3:.2f} ms/step, sequential {seq_ms:.2f} ms/request")
    return out


def copy_shift(af, w, shape, pids, pool, K=7, steps=12, reps=10):
    """The paper's physical-copy InPlaceKVShift against the index rotation: the same pipeline
    (K = 7) with stage s kept in slot s and every live stage's keys and values copied one slot
    along after each step (af_ring_shift_stages); and that copy alone, on a steady-state ring
    (stages of 276 .. 281 positions, all 32 layers), with the bytes it moves."""
    import torch
    from paper_2512_20276_amd.pipeline import Pipeline
    L_P = int(pids.numel())
    ring = af.Ring(shape.n_layers, K, 288, shape.n_heads, shape.head_dim, dtype=torch.bfloat16)
    pipe = Pipeline(w, ring, K, pids, lambda t: pool[t % len(pool)], keep_history=False, shift="copy")
    for _ in range(K + 1):
        pipe.step()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        pipe.step()
    torch.cuda.synchronize()
    dt = (time.perf_counter() - t0) / steps
    ring.close()
    # the copy alone: K - 1 live stages of L_P .. L_P + K - 2 positions
    ring = af.Ring(shape.n_layers, K, 288, shape.n_heads, shape.head_dim, dtype=torch.bfloat16)
    lens = [L_P + s for s in range(K - 1)]
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    total_ms = 0.0
    for r in range(reps + 1):
        ring.reset()
        for s, n in enumerate(lens):
            ring.append(s, n)
        ring.append(10 ** 6, 1)   # the last stage's slot, released: the finished request
        ring.release(10 ** 6)
        torch.cuda.synchronize()
        e0.record()
        ring.shift_stages(K)
        e1.record()
        torch.cuda.synchronize()
        if r:
            total_ms += e0.elapsed_time(e1)
    ring.close()
    shift_ms = total_ms / reps
    moved = 2 * sum(lens) * shape.n_heads * shape.head_dim * 2 * 2 * shape.n_layers  # read + write
    return {"ms_per_step": round(dt * 1e3, 3), "packed_steps_per_s": round(1 / dt, 3),
            "shift_ms_per_step": round(shift_ms, 4), "shift_bytes_per_step": moved,
            "shift_GB/s": round(moved / (shift_ms * 1e-3) / 1e9, 1),
            "note": "stage s kept in slot s; K - 1 stages' keys and values copied one slot along per step"}


def naive_pipe(af, w, shape, pids, pool, packed_ms, K=7, steps=12):
    """The pipeline without the unified ring (the paper's Naive Pipe ablation): per-request
    caches, every layer's histories gathered into one contiguous buffer and the new rows
    scattered back, the host waiting for the device after each layer and building the next
    batch from host-side tokens; and the same with the per-layer waits left out (the copies'
    cost alone).  Wall-clock ms per steady-state step (K = 7, M = 282)."""
    import torch
    from paper_2512_20276_amd.naive_pipe import NaivePipeline
    out = {}
    for name, sync in (("host_sync_per_layer", True), ("copies_only", False)):
        pipe = NaivePipeline(w, K, pids, lambda t: pool[t % len(pool)], sync_per_layer=sync)
        for _ in range(K + 1):
            pipe.step()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(steps):
            pipe.step()
        torch.cuda.synchronize()
        dt = (time.perf_counter() - t0) / steps
        out[name] = {"ms_per_step": round(dt * 1e3, 3), "packed_steps_per_s": round(1 / dt, 3),
                     "ring_speedup": round(dt * 1e3 / packed_ms, 3)}
        out["copy_bytes_per_step"] = pipe.copy_bytes
        pipe.close()
    out["note"] = ("per layer: K - 1 histories gathered and K new rows scattered back (copy_bytes: bytes "
                   "copied, each read once and written once); ring_speedup = this ms per step / the ring "
                   "pipeline's")
    return out


# ----------------------------------------------------------------------------- cpu baseline
def cpu_baseline(n_big_steps: int = 2):
    """The oracle as it stands (float64 NumPy with bf16 storage rounding, never tuned for speed)
    on the host cores, on bounded samples of the workloads:
      * config 1: the tiny fp32-storage decoder's packed step 2 of a K = 3 pipeline (32 + 1 + 1 rows);
      * config 2: one 7B-shape layer at the 282-row packed step (276 prefill + 6 decode rows);
      * config 3: n_big_steps whole 282-row packed steps through all 32 layers and the LM head of
        the 7 emitting rows; the weights are drawn one layer at a time and streamed (host memory
        holds one float64 layer), and each layer is applied to every step's rows before the next
        layer is drawn, so only the oracle's own arithmetic is timed.
    The headline value is packed tokens/s at the median config-3 step."""
    import numpy as np
    import torch
    import threadpoolctl

    import oracle
    from oracle.pipeline import PipelineOracle
    import workload as wl

    info = threadpoolctl.threadpool_info()
    blas_threads = max([i.get("num_threads", 1) for i in info if i.get("user_api") == "blas"] or [1])
    cores = len(os.sched_getaffinity(0))
    to64 = lambda t: t.detach().to("cpu", torch.float64).numpy()
    out = {}

    # config 1: the tiny decoder's step 2 (warm-up steps 0 and 1 untimed)
    tiny = wl.TINY
    g, ls = wl.model_weights(tiny, seed=0)
    tmodel = oracle.OracleModel(tiny, {k: to64(v) for k, v in g.items()},
                                [{k: to64(v) for k, v in lw.items()} for lw in ls], storage="f32")

    def tiny_prefill(t):
        ids = wl.draw_ids(("prompt", 0, t), 32, tiny.vocab).numpy().astype(np.int64)
        return ids, np.zeros((32, tiny.d_model))

    tpipe = PipelineOracle(tmodel, 3, 4, 64, tiny_prefill)
    tpipe.step()
    tpipe.step()
    t0 = time.perf_counter()
    st = tpipe.step()
    t1 = time.perf_counter() - t0
    out["config1_step"] = {"M": int(len(st["ids"])), "seconds": round(t1, 4),
                           "tokens_per_s": round(len(st["ids"]) / t1, 1)}
    log(f"cpu oracle: config 1 step {t1 * 1e3:.1f} ms")

    # configs 2 and 3: 282-row packed steps of the 7B shape, layer by layer
    shape = wl.LLAMA7B
    H, hd, D, L = shape.n_heads, shape.head_dim, shape.d_model, shape.n_layers
    glob = {k: to64(v) for k, v in wl.global_weights(shape, seed=0, device="cuda").items()}
    rng = np.random.default_rng(0)
    segs = [oracle.Segment(0, 276, 2, 0, 10)] + [oracle.Segment(276 + s - 1, 1, (2 - s) % 8, 276 + s - 1, 10 - s)
                                                 for s in range(1, 7)]
    steps = []
    for b in range(n_big_steps):
        # one layer of ring history (N(0, 1), bf16 values), which every layer of the sample reads
        kv = oracle.OracleRingKV(1, 8, 288, H, hd)
        for sg in segs:
            if sg.pos0:
                kv.k[0, sg.slot, :sg.pos0] = oracle.round_storage(rng.standard_normal((sg.pos0, H, hd)), "bf16")
                kv.v[0, sg.slot, :sg.pos0] = oracle.round_storage(rng.standard_normal((sg.pos0, H, hd)), "bf16")
        x = oracle.round_storage(rng.standard_normal((282, D)), "bf16")
        steps.append({"kv": kv, "h": x, "layer_s": []})
    for l in range(L):
        lw = {k: to64(v) for k, v in wl.layer_weights(shape, l, seed=0, device="cuda").items()}
        model = oracle.OracleModel(shape.with_layers(1), glob, [lw], storage="bf16")
        for stp in steps:
            t0 = time.perf_counter()
            stp["h"] = model.layer_packed(0, stp["h"], segs, stp["kv"])
            stp["layer_s"].append(time.perf_counter() - t0)
        del model, lw
        if l % 8 == 7:
            log(f"cpu oracle: {l + 1} of {L} layers of {n_big_steps} steps")
    torch.cuda.empty_cache()
    head_model = oracle.OracleModel(shape.with_layers(0), glob, [], storage="bf16")
    step_s = []
    for stp in steps:
        t0 = time.perf_counter()
        head_model.logits(stp["h"][[s.q_start + s.q_len - 1 for s in segs]])
        step_s.append(sum(stp["layer_s"]) + time.perf_counter() - t0)
    layer_s = sorted(t for stp in steps for t in stp["layer_s"])
    q = lambda v, f: v[min(len(v) - 1, int(f * len(v)))]
    out["config2_layer_step"] = {"M": 282, "median_s": round(q(layer_s, 0.5), 4), "p10_s": round(q(layer_s, 0.1), 4),
                                 "p90_s": round(q(layer_s, 0.9), 4), "samples": len(layer_s)}
    med = sorted(step_s)[len(step_s) // 2]
    out["config3_steps"] = {"M": 282, "layers": L, "seconds": [round(t, 3) for t in step_s],
                            "median_s": round(med, 3)}
    log(f"cpu oracle: config 3 steps {[round(t, 2) for t in step_s]} s")
    return {"value": round(282.0 / med, 2), "unit": "tokens/s", "cores": cores, "blas_threads": int(blas_threads),
            "kind": "oracle", "precision": "float64 arithmetic, bf16 storage rounding (fp32 for config 1)",
            "sample": f"{n_big_steps} whole 282-row packed steps of the 32-layer 7B shape (weights streamed a layer "
                      f"at a time, LM head on 7 rows), median {med:.1f} s/step; plus one config-1 step and the "
                      f"config-2 layer steps they contain",
            **out}


# ----------------------------------------------------------------------------- main
def main():
    args = parse()
    if args.summarize_stats:
        summarize_stats(args.summarize_stats)
        return
    if args.summarize_pmc:
        summarize_pmc(*args.summarize_pmc)
        return
    if args.summarize_mfma:
        summarize_mfma(*args.summarize_mfma)
        return
    if args.summarize_stalls:
        summarize_stalls(*args.summarize_stalls)
        return
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py measures one GPU: this build has no multi-GPU path (each MI355X would run its "
              "own independent pipelines); run with --gpus 1", file=sys.stderr)
        sys.exit(2)
    import torch

    import paper_2512_20276_amd as af
    import workload as wl
    from paper_2512_20276_amd.pipeline import Pipeline

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = "cuda"
    shape = wl.LLAMA7B
    K, L_V, L_T, n_slots, max_pos = 7, 256, 20, 8, 288
    L_P = L_V + L_T
    M = L_P + K - 1
    D, F, V, H, hd = shape.d_model, shape.d_ff, shape.vocab, shape.n_heads, shape.head_dim
    if args.warmup < K - 1:
        log(f"warm-up raised to {K - 1} so that every timed step is a full packed step")
        args.warmup = K - 1

    t0 = time.time()
    g, layers = wl.model_weights(shape, seed=0, device=dev)
    w = af.Weights(shape, g, layers)
    del g, layers
    torch.cuda.empty_cache()
    ring = af.Ring(shape.n_layers, n_slots, max_pos, H, hd, dtype=torch.bfloat16)
    text = wl.draw_ids(("instruction", 0), L_T, V, device=dev)
    pids = torch.cat([torch.full((L_V,), -1, dtype=torch.int32, device=dev), text])
    pool = []
    for i in range(8):   # eight distinct camera frames, reused cyclically
        e = torch.zeros((M, D), dtype=torch.bfloat16, device=dev)
        e[:L_V] = wl.draw(("vision", 0, i), (L_V, D), device=dev)
        pool.append(e)
    pipe = Pipeline(w, ring, K, pids, lambda t: pool[t % len(pool)], keep_history=False)
    torch.cuda.synchronize()
    if args.copy_calibration:
        src = torch.ones(COPY_BYTES // 4, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        torch.neg(src, out=dst)   # one elementwise pass: every byte read once and written once
        torch.cuda.synchronize()
        del src, dst
        torch.cuda.empty_cache()
    log(f"setup {time.time() - t0:.1f} s; warm-up {args.warmup} steps")

    for _ in range(args.warmup):
        pipe.step()
    torch.cuda.synchronize()
    log(f"timed: {args.steps} steps")
    t0 = time.perf_counter()
    Ms = []
    for _ in range(args.steps):
        Ms.append(pipe.step().M)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    assert all(m == M for m in Ms), Ms
    ms_step = elapsed / args.steps * 1e3
    steps_s = args.steps / elapsed
    tokens_s = M * steps_s
    log(f"{ms_step:.3f} ms/step, {tokens_s:.0f} packed tokens/s")

    out = {"metric": METRIC, "value": round(tokens_s, 1), "unit": "tokens/s", "n_gpus": 1,
           "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms_step, 4),
           "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
           "data": "synthetic (seeded N(0,1) vision rows, fixed instruction ids, random-init N(0,0.02) weights)",
           "config": {"workload": "7B-shape 32-layer packed step, K=7 pipeline steady state: 276 prefill + 6 decode "
                                  "rows (M=282), ring 8 slots x 288, LM head + argmax on 7 rows",
                      "M": M, "layers": shape.n_layers, "K": K, "prefill_rows": L_P, "decode_rows": K - 1},
           "packed_steps_per_s": round(steps_s, 3),
           "action_tokens_per_s": round(K * steps_s, 2)}

    if not args.no_timing_pass:
        w.timing_enable((1 << af.AF_K_COUNT) - 1)
        segs_seen = None
        t1 = time.perf_counter()
        for _ in range(args.steps):
            r = pipe.step()
            segs_seen = r.segments
        torch.cuda.synchronize()
        t_inst = time.perf_counter() - t1
        tm = w.timing_read()
        w.timing_enable(0)
        work = gemm_work(M, D, F, V, K)
        per_step = {k: round(ms / args.steps, 4) for k, (ms, n) in tm.items()}
        gemm_ms = sum(tm[k][0] for k in ("gemm_qkv", "gemm_o", "gemm_gateup", "gemm_down")) / args.steps
        gemm_flops = sum(work[k][0] for k in ("gemm_qkv", "gemm_o", "gemm_gateup", "gemm_down")) * shape.n_layers
        mfma_frac = gemm_flops / (gemm_ms * 1e-3) / (PEAK_BF16_TFLOPS * 1e12)
        ga_ms, ga_n = tm["gemm_gateup"]
        ga_avg = ga_ms / ga_n
        ga_flops, _ = work["gemm_gateup"]
        ga_bytes = 2 * (2 * F * D)   # algorithmic bytes: the gate and up weights, each read once
        ga_gbs = ga_bytes / (ga_avg * 1e-3) / 1e9
        at_ms, at_n = tm["attention"]
        at_bytes = attention_bytes(segs_seen, H, hd)
        at_gbs = at_bytes / (at_ms / at_n * 1e-3) / 1e9
        out["roofline"] = {"kernel": "gemm32c_kernel<5, 6, EPI_SWIGLU> (gate/up projection, SwiGLU epilogue)",
                           "bound": "hbm", "achieved": round(ga_gbs, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                           "frac": round(ga_gbs / PEAK_HBM_GBS, 4), "traffic": measured_traffic(),
                           "bytes_per_launch": ga_bytes, "bytes_counted": "gate + up weights (2 x 11008 x 4096 bf16)",
                           "avg_launch_us": round(ga_avg * 1e3, 2),
                           "duration": f"average of {ga_n} launches, HIP events on the launch stream (timing pass)",
                           "tflops": round(ga_flops / (ga_avg * 1e-3) / 1e12, 1),
                           "frac_mfma": round(ga_flops / (ga_avg * 1e-3) / (PEAK_BF16_TFLOPS * 1e12), 4)}
        out["mfma_frac_projection_gemms"] = round(mfma_frac, 4)
        out["projection_gemm_tflops"] = round(gemm_flops / (gemm_ms * 1e-3) / 1e12, 1)
        out["attention_hbm"] = {"GB/s": round(at_gbs, 1), "frac": round(at_gbs / PEAK_HBM_GBS, 4),
                                "bytes_per_launch": at_bytes, "avg_launch_us": round(at_ms / at_n * 1e3, 2)}
        out["kernel_ms_per_step"] = per_step
        out["kernel_sum_ms_per_step"] = round(sum(ms for ms, _ in tm.values()) / args.steps, 4)
        out["timing_pass_ms_per_step"] = round(t_inst / args.steps * 1e3, 4)
        log(f"timing pass: {json.dumps(per_step)}")

        # per-step GPU time: an event pair around every step on the launch stream, no host waits
        evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
               for _ in range(args.steps)]
        for a, b in evs:
            a.record()
            pipe.step()
            b.record()
        torch.cuda.synchronize()
        st_ms = sorted(a.elapsed_time(b) for a, b in evs)
        q = lambda f: st_ms[min(len(st_ms) - 1, int(f * len(st_ms)))]
        out["step_ms_distribution"] = {"median": round(q(0.5), 4), "p10": round(q(0.1), 4), "p90": round(q(0.9), 4),
                                       "steps": len(st_ms), "how": "HIP events around each step, no host waits"}

    extras = () if args.no_extra else tuple(args.extra or EXTRAS)
    if "sequential" in extras:
        log("sequential baseline (one request at a time, same kernels)")
        seq_ms = sequential_baseline(af, w, shape, pids, pool, K)
        out["sequential_baseline"] = {
            "ms_per_request": round(seq_ms, 3), "requests_per_s": round(1e3 / seq_ms, 3),
            "packed_speedup": round(steps_s / (1e3 / seq_ms), 3),
            "note": "one request = 276-row prefill + 6 single-row decodes through 32 layers; the packed "
                    "pipeline completes one request per step"}
    if "attention_stress" in extras:
        log("decode-heavy attention (8 pipelines x (276 + 7), 64 slots)")
        out["attention_stress"] = decode_heavy_attention(af, w, shape)
    if "sweep" in extras:
        log("packed-mix sweep (one layer, 16 points)")
        out["sweep"] = sweep(af, w, shape)
    if "stress" in extras:
        log("stress workload (8 pipelines, M = 2264, 32 layers)")
        out["stress"] = stress(af, w, shape)
    if "k_sweep" in extras:
        log("K sweep (K = 7, 16, 24, 32 x prefill 276, 320, 512)")
        out["k_sweep"] = k_sweep(af, w, shape)
    if "copy_shift" in extras:
        log("physical-copy stage shift (the paper's InPlaceKVShift copy) against the rotation")
        out["copy_shift"] = copy_shift(af, w, shape, pids, pool, K)
    if "naive_pipe" in extras:
        log("naive pipe (per-request caches, per-layer gather/scatter, host-coordinated)")
        out["naive_pipe"] = naive_pipe(af, w, shape, pids, pool, ms_step, K)
    ring.close()
    w.close()
    torch.cuda.empty_cache()
    if not args.no_cpu_baseline:
        log("cpu baseline (oracle sample)")
        out["cpu_baseline"] = cpu_baseline(args.cpu_steps)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
