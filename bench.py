"""Benchmark of the FedOptima server hot path on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--config 1..10, default 4] [--pipeline]

One step = one pass of the server's hot path over one activation batch:
an arriving batch is copied into the HBM activation pool (Alg. 2 put() with
flow control), the Task Scheduler picks the device with the smallest
consumption counter (Alg. 3 get()), the server trains M_s on that batch
(Alg. 4: forward, loss, backward, SGD) and the slot is recycled.  For the
workloads that aggregate device-side models (tiny CNN, ResNet, 128-device
VGG) one model arrival is also aggregated per step.  The default workload is
the BERT-base-shaped transformer split (B = 32, L = 128, d = 768, 10 layers,
lengths uniform on [32, 128]), the workload the bf16 MFMA target is stated on.

Printed as one JSON line:
  value          server training throughput (samples/s) with inputs resident in HBM
  mfu            useful FLOPs per step / step time / bf16 dense MFMA peak
  roofline       the dominant kernel (the one with the largest share of step time)
                 measured live with HIP events over the timed steps
  aggregate      the aggregation kernel at 1 GiB vectors (HBM roofline) and at the
                 workload sizes
  cpu_baseline   the oracle (fp32 NumPy) timed on the host cores on a bounded sample
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2516.6   # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0       # MI355X HBM3E


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=None, help="timed steps (transformer 30, 128-device VGG 1000)")
    ap.add_argument("--warmup", type=int, default=None, help="untimed steps (transformer 5, 128-device VGG 10)")
    ap.add_argument("--config", type=int, default=4, help="1-3: the parity workloads' step loops; 4: "
                    "transformer (default); 5: 128-device VGG with Poisson arrivals; 6: the device-side "
                    "iteration of the VGG split; 7, 8, 9, 10: the paper's Transformer-6 / Transformer-12 / VGG-5 / "
                    "MobileNetV3-Large server parts")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--pipeline", action="store_true",
                    help="the concurrent pipeline (Receiver and Compute Engine threads) on the 128-device VGG "
                         "workload: throughput T(p), retention R(p) = T(p)/T(0) and server idle time under "
                         "device dropout p")
    ap.add_argument("--pipeline-seconds", type=float, default=3.0, help="wall-clock seconds per pipeline run")
    ap.add_argument("--cpu-sample-steps", type=int, default=3,
                    help="fp32 oracle steps at the workload's own batch timed for cpu_baseline")
    ap.add_argument("--calib-copy", action="store_true",
                    help="also run a 1 GiB device-to-device copy (the HBM counter calibration kernel)")
    ap.add_argument("--summarize-pmc", nargs=2, metavar=("FETCH_CSV", "WRITE_CSV"),
                    help="turn two rocprofv3 --pmc runs (FETCH_SIZE, WRITE_SIZE) of this bench with "
                         "--calib-copy into the HBM traffic summary (JSON on stdout)")
    ap.add_argument("--summarize-trace", metavar="KERNEL_STATS_CSV",
                    help="print the per-kernel table of a rocprofv3 --kernel-trace --stats summary and exit")
    ap.add_argument("--summarize-counters", nargs="+", metavar="CSV",
                    help="turn rocprofv3 --pmc runs of this bench (MFMA and L2 counters, any number of "
                         "passes) into a per-kernel table (Markdown on stdout)")
    return ap.parse_args()


def cpu_baseline(cid, sample_steps):
    """The oracle in fp32 on the host cores over a bounded sample of the workload."""
    import fo_synth as S
    import oracle
    try:
        from threadpoolctl import threadpool_info
        cores = max([i.get("num_threads", 1) for i in threadpool_info()] or [os.cpu_count() or 1])
    except Exception:  # pragma: no cover
        cores = os.cpu_count() or 1
    Bs = S.get_config(cid).batch  # the headline workload's own batch
    theta = S.init_params(cid)
    acts = S.make_acts(cid, sample_steps, batch=Bs, sub=99)
    labels = S.make_labels(cid, sample_steps, batch=Bs, sub=99)
    lengths = (S.make_lengths(cid, sample_steps, batch=Bs, sub=99) if cid in (4, 7, 8)
               else [None] * sample_steps)
    t0 = time.perf_counter()
    cfg = S.get_config(cid)
    mom = None
    for i in range(sample_steps):
        r = oracle.server_step(cid, theta, acts[i], labels[i], lengths[i], lr=cfg.lr, momentum=cfg.momentum,
                               mom_buf=mom, dt=np.float32)
        theta = r["params"].astype(np.float32)
        mom = r["momentum"]
    dt = time.perf_counter() - t0
    return {"value": round(Bs * sample_steps / dt, 3), "unit": "samples/s", "cores": int(cores), "kind": "oracle",
            "sample": f"{sample_steps} consecutive fp32 oracle steps at batch {Bs} (the workload's batch) "
                      f"on fresh seeded batches of the same workload ({dt:.1f} s)"}


# ---------------------------------------------------------------- HBM traffic
# The kernels whose HBM bytes are taken from rocprofv3 counters: (name prefix in
# the profiler's kernel names, the sources that define them).
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "hbm_traffic_bert_step.txt")
GEMM_SOURCES = ["paper_2504_13850_amd/csrc/k_gemm.hip", "paper_2504_13850_amd/csrc/gemm.h",
                "paper_2504_13850_amd/csrc/common.h"]
TRAFFIC_KERNELS = {
    # compensated forward products, input gradients, weight gradients of the transformer step
    "gemm_comp_dma_kernel<3>": ("gemm_comp_dma_kernel<3, 2, fo::(anonymous namespace)::DmaRKc>", GEMM_SOURCES),
    "gemm_rk_krt_dma_kernel": ("gemm_rk_krt_dma_kernel<32, 4>", GEMM_SOURCES),
    "gemm_wgrad_dma_kernel": ("gemm_wgrad_dma_kernel<32, 4>", GEMM_SOURCES),
    "gemm_wgrad_tall_kernel": ("gemm_wgrad_tall_kernel<32, 3>", GEMM_SOURCES),
    "agg_lerp_kernel": ("agg_lerp_kernel(", ["paper_2504_13850_amd/csrc/k_update.hip"]),
}
CALIB_BYTES = 1 << 30
# `traffic` is not measured by this run: it is read from the committed summary
# of two rocprofv3 counter passes, and only while the kernel's sources still
# hash to what they were when the counters were taken (else null).
TRAFFIC_SOURCE = ("stored rocprofv3 FETCH_SIZE + WRITE_SIZE per launch from profiles/hbm_traffic_bert_step.txt "
                  "(null when the kernel's sources changed since)")


def source_hash(files):
    import hashlib
    h = hashlib.sha256()
    for f in files:
        with open(os.path.join(ROOT, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def summarize_pmc(fetch_csv, write_csv):
    """Per-dispatch FETCH_SIZE / WRITE_SIZE (KiB) of the traffic kernels, scaled
    by what the same counters read for the 1 GiB calibration copy."""
    import csv
    import statistics

    def read(path, counter):
        rows = {}
        with open(path) as fh:
            for r in csv.DictReader(fh):
                if r["Counter_Name"] != counter:
                    continue
                key = r["Dispatch_Id"]
                rows[key] = (r["Kernel_Name"], rows.get(key, (None, 0.0))[1] + float(r["Counter_Value"]))
        return list(rows.values())

    out = {"counters_kib_per_dispatch": {}, "calibration": {}}
    for counter, path in (("FETCH_SIZE", fetch_csv), ("WRITE_SIZE", write_csv)):
        rows = read(path, counter)
        copies = [v for n, v in rows if "copyBuffer" in n and v * 1024 > CALIB_BYTES / 2]
        if not copies:
            raise SystemExit(f"no calibration copy found in {path}")
        factor = (CALIB_BYTES / 1024) / statistics.mean(copies)
        out["calibration"][counter] = {"copy_bytes": CALIB_BYTES, "dispatches": len(copies),
                                       "mean_kib": round(statistics.mean(copies), 1), "factor": round(factor, 5)}
        for name, (prefix, _) in TRAFFIC_KERNELS.items():
            vals = [v for n, v in rows if prefix in n]
            if name == "agg_lerp_kernel":  # the 1 GiB sweep calls only
                vals = [v for v in vals if v * 1024 > (1 << 29)]
            if vals:
                out["counters_kib_per_dispatch"].setdefault(name, {})[counter] = {
                    "dispatches": len(vals), "mean_kib": round(statistics.mean(vals), 1)}
    kern = {}
    for name, (prefix, files) in TRAFFIC_KERNELS.items():
        c = out["counters_kib_per_dispatch"].get(name, {})
        if "FETCH_SIZE" not in c or "WRITE_SIZE" not in c:
            continue
        rd = c["FETCH_SIZE"]["mean_kib"] * 1024 * out["calibration"]["FETCH_SIZE"]["factor"]
        wr = c["WRITE_SIZE"]["mean_kib"] * 1024 * out["calibration"]["WRITE_SIZE"]["factor"]
        kern[name] = {"read_bytes_per_launch": round(rd), "write_bytes_per_launch": round(wr),
                      "bytes_per_launch": round(rd + wr), "source_sha256": source_hash(files)}
    out["kernels"] = kern
    return out


def summarize_trace(path, top=25):
    """Markdown table of a rocprofv3 kernel_stats.csv: calls, average and total
    time and share per kernel (names shortened)."""
    import csv
    rows = []
    with open(path) as fh:
        for r in csv.DictReader(fh):
            name = r["Name"].replace("void ", "").replace("fo::(anonymous namespace)::", "fo::")
            name = name.split("(fo::")[0].split("(unsigned")[0].split("(float")[0].split("(int")[0]
            name = name.split("(__hip")[0].split("(const")[0].split("(long")[0]
            rows.append((float(r["TotalDurationNs"]), name, int(r["Calls"]), float(r["AverageNs"]),
                         float(r["Percentage"])))
    rows.sort(key=lambda t: -t[0])
    out = ["| kernel | calls | avg us | total ms | share % |", "|---|---:|---:|---:|---:|"]
    for tot, name, calls, avg, pct in rows[:top]:
        out.append(f"| `{name[:90]}` | {calls} | {avg / 1e3:.1f} | {tot / 1e6:.2f} | {pct:.2f} |")
    return "\n".join(out)


def summarize_counters(paths, top=12):
    """Per-kernel averages of rocprofv3 --pmc counter passes over this bench.

    Executed MFMA work is SQ_INSTS_VALU_MFMA_MOPS_BF16 x 512 FLOP (the unit the
    counter counts in; it reproduces 2*M*N*K per pass of each product).  L2
    requests are TCC_HIT + TCC_MISS (64-byte requests for these kernels).
    Busy fractions divide by the dispatch's GRBM_GUI_ACTIVE / 8 (that counter
    sums the eight XCDs) and by the unit count: 128 L2 channels, 256 CUs for
    the texture address (TA) and data (TD) units."""
    import csv
    from collections import defaultdict
    disp = defaultdict(dict)  # (path, dispatch) -> counters
    info = {}
    for path in paths:
        with open(path) as fh:
            for r in csv.DictReader(fh):
                key = (path, r["Dispatch_Id"])
                c = disp[key]
                c[r["Counter_Name"]] = c.get(r["Counter_Name"], 0.0) + float(r["Counter_Value"])
                name = r["Kernel_Name"].replace("void ", "").replace("fo::(anonymous namespace)::", "")
                name = name.split("(fo::")[0].split("(unsigned")[0].split("(float")[0].split("(int")[0]
                info[key] = (name, (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) * 1e-9)
    per = defaultdict(lambda: defaultdict(list))
    calls = defaultdict(lambda: defaultdict(int))  # dispatches per pass
    for key, c in disp.items():
        name, dur = info[key]
        if "at::native" in name or "__amd_rocclr" in name:  # the bench's own setup and copies
            continue
        calls[name][key[0]] += 1
        per[name]["dur"].append(dur)
        for k, v in c.items():
            per[name][k].append(v)
    mean = lambda xs: sum(xs) / len(xs) if xs else float("nan")
    rows = []
    for name, c in per.items():
        d = mean(c["dur"])
        cyc = {k: mean(v) / 8 for k, v in c.items() if k == "GRBM_GUI_ACTIVE"}.get("GRBM_GUI_ACTIVE")
        g = lambda k: mean(c[k]) if c.get(k) else None
        flop = g("SQ_INSTS_VALU_MFMA_MOPS_BF16")
        hit, miss = g("TCC_HIT"), g("TCC_MISS")
        frac = lambda k, units: (g(k) / units / cyc) if (g(k) is not None and cyc) else None
        n = max(calls[name].values())
        rows.append((d * n, name, {
            "dispatches": n, "avg_us": d * 1e6,
            "exec_tflops": flop * 512 / d / 1e12 if flop else None,
            "pct_peak": 100 * flop * 512 / d / 1e12 / PEAK_BF16_TFLOPS if flop else None,
            "l2_req": (hit + miss) if hit is not None else None,
            "l2_hit": hit / (hit + miss) if hit is not None and hit + miss > 0 else None,
            "l2_gbs": (hit + miss) * 64 / d / 1e9 if hit is not None else None,
            "l2_busy": frac("TCC_BUSY", 128), "td_busy": frac("TD_TD_BUSY", 256),
            "td_wait_l2": frac("TD_TC_STALL", 256), "ta_busy": frac("TA_TA_BUSY", 256)}))
    rows.sort(key=lambda r: -r[0])
    cols = [("dispatches", "dispatches per pass", "{:.0f}"), ("avg_us", "avg us", "{:.1f}"),
            ("exec_tflops", "MFMA TFLOP/s executed", "{:.0f}"), ("pct_peak", "% of bf16 peak", "{:.1f}"),
            ("l2_req", "L2 requests", "{:.3g}"), ("l2_hit", "L2 hit", "{:.2f}"),
            ("l2_gbs", "L2 GB/s (64 B req.)", "{:.0f}"), ("l2_busy", "L2 busy", "{:.2f}"),
            ("td_busy", "TD busy", "{:.2f}"), ("td_wait_l2", "TD waits on L2", "{:.2f}"),
            ("ta_busy", "TA busy", "{:.2f}")]
    out = ["| kernel | " + " | ".join(h for _, h, _ in cols) + " |",
           "|---|" + "---:|" * len(cols)]
    for _, name, v in rows[:top]:
        cells = [("-" if v[k] is None else f.format(v[k])) for k, _, f in cols]
        out.append(f"| `{name}` | " + " | ".join(cells) + " |")
    # latency passes, when given: average cycles of an L1 -> L2 read
    # (TCP_TCC_READ_REQ_LATENCY / TCP_TCC_READ_REQ), of an L2 -> fabric read
    # (TCC_EA0_RDREQ_LEVEL / TCC_EA0_RDREQ), the fraction of wave cycles spent
    # waiting (SQ_WAIT_ANY, SQ_WAIT_INST_ANY / SQ_WAVE_CYCLES) and the vector
    # memory instructions in flight per wave (SQ_INST_LEVEL_VMEM / SQ_INSTS_VMEM_RD)
    lat = []
    for _, name, _v in rows[:top]:
        c = per[name]
        g = lambda k: mean(c[k]) if c.get(k) else None
        ratio = lambda a, b: (g(a) / g(b)) if g(a) is not None and g(b) else None
        v = {"l1l2": ratio("TCP_TCC_READ_REQ_LATENCY_sum", "TCP_TCC_READ_REQ_sum"),
             "ea": ratio("TCC_EA0_RDREQ_LEVEL_sum", "TCC_EA0_RDREQ_sum"),
             "wait": ratio("SQ_WAIT_ANY", "SQ_WAVE_CYCLES"), "wait_inst": ratio("SQ_WAIT_INST_ANY", "SQ_WAVE_CYCLES"),
             "vmem_level": ratio("SQ_INST_LEVEL_VMEM", "SQ_INSTS_VMEM_RD"),
             "lds_fifo": g("SQ_LDS_DATA_FIFO_FULL")}
        if any(x is not None for x in v.values()):
            lat.append((name, v))
    if lat:
        lc = [("l1l2", "L1->L2 read latency (cyc)", "{:.0f}"), ("ea", "L2->fabric read latency (cyc)", "{:.0f}"),
              ("wait", "wave cycles waiting", "{:.2f}"), ("wait_inst", "waiting to issue", "{:.2f}"),
              ("vmem_level", "vector memory ops in flight per issue", "{:.0f}"),
              ("lds_fifo", "LDS data FIFO full (cyc)", "{:.3g}")]
        out += ["", "| kernel | " + " | ".join(h for _, h, _ in lc) + " |", "|---|" + "---:|" * len(lc)]
        for name, v in lat:
            out.append(f"| `{name}` | " + " | ".join("-" if v[k] is None else f.format(v[k]) for k, _, f in lc) + " |")
    return "\n".join(out)


def padded_bert_flops(B, L, d=768, ff=3072, layers=10, classes=2):
    """Training FLOPs of the transformer step with every sequence padded to L
    tokens and no first-token pruning: per layer the forward products
    2 L (3 d d + d d + 2 d ff) and attention 4 d L^2 per sequence, times three
    for forward, input and weight gradients, less the first layer's input
    gradient (2 L 3 d d); plus the pooler and classifier (forward and both
    gradients)."""
    fwd_layer = 2 * L * (3 * d * d + d * d + 2 * d * ff) + 4 * d * L * L
    per_seq = layers * 3 * fwd_layer - 2 * L * 3 * d * d
    head = 3 * 2 * (d * d + d * classes)
    return B * (per_seq + head)


def traffic_for(name):
    """HBM bytes per launch from the committed counter summary, or None when it
    is missing or the kernel's source changed since the counters were taken."""
    try:
        with open(TRAFFIC_FILE) as fh:
            summary = json.load(fh)
        k = summary["kernels"][name]
        if k["source_sha256"] != source_hash(TRAFFIC_KERNELS[name][1]):
            return None
        return k["bytes_per_launch"]
    except (OSError, KeyError, ValueError):
        return None


def calib_copy(torch):
    src = torch.empty(CALIB_BYTES, dtype=torch.uint8, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    del src, dst


def bench_aggregate(A, torch, stream):
    """HBM roofline of the aggregation kernel: 1 GiB fp32 vectors (12 B/element
    per call: read global + local, write global), plus latency at workload sizes."""
    n = 1 << 28
    g = torch.empty(n, device="cuda", dtype=torch.float32).normal_(0, 0.02)
    l = torch.empty(n, device="cuda", dtype=torch.float32).normal_(0, 0.02)
    A.fo_set_stream(stream)
    for _ in range(3):
        A.fo_async_aggregate(g, l, 1.0, 3)
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    reps = 20
    torch.cuda.synchronize()
    ev0.record(stream)
    for _ in range(reps):
        A.fo_async_aggregate(g, l, 1.0, 3)
    ev1.record(stream)
    torch.cuda.synchronize()
    ms = ev0.elapsed_time(ev1) / reps
    gbs = 12.0 * n / (ms * 1e-3) / 1e9
    small = {}
    for m in (10_000, 38_720, 157_504):
        gs, ls = g[:m], l[:m]
        for _ in range(3):
            A.fo_async_aggregate(gs, ls, 1.0, 1)
        torch.cuda.synchronize()
        ev0.record(stream)
        for _ in range(50):
            A.fo_async_aggregate(gs, ls, 1.0, 1)
        ev1.record(stream)
        torch.cuda.synchronize()
        us = ev0.elapsed_time(ev1) / 50 * 1e3
        small[str(m)] = {"us_per_call": round(us, 2), "GB/s": round(12.0 * m / (us * 1e-6) / 1e9, 1)}
    del g, l
    return {"kernel": "agg_lerp_kernel", "n": n, "bytes_per_call": 12 * n, "ms_per_call": round(ms, 4),
            "achieved_GBps": round(gbs, 1), "peak_GBps": PEAK_HBM_GBS, "frac": round(gbs / PEAK_HBM_GBS, 4),
            "workload_sizes": small}


VGG_STEP_GFLOP = 102.9  # useful FLOPs of one VGG-16 split server step at B = 64 (fwd + dgrad + wgrad)
PEAK_F32_TFLOPS = 157.3  # MI355X fp32 vector

# The step-loop workloads: K devices with one batch queued each, one arrival and
# one step per iteration (plus one model aggregation where the workload has a
# device-side model).  gflop: useful FLOPs of a step where no kernel records them.
WORKLOADS = {
    1: {"workload": "tiny CNN split server step (fp32): conv3x3 32->64, maxpool, conv3x3 64->64, GAP, "
                    "linear 64->10, batch 16 of [32,16,16], 4 devices, aggregation of 10,000 params per step "
                    "(alpha 0.5, staleness = device id)", "peak": PEAK_F32_TFLOPS, "gflop": 0.5285},
    2: {"workload": "vgg16 split server step, batch 64 of [64,16,16] bf16 activations, 16 devices",
        "peak": PEAK_BF16_TFLOPS, "gflop": VGG_STEP_GFLOP},
    3: {"workload": "resnet18 split server step (layer2-4, BatchNorm train mode, momentum 0.9), batch 32 of "
                    "[64,16,16] bf16 activations, 32 devices, aggregation of 157,504 params per step "
                    "(alpha 1, staleness U{0..8})", "peak": PEAK_BF16_TFLOPS, "gflop": 19.0},
    4: {"workload": "bert-base split server step: 10 post-LN encoder layers d=768 h=12 ffn=3072, "
                    "batch 32 x 128 tokens, lengths U[32,128], 16 devices, plain SGD",
        "peak": PEAK_BF16_TFLOPS, "gflop": 1099.0},
    7: {"workload": "Transformer-6 split server step (fp32): 6 post-LN encoder layers d=100 h=5 ffn=100 ReLU, "
                    "classifier on the first token, batch 16 x 64 tokens, lengths U[4,64], 8 devices",
        "peak": PEAK_F32_TFLOPS, "gflop": None},
    8: {"workload": "Transformer-12 split server step (fp32): 12 post-LN encoder layers d=100 h=50 ffn=100 ReLU, "
                    "classifier on the first token, batch 16 x 256 tokens, lengths U[16,256], 16 devices",
        "peak": PEAK_F32_TFLOPS, "gflop": None},
    9: {"workload": "VGG-5 split server step (fp32): conv3x3 64->64 + batch norm + ReLU, maxpool, fc 1024-128-10, "
                    "batch 32 of [64,8,8], 8 devices",
        # the convolution's forward and weight gradient (no input gradient), both fc layers three times
        "peak": PEAK_F32_TFLOPS, "gflop": 32 * (2 * 2 * 64 * 576 * 64 + 3 * (2 * 1024 * 128 + 2 * 128 * 10)) / 1e9},
    10: {"workload": "MobileNetV3-Large split server step (fp32): 8 bottlenecks (depthwise conv, squeeze-excitation, "
                     "hard-swish), conv1x1 960, pool, fc 960-1280-200, batch 32 of [80,4,4], 16 devices",
         "peak": PEAK_F32_TFLOPS, "gflop": None},
}


def mbv3_gflop():
    """FLOPs of the MobileNetV3 step (config 10, batch 32) from the
    pre-processor's unit table of MobileNetV3-Large at 64x64: the forward of the
    units after the split, three times, less the first unit's input gradient
    (its expansion product)."""
    import ctypes  # noqa: F401
    from paper_2504_13850_amd import api as A
    units = A.fo_net_units(A.FO_NET_MOBILENETV3_LARGE, 200, 64)
    fwd = sum(u.fwd_flops for u in list(units)[8:])
    first_dx = 2 * 80 * 200 * 16  # expansion of the first server block: 80 -> 200 channels on 4x4
    return 32 * (3 * fwd - first_dx) / 1e9


def tfsmall_gflop(cid):
    """FLOPs the fp32 transformer step executes (padded [B][L] layout): per
    encoder layer and sequence 2 L d (3d + d + 2 ffn) + 4 d L^2, three times
    (forward, input and weight gradients) less the first layer's input
    gradient, plus the classifier."""
    L, layers = (64, 6) if cid == 7 else (256, 12)
    d, ff, B = 100, 100, 16
    fwd = 2 * L * d * (3 * d + d + 2 * ff) + 4 * d * L * L
    per_seq = layers * 3 * fwd - 2 * L * 3 * d * d + 3 * 2 * d * 2
    return B * per_seq / 1e9


def fused_aggregation(A, torch, n, m):
    """One fused drain of m model messages into an n-element global: µs and GB/s
    against its (m + 2) * 4 * n algorithmic bytes."""
    g = torch.zeros(n, device="cuda", dtype=torch.float32)
    locs = [torch.full((n,), float(i + 1), device="cuda", dtype=torch.float32) for i in range(m)]
    q = A.fo_queues_create(m, 0, 1, False, 2 * m)
    try:
        def queue_models():
            for k in range(m):
                A.fo_queues_push_model(q, k, locs[k], 0)
            if A.fo_pick_device(q) != -2:
                raise RuntimeError("fused aggregation: no model pending")
        queue_models()
        A.fo_aggregate_pending_all(q, g, 1.0)
        torch.cuda.synchronize()
        reps = 10
        ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        ms = 0.0
        for _ in range(reps):
            queue_models()  # host bookkeeping only, outside the timed span
            torch.cuda.synchronize()
            ev0.record()
            applied, _ = A.fo_aggregate_pending_all(q, g, 1.0)
            ev1.record()
            torch.cuda.synchronize()
            ms += ev0.elapsed_time(ev1)
            assert applied == m
        us = ms / reps * 1e3
        nbytes = (m + 2) * 4 * n
        return {"n": n, "arrivals": m, "us_per_drain": round(us, 2), "bytes": nbytes,
                "GB/s": round(nbytes / (us * 1e-6) / 1e9, 1), "frac_of_hbm": round(nbytes / (us * 1e-6) / 1e9 / PEAK_HBM_GBS, 4)}
    finally:
        A.fo_queues_destroy(q)


def bench_vgg128(args, A, torch, S):
    """The 128-device VGG-16 split workload: lognormal device rates, Poisson
    arrivals per server step, each arrival an activation batch (flow-controlled
    put into a 64 GiB HBM pool, copied from a bank of 256 distinct batches) and a
    model message (staleness-weighted aggregation of the 38,720-parameter
    device-side part, fused per drain); then one pick and one server step."""
    cid = 5
    cfg = S.get_config(cid)
    K, B = cfg.n_devices, cfg.batch
    stream = torch.cuda.current_stream()
    steps, warm = args.steps, args.warmup
    rates = S.make_arrival_rates(cid)
    counts = S.make_arrival_counts(cid, rates, warm + steps)
    bank_n = cfg.extra["bank"]
    acts_d = torch.from_numpy(S.make_acts(cid, bank_n).view(np.int16)).cuda()
    labels_d = torch.from_numpy(S.make_labels(cid, bank_n)).cuda()
    model = A.fo_model_create(cid, B, S.init_params(cid), stream)
    slot_bytes = int(acts_d[0].numel()) * 2
    n_slots = cfg.extra["pool_bytes"] // slot_bytes
    q = A.fo_queues_create(K, slot_bytes, B, False, n_slots, stream)
    A.fo_set_max_delay(-1)
    n = cfg.agg_n
    glob = torch.from_numpy(S.make_global_vector(cid)).cuda()
    locs = torch.from_numpy(S.make_local_vectors(cid, K)).cuda()
    dev_version = np.zeros(K, np.int64)
    seq = [0]
    tallies = {"arrivals": 0, "applied": 0, "skipped": 0, "drains": 0, "idle_steps": 0}
    # raw device addresses of the bank's batches and labels and of the device-side models
    acts_base, lab_base, loc_base = (np.uint64(t.data_ptr()) for t in (acts_d, labels_d, locs))
    act_stride, lab_stride, loc_stride = np.uint64(slot_bytes), np.uint64(4 * B), np.uint64(4 * n)

    def one_step(t):
        # this step's arrivals, in device order: one activation send attempt and one
        # model message each (Alg. 2 put()), handed over in two calls
        senders = np.repeat(np.arange(K, dtype=np.int32), counts[t])
        m = int(senders.size)
        if m:
            idx = (np.uint64(seq[0]) + np.arange(m, dtype=np.uint64)) % np.uint64(bank_n)
            seq[0] += m
            A.fo_queues_push_batch(q, senders, acts_base + idx * act_stride, lab_base + idx * lab_stride)
            A.fo_queues_push_model_batch(q, senders, loc_base + senders.astype(np.uint64) * loc_stride, n,
                                         dev_version[senders])
        tallies["arrivals"] += m
        k = A.fo_pick_device(q)
        if k == -2:  # Alg. 3: models first
            applied, skipped = A.fo_aggregate_pending_all(q, glob, 1.0)
            tallies["applied"] += applied
            tallies["skipped"] += skipped
            tallies["drains"] += 1
            # each sender receives the aggregated global (Alg. 4)
            dev_version[senders] = A.fo_queues_stats(q).version
            k = A.fo_pick_device(q)
        if k < 0:
            tallies["idle_steps"] += 1
            return
        fa, lab, _, _ = A.fo_queues_in_service(q)
        A.fo_server_step(model, fa, lab, k)
        A.fo_queues_release(q)

    try:
        for t in range(warm):
            one_step(t)
        torch.cuda.synchronize()
        st0 = A.fo_queues_stats(q)
        ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        ev0.record(stream)
        wall0 = time.perf_counter()
        for t in range(warm, warm + steps):
            one_step(t)
        ev1.record(stream)
        torch.cuda.synchronize()
        wall = time.perf_counter() - wall0
        ms = ev0.elapsed_time(ev1)
        st = A.fo_queues_stats(q)
        trained = st.picks - st0.picks
        # the server step alone on a resident batch, for the step-only rate and MFU
        k = A.fo_pick_device(q)
        assert k >= 0
        fa, lab, _, _ = A.fo_queues_in_service(q)
        for _ in range(3):
            A.fo_server_step(model, fa, lab, k)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(20):
            A.fo_server_step(model, fa, lab, k)
        e1.record(stream)
        torch.cuda.synchronize()
        A.fo_queues_release(q)
        step_ms = e0.elapsed_time(e1) / 20
    finally:
        A.fo_queues_destroy(q)
        A.fo_model_destroy(model)
    fused = [fused_aggregation(A, torch, n, 64), fused_aggregation(A, torch, 1 << 24, 16)]
    value = B * trained / (ms * 1e-3)
    out = {
        "metric": "server train samples/s (128-device loop: arrivals, flow control, fused aggregation, pick, step)",
        "value": round(value, 2), "unit": "samples/s", "n_gpus": 1, "steps": steps, "warmup": warm,
        "ms_per_step": round(ms / steps, 4), "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16", "data": "synthetic",
        "config": {"workload": "vgg16 split server step, batch 64 of [64,16,16] bf16 activations, 128 devices, "
                               "arrivals Poisson(lambda_k), lambda_k ~ LogNormal(0,1), 64 GiB activation pool, "
                               "aggregation of the 38,720-parameter device part per arrival (alpha 1, no delay cap)",
                   "global_batch": B, "parallelism": "single-gpu"},
        "loop": {"trained_batches": trained, "idle_steps": tallies["idle_steps"],
                 "arrivals": tallies["arrivals"], "admitted": st.admitted - st0.admitted,
                 "refused": st.refused - st0.refused, "refused_total": st.refused,
                 "pool_slots": n_slots, "omega": st.omega, "pool_peak_occupancy": st.peak_queued,
                 "models_applied": tallies["applied"], "models_skipped": tallies["skipped"],
                 "fused_drains": tallies["drains"], "host_wall_ms_per_step": round(wall / steps * 1e3, 3)},
        "step_only": {"ms": round(step_ms, 4), "samples_per_s": round(B / (step_ms * 1e-3), 1),
                      "mfu": round(VGG_STEP_GFLOP * 1e9 / (step_ms * 1e-3) / (PEAK_BF16_TFLOPS * 1e12), 4)},
        "fused_aggregation": fused,
    }
    print(json.dumps(out), flush=True)


def bench_pipeline(args, A, torch, S):
    """The concurrent pipeline (fo_pipeline_run) on the 128-device VGG-16 split
    workload: config 5's server model, 64 GiB pool, bank of activation batches
    and 38,720-parameter device models.  Device k's local iteration takes
    step_ms / lambda_k (lambda_k ~ LogNormal(0,1) arrivals per server step, as in
    the step loop: server-bound), or, in the balanced regime, periods scaled so
    that all devices together send one batch per server step time.  Each run
    lasts --pipeline-seconds; dropout draws every 0.25 s, slow-down factors
    U[1, 2]; a model message every local iteration (H = 1), alpha 1."""
    cid = 5
    cfg = S.get_config(cid)
    K, B = cfg.n_devices, cfg.batch
    stream = torch.cuda.current_stream()
    pool_stream = torch.cuda.Stream()
    bank_n = cfg.extra["bank"]
    acts_d = torch.from_numpy(S.make_acts(cid, bank_n).view(np.int16)).cuda()
    labels_d = torch.from_numpy(S.make_labels(cid, bank_n)).cuda()
    locs = torch.from_numpy(S.make_local_vectors(cid, K)).cuda()
    slot_bytes = int(acts_d[0].numel()) * 2
    n_slots = cfg.extra["pool_bytes"] // slot_bytes
    rates = S.make_arrival_rates(cid)
    A.fo_set_max_delay(-1)
    # the server step alone, for the device periods
    model = A.fo_model_create(cid, B, S.init_params(cid), stream)
    for _ in range(3):
        A.fo_server_step(model, (acts_d[0], None, B), labels_d[0], 0)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(20):
        A.fo_server_step(model, (acts_d[0], None, B), labels_d[0], 0)
    e1.record(stream)
    torch.cuda.synchronize()
    step_s = e0.elapsed_time(e1) / 20 * 1e-3
    A.fo_model_destroy(model)
    regimes = {"workload rates (server-bound)": step_s / rates,
               "balanced": step_s / rates * float(rates.sum())}
    runs = []
    for regime, periods in regimes.items():
        T0 = None
        for p in (0.0, 0.25, 0.5):
            model = A.fo_model_create(cid, B, S.init_params(cid), stream)
            q = A.fo_queues_create(K, slot_bytes, B, False, n_slots, pool_stream)
            glob = torch.from_numpy(S.make_global_vector(cid)).cuda()
            try:
                st = A.fo_pipeline_run(q, model, glob, dict(
                    seconds=args.pipeline_seconds, iter_seconds=periods, H=1, p_drop=p, interval_seconds=0.25,
                    slow_max=2.0, seed=17, bank_x=acts_d, bank_labels=labels_d, bank_n=bank_n, local_bank=locs,
                    n_local=K, alpha=1.0, max_inflight=2))
            finally:
                A.fo_queues_destroy(q)
                A.fo_model_destroy(model)
            T = st.samples / st.wall_seconds
            T0 = T if p == 0.0 else T0
            runs.append({"regime": regime, "p": p, "T_samples_per_s": round(T, 1), "R": round(T / T0, 3),
                         "server_idle_fraction": round(st.idle_seconds / st.wall_seconds, 4),
                         "steps": st.steps, "sent": st.sent, "not_sent": st.not_sent,
                         "aggregations": st.aggregations, "leaves": st.leaves, "rejoins": st.rejoins,
                         "wall_s": round(st.wall_seconds, 3)})
            print(json.dumps(runs[-1]), flush=True)
    print(json.dumps({"metric": "concurrent pipeline: server train samples/s T(p) and retention R(p) under "
                                "device dropout p (Sec. 6.4)",
                      "unit": "samples/s", "n_gpus": 1, "dtype": "bf16", "data": "synthetic",
                      "step_only_ms": round(step_s * 1e3, 4),
                      "config": {"workload": "vgg16 split server step, batch 64 of [64,16,16] bf16 activations, "
                                             "128 emulated devices, 64 GiB activation pool, counter-based "
                                             "scheduler, dropout draws every 0.25 s, slow-down U[1,2]",
                                 "parallelism": "single-gpu"},
                      "runs": runs}), flush=True)


def device_flops_per_sample():
    """Useful FLOPs of one device-side training iteration per sample (config 6):
    forward of conv1 (3->64 at 32x32), conv2 (64->64 at 32x32), the auxiliary
    conv (64->64 at 16x16) and linear (64->10); input and weight gradients of
    all but conv1, whose input is data (weight gradient only)."""
    conv1 = 2 * 32 * 32 * 64 * 27
    conv2 = 2 * 32 * 32 * 64 * 576
    aux = 2 * 16 * 16 * 64 * 576
    fc = 2 * 64 * 10
    return (conv1 + conv2 + aux + fc) + (conv1 + 2 * conv2 + 2 * aux + 2 * fc)


def bench_device(args, A, torch, S):
    """The device-side iteration of Alg. 1 (config 6) on one GPU: device
    network, the activations it sends, auxiliary network, local loss,
    backward and SGD, over a bank of CIFAR-10-shaped input batches."""
    cid = 6
    cfg = S.get_config(cid)
    B = cfg.batch
    stream = torch.cuda.current_stream()
    bank_n = 8
    xs = torch.from_numpy(S.make_acts(cid, bank_n)).cuda()
    labs = torch.from_numpy(S.make_labels(cid, bank_n)).cuda()
    out = torch.empty((bank_n, B * 64 * 16 * 16), dtype=torch.int16, device="cuda")
    model = A.fo_model_create(cid, B, S.init_params(cid), stream)
    try:
        def run(t0, n):
            for t in range(t0, t0 + n):
                i = t % bank_n
                A.fo_device_step(model, xs[i], labs[i], B, out[i])
        run(0, args.warmup)
        torch.cuda.synchronize()
        ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        ev0.record(stream)
        run(args.warmup, args.steps)
        ev1.record(stream)
        torch.cuda.synchronize()
        ms = ev0.elapsed_time(ev1) / args.steps
        A.fo_profile_enable(100 * args.steps)
        run(0, args.steps)
        torch.cuda.synchronize()
        stats = A.fo_profile_read(64)
        A.fo_profile_enable(0)
    finally:
        A.fo_model_destroy(model)
    flops = device_flops_per_sample() * B
    kernels = [{"name": s["name"], "launches": s["launches"], "ms_per_step": round(s["ms"] / args.steps, 4),
                "TFLOP/s": round(s["flops"] / max(s["ms"], 1e-9) / 1e9, 1) if s["flops"] else None}
               for s in sorted(stats, key=lambda s: -s["ms"])]
    out_line = {
        "metric": "device-side train samples/s (Alg. 1: device network, activations sent, auxiliary network, "
                  "local loss, backward, SGD)",
        "value": round(B / (ms * 1e-3), 2), "unit": "samples/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms, 4), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": "vgg16 split device side: conv3x3 3->64, conv3x3 64->64, maxpool (sends "
                               "[64,16,16]), auxiliary conv3x3 64->64 + avgpool + linear 64->10, batch 64 of "
                               "32x32 RGB", "global_batch": B, "parallelism": "single-gpu"},
        "mfu": round(flops / (ms * 1e-3) / (PEAK_BF16_TFLOPS * 1e12), 5),
        "useful_gflop_per_step": round(flops / 1e9, 3),
        "kernels": kernels[:10],
    }
    print(json.dumps(out_line), flush=True)


def main():
    args = parse()
    if args.summarize_pmc:
        print(json.dumps(summarize_pmc(*args.summarize_pmc), indent=1))
        return
    if args.summarize_trace:
        print(summarize_trace(args.summarize_trace))
        return
    if args.summarize_counters:
        print(summarize_counters(args.summarize_counters))
        return
    if args.gpus != 1:
        sys.stderr.write("bench.py measures one GPU only: this build has no multi-GPU path "
                         f"(asked for --gpus {args.gpus}).\n")
        sys.exit(2)
    import torch
    import fo_synth as S
    from paper_2504_13850_amd import api as A

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    cid = args.config
    if args.pipeline:
        bench_pipeline(args, A, torch, S)
        return
    if cid == 6:
        args.steps = 30 if args.steps is None else args.steps
        args.warmup = 5 if args.warmup is None else args.warmup
        bench_device(args, A, torch, S)
        return
    if cid == 5:
        args.steps = 1000 if args.steps is None else args.steps
        args.warmup = 10 if args.warmup is None else args.warmup
        bench_vgg128(args, A, torch, S)
        return
    if cid not in WORKLOADS:
        raise SystemExit("bench.py: --config 1..10 (4, the transformer, is the default)")
    args.steps = 30 if args.steps is None else args.steps
    args.warmup = 5 if args.warmup is None else args.warmup
    cfg = S.get_config(cid)
    B, K = cfg.batch, cfg.n_devices
    bert = cfg.family in ("bert", "tfsmall")  # batches carry sequence lengths
    stream = torch.cuda.current_stream()

    # ---------------- synthetic inputs, resident in HBM before timing
    bank_n = 16
    acts_h = S.make_acts(cid, bank_n)                 # fp32, or bf16 bits, [n, B, ...]
    labels_h = S.make_labels(cid, bank_n)
    acts_d = torch.from_numpy(acts_h if cfg.dtype == "f32" else acts_h.view(np.int16)).cuda()
    labels_d = torch.from_numpy(labels_h).cuda()
    lengths_d = torch.from_numpy(S.make_lengths(cid, bank_n)).cuda() if bert else None
    del acts_h
    theta = S.init_params(cid)
    model = A.fo_model_create(cid, B, theta, stream)
    slot_bytes = int(acts_d[0].numel() * acts_d.element_size())
    q = A.fo_queues_create(K, slot_bytes, B, bert, 3 * K, stream)
    # device-side models aggregated once per step (Alg. 4, model branch), where the workload has them
    agg_glob = agg_locs = agg_stale = None
    if cfg.agg_n:
        agg_glob = torch.from_numpy(S.make_global_vector(cid)).cuda()
        agg_locs = torch.from_numpy(S.make_local_vectors(cid, K)).cuda()
        agg_stale = S.make_staleness(cid, args.warmup + 2 * args.steps, 8) if cid == 3 else None
        A.fo_set_stream(stream)

    arrivals = [0]

    def push(k):
        i = arrivals[0] % bank_n
        arrivals[0] += 1
        st = A.fo_queues_push(q, k, acts_d[i], labels_d[i], lengths_d[i] if bert else None)
        return i if st == A.FO_OK else None

    # every device starts with one batch queued
    for k in range(K):
        push(k)

    def one_step(t):
        # arrival from device t % K (Alg. 2 put(), flow control), then get() and train
        push(t % K)
        k = A.fo_pick_device(q)
        fa, lab, seq, slot = A.fo_queues_in_service(q)
        A.fo_server_step(model, fa, lab, k)
        A.fo_queues_release(q)
        if agg_glob is not None:  # one model arrival: device k's local model, staleness as in the workload
            s = k if cid == 1 else int(agg_stale[t])
            A.fo_async_aggregate(agg_glob, agg_locs[k], cfg.agg_alpha, s)
        return k

    for t in range(args.warmup):
        one_step(t)
    torch.cuda.synchronize()

    def timed(nsteps, t0, profile):
        if profile:
            A.fo_profile_enable(400 * nsteps)
        ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        ev0.record(stream)
        t_wall = time.perf_counter()
        for t in range(t0, t0 + nsteps):
            one_step(t)
        ev1.record(stream)
        torch.cuda.synchronize()
        wall = time.perf_counter() - t_wall
        stats = None
        if profile:
            stats = A.fo_profile_read(64)
            A.fo_profile_enable(0)
        return ev0.elapsed_time(ev1), wall, stats

    # ---------------- timed region (headline), then the same steps again with kernel events
    ms_total, wall, _ = timed(args.steps, args.warmup, False)
    ms_prof, _, stats = timed(args.steps, args.warmup + args.steps, True)
    ms_step = ms_total / args.steps
    samples_s = B * args.steps / (ms_total * 1e-3)

    wl = WORKLOADS[cid]
    peak = wl["peak"]
    # useful FLOPs per step from the kernels' own records (valid tokens only), or
    # the workload's fixed count where its kernels carry no records (fp32 CNN)
    alg_flops = sum(s["flops"] for s in stats)
    mfma_flops = sum(s["mfma_flops"] for s in stats)
    gflop = wl["gflop"] if wl["gflop"] is not None else (tfsmall_gflop(cid) if cid in (7, 8) else mbv3_gflop())
    flops_step = alg_flops / args.steps if alg_flops else gflop * 1e9
    mfu = flops_step / (ms_step * 1e-3) / (peak * 1e12)
    gemms = [s for s in stats if s["name"].startswith("gemm")]
    if gemms:
        dom = max(gemms, key=lambda s: s["ms"])
        dom_tflops = dom["flops"] / (dom["ms"] * 1e-3) / 1e12
        roofline = {"bound": "mfma", "kernel": dom["name"], "achieved": round(dom_tflops, 1), "peak": peak,
                    "unit": "TFLOP/s", "frac": round(dom_tflops / peak, 4), "launches": dom["launches"],
                    "avg_launch_us": round(dom["ms"] / dom["launches"] * 1e3, 2), "traffic": traffic_for(dom["name"]),
                    "traffic_source": TRAFFIC_SOURCE}
    else:  # the fp32 direct-convolution CNN: the whole step against the fp32 vector peak
        roofline = {"bound": "alu", "kernel": "whole step (fp32 FMA kernels, not instrumented)",
                    "achieved": round(flops_step / (ms_step * 1e-3) / 1e12, 3), "peak": peak, "unit": "TFLOP/s",
                    "frac": round(mfu, 5), "traffic": None}
    kernels = [{"name": s["name"], "launches": s["launches"], "ms_per_step": round(s["ms"] / args.steps, 4),
                "TFLOP/s": round(s["flops"] / max(s["ms"], 1e-9) / 1e9, 1) if s["flops"] else None}
               for s in sorted(stats, key=lambda s: -s["ms"])]

    agg = bench_aggregate(A, torch, stream)
    t_agg = traffic_for("agg_lerp_kernel")
    agg["traffic"] = t_agg
    agg["traffic_source"] = TRAFFIC_SOURCE
    agg["traffic_frac_of_algorithmic"] = round(t_agg / agg["bytes_per_call"], 4) if t_agg else None
    if args.calib_copy:
        calib_copy(torch)
    A.fo_queues_destroy(q)
    A.fo_model_destroy(model)

    cpu = None if args.no_cpu_baseline else cpu_baseline(cid, args.cpu_sample_steps)

    config = {"workload": wl["workload"], "global_batch": B, "parallelism": "single-gpu"}
    if bert:
        config["seq_len"] = cfg.in_shape[0]
    if bert:  # every sequence at its full 128 tokens: the work a padded run would do (context only)
        out_extra = {"padded_dense_tflop_per_step": round(padded_bert_flops(B, cfg.in_shape[0]) / 1e12, 4)}
    else:
        out_extra = {}
    out = {
        "metric": "server train samples/s + % bf16 MFMA peak; async-aggregate HBM GB/s",
        "value": round(samples_s, 2),
        "unit": "samples/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32" if cfg.dtype == "f32" else "bf16",
        "data": "synthetic",
        "config": config,
        "mfu": round(mfu, 5),
        "mfu_peak_tflops": peak,
        "useful_tflop_per_step": round(flops_step / 1e12, 6),
        "mfma_tflop_per_step_executed": round(mfma_flops / args.steps / 1e12, 4),
        **out_extra,
        "roofline": roofline,
        "aggregate": agg,
        "kernels": kernels[:12],
        "host_wall_ms_per_step": round(wall / args.steps * 1e3, 3),
        "profiled_ms_per_step": round(ms_prof / args.steps, 4),
        "cpu_baseline": cpu,
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
