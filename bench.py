#!/usr/bin/env python3
"""Benchmark of the fused sub-kernels on one MI355X.

One step = one launch of every fused sub-kernel at its workload shape:
  pw_256x1024     pointwise GELU_erf(x*s + b) + r, fp32 [256, 1024]
  sm_8192x4096    row softmax, scale + bf16 additive mask, bf16 [8192, 4096]
  ln_16384x4096   LayerNorm + residual, bf16 [16384, 4096]
  ep_8192x8192    GEMM epilogue (+bias, *scale, sigmoid, row sum) on C bf16 [8192, 8192]
  blk_ln1         block LayerNorm 1, bf16 [16384, 1024]
  blk_sm          block causal softmax, bf16 [32, 16, 512, 512], scale 1/8
  blk_ln2         block LayerNorm 2 + residual, bf16 [16384, 1024]
  blk_gelu        block bias + GELU_erf, bf16 [16384, 4096]
  blk_res         block residual add, bf16 [16384, 1024]
The GEMMs (the fixed library calls) run once before timing to produce the
resident inputs of the epilogue and block sub-kernels; they are reported
separately as context, never inside `value`.

`value` = compulsory bytes of one step (each input read once, each output
written once; the causal upper triangle is not read) / step time, in GB/s.
Inputs are resident in HBM when timing starts.  Every kernel in a step is
separated from its previous launch by more than the 256 MB Infinity Cache of
other traffic, so inputs come from HBM (pw_256x1024, 3 MiB, stays cache
resident and is latency-bound).

Setup ends with a settle pass: steps back to back for at least 25 ms of GPU
time (--settle-ms), so that the engine clock has left the dip it takes in
the first milliseconds of load after idling.  The W warmup steps and the K
timed steps are then enqueued back to back, without a host synchronisation.

Timing: the K timed steps are bracketed by two events; inside them only the
dominant kernel (the longest, picked from the warmup steps) is bracketed, for
`roofline.achieved`.  Every event is a timing-only HIP event (created with
hipEventDisableSystemFence: recording it skips the system-scope cache
writeback and invalidation of a default event, which costs the GPU about 3 us
per event; a timing-only one costs about 1 us).  Events after every kernel
would still lengthen the step by about 3 %, so the per-kernel breakdown comes
from a separate pass after the timed region (medians, with the means beside
them), followed by the same pass over the step's access-shape floors
(libaccessfloor.so: each launch's bytes moved in its launch shape with none of
the arithmetic) when that library is built.

Prints one JSON line.  Two GPU-free modes turn rocprofv3 CSV output of this
script into the summaries under profiles/:
  --report-trace STATS_CSV          per-kernel durations (Markdown table)
  --write-traffic FETCH_CSV WRITE_CSV
                                    HBM bytes per launch -> profiles/traffic.json
A third GPU mode, --long-rows, times softmax and LayerNorm/RMSNorm rows past
the register-resident widths (16392 ... 262144 columns) and prints a Markdown
table (not part of the step).
"""
from __future__ import annotations

import argparse
import hashlib
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

from paper_2609_30059_amd.timing import TimingEvent  # noqa: E402

PEAK_HBM_GBS = 8000.0
SETTLE_MS = 25.0       # back-to-back steps before the warmup (do_bench-style warm-up)
METRIC = "achieved HBM GB/s and % of MI355X peak per fused sub-kernel; oracle match"
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic.json")
KERNEL_SOURCES = {
    "pw": "pointwise.hip", "sm": "softmax.hip", "ln": "layernorm.hip", "ep": "epilogue.hip",
}



# Each bench kernel by its (demangled, anonymous-namespace-free) kernel name in
# rocprofv3 output: the template arguments tell the launches apart.
KERNEL_PATTERNS = {
    "pw_256x1024": r"pointwise_kernel<float, 1, true, true, 1>",       # one row per trip
    "pw_262144x1024": r"pointwise_kernel<float, 1, true, true, 4>",    # four rows per trip
    "sm_8192x4096": r"softmax_kernel<unsigned short, unsigned short, true,",
    "ln_16384x4096": r"layernorm_kernel<unsigned short, true, false, 2,",
    "ep_8192x8192": r"epilogue_lds_kernel<unsigned short, unsigned short, 2,",
    "blk_ln1": r"layernorm_wave_kernel<unsigned short, false, false, 16,",
    "blk_sm": r"softmax_kernel<unsigned short, unsigned short, false,",
    "blk_ln2": r"layernorm_wave_kernel<unsigned short, true, false, 16,",
    "blk_gelu": r"pointwise_kernel<unsigned short, 1, false,",
    "blk_res": r"pointwise_flat_kernel<unsigned short, 0, true,",
    "copy_1GiB": r"copy128_kernel",
}
KIND = {"pw_256x1024": "pw", "pw_262144x1024": "pw", "sm_8192x4096": "sm",
        "ln_16384x4096": "ln", "ep_8192x8192": "ep", "blk_ln1": "ln", "blk_sm": "sm",
        "blk_ln2": "ln", "blk_gelu": "pw", "blk_res": "pw"}
# compulsory bytes per launch (block: batch 32, seq 512, hidden 1024, 16 heads, MLP 4096)
_T, _H, _F, _NH, _S = 32 * 512, 1024, 4096, 16, 512
STEP_BYTES = {
    "pw_256x1024": 256 * 1024 * 4 * 3 + 1024 * 4,
    "pw_262144x1024": 262144 * 1024 * 4 * 3 + 1024 * 4,    # context, not in the step
    "sm_8192x4096": 8192 * 4096 * 2 * 3,
    "ln_16384x4096": 16384 * 4096 * 2 * 4 + 4096 * 2 * 2,
    "ep_8192x8192": 8192 * 8192 * 2 + 8192 * (2 + 4) + 8192 * 4,
    "blk_ln1": _T * _H * 2 * 2 + _H * 2 * 2,
    "blk_sm": 32 * _NH * (_S * (_S + 1) // 2) * 2 + 32 * _NH * _S * _S * 2,
    "blk_ln2": _T * _H * 2 * 4 + _H * 2 * 2,
    "blk_gelu": _T * _F * 2 * 2 + _F * 2,
    "blk_res": _T * _H * 2 * 3,
    "copy_1GiB": 2 << 30,
}


def _match(names, label):
    import re
    hits = [n for n in names if re.search(KERNEL_PATTERNS[label], n)]
    if len(hits) > 1:
        raise ValueError(f"{label}: pattern matches {len(hits)} kernels: {hits}")
    return hits[0] if hits else None


def report_trace(stats_csv: str, every: bool = False) -> None:
    """Markdown table of the bench kernels' rocprofv3 durations; with `every`,
    of every kernel of this library in the stats file (by name, without byte
    counts)."""
    import csv
    rows = {}
    with open(stats_csv, newline="") as f:
        for r in csv.DictReader(f):
            rows[r["Name"].replace("(anonymous namespace)::", "")] = r
    total = sum(float(r["TotalDurationNs"]) for r in rows.values())
    if every:
        print("| kernel | calls | avg us | min us | max us | % of GPU time |")
        print("|---|---|---|---|---|---|")
        ours = {n: r for n, r in rows.items() if "fs::" in n}
        for n, r in sorted(ours.items(), key=lambda kv: -float(kv[1]["TotalDurationNs"])):
            short = n.split("(")[0].replace("void ", "").replace("fs::", "")
            print(f"| `{short}` | {r['Calls']} | {float(r['AverageNs']) / 1e3:.2f} | "
                  f"{float(r['MinNs']) / 1e3:.2f} | {float(r['MaxNs']) / 1e3:.2f} | "
                  f"{100 * float(r['TotalDurationNs']) / total:.1f} |")
        return
    print("| kernel | calls | avg us | min us | max us | % of GPU time | GB/s (avg) | % of 8 TB/s |")
    print("|---|---|---|---|---|---|---|---|")
    for label in KERNEL_PATTERNS:
        n = _match(rows, label)
        if n is None:
            continue
        r = rows[n]
        avg = float(r["AverageNs"])
        gbs = STEP_BYTES[label] / avg
        print(f"| {label} | {r['Calls']} | {avg / 1e3:.2f} | {float(r['MinNs']) / 1e3:.2f} | "
              f"{float(r['MaxNs']) / 1e3:.2f} | {100 * float(r['TotalDurationNs']) / total:.1f} | "
              f"{gbs:.0f} | {100 * gbs / PEAK_HBM_GBS:.1f} |")


def write_traffic(fetch_csv: str, write_csv: str, measured_at: str, cmd_fetch: str,
                  cmd_write: str) -> dict:
    """HBM bytes per launch of every bench kernel from FETCH_SIZE and
    WRITE_SIZE runs, each counter scaled by what it reads for the 1 GiB
    calibration copy of the same run; written to profiles/traffic.json with
    the hash of each kernel's sources (bench.py reports a kernel's traffic
    only while its sources still hash the same)."""
    from paper_2609_30059_amd import tiers
    prof = {}
    tiers.read_counters(fetch_csv, prof)
    tiers.read_counters(write_csv, prof)
    fs_, ws_ = tiers.copy_scales(prof, KERNEL_PATTERNS["copy_1GiB"], float(1 << 30),
                                 float(1 << 30))
    out = {"fetch_scale": fs_, "write_scale": ws_, "measured_at": measured_at,
           "command_fetch": cmd_fetch, "command_write": cmd_write}
    for label in KERNEL_PATTERNS:
        n = _match(prof, label)
        if n is None or label not in KIND:
            continue
        p = prof[n]
        out[label] = {"source_hash": source_hash(KIND[label]),
                      "fetch_kib": round(p.fetch_kib, 1), "write_kib": round(p.write_kib, 1),
                      "bytes_per_launch": round(p.hbm_bytes(fs_, ws_)),
                      "algorithmic_bytes": STEP_BYTES[label]}
    with open(TRAFFIC_FILE, "w") as f:
        json.dump(out, f, indent=1)
        f.write("\n")
    return out


def source_hash(kind: str) -> str:
    csrc = os.path.join(ROOT, "paper_2609_30059_amd", "csrc")
    h = hashlib.sha256()
    for f in (KERNEL_SOURCES[kind], "device_common.hpp"):
        with open(os.path.join(csrc, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def parse():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawTextHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--settle-ms", type=float, default=SETTLE_MS,
                    help="GPU time of back-to-back steps run before the warmup steps")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-copy-reference", action="store_true",
                    help="skip the same-size copies (profiling runs: every copy dispatch is "
                         "then the 1 GiB calibration that scales the byte counters)")
    ap.add_argument("--cpu-sample", type=float, default=1.0,
                    help="fraction of each sub-kernel's rows the CPU oracle baseline runs over")
    ap.add_argument("--report-trace", metavar="STATS_CSV",
                    help="print the bench kernels' durations from a rocprofv3 kernel-stats CSV")
    ap.add_argument("--all-kernels", action="store_true",
                    help="with --report-trace: list every kernel of the stats file")
    ap.add_argument("--write-traffic", nargs=2, metavar=("FETCH_CSV", "WRITE_CSV"),
                    help="write profiles/traffic.json from FETCH_SIZE and WRITE_SIZE runs")
    ap.add_argument("--measured-at", default="", help="commit the counter runs measured")
    ap.add_argument("--commands", nargs=2, default=("", ""), metavar=("FETCH_CMD", "WRITE_CMD"),
                    help="the rocprofv3 commands of the two counter runs (recorded)")
    ap.add_argument("--program-costs", action="store_true",
                    help="pointwise programs of growing arithmetic against the fixed chain, and "
                         "the row reductions (sum, max, log-sum-exp), each launch after a "
                         "read-only 1 GiB pass")
    ap.add_argument("--long-rows", action="store_true",
                    help="time long-row softmax and LayerNorm/RMSNorm and print a Markdown table")
    ap.add_argument("--odd-rows", action="store_true",
                    help="time rows that are not whole 16-byte vectors (the aligned-body "
                         "variants) and print a Markdown table")
    ap.add_argument("--report-counters", nargs="+", metavar="COUNTER_CSV",
                    help="LDS and occupancy table from rocprofv3 --pmc counter-collection CSVs")
    ap.add_argument("--epilogue-context", action="store_true",
                    help="launch the GEMM epilogue in four contexts separated by pauses "
                         "(run under a kernel trace)")
    ap.add_argument("--report-context", metavar="TRACE_CSV",
                    help="the --epilogue-context table from a rocprofv3 kernel-trace CSV")
    ap.add_argument("--copy-floor", action="store_true",
                    help="time the short block kernels next to copies moving the same bytes, "
                         "each after a read-only 1 GiB pass (run under a kernel trace)")
    ap.add_argument("--clock-transient", action="store_true",
                    help="bench steps right after an idle pause, each followed by an "
                         "engine-clock probe (run under a kernel trace)")
    ap.add_argument("--report-transient", nargs=2, metavar=("TRACE_CSV", "LOG"),
                    help="the --clock-transient table from its kernel trace and printed lines")
    ap.add_argument("--report-floor", metavar="TRACE_CSV",
                    help="the --copy-floor table from a rocprofv3 kernel-trace CSV")
    ap.add_argument("--access-floors", action="store_true",
                    help="time every step sub-kernel next to its access-shape floor "
                         "(libaccessfloor.so), each after a read-only 1 GiB pass (run under "
                         "a kernel trace)")
    ap.add_argument("--report-floors", metavar="TRACE_CSV",
                    help="the --access-floors table from a rocprofv3 kernel-trace CSV")
    return ap.parse_args()


# ---------------------------------------------------------------------------
# workload
# ---------------------------------------------------------------------------
class Workload:
    def __init__(self, seed):
        import numpy as np
        import torch

        import fusedsub_data as fd
        import paper_2609_30059_amd as fs
        self.fs, self.torch, self.np, self.fd = fs, torch, np, fd
        dev = "cuda"
        self.host = {}

        def d(t):
            if t is None:
                return None
            if t.dtype == "f32":
                return torch.from_numpy(t.data).to(dev)
            return torch.from_numpy(t.data.view(np.int16)).view(torch.bfloat16).to(dev)

        # pointwise_256x1024
        h1 = fd.make_inputs("pointwise_256x1024", seed)
        self.host["pointwise_256x1024"] = h1
        self.pw = dict(x=d(h1["x"]), b=d(h1["bias"]), r=d(h1["residual"]), s=h1["scale"])
        self.pw["y"] = torch.empty_like(self.pw["x"])
        # the same chain at bandwidth scale, [262144, 1024] (the [256, 1024]
        # draws repeated), measured as context outside the step
        reps = 262144 // 256
        self.pwbw = dict(x=self.pw["x"].repeat(reps, 1), r=self.pw["r"].repeat(reps, 1))
        self.pwbw["y"] = torch.empty_like(self.pwbw["x"])
        # softmax_8192x4096
        h2 = fd.make_inputs("softmax_8192x4096", seed)
        self.host["softmax_8192x4096"] = h2
        self.sm = dict(x=d(h2["x"]), m=d(h2["mask"]), s=h2["scale"])
        self.sm["y"] = torch.empty_like(self.sm["x"])
        # the same mask as bytes (nonzero = excluded), measured as context
        self.sm["m8"] = (self.sm["m"] != 0).to(torch.uint8)
        # layernorm_16384x4096
        h3 = fd.make_inputs("layernorm_16384x4096", seed)
        self.host["layernorm_16384x4096"] = h3
        self.ln = dict(x=d(h3["x"]), r=d(h3["residual"]), g=d(h3["gamma"]), b=d(h3["beta"]),
                       eps=h3["eps"])
        self.ln["y"] = torch.empty_like(self.ln["x"])
        self.ln["ro"] = torch.empty_like(self.ln["x"])
        # GEMM [8192, 4096] x [4096, 8192] once (library call), then the epilogue on its output
        h4 = fd.make_inputs("gemm_epilogue_8192x8192x4096", seed)
        self.host["gemm_epilogue_8192x8192x4096"] = h4
        a, b = d(h4["a"]), d(h4["b"])
        self.ep = dict(bias=d(h4["bias"]), scale=d(h4["col_scale"]))
        self.ep["c"] = fs.gemm(a, b)
        self.ep["out"] = torch.empty(self.ep["c"].shape[0], dtype=torch.float32, device=dev)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(3):
            fs.gemm(a, b, out=self.ep["c"])
        torch.cuda.synchronize()
        self.gemm_8192x8192x4096_ms = (time.perf_counter() - t0) / 3 * 1e3
        del a, b
        # block_32x512x1024: one full forward pass makes every block sub-kernel input resident
        h5 = fd.make_inputs("block_32x512x1024", seed)
        self.host["block_32x512x1024"] = {k: h5[k] for k in ("x", "eps", "heads")}
        params = {k: d(h5[k]) for k in fs.block.PARAM_NAMES}
        self.blk = fs.TransformerBlock(params, heads=h5["heads"], eps=h5["eps"])
        self.bx = d(h5["x"])
        self.buf = self.blk.forward(self.bx)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(3):
            self.blk.forward(self.bx, self.buf)
        torch.cuda.synchronize()
        self.block_e2e_ms = (time.perf_counter() - t0) / 3 * 1e3

        B, S, H = self.bx.shape
        NH, F = self.blk.heads, self.blk.mlp
        T = B * S
        causal_read = B * NH * (S * (S + 1) // 2) * 2
        # (name, kind, compulsory bytes, launch closure)
        fsb = self.blk
        p = fsb.p
        x2 = self.bx.view(T, H)
        buf = self.buf
        self.kernels = [
            ("pw_256x1024", "pw", 256 * 1024 * 4 * 3 + 1024 * 4,
             lambda: fs.pointwise_chain(self.pw["x"], self.pw["b"], self.pw["r"], self.pw["s"],
                                        "gelu_erf", out=self.pw["y"])),
            ("sm_8192x4096", "sm", 8192 * 4096 * 2 * 3,
             lambda: fs.row_softmax(self.sm["x"], self.sm["m"], self.sm["s"], out=self.sm["y"])),
            ("ln_16384x4096", "ln", 16384 * 4096 * 2 * 4 + 4096 * 2 * 2,
             lambda: fs.layernorm_residual(self.ln["x"], self.ln["r"], self.ln["g"], self.ln["b"],
                                           self.ln["eps"], out=self.ln["y"],
                                           residual_out=self.ln["ro"])),
            ("ep_8192x8192", "ep", 8192 * 8192 * 2 + 8192 * (2 + 4) + 8192 * 4,
             lambda: fs.gemm_epilogue_reduce(self.ep["c"], self.ep["bias"], self.ep["scale"],
                                             "sigmoid", "sum", out=self.ep["out"])),
            ("blk_ln1", "ln", T * H * 2 * 2 + H * 2 * 2,
             lambda: fs.layernorm_residual(x2, None, p["ln1_gamma"], p["ln1_beta"], fsb.eps,
                                           out=buf["a"])),
            ("blk_sm", "sm", causal_read + B * NH * S * S * 2,
             lambda: fs.row_softmax(buf["scores"], None, 1.0 / math.sqrt(fsb.dh),
                                    causal_q_len=S, out=buf["probs"])),
            ("blk_ln2", "ln", T * H * 2 * 4 + H * 2 * 2,
             lambda: fs.layernorm_residual(buf["att"], x2, p["ln2_gamma"], p["ln2_beta"],
                                           fsb.eps, out=buf["m"], residual_out=buf["h1"])),
            ("blk_gelu", "pw", T * F * 2 * 2 + F * 2,
             lambda: fs.pointwise_chain(buf["u"], p["b_1"], None, 1.0, "gelu_erf",
                                        out=buf["g"])),
            ("blk_res", "pw", T * H * 2 * 3,
             lambda: fs.pointwise_chain(buf["d"], None, buf["h1"], 1.0, "none",
                                        out=buf["out"])),
        ]
        self.step_bytes = sum(k[2] for k in self.kernels)
        for name, _, nbytes, _ in self.kernels:
            assert nbytes == STEP_BYTES[name], name
        # one launch of each kernel, so that loading its code object is not
        # part of any measured interval
        for _, _, _, fn in self.kernels:
            fn()
        torch.cuda.synchronize()

    def step(self, events=None):
        for i, (_, _, _, fn) in enumerate(self.kernels):
            fn()
            if events is not None:
                events[i + 1].record()

    def copy_calibration(self, nbytes=1 << 30, iters=10):
        torch, fs = self.torch, self.fs
        src = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
        dst = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
        fs.copy_(dst, src)
        torch.cuda.synchronize()
        e0, e1 = TimingEvent(), TimingEvent()
        e0.record()
        for _ in range(iters):
            fs.copy_(dst, src)
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / iters
        del src, dst
        return 2 * nbytes / (ms * 1e-3) / 1e9

    def pointwise_bandwidth_scale(self, reps):
        """Median launch interval of the fp32 chain at [262144, 1024] (3 GiB
        moved): the 3 MiB workload is latency-bound, this one carries the
        chain's bandwidth.  Each launch is bracketed by its own two events."""
        torch, fs, p = self.torch, self.fs, self.pwbw
        fn = lambda: fs.pointwise_chain(p["x"], self.pw["b"], p["r"], self.pw["s"], "gelu_erf",
                                        out=p["y"])
        fn()
        torch.cuda.synchronize()
        evs = [(TimingEvent(), TimingEvent())
               for _ in range(reps)]
        for a, b in evs:
            a.record()
            fn()
            b.record()
        torch.cuda.synchronize()
        ts = sorted(a.elapsed_time(b) for a, b in evs)
        return ts[reps // 2]

    def softmax_byte_mask(self, reps):
        """Median launch intervals of the [8192, 4096] softmax with its mask
        as bytes and, alternating with it, as the additive bf16 mask; each
        launch follows a read-only pass over 1 GiB (inputs come from HBM) and
        is bracketed by its own two events.  Returns (byte us, additive us)."""
        torch, fs, p = self.torch, self.fs, self.sm
        scrub = torch.zeros(8192, 65536, dtype=torch.bfloat16, device="cuda")
        sink = torch.empty(8192, dtype=torch.float32, device="cuda")
        fns = [lambda: fs.row_softmax(p["x"], p["m8"], p["s"], out=p["y"]),
               lambda: fs.row_softmax(p["x"], p["m"], p["s"], out=p["y"])]
        ts = [[], []]
        for rep in range(reps + 1):            # the first repetition is a warm-up
            for i, fn in enumerate(fns):
                fs.row_reduce(scrub, "sum", out=sink)
                a, b = TimingEvent(), TimingEvent()
                a.record()
                fn()
                b.record()
                torch.cuda.synchronize()
                if rep:
                    ts[i].append(a.elapsed_time(b))
        del scrub
        return tuple(sorted(t)[reps // 2] * 1e3 for t in ts)

    def pointwise_program(self, reps):
        """Median launch intervals of a fused pointwise program -- bias, a
        multiply, a hardtanh and a GELU on the block's bf16 [16384, 4096]
        MLP activations -- and, alternating with it, of the fixed bias + GELU
        chain on the same tensors; each launch after a read-only pass over
        1 GiB, with its own events.  Returns (program us, chain us, bytes)."""
        torch, fs = self.torch, self.fs
        g = torch.Generator(device="cuda").manual_seed(7)
        x = (0.5 * torch.randn(16384, 4096, device="cuda", generator=g)).to(torch.bfloat16)
        b = (0.02 * torch.randn(4096, device="cuda", generator=g)).to(torch.bfloat16)
        y = torch.empty_like(x)
        ops = [("add_bias",), ("scale", 0.5), ("clamp", -1.0, 1.0), ("gelu_erf",)]
        scrub = torch.zeros(8192, 65536, dtype=torch.bfloat16, device="cuda")
        sink = torch.empty(8192, dtype=torch.float32, device="cuda")
        fns = [lambda: fs.pointwise_program(x, ops, bias=b, out=y),
               lambda: fs.pointwise_chain(x, b, None, 1.0, "gelu_erf", out=y)]
        ts = [[], []]
        for rep in range(reps + 1):            # the first repetition is a warm-up
            for i, fn in enumerate(fns):
                fs.row_reduce(scrub, "sum", out=sink)
                e0, e1 = TimingEvent(), TimingEvent()
                e0.record()
                fn()
                e1.record()
                torch.cuda.synchronize()
                if rep:
                    ts[i].append(e0.elapsed_time(e1))
        del scrub, x, y
        nbytes = 16384 * 4096 * 2 * 2 + 4096 * 2
        return (*(sorted(t)[reps // 2] * 1e3 for t in ts), nbytes)

    def same_size_copies(self, sizes, reps):
        """Median interval of a calibration copy moving the same number of
        bytes as each kernel (half read, half written), timed like the
        per-kernel pass (an event after every launch).  Successive copies
        take different slices of 1 GiB buffers, so their inputs come from
        HBM, not the Infinity Cache."""
        torch, fs = self.torch, self.fs
        span = 1 << 30
        src = torch.empty(span, dtype=torch.uint8, device="cuda")
        dst = torch.empty(span, dtype=torch.uint8, device="cuda")
        out = []
        for nbytes in sizes:
            half = (nbytes // 2 + 4095) // 4096 * 4096
            evs = [TimingEvent() for _ in range(reps + 1)]
            off = 0
            evs[0].record()
            for i in range(reps):
                if off + half > span:
                    off = 0
                fs.copy_(dst[off:off + half], src[off:off + half])
                off += half
                evs[i + 1].record()
            torch.cuda.synchronize()
            ts = sorted(evs[i].elapsed_time(evs[i + 1]) for i in range(reps))
            out.append(ts[reps // 2])
        del src, dst
        return out


# ---------------------------------------------------------------------------
# CPU baseline: the float64 oracle over the same step, on the host
# ---------------------------------------------------------------------------
def cpu_baseline(wl: Workload, frac: float):
    """Times the float64 oracle, one thread, over the rows of every sub-kernel
    of one step (``frac`` of the rows of each; 1.0 = the whole step).  Host
    inputs come from the seeded generators at the same shapes and
    distributions (their generation is not timed); nothing is read back from
    the device.  Rows are independent, so the oracle runs in row chunks to
    bound memory."""
    import numpy as np
    from threadpoolctl import threadpool_limits

    import oracle
    fd = wl.fd
    h = wl.host
    blk = wl.blk
    H, F = blk.hidden, blk.mlp
    B, S = wl.bx.shape[0], wl.bx.shape[1]
    T = B * S
    eps = blk.eps
    seed = 7
    g64 = {k: v.float().cpu().numpy().astype(np.float64) for k, v in blk.p.items()}
    # host stand-ins for the resident block activations (same shapes and dtypes)
    blk_x = h["block_32x512x1024"]["x"].f64().reshape(T, H)
    scores = fd.softmax_inputs(seed, B * blk.heads * S, S, "bf16", sigma=1.0, mask_dtype=None)
    att = fd.layernorm_inputs(seed, T, H, "bf16")
    u = fd.pointwise_inputs(seed, T, F, "bf16", with_residual=False)
    dres = fd.pointwise_inputs(seed + 1, T, H, "bf16", with_bias=False)
    epi = fd.epilogue_inputs(seed, 8192, 8192)
    c1, c2, c3 = h["pointwise_256x1024"], h["softmax_8192x4096"], h["layernorm_16384x4096"]

    def n(rows):
        return max(1, int(rows * frac))

    # (name, rows, chunk, bytes per row, fn(lo, hi)) -- f64 conversion of the
    # inputs is part of the oracle's work and is timed
    jobs = [
        ("pw_256x1024", 256, 256, 1024 * 12,
         lambda lo, hi: oracle.pointwise_chain(c1["x"].rows(slice(lo, hi)).f64(), c1["bias"].f64(),
                                               c1["residual"].rows(slice(lo, hi)).f64(),
                                               c1["scale"], "gelu_erf")),
        ("sm_8192x4096", n(8192), 1024, 4096 * 6,
         lambda lo, hi: oracle.row_softmax(c2["x"].rows(slice(lo, hi)).f64(),
                                           c2["mask"].rows(slice(lo, hi)).f64(), c2["scale"])),
        ("ln_16384x4096", n(16384), 1024, 4096 * 8,
         lambda lo, hi: (oracle.layernorm_residual(c3["x"].rows(slice(lo, hi)).f64(),
                                                   c3["residual"].rows(slice(lo, hi)).f64(),
                                                   c3["gamma"].f64(), c3["beta"].f64(), c3["eps"]),
                         oracle.residual_store_bf16(c3["x"].rows(slice(lo, hi)).f64(),
                                                    c3["residual"].rows(slice(lo, hi)).f64()))),
        ("ep_8192x8192", n(8192), 512, 8192 * 2 + 4,
         lambda lo, hi: oracle.gemm_epilogue_reduce(epi["c"].rows(slice(lo, hi)).f64(),
                                                    epi["bias"].f64(), epi["col_scale"].f64(),
                                                    "sigmoid", "sum")),
        ("blk_ln1", n(T), 4096, H * 4,
         lambda lo, hi: oracle.layernorm_residual(blk_x[lo:hi], None, g64["ln1_gamma"],
                                                  g64["ln1_beta"], eps)),
        ("blk_sm", n(B * blk.heads * S), 16384, 3 * S + 1,   # mean causal row: (S+1) read, 2S written
         lambda lo, hi: oracle.row_softmax(scores["x"].rows(slice(lo, hi)).f64(), None,
                                           1.0 / math.sqrt(blk.dh), causal_q_len=S)),
        ("blk_ln2", n(T), 4096, H * 8,
         lambda lo, hi: oracle.layernorm_residual(att["x"].rows(slice(lo, hi)).f64(),
                                                  att["residual"].rows(slice(lo, hi)).f64(),
                                                  g64["ln2_gamma"], g64["ln2_beta"], eps)),
        ("blk_gelu", n(T), 2048, F * 4,
         lambda lo, hi: oracle.pointwise_chain(u["x"].rows(slice(lo, hi)).f64(), g64["b_1"], None,
                                               1.0, "gelu_erf")),
        ("blk_res", n(T), 4096, H * 6,
         lambda lo, hi: oracle.pointwise_chain(dres["x"].rows(slice(lo, hi)).f64(), None,
                                               dres["residual"].rows(slice(lo, hi)).f64(), 1.0,
                                               "none")),
    ]
    per = {}
    total_bytes = 0
    total_s = 0.0
    with threadpool_limits(limits=1):
        for name, rows, chunk, bpr, fn in jobs:
            t0 = time.perf_counter()
            for lo in range(0, rows, chunk):
                fn(lo, min(rows, lo + chunk))
            dt = time.perf_counter() - t0
            nbytes = rows * bpr
            per[name] = {"rows": rows, "s": round(dt, 3), "GB/s": round(nbytes / dt / 1e9, 4)}
            total_bytes += nbytes
            total_s += dt
    return {"value": round(total_bytes / total_s / 1e9, 4), "unit": "GB/s", "cores": 1,
            "kind": "oracle", "seconds": round(total_s, 2),
            "sample": f"float64 oracle, one thread, over "
                      f"{'all' if frac >= 1 else f'a fraction {frac:g}'} of the rows of every "
                      f"sub-kernel of one step ({total_bytes} compulsory bytes), on host "
                      f"inputs of the same shapes from the seeded generators",
            "cpu_model": cpu_model(), "affinity_cores": len(os.sched_getaffinity(0)),
            "per_kernel": per, "blas_legs": blas_legs(wl)}


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def blas_legs(wl: "Workload", gemm_rows: int = 512, block_seqs: int = 2):
    """The float64 legs that run through BLAS, each on a bounded sample, with
    the BLAS thread count set to the process's affinity cores: the product
    A.B of the GEMM-epilogue workload (its first rows) and the whole-block
    oracle (its first sequences).  Each reports its time on the sample and
    the time the whole workload would take at that rate."""
    import numpy as np
    from threadpoolctl import threadpool_limits

    import oracle
    threads = len(os.sched_getaffinity(0))
    h4 = wl.host["gemm_epilogue_8192x8192x4096"]
    m, k = h4["a"].shape
    n = h4["b"].shape[1]
    blk = wl.blk
    p64 = {k_: v.float().cpu().numpy().astype(np.float64) for k_, v in blk.p.items()}
    x64 = wl.host["block_32x512x1024"]["x"].f64()
    out = {"threads": threads}
    with threadpool_limits(limits=threads, user_api="blas"):
        a = h4["a"].rows(slice(0, gemm_rows)).f64()
        b = h4["b"].f64()
        t0 = time.perf_counter()
        a @ b
        dt = time.perf_counter() - t0
        flop = 2.0 * gemm_rows * k * n
        out["gemm_f64"] = {"shape": [m, k, n], "rows_sampled": gemm_rows, "s": round(dt, 3),
                           "GFLOP/s": round(flop / dt / 1e9, 1),
                           "full_s_at_this_rate": round(dt * m / gemm_rows, 2)}
        t0 = time.perf_counter()
        oracle.block_forward(x64[:block_seqs], p64, blk.heads, blk.eps)
        dt = time.perf_counter() - t0
        out["block_forward_f64"] = {"sequences_sampled": block_seqs, "s": round(dt, 3),
                                    "s_per_sequence": round(dt / block_seqs, 3),
                                    "full_s_at_this_rate": round(dt * x64.shape[0] / block_seqs, 2)}
    return out


def load_traffic():
    try:
        with open(TRAFFIC_FILE) as f:
            return json.load(f)
    except (OSError, ValueError):
        return {}


# widths of the long-row table: the 16-wave register rungs (16392, 32768), the
# row cache (49152, 65536), the row cache with a streamed tail (98304 and up);
# 50257 columns are not a whole number of 16-byte vectors (element-wise loads)
LONG_ROW_WIDTHS = (16392, 32768, 49152, 50257, 65536, 98304, 131072, 262144)
# (name, dtype, bytes per element of one launch): compulsory reads + writes
LONG_ROW_CASES = (
    ("softmax bf16 + bf16 mask", "bf16", 6),
    ("softmax bf16 + byte mask", "bf16", 5),
    ("softmax bf16", "bf16", 4),
    ("softmax fp32", "f32", 8),
    ("LayerNorm + residual bf16", "bf16", 8),
    ("RMSNorm + residual bf16", "bf16", 8),
    ("LayerNorm + residual fp32", "f32", 16),
)


def long_rows(reps: int = 9) -> None:
    """Median launch time of each long-row case: 256 MiB per bf16 input
    (128 MiB of rows for fp32), a 512 MiB scrub between launches so that every
    launch reads HBM, one event pair per launch."""
    import torch
    import paper_2609_30059_amd as fs
    torch.cuda.set_device(0)
    dev = "cuda"
    scrub = torch.empty(512 << 20, dtype=torch.uint8, device=dev)
    g = torch.Generator(device=dev)
    results = {}
    for cols in LONG_ROW_WIDTHS:
        for name, dt, bpe in LONG_ROW_CASES:
            tdt = torch.bfloat16 if dt == "bf16" else torch.float32
            rows = (128 << 20) // cols if dt == "bf16" else (32 << 20) // cols
            g.manual_seed(cols)
            x = (torch.randn(rows, cols, device=dev, generator=g) * 3).to(tdt)
            y = torch.empty_like(x)
            if name.startswith("softmax"):
                m = None
                if "bf16 mask" in name:
                    m = torch.where(torch.rand(rows, cols, device=dev, generator=g) < 0.1,
                                    float("-inf"), 0.0).to(tdt)
                elif "byte mask" in name:
                    m = (torch.rand(rows, cols, device=dev, generator=g) < 0.1).to(torch.uint8)
                fn = lambda: fs.row_softmax(x, m, 0.125, out=y)
            else:
                r = torch.randn(rows, cols, device=dev, generator=g).to(tdt)
                ro = torch.empty_like(x)
                gam = (torch.randn(cols, device=dev, generator=g) * 0.1 + 1).to(tdt)
                bet = (torch.randn(cols, device=dev, generator=g) * 0.1).to(tdt)
                if name.startswith("RMS"):
                    fn = lambda: fs.rmsnorm_residual(x, r, gam, 1e-5, out=y, residual_out=ro)
                else:
                    fn = lambda: fs.layernorm_residual(x, r, gam, bet, 1e-5, out=y,
                                                       residual_out=ro)
            fn()
            torch.cuda.synchronize()
            ts = []
            for i in range(reps):
                scrub.fill_(i & 0xFF)
                e0 = TimingEvent()
                e1 = TimingEvent()
                e0.record()
                fn()
                e1.record()
                torch.cuda.synchronize()
                ts.append(e0.elapsed_time(e1) * 1e3)
            us = sorted(ts)[reps // 2]
            results[(cols, name)] = (us, bpe * x.numel() / us / 1e3)
            print(f"  {cols:>6} {name:<28} {us:8.1f} us {results[(cols, name)][1]:6.0f} GB/s",
                  file=sys.stderr, flush=True)
            del x, y
    names = [c[0] for c in LONG_ROW_CASES]
    print("| columns | " + " | ".join(names) + " |")
    print("|---" * (len(names) + 1) + "|")
    for cols in LONG_ROW_WIDTHS:
        cells = [f"{results[(cols, n)][1]:.0f}" for n in names]
        print(f"| {cols} | " + " | ".join(cells) + " |")


# widths of the odd-row table: rows that are not whole 16-byte vectors, whose
# operands share one 16-byte phase per row (contiguous tensors), so each row's
# aligned body is read 16 bytes at a time
ODD_ROW_WIDTHS = (1001, 4095, 16383)
ODD_ROW_CASES = (
    ("softmax bf16 + bf16 mask", 6),
    ("softmax bf16 + byte mask", 5),
    ("LayerNorm + residual bf16", 8),
    ("bias + GELU bf16", 4),
    ("GEMM epilogue bf16 (sigmoid, row sum)", 2),
    ("row sum bf16", 2),
)


def program_costs(reps: int = 11) -> None:
    """Median event interval of pointwise programs of growing arithmetic on
    bf16 [16384, 4096] against the fixed chain (and on rows of 4095 columns),
    of the GEMM epilogue's reductions, and of the row reductions on
    bf16 [16384, 4096] and fp32 [8192, 4096]; every launch follows a
    read-only pass over 1 GiB."""
    import torch
    import paper_2609_30059_amd as fs
    torch.cuda.set_device(0)
    g = torch.Generator(device="cuda").manual_seed(7)
    x = (0.5 * torch.randn(16384, 4096, device="cuda", generator=g)).to(torch.bfloat16)
    b = (0.02 * torch.randn(4096, device="cuda", generator=g)).to(torch.bfloat16)
    y = torch.empty_like(x)
    scrub = torch.zeros(8192, 65536, dtype=torch.bfloat16, device="cuda")
    sink = torch.empty(8192, dtype=torch.float32, device="cuda")
    prog = lambda ops, **kw: (lambda: fs.pointwise_program(x, ops, out=y, **kw))   # noqa: E731
    cases = [
        ("fixed chain: none", 4, lambda: fs.pointwise_chain(x, None, None, 1.0, "none", out=y)),
        ("fixed chain: bias + GELU", 4, lambda: fs.pointwise_chain(x, b, None, 1.0, "gelu_erf",
                                                                   out=y)),
        ("program: (empty, a copy)", 4, prog([])),
        ("program: scale", 4, prog([("scale", 0.5)])),
        ("program: GELU", 4, prog([("gelu_erf",)])),
        ("program: bias, GELU", 4, prog([("add_bias",), ("gelu_erf",)], bias=b)),
        ("program: bias, scale, GELU", 4, prog([("add_bias",), ("scale", 0.5), ("gelu_erf",)],
                                               bias=b)),
        ("program: bias, scale, clamp, GELU", 4,
         prog([("add_bias",), ("scale", 0.5), ("clamp", -1.0, 1.0), ("gelu_erf",)], bias=b)),
        ("program: 8 x scale", 4, prog([("scale", 1.0)] * 8)),
        ("program: GELU, GELU", 4, prog([("gelu_erf",), ("gelu_erf",)])),
    ]
    # rows of 4095 columns (not whole 16-byte vectors): the aligned-body path
    # where x and y start each row at one phase, the element-wise path where
    # y sits one element further (bytes per element scaled to [16384, 4095])
    xo = x[:, :4095].contiguous()
    yo = torch.empty_like(xo)
    ye = torch.empty(xo.numel() + 1, dtype=xo.dtype, device="cuda")[1:].view(xo.shape)
    odd = 4 * 4095 / 4096
    bg = [("add_bias",), ("gelu_erf",)]
    cases += [
        ("fixed chain: bias + GELU, [16384, 4095]", odd,
         lambda: fs.pointwise_chain(xo, b[:4095], None, 1.0, "gelu_erf", out=yo)),
        ("program: (empty), [16384, 4095]", odd, lambda: fs.pointwise_program(xo, [], out=yo)),
        ("program: (empty), [16384, 4095], y at another phase (element-wise)", odd,
         lambda: fs.pointwise_program(xo, [], out=ye)),
        ("program: bias, scale, [16384, 4095]", odd,
         lambda: fs.pointwise_program(xo, [("add_bias",), ("scale", 0.5)], bias=b[:4095],
                                      out=yo)),
        ("program: bias, scale, [16384, 4095], y at another phase (element-wise)", odd,
         lambda: fs.pointwise_program(xo, [("add_bias",), ("scale", 0.5)], bias=b[:4095],
                                      out=ye)),
        ("program: bias, GELU, [16384, 4095]", odd,
         lambda: fs.pointwise_program(xo, bg, bias=b[:4095], out=yo)),
        ("program: bias, GELU, [16384, 4095], y at another phase (element-wise)", odd,
         lambda: fs.pointwise_program(xo, bg, bias=b[:4095], out=ye)),
        ("program: bias, scale, clamp, GELU, [16384, 4095]", odd,
         lambda: fs.pointwise_program(xo, [("add_bias",), ("scale", 0.5), ("clamp", -1.0, 1.0),
                                           ("gelu_erf",)], bias=b[:4095], out=yo)),
    ]
    xf = (2 * torch.randn(8192, 4096, device="cuda", generator=g))
    o = torch.empty(16384, device="cuda")
    # the GEMM epilogue with each reduction on a bf16 C [8192, 8192] (the sum
    # and mean in one kernel family, max and log-sum-exp in another)
    ce = (0.0256 * torch.randn(8192, 8192, device="cuda", generator=g)).to(torch.bfloat16)
    be = (torch.rand(8192, device="cuda", generator=g) - 0.5).to(torch.bfloat16)
    se = torch.rand(8192, device="cuda", generator=g) + 0.5
    for red in ("sum", "max", "logsumexp"):
        cases.append((f"epilogue sigmoid {red}, bf16 C [8192, 8192]", -1,
                      (lambda red=red: fs.gemm_epilogue_reduce(ce, be, se, "sigmoid", red,
                                                               out=o[:8192]))))
    for name, t in (("bf16 [16384, 4096]", x), ("fp32 [8192, 4096]", xf)):
        for op in ("sum", "max", "logsumexp"):
            cases.append((f"row {op}, {name}", 0,
                          (lambda t=t, op=op: fs.row_reduce(t, op, out=o[:t.shape[0]]))))
    times = {n: [] for n, _, _ in cases}
    for rep in range(reps + 1):            # the first repetition is a warm-up
        for name, _, fn in cases:
            fs.row_reduce(scrub, "sum", out=sink)
            e0, e1 = TimingEvent(), TimingEvent()
            e0.record()
            fn()
            e1.record()
            torch.cuda.synchronize()
            if rep:
                times[name].append(e0.elapsed_time(e1) * 1e3)
    print("| case | us (events) | GB/s | % of 8 TB/s |")
    print("|---|---|---|---|")
    for name, bpe, _ in cases:
        us = sorted(times[name])[reps // 2]
        nbytes = (x.numel() * bpe if bpe > 0 else ce.numel() * 2 if bpe < 0 else
                  (x.numel() * 2 if "bf16" in name else xf.numel() * 4))
        gbs = nbytes / us / 1e3
        print(f"| {name} | {us:.2f} | {gbs:.0f} | {100 * gbs / PEAK_HBM_GBS:.1f} |")


def odd_rows(reps: int = 9) -> None:
    """Median launch time of each odd-row case: 64 MiB per bf16 input, a
    512 MiB scrub between launches, one event pair per launch."""
    import torch
    import paper_2609_30059_amd as fs
    torch.cuda.set_device(0)
    dev = "cuda"
    scrub = torch.empty(512 << 20, dtype=torch.uint8, device=dev)
    g = torch.Generator(device=dev)
    results = {}
    for cols in ODD_ROW_WIDTHS:
        rows = (32 << 20) // cols
        g.manual_seed(cols)
        rn = lambda *sh: torch.randn(*sh, device=dev, generator=g)
        x = (rn(rows, cols) * 3).to(torch.bfloat16)
        y = torch.empty_like(x)
        for name, bpe in ODD_ROW_CASES:
            if name.startswith("softmax"):
                masked = torch.rand(rows, cols, device=dev, generator=g) < 0.1
                if "byte mask" in name:
                    m = masked.to(torch.uint8)
                else:
                    m = torch.where(masked, float("-inf"), 0.0).to(torch.bfloat16)
                fn = lambda: fs.row_softmax(x, m, 0.125, out=y)
            elif name.startswith("LayerNorm"):
                r = rn(rows, cols).to(torch.bfloat16)
                ro = torch.empty_like(x)
                gam = (rn(cols) * 0.1 + 1).to(torch.bfloat16)
                bet = (rn(cols) * 0.1).to(torch.bfloat16)
                fn = lambda: fs.layernorm_residual(x, r, gam, bet, 1e-5, out=y, residual_out=ro)
            elif name.startswith("bias"):
                b = (rn(cols) * 0.02).to(torch.bfloat16)
                fn = lambda: fs.pointwise_chain(x, b, None, 1.0, "gelu_erf", out=y)
            elif name.startswith("GEMM"):
                b = (torch.rand(cols, device=dev, generator=g) - 0.5).to(torch.bfloat16)
                sc = torch.rand(cols, device=dev, generator=g) + 0.5
                o = torch.empty(rows, dtype=torch.float32, device=dev)
                fn = lambda: fs.gemm_epilogue_reduce(x, b, sc, "sigmoid", "sum", out=o)
            else:
                o = torch.empty(rows, dtype=torch.float32, device=dev)
                fn = lambda: fs.row_reduce(x, "sum", out=o)
            fn()
            torch.cuda.synchronize()
            ts = []
            for i in range(reps):
                scrub.fill_(i & 0xFF)
                e0 = TimingEvent()
                e1 = TimingEvent()
                e0.record()
                fn()
                e1.record()
                torch.cuda.synchronize()
                ts.append(e0.elapsed_time(e1) * 1e3)
            us = sorted(ts)[reps // 2]
            results[(cols, name)] = (us, bpe * x.numel() / us / 1e3)
            print(f"  {cols:>6} {name:<40} {us:8.1f} us {results[(cols, name)][1]:6.0f} GB/s",
                  file=sys.stderr, flush=True)
    names = [c[0] for c in ODD_ROW_CASES]
    print("| columns | " + " | ".join(names) + " |")
    print("|---" * (len(names) + 1) + "|")
    for cols in ODD_ROW_WIDTHS:
        cells = [f"{results[(cols, n)][1]:.0f}" for n in names]
        print(f"| {cols} | " + " | ".join(cells) + " |")


def short_kernel_name(name: str) -> str:
    """A library kernel's name without the namespace, return type and
    parameter list (its template arguments kept)."""
    n = name.replace("(anonymous namespace)::", "").replace("void ", "").replace("fs::", "")
    depth = 0
    for i, ch in enumerate(n):
        if ch == "<":
            depth += 1
        elif ch == ">":
            depth -= 1
        elif ch == "(" and depth == 0:
            return n[:i]
    return n


def report_counters(paths) -> None:
    """Per-launch averages of the LDS and occupancy counters of the library's
    kernels, from one or more rocprofv3 --pmc counter-collection CSVs (one
    per counter pass); launches are grouped by kernel, grid and workgroup."""
    import csv
    acc = {}
    meta = {}
    for path in paths:
        with open(path, newline="") as f:
            for r in csv.DictReader(f):
                if "fs::" not in r["Kernel_Name"]:
                    continue
                key = (short_kernel_name(r["Kernel_Name"]), int(r["Grid_Size"]),
                       int(r["Workgroup_Size"]))
                meta[key] = (int(r["VGPR_Count"]) + int(r.get("Accum_VGPR_Count") or 0),
                             int(r["LDS_Block_Size"]))
                d = acc.setdefault(key, {}).setdefault(r["Counter_Name"], {})
                d[r["Dispatch_Id"]] = float(r["Counter_Value"])
    avg = {k: {c: sum(v.values()) / len(v) for c, v in cs.items()} for k, cs in acc.items()}
    cols = ("OccupancyPercent", "SQ_INSTS_LDS", "SQ_LDS_IDX_ACTIVE", "SQ_LDS_BANK_CONFLICT",
            "SQ_LDS_ADDR_CONFLICT", "LDSBankConflict")
    print("| kernel | grid x wg | VGPRs | static LDS B | waves/CU (occupancy) | LDS instr | "
          "LDS active cyc | bank-conflict cyc | conflict / active | addr-conflict cyc | "
          "LDSBankConflict % |")
    print("|---|---|---|---|---|---|---|---|---|---|---|")

    def f(v, fmt):
        return "--" if v is None else format(v, fmt)
    for key in sorted(avg, key=lambda k: (k[0], k[1])):
        a = avg[key]
        occ, ins, act, bank, addr, pct = (a.get(c) for c in cols)
        ratio = bank / act if bank is not None and act else None
        waves = None if occ is None else occ * 32 / 100
        print(f"| `{key[0]}` | {key[1] // key[2]} x {key[2]} | {meta[key][0]} | {meta[key][1]} | "
              f"{f(waves, '.1f')} ({f(occ, '.0f')} %) | {f(ins, '.0f')} | {f(act, '.0f')} | "
              f"{f(bank, '.0f')} | {f(ratio, '.4f')} | {f(addr, '.0f')} | {f(pct, '.3f')} |")


# --epilogue-context: the GEMM epilogue (a read-only stream with a sigmoid per
# element) launched in four contexts, each a warm-up of 3 and then CONTEXT_REPS
# repetitions, every block of launches separated by a pause
CONTEXT_STEPS, CONTEXT_STEP_TAIL, CONTEXT_REPS = 100, 60, 20
# (label, measured kernel, launches after the 3 warm-up ones)
CONTEXTS = (("inside full bench steps", "ep", CONTEXT_STEPS),
            ("a plain row sum over the same C in its place in full bench steps", "rowsum",
             CONTEXT_STEPS),
            ("right after the [16384, 4096] LayerNorm", "ep", CONTEXT_REPS),
            ("after a read-only 1 GiB pass", "ep", CONTEXT_REPS),
            ("back to back", "ep", CONTEXT_REPS))
CONTEXT_PAUSE_S = 0.3
CONTEXT_PATTERNS = {"ep": KERNEL_PATTERNS["ep_8192x8192"],
                    "rowsum": r"reduce_kernel<unsigned short,"}
CONTEXT_BYTES = {"ep": STEP_BYTES["ep_8192x8192"], "rowsum": 8192 * 8192 * 2 + 8192 * 4}


def epilogue_context(seed: int = 0) -> None:
    """The GEMM epilogue on the bench's C in the contexts of CONTEXTS, each
    block of launches after a pause (run under a kernel trace).  The second
    context runs the bench step with a plain row sum over the same C (the
    read-only floor of those bytes) where the epilogue would be."""
    import torch
    import paper_2609_30059_amd as fs
    torch.cuda.set_device(0)
    wl = Workload(seed)
    k = {name: fn for name, _, _, fn in wl.kernels}
    scrub = torch.zeros(8192, 65536, dtype=torch.bfloat16, device="cuda")     # 1 GiB
    sink = torch.empty(8192, dtype=torch.float32, device="cuda")
    ep = k["ep_8192x8192"]
    c = wl.ep["c"]

    def step_with_rowsum():
        for name, _, _, fn in wl.kernels:
            if name == "ep_8192x8192":
                fs.row_reduce(c, "sum", out=sink)
            else:
                fn()

    fns = (wl.step, step_with_rowsum, lambda: (k["ln_16384x4096"](), ep()),
           lambda: (fs.row_reduce(scrub, "sum", out=sink), ep()), ep)
    for fn, (_, _, reps) in zip(fns, CONTEXTS):
        for n in (3, reps):
            torch.cuda.synchronize()
            time.sleep(CONTEXT_PAUSE_S)
            for _ in range(n):
                fn()
    torch.cuda.synchronize()
    time.sleep(CONTEXT_PAUSE_S)


def report_context(trace_csv: str) -> None:
    """Median dispatch time of each context's kernel in --epilogue-context:
    the trace is split at pauses (gaps above half the pause); the last
    2 x len(CONTEXTS) blocks are the warm-up and timed blocks of each
    context, in order.  Step contexts report their last CONTEXT_STEP_TAIL
    launches (the first milliseconds of load after a pause run at a lower
    engine clock)."""
    import csv
    import re
    rows = []
    with open(trace_csv, newline="") as f:
        for r in csv.DictReader(f):
            rows.append((int(r["Start_Timestamp"]), int(r["End_Timestamp"]),
                         r["Kernel_Name"].replace("(anonymous namespace)::", "")))
    rows.sort()
    blocks, cur, last = [], [], None
    for s, e, n in rows:
        if last is not None and s - last > CONTEXT_PAUSE_S * 0.5e9:
            blocks.append(cur)
            cur = []
        cur.append((s, e, n))
        last = e
    blocks.append(cur)
    need = 2 * len(CONTEXTS)
    if len(blocks) < need:
        raise ValueError(f"{len(blocks)} blocks in the trace, expected at least {need}")
    timed = blocks[-need:][1::2]
    print("| context | kernel | launches | median us | q1 us | q3 us | min us | max us | "
          "% of 8 TB/s (median) |")
    print("|---|---|---|---|---|---|---|---|---|")
    for (name, kind, reps), b in zip(CONTEXTS, timed):
        v = [(e - s) / 1e3 for s, e, n in b if re.search(CONTEXT_PATTERNS[kind], n)]
        if reps == CONTEXT_STEPS:
            v = v[-CONTEXT_STEP_TAIL:]
        v = sorted(v)
        med = v[len(v) // 2]
        label = "epilogue" if kind == "ep" else "row sum"
        print(f"| {name} | {label} | {len(v)} | {med:.2f} | {v[len(v) // 4]:.2f} | "
              f"{v[3 * len(v) // 4]:.2f} | {v[0]:.2f} | {v[-1]:.2f} | "
              f"{100 * CONTEXT_BYTES[kind] / med / 1e3 / PEAK_HBM_GBS:.1f} |")


# --copy-floor: each short block sub-kernel next to the calibration copy moving
# the same number of bytes (half read, half written), in this order every
# repetition, each launch after a read-only pass over 1 GiB (HBM-cold inputs
# and no dirty lines left in the Infinity Cache, as in the bench step)
FLOOR_CASES = (("copy_64MiB", 64 << 20), ("blk_ln1", None), ("copy_96MiB", 96 << 20),
               ("blk_res", None), ("copy_128MiB", 128 << 20), ("blk_ln2", None))
FLOOR_REPS = 15


def copy_floor(reps: int = FLOOR_REPS) -> None:
    import torch
    import paper_2609_30059_amd as fs
    torch.cuda.set_device(0)
    dev = "cuda"
    g = torch.Generator(device=dev)
    g.manual_seed(0)
    T, H = 16384, 1024
    bf = torch.bfloat16
    rn = lambda *sh: torch.randn(*sh, device=dev, generator=g).to(bf)
    x, r, att = rn(T, H), rn(T, H), rn(T, H)
    gam, bet = (rn(H) * 0.1 + 1).to(bf), (rn(H) * 0.1).to(bf)
    a, m, h1, out = (torch.empty(T, H, dtype=bf, device=dev) for _ in range(4))
    span = 1 << 30
    src = torch.empty(span, dtype=torch.uint8, device=dev)
    dst = torch.empty(span, dtype=torch.uint8, device=dev)
    scrub = torch.zeros(8192, 65536, dtype=bf, device=dev)          # 1 GiB, read only
    sink = torch.empty(8192, dtype=torch.float32, device=dev)
    offs = {}

    def copy(nbytes):
        half = nbytes // 2
        def fn():
            o = offs.get(nbytes, 0)
            o = 0 if o + half > span else o
            fs.copy_(dst[o:o + half], src[o:o + half])
            offs[nbytes] = o + half
        return fn
    kern = {
        "blk_ln1": lambda: fs.layernorm_residual(x, None, gam, bet, 1e-5, out=a),
        "blk_res": lambda: fs.pointwise_chain(x, None, r, 1.0, "none", out=out),
        "blk_ln2": lambda: fs.layernorm_residual(att, x, gam, bet, 1e-5, out=m, residual_out=h1),
    }
    cases = [(name, copy(nb) if nb else kern[name]) for name, nb in FLOOR_CASES]
    times = {name: [] for name, _ in cases}
    for rep in range(reps + 1):            # the first repetition is a warm-up
        for name, fn in cases:
            fs.row_reduce(scrub, "sum", out=sink)
            e0, e1 = TimingEvent(), TimingEvent()
            e0.record()
            fn()
            e1.record()
            torch.cuda.synchronize()
            if rep:
                times[name].append(e0.elapsed_time(e1) * 1e3)
    print("| case | median us (events) | min us |")
    print("|---|---|---|")
    for name, _ in cases:
        ts = sorted(times[name])
        print(f"| {name} | {ts[len(ts) // 2]:.2f} | {ts[0]:.2f} |")


def floor_bytes(label: str) -> int:
    for name, nb in FLOOR_CASES:
        if name == label and nb:
            return nb
    return STEP_BYTES[label]


def report_floor(trace_csv: str) -> None:
    """Median dispatch duration of every --copy-floor case from a rocprofv3
    kernel-trace CSV: the copies and kernels are told apart by their fixed
    order within each repetition (the read-only passes between them are
    skipped, the warm-up repetition dropped)."""
    import csv
    import re
    labels = [name for name, _ in FLOOR_CASES]
    pats = [r"copy128_kernel" if nb else KERNEL_PATTERNS[name] for name, nb in FLOOR_CASES]
    seq = []
    with open(trace_csv, newline="") as f:
        for row in csv.DictReader(f):
            n = row["Kernel_Name"].replace("(anonymous namespace)::", "")
            if any(re.search(p, n) for p in pats):
                seq.append((n, (int(row["End_Timestamp"]) - int(row["Start_Timestamp"])) / 1e3))
    per = len(labels)
    if len(seq) % per:
        raise ValueError(f"{len(seq)} matching dispatches is not a multiple of {per}")
    got = {l: [] for l in labels}
    for i, (n, us) in enumerate(seq):
        label, pat = labels[i % per], pats[i % per]
        if not re.search(pat, n):
            raise ValueError(f"dispatch {i}: expected {label}, got {n}")
        if i >= per:
            got[label].append(us)
    med = {l: sorted(v)[len(v) // 2] for l, v in got.items()}
    print("| case | dispatches | median us | min us | bytes | GB/s | % of 8 TB/s | vs same-size copy |")
    print("|---|---|---|---|---|---|---|---|")
    copy_of = {}
    for i, (name, nb) in enumerate(FLOOR_CASES):
        if nb:
            copy_of[FLOOR_CASES[i + 1][0]] = name
    for name, nb in FLOOR_CASES:
        b = floor_bytes(name)
        gbs = b / med[name] / 1e3
        ratio = f"{med[name] / med[copy_of[name]]:.3f}" if name in copy_of else "--"
        print(f"| {name} | {len(got[name])} | {med[name]:.2f} | {min(got[name]):.2f} | {b} | "
              f"{gbs:.0f} | {100 * gbs / PEAK_HBM_GBS:.1f} | {ratio} |")



# --access-floors: every sub-kernel of the step next to its access-shape floor
# (libaccessfloor.so: a kernel moving the same bytes in the same launch shape
# with none of the arithmetic), alternating, each launch after a read-only
# pass over 1 GiB, in this order every repetition
FLOOR_SHAPES = ("pw_256x1024", "pw_262144x1024", "sm_8192x4096", "ln_16384x4096",
                "ep_8192x8192", "blk_ln1", "blk_sm", "blk_ln2", "blk_gelu", "blk_res")
ACCESS_FLOOR_REPS = 10


def access_floor_operands(wl):
    """(in0, in1, out0, out1) of each step launch, in fsx_access_floor's shape
    order: the floor reads the sub-kernel's own inputs and writes its outputs."""
    T, H = wl.bx.shape[0] * wl.bx.shape[1], wl.bx.shape[2]
    x2, buf = wl.bx.view(T, H), wl.buf
    return {
        "pw_256x1024": (wl.pw["x"], wl.pw["r"], wl.pw["y"], None),
        "pw_262144x1024": (wl.pwbw["x"], wl.pwbw["r"], wl.pwbw["y"], None),
        "sm_8192x4096": (wl.sm["x"], wl.sm["m"], wl.sm["y"], None),
        "ln_16384x4096": (wl.ln["x"], wl.ln["r"], wl.ln["y"], wl.ln["ro"]),
        "ep_8192x8192": (wl.ep["c"], None, wl.ep["out"], None),
        "blk_ln1": (x2, None, buf["a"], None),
        "blk_sm": (buf["scores"], None, buf["probs"], None),
        "blk_ln2": (buf["att"], x2, buf["m"], buf["h1"]),
        "blk_gelu": (buf["u"], None, buf["g"], None),
        "blk_res": (buf["d"], buf["h1"], buf["out"], None),
    }


def floor_launchers(wl):
    """{step launch name: closure launching its access-shape floor on the
    current stream} from libaccessfloor.so, or None when it is not built.
    The floors read the sub-kernels' inputs and overwrite their outputs."""
    import ctypes
    import torch
    from paper_2609_30059_amd import build as B
    if not os.path.exists(B.LIB_ACCESS_FLOOR):
        return None
    lib = ctypes.CDLL(B.LIB_ACCESS_FLOOR)
    sz = ctypes.c_size_t
    lib.fsx_access_floor.argtypes = [ctypes.c_int, ctypes.c_void_p, sz, ctypes.c_void_p, sz,
                                     ctypes.c_void_p, sz, ctypes.c_void_p, sz, ctypes.c_int,
                                     ctypes.c_void_p]
    lib.fsx_access_floor.restype = ctypes.c_int
    lib.fsx_access_floor_shapes.restype = ctypes.c_int
    if lib.fsx_access_floor_shapes() != len(FLOOR_SHAPES):
        raise RuntimeError("libaccessfloor.so does not match bench.py's shape list")
    cus = torch.cuda.get_device_properties(torch.cuda.current_device()).multi_processor_count
    ops = access_floor_operands(wl)

    def floor(shape):
        args = []
        for t in ops[FLOOR_SHAPES[shape]]:
            args += [None, 0] if t is None else [t.data_ptr(), t.numel() * t.element_size()]
        def fn():
            rc = lib.fsx_access_floor(shape, *args, cus, torch.cuda.current_stream().cuda_stream)
            if rc != 0:
                raise RuntimeError(f"fsx_access_floor({FLOOR_SHAPES[shape]}) returned {rc}")
        return fn
    return {name: floor(i) for i, name in enumerate(FLOOR_SHAPES)}


def access_floors(seed: int = 0, reps: int = ACCESS_FLOOR_REPS) -> None:
    """Prints the median event interval of every step sub-kernel and of its
    floor; run under a kernel trace for dispatch durations (--report-floors)."""
    import torch
    from paper_2609_30059_amd import build as B
    import paper_2609_30059_amd as fs
    torch.cuda.set_device(0)
    wl = Workload(seed)
    floors = floor_launchers(wl)
    if floors is None:
        raise RuntimeError(f"{B.LIB_ACCESS_FLOOR} is not built (python -m paper_2609_30059_amd.build)")
    real = {name: fn for name, _, _, fn in wl.kernels}
    real["pw_262144x1024"] = lambda: fs.pointwise_chain(
        wl.pwbw["x"], wl.pw["b"], wl.pwbw["r"], wl.pw["s"], "gelu_erf", out=wl.pwbw["y"])

    scrub = torch.zeros(8192, 65536, dtype=torch.bfloat16, device="cuda")   # 1 GiB, read only
    sink = torch.empty(8192, dtype=torch.float32, device="cuda")
    cases = []
    for name in FLOOR_SHAPES:
        cases += [(name, "kernel", real[name]), (name, "floor", floors[name])]
    times = {(n, k): [] for n, k, _ in cases}
    for rep in range(reps + 1):            # the first repetition is a warm-up
        for name, kind, fn in cases:
            fs.row_reduce(scrub, "sum", out=sink)
            e0, e1 = TimingEvent(), TimingEvent()
            e0.record()
            fn()
            e1.record()
            torch.cuda.synchronize()
            if rep:
                times[(name, kind)].append(e0.elapsed_time(e1) * 1e3)
    print("| kernel | kernel us (events) | floor us (events) | kernel / floor |")
    print("|---|---|---|---|")
    for name in FLOOR_SHAPES:
        k, f = (sorted(times[(name, c)])[reps // 2] for c in ("kernel", "floor"))
        print(f"| {name} | {k:.2f} | {f:.2f} | {k / f:.3f} |")


def report_floors(trace_csv: str) -> None:
    """Median dispatch durations of every --access-floors case from a rocprofv3
    kernel-trace CSV.  Each repetition launches, per step kernel, a read-only
    pass, the kernel, a read-only pass and its floor; the read-only passes
    are dropped and the rest assigned in that fixed order (the warm-up
    repetition dropped).  The sub-kernels must match their kernel-name
    patterns and the floors floor_rows_kernel."""
    import csv
    import re
    seq = []
    with open(trace_csv, newline="") as f:
        for row in csv.DictReader(f):
            n = row["Kernel_Name"].replace("(anonymous namespace)::", "")
            seq.append((int(row["Start_Timestamp"]), n,
                        (int(row["End_Timestamp"]) - int(row["Start_Timestamp"])) / 1e3))
    seq.sort()
    # the measured launches begin after the Workload setup: from the first
    # floor dispatch back to the kernel launched right before it
    first = next(i for i, (_, n, _) in enumerate(seq) if "floor_rows_kernel" in n)
    pats = [KERNEL_PATTERNS[n] for n in FLOOR_SHAPES] + [r"floor_rows_kernel"]
    body = [(n, us) for _, n, us in seq[first - 2:] if any(re.search(p, n) for p in pats)]
    per = 2 * len(FLOOR_SHAPES)
    if len(body) % per:
        raise ValueError(f"{len(body)} measured dispatches is not a multiple of {per}")
    got = {}
    for i, (n, us) in enumerate(body):
        name, kind = FLOOR_SHAPES[(i % per) // 2], ("kernel", "floor")[i % 2]
        pat = KERNEL_PATTERNS[name] if kind == "kernel" else r"floor_rows_kernel"
        if not re.search(pat, n):
            raise ValueError(f"dispatch {i}: expected the {kind} of {name}, got {n[:120]}")
        if i >= per:
            got.setdefault((name, kind), []).append(us)
    print("| kernel | compulsory bytes | kernel us | floor us | kernel / floor | kernel % of 8 TB/s "
          "| floor % of 8 TB/s |")
    print("|---|---|---|---|---|---|---|")
    for name in FLOOR_SHAPES:
        k, f = (sorted(got[(name, c)])[len(got[(name, c)]) // 2] for c in ("kernel", "floor"))
        b = STEP_BYTES[name]
        print(f"| {name} | {b} | {k:.2f} | {f:.2f} | {k / f:.3f} | "
              f"{100 * b / k / 1e3 / PEAK_HBM_GBS:.1f} | {100 * b / f / 1e3 / PEAK_HBM_GBS:.1f} |")


# ---------------------------------------------------------------------------
# clock transient: the step after an idle pause, with an engine-clock reading
# after every step
# ---------------------------------------------------------------------------
TRANSIENT_STEPS = 160
TRANSIENT_PAUSE_S = 0.5
TRANSIENT_PROBE_ITERS = 60     # about 7 us of FMAs per SIMD per probe


def clock_transient(steps: int = TRANSIENT_STEPS) -> None:
    """After an idle pause, ``steps`` bench steps back to back, each followed
    by the engine-clock probe (libclockprobe.so); run under a kernel trace.
    Prints one line per step, ``clock step S MHZ MHz``."""
    import ctypes
    import torch
    from paper_2609_30059_amd import build as B
    if not os.path.exists(B.LIB_CLOCK_PROBE):
        raise RuntimeError(f"{B.LIB_CLOCK_PROBE} is not built (python -m paper_2609_30059_amd.build)")
    lib = ctypes.CDLL(B.LIB_CLOCK_PROBE)
    lib.fsx_clock_probe.argtypes = [ctypes.c_void_p, ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                    ctypes.c_int, ctypes.c_void_p]
    torch.cuda.set_device(0)
    wl = Workload(0)
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    buf = torch.zeros(2 * steps, dtype=torch.int64, device="cuda")
    for _ in range(3):
        wl.step()
    torch.cuda.synchronize()
    time.sleep(TRANSIENT_PAUSE_S)
    stream = torch.cuda.current_stream().cuda_stream
    for st in range(steps):
        wl.step()
        rc = lib.fsx_clock_probe(buf.data_ptr(), st, steps, cus * 4, TRANSIENT_PROBE_ITERS, stream)
        if rc != 0:
            raise RuntimeError(f"fsx_clock_probe failed ({rc})")
    torch.cuda.synchronize()
    v = buf.cpu().tolist()
    for st in range(steps):
        mhz = v[2 * st] / (v[2 * st + 1] / 100.0) if v[2 * st + 1] else 0.0
        print(f"clock step {st} {mhz:.0f} MHz", flush=True)


def transient_table(trace_csv: str, log: str, every: int = 8):
    """Rows of (step, ms since the first step, MHz, {kernel: us}) from a
    --clock-transient kernel trace and its printed clock lines; the probe
    launch closes each step."""
    import csv
    import re
    clocks = {}
    with open(log) as f:
        for line in f:
            m = re.match(r"clock step (\d+) (\d+) MHz", line)
            if m:
                clocks[int(m.group(1))] = int(m.group(2))
    with open(trace_csv) as f:
        rows = sorted(csv.DictReader(f), key=lambda r: int(r["Start_Timestamp"]))
    steps, cur, t_first = [], {}, None
    for r in rows:
        name = r["Kernel_Name"]
        if "clock_probe_kernel" in name:
            if cur:
                steps.append(cur)
            cur = {}
            continue
        label = next((k for k, pat in KERNEL_PATTERNS.items()
                      if k in KIND and re.search(re.escape(pat), name)), None)
        if label:
            if label == "pw_256x1024":
                cur["_t"] = int(r["Start_Timestamp"])      # the step's first kernel
            cur[label] = (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3
    steps = [st for st in steps if st][-len(clocks):] if clocks else steps
    out = []
    for i, st in enumerate(steps):
        if t_first is None:
            t_first = st["_t"]
        out.append((i, (st["_t"] - t_first) / 1e6, clocks.get(i, 0),
                    {k: v for k, v in st.items() if k != "_t"}))
    return out


def report_transient(trace_csv: str, log: str) -> None:
    """Markdown: the per-step table (every 8th step) and, per kernel, the
    median duration over the steps whose clock sits below 90 % of the
    sustained clock (median of the last 60 steps) against the last 60 steps."""
    tab = transient_table(trace_csv, log)
    names = [k for k in KIND if k != "pw_262144x1024" and any(k in t[3] for t in tab)]
    print("| step | ms | MHz | " + " | ".join(names) + " |")
    print("|---" * (3 + len(names)) + "|")
    for i, ms, mhz, d in tab[::8]:
        print(f"| {i} | {ms:.1f} | {mhz} | " + " | ".join(f"{d.get(k, 0):.2f}" for k in names) + " |")
    tail = tab[-60:]
    med = lambda v: sorted(v)[len(v) // 2] if v else float("nan")
    steady = med([t[2] for t in tail])
    dip = [t for t in tab if t[2] and t[2] < 0.9 * steady]
    print()
    print(f"sustained clock (median of the last {len(tail)} steps): {steady} MHz; "
          f"{len(dip)} steps below 90 % of it"
          + (f", from {dip[0][1]:.1f} to {dip[-1][1]:.1f} ms, lowest {min(t[2] for t in dip)} MHz"
             if dip else ""))
    print()
    print("| kernel | median us, dip steps | median us, last 60 steps | ratio |")
    print("|---|---|---|---|")
    for k in names:
        a = med([t[3][k] for t in dip if k in t[3]])
        b = med([t[3][k] for t in tail if k in t[3]])
        print(f"| {k} | {a:.2f} | {b:.2f} | {a / b:.3f} |")


def main():
    args = parse()
    if args.program_costs:
        program_costs()
        return
    if args.long_rows:
        long_rows()
        return
    if args.copy_floor:
        copy_floor()
        return
    if args.access_floors:
        access_floors(args.seed)
        return
    if args.report_floors:
        report_floors(args.report_floors)
        return
    if args.clock_transient:
        clock_transient()
        return
    if args.report_transient:
        report_transient(*args.report_transient)
        return
    if args.epilogue_context:
        epilogue_context(args.seed)
        return
    if args.report_context:
        report_context(args.report_context)
        return
    if args.odd_rows:
        odd_rows()
        return
    if args.report_counters:
        report_counters(args.report_counters)
        return
    if args.report_floor:
        report_floor(args.report_floor)
        return
    if args.report_trace:
        report_trace(args.report_trace, args.all_kernels)
        return
    if args.write_traffic:
        out = write_traffic(*args.write_traffic, args.measured_at, *args.commands)
        print(json.dumps(out, indent=1))
        return
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (got --gpus {args.gpus}): every sub-kernel shards "
              f"by rows with no exchange, so each GPU of a larger job runs this same "
              f"single-GPU workload on its rows.", file=sys.stderr)
        sys.exit(2)
    import torch
    torch.cuda.set_device(0)
    t_setup = time.perf_counter()
    wl = Workload(args.seed)
    copy_gbs = wl.copy_calibration()
    setup_s = time.perf_counter() - t_setup

    nk = len(wl.kernels)

    def interval_pass(steps, reduce=lambda v: sum(v) / len(v)):
        """Per-kernel intervals between events recorded after every kernel."""
        evs = [[TimingEvent() for _ in range(nk + 1)]
               for _ in range(steps)]
        for s in range(steps):
            evs[s][0].record()
            wl.step(evs[s])
        torch.cuda.synchronize()
        return [reduce([evs[s][i].elapsed_time(evs[s][i + 1]) for s in range(steps)])
                for i in range(nk)]

    # settle (part of the setup, untimed): steps back to back for at least
    # SETTLE_MS of GPU time.  For the first few milliseconds of load after an
    # idle GPU the engine clock dips well below its sustained value and the
    # kernels with the most issue work per byte slow down with it; the timed
    # steps are to see the sustained state.  The medians of the settle pass's
    # per-kernel intervals pick the dominant kernel.
    settle_ms, settle_steps, settle_per = 0.0, 0, None
    while settle_ms < args.settle_ms:
        n = max(1, min(20, int(args.settle_ms / 0.3)))
        per_s = interval_pass(n, lambda v: sorted(v)[len(v) // 2])
        settle_per = per_s
        settle_ms += sum(per_s) * n
        settle_steps += n
    if settle_per is not None:
        dom = max(range(nk), key=lambda i: settle_per[i])
    else:
        dom = max(range(nk), key=lambda i: wl.kernels[i][2])

    # timed region: exactly K steps, right behind the W warmup steps (no host
    # synchronisation between them, so the GPU does not idle).  Events mark
    # its two ends and bracket the dominant kernel of every step; no other
    # event sits between kernels (a timing-only event still costs the GPU
    # about 1 us, so one after every kernel would inflate the step by about 3 %).
    t_beg = TimingEvent()
    t_end = TimingEvent()
    dev = [(TimingEvent(), TimingEvent())
           for _ in range(args.steps)]
    dom_fn = wl.kernels[dom][3]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.warmup):
        wl.step()
    t_beg.record()
    for s in range(args.steps):
        for i, (_, _, _, fn) in enumerate(wl.kernels):
            if i == dom:
                dev[s][0].record()
                dom_fn()
                dev[s][1].record()
            else:
                fn()
    t_end.record()
    torch.cuda.synchronize()
    wall_s = time.perf_counter() - t0
    step_ms = t_beg.elapsed_time(t_end) / args.steps
    dom_ms = sum(a.elapsed_time(b) for a, b in dev) / args.steps
    value = wl.step_bytes / (step_ms * 1e-3) / 1e9

    # per-kernel breakdown (context, after the timed region): K more steps with
    # an event after every kernel; each interval includes that event's cost
    # medians (do_bench's statistic) and means of the same intervals
    per_all = interval_pass(args.steps, lambda v: v)
    per = [sorted(v)[len(v) // 2] for v in per_all]
    per_mean = [sum(v) / len(v) for v in per_all]
    # the practical ceiling of a kernel that moves as many bytes: a copy of
    # that size, measured the same way
    copies = ([float("nan")] * nk if args.no_copy_reference
              else wl.same_size_copies([k[2] for k in wl.kernels], max(args.steps, 5)))

    bw_ms = wl.pointwise_bandwidth_scale(max(args.steps // 5, 5))
    bw_bytes = STEP_BYTES["pw_262144x1024"]
    sm8_us, sm_add_us = wl.softmax_byte_mask(max(args.steps // 5, 5))
    sm8_bytes = 8192 * 4096 * (2 + 1 + 2)
    prog_us, prog_chain_us, prog_bytes = wl.pointwise_program(max(args.steps // 5, 5))

    # access-shape floors (libaccessfloor.so): K steps of the step's launches
    # each replaced by its floor, timed like the per-kernel pass.  Last of the
    # GPU measurements: the floors overwrite the sub-kernels' outputs.
    floors = floor_launchers(wl)
    floor_med = [None] * nk
    if floors is not None:
        fl_fns = [floors[name] for name, _, _, _ in wl.kernels]
        for f in fl_fns:
            f()
        torch.cuda.synchronize()
        fev = [[TimingEvent() for _ in range(nk + 1)] for _ in range(args.steps)]
        for row in fev:
            row[0].record()
            for i, f in enumerate(fl_fns):
                f()
                row[i + 1].record()
        torch.cuda.synchronize()
        floor_med = [sorted(fev[st][i].elapsed_time(fev[st][i + 1]) for st in range(args.steps))
                     [args.steps // 2] for i in range(nk)]

    traffic = load_traffic()
    per_kernel = {}
    for (name, kind, nbytes, _), ms, mms, cms, fms in zip(wl.kernels, per, per_mean, copies,
                                                          floor_med):
        gbs = nbytes / (ms * 1e-3) / 1e9
        per_kernel[name] = {"us": round(ms * 1e3, 2), "mean_us": round(mms * 1e3, 2),
                            "bytes": nbytes, "GB/s": round(gbs, 1),
                            "frac": round(gbs / PEAK_HBM_GBS, 4),
                            "same_size_copy_us": None if cms != cms else round(cms * 1e3, 2),
                            "floor_us": None if fms is None else round(fms * 1e3, 2),
                            "vs_floor": None if fms is None else round(ms / fms, 3)}
    dname, dkind, dbytes, _ = wl.kernels[dom]
    achieved = dbytes / (dom_ms * 1e-3) / 1e9
    t = traffic.get(dname)
    tr = None
    if t and t.get("source_hash") == source_hash(dkind):
        tr = t.get("bytes_per_launch")

    out = {
        "metric": METRIC,
        "value": round(value, 1),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "settle": {"steps": settle_steps, "gpu_ms": round(settle_ms, 1)},
        "ms_per_step": round(step_ms, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {
            "workload": "one launch of each fused sub-kernel at its workload shape: "
                        "pointwise fp32 [256,1024]; softmax bf16 [8192,4096] + mask; "
                        "LayerNorm+residual bf16 [16384,4096]; GEMM epilogue+row-sum on "
                        "bf16 C [8192,8192]; block (32x512, hidden 1024, 16 heads, MLP 4096) "
                        "LN1, causal softmax, LN2+residual, bias+GELU, residual add",
            "step_bytes": wl.step_bytes,
            "io_dtypes": "bf16 (fp32 for the pointwise [256,1024] chain)",
        },
        "roofline": {"kernel": dname, "bound": "hbm", "achieved": round(achieved, 1),
                     "peak": PEAK_HBM_GBS, "unit": "GB/s",
                     "frac": round(achieved / PEAK_HBM_GBS, 4), "traffic": tr,
                     "algorithmic_bytes": dbytes, "launch_us": round(dom_ms * 1e3, 2)},
        "per_kernel": per_kernel,
        "per_kernel_note": "intervals between events recorded after every kernel, in a pass "
                           "of K steps after the timed region; us, GB/s and frac from the median "
                           "interval, mean_us the mean; each interval includes the cost of one "
                           "timing-only event (about 1 us). "
                           "same_size_copy_us: the calibration copy moving the same bytes "
                           "(half read, half written), timed the same way; floor_us: the launch's "
                           "access-shape floor (libaccessfloor.so: the same bytes in the same "
                           "launch shape, none of the arithmetic), median over K steps of floors "
                           "timed the same way; vs_floor = us / floor_us",
        "copy_calibration_GBs": round(copy_gbs, 1),
        "context": {"pointwise_bandwidth_scale": {
                        "shape": [262144, 1024], "dtype": "f32", "bytes": bw_bytes,
                        "us": round(bw_ms * 1e3, 2),
                        "GB/s": round(bw_bytes / (bw_ms * 1e-3) / 1e9, 1),
                        "frac": round(bw_bytes / (bw_ms * 1e-3) / 1e9 / PEAK_HBM_GBS, 4)},
                    "softmax_byte_mask": {
                        "shape": [8192, 4096], "dtype": "bf16", "mask": "u8", "bytes": sm8_bytes,
                        "us": round(sm8_us, 2),
                        "GB/s": round(sm8_bytes / (sm8_us * 1e-6) / 1e9, 1),
                        "frac": round(sm8_bytes / (sm8_us * 1e-6) / 1e9 / PEAK_HBM_GBS, 4),
                        "additive_bf16_mask_us": round(sm_add_us, 2),
                        "note": "each launch after a 1 GiB read-only pass, with its own events"},
                    "pointwise_program": {
                        "ops": "add_bias, scale 0.5, clamp [-1, 1], gelu_erf",
                        "shape": [16384, 4096], "dtype": "bf16", "bytes": prog_bytes,
                        "us": round(prog_us, 2),
                        "GB/s": round(prog_bytes / (prog_us * 1e-6) / 1e9, 1),
                        "frac": round(prog_bytes / (prog_us * 1e-6) / 1e9 / PEAK_HBM_GBS, 4),
                        "fixed_bias_gelu_chain_us": round(prog_chain_us, 2),
                        "note": "each launch after a 1 GiB read-only pass, with its own events"},
                    "block_forward_ms_with_gemms": round(wl.block_e2e_ms, 3),
                    "gemm_8192x8192x4096_ms": round(wl.gemm_8192x8192x4096_ms, 3),
                    "wall_s_warmup_and_timed": round(wall_s, 4), "setup_s": round(setup_s, 1),
                    "paper_geomean_speedups_vs_torch_compile_H200":
                        {"L1": 1.40, "L2": 1.15, "L3": 1.07}},
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(wl, args.cpu_sample)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
