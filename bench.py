#!/usr/bin/env python3
"""Benchmark of the fused sub-kernels on one MI355X.

One step = one launch of every fused sub-kernel at its workload shape:
  pw_cfg1    pointwise GELU_erf(x*s + b) + r, fp32 [256, 1024]
  sm_cfg2    row softmax, scale + bf16 additive mask, bf16 [8192, 4096]
  ln_cfg3    LayerNorm + residual, bf16 [16384, 4096]
  ep_cfg4    GEMM epilogue (+bias, *scale, sigmoid, row sum) on C bf16 [8192, 8192]
  blk_ln1    block LayerNorm 1, bf16 [16384, 1024]
  blk_sm     block causal softmax, bf16 [32, 16, 512, 512], scale 1/8
  blk_ln2    block LayerNorm 2 + residual, bf16 [16384, 1024]
  blk_gelu   block bias + GELU_erf, bf16 [16384, 4096]
  blk_res    block residual add, bf16 [16384, 1024]
The GEMMs (the fixed library calls) run once before timing to produce the
resident inputs of the epilogue and block sub-kernels; they are reported
separately as context, never inside `value`.

`value` = compulsory bytes of one step (each input read once, each output
written once; the causal upper triangle is not read) / step time, in GB/s.
Inputs are resident in HBM when timing starts.  Every kernel in a step is
separated from its previous launch by more than the 256 MB Infinity Cache of
other traffic, so inputs come from HBM (pw_cfg1, 3 MiB, stays cache
resident and is latency-bound).

Prints one JSON line.
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

PEAK_HBM_GBS = 8000.0
METRIC = "achieved HBM GB/s and % of MI355X peak per fused sub-kernel; oracle match"
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic.json")
KERNEL_SOURCES = {
    "pw": "pointwise.hip", "sm": "softmax.hip", "ln": "layernorm.hip", "ep": "epilogue.hip",
}


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
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-sample-scale", type=float, default=1.0,
                    help="scales the rows of the CPU oracle sample")
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

        # cfg1
        h1 = fd.make_inputs("cfg1", seed)
        self.host["cfg1"] = h1
        self.pw = dict(x=d(h1["x"]), b=d(h1["bias"]), r=d(h1["residual"]), s=h1["scale"])
        self.pw["y"] = torch.empty_like(self.pw["x"])
        # cfg2
        h2 = fd.make_inputs("cfg2", seed)
        self.host["cfg2"] = h2
        self.sm = dict(x=d(h2["x"]), m=d(h2["mask"]), s=h2["scale"])
        self.sm["y"] = torch.empty_like(self.sm["x"])
        # cfg3
        h3 = fd.make_inputs("cfg3", seed)
        self.host["cfg3"] = h3
        self.ln = dict(x=d(h3["x"]), r=d(h3["residual"]), g=d(h3["gamma"]), b=d(h3["beta"]),
                       eps=h3["eps"])
        self.ln["y"] = torch.empty_like(self.ln["x"])
        self.ln["ro"] = torch.empty_like(self.ln["x"])
        # cfg4: GEMM once (library call), then the epilogue on its output
        h4 = fd.make_inputs("cfg4", seed)
        self.host["cfg4"] = h4
        a, b = d(h4["a"]), d(h4["b"])
        self.ep = dict(bias=d(h4["bias"]), scale=d(h4["col_scale"]))
        self.ep["c"] = fs.gemm(a, b)
        self.ep["out"] = torch.empty(self.ep["c"].shape[0], dtype=torch.float32, device=dev)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(3):
            fs.gemm(a, b, out=self.ep["c"])
        torch.cuda.synchronize()
        self.gemm_cfg4_ms = (time.perf_counter() - t0) / 3 * 1e3
        del a, b
        # cfg5: one full forward pass makes every block sub-kernel input resident
        h5 = fd.make_inputs("cfg5", seed)
        self.host["cfg5"] = {k: h5[k] for k in ("x", "eps", "heads")}
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
            ("pw_cfg1", "pw", 256 * 1024 * 4 * 3 + 1024 * 4,
             lambda: fs.pointwise_chain(self.pw["x"], self.pw["b"], self.pw["r"], self.pw["s"],
                                        "gelu_erf", out=self.pw["y"])),
            ("sm_cfg2", "sm", 8192 * 4096 * 2 * 3,
             lambda: fs.row_softmax(self.sm["x"], self.sm["m"], self.sm["s"], out=self.sm["y"])),
            ("ln_cfg3", "ln", 16384 * 4096 * 2 * 4 + 4096 * 2 * 2,
             lambda: fs.layernorm_residual(self.ln["x"], self.ln["r"], self.ln["g"], self.ln["b"],
                                           self.ln["eps"], out=self.ln["y"],
                                           residual_out=self.ln["ro"])),
            ("ep_cfg4", "ep", 8192 * 8192 * 2 + 8192 * (2 + 4) + 8192 * 4,
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
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(iters):
            fs.copy_(dst, src)
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / iters
        del src, dst
        return 2 * nbytes / (ms * 1e-3) / 1e9


# ---------------------------------------------------------------------------
# CPU baseline: the float64 oracle on a bounded sample of the same step
# ---------------------------------------------------------------------------
def cpu_baseline(wl: Workload, scale: float):
    import numpy as np
    from threadpoolctl import threadpool_limits

    import oracle
    fd = wl.fd
    h = wl.host
    n = lambda r: max(1, int(r * scale))   # noqa: E731
    sample = {"pw_cfg1": n(256), "sm_cfg2": n(64), "ln_cfg3": n(128), "ep_cfg4": n(64),
              "blk_ln1": n(512), "blk_sm": n(512), "blk_ln2": n(512), "blk_gelu": n(256),
              "blk_res": n(512)}
    rng = np.random.default_rng(1)
    # block intermediates of the sample rows, read back from the resident
    # device inputs of each block sub-kernel (inputs, not results, of the
    # kernels being timed)
    torch = wl.torch

    def rows_of(t, r):
        v = t.reshape(-1, t.shape[-1])[:r]
        return v.float().cpu().numpy().astype(np.float64)

    blk = wl.blk
    pw = {k: v.float().cpu().numpy().astype(np.float64) for k, v in blk.p.items()}
    total_bytes = 0
    t_total = 0.0
    with threadpool_limits(limits=1):
        def timed(fn):
            t0 = time.perf_counter()
            fn()
            return time.perf_counter() - t0
        r = sample["pw_cfg1"]
        c1 = h["cfg1"]
        x, rr = c1["x"].rows(slice(0, r)).f64(), c1["residual"].rows(slice(0, r)).f64()
        t_total += timed(lambda: oracle.pointwise_chain(x, c1["bias"].f64(), rr, c1["scale"],
                                                        "gelu_erf"))
        total_bytes += r * 1024 * 12
        r = sample["sm_cfg2"]
        c2 = h["cfg2"]
        x, m = c2["x"].rows(slice(0, r)).f64(), c2["mask"].rows(slice(0, r)).f64()
        t_total += timed(lambda: oracle.row_softmax(x, m, c2["scale"]))
        total_bytes += r * 4096 * 6
        r = sample["ln_cfg3"]
        c3 = h["cfg3"]
        x, rr = c3["x"].rows(slice(0, r)).f64(), c3["residual"].rows(slice(0, r)).f64()
        g, b = c3["gamma"].f64(), c3["beta"].f64()
        t_total += timed(lambda: (oracle.layernorm_residual(x, rr, g, b, c3["eps"]),
                                  oracle.residual_store_bf16(x, rr)))
        total_bytes += r * 4096 * 8
        r = sample["ep_cfg4"]
        c4 = h["cfg4"]
        cm = rows_of(wl.ep["c"], r)
        t_total += timed(lambda: oracle.gemm_epilogue_reduce(cm, c4["bias"].f64(),
                                                             c4["col_scale"].f64(), "sigmoid",
                                                             "sum"))
        total_bytes += r * 8192 * 2 + r * 4
        buf = wl.buf
        H = blk.hidden
        r = sample["blk_ln1"]
        x = rows_of(wl.bx, r)
        t_total += timed(lambda: oracle.layernorm_residual(x, None, pw["ln1_gamma"],
                                                           pw["ln1_beta"], blk.eps))
        total_bytes += r * H * 4
        r = sample["blk_sm"]
        sc = rows_of(buf["scores"], r)
        S = buf["scores"].shape[-1]
        t_total += timed(lambda: oracle.row_softmax(sc, None, 1.0 / math.sqrt(blk.dh),
                                                    causal_q_len=S))
        total_bytes += (r * (S + 1) // 2) * 2 + r * S * 2
        r = sample["blk_ln2"]
        att, x = rows_of(buf["att"], r), rows_of(wl.bx, r)
        t_total += timed(lambda: oracle.layernorm_residual(att, x, pw["ln2_gamma"],
                                                           pw["ln2_beta"], blk.eps))
        total_bytes += r * H * 8
        r = sample["blk_gelu"]
        u = rows_of(buf["u"], r)
        t_total += timed(lambda: oracle.pointwise_chain(u, pw["b_1"], None, 1.0, "gelu_erf"))
        total_bytes += r * blk.mlp * 4
        r = sample["blk_res"]
        dd, h1 = rows_of(buf["d"], r), rows_of(buf["h1"], r)
        t_total += timed(lambda: oracle.pointwise_chain(dd, None, h1, 1.0, "none"))
        total_bytes += r * H * 6
    del rng, torch
    desc = ", ".join(f"{k} {v} rows" for k, v in sample.items())
    return {"value": round(total_bytes / t_total / 1e9, 4), "unit": "GB/s", "cores": 1,
            "kind": "oracle", "seconds": round(t_total, 3),
            "sample": f"float64 oracle, one thread, on the first rows of each sub-kernel's "
                      f"input ({desc}); {total_bytes} compulsory bytes"}


def load_traffic():
    try:
        with open(TRAFFIC_FILE) as f:
            return json.load(f)
    except (OSError, ValueError):
        return {}


def main():
    args = parse()
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
    for _ in range(args.warmup):
        wl.step()
    torch.cuda.synchronize()

    # timed region: K steps, boundary events between consecutive kernels
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(nk + 1)]
           for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for s in range(args.steps):
        evs[s][0].record()
        wl.step(evs[s])
    torch.cuda.synchronize()
    wall_s = time.perf_counter() - t0

    per = [0.0] * nk
    step_ms = 0.0
    for s in range(args.steps):
        for i in range(nk):
            per[i] += evs[s][i].elapsed_time(evs[s][i + 1])
        step_ms += evs[s][0].elapsed_time(evs[s][nk])
    per = [p / args.steps for p in per]
    step_ms /= args.steps
    value = wl.step_bytes / (step_ms * 1e-3) / 1e9

    traffic = load_traffic()
    per_kernel = {}
    for (name, kind, nbytes, _), ms in zip(wl.kernels, per):
        gbs = nbytes / (ms * 1e-3) / 1e9
        per_kernel[name] = {"us": round(ms * 1e3, 2), "bytes": nbytes, "GB/s": round(gbs, 1),
                            "frac": round(gbs / PEAK_HBM_GBS, 4)}
    dom = max(range(nk), key=lambda i: per[i])
    dname, dkind, dbytes, _ = wl.kernels[dom]
    achieved = dbytes / (per[dom] * 1e-3) / 1e9
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
                     "algorithmic_bytes": dbytes},
        "per_kernel": per_kernel,
        "copy_calibration_GBs": round(copy_gbs, 1),
        "context": {"block_forward_ms_with_gemms": round(wl.block_e2e_ms, 3),
                    "gemm_cfg4_ms": round(wl.gemm_cfg4_ms, 3),
                    "wall_s_timed_region": round(wall_s, 4), "setup_s": round(setup_s, 1),
                    "paper_geomean_speedups_vs_torch_compile_H200":
                        {"L1": 1.40, "L2": 1.15, "L3": 1.07}},
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(wl, args.cpu_sample_scale)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
