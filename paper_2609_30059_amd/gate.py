"""Model-level performance gate for the stitched transformer block.

KernelOPT accepts an optimised sub-kernel only if the re-stitched model is
not slower than the compiler's model beyond a noise margin (Gate 4,
Section 4.4, Eq. 5):

    V_perf(k, k0) = 1[ tau_M(k0 -> k) <= gamma * tau_M(k0) ],   gamma = 1.03

where tau_M is the wall-clock time of the whole model, measured by a
do_bench-style loop (25 ms warm-up, 100 ms of repetitions, Section 4.4 and
Table 5) in a separate process per measurement so that no device state
leaks from one into the next.

Here M(k0) is the same pre-LN block with the same hipBLASLt GEMM calls but
its five sub-kernels computed by PyTorch eager operators (the unfused
baseline), and M(k0 -> k) is the block with the libfusedsub kernels.  Three
more models are timed for context only: the fused block captured once as a
HIP graph and replayed (the same launches without per-launch host work), the
whole block written in plain PyTorch eager (its GEMMs included), and that
eager block under torch.compile.

Run ``python -m paper_2609_30059_amd.gate`` for the JSON report.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import statistics
import subprocess
import sys
from typing import Callable, Dict, Optional

from .timing import TimingEvent

GAMMA = 1.03

VARIANTS = ("fused", "fused_graph", "eager_subkernels", "eager", "compiled")


def perf_gate(tau_candidate: float, tau_baseline: float, gamma: float = GAMMA) -> bool:
    """Eq. 5: the candidate model passes if its time is at most gamma times
    the baseline model's time.  Times must be positive and finite."""
    for name, v in (("tau_candidate", tau_candidate), ("tau_baseline", tau_baseline),
                    ("gamma", gamma)):
        if not (isinstance(v, (int, float)) and math.isfinite(v) and v > 0):
            raise ValueError(f"{name} must be a positive finite number, got {v!r}")
    return tau_candidate <= gamma * tau_baseline


# ---------------------------------------------------------------------------
# timing
# ---------------------------------------------------------------------------
def bench_plan(estimate_ms: float, warmup_ms: float = 25.0, rep_ms: float = 100.0):
    """Warm-up and repetition counts that fill the requested budgets given one
    call's estimated time (at least one of each)."""
    if not (estimate_ms > 0 and math.isfinite(estimate_ms)):
        raise ValueError("estimate_ms must be positive and finite")
    return max(1, int(warmup_ms / estimate_ms)), max(1, int(rep_ms / estimate_ms))


def do_bench(fn: Callable[[], object], warmup_ms: float = 25.0, rep_ms: float = 100.0,
             flush_bytes: int = 512 << 20) -> Dict[str, float]:
    """Time fn on the current stream with device events: one call, a
    five-call estimate, warm-up calls for warmup_ms, then rep_ms of timed
    calls, each after a clear of a flush_bytes buffer (larger than the
    last-level cache) outside its timed region.  Returns the median, min and
    mean per call in ms."""
    import torch
    fn()
    torch.cuda.synchronize()
    flush = torch.empty(flush_bytes, dtype=torch.uint8, device="cuda") if flush_bytes else None
    e0, e1 = TimingEvent(), TimingEvent()
    e0.record()
    for _ in range(5):
        fn()
    e1.record()
    torch.cuda.synchronize()
    n_warm, n_rep = bench_plan(e0.elapsed_time(e1) / 5, warmup_ms, rep_ms)
    for _ in range(n_warm):
        fn()
    starts = [TimingEvent() for _ in range(n_rep)]
    ends = [TimingEvent() for _ in range(n_rep)]
    for i in range(n_rep):
        if flush is not None:
            flush.zero_()
        starts[i].record()
        fn()
        ends[i].record()
    torch.cuda.synchronize()
    t = [s.elapsed_time(e) for s, e in zip(starts, ends)]
    return {"median_ms": statistics.median(t), "min_ms": min(t), "mean_ms": statistics.fmean(t),
            "reps": n_rep}


# ---------------------------------------------------------------------------
# the baseline models
# ---------------------------------------------------------------------------
def _baseline_block_class():
    import torch
    import torch.nn.functional as F

    from .block import TransformerBlock

    class EagerSubkernelBlock(TransformerBlock):
        """The block with the same GEMM calls and PyTorch eager sub-kernels:
        the model M(k0) of Eq. 5.  Each stage returns a new tensor, as eager
        code does, and the GEMMs read it from the activation dictionary."""

        _causal = None

        def layernorm1(self, x2, buf):
            p = self.p
            buf["a"] = F.layer_norm(x2, (self.hidden,), p["ln1_gamma"], p["ln1_beta"], self.eps)

        def softmax(self, buf, seq):
            if self._causal is None or self._causal.shape[0] != seq:
                self._causal = torch.ones(seq, seq, dtype=torch.bool,
                                          device=buf["scores"].device).triu_(1)
            s = buf["scores"] * (1.0 / math.sqrt(self.dh))
            s = s.masked_fill(self._causal, float("-inf"))
            buf["probs"] = torch.softmax(s, dim=-1)

        def layernorm2_residual(self, x2, buf):
            p = self.p
            buf["h1"] = buf["att"] + x2
            buf["m"] = F.layer_norm(buf["h1"], (self.hidden,), p["ln2_gamma"], p["ln2_beta"],
                                    self.eps)

        def bias_gelu(self, buf):
            buf["g"] = F.gelu(buf["u"] + self.p["b_1"])

        def residual_add(self, buf):
            buf["out"] = buf["d"] + buf["h1"]

    return EagerSubkernelBlock


def eager_block(p: Dict[str, "object"], x, heads: int, eps: float):
    """The whole block in plain PyTorch eager (GEMMs included), the way a
    model author writes it.  Context only: its GEMMs differ from the
    library calls of the stitched block."""
    import torch
    import torch.nn.functional as F
    B, S, H = x.shape
    dh = H // heads
    x2 = x.reshape(B * S, H)
    a = F.layer_norm(x2, (H,), p["ln1_gamma"], p["ln1_beta"], eps)
    qkv = torch.addmm(p["b_qkv"], a, p["w_qkv"])
    qkv = qkv.view(B, S, 3, heads, dh).permute(2, 0, 3, 1, 4)
    q, k, v = qkv[0].contiguous(), qkv[1].contiguous(), qkv[2].contiguous()
    s = torch.matmul(q, k.transpose(-1, -2).contiguous()) * (1.0 / math.sqrt(dh))
    causal = torch.ones(S, S, dtype=torch.bool, device=x.device).triu_(1)
    pr = torch.softmax(s.masked_fill(causal, float("-inf")), dim=-1)
    o = torch.matmul(pr, v).transpose(1, 2).reshape(B * S, H)
    att = torch.addmm(p["b_o"], o, p["w_o"])
    h1 = att + x2
    m = F.layer_norm(h1, (H,), p["ln2_gamma"], p["ln2_beta"], eps)
    g = F.gelu(torch.addmm(p["b_1"], m, p["w_1"]))
    d = torch.addmm(p["b_2"], g, p["w_2"])
    return d + h1


# ---------------------------------------------------------------------------
# one measurement (runs in its own process)
# ---------------------------------------------------------------------------
def _device_inputs(seed: int, dims: Optional[Dict[str, int]] = None):
    import numpy as np
    import torch

    import fusedsub_data as fd
    from .block import PARAM_NAMES
    h = fd.block_inputs(seed, **(dims or fd.BLOCK_DIMS))

    def dev(t):
        return torch.from_numpy(t.data.view(np.int16)).view(torch.bfloat16).cuda()

    return {k: dev(h[k]) for k in PARAM_NAMES}, dev(h["x"]), h["heads"], h["eps"]


def measure(variant: str, seed: int = 0, warmup_ms: float = 25.0, rep_ms: float = 100.0,
            dims: Optional[Dict[str, int]] = None) -> Dict[str, object]:
    """Time one model variant on the block workload; returns the timing and a
    checksum of its output."""
    import torch

    from .block import TransformerBlock
    if variant not in VARIANTS:
        raise ValueError(f"variant must be one of {VARIANTS}")
    params, x, heads, eps = _device_inputs(seed, dims)
    if variant in ("fused", "fused_graph", "eager_subkernels"):
        cls = _baseline_block_class() if variant == "eager_subkernels" else TransformerBlock
        blk = cls(params, heads=heads, eps=eps)
        buf = blk.alloc(*x.shape[:2], x.device)
        fn = lambda: blk.forward(x, buf)              # noqa: E731
        get = lambda: buf["out"]                      # noqa: E731
        if variant == "fused_graph":
            fn = _captured(fn)
    else:
        f = eager_block if variant == "eager" else torch.compile(eager_block)
        res = {}
        fn = lambda: res.__setitem__("out", f(params, x, heads, eps))   # noqa: E731
        get = lambda: res["out"]                      # noqa: E731
    t = do_bench(fn, warmup_ms, rep_ms)
    out = get().float()
    t.update(variant=variant, out_abs_mean=float(out.abs().mean()),
             out_finite=bool(torch.isfinite(out).all()))
    return t


def _captured(fn: Callable[[], object]) -> Callable[[], object]:
    """fn captured once as a HIP graph (after a warm-up call on a side stream
    that creates the GEMM plans and loads every kernel); returns its replay."""
    import torch
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        fn()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        fn()
    torch.cuda.synchronize()
    return g.replay


def run_isolated(variant: str, seed: int, warmup_ms: float, rep_ms: float,
                 timeout_s: float = 600.0) -> Dict[str, object]:
    """measure() in a child process (started fresh, never exec'd over this
    one); returns its JSON result."""
    cmd = [sys.executable, "-m", "paper_2609_30059_amd.gate", "--variant", variant,
           "--seed", str(seed), "--warmup-ms", str(warmup_ms), "--rep-ms", str(rep_ms)]
    r = subprocess.run(cmd, capture_output=True, text=True, timeout=timeout_s,
                       cwd=os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
    if r.returncode != 0:
        raise RuntimeError(f"{variant} measurement failed ({r.returncode}):\n{r.stderr[-2000:]}")
    return json.loads(r.stdout.strip().splitlines()[-1])


def report(results: Dict[str, Dict[str, object]], gamma: float = GAMMA) -> Dict[str, object]:
    """The gate verdict from the measured variants."""
    tf = results["fused"]["median_ms"]
    tb = results["eager_subkernels"]["median_ms"]
    out = {"gate": "V_perf", "gamma": gamma, "tau_candidate_ms": tf, "tau_baseline_ms": tb,
           "speedup": tb / tf, "pass": perf_gate(tf, tb, gamma),
           "variants": {k: v["median_ms"] for k, v in results.items()}}
    for ctx in ("eager", "compiled"):
        if ctx in results:
            out[f"speedup_vs_{ctx}"] = results[ctx]["median_ms"] / tf
    if "fused_graph" in results:
        out["graph_replay_speedup"] = tf / results["fused_graph"]["median_ms"]
    return out


def main(argv=None) -> int:
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("--variant", choices=VARIANTS, help="time one variant in this process")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--warmup-ms", type=float, default=25.0)
    ap.add_argument("--rep-ms", type=float, default=100.0)
    ap.add_argument("--gamma", type=float, default=GAMMA)
    ap.add_argument("--compile", action="store_true", help="also time torch.compile")
    a = ap.parse_args(argv)
    if a.variant:
        print(json.dumps(measure(a.variant, a.seed, a.warmup_ms, a.rep_ms)), flush=True)
        return 0
    variants = (["fused", "fused_graph", "eager_subkernels", "eager"]
                + (["compiled"] if a.compile else []))
    results = {}
    for v in variants:
        results[v] = run_isolated(v, a.seed, a.warmup_ms, a.rep_ms)
        print(f"# {v}: {results[v]['median_ms']:.4f} ms", file=sys.stderr, flush=True)
    print(json.dumps(report(results, a.gamma)), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
