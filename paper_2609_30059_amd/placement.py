"""Epilogue placement study: where a thin epilogue after a library GEMM is
cheapest on MI355X.

KernelOPT keeps GEMMs as library calls and rewrites only the generated
sub-kernels around them; it reports that in GEMM-dominated models a thin
epilogue gains little and an extra dispatch can make the model slower
(Section 6.2, library dominance; Section 6.3).  This module measures the alternatives for the two
epilogues of this library:

GEMM + bias/scale/sigmoid + row sum  (C = A @ B, A [8192, 4096], B [4096, 8192])
  gemm_only       the GEMM alone (the reference for marginal costs)
  separate_cold   fs_gemm_epilogue_reduce on C after a cache flush
  separate_hot    the same epilogue right after the GEMM, while C (128 MiB)
                  may still sit in the 256 MB last-level cache
  library_affine  hipBLASLt applies the column scale (as its alpha vector)
                  and scale * bias (fp32) in its own epilogue; the sigmoid
                  and row sum stay in fs_gemm_epilogue_reduce.  (hipBLASLt's
                  SIGMOID epilogue is not usable: with this ROCm release it
                  leaves bf16 output untouched.)

Block MLP epilogues ([16384, 1024] @ [1024, 4096] and back)
  subkernel       GEMM, then fs_pointwise_chain (bias + GELU_erf), and GEMM
                  with bias, then fs_pointwise_chain (+ residual)
  library         hipBLASLt GELU_BIAS epilogue (its own GELU approximation)
                  and the residual read as beta * C inside the second GEMM

The report gives the times and how far the placements' results differ;
their accuracy against the float64 definitions is checked by the GPU tests.
Run ``python -m paper_2609_30059_amd.placement`` for the JSON report.
"""
from __future__ import annotations

import argparse
import json
import statistics
import sys
from typing import Dict

from . import ops
from .block import TransformerBlock
from .gate import do_bench
from .timing import TimingEvent

LLC_FLUSH_BYTES = 512 << 20


def _events(n):
    import torch
    return [TimingEvent() for _ in range(n)]


def time_pair(first, second, reps: int = 30, flush: bool = True) -> Dict[str, float]:
    """Median device time of `first`, of `second` run right after it, and of
    the pair, each rep after an optional cache flush."""
    import torch
    buf = torch.empty(LLC_FLUSH_BYTES, dtype=torch.uint8, device="cuda") if flush else None
    first()
    second()
    torch.cuda.synchronize()
    e = [_events(3) for _ in range(reps)]
    for ev in e:
        if buf is not None:
            buf.zero_()
        ev[0].record()
        first()
        ev[1].record()
        second()
        ev[2].record()
    torch.cuda.synchronize()
    t1 = [a.elapsed_time(b) for a, b, _ in e]
    t2 = [b.elapsed_time(c) for _, b, c in e]
    return {"first_ms": statistics.median(t1), "second_ms": statistics.median(t2),
            "pair_ms": statistics.median([x + y for x, y in zip(t1, t2)])}


def time_cold(fn, reps: int = 30) -> float:
    """Median device time of fn, each rep after a cache flush."""
    import torch
    buf = torch.empty(LLC_FLUSH_BYTES, dtype=torch.uint8, device="cuda")
    fn()
    torch.cuda.synchronize()
    e = [_events(2) for _ in range(reps)]
    for ev in e:
        buf.zero_()
        ev[0].record()
        fn()
        ev[1].record()
    torch.cuda.synchronize()
    return statistics.median(a.elapsed_time(b) for a, b in e)


# ---------------------------------------------------------------------------
# the GEMM + sigmoid row-sum epilogue
# ---------------------------------------------------------------------------
def epilogue_study(seed: int = 0, rows: int = 8192, cols: int = 8192, k: int = 4096,
                   reps: int = 30) -> Dict[str, object]:
    import numpy as np
    import torch

    import fusedsub_data as fd
    h = fd.gemm_epilogue_inputs(seed, rows, cols, k)

    def dev(t):
        if t.dtype == "f32":
            return torch.from_numpy(t.data).cuda()
        return torch.from_numpy(t.data.view(np.int16)).view(torch.bfloat16).cuda()

    a, b, bias, scale = dev(h["a"]), dev(h["b"]), dev(h["bias"]), dev(h["col_scale"])
    c = torch.empty(rows, cols, dtype=torch.bfloat16, device="cuda")
    zc = torch.empty_like(c)
    out_sep = torch.empty(rows, dtype=torch.float32, device="cuda")
    out_lib = torch.empty_like(out_sep)
    # (C + bias) * scale = scale * C + scale * bias: the library form takes the
    # column scale as its alpha vector and scale * bias as an fp32 bias
    sbias = (bias.float() * scale).contiguous()

    def gemm():
        ops.gemm(a, b, out=c)

    def epi():
        ops.gemm_epilogue_reduce(c, bias, scale, "sigmoid", "sum", out=out_sep)

    def lib_gemm():
        ops.gemm(a, b, bias=sbias, col_scale=scale, out=zc)

    def lib_sum():
        ops.gemm_epilogue_reduce(zc, None, None, "sigmoid", "sum", out=out_lib)

    res: Dict[str, object] = {"shape": {"m": rows, "n": cols, "k": k}}
    hot = time_pair(gemm, epi, reps)
    res["gemm_only_ms"] = hot["first_ms"]
    res["separate_hot"] = {"epilogue_ms": hot["second_ms"], "total_ms": hot["pair_ms"]}
    res["separate_cold"] = {"epilogue_ms": time_cold(epi, reps)}
    res["separate_cold"]["total_ms"] = res["gemm_only_ms"] + res["separate_cold"]["epilogue_ms"]
    lib = time_pair(lib_gemm, lib_sum, reps)
    res["library_affine"] = {"gemm_ms": lib["first_ms"], "epilogue_ms": lib["second_ms"],
                             "total_ms": lib["pair_ms"]}
    # how far the two placements' results are apart (their accuracy against
    # the float64 definition is checked by the GPU tests)
    epi()
    lib_gemm()
    lib_sum()
    torch.cuda.synchronize()
    res["library_vs_separate_max_abs_diff"] = float((out_lib - out_sep).abs().max())
    res["row_sum_magnitude"] = float(out_sep.abs().mean())
    return res


# ---------------------------------------------------------------------------
# the block's MLP epilogues
# ---------------------------------------------------------------------------
class LibraryEpilogueBlock(TransformerBlock):
    """The block with its MLP epilogues inside the hipBLASLt calls: bias +
    GELU in the first GEMM's epilogue (hipBLASLt's GELU, an approximation of
    the erf form) and the residual read as beta * C by the second GEMM."""

    def mlp_up(self, buf):
        ops.gemm(buf["m"], self.p["w_1"], bias=self.p["b_1"], act="gelu", out=buf["g"])

    def mlp_down(self, buf):
        ops.gemm(buf["g"], self.p["w_2"], bias=self.p["b_2"], c_in=buf["h1"], beta=1.0,
                 out=buf["out"])


def mlp_study(seed: int = 0, reps: int = 30) -> Dict[str, object]:
    import numpy as np
    import torch

    import fusedsub_data as fd
    from .block import PARAM_NAMES
    h = fd.make_inputs("block_32x512x1024", seed)

    def dev(t):
        return torch.from_numpy(t.data.view(np.int16)).view(torch.bfloat16).cuda()

    params = {k: dev(h[k]) for k in PARAM_NAMES}
    x = dev(h["x"])
    sub = TransformerBlock(params, heads=h["heads"], eps=h["eps"])
    lib = LibraryEpilogueBlock(params, heads=h["heads"], eps=h["eps"])
    bs, bl = sub.alloc(*x.shape[:2], x.device), lib.alloc(*x.shape[:2], x.device)
    sub.forward(x, bs)
    lib.forward(x, bl)
    torch.cuda.synchronize()
    res: Dict[str, object] = {}
    up_s = time_pair(lambda: ops.gemm(bs["m"], params["w_1"], out=bs["u"]),
                     lambda: sub.bias_gelu(bs), reps)
    up_l = time_cold(lambda: lib.mlp_up(bl), reps)
    dn_s = time_pair(lambda: ops.gemm(bs["g"], params["w_2"], bias=params["b_2"], out=bs["d"]),
                     lambda: sub.residual_add(bs), reps)
    dn_l = time_cold(lambda: lib.mlp_down(bl), reps)
    res["bias_gelu"] = {"subkernel": {"gemm_ms": up_s["first_ms"], "epilogue_ms": up_s["second_ms"],
                                      "total_ms": up_s["pair_ms"]},
                        "library_ms": up_l}
    res["residual"] = {"subkernel": {"gemm_ms": dn_s["first_ms"], "epilogue_ms": dn_s["second_ms"],
                                     "total_ms": dn_s["pair_ms"]},
                       "library_ms": dn_l}
    res["block_ms"] = {"subkernel": do_bench(lambda: sub.forward(x, bs))["median_ms"],
                       "library": do_bench(lambda: lib.forward(x, bl))["median_ms"]}
    # how far the placements are apart: GELU output on the same GEMM input
    # and the block output (accuracy against float64 is in the GPU tests)
    ops.gemm(bs["m"], params["w_1"], out=bs["u"])
    sub.bias_gelu(bs)
    lib.mlp_up(bl)
    torch.cuda.synchronize()
    res["gelu_max_abs_diff"] = float((bs["g"].float() - bl["g"].float()).abs().max())
    res["out_max_abs_diff"] = float((bs["out"].float() - bl["out"].float()).abs().max())
    return res


def main(argv=None) -> int:
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--reps", type=int, default=30)
    ap.add_argument("--only", choices=["epilogue", "mlp"])
    a = ap.parse_args(argv)
    out = {}
    if a.only in (None, "epilogue"):
        out["gemm_sigmoid_row_sum"] = epilogue_study(a.seed, reps=a.reps)
        print("# epilogue study done", file=sys.stderr, flush=True)
    if a.only in (None, "mlp"):
        out["block_mlp"] = mlp_study(a.seed, reps=a.reps)
        print("# mlp study done", file=sys.stderr, flush=True)
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
