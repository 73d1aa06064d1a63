"""Deterministic bottleneck-tier classifier over hardware counters.

KernelOPT's strategy analyst sorts every profiled kernel into one of four
tiers from its speed-of-light (SOL) throughputs before planning (Section
4.2, Agent Architecture):

  near-optimal    either SOL above 80 %
  memory-bound    SOL_mem > SOL_comp, both at most 80 %
  compute-bound   SOL_comp > SOL_mem, both at most 80 %
  underutilized   SOL_mem == SOL_comp, both at most 80 %

On MI355X the two SOL figures come from rocprofv3 counters and the kernel
duration t of a kernel-trace run:

  SOL_mem  = (FETCH_SIZE + WRITE_SIZE) bytes / t / 8 TB/s, each counter
             scaled by what it reads for a copy kernel of known size (the
             calibration dispatch of the same run);
  SOL_comp = the busiest issue pipe, as a fraction of its capacity at the
             2.4 GHz peak engine clock:
               VALU  (2 (N_valu - N_mfma - N_trans) + 8 N_trans) / (1024 SIMDs * f * t)
                     (issue costs measured on MI355X by csrc/issue_rate.hip:
                     a wave64 fp32 FMA occupies a SIMD for 2.3 cycles -- the
                     157 TFLOP/s fp32 vector peak without packed math -- and
                     v_exp_f32 / v_rcp_f32 for 8.3, a quarter of that rate)
               SALU  N_salu / (256 CUs * f * t)      (one scalar issue per CU cycle)
               MFMA  MfmaUtil / 100                  (matrix-core busy cycles)
             from SQ_INSTS_VALU, SQ_INSTS_MFMA, SQ_INSTS_VALU_TRANS_F32,
             SQ_INSTS_SALU and MfmaUtil.  rocprofv3's derived VALUBusy sums
             per-wave active cycles and can exceed 100 %; it is reported for
             context only.

The classifier is used as a reporting tool: ``python -m
paper_2609_30059_amd.tiers`` reads the CSV output of the rocprofv3 runs and
prints one Markdown table row per kernel.
"""
from __future__ import annotations

import argparse
import csv
import math
import re
import sys
from dataclasses import dataclass, field
from typing import Dict, Iterable, List, Optional, Tuple

NEAR_OPTIMAL = 0.80
HBM_PEAK_BYTES_PER_S = 8.0e12
SIMDS = 1024                 # 256 CUs x 4 SIMDs
CUS = 256
CLOCK_HZ = 2.4e9             # peak engine clock
VALU_CYCLES = 2.0            # SIMD cycles per wave64 VALU instruction
TRANS_CYCLES = 8.0           # SIMD cycles per wave64 fp32 transcendental

TIERS = ("near-optimal", "memory-bound", "compute-bound", "underutilized")


def classify(sol_mem: float, sol_comp: float, near: float = NEAR_OPTIMAL,
             tie: float = 0.0) -> str:
    """The tier of a kernel from its two SOL fractions (0..1).  `tie` is the
    band within which the two count as equal (0: exactly equal)."""
    for name, v in (("sol_mem", sol_mem), ("sol_comp", sol_comp)):
        if not (isinstance(v, (int, float)) and math.isfinite(v) and v >= 0):
            raise ValueError(f"{name} must be a finite fraction >= 0, got {v!r}")
    if not (0 < near and tie >= 0):
        raise ValueError("near must be > 0 and tie >= 0")
    if sol_mem > near or sol_comp > near:
        return "near-optimal"
    if abs(sol_mem - sol_comp) <= tie:
        return "underutilized"
    return "memory-bound" if sol_mem > sol_comp else "compute-bound"


@dataclass
class KernelProfile:
    """Per-dispatch averages of one kernel's counters."""
    name: str
    duration_ns: float = float("nan")
    fetch_kib: float = float("nan")        # FETCH_SIZE as the counter reads it
    write_kib: float = float("nan")        # WRITE_SIZE as the counter reads it
    raw: Dict[str, float] = field(default_factory=dict)    # every other counter

    def hbm_bytes(self, fetch_scale: float, write_scale: float) -> float:
        return (self.fetch_kib * fetch_scale + self.write_kib * write_scale) * 1024.0

    def pipes(self) -> Dict[str, float]:
        """Issue-pipe utilisations (fractions) that the counters allow."""
        if not (self.duration_ns > 0):
            raise ValueError(f"{self.name}: no duration")
        cyc = CLOCK_HZ * self.duration_ns * 1e-9
        r, out = self.raw, {}
        if "SQ_INSTS_VALU" in r:
            trans = r.get("SQ_INSTS_VALU_TRANS_F32", 0.0)
            plain = max(r["SQ_INSTS_VALU"] - r.get("SQ_INSTS_MFMA", 0.0) - trans, 0.0)
            out["VALU"] = (VALU_CYCLES * plain + TRANS_CYCLES * trans) / (SIMDS * cyc)
        if "SQ_INSTS_SALU" in r:
            out["SALU"] = r["SQ_INSTS_SALU"] / (CUS * cyc)
        if "MfmaUtil" in r:
            out["MFMA"] = r["MfmaUtil"] / 100.0
        return out

    def sol(self, fetch_scale: float = 1.0, write_scale: float = 1.0,
            peak: float = HBM_PEAK_BYTES_PER_S) -> Tuple[float, float]:
        """(SOL_mem, SOL_comp) as fractions."""
        if not (self.duration_ns > 0):
            raise ValueError(f"{self.name}: no duration")
        mem = self.hbm_bytes(fetch_scale, write_scale) / (self.duration_ns * 1e-9) / peak
        p = self.pipes()
        return mem, (max(p.values()) if p else 0.0)


def copy_scales(profiles: Dict[str, KernelProfile], pattern: str, read_bytes: float,
                write_bytes: float) -> Tuple[float, float]:
    """Counter scale factors from the calibration copy kernel: bytes it moves
    per dispatch divided by what FETCH_SIZE and WRITE_SIZE read for it."""
    hits = [p for n, p in profiles.items() if re.search(pattern, n)]
    if len(hits) != 1:
        raise ValueError(f"calibration pattern {pattern!r} matches {len(hits)} kernels")
    p = hits[0]
    return read_bytes / (p.fetch_kib * 1024.0), write_bytes / (p.write_kib * 1024.0)


# ---------------------------------------------------------------------------
# rocprofv3 CSV output
# ---------------------------------------------------------------------------
def _short(name: str) -> str:
    return name.replace("(anonymous namespace)::", "")


def label(name: str) -> str:
    """A table label: a kernel's name with its template arguments, without
    the return type, namespace and parameter list (library kernels keep
    their first 64 characters)."""
    n = re.sub(r"^void ", "", name)
    n = n.replace("fs::", "")
    depth, cut = 0, len(n)
    for i, ch in enumerate(n):
        if ch == "<":
            depth += 1
        elif ch == ">":
            depth -= 1
        elif ch == "(" and depth == 0 and i > 0:
            cut = i
            break
    n = n[:cut]
    return n if len(n) <= 64 or "<" in n else n[:64] + "..."


def read_kernel_stats(path: str, into: Dict[str, KernelProfile]) -> None:
    """Average durations from a ``*_kernel_stats.csv`` (--kernel-trace --stats)."""
    with open(path, newline="") as f:
        for r in csv.DictReader(f):
            n = _short(r["Name"])
            into.setdefault(n, KernelProfile(n)).duration_ns = float(r["AverageNs"])


def read_counters(path: str, into: Dict[str, KernelProfile]) -> None:
    """Per-dispatch averages of every counter in a ``*_counter_collection.csv``."""
    acc: Dict[Tuple[str, str], List[float]] = {}
    with open(path, newline="") as f:
        for r in csv.DictReader(f):
            key = (_short(r["Kernel_Name"]), r["Counter_Name"])
            acc.setdefault(key, []).append(float(r["Counter_Value"]))
    for (n, c), vals in acc.items():
        p = into.setdefault(n, KernelProfile(n))
        v = sum(vals) / len(vals)
        if c == "FETCH_SIZE":
            p.fetch_kib = v
        elif c == "WRITE_SIZE":
            p.write_kib = v
        else:
            p.raw[c] = v


def table(profiles: Iterable[KernelProfile], fetch_scale: float, write_scale: float,
          label=lambda n: n, near: float = NEAR_OPTIMAL, tie: float = 0.0) -> List[str]:
    """Markdown rows: kernel, duration, HBM GB/s, SOL_mem, SOL_comp (and the
    pipe that sets it), rocprofv3's VALUBusy for context, tier."""
    rows = ["| kernel | avg us | HBM GB/s | SOL_mem % | SOL_comp % (pipe) | VALUBusy % | tier |",
            "|---|---|---|---|---|---|---|"]
    for p in profiles:
        if not (p.duration_ns > 0) or math.isnan(p.fetch_kib) or math.isnan(p.write_kib):
            continue
        mem, comp = p.sol(fetch_scale, write_scale)
        pp = p.pipes()
        pipe = max(pp, key=pp.get) if pp else "-"
        gbs = p.hbm_bytes(fetch_scale, write_scale) / (p.duration_ns * 1e-9) / 1e9
        vb = f"{p.raw['VALUBusy']:.1f}" if "VALUBusy" in p.raw else "-"
        rows.append(f"| {label(p.name)} | {p.duration_ns / 1e3:.1f} | {gbs:.0f} | {100 * mem:.1f} | "
                    f"{100 * comp:.1f} ({pipe}) | {vb} | {classify(mem, comp, near, tie)} |")
    return rows


def main(argv: Optional[List[str]] = None) -> int:
    ap = argparse.ArgumentParser(description="Bottleneck tiers from rocprofv3 CSV output")
    ap.add_argument("--stats", required=True, help="*_kernel_stats.csv of a kernel-trace run")
    ap.add_argument("--counters", nargs="+", required=True,
                    help="*_counter_collection.csv files (FETCH_SIZE, WRITE_SIZE, pipes)")
    ap.add_argument("--calibration", default=r"copy128_kernel",
                    help="regex of the calibration copy kernel")
    ap.add_argument("--calibration-bytes", type=float, default=float(1 << 30),
                    help="bytes the calibration kernel reads (and writes) per dispatch")
    ap.add_argument("--tie", type=float, default=0.0)
    a = ap.parse_args(argv)
    prof: Dict[str, KernelProfile] = {}
    read_kernel_stats(a.stats, prof)
    for c in a.counters:
        read_counters(c, prof)
    fs_, ws_ = copy_scales(prof, a.calibration, a.calibration_bytes, a.calibration_bytes)
    print(f"FETCH_SIZE scale x{fs_:.4f}, WRITE_SIZE scale x{ws_:.4f}")
    by_time = sorted(prof.values(), key=lambda p: -p.duration_ns if p.duration_ns > 0 else 0.0)
    for line in table(by_time, fs_, ws_, label=label, tie=a.tie):
        print(line)
    return 0


if __name__ == "__main__":
    sys.exit(main())
