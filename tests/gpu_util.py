"""Helpers of the GPU parity tests: device transfer of the seeded inputs,
tolerance checks, guard-band buffers and the error-ratio diagnostic of the
paper's float64 fallback (Section 4.4, Gate 3, Eq. 4)."""
from __future__ import annotations

import json
import os
import sys

import numpy as np
import pytest
import torch

import fusedsub_data as fd

# tolerance contract (elementwise |got - ref| <= atol + rtol*|ref|)
TOL = {"f32": (1e-5, 1e-4), "bf16": (1e-2, 2e-2)}
SEEDS = (0, 1, 2, 3, 4)


def gpu_available() -> bool:
    return torch.cuda.is_available()


requires_gpu = pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a GPU")


def announce(*parts):
    """Name the case on stdout before the GPU step runs (it survives a lost
    process)."""
    print("[case]", *parts, flush=True)
    sys.stdout.flush()


def dev(t: fd.Tensor, device="cuda") -> torch.Tensor:
    if t is None:
        return None
    if t.dtype == "f32":
        return torch.from_numpy(np.ascontiguousarray(t.data)).to(device)
    if t.dtype == "u8":
        return torch.from_numpy(np.ascontiguousarray(t.data)).to(device)
    return torch.from_numpy(np.ascontiguousarray(t.data).view(np.int16)).view(
        torch.bfloat16).to(device)


def host64(x: torch.Tensor) -> np.ndarray:
    if x.dtype == torch.bfloat16:
        return x.detach().float().cpu().numpy().astype(np.float64)
    return x.detach().cpu().numpy().astype(np.float64)


def host_bits(x: torch.Tensor) -> np.ndarray:
    """Raw storage of a device tensor (bf16 -> uint16 bits, fp32 -> uint32 bits)."""
    if x.dtype == torch.bfloat16:
        return x.detach().cpu().view(torch.int16).numpy().view(np.uint16)
    return x.detach().cpu().view(torch.int32).numpy().view(np.uint32)


def assert_close(name, got, ref, atol, rtol):
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert got.shape == ref.shape, f"{name}: shape {got.shape} vs {ref.shape}"
    with np.errstate(invalid="ignore"):          # inf - inf where both are infinite
        err = np.abs(got - ref)
    ok = err <= atol + rtol * np.abs(ref)
    ok &= ~np.isnan(got)
    # identical infinities are equal
    ok |= (got == ref) & np.isinf(ref)
    if not ok.all():
        bad = np.argwhere(~ok)
        i = tuple(bad[0])
        worst = tuple(np.unravel_index(np.argmax(np.where(ok, -1, np.nan_to_num(err, nan=np.inf))),
                                       err.shape))
        raise AssertionError(
            f"{name}: {len(bad)} / {ok.size} elements out of tolerance (atol={atol}, rtol={rtol});"
            f" first at {i}: got {got[i]!r} ref {ref[i]!r}; worst at {worst}: got {got[worst]!r}"
            f" ref {ref[worst]!r}")


def rho(o32, r32, r64):
    """Gate-3 error ratio d_opt / d_ref (Eq. 4) with its degenerate case."""
    d_ref = np.max(np.abs(np.asarray(r32, np.float64) - r64))
    d_opt = np.max(np.abs(np.asarray(o32, np.float64) - r64))
    return rho_from_distances(d_opt, d_ref, np.max(np.abs(r32)))


def rho_from_distances(d_opt, d_ref, ref_scale):
    """Eq. 4 from the two largest deviations from the float64 result: the
    optimised output's (d_opt) and the unfused reference's (d_ref).  When the
    reference is itself within 1e-8 of the float64 result, the ratio is taken
    against the reference's magnitude instead (the degenerate case)."""
    if d_ref >= 1e-8:
        return float(d_opt / d_ref)
    return float(d_opt / max(ref_scale, 1e-12))


RHO_LIMIT = 10.0


def record_diag(case, **values):
    """Append {case, **values} to the FS_RHO_LOG file as one JSON line (when
    set) and print it."""
    path = os.environ.get("FS_RHO_LOG")
    if path:
        with open(path, "a") as f:
            f.write(json.dumps({"case": case, **{k: float(v) for k, v in values.items()}}) + "\n")
    print(f"[diag] {case}: {values}", flush=True)


def record_rho(case, d_opt, d_ref, ref_scale, limit=RHO_LIMIT):
    """Check the Gate-3 ratio of one case and, when FS_RHO_LOG names a file,
    append {case, rho, d_opt, d_ref} to it as one JSON line."""
    r = rho_from_distances(d_opt, d_ref, ref_scale)
    path = os.environ.get("FS_RHO_LOG")
    if path:
        with open(path, "a") as f:
            f.write(json.dumps({"case": case, "rho": r, "d_opt": float(d_opt),
                                "d_ref": float(d_ref)}) + "\n")
    print(f"[rho] {case}: {r:.4g} (d_opt {d_opt:.3g}, d_ref {d_ref:.3g})", flush=True)
    assert r <= limit, f"{case}: rho = {r:.3g} above {limit}"
    return r


class Guarded:
    """A [rows, ld] device buffer filled with a sentinel, with red zones before
    and after; ``view`` is the [rows, cols] window handed to a kernel."""

    def __init__(self, rows, cols, ld, dtype, device="cuda", pad=4096, offset=0):
        es = torch.tensor([], dtype=dtype).element_size()
        self.rows, self.cols, self.ld, self.pad, self.offset = rows, cols, ld, pad, offset
        n = pad + offset + max(rows * ld, 1) + pad
        self.base = torch.empty(n, dtype=dtype, device=device)
        self.base.view(torch.int16 if es == 2 else torch.int32).fill_(0x7A5C if es == 2 else 0x7A5C3E1F)
        self.snapshot = host_bits(self.base).copy()
        start = pad + offset
        self.view = self.base[start:start + rows * ld].view(rows, ld)[:, :cols] if rows else \
            self.base[start:start].view(0, cols)

    def check_untouched(self, name):
        now = host_bits(self.base)
        start = self.pad + self.offset
        written = np.zeros(now.shape, dtype=bool)
        for r in range(self.rows):
            written[start + r * self.ld:start + r * self.ld + self.cols] = True
        changed = (now != self.snapshot) & ~written
        assert not changed.any(), f"{name}: {changed.sum()} guard elements modified " \
                                  f"(first at {np.argwhere(changed)[0][0] - start})"


def bf16_ulp_close(name, got, ref_f64, ulps=1.0, atol=1e-6):
    """|got - ref| <= ulps * 2^-8 * |ref| + atol: round-to-nearest of an fp32
    result to bf16 is off by at most 2^-8 |ref| (half a unit in the last
    place); ``atol`` covers the fp32 error of results that cancel."""
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref_f64, np.float64)
    assert_close(name + " (bf16 rounding)", got, ref, atol, ulps * 2.0 ** -8)


def softmax_supplementary(name, got, ref, masked):
    """The contract atol (1e-2) exceeds every probability of a 4096-wide row,
    so also: about one bf16 rounding of the exact value, row sums near 1,
    masked entries exactly +0."""
    assert_close(name + " supplementary", got, ref, 1e-6, 8e-3)
    sums = got.sum(axis=1)
    live = ref.sum(axis=1) > 0
    np.testing.assert_allclose(sums[live], 1.0, atol=2e-2, err_msg=name + " row sums")
    assert np.all(got[masked] == 0.0), name + " masked entries not zero"
    assert not np.any(np.signbit(got[masked])), name + " masked entries are -0"


def f64_rows(t: fd.Tensor, r0: int, r1: int) -> np.ndarray:
    """Exact float64 values of rows r0..r1 of a host tensor."""
    return fd.Tensor(t.data[r0:r1], t.dtype).f64()


def max_abs_dev(a, b) -> float:
    """max |a - b|, with NaN counted as an infinite deviation."""
    d = np.abs(np.asarray(a, np.float64) - np.asarray(b, np.float64))
    return float(np.inf) if np.isnan(d).any() else float(d.max(initial=0.0))

