"""Host tests of bench.py's profile tooling: the kernel-name patterns that tell
the bench kernels apart in rocprofv3 output, the compulsory-byte formulas, the
traffic.json writer and the duration report."""
import importlib.util
import json
import os

import pytest

from paper_2609_30059_amd import tiers as T

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
_spec = importlib.util.spec_from_file_location("bench", os.path.join(ROOT, "bench.py"))
bench = importlib.util.module_from_spec(_spec)
_spec.loader.exec_module(bench)

# kernel names as rocprofv3 prints them (anonymous namespace removed), one per
# bench kernel, plus library and runtime kernels that must match nothing
NAMES = {
    "pw_256x1024": "void fs::pointwise_kernel<float, 1, true, true, 1>(float const*, long, float const*, float const*, long, float*, long, long, int, float, int)",
    "pw_262144x1024": "void fs::pointwise_kernel<float, 1, true, true, 4>(float const*, long, float const*, float const*, long, float*, long, long, int, float, int)",
    "sm_8192x4096": "void fs::softmax_kernel<unsigned short, unsigned short, true, 2, 32, true, 1, 1>(unsigned short const*, long)",
    "ln_16384x4096": "void fs::layernorm_kernel<unsigned short, true, false, 2, 32, true, 1, 1>(unsigned short const*, long)",
    "ep_8192x8192": "void fs::epilogue_lds_kernel<unsigned short, unsigned short, 2, 16, 2, 16, true>(unsigned short const*, long)",
    "blk_ln1": "void fs::layernorm_wave_kernel<unsigned short, false, false, 16, 1>(unsigned short const*, long)",
    "blk_sm": "void fs::softmax_kernel<unsigned short, unsigned short, false, 1, 8, true, 4, 2>(unsigned short const*, long)",
    "blk_ln2": "void fs::layernorm_wave_kernel<unsigned short, true, false, 16, 1>(unsigned short const*, long)",
    "blk_gelu": "void fs::pointwise_kernel<unsigned short, 1, false, true, 4>(unsigned short const*, long)",
    "blk_res": "void fs::pointwise_flat_kernel<unsigned short, 0, true, 4>(unsigned short const*, long)",
    "copy_1GiB": "void fs::copy128_kernel<4>(unsigned int __vector(4) const*, unsigned int __vector(4)*, long)",
}
OTHERS = [
    "void fs::layernorm_kernel<unsigned short, false, false, 1, 16, true, 4, 1>(unsigned short const*, long)",
    "void fs::pointwise_kernel<unsigned short, 0, true, true, 4>(unsigned short const*, long)",
    "void fs::copy_strided_kernel<unsigned int __vector(4), 4>(unsigned int __vector(4) const*, long)",
    "Cijk_Ailk_Bljk_BBS_BH_Bias_HA_S_SAV_UserArgs_MT256x256x64_MI16x16x1_SN_LDSB1",
    "__amd_rocclr_copyBuffer",
]


def test_every_bench_kernel_matches_exactly_one_name():
    names = list(NAMES.values()) + OTHERS
    for label in bench.KERNEL_PATTERNS:
        assert bench._match(names, label) == NAMES[label], label
    assert set(bench.KERNEL_PATTERNS) == set(NAMES)
    with pytest.raises(ValueError):       # two candidates for one label
        bench._match([NAMES["blk_ln1"], NAMES["blk_ln1"] + " "], "blk_ln1")


def test_compulsory_bytes():
    T_, H, F = 32 * 512, 1024, 4096
    live = sum(p + 1 for p in range(512))                       # lower triangle with diagonal
    assert live == 512 * 513 // 2
    assert bench.STEP_BYTES["blk_sm"] == 32 * 16 * (live * 2 + 512 * 512 * 2)
    assert bench.STEP_BYTES["blk_ln2"] == T_ * H * 2 * 4 + 2 * H * 2   # x, res in; y, res out
    assert bench.STEP_BYTES["blk_gelu"] == T_ * F * 2 * 2 + F * 2
    assert bench.STEP_BYTES["ep_8192x8192"] == 8192 * 8192 * 2 + 8192 * 2 + 8192 * 4 + 8192 * 4
    assert bench.STEP_BYTES["copy_1GiB"] == 2 << 30
    assert bench.STEP_BYTES["pw_262144x1024"] == 3 * (1 << 30) + 4096
    assert set(bench.KIND) == set(bench.STEP_BYTES) - {"copy_1GiB"}


def _counters(path, counter, per_label):
    with open(path, "w") as f:
        f.write("Dispatch_Id,Kernel_Name,Counter_Name,Counter_Value\n")
        for i, (label, v) in enumerate(per_label.items()):
            f.write(f'{i},"{NAMES[label]}",{counter},{v}\n')


def test_write_traffic_scales_by_the_copy(tmp_path, monkeypatch):
    monkeypatch.setattr(bench, "TRAFFIC_FILE", str(tmp_path / "traffic.json"))
    # the copy moves 1 GiB each way; FETCH_SIZE reads half of it, WRITE_SIZE all
    fetch = {"copy_1GiB": 524288, "ln_16384x4096": 131072, "ep_8192x8192": 65536}
    write = {"copy_1GiB": 1048576, "ln_16384x4096": 262144, "ep_8192x8192": 32}
    _counters(tmp_path / "f.csv", "FETCH_SIZE", fetch)
    _counters(tmp_path / "w.csv", "WRITE_SIZE", write)
    out = bench.write_traffic(str(tmp_path / "f.csv"), str(tmp_path / "w.csv"), "abc", "F", "W")
    assert out["fetch_scale"] == 2.0 and out["write_scale"] == 1.0
    assert out["ln_16384x4096"]["bytes_per_launch"] == (2 * 131072 + 262144) * 1024
    assert out["ep_8192x8192"]["bytes_per_launch"] == (2 * 65536 + 32) * 1024
    assert out["ln_16384x4096"]["source_hash"] == bench.source_hash("ln")
    assert "pw_256x1024" not in out and "copy_1GiB" not in out
    assert json.load(open(tmp_path / "traffic.json"))["measured_at"] == "abc"


def test_report_trace(tmp_path, capsys):
    p = tmp_path / "s.csv"
    p.write_text('"Name","Calls","TotalDurationNs","AverageNs","Percentage","MinNs","MaxNs"\n'
                 f'"{NAMES["ln_16384x4096"]}",4,352000,88000,80,87000,89000\n'
                 f'"{OTHERS[1]}",1,88000,88000,20,88000,88000\n')
    bench.report_trace(str(p))
    rows = [l for l in capsys.readouterr().out.splitlines() if l.startswith("| ln_16384x4096")]
    gbs = bench.STEP_BYTES["ln_16384x4096"] / 88000
    assert rows == [f"| ln_16384x4096 | 4 | 88.00 | 87.00 | 89.00 | 80.0 | {gbs:.0f} | "
                    f"{100 * gbs / 8000:.1f} |"]


def test_report_trace_every_library_kernel(tmp_path, capsys):
    p = tmp_path / "s.csv"
    p.write_text('"Name","Calls","TotalDurationNs","AverageNs","Percentage","MinNs","MaxNs"\n'
                 '"void fs::(anonymous namespace)::softmax_cached_kernel<unsigned short, true>'
                 '(unsigned short const*, long)",3,300000,100000,60,90000,110000\n'
                 '"void at::native::fill_kernel<float>(float*)",2,200000,100000,40,100000,100000\n')
    bench.report_trace(str(p), every=True)
    out = capsys.readouterr().out.splitlines()
    assert out[2] == "| `softmax_cached_kernel<unsigned short, true>` | 3 | 100.00 | 90.00 | 110.00 | 60.0 |"
    assert len(out) == 3                      # torch's own kernels are not listed


def test_long_row_widths_span_every_long_row_path():
    # the 16-wave register rungs, the row cache with and without a tail
    w = bench.LONG_ROW_WIDTHS
    assert any(16384 < c <= 32768 for c in w)
    assert any(32768 < c <= 65536 for c in w)
    assert any(c > 65536 for c in w)
    assert any(c % 8 for c in w)              # element-wise loads (not whole 16-byte vectors)
    assert sum(c % 8 == 0 for c in w) >= 6    # the 16-byte path at every other width


def test_tier_labels():
    assert T.label("void fs::layernorm_kernel<unsigned short, true, false>(unsigned short const*, long)") \
        == "layernorm_kernel<unsigned short, true, false>"
    assert T.label("void fs::copy_strided_kernel<unsigned int __vector(4), 4>(int)") \
        == "copy_strided_kernel<unsigned int __vector(4), 4>"
    long_name = "Cijk_" + "A" * 100
    assert T.label(long_name) == long_name[:64] + "..."
    assert T.label("__amd_rocclr_copyBuffer") == "__amd_rocclr_copyBuffer"


def test_more_than_one_gpu_exits_with_the_reason():
    import subprocess
    import sys
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU only" in r.stderr and r.stdout == ""


def _trace(path, seq):
    with open(path, "w") as f:
        f.write("Kernel_Name,Start_Timestamp,End_Timestamp\n")
        t = 0
        for name, us in seq:
            f.write(f'"{name}",{t},{t + int(us * 1000)}\n')
            t += int(us * 1000) + 5000


def test_report_floor_splits_the_dispatches_by_order(tmp_path, capsys):
    scrub = "void fs::reduce_kernel<unsigned short, 0, 8, 4, true, false>(unsigned short const*, long)"
    copy = NAMES["copy_1GiB"]
    order = [(copy, 12.0), (NAMES["blk_ln1"], 13.0), (copy, 17.0), (NAMES["blk_res"], 16.0),
             (copy, 23.0), (NAMES["blk_ln2"], 23.5)]
    seq = []
    for rep in range(3):                        # the first repetition is the warm-up
        for name, us in order:
            seq.append((scrub, 100.0))
            seq.append((name, us * 10 if rep == 0 else us + rep * 0.1))
    p = tmp_path / "trace.csv"
    _trace(p, seq)
    bench.report_floor(str(p))
    out = capsys.readouterr().out
    rows = {l.split("|")[1].strip(): l.split("|") for l in out.splitlines()[2:]}
    assert float(rows["blk_ln1"][3]) == pytest.approx(13.2)          # median of 13.1, 13.2
    assert rows["blk_ln1"][8].strip() == f"{13.2 / 12.2:.3f}"         # against copy_64MiB
    assert rows["copy_96MiB"][2].strip() == "2"
    # a dispatch out of order is an error, not a silent relabelling
    bad = seq[:]
    bad[3], bad[7] = bad[7], bad[3]
    _trace(p, bad)
    with pytest.raises(ValueError):
        bench.report_floor(str(p))


def test_report_floors_pairs_each_kernel_with_its_floor(tmp_path, capsys):
    scrub = "void fs::reduce_kernel<unsigned short, 0, 8, 4, true, false>(unsigned short const*, long)"
    floor = ("void (anonymous namespace)::floor_rows_kernel<2, 1, 4, 1, 1, 1, false, false>"
             "(unsigned int __vector(4) const*, long)")
    # the setup launches every step kernel (and a block forward) before the
    # measured repetitions; those dispatches are not part of the table
    seq = [(NAMES[n], 50.0) for n in bench.FLOOR_SHAPES]
    for rep in range(4):                        # the first repetition is the warm-up
        for i, name in enumerate(bench.FLOOR_SHAPES):
            seq.append((scrub, 150.0))
            seq.append((NAMES[name], 1000.0 if rep == 0 else 20.0 + i + rep * 0.1))
            seq.append((scrub, 150.0))
            seq.append((floor, 1000.0 if rep == 0 else 10.0 + i))
    p = tmp_path / "trace.csv"
    _trace(p, seq)
    bench.report_floors(str(p))
    out = capsys.readouterr().out
    rows = {l.split("|")[1].strip(): [c.strip() for c in l.split("|")] for l in out.splitlines()[2:]}
    assert set(rows) == set(bench.FLOOR_SHAPES)
    ln = rows["ln_16384x4096"]                  # shape 3: kernel 23.2 (median of 23.1..23.3), floor 13
    assert float(ln[3]) == pytest.approx(23.2) and float(ln[4]) == pytest.approx(13.0)
    assert ln[5] == f"{23.2 / 13.0:.3f}"
    assert int(ln[2]) == bench.STEP_BYTES["ln_16384x4096"]
    # a floor where a kernel belongs is an error, not a silent relabelling
    bad = seq[:]
    k = len(bench.FLOOR_SHAPES) + 4 * 3 + 1     # the kernel of the fourth case, first repetition
    bad[k] = (floor, 20.0)
    _trace(p, bad)
    with pytest.raises(ValueError):
        bench.report_floors(str(p))


def test_access_floor_refuses_bad_arguments_before_any_launch():
    """The access-floor library checks shapes, buffer sizes, alignment and the
    CU count on the host and launches nothing when one is wrong (the pointers
    below are never dereferenced)."""
    import ctypes
    import subprocess
    from paper_2609_30059_amd import build as B
    lib = ctypes.CDLL(B.LIB_ACCESS_FLOOR)
    f = lib.fsx_access_floor
    sz = ctypes.c_size_t
    f.argtypes = [ctypes.c_int, ctypes.c_void_p, sz, ctypes.c_void_p, sz, ctypes.c_void_p, sz,
                  ctypes.c_void_p, sz, ctypes.c_int, ctypes.c_void_p]
    f.restype = ctypes.c_int
    lib.fsx_access_floor_shapes.restype = ctypes.c_int
    assert lib.fsx_access_floor_shapes() == len(bench.FLOOR_SHAPES)
    p, big = 1 << 20, 1 << 31                   # a 16-byte-aligned stand-in address, ample sizes
    ln = bench.FLOOR_SHAPES.index("ln_16384x4096")
    need = 16384 * 4096 * 2
    assert f(-1, p, big, p, big, p, big, p, big, 256, None) == -2
    assert f(len(bench.FLOOR_SHAPES), p, big, p, big, p, big, p, big, 256, None) == -2
    assert f(ln, p, big, p, big, p, big, p, big, 0, None) == -3
    assert f(ln, None, big, p, big, p, big, p, big, 256, None) == -1
    assert f(ln, p + 8, big, p, big, p, big, p, big, 256, None) == -1      # misaligned
    assert f(ln, p, need - 16, p, big, p, big, p, big, 256, None) == -1    # x too small
    assert f(ln, p, need, p, need, p, need, None, 0, 256, None) == -1      # residual_out missing
    ep = bench.FLOOR_SHAPES.index("ep_8192x8192")
    assert f(ep, p, 8192 * 8192 * 2, None, 0, p, 8, None, 0, 256, None) == -1   # out < 16 bytes
    out = subprocess.run(["nm", "-D", "--defined-only", B.LIB_ACCESS_FLOOR], capture_output=True,
                         text=True).stdout
    assert {l.split()[-1] for l in out.splitlines() if " T " in l} == {
        "fsx_access_floor", "fsx_access_floor_shapes", "fsx_access_floor_bytes"}


def test_access_floors_move_the_sub_kernels_bytes():
    """Each floor reads and writes the compulsory bytes of the step launch it
    stands in for: exactly, less the broadcast vectors (bias, gamma/beta,
    column scales) and the epilogue's row sums it does not move; the causal
    shape reads whole 16-byte vectors up to each row's diagonal, 1.4 % above
    the element count of the lower triangle."""
    import ctypes
    from paper_2609_30059_amd import build as B
    lib = ctypes.CDLL(B.LIB_ACCESS_FLOOR)
    lib.fsx_access_floor_bytes.restype = ctypes.c_int64
    lib.fsx_access_floor_bytes.argtypes = [ctypes.c_int]
    small = {"pw_256x1024": 1024 * 4, "pw_262144x1024": 1024 * 4, "ln_16384x4096": 2 * 4096 * 2,
             "ep_8192x8192": 8192 * (2 + 4) + 8192 * 4, "blk_ln1": 2 * 1024 * 2,
             "blk_ln2": 2 * 1024 * 2, "blk_gelu": 4096 * 2}
    for i, name in enumerate(bench.FLOOR_SHAPES):
        got = lib.fsx_access_floor_bytes(i)
        want = bench.STEP_BYTES[name] - small.get(name, 0)
        if name == "blk_sm":
            assert want < got < want * 1.015, (name, got, want)
        else:
            assert got == want, (name, got, want)
    assert lib.fsx_access_floor_bytes(-1) == -1
    assert lib.fsx_access_floor_bytes(len(bench.FLOOR_SHAPES)) == -1


def test_short_kernel_name_keeps_template_arguments():
    n = ("void fs::(anonymous namespace)::softmax_cached_kernel<unsigned short, unsigned short, "
         "true, false, true, 32, 32, false>(unsigned short const*, long, float)")
    assert bench.short_kernel_name(n) == ("softmax_cached_kernel<unsigned short, unsigned short, "
                                          "true, false, true, 32, 32, false>")


def test_report_counters_groups_launches_and_averages(tmp_path, capsys):
    hdr = ("Correlation_Id,Dispatch_Id,Agent_Id,Queue_Id,Process_Id,Thread_Id,Grid_Size,Kernel_Id,"
           "Kernel_Name,Workgroup_Size,LDS_Block_Size,Scratch_Size,VGPR_Count,Accum_VGPR_Count,"
           "SGPR_Count,Counter_Name,Counter_Value,Start_Timestamp,End_Timestamp\n")
    k = "void fs::(anonymous namespace)::epilogue_lds_kernel<unsigned short, 2>(unsigned short const*)"
    lds = tmp_path / "lds.csv"
    occ = tmp_path / "occ.csv"
    with open(lds, "w") as f:
        f.write(hdr)
        for d, (act, bank) in enumerate([(1000, 10), (3000, 30)]):
            for c, v in (("SQ_LDS_IDX_ACTIVE", act), ("SQ_LDS_BANK_CONFLICT", bank)):
                f.write(f'1,{d},1,1,1,1,262144,3,"{k}",512,0,0,28,0,32,{c},{v},0,1\n')
        f.write(f'1,9,1,1,1,1,4096,3,"__amd_rocclr_fillBuffer",256,0,0,8,0,16,SQ_LDS_IDX_ACTIVE,5,0,1\n')
    with open(occ, "w") as f:
        f.write(hdr)
        for d, v in enumerate([50.0, 100.0]):
            f.write(f'1,{10 + d},1,1,1,1,262144,3,"{k}",512,0,0,28,0,32,OccupancyPercent,{v},0,1\n')
    bench.report_counters([str(lds), str(occ)])
    out = capsys.readouterr().out.splitlines()
    rows = [l for l in out if l.startswith("| `")]
    assert len(rows) == 1                                     # runtime kernels are skipped
    cells = [c.strip() for c in rows[0].split("|")]
    assert cells[2] == "512 x 512" and cells[3] == "28"
    assert cells[5] == "24.0 (75 %)"                          # mean occupancy 75 % of 32 waves
    assert cells[7] == "2000" and cells[8] == "20" and cells[9] == "0.0100"


def test_report_context_takes_the_timed_blocks(tmp_path, capsys):
    ep = NAMES["ep_8192x8192"]
    rowsum = "void fs::reduce_kernel<unsigned short, 0, 1, 16, 4, 1>(unsigned short const*, long)"
    other = NAMES["ln_16384x4096"]
    pause = int(bench.CONTEXT_PAUSE_S * 1e9)
    t = 0
    # setup launches first, then a warm-up and a timed block per context; step
    # contexts report only their last CONTEXT_STEP_TAIL launches
    blocks = [[(ep, 30.0), (other, 90.0)]]
    for i, (_, kind, reps) in enumerate(bench.CONTEXTS):
        name = ep if kind == "ep" else rowsum
        blocks.append([(name, 99.0)] * 3)
        head = reps - bench.CONTEXT_STEP_TAIL if reps == bench.CONTEXT_STEPS else 0
        blocks.append([(other, 90.0), (name, 50.0)] * head
                      + [(other, 90.0), (name, 20.0 + i)] * (reps - head))
    with open(tmp_path / "t.csv", "w") as f:
        f.write("Kernel_Name,Start_Timestamp,End_Timestamp\n")
        for b in blocks:
            t += pause
            for name, us in b:
                f.write(f'"{name}",{t},{t + int(us * 1000)}\n')
                t += int(us * 1000) + 3000
    bench.report_context(str(tmp_path / "t.csv"))
    out = [l for l in capsys.readouterr().out.splitlines()[2:]]
    assert len(out) == len(bench.CONTEXTS)
    for i, (line, (_, kind, reps)) in enumerate(zip(out, bench.CONTEXTS)):
        cells = [c.strip() for c in line.split("|")]
        n = bench.CONTEXT_STEP_TAIL if reps == bench.CONTEXT_STEPS else reps
        assert cells[2] == ("epilogue" if kind == "ep" else "row sum")
        assert cells[3] == str(n) and float(cells[4]) == 20.0 + i


def test_timing_events_use_the_runtime_torch_loaded():
    """The timing-only events resolve HIP from the runtime torch has already
    loaded (the same one that owns torch's streams), never a second copy."""
    import ctypes
    import torch  # noqa: F401
    from paper_2609_30059_amd import timing
    if torch.cuda.is_available():
        ev = bench.TimingEvent()
        assert ev.ev.value
    else:
        with pytest.raises(RuntimeError, match="hipEventCreateWithFlags"):
            bench.TimingEvent()
    addr = ctypes.cast(timing._HIP.hipEventCreateWithFlags, ctypes.c_void_p).value
    spans = []
    for line in open("/proc/self/maps").read().splitlines():
        parts = line.split()
        if len(parts) >= 6 and "libamdhip64" in parts[5]:
            lo, hi = (int(v, 16) for v in parts[0].split("-"))
            spans.append((lo, hi, parts[5]))
    owners = {p for lo, hi, p in spans if lo <= addr < hi}
    assert len({p for _, _, p in spans}) == 1, spans
    assert len(owners) == 1


def test_report_transient_pairs_steps_with_clocks(tmp_path, capsys):
    """Warm-up steps before the first probe fold into step 0 (its last
    launches count); each probe closes a step; the dip steps are those below
    90 % of the median clock of the last 60 steps."""
    order = ["pw_256x1024", "sm_8192x4096", "ln_16384x4096", "ep_8192x8192", "blk_ln1",
             "blk_sm", "blk_ln2", "blk_gelu", "blk_res"]
    probe = "void (anonymous namespace)::clock_probe_kernel(unsigned long long*, int, int)"
    steps = 80
    clocks = [1500 if 2 <= s < 12 else 2000 for s in range(steps)]
    t = 0
    with open(tmp_path / "t.csv", "w") as f:
        f.write("Kernel_Name,Start_Timestamp,End_Timestamp\n")
        for _ in range(3):                          # warm-up steps, no probe
            for k in order:
                f.write(f'"{NAMES[k]}",{t},{t + 99000}\n')
                t += 100000
        t += 500_000_000
        for s in range(steps):
            for k in order:
                us = 30.0 if (k == "ep_8192x8192" and clocks[s] < 2000) else 20.0
                f.write(f'"{NAMES[k]}",{t},{t + int(us * 1000)}\n')
                t += int(us * 1000) + 1000
            f.write(f'"{probe}",{t},{t + 7000}\n')
            t += 8000
    with open(tmp_path / "log", "w") as f:
        for s in range(steps):
            f.write(f"clock step {s} {clocks[s]} MHz\n")
    tab = bench.transient_table(str(tmp_path / "t.csv"), str(tmp_path / "log"))
    assert len(tab) == steps
    assert tab[0][1] == 0.0 and tab[0][3]["ep_8192x8192"] == 20.0
    assert [row[2] for row in tab] == clocks
    bench.report_transient(str(tmp_path / "t.csv"), str(tmp_path / "log"))
    out = capsys.readouterr().out
    assert "sustained clock (median of the last 60 steps): 2000 MHz; 10 steps below" in out
    ep_line = [l for l in out.splitlines() if l.startswith("| ep_8192x8192 |")][0]
    cells = [c.strip() for c in ep_line.split("|")]
    assert float(cells[2]) == 30.0 and float(cells[3]) == 20.0 and float(cells[4]) == 1.5


def test_clock_probe_refuses_bad_arguments_before_any_launch():
    """The engine-clock probe checks its arguments on the host and launches
    nothing for a null buffer, a slot out of range, an empty grid or a
    negative trip count (the pointer below is never dereferenced)."""
    import ctypes
    import subprocess
    from paper_2609_30059_amd import build as B
    lib = ctypes.CDLL(B.LIB_CLOCK_PROBE)
    f = lib.fsx_clock_probe
    f.argtypes = [ctypes.c_void_p, ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int,
                  ctypes.c_void_p]
    f.restype = ctypes.c_int
    fake = ctypes.c_void_p(64)
    assert f(None, 0, 1, 1, 1, None) == -1
    assert f(fake, -1, 4, 1, 1, None) == -1
    assert f(fake, 4, 4, 1, 1, None) == -1
    assert f(fake, 0, 4, 0, 1, None) == -1
    assert f(fake, 0, 4, 1, -1, None) == -1
    out = subprocess.run(["nm", "-D", "--defined-only", B.LIB_CLOCK_PROBE], capture_output=True,
                         text=True).stdout
    assert {l.split()[-1] for l in out.splitlines() if " T " in l} == {"fsx_clock_probe"}
