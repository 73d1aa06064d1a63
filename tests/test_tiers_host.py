"""Host tests of the bottleneck-tier classifier (Section 4.2): the four
tiers at and around their boundaries, SOL from scaled counters, and parsing
of rocprofv3 CSV output."""
import math

import pytest

from paper_2609_30059_amd import tiers as T


@pytest.mark.parametrize("mem,comp,want", [
    (0.81, 0.10, "near-optimal"), (0.10, 0.81, "near-optimal"), (0.95, 0.95, "near-optimal"),
    (0.80, 0.50, "memory-bound"),            # 80 % itself is not above the threshold
    (0.50, 0.80, "compute-bound"),
    (0.30, 0.30, "underutilized"), (0.0, 0.0, "underutilized"),
    (0.31, 0.30, "memory-bound"), (0.30, 0.31, "compute-bound"),
])
def test_tiers_and_boundaries(mem, comp, want):
    assert T.classify(mem, comp) == want


def test_tie_band_and_threshold_parameters():
    assert T.classify(0.31, 0.30, tie=0.02) == "underutilized"
    assert T.classify(0.40, 0.30, tie=0.02) == "memory-bound"
    assert T.classify(0.70, 0.1, near=0.6) == "near-optimal"
    for bad in (-0.1, float("nan"), float("inf")):
        with pytest.raises(ValueError):
            T.classify(bad, 0.1)
        with pytest.raises(ValueError):
            T.classify(0.1, bad)


def test_sol_from_scaled_counters():
    # 1 GiB read + 1 GiB written in 0.5 ms with counters reading half the
    # reads (scale 2) and all the writes: 4.295 TB/s = 53.7 % of 8 TB/s
    cyc = 2.4e9 * 5e-4                                  # engine cycles in 0.5 ms
    p = T.KernelProfile("k", duration_ns=5e5, fetch_kib=(1 << 20) / 2, write_kib=1 << 20,
                        raw={"SQ_INSTS_VALU": 0.1 * 1024 * cyc / T.VALU_CYCLES + 1000.0,
                             "SQ_INSTS_MFMA": 1000.0,      # counted among VALU, removed
                             "SQ_INSTS_SALU": 0.05 * 256 * cyc, "MfmaUtil": 2.0,
                             "VALUBusy": 130.0})          # context only, never the SOL
    mem, comp = p.sol(2.0, 1.0)
    assert math.isclose(mem, 2 * (1 << 30) / 5e-4 / 8e12)
    pp = p.pipes()
    assert math.isclose(pp["VALU"], 0.1) and math.isclose(pp["SALU"], 0.05)
    assert pp["MFMA"] == 0.02 and comp == pp["VALU"]
    assert T.classify(mem, comp) == "memory-bound"
    # a transcendental costs four FMA issue slots (2 and 8 cycles per wave64)
    assert (T.VALU_CYCLES, T.TRANS_CYCLES) == (2.0, 8.0)
    q = T.KernelProfile("t", duration_ns=5e5, raw={"SQ_INSTS_VALU": 1024 * cyc / 8,
                                                   "SQ_INSTS_VALU_TRANS_F32": 1024 * cyc / 8})
    assert math.isclose(q.pipes()["VALU"], 1.0)
    q4 = T.KernelProfile("f", duration_ns=5e5, raw={"SQ_INSTS_VALU": 4 * 1024 * cyc / 8})
    assert math.isclose(q4.pipes()["VALU"], 1.0)
    with pytest.raises(ValueError):
        T.KernelProfile("empty").sol()


def test_reads_rocprof_csv_and_calibrates(tmp_path):
    stats = tmp_path / "run_kernel_stats.csv"
    stats.write_text('"Name","Calls","TotalDurationNs","AverageNs","Percentage","MinNs","MaxNs"\n'
                     '"void fs::(anonymous namespace)::copy128_kernel(x)",2,600000,300000,50,1,1\n'
                     '"void fs::(anonymous namespace)::softmax_kernel<a>(b)",4,400000,100000,50,1,1\n')
    fetch = tmp_path / "fetch_counter_collection.csv"
    fetch.write_text("Dispatch_Id,Kernel_Name,Counter_Name,Counter_Value\n"
                     "1,void fs::(anonymous namespace)::copy128_kernel(x),FETCH_SIZE,524288\n"
                     "2,void fs::(anonymous namespace)::copy128_kernel(x),FETCH_SIZE,524288\n"
                     "3,void fs::(anonymous namespace)::softmax_kernel<a>(b),FETCH_SIZE,65536\n"
                     "4,void fs::(anonymous namespace)::softmax_kernel<a>(b),FETCH_SIZE,65536\n")
    write = tmp_path / "write_counter_collection.csv"
    write.write_text("Dispatch_Id,Kernel_Name,Counter_Name,Counter_Value\n"
                     "1,void fs::(anonymous namespace)::copy128_kernel(x),WRITE_SIZE,1048576\n"
                     "3,void fs::(anonymous namespace)::softmax_kernel<a>(b),WRITE_SIZE,65536\n")
    pipes = tmp_path / "pipes_counter_collection.csv"
    pipes.write_text("Dispatch_Id,Kernel_Name,Counter_Name,Counter_Value\n"
                     "3,void fs::(anonymous namespace)::softmax_kernel<a>(b),SQ_INSTS_VALU,3072000\n"
                     "4,void fs::(anonymous namespace)::softmax_kernel<a>(b),SQ_INSTS_VALU,4608000\n"
                     "3,void fs::(anonymous namespace)::softmax_kernel<a>(b),MfmaUtil,0\n"
                     "3,void fs::(anonymous namespace)::softmax_kernel<a>(b),VALUBusy,90\n")
    prof = {}
    T.read_kernel_stats(str(stats), prof)
    for f in (fetch, write, pipes):
        T.read_counters(str(f), prof)
    sm = prof["void fs::softmax_kernel<a>(b)"]
    assert sm.duration_ns == 100000 and sm.fetch_kib == 65536
    assert sm.raw["SQ_INSTS_VALU"] == 3840000             # per-dispatch average
    # 2 * 3.84e6 / (1024 * 2.4e9 * 1e-4) = 3.125 %
    fs_, ws_ = T.copy_scales(prof, "copy128_kernel", float(1 << 30), float(1 << 30))
    assert fs_ == 2.0 and ws_ == 1.0
    rows = T.table([sm], fs_, ws_)
    # (2 * 64 + 64) MiB in 100 us = 2013 GB/s = 25.2 % of 8 TB/s > VALU 3.125 %
    assert rows[2] == ("| void fs::softmax_kernel<a>(b) | 100.0 | 2013 | 25.2 | 3.1 (VALU) | 90.0 "
                       "| memory-bound |")
    with pytest.raises(ValueError):
        T.copy_scales(prof, "nothing", 1.0, 1.0)
    assert T.main(["--stats", str(stats), "--counters", str(fetch), str(write), str(pipes)]) == 0
