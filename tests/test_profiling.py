"""The counter summaries behind the bench's traffic and matrix-op figures, on small
hand-made rocprofv3 CSVs (no GPU)."""
import csv
import json

from paper_2606_13097_amd import profiling

FIELDS = ["Correlation_Id", "Dispatch_Id", "Agent_Id", "Queue_Id", "Process_Id", "Thread_Id", "Grid_Size",
          "Kernel_Id", "Kernel_Name", "Workgroup_Size", "LDS_Block_Size", "Scratch_Size", "VGPR_Count",
          "Accum_VGPR_Count", "SGPR_Count", "Counter_Name", "Counter_Value", "Start_Timestamp", "End_Timestamp"]


def _csv(path, rows):
    """rows: (dispatch, kernel, counter, value)"""
    with open(path, "w", newline="") as f:
        w = csv.DictWriter(f, FIELDS)
        w.writeheader()
        for d, k, c, v in rows:
            w.writerow({**{x: 0 for x in FIELDS}, "Dispatch_Id": d, "Kernel_Name": k, "Counter_Name": c,
                        "Counter_Value": v})
    return str(path)


class _Args:
    def __init__(self, **kw):
        self.__dict__.update(kw)


def test_traffic_calibrates_each_counter_by_the_copy(tmp_path):
    k = "fcg::graft_kernel<unsigned short, 128, false>(...)"
    fetch = _csv(tmp_path / "f.csv", [(1, k, "FETCH_SIZE", 999.0), (2, k, "FETCH_SIZE", 100.0),
                                      (3, "other", "FETCH_SIZE", 5.0), (4, k, "FETCH_SIZE", 300.0)])
    write = _csv(tmp_path / "w.csv", [(1, k, "WRITE_SIZE", 999.0), (2, k, "WRITE_SIZE", 50.0),
                                      (4, k, "WRITE_SIZE", 150.0)])
    # a 1 MiB copy reads half its bytes on FETCH_SIZE and all of them on WRITE_SIZE
    cf = _csv(tmp_path / "cf.csv", [(1, "__amd_rocclr_copyBuffer", "FETCH_SIZE", 512.0)])
    cw = _csv(tmp_path / "cw.csv", [(1, "__amd_rocclr_copyBuffer", "WRITE_SIZE", 1024.0)])
    d = profiling.traffic(_Args(kernel="graft_kernel", source="csrc/k_graft.hip", fetch=fetch, write=write,
                                copy_fetch=cf, copy_write=cw, copy_kernel="copyBuffer", copy_bytes=float(1 << 20),
                                skip=1, take=0, command="c"))
    assert d["dispatches"] == 2                               # first one skipped, other kernels ignored
    assert d["fetch_factor"] == 2.0 and d["write_factor"] == 1.0
    assert d["fetch_kib_avg"] == 200.0 and d["write_kib_avg"] == 100.0
    assert d["traffic_bytes_per_launch"] == 200.0 * 1024 * 2 + 100.0 * 1024
    assert d["source_sha256"] == profiling.source_sha256("csrc/k_graft.hip")
    json.dumps(d)


def test_mfma_ops_sum_rows_per_dispatch_and_take_the_gemm_unit(tmp_path):
    k = "fcg::attn_prefill_mfma_kernel<128, false, 4, 2>(...)"
    m = profiling.MOPS
    ops = _csv(tmp_path / "o.csv", [(5, k, m, 7.0), (6, k, m, 10.0), (6, k, m, 6.0), (7, k, m, 4.0),
                                    (8, "x", m, 100.0)])
    gemm = _csv(tmp_path / "g.csv", [(1, "Cijk_gemm", m, 1000.0), (2, "elementwise", m, 0.0)])
    d = profiling.mfma(_Args(kernel="attn_prefill_mfma_kernel", source="csrc/k_attn_mfma.hip", ops=ops,
                             gemm_ops=gemm, gemm_flops=512000.0, skip=1, take=1, command="c"))
    assert d["flops_per_op"] == 512.0
    assert d["dispatches"] == 1 and d["ops_avg"] == 16.0      # dispatch 6: two rows summed
    assert d["counter_flops_per_launch"] == 16.0 * 512.0


def test_source_hash_covers_every_listed_file():
    a = profiling.source_sha256("csrc/k_decode_mfma.hip")
    ab = profiling.source_sha256("csrc/k_decode_mfma.hip+csrc/decode_common.hpp")
    assert a != ab and len(ab) == 64


def test_bench_reports_counter_traffic_only_for_the_workload_it_was_taken_on():
    """The committed traffic summaries are per workload: a bench line of another workload
    carries no traffic figure rather than the 7B one."""
    import importlib.util
    import os
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    spec = importlib.util.spec_from_file_location("fcg_bench", os.path.join(root, "bench.py"))
    bench = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(bench)
    assert bench.measured_traffic("graft_long16k_traffic.json", "long16k") is None   # no such summary
    assert bench.measured_traffic("prefill_7b_traffic.json", "34b") is None
    assert bench.measured_traffic("graft_batched_traffic.json", "7b") is None
    got = bench.measured_traffic("prefill_7b_traffic.json", "7b")
    with open(os.path.join(root, "profiles", "prefill_7b_traffic.json")) as f:
        d = json.load(f)
    if d["source_sha256"] == profiling.source_sha256(d["source"]):
        assert got == int(round(d["traffic_bytes_per_launch"]))
    else:                                   # kernel changed since the counters were taken
        assert got is None
