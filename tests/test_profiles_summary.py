"""Host logic of the rocprofv3 summaries (CPU): kernel-name mapping, the copy
calibration of the byte counters and the executed-MFMA ratio, on small
hand-written CSV files in the layout rocprofv3 writes."""
import csv
import json
import os
import sys

import pytest

from paper_2607_05380_amd import profiles_summary as ps


@pytest.mark.parametrize("kernel,name", [
    ("_ZN7tabpack12_GLOBAL__N_117gemm_kernel_smallIDF16bLi1ELi1ELi3EEEvNS_8GemmArgsE", "gemm_bf16_rmaj_rmaj_dw"),
    ("void tabpack::(anonymous namespace)::gemm_kernel_small<__bf16, 0, 1, 3>(tabpack::GemmArgs)",
     "gemm_bf16_kmaj_rmaj_dw"),
    ("_ZN7tabpack12_GLOBAL__N_116gemm_kernel_tallILi0ELi1ELi2EEEvNS_8GemmArgsE", "gemm_bf16_kmaj_rmaj_dx"),
    ("void tabpack::(anonymous namespace)::gemm_kernel<float, 0, 1, 4>(tabpack::GemmArgs)", "gemm_f32_kmaj_rmaj_ns"),
    ("_ZN7tabpack12_GLOBAL__N_111gemm_kernelIDF16bLi0ELi0ELi1EEEvNS_8GemmArgsE", "gemm_bf16_kmaj_kmaj_fwd_eval"),
    ("_ZN7tabpack12_GLOBAL__N_120gemm_kernel_emb_wideILi0EEEvNS_8GemmArgsE", "gemm_bf16_emb_kmaj_fwd"),
    ("void tabpack::(anonymous namespace)::gemm_kernel_emb_wide<1>(tabpack::GemmArgs)", "gemm_bf16_emb_kmaj_fwd_eval"),
    ("void tabpack::(anonymous namespace)::muon_update_kernel<__bf16>(...)", "muon_update"),
    ("void tabpack::(anonymous namespace)::select_partial_kernel(...)", "select_partial"),
    ("void at::native::elementwise_kernel<128, 4>(...)", None),
])
def test_short_name(kernel, name):
    assert ps.short_name(kernel) == name


def _write_pmc(d, rows):
    os.makedirs(d, exist_ok=True)
    with open(os.path.join(d, "run_counter_collection.csv"), "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=["Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value"])
        w.writeheader()
        for r in rows:
            w.writerow(dict(zip(["Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value"], r)))


DW = "_ZN7tabpack12_GLOBAL__N_117gemm_kernel_smallIDF16bLi1ELi1ELi3EEEvNS_8GemmArgsE"
COPY = "__amd_rocclr_copyBuffer"
STREAM = "tabpack::(anonymous namespace)::stream_copy_kernel(float vector[4] const*, float vector[4]*, long)"


def test_traffic_scales_by_the_stream_copy(tmp_path, monkeypatch):
    # the library's streaming copy reads FETCH 2x and WRITE 1.5x of its 256 MiB;
    # a kernel's counters are divided by those factors (raw values kept too);
    # values per XCC row are summed per dispatch; torch's copy is only reported
    mib = 1024
    _write_pmc(tmp_path / "f", [(1, STREAM, "FETCH_SIZE", 512 * mib), (2, DW, "FETCH_SIZE", 600),
                                (2, DW, "FETCH_SIZE", 400), (3, DW, "FETCH_SIZE", 3000),
                                (4, COPY, "FETCH_SIZE", 256 * mib)])
    _write_pmc(tmp_path / "w", [(1, STREAM, "WRITE_SIZE", 384 * mib), (2, DW, "WRITE_SIZE", 150),
                                (3, DW, "WRITE_SIZE", 450), (4, COPY, "WRITE_SIZE", 512 * mib)])
    out = tmp_path / "t"
    monkeypatch.setattr(sys, "argv", ["ps", "traffic", str(tmp_path / "f"), str(tmp_path / "w"), "wl", str(out)])
    ps.main()
    rec = json.load(open(str(out) + ".json"))
    k = rec["kernels"]["gemm_bf16_rmaj_rmaj_dw"]
    assert rec["copy_factor"] == {"fetch": 2.0, "write": 1.5}
    assert rec["torch_copy_factor"] == {"fetch": 1.0, "write": 2.0}
    assert k["dispatches"] == 2
    assert k["fetch_bytes"] == pytest.approx((1000 + 3000) / 2 * 1024 / 2.0)
    assert k["write_bytes"] == pytest.approx((150 + 450) / 2 * 1024 / 1.5)
    assert k["write_raw_bytes"] == pytest.approx((150 + 450) / 2 * 1024)


def test_busy_time_is_the_union_of_intervals(tmp_path):
    assert ps.busy_ns([(0, 10), (5, 12), (20, 25), (24, 30), (40, 41)]) == 12 + 10 + 1
    assert ps.busy_ns([]) == 0
    d = tmp_path / "k"
    os.makedirs(d)
    with open(d / "run_kernel_trace.csv", "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=["Kernel_Name", "Start_Timestamp", "End_Timestamp"])
        w.writeheader()
        for a, b in ((100, 200), (150, 260), (300, 310)):
            w.writerow({"Kernel_Name": DW, "Start_Timestamp": a, "End_Timestamp": b})
        w.writerow({"Kernel_Name": COPY, "Start_Timestamp": 0, "End_Timestamp": 1000})
    assert ps.trace_busy(str(d)) == {"gemm_bf16_rmaj_rmaj_dw": (3, 170)}


def test_mfma_ratio(tmp_path, monkeypatch):
    _write_pmc(tmp_path / "m", [(1, DW, "SQ_INSTS_VALU_MFMA_MOPS_BF16", 1000), (2, DW, "SQ_INSTS_VALU_MFMA_MOPS_BF16",
                                                                              1400)])
    log = tmp_path / "bench.log"
    log.write_text("[bench] text\n" + json.dumps({"kernels": [{"name": "gemm_bf16_rmaj_rmaj_dw",
                                                                "flops_per_launch": 1200 * 512 / 1.2}]}) + "\n")
    out = tmp_path / "m.md"
    monkeypatch.setattr(sys, "argv", ["ps", "mfma", str(tmp_path / "m"), str(log), "wl", str(out)])
    ps.main()
    text = out.read_text()
    assert "| gemm_bf16_rmaj_rmaj_dw | 2 |" in text and "1.200 |" in text
    assert "executed / algorithmic = 1.200" in text
