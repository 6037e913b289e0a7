"""bench.py's measurement plumbing on the CPU: the peak-rate library loads and rejects bad
arguments before any launch, and the rocprofv3 summariser turns kernel-trace and counter
csv files into a summary whose machine-readable record gives the sparse attention
kernel's HBM bytes (counter units scaled by a plain copy of known size)."""
import csv
import ctypes
import importlib.util
import os
import sys
import types

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _bench():
    spec = importlib.util.spec_from_file_location("bench_under_test", os.path.join(ROOT, "bench.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


def test_peaks_library_exports_and_validates():
    path = os.path.join(ROOT, "paper_2609_01925_amd", "libcrisp_peaks.so")
    if not os.path.exists(path):
        pytest.skip("libcrisp_peaks.so not built")
    lib = ctypes.CDLL(path)
    lib.crisp_peak_mfma_flop.restype = ctypes.c_double
    lib.crisp_peak_mfma_flop.argtypes = [ctypes.c_int, ctypes.c_int]
    assert lib.crisp_peak_mfma_flop(2048, 10) == 2048 * 4 * 10 * 4 * 32768.0
    lib.crisp_peak_mfma_bf16.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p]
    lib.crisp_peak_copy.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t, ctypes.c_int, ctypes.c_void_p]
    assert lib.crisp_peak_mfma_bf16(0, 10, ctypes.c_void_p(16), None) != 0      # no workgroups
    assert lib.crisp_peak_mfma_bf16(8, 10, None, None) != 0                     # no output
    lib.crisp_peak_mfma_bf16_toggling.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p,
                                                  ctypes.c_void_p]
    assert lib.crisp_peak_mfma_bf16_toggling(8, 12, ctypes.c_void_p(16), ctypes.c_void_p(16), None) != 0  # 12 % 8
    assert lib.crisp_peak_mfma_bf16_toggling(8, 16, ctypes.c_void_p(8), ctypes.c_void_p(16), None) != 0   # misaligned
    assert lib.crisp_peak_copy(ctypes.c_void_p(16), ctypes.c_void_p(32), 15, 1, None) != 0   # not 16-byte words
    assert lib.crisp_peak_copy(ctypes.c_void_p(8), ctypes.c_void_p(32), 16, 1, None) != 0    # misaligned
    lib.crisp_peak_lds_bytes_per_wave.restype = ctypes.c_double
    lib.crisp_peak_lds_bytes_per_wave.argtypes = [ctypes.c_int, ctypes.c_int]
    assert lib.crisp_peak_lds_bytes_per_wave(0, 10) == 10 * 8 * 64 * 16.0   # ds_read_b128
    assert lib.crisp_peak_lds_bytes_per_wave(1, 10) == 10 * 8 * 64 * 8.0    # ds_read_b64_tr_b16
    six = [ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p]
    lib.crisp_peak_lds_read.argtypes = six
    lib.crisp_peak_valu.argtypes = six
    assert lib.crisp_peak_lds_read(3, 8, 10, ctypes.c_void_p(16), ctypes.c_void_p(16), None) != 0   # no such kind
    assert lib.crisp_peak_lds_read(0, 8, 10, None, ctypes.c_void_p(16), None) != 0                  # no output
    assert lib.crisp_peak_valu(3, 8, 10, ctypes.c_void_p(16), ctypes.c_void_p(16), None) != 0       # no such kind
    assert lib.crisp_peak_valu(0, 0, 10, ctypes.c_void_p(16), ctypes.c_void_p(16), None) != 0       # no workgroups


def _write_csv(path, rows):
    with open(path, "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=list(rows[0]))
        w.writeheader()
        w.writerows(rows)


def test_summary_scales_counters_and_feeds_the_traffic_field(tmp_path, monkeypatch):
    b = _bench()
    attn = "void crisp::(anonymous namespace)::attn_kernel<128, false>(crisp::(anonymous namespace)::AttnArgs)"
    copy = "(anonymous namespace)::peak_copy(unsigned int const*, unsigned int*, unsigned long)"
    (tmp_path / "trace").mkdir()
    _write_csv(tmp_path / "trace" / "t_kernel_stats.csv", [
        {"Name": attn, "Calls": 3, "TotalDurationNs": 3e7, "AverageNs": 1e7, "Percentage": 90, "MinNs": 9e6,
         "MaxNs": 11e6, "StdDev": 0}])
    for counter, unit_attn, unit_copy in (("FETCH_SIZE", 500.0, 524288.0), ("WRITE_SIZE", 100.0, 1048576.0)):
        d = tmp_path / counter
        d.mkdir()
        rows = []
        for kid, (name, val) in enumerate(((attn, unit_attn), (attn, unit_attn * 3), (attn, unit_attn),
                                           (copy, unit_copy))):
            rows.append({"Correlation_Id": kid, "Dispatch_Id": kid, "Agent_Id": 1, "Queue_Id": 1, "Process_Id": 1,
                         "Thread_Id": 1, "Grid_Size": 1024, "Kernel_Id": kid, "Kernel_Name": name,
                         "Workgroup_Size": 256, "LDS_Block_Size": 0, "Scratch_Size": 0, "VGPR_Count": 0,
                         "Accum_VGPR_Count": 0, "SGPR_Count": 0, "Counter_Name": counter, "Counter_Value": val,
                         "Start_Timestamp": 0, "End_Timestamp": 1000000})
        _write_csv(d / f"{counter}_counter_collection.csv", rows)
    monkeypatch.setattr(b, "ROOT", str(tmp_path))
    os.makedirs(tmp_path / "paper_2609_01925_amd" / "csrc")
    with open(tmp_path / "paper_2609_01925_amd" / "csrc" / "attn.hip", "w") as f:
        f.write("// kernel source stand-in\n")
    args = types.SimpleNamespace(summarize=str(tmp_path), label="crisp_kernels_test-layer", command=["cmd a"])
    b.summarize(args)
    text = open(tmp_path / "profiles" / "crisp_kernels_test-layer.md").read()
    assert "| attn_kernel<128, false> | 3 | 10000.0 |" in text and "cmd a" in text
    # median over dispatches (500 units), scaled by the copy: 2 KiB per FETCH unit, 1 KiB per WRITE unit
    want = 500.0 * (1 << 30) / 524288.0 + 100.0 * (1 << 30) / 1048576.0
    h = b.src_hash(str(tmp_path / "paper_2609_01925_amd" / "csrc" / "attn.hip"))
    assert b.attn_traffic(h, "test-layer") == pytest.approx(want)
    assert b.attn_traffic("0" * 16, "test-layer") is None      # taken on another kernel source


def test_summary_splits_simd_cycles_into_mfma_and_valu_overlap(tmp_path, monkeypatch):
    """MFMA busy, VALU busy (issue of MFMAs taken out), both at once, VALU with the MFMA idle and
    neither, as fractions of GRBM_GUI_ACTIVE / 8 XCDs x 1024 SIMDs."""
    b = _bench()
    attn = "void crisp::(anonymous namespace)::attn_kernel<128, false>(crisp::(anonymous namespace)::AttnArgs)"
    grbm = 8 * 1000.0                      # 1000 cycles per XCD -> 1.024e6 SIMD-cycles
    simd = 1000.0 * 1024
    vals = {"GRBM_GUI_ACTIVE": grbm, "SQ_VALU_MFMA_BUSY_CYCLES": 0.7 * simd, "SQ_VALU_MFMA_COEXEC_CYCLES": 0.25 * simd,
            # quad-cycles: 0.4 of the SIMD-cycles of VALU work plus the issue of 1000 MFMAs (4 cycles each)
            "SQ_ACTIVE_INST_VALU": (0.4 * simd + 4 * 1000.0) / 4, "SQ_INSTS_MFMA": 1000.0,
            "SQ_WAIT_INST_ANY": 30.0, "SQ_WAVE_CYCLES": 100.0}
    d = tmp_path / "stall"
    d.mkdir()
    rows = [{"Kernel_Name": attn, "Counter_Name": c, "Counter_Value": v, "Start_Timestamp": 0,
             "End_Timestamp": 1000000} for c, v in vals.items()]
    _write_csv(d / "pmc_counter_collection.csv", rows)
    monkeypatch.setattr(b, "ROOT", str(tmp_path))
    os.makedirs(tmp_path / "paper_2609_01925_amd" / "csrc")
    args = types.SimpleNamespace(summarize=str(tmp_path), label="crisp_kernels_overlap", command=["cmd"])
    b.summarize(args)
    text = open(tmp_path / "profiles" / "crisp_kernels_overlap.md").read()
    # MFMA 70, VALU 40, together 25, VALU alone 15, neither 100 - 70 - 15 = 15, waiting 30
    assert "| attn_kernel<128, false> | 70.0 | 40.0 | 25.0 | 15.0 | 15.0 | 30.0 |" in text


def test_record_names_the_workload_manifest():
    b = _bench()
    m = b.manifest_id()
    from workloads import GEN_VERSION
    assert m["gen_version"] == GEN_VERSION
    assert m["manifests_sha"] == b.src_hash(os.path.join(ROOT, "tests", "golden", "manifests.json"))
