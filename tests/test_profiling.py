"""The profiling helpers: traffic records scale counters by the copy
calibration, belong to the kernel sources they were made from, and the
benchmark ignores them once those sources change."""
import json

from paper_2606_00746_amd import profiling

HEADER = ('"Correlation_Id","Dispatch_Id","Agent_Id","Queue_Id","Process_Id","Thread_Id",'
          '"Grid_Size","Kernel_Id","Kernel_Name","Workgroup_Size","LDS_Block_Size",'
          '"Scratch_Size","VGPR_Count","Accum_VGPR_Count","SGPR_Count","Counter_Name",'
          '"Counter_Value","Start_Timestamp","End_Timestamp"\n')


def _csv(path, counter, rows):
    with open(path, "w") as f:
        f.write(HEADER)
        for i, (kernel, value) in enumerate(rows):
            f.write(f'{i},{i},"Agent 1",1,1,1,64,1,"{kernel}",256,0,0,8,0,16,"{counter}",{value},0,1\n')


def test_traffic_record_scales_by_copy(tmp_path):
    copy = "__amd_rocclr_copyBuffer(char const*, char*)"
    fwd = "void gspn::(anonymous namespace)::fwd_med_kernel<64, 64>(int)"
    bwd = "void gspn::(anonymous namespace)::bwd_med_kernel<64, 64, 1>(int)"
    dws = "void gspn::(anonymous namespace)::dw_sum_kernel<64>(int)"
    # a small upload copy first, then the 4 MiB calibration copy: its counter
    # reads half the bytes for FETCH_SIZE and all of them for WRITE_SIZE
    # two calls of each kind
    _csv(tmp_path / "f.csv", "FETCH_SIZE", [(copy, 1.0), (copy, 2048.0), (fwd, 100.0), (bwd, 300.0),
                                           (dws, 50.0), (fwd, 100.0), (bwd, 300.0), (dws, 50.0)])
    _csv(tmp_path / "w.csv", "WRITE_SIZE", [(copy, 2.0), (copy, 4096.0), (fwd, 10.0), (bwd, 200.0),
                                           (dws, 5.0), (fwd, 10.0), (bwd, 200.0), (dws, 5.0)])
    rec = profiling.traffic_record(str(tmp_path / "f.csv"), str(tmp_path / "w.csv"), "wl", 4, "cmd",
                                   calls=2)
    assert rec["copy_calibration"]["fetch_scale"] == 2.0
    assert rec["copy_calibration"]["write_scale"] == 1.0
    assert rec["kernels"]["fwd_med_kernel<64, 64>"]["fetch_bytes"] == 200 * 1024
    assert rec["bytes_per_call"]["fwd"] == (200 + 10) * 1024
    assert rec["bytes_per_call"]["bwd"] == (600 + 200 + 100 + 5) * 1024
    assert rec["source_hash"] == profiling.source_hash(sorted(rec["kernels"]))
    # the record depends on its kernels' family and the shared sources only
    assert "scan_med.hip" in rec["source_files"] and "api.cpp" in rec["source_files"]
    assert "scan_wide.hip" not in rec["source_files"]


def test_traffic_counts_every_dispatch_of_a_call(tmp_path):
    # a call that runs its scan and its direction sum in 4 rounds: 3 calls,
    # 12 dispatches of each kernel
    copy = "__amd_rocclr_copyBuffer(char const*, char*)"
    scan = "void gspn::(anonymous namespace)::fwd_wide_kernel<4, 256, 256>(int)"
    summ = "void gspn::(anonymous namespace)::sum_wide_kernel(float)"
    rows_f = [(copy, 512.0)] + [(scan, 100.0), (summ, 40.0)] * 12
    rows_w = [(copy, 1024.0)] + [(scan, 80.0), (summ, 8.0)] * 12
    _csv(tmp_path / "f.csv", "FETCH_SIZE", rows_f)
    _csv(tmp_path / "w.csv", "WRITE_SIZE", rows_w)
    rec = profiling.traffic_record(str(tmp_path / "f.csv"), str(tmp_path / "w.csv"), "wl", 1, "cmd",
                                   calls=3)
    assert rec["kernels"]["sum_wide_kernel"]["dispatches_per_call"] == 4
    assert rec["bytes_per_call"]["fwd"] == 4 * (200 + 80 + 80 + 8) * 1024


def test_traffic_ignored_for_other_sources(tmp_path):
    kern = {"bwd_med_kernel<64, 64, false, false>": {}}
    rec = {"source_hash": profiling.source_hash(sorted(kern)), "kernels": kern,
           "bytes_per_call": {"bwd": 123}}
    p = tmp_path / "t.txt"
    p.write_text(json.dumps(rec))
    assert profiling.load_traffic(str(p), "bwd") == 123
    rec["source_hash"] = "0" * 64
    p.write_text(json.dumps(rec))
    assert profiling.load_traffic(str(p), "bwd") is None
    assert profiling.load_traffic(str(tmp_path / "missing.txt"), "bwd") is None


def test_kernels_map_to_calls():
    assert profiling.call_of("void gspn::(anonymous namespace)::sum_wide_kernel(float)") == "fwd"
    assert profiling.call_of("gspn::(anonymous namespace)::dw_reduce_kernel(float)") == "bwd"
    assert profiling.call_of("__amd_rocclr_copyBuffer") is None


def test_waves_summary_shares(tmp_path):
    bwd = "void gspn::(anonymous namespace)::bwd_med_kernel<64, 64, 0>(int)"
    p = tmp_path / "sq.csv"
    with open(p, "w") as f:
        f.write(HEADER)
        i = 0
        # two dispatches; the shares use the mean of each counter
        for wave, wait, valu in ((1000.0, 600.0, 200.0), (3000.0, 1400.0, 600.0)):
            for name, v in (("SQ_WAVE_CYCLES", wave), ("SQ_WAIT_ANY", wait),
                            ("SQ_ACTIVE_INST_VALU", valu)):
                f.write(f'{i},{i},"Agent 1",1,1,1,64,1,"{bwd}",256,0,0,8,0,16,"{name}",{v},0,1\n')
                i += 1
        f.write(f'{i},{i},"Agent 1",1,1,1,64,1,"__amd_rocclr_copyBuffer",256,0,0,8,0,16,'
                f'"SQ_WAVE_CYCLES",5,0,1\n')
    text = profiling.waves_summary(str(p), str(tmp_path / "o.txt"), "cmd")
    row = [ln for ln in text.splitlines() if ln.startswith("bwd_med_kernel")]
    assert len(row) == 1 and "copyBuffer" not in text
    f = row[0].split()
    # kernel name has spaces: read the numeric columns from the right
    wait, valu = float(f[-6]), float(f[-3])
    assert abs(wait - 0.5) < 1e-3 and abs(valu - 0.2) < 1e-3


def test_relayout_kernels_belong_to_the_call_they_precede(tmp_path):
    # pixel-major calls: the weight re-layout precedes the forward scan; the
    # weight and lambda/u re-layouts precede the backward scan
    copy = "__amd_rocclr_copyBuffer(char const*, char*)"
    rel = "void gspn::(anonymous namespace)::to_blocked_kernel<64>(int)"
    fwd = "void gspn::(anonymous namespace)::fwd_pm_kernel<64>(int)"
    bwd = "void gspn::(anonymous namespace)::bwd_med_kernel<64, 64, 1>(int)"
    flush = "void at::native::reduce_kernel<512, 1>(int)"
    step = [(flush, 999.0), (rel, 10.0), (fwd, 100.0), (flush, 999.0), (rel, 10.0), (rel, 20.0),
            (rel, 20.0), (bwd, 300.0)]
    _csv(tmp_path / "f.csv", "FETCH_SIZE", [(copy, 2048.0)] + step * 2)
    _csv(tmp_path / "w.csv", "WRITE_SIZE", [(copy, 4096.0)] + step * 2)
    rec = profiling.traffic_record(str(tmp_path / "f.csv"), str(tmp_path / "w.csv"), "wl", 4, "cmd",
                                   calls=2)
    assert rec["kernels"]["to_blocked_kernel<64> [fwd]"]["dispatches_per_call"] == 1
    assert rec["kernels"]["to_blocked_kernel<64> [bwd]"]["dispatches_per_call"] == 3
    assert rec["bytes_per_call"]["fwd"] == (2 * 10 + 10 + 2 * 100 + 100) * 1024
    assert rec["bytes_per_call"]["bwd"] == (2 * 50 + 50 + 2 * 300 + 300) * 1024
    assert "scan_pm.hip" in rec["source_files"]


def test_normalization_kernels_belong_to_their_calls(tmp_path):
    # _norm calls: the weights are formed at the start of each call; the
    # logits' gradient ends the backward (it follows the backward's scans and
    # precedes the next step's forward, which forms its weights again)
    copy = "__amd_rocclr_copyBuffer(char const*, char*)"
    norm = "void gspn::(anonymous namespace)::norm_pm_kernel<unsigned short>(int)"
    fwd = "void gspn::(anonymous namespace)::fwd_pm_kernel<64>(int)"
    bwd = "void gspn::(anonymous namespace)::bwd_med_kernel<64, 64, 1>(int)"
    dws = "void gspn::(anonymous namespace)::dw_sum_pm_kernel<64>(int)"
    flush = "void at::native::reduce_kernel<512, 1>(int)"
    step = [(flush, 999.0), (norm, 5.0), (fwd, 100.0), (norm, 7.0), (bwd, 300.0), (dws, 30.0),
            (norm, 11.0)]
    _csv(tmp_path / "f.csv", "FETCH_SIZE", [(copy, 2048.0)] + step * 2)
    _csv(tmp_path / "w.csv", "WRITE_SIZE", [(copy, 4096.0)] + step * 2)
    rec = profiling.traffic_record(str(tmp_path / "f.csv"), str(tmp_path / "w.csv"), "wl", 4, "cmd",
                                   calls=2)
    assert rec["kernels"]["norm_pm_kernel<unsigned short> [fwd]"]["dispatches_per_call"] == 1
    assert rec["kernels"]["norm_pm_kernel<unsigned short> [bwd]"]["dispatches_per_call"] == 2
    assert rec["bytes_per_call"]["fwd"] == (2 * 105 + 105) * 1024
    assert rec["bytes_per_call"]["bwd"] == (2 * 348 + 348) * 1024
    assert "scan_norm.hip" in rec["source_files"]


def test_kernels_after_the_last_scan_belong_to_its_call(tmp_path):
    # one channel per group: the horizontal weight gradients leave the
    # backward's scan in the blocked order and are turned pixel-major by a
    # re-layout launch that ends the backward; the next step's forward starts
    # with the same kind of launch
    copy = "__amd_rocclr_copyBuffer(char const*, char*)"
    rel = "void gspn::(anonymous namespace)::pieces_kernel(int)"
    fwd = "void gspn::(anonymous namespace)::fwd_pm_kernel<64>(int)"
    bwd = "void gspn::(anonymous namespace)::bwd_med_kernel<64, 64, 1>(int)"
    flush = "void at::native::reduce_kernel<512, 1>(int)"
    step = [(flush, 999.0), (rel, 3.0), (fwd, 100.0), (bwd, 300.0), (rel, 20.0)]
    _csv(tmp_path / "f.csv", "FETCH_SIZE", [(copy, 2048.0)] + step * 3)
    _csv(tmp_path / "w.csv", "WRITE_SIZE", [(copy, 4096.0)] + step * 3)
    rec = profiling.traffic_record(str(tmp_path / "f.csv"), str(tmp_path / "w.csv"), "wl", 4, "cmd",
                                   calls=3)
    assert rec["kernels"]["pieces_kernel [fwd]"]["dispatches_per_call"] == 1
    assert rec["kernels"]["pieces_kernel [bwd]"]["dispatches_per_call"] == 1
    assert rec["bytes_per_call"]["fwd"] == (2 * 103 + 103) * 1024
    assert rec["bytes_per_call"]["bwd"] == (2 * 320 + 320) * 1024
