"""bench.py's traffic summary: counter passes (KiB per dispatch) scaled by
the 1 GiB copy calibration into HBM bytes per launch of each kernel class."""
import csv
import json
import os

import bench

FIELDS = ["Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value"]


def write_pass(d, sub, counter, rows):
    os.makedirs(os.path.join(d, sub))
    with open(os.path.join(d, sub, "run_counter_collection.csv"), "w", newline="") as fh:
        w = csv.DictWriter(fh, FIELDS)
        w.writeheader()
        for i, (name, v) in enumerate(rows):
            w.writerow({"Dispatch_Id": i, "Kernel_Name": name, "Counter_Name": counter, "Counter_Value": v})


def test_summarize_traffic(tmp_path, monkeypatch):
    d = str(tmp_path / "pmc")
    out = tmp_path / "traffic_mlp1000_n8.json"
    monkeypatch.setattr(bench, "TRAFFIC_FILE", str(tmp_path / "traffic_{}.json"))
    # the copy reads 2^30 bytes and writes 2^30: FETCH reads half (factor 2), WRITE all (factor 1)
    copy = "void at::native::elementwise_kernel<copy>"
    write_pass(d, "copy_FETCH_SIZE", "FETCH_SIZE", [("fill", 3.0), (copy, (1 << 20) / 2)])
    write_pass(d, "copy_WRITE_SIZE", "WRITE_SIZE", [(copy, 1 << 20)])
    bwd = "void agn::(anonymous namespace)::gemm_f32_dl_bwd_kernel<false>(agn::GemmArgs, agn::GemmArgs)"
    commit = "void agn::(anonymous namespace)::commit_kernel<false>(agn::CommitArgs)"
    write_pass(d, "bench_FETCH_SIZE", "FETCH_SIZE", [(bwd, 100.0), (bwd, 300.0), (commit, 50.0)])
    write_pass(d, "bench_WRITE_SIZE", "WRITE_SIZE", [(bwd, 10.0), (bwd, 30.0), (commit, 5.0)])
    bench.summarize_traffic(d, "mlp1000_n8")
    t = json.loads(out.read_text())
    assert t["workload"] == "mlp1000_n8"
    assert t["kernel_source_sha256"] == bench.kernel_source_digest()
    b = t["classes"]["bwd"]
    assert b["fetch_bytes_per_launch"] == 200.0 * 1024 * 2
    assert b["write_bytes_per_launch"] == 20.0 * 1024
    assert b["hbm_bytes_per_launch"] == 200.0 * 1024 * 2 + 20.0 * 1024
    assert b["launches_sampled"] == 2
    assert t["classes"]["commit"]["hbm_bytes_per_launch"] == 50.0 * 1024 * 2 + 5.0 * 1024
    # stored values apply only to these sources and this workload
    assert bench.stored_traffic("mlp1000_n8", "bwd") == b["hbm_bytes_per_launch"]
    assert bench.stored_traffic("wide_bf16", "bwd") is None


def test_traffic_classes():
    assert bench.traffic_class("agn::(anonymous namespace)::gemm_bf16_dl_bwd_kernel(agn::GemmArgs)") == "bwd"
    assert bench.traffic_class("void agn::(anonymous namespace)::gemm_bf16_dl_kernel<false, false, 3>(x)") == "dw_first"
    assert bench.traffic_class("void agn::(anonymous namespace)::gemm_f32_dl_dw_kernel<true>(x)") == "dw_first"
    assert bench.traffic_class("void agn::(anonymous namespace)::gemm_f32_strip_dw_kernel<false>(agn::GemmArgs)") == "dw_first"
    assert bench.traffic_class("void agn::(anonymous namespace)::gemm_f32_strip_bwd_kernel<false, false>(x)") == "bwd"
    assert bench.traffic_class("void agn::(anonymous namespace)::gemm_bf16_dl_big_kernel<0>(agn::GemmArgs)") == "fwd"
    assert bench.traffic_class("void agn::(anonymous namespace)::gemm_f32_dl_fwd8_kernel<0>(agn::GemmArgs)") == "fwd"
    assert bench.traffic_class("void agn::(anonymous namespace)::head_dw_kernel<10>(x)") == "output_dw"
    assert bench.traffic_class("void agn::(anonymous namespace)::head_kernel<10, 16, false>(x)") == "output"
    assert bench.traffic_class("__amd_rocclr_fillBufferAligned") is None
