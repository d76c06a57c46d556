"""Host-side logic of bench.py (no GPU needed): the one-GPU refusal, the
filter on profiler kernel names, and the copy-calibrated HBM traffic
summaries that feed `roofline.traffic`."""
import csv
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402


def test_refuses_more_than_one_gpu():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert r.stdout == ""
    assert "one GPU" in r.stderr


def test_headline_instance_filter():
    solve_bf16 = "_ZN2ea12_GLOBAL__N_112solve_kernelIDF16bLi128ELi2EEEvNS_7TauArgsE"
    solve_f32 = "_ZN2ea12_GLOBAL__N_112solve_kernelIfLi128ELi2EEEvNS_7TauArgsE"
    assert bench.headline_instance(solve_bf16, 128)
    assert not bench.headline_instance(solve_bf16, 64)
    assert not bench.headline_instance(solve_f32, 128)
    dkdv2 = "void ea::(anonymous namespace)::dkdv2_kernel<128, 2>(ea::BwdArgs)"
    assert bench.headline_instance(dkdv2, 128)
    assert not bench.headline_instance(dkdv2, 64)
    assert bench.headline_instance("void ea::fwd_kernel<__bf16, 64, 2, true>(ea::FwdArgs)", 64)


def _counter_csv(path, counter, rows):
    with open(path, "w", newline="") as fh:
        w = csv.DictWriter(fh, fieldnames=["Kernel_Name", "Counter_Name", "Counter_Value"])
        w.writeheader()
        for name, value in rows:
            w.writerow({"Kernel_Name": name, "Counter_Name": counter, "Counter_Value": value})


def test_traffic_summary_round_trip(tmp_path, monkeypatch):
    monkeypatch.setattr(bench, "traffic_path", lambda k: str(tmp_path / ("traffic_%s.md" % k)))
    copy = "__amd_rocclr_copyBuffer"
    solve = "_ZN2ea12_GLOBAL__N_112solve_kernelIDF16bLi128ELi2EEEvNS_7TauArgsE"
    solve_f32 = "_ZN2ea12_GLOBAL__N_112solve_kernelIfLi128ELi2EEEvNS_7TauArgsE"
    fetch = tmp_path / "fetch.csv"
    write = tmp_path / "write.csv"
    # the 1024 MiB copy reads back as half its size and writes its size: the
    # read counter is scaled by 2, the write counter by 1
    _counter_csv(fetch, "FETCH_SIZE", [(copy, 524288), (solve, 1000), (solve, 3000),
                                       (solve_f32, 10 ** 9)])
    _counter_csv(write, "WRITE_SIZE", [(copy, 1048576), (solve, 500), (solve, 500),
                                       (solve_f32, 10 ** 9)])
    bench.write_traffic(str(fetch), str(write), 1024, "cmd", head_dim=128)
    text = (tmp_path / "traffic_tau_solve.md").read_text()
    assert "- hbm_read_bytes_per_launch: %d" % (2000 * 1024 * 2) in text
    assert "- hbm_write_bytes_per_launch: %d" % (500 * 1024) in text
    assert bench.measured_traffic("tau_solve") == 2000 * 1024 * 2 + 500 * 1024
    # kernels without dispatches in the counter files get no summary
    assert not (tmp_path / "traffic_bwd_dq.md").exists()
    # a summary taken on other sources no longer counts
    (tmp_path / "traffic_tau_solve.md").write_text(
        text.replace(bench.sources_sha256("tau_solve"), "0" * 64))
    assert bench.measured_traffic("tau_solve") is None


def test_mfma_summary_round_trip(tmp_path, monkeypatch):
    monkeypatch.setattr(bench, "mfma_path", lambda k: str(tmp_path / ("mfma_%s.md" % k)))
    dkdv = "void ea::(anonymous namespace)::dkdv2_kernel<128, 2>(ea::BwdArgs)"
    dkdv64 = "void ea::(anonymous namespace)::dkdv2_kernel<64, 2>(ea::BwdArgs)"
    pmc = tmp_path / "pmc.csv"
    with open(pmc, "w", newline="") as fh:
        w = csv.DictWriter(fh, fieldnames=["Kernel_Name", "Counter_Name", "Counter_Value"])
        w.writeheader()
        for name, util, mops in ((dkdv, 40.0, 1000), (dkdv, 42.0, 1000), (dkdv64, 90.0, 5)):
            w.writerow({"Kernel_Name": name, "Counter_Name": "MfmaUtil", "Counter_Value": util})
            w.writerow({"Kernel_Name": name, "Counter_Name": "SQ_INSTS_VALU_MFMA_MOPS_BF16",
                        "Counter_Value": mops})
    bench.write_mfma(str(pmc), "cmd", head_dim=128)
    busy, flops = bench.measured_mfma("bwd_dkdv")
    assert abs(busy - 0.41) < 1e-9 and flops == 1000 * 512
    assert bench.measured_mfma("bwd_dq") is None
    text = (tmp_path / "mfma_bwd_dkdv.md").read_text()
    (tmp_path / "mfma_bwd_dkdv.md").write_text(
        text.replace(bench.sources_sha256("bwd_dkdv"), "0" * 64))
    assert bench.measured_mfma("bwd_dkdv") is None
