"""Host logic of the rocprofv3 summary tool on small synthetic counter files."""
import csv
import json

from paper_2310_08152_amd import rocprof_summary as R

FIELDS = ["Dispatch_Id", "Grid_Size", "Kernel_Name", "Counter_Name", "Counter_Value",
          "Start_Timestamp", "End_Timestamp"]


def write_csv(path, rows):
    with open(path, "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=FIELDS)
        w.writeheader()
        for r in rows:
            w.writerow(dict(zip(FIELDS, r)))


def test_traffic_calibration(tmp_path):
    # the copy kernel moves 1 MiB each way; FETCH_SIZE reads half of it, WRITE_SIZE all of it
    fetch, write, out = tmp_path / "f.csv", tmp_path / "w.csv", tmp_path / "o.json"
    write_csv(fetch, [(1, 4096, "copyBuffer", "FETCH_SIZE", 512.0, 0, 10),
                      (2, 256, "my_kernel", "FETCH_SIZE", 100.0, 20, 30),
                      (3, 256, "my_kernel", "FETCH_SIZE", 300.0, 40, 50)])
    write_csv(write, [(1, 4096, "copyBuffer", "WRITE_SIZE", 1024.0, 0, 10),
                      (2, 256, "my_kernel", "WRITE_SIZE", 50.0, 20, 30),
                      (3, 256, "my_kernel", "WRITE_SIZE", 50.0, 40, 50)])
    R.main(["traffic", str(fetch), str(write), str(out), "--workload", "w", "--kernel",
            "my_kernel", "--cal-kernel", "copyBuffer", "--cal-bytes", str(1 << 20),
            "--sources", "paper_2310_08152_amd/rocprof_summary.py",
            "--command-fetch", "cf", "--command-write", "cw"])
    d = json.load(open(out))
    assert d["calibration"]["fetch_factor"] == 2.0 and d["calibration"]["write_factor"] == 1.0
    k = d["kernels"]["my_kernel"]
    assert k["dispatches"] == 2
    assert k["hbm_bytes"] == 200.0 * 1024 * 2.0 + 50.0 * 1024


def test_pmc_mfma_share_and_flops(tmp_path):
    # one dispatch of 1 ms on 8 XCDs at 2 GHz: 2e6 busy clocks per XCD; the matrix
    # cores of all 1024 SIMDs busy a quarter of them; 1000 MFMA instructions of 64 MOPS
    a, b, out = tmp_path / "a.csv", tmp_path / "b.csv", tmp_path / "o.md"
    t0, t1 = 1_000_000, 2_000_000
    busy = 0.25 * 1024 * 2e6
    write_csv(a, [(7, 1, "k_attn<80>", "GRBM_GUI_ACTIVE", 8 * 2e6, t0, t1),
                  (7, 1, "k_attn<80>", "SQ_VALU_MFMA_BUSY_CYCLES", busy, t0, t1),
                  (7, 1, "k_attn<80>", "SQ_INSTS_MFMA", busy / 32, t0, t1),
                  (7, 1, "k_attn<80>", "SQ_INSTS_VALU_MFMA_MOPS_BF16", 64 * busy / 32, t0, t1),
                  (7, 1, "k_attn<80>", "SQ_WAVES", 100.0, t0, t1),
                  (7, 1, "k_attn<80>", "SQ_WAVE_CYCLES", 1000.0, t0, t1),
                  (8, 1, "other", "SQ_WAVES", 5.0, t0, t1)])
    write_csv(b, [(7, 1, "k_attn<80>", "SQ_INSTS_VALU", 500.0, t0, t1 + 1000),
                  (7, 1, "k_attn<80>", "SQ_WAIT_ANY", 400.0, t0, t1 + 1000)])
    js = tmp_path / "o.json"
    R.main(["pmc", str(out), "t", "--csv", str(a), "--csv", str(b), "--command", "c",
            "--kernel", "k_attn", "--json", str(js), "--workload", "w",
            "--sources", "paper_2310_08152_amd/rocprof_summary.py"])
    d = json.load(open(js))
    assert d["workload"] == "w" and len(d["sources_hash"]) == 16
    assert d["kernels"]["k_attn"]["mfma_busy"] == 0.25
    text = open(out).read()
    row = [ln for ln in text.splitlines() if ln.startswith("| `k_attn`")][0].split("|")
    clock, share, tflops = float(row[4]), float(row[5]), float(row[6])
    assert clock == 2.0 and share == 0.25
    # 64 MOPS x 512 flops per instruction, over 1 ms of the pass that counted them
    assert abs(tflops - 512 * 64 * busy / 32 / 1e-3 / 1e12) < 0.05
    assert "VALU 5" in text and "WAIT_ANY 0.400" in text
    assert "MFMA busy clocks per MFMA instruction: 32.00" in text
