"""CPU: the rocprofv3 counter summaries (paper_1907_02154_amd.traffic) on small
synthetic counter-run directories."""
import csv
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
K1 = "void miconv::(anonymous namespace)::igemm_wave_f32_kernel<1, 1, 8, 1, 1>(miconv::ConvArgs)"
K2 = "miconv::(anonymous namespace)::splitk_reduce_kernel(miconv::ConvArgs)"
COPY = "__amd_rocclr_copyBuffer"


def run_dir(tmp, name, rows):
    d = os.path.join(tmp, name, "host", "1")
    os.makedirs(d)
    with open(os.path.join(d, "run_counter_collection.csv"), "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=["Kernel_Name", "Counter_Name", "Counter_Value"])
        w.writeheader()
        for k, c, v in rows:
            w.writerow(dict(Kernel_Name=k, Counter_Name=c, Counter_Value=v))
    return os.path.join(tmp, name)


def traffic(*args):
    r = subprocess.run([sys.executable, "-m", "paper_1907_02154_amd.traffic", *args], cwd=ROOT,
                       capture_output=True, text=True, check=True)
    return r.stdout


def test_fetch_write_calibrated(tmp_path):
    t = str(tmp_path)
    fetch = run_dir(t, "f", [(K1, "FETCH_SIZE", 10), (K1, "FETCH_SIZE", 30), (K2, "FETCH_SIZE", 4)])
    write = run_dir(t, "w", [(K1, "WRITE_SIZE", 8), (K1, "WRITE_SIZE", 8), (K2, "WRITE_SIZE", 2)])
    # a 1 MiB copy whose counters read 512 KiB fetched and 1024 KiB written: scales 2 and 1
    cf = run_dir(t, "cf", [(COPY, "FETCH_SIZE", 512)])
    cw = run_dir(t, "cw", [(COPY, "WRITE_SIZE", 1024)])
    out = traffic("--fetch", fetch, "--write", write, "--copy-fetch", cf, "--copy-write", cw,
                  "--copy-bytes", str(1 << 20))
    rows = {l.split("\t")[0]: l.split("\t") for l in out.splitlines() if not l.startswith("#")}
    wave = rows["igemm_wave_f32_kernel<1, 1, 8, 1, 1>"]
    assert wave[2] == str(20 * 1024 * 2) and wave[3] == str(8 * 1024) and wave[6] == "2"
    red = rows["splitk_reduce_kernel"]
    assert red[2] == str(4 * 1024 * 2) and red[3] == str(2 * 1024)
    assert len(wave[1]) == 12    # SHA-1 prefix of conv_wave_f32.hip


def test_counter_means_filtered(tmp_path):
    t = str(tmp_path)
    a = run_dir(t, "a", [(K1, "SQ_INSTS_MFMA", 100), (K1, "SQ_INSTS_MFMA", 300), (K2, "SQ_INSTS_MFMA", 7)])
    b = run_dir(t, "b", [(K1, "GRBM_GUI_ACTIVE", 50), (K1, "GRBM_GUI_ACTIVE", 70)])
    out = traffic("--counters", a, b, "--match", "wave")
    assert "splitk_reduce" not in out
    lines = out.splitlines()
    assert lines[0].startswith("igemm_wave_f32_kernel<1, 1, 8, 1, 1>\tsource_sha1 ") and lines[0].endswith(
        "dispatches 2")
    assert "\tGRBM_GUI_ACTIVE\t60.0" in lines and "\tSQ_INSTS_MFMA\t200.0" in lines
