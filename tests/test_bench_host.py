"""Host-side pieces of bench.py: the algorithmic byte and MFMA flop counts
against hand-counted closed forms, the committed counter summaries' source
check, and the one-GPU guard."""

import os
import subprocess
import sys

import pytest

import bench
from workload import get_config


def _cfg():
    # 2 layers, 4 query / 2 KV heads, d=64, two prompts of 40 and 64 tokens, m=2.
    return get_config("tiny_f32").with_(layers=2, prompt_lens=(40, 64), samples_per_prompt=4, slots_per_prompt=2)


def test_algorithmic_bytes_closed_form():
    cfg = _cfg()
    # Step 0: prompt 0 slot 0 at t=1, prompt 1 slot 1 at t=3.  Step 1: only prompt 1 slot 0 at t=2.
    log = [[(0, 0, 1), None, None, (1, 2, 3)], [None, None, (1, 0, 2), None]]
    kvrow = 2 * 64 * 4
    qo = 4 * 64 * (4 + 4)
    step0 = 2 * 40 * kvrow + 2 * 64 * kvrow + (2 * 0 * kvrow + 4 * kvrow + qo) + (2 * 2 * kvrow + 4 * kvrow + qo)
    step1 = 2 * 64 * kvrow + (2 * 1 * kvrow + 4 * kvrow + qo)
    assert bench.algorithmic_bytes(cfg, log) == 2 * (step0 + step1)
    # A 1-byte cache shrinks only the stored K/V terms: the caller's new rows stay 4 bytes.
    kv8 = 2 * 64 * 1
    step0_8 = 2 * 40 * kv8 + 2 * 64 * kv8 + (0 + 2 * kvrow + 2 * kv8 + qo) + (2 * 2 * kv8 + 2 * kvrow + 2 * kv8 + qo)
    step1_8 = 2 * 64 * kv8 + (2 * 1 * kv8 + 2 * kvrow + 2 * kv8 + qo)
    assert bench.algorithmic_bytes(cfg, log, kv_bytes=1) == 2 * (step0_8 + step1_8)


def test_mfma_flops_closed_form():
    cfg = _cfg()  # m * hpk = 4 rows -> one 16-row tile; prompts padded to 64 and 64 tokens
    log = [[(0, 0, 1), None, None, (1, 2, 3)], [None, None, (1, 0, 2), None], [None] * 4]
    per = [4 * 16 * 64 * 64 * 2, 4 * 16 * 64 * 64 * 2]
    assert bench.mfma_flops(cfg, log) == 2 * (per[0] + per[1] + per[1])
    big = get_config("qwen3_1p7b_g64")
    one = [[(0, 0, 1)] + [None] * 15]
    assert bench.mfma_flops(big, one) == 28 * 4 * 32 * 2048 * 128 * 8


def test_summaries_follow_kernel_source(tmp_path, monkeypatch):
    pattern = tmp_path / "t_{workload}.txt"
    (tmp_path / "t_w.txt").write_text(f"# header = ignored\nkernel_source_sha256 = {bench.kernel_source_hash()}\n"
                                      "traffic_bytes_per_launch = 123\n")
    monkeypatch.setattr(bench, "TRAFFIC_FILE", str(pattern))
    assert bench.read_traffic("w") == 123.0
    (tmp_path / "t_w.txt").write_text("kernel_source_sha256 = 00\ntraffic_bytes_per_launch = 123\n")
    assert bench.read_traffic("w") is None
    assert bench.read_traffic("absent") is None


@pytest.mark.parametrize("name", ["traffic", "mfma"])
def test_committed_summaries_parse(name):
    path = (bench.TRAFFIC_FILE if name == "traffic" else bench.MFMA_FILE).format(workload="qwen3_1p7b_g64")
    assert os.path.exists(path)
    kv = {}
    for ln in open(path):
        if "=" in ln and not ln.startswith("#"):
            k, v = ln.split("=", 1)
            kv[k.strip()] = v.strip()
    assert len(kv["kernel_source_sha256"]) == 64
    if name == "mfma":
        assert kv["mfma_flops_per_launch"] == kv["expected_mfma_flops_per_launch"]


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, bench.__file__, "--gpus", "2"], capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr


def test_calibration_library_exports():
    import ctypes

    assert os.path.exists(bench.CALIB_LIB), "build the libraries first (python -m paper_2506_22950_amd.build)"
    lib = ctypes.CDLL(bench.CALIB_LIB)
    fn = lib.infs_calib_stream_read
    fn.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p]
    fn.restype = ctypes.c_int
    # Argument errors are refused on the host, before any launch.
    assert fn(None, 1 << 20, 256, None, None) != 0
    assert fn(ctypes.c_void_p(256), 1000, 256, None, ctypes.c_void_p(256)) != 0
    assert fn(ctypes.c_void_p(8), 1 << 20, 256, None, ctypes.c_void_p(256)) != 0
