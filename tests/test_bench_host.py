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
    # bf16, 2 layers, 16 query / 8 KV heads, d=128, prompts of 40 and 64 tokens, m=2:
    # m * hpk = 4 rows -> one 16-row tile; both prompts padded to 64 tokens.
    cfg = get_config("qwen3_1p7b_g64").with_(layers=2, prompt_lens=(40, 64), samples_per_prompt=4,
                                             slots_per_prompt=2)
    log = [[(0, 0, 1), None, None, (1, 2, 3)], [None, None, (1, 0, 2), None], [None] * 4]
    per = [4 * 16 * 64 * 128 * 8, 4 * 16 * 64 * 128 * 8]
    tile = 2 * 16 * 16 * 32
    pair = (2 * 4 + 8 + 1) * tile * 8  # two S^T tiles of 4 k-steps, 8 O^T tiles, the row-sum tile; 8 KV heads
    # responses: t=1 stores nothing (its only token is the newest, folded in apart); t=3 and t=2: one pair
    assert bench.mfma_flops(cfg, log) == 2 * (per[0] + per[1] + pair + per[1] + pair)
    big = get_config("qwen3_1p7b_g64")
    one = [[(0, 0, 1)] + [None] * 15]
    assert bench.mfma_flops(big, one) == 28 * 4 * 32 * 2048 * 128 * 8
    # t=300, chunks of 256: four wavefronts of 64 stored tokens (2 pairs each), then 43 stored tokens
    # (299 minus 256, the newest apart) on the next chunk's first wavefront (2 pairs): 10 pairs
    long = [[(0, 0, 300)] + [None] * 15]
    assert bench.mfma_flops(big, long) - bench.mfma_flops(big, one) == 28 * 10 * pair
    assert bench.mfma_flops(get_config("tiny_f32"), log) == 0  # fp32 contexts issue no MFMA
    # Step launch with 64 work-groups per KV head (8 prefix chunks of 256 tokens): one 300-token
    # response fits the chunks, so the count is the same.  Sixteen of 900 tokens (57 pages) are 64
    # chunks for the chunk plan's 54 response work-groups, so the plan keeps 8 prefix work-groups
    # and cuts each response into 3 pieces of 19 pages for the other 52: wavefronts of 5 pages
    # (80 tokens, 3 pairs) and a last one of 4 pages (2 pairs; in the last piece 51 stored tokens,
    # the newest apart: 2) -- 33 pairs against the chunks' 8 + 8 + 8 + 5 = 29.
    assert bench.mfma_flops(big, long, nj=64) == bench.mfma_flops(big, long)
    many = [[(0, i, 900) for i in range(16)]]
    assert bench.mfma_flops(big, many, nj=64) - bench.mfma_flops(big, many) == 28 * 16 * 4 * pair


def test_launches_per_entry():
    cfg = get_config("qwen3_1p7b_g64")
    log = [[None] * 16] * 5
    assert bench.entry_launches(cfg, log, "decode_step_layers") == 5
    assert bench.entry_launches(cfg, log, "decode_step") == 5 * cfg.layers


def test_summaries_follow_kernel_source(tmp_path, monkeypatch):
    pattern = tmp_path / "t_{kernel}_{workload}.txt"
    (tmp_path / "t_k_w.txt").write_text(f"# header = ignored\nkernel_source_sha256 = {bench.kernel_source_hash()}\n"
                                        "traffic_bytes_per_launch = 123\n")
    monkeypatch.setattr(bench, "TRAFFIC_FILE", str(pattern))
    assert bench.read_traffic("w", "k") == 123.0
    assert bench.read_traffic("w", "other") is None
    (tmp_path / "t_k_w.txt").write_text("kernel_source_sha256 = 00\ntraffic_bytes_per_launch = 123\n")
    assert bench.read_traffic("w", "k") is None
    assert bench.read_traffic("absent", "k") is None


@pytest.mark.parametrize("name", ["traffic", "mfma"])
def test_committed_summaries_parse(name):
    path = (bench.TRAFFIC_FILE if name == "traffic" else bench.MFMA_FILE).format(kernel="layers_kernel",
                                                                               workload="qwen3_1p7b_g64")
    assert os.path.exists(path)
    kv = {}
    for ln in open(path):
        if "=" in ln and not ln.startswith("#"):
            k, v = ln.split("=", 1)
            kv[k.strip()] = v.strip()
    assert len(kv["kernel_source_sha256"]) == 64
    assert kv["kernel"] == "layers_kernel"
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
