"""Host-side logic on the CPU: the benchmark's one-GPU contract and the work
and byte models its roofline figures use."""
import os
import subprocess
import sys

import pytest

from paper_2603_14806_amd import perf

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.mark.parametrize("n", [2, 8])
def test_bench_refuses_more_than_one_gpu(n):
    """bench.py --gpus N > 1 exits with a message before touching a GPU."""
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", str(n)],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU only" in r.stderr
    assert r.stdout == ""


def test_flop_model_matches_its_definition():
    """Per direction: projections 2 N^2 c_z 4c, contraction 2 N^3 c, epilogue
    2 N^2 (c_z^2 + c_z c); N = 4096, c_z = c = 128 gives the 17.59 TFLOP of
    one contraction."""
    f = perf.flops(4096)
    assert f["contract"] == 2 * 4096 ** 3 * 128
    assert abs(f["contract"] / 1e12 - 17.592) < 1e-3
    assert f["project"] == 2 * 4096 ** 2 * 128 * 512
    assert f["epilogue"] == 2 * 4096 ** 2 * (128 * 128 + 128 * 128)
    assert f["total"] == f["project"] + f["contract"] + f["epilogue"]


def test_byte_model_matches_the_tensors_moved():
    """Compulsory bytes per direction at N = 4096: K1 reads z (bf16) and
    writes A, B (bf16); K2 reads A, B and writes C (fp32); K3 reads C and z
    and writes the fp32 output."""
    P = 4096 ** 2
    b = perf.bytes_moved(4096)
    assert b["project"] == P * 128 * 2 + 2 * P * 128 * 2
    assert b["contract"] == 2 * P * 128 * 2 + P * 128 * 4
    assert b["epilogue"] == P * 128 * 4 + P * 128 * 2 + P * 128 * 4
    assert abs(b["epilogue"] / 1e9 - 21.47) < 0.01


def test_backward_model():
    """The saved-forward backward: two N^3 products and 10240 bytes per pair;
    the recomputing one adds a third product and 768 bytes per pair."""
    s = perf.backward_layer_work(4096, recompute=False)
    r = perf.backward_layer_work(4096, recompute=True)
    assert s["mfma_flops"] == 2 * 2 * 4096 ** 3 * 128
    assert r["mfma_flops"] == 3 * 2 * 4096 ** 3 * 128
    per_pair_saved = s["hbm_bytes"] / 4096 ** 2
    per_pair_full = r["hbm_bytes"] / 4096 ** 2
    assert per_pair_full == 10240
    assert per_pair_full - per_pair_saved == 128 * 2 + 2 * 128 * 2
    floor = 1e3 * (s["mfma_flops"] / (perf.PEAK_BF16_TFLOPS * 1e12) + s["hbm_bytes"] / (perf.PEAK_HBM_GBS * 1e9))
    assert abs(s["floor_ms"] - floor) < 1e-9


def test_peaks():
    """Published MI355X peaks the roofline fractions divide by."""
    assert abs(perf.PEAK_BF16_TFLOPS - 256 * 4096 * 2.4e9 / 1e12) < 0.1
    assert perf.PEAK_HBM_GBS == 8000.0
    assert perf.PEAK_LANE_OPS == 256 * 4 * 32 * 2.4e9
    assert abs(perf.PEAK_LANE_OPS / perf.TRIATTN_SLOTS / 1e12 - 9.25) < 0.01
