"""Host-side parts of bench.py, on the CPU: the one-GPU guard, the count of
algorithmic bytes (inputs read once, state read and written, outputs
written: the rows of Sec. 3.1 and Alg. 2 the step touches), and the rule that
counter-measured traffic is reported only for the kernel source it was
measured on."""
import os
import subprocess
import sys

import pytest

import bench
from synth.configs import BY_NAME

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.mark.parametrize("argv,env", [(["--gpus", "2"], {}), (["--gpus", "8"], {}), ([], {"WORLD_SIZE": "2"})])
def test_more_than_one_gpu_is_refused_with_a_message(argv, env):
    e = dict(os.environ, **env)
    p = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), *argv], env=e, capture_output=True,
                       text=True, timeout=60)
    assert p.returncode == 2
    assert "one GPU" in p.stderr
    assert p.stdout == ""


def test_algorithmic_bytes_of_a_hand_sized_step():
    # c0 shapes (Adagrad, D = 16, P = 65,536, N = 20,480) with hand-picked counts
    w = BY_NAME["c0"]
    dense, sparse = bench.algorithmic_bytes(w, K_eff=3, N_act=15_360, U=5_000, U_act=4_000, id_tag=False)
    assert dense == 3 * 65_536 * 4 + 4 * 65_536 * 4 == 1_835_008
    # IDs 8 B each, kept rows, touched rows with their accumulator read and
    # written, and per distinct ID its value, offset, c_r and W_r
    assert sparse == 163_840 + 983_040 + 1_024_000 + 120_000 == 2_290_880
    _, tagged = bench.algorithmic_bytes(w, K_eff=3, N_act=15_360, U=5_000, U_act=4_000, id_tag=True)
    assert tagged - sparse == 5_000 * 4 + 4_000 * 4   # tags read for every ID, written for the touched ones


def test_algorithmic_bytes_with_adam_count_two_slots():
    w = BY_NAME["c3"]
    dense, sparse = bench.algorithmic_bytes(w, K_eff=0, N_act=0, U=0, U_act=1, id_tag=False)
    assert dense == 6 * w.P * 4          # parameters, m and v, each read and written
    assert sparse == w.N * 8 + 6 * w.D * 4


def test_algorithmic_bytes_of_the_recorded_c4_step():
    # the realised counts of a c4 run and the step bytes that run reported
    w = BY_NAME["c4"]
    dense, sparse = bench.algorithmic_bytes(w, K_eff=245, N_act=62_720_000, U=8_197_113, U_act=7_911_716,
                                            id_tag=False)
    assert dense == 15_936_000_000
    assert dense + sparse == 28_735_977_304


def test_traffic_is_reported_only_for_the_source_it_was_measured_on(monkeypatch):
    key = "aggregate_dense_kernel<1, false, 16>"
    t = bench.measured_traffic(key, "c4")
    assert t is not None and abs(t - 15_936_000_000) / 15_936_000_000 < 1e-3
    assert bench.measured_traffic(key, "c2") is None          # never measured there
    monkeypatch.setattr(bench, "kernel_source_sha", lambda path: "0" * 16)
    assert bench.measured_traffic(key, "c4") is None          # the kernel changed since
