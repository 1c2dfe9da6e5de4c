"""The cross-workgroup protocols of the step kernel (grid barrier with epoch
recovery, watchdog, tagged hand-offs and their tag ranges), modelled with
host threads and std::atomic under ThreadSanitizer, on the library's own
protocol arithmetic (csrc/kl_sync.h).  CPU only."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "tests", "cpu", "sync_model.cpp")
INC = os.path.join(ROOT, "paper_2410_23668_amd", "csrc")


@pytest.fixture(scope="module")
def model(tmp_path_factory):
    gxx = shutil.which("g++")
    if gxx is None:
        pytest.skip("g++ not available")
    exe = str(tmp_path_factory.mktemp("sync") / "sync_model")
    subprocess.run([gxx, "-std=c++17", "-O1", "-g", "-fsanitize=thread", "-pthread", "-DKL_HD=",
                    "-I", INC, "-o", exe, SRC], check=True)
    return exe


def test_protocols_hold_under_thread_sanitizer(model):
    r = subprocess.run([model], capture_output=True, text=True, timeout=300)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "sync model OK" in r.stdout
    assert "ThreadSanitizer" not in r.stderr


def test_model_catches_a_planted_early_barrier(model):
    # the same check with barrier k waiting for barrier k - 1's target: the
    # model (or ThreadSanitizer) must report it
    r = subprocess.run([model, "--plant-early-barrier"], capture_output=True, text=True,
                       timeout=300)
    assert r.returncode != 0
    assert "FAIL" in r.stderr or "ThreadSanitizer" in r.stderr
