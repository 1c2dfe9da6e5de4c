"""The packed weight layout on the host: the library's own packing plan
(csrc/kl_layout.h: geometry, packing jobs, row maps and the per-chunk body
the packing kernel runs) packs seeded matrices, and every packed element is
read back the way the kernel's consumers interpret it (RoPE pairs, gate/up
interleave, O projection per query head, down projection per column block,
LM head padding).  CPU only."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_pack_unpack_round_trip(tmp_path):
    gxx = shutil.which("g++")
    if gxx is None:
        pytest.skip("g++ not available")
    exe = str(tmp_path / "pack_roundtrip")
    subprocess.run([gxx, "-std=c++17", "-O2", "-DKL_HD=",
                    "-I", os.path.join(ROOT, "paper_2410_23668_amd", "csrc"),
                    "-I", os.path.join(ROOT, "include"),
                    "-o", exe, os.path.join(ROOT, "tests", "cpu", "pack_roundtrip.cpp")],
                   check=True)
    r = subprocess.run([exe], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "pack round trip OK" in r.stdout
