"""The NS GEMM tile schedules (csrc/gemm_schedule.h, plain host C++) built with g++ and checked on the
CPU: every tile of every problem exactly once (every K range of a split Gram tile once), whole rounds
of XCD groups, the deal's balance and determinism, on random launches and on the owner shares' own
launches; and the Gram launches' K splits on hand-worked cases, with and without the partial-tile
budget."""
import os
import subprocess
import tempfile

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_schedules_cover_every_tile_once():
    with tempfile.TemporaryDirectory() as d:
        exe = os.path.join(d, "schedule_check")
        subprocess.run(["g++", "-O1", "-std=c++17", "-Wall", "-Werror",
                        "-I", os.path.join(ROOT, "paper_2607_05895_amd", "csrc"),
                        os.path.join(ROOT, "tests", "cpp", "schedule_check.cpp"), "-o", exe], check=True)
        res = subprocess.run([exe], capture_output=True, text=True, timeout=120)
    print(res.stdout)
    assert res.returncode == 0, res.stdout + res.stderr
    assert "schedule check ok" in res.stdout
