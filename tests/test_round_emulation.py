"""The bucketed insert's per-tensor hash rounds (bl_round in bloom.hip, the
kernels' own function compiled for the host with UBSan): over random item
counts below the planned capacity, planned hashes per round and hash counts
up to 32, the rounds the launcher issues insert every hash of a tensor
exactly once, in order, and no round writes more position records than the
tensor's region holds.  Host code only: no GPU."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2102_03112_amd", "csrc")
EMU = os.path.join(ROOT, "tests", "emu")


def test_insert_rounds_on_the_host(tmp_path):
    gxx = shutil.which("g++")
    if not gxx:
        pytest.skip("g++ not found")
    lines = open(os.path.join(CSRC, "bloom.hip")).readlines()
    a = next(i for i, l in enumerate(lines) if l.startswith("// The hashes [*a, *b) of tensor td in round r"))
    b = next(i for i, l in enumerate(lines) if i > a and l.startswith("}"))
    (tmp_path / "ext_round.inc").write_text("".join(lines[a:b + 1]))
    exe = tmp_path / "round_emu"
    cmd = [gxx, "-std=c++17", "-O1", "-g", "-fsanitize=address,undefined", "-fno-sanitize-recover=undefined",
           f"-I{tmp_path}", f"-I{EMU}", f"-I{CSRC}", "-o", str(exe), os.path.join(EMU, "round_emu.cpp"),
           os.path.join(EMU, "emu_rt.cpp"), "-lpthread"]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-3000:]
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0")
    r = subprocess.run([str(exe), "7", "200000"], capture_output=True, text=True, timeout=300, env=env)
    assert r.returncode == 0, (r.stdout + r.stderr)[-3000:]
    assert r.stdout.startswith("OK"), r.stdout
