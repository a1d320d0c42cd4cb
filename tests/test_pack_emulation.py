"""Host emulation of the reorder-map packing that the fit launch's packing
blocks run (pack_sigma_words and the search it starts from, cut out of
valuefit.hip): compiled by g++ against the same stand-in for the HIP device
runtime as the bucketed query's emulation (tests/emu), with AddressSanitizer
and UBSan, and run for every thread of a launch over tensors of random sizes
(empty ones, maps of fewer and of at least 16 bits per entry).  Each
tensor's words must equal a direct LSB-first packing of its entries
(section 5.1's reorder map at b = ceil(log2 n) bits).  Host code only: no
GPU."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2102_03112_amd", "csrc")
EMU = os.path.join(ROOT, "tests", "emu")


@pytest.fixture(scope="module")
def emulator(tmp_path_factory):
    gxx = shutil.which("g++")
    if not gxx:
        pytest.skip("g++ not found")
    d = tmp_path_factory.mktemp("pack_emu")
    lines = open(os.path.join(CSRC, "valuefit.hip")).readlines()
    a = next(i for i, l in enumerate(lines) if l.startswith("// Reorder map packing"))
    b = next(i for i, l in enumerate(lines) if i > a and l.startswith("// Standalone value decode"))
    # from the rule line above the section's title to the line before the next
    (d / "ext_pack.inc").write_text("".join(lines[a - 1:b - 1]))
    exe = d / "pack_emu"
    cmd = [gxx, "-std=c++17", "-O1", "-g", "-fsanitize=address,undefined", "-fno-sanitize-recover=undefined",
           f"-I{d}", f"-I{EMU}", f"-I{CSRC}", "-o", str(exe), os.path.join(EMU, "pack_emu.cpp"),
           os.path.join(EMU, "emu_rt.cpp"), "-lpthread"]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-3000:]
    return str(exe)


CASES = [
    # seed, tensors, largest map, threads of the launch
    (1, 1, 70_000, 1024),        # one tensor
    (2, 24, 200_000, 8 * 1024),  # many tensors, several words per thread
    (3, 40, 5_000, 3 * 1024),    # small maps (b < 16 for most), empty tensors
    (4, 7, 1_500_000, 512),      # long walks per thread (b = 21)
]


@pytest.mark.parametrize("seed,nt,max_nv,threads", CASES)
def test_reorder_map_packing_on_the_host(emulator, seed, nt, max_nv, threads):
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0")
    r = subprocess.run([emulator, str(seed), str(nt), str(max_nv), str(threads)], capture_output=True, text=True,
                       timeout=600, env=env)
    assert r.returncode == 0, (r.stdout + r.stderr)[-3000:]
    assert r.stdout.startswith("OK"), r.stdout
